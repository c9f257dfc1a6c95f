// Pairwise contraction steps of the factorised weights (the greedy two-
// operand order of Sec. 4.2) as batched complex GEMMs on the matrix cores.
//
// A step R[res] = sum_red A[..] B[..] sorts its indices into four classes:
// batch (in A, B and R), M (in A and R only), N (in B and R only) and K (the
// contracted ones).  Each class is flattened in mixed radix (innermost last),
// so the step reads R[bt][m][n] = sum_k A[bt][m][k] B[bt][n][k], and every
// operand is reached through per-class strides: any index order, no
// transposed copies.  A work-group owns a TM x TN tile of one batch entry and
// walks K in stages of 16 through LDS (operands converted to fp32 and
// conjugated on the way in); each complex product is three real
// v_mfma_f32_16x16x4_f32 products (Gauss: ar br, ai bi, (ar + ai)(br + bi)),
// fp32 accumulation.  When both operands are stored in fp16 (the spectra,
// the factors and the fp16 intermediates of the half-precision mode) the
// tiles stay fp16 in LDS and each complex product is four real
// v_mfma_f32_16x16x16_f16 products (ar br - ai bi, ar bi + ai br): the
// products of fp16 values are exact in the fp32 accumulator, so this equals
// the fp32 form up to summation order, with a quarter of its matrix-core time.  Long reductions over few results are split over work-groups
// (split-K); the partial sums are then added in split order by a second
// kernel, so the result does not depend on scheduling.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <climits>
#include <type_traits>
#include <utility>
#include <vector>

#include "fno_device.h"

namespace fno {

namespace {

constexpr int GM_SUB = PW_MAXIDX;  // sub-indices per class
constexpr int GM_TK = 16;          // k per LDS stage, fp32 tiles (four MFMA k-steps)
constexpr int GM_TKH = 16;         // k per LDS stage, fp16 tiles (one MFMA k-step;
                                   // 32 measured slower)
// LDS row stride (elements) of a stage tk deep: 16 rows of a fragment read
// start in disjoint banks
__host__ __device__ constexpr int gm_ls(int tk) { return tk + 4; }
constexpr int GM_KCHUNK = 2048;    // most contracted elements per work-group
enum { CL_BT = 0, CL_M = 1, CL_N = 2, CL_K = 3 };

struct GemmClass {
  int n;                                     // sub-indices, innermost last
  int32_t ext[GM_SUB];
  uint32_t mag[GM_SUB], shr[GM_SUB];           // division by ext (div_magic)
  int64_t sa[GM_SUB], sb[GM_SUB], sr[GM_SUB];  // element strides (0: absent)
  int csub;                                  // last spatial axis (c(t)), -1 none
  int64_t size;
};

struct GemmArgs {
  const void* a;
  const void* b;
  void* out;
  float* part;  // split-K partial sums [splits][Bt][M][N] complex, or null
  int a_elem, b_elem, out_elem, conj_a, conj_b;
  GemmClass c[4];
  int a_kfast, b_kfast;  // staging order: lanes along k (else along m / n)
  int a_vec, b_vec;      // quads of k consecutive and 4-aligned in memory
  int tiles_m, tiles_n, splits, kchunk;
  float scale;
  int Nb;
};

// Offsets of flat index v of class c in A, B and R, and the c(t) factor.
__device__ __forceinline__ void cls_decode(const GemmClass& c, uint32_t v, int Nb, int32_t& oa,
                                           int32_t& ob, int64_t& orr, float& mult) {
  oa = 0;
  ob = 0;
  orr = 0;
  mult = 1.0f;
#pragma unroll
  for (int j = GM_SUB - 1; j >= 0; --j) {
    if (j < c.n) {
      const uint32_t q = fast_div(v, c.mag[j], c.shr[j]);
      const uint32_t d = v - q * (uint32_t)c.ext[j];
      v = q;
      oa += (int32_t)(d * c.sa[j]);
      ob += (int32_t)(d * c.sb[j]);
      orr += (int64_t)d * c.sr[j];
      if (j == c.csub) mult = (d == 0 || 2 * (int)d == Nb) ? 1.0f : 2.0f;
    }
  }
}

__device__ __forceinline__ f2 load_c(const void* p, int elem, int32_t off) {
  if (elem == ELEM_F16) {
    const h2 v = reinterpret_cast<const h2*>(p)[off];
    return f2{(float)v[0], (float)v[1]};
  }
  return reinterpret_cast<const f2*>(p)[off];
}

__device__ __forceinline__ void store_c(void* p, int elem, int64_t off, float re, float im) {
  if (elem == ELEM_F16)
    reinterpret_cast<h2*>(p)[off] = h2{to_h(re), to_h(im)};
  else
    reinterpret_cast<f2*>(p)[off] = f2{re, im};
}

// One operand tile (rows x TK) of a stage into registers.  With 64 or
// more rows a thread takes four consecutive k of one row (four loads) and
// writes them to LDS as one 16-byte (fp32) or 8-byte (fp16) access in the layout the MFMA fragments
// are read in (no bank conflicts); lanes run along the row's k quads
// (KFAST) or along the rows.  Smaller tiles: one element per thread.
template <int ROWS, int TK>
struct TileLoader {
  static constexpr int NE = ROWS * TK / 256;
  static constexpr bool QUAD = ROWS >= 64;
  static constexpr int QPR = TK / 4;  // k quads per row
  static constexpr int LS = gm_ls(TK);
  static_assert(NE >= 1 && (!QUAD || NE % 4 == 0), "tile shape");
  float re[NE], im[NE];
  __device__ __forceinline__ static void slot(bool kfast, int e, int& r, int& kk) {
    const int t = threadIdx.x;
    if (QUAD) {
      const int q = e >> 2, j = e & 3;  // quad q of this thread, element j
      if (kfast) {
        kk = (t % QPR) * 4 + j;
        r = t / QPR + (256 / QPR) * q;
      } else {
        r = t % ROWS;
        kk = (t / ROWS + (256 / ROWS) * q) * 4 + j;
      }
    } else if (kfast) {
      kk = t % TK;
      r = t / TK + (256 / TK) * e;
    } else {
      r = t % ROWS;
      kk = t / ROWS + (256 / ROWS) * e;
    }
  }
  // vec: the four k of a quad are consecutive elements in memory, starting
  // at an offset that is a multiple of four (checked on the host): one 16-byte
  // (fp16) or two 16-byte (fp32) loads per quad instead of four, so the
  // address unit sees a quarter of the instructions.
  __device__ __forceinline__ void load(const void* p, int elem, int conj, bool kfast, bool vec,
                                       int32_t base, const int32_t* roff, const int32_t* koff,
                                       int k0, int klen) {
    if (QUAD && kfast && vec) {
#pragma unroll
      for (int q = 0; q < NE / 4; ++q) {
        int r, kk;
        slot(kfast, 4 * q, r, kk);
        const int32_t ro = roff[r];
        f4 vr = f4zero(), vi = f4zero();
        // klen is a multiple of four, so a quad is either whole or outside
        if (ro >= 0 && k0 + kk < klen) {
          const int32_t off = base + ro + koff[k0 + kk];
          if (elem == ELEM_F16) {
            const h8 v = *reinterpret_cast<const h8*>(reinterpret_cast<const h2*>(p) + off);
            vr = f4{(float)v[0], (float)v[2], (float)v[4], (float)v[6]};
            vi = f4{(float)v[1], (float)v[3], (float)v[5], (float)v[7]};
          } else {
            const f4* fp = reinterpret_cast<const f4*>(reinterpret_cast<const f2*>(p) + off);
            const f4 v0 = fp[0], v1 = fp[1];
            vr = f4{v0[0], v0[2], v1[0], v1[2]};
            vi = f4{v0[1], v0[3], v1[1], v1[3]};
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          re[4 * q + j] = vr[j];
          im[4 * q + j] = conj ? -vi[j] : vi[j];
        }
      }
      return;
    }
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      int r, kk;
      slot(kfast, e, r, kk);
      const int32_t ro = roff[r];
      f2 v = f2{0.0f, 0.0f};
      if (ro >= 0 && k0 + kk < klen) v = load_c(p, elem, base + ro + koff[k0 + kk]);
      re[e] = v[0];
      im[e] = conj ? -v[1] : v[1];
    }
  }
  // ST float: the fp32 tiles; ST _Float16: fp16 tiles (values loaded from
  // fp16 storage, so the conversion back is exact).
  template <typename ST>
  __device__ __forceinline__ void store(bool kfast, ST* lre, ST* lim) const {
    typedef ST v4 __attribute__((ext_vector_type(4)));
    if (QUAD) {
#pragma unroll
      for (int q = 0; q < NE / 4; ++q) {
        int r, kk;
        slot(kfast, 4 * q, r, kk);
        *reinterpret_cast<v4*>(lre + r * LS + kk) =
            v4{(ST)re[4 * q], (ST)re[4 * q + 1], (ST)re[4 * q + 2], (ST)re[4 * q + 3]};
        *reinterpret_cast<v4*>(lim + r * LS + kk) =
            v4{(ST)im[4 * q], (ST)im[4 * q + 1], (ST)im[4 * q + 2], (ST)im[4 * q + 3]};
      }
    } else {
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        int r, kk;
        slot(kfast, e, r, kk);
        lre[r * LS + kk] = (ST)re[e];
        lim[r * LS + kk] = (ST)im[e];
      }
    }
  }
};

// TM x TN result tile per work-group of four waves, WGM of them along M.
// H: both operands stored in fp16 (fp16 tiles, fp16 matrix-core products).
template <int TM, int TN, int WGM, bool H>
__global__ __launch_bounds__(256) void pair_gemm_kernel(GemmArgs g) {
  constexpr int WGN = 4 / WGM;
  constexpr int WM = TM / WGM, WN = TN / WGN;
  constexpr int FM = WM / 16, FN = WN / 16;
  static_assert(FM >= 1 && FN >= 1 && WM % 16 == 0 && WN % 16 == 0, "tile shape");
  typedef typename std::conditional<H, _Float16, float>::type ST;
  constexpr int TK = H ? GM_TKH : GM_TK;
  constexpr int LS = gm_ls(TK);
  __shared__ __align__(16) ST As[2][TM * LS];
  __shared__ __align__(16) ST Bs[2][TN * LS];
  __shared__ int32_t moA[TM], noB[TN];
  __shared__ int64_t moR[TM], noR[TN];
  __shared__ float mmul[TM], nmul[TN];
  __shared__ int32_t koA[GM_KCHUNK], koB[GM_KCHUNK];

  const int tid = threadIdx.x;
  uint32_t bid = blockIdx.x;
  const int tn = (int)(bid % (uint32_t)g.tiles_n);
  bid /= (uint32_t)g.tiles_n;
  const int tm = (int)(bid % (uint32_t)g.tiles_m);
  bid /= (uint32_t)g.tiles_m;
  const uint32_t bt = bid % (uint32_t)g.c[CL_BT].size;
  const int sp = (int)(bid / (uint32_t)g.c[CL_BT].size);
  const int64_t M = g.c[CL_M].size, N = g.c[CL_N].size, K = g.c[CL_K].size;
  const int64_t m0 = (int64_t)tm * TM, n0 = (int64_t)tn * TN;
  const int64_t kb = (int64_t)sp * g.kchunk;
  const int klen = (int)std::min<int64_t>(g.kchunk, K - kb);

  int32_t baA, baB;
  int64_t baR;
  float bmul;
  cls_decode(g.c[CL_BT], bt, g.Nb, baA, baB, baR, bmul);
  for (int i = tid; i < TM; i += 256) {
    int32_t oa = -1, ob;
    int64_t orr = 0;
    float mu = 1.0f;
    if (m0 + i < M) cls_decode(g.c[CL_M], (uint32_t)(m0 + i), g.Nb, oa, ob, orr, mu);
    moA[i] = oa;
    moR[i] = orr;
    mmul[i] = mu;
  }
  for (int i = tid; i < TN; i += 256) {
    int32_t oa, ob = -1;
    int64_t orr = 0;
    float mu = 1.0f;
    if (n0 + i < N) cls_decode(g.c[CL_N], (uint32_t)(n0 + i), g.Nb, oa, ob, orr, mu);
    noB[i] = ob;
    noR[i] = orr;
    nmul[i] = mu;
  }
  for (int i = tid; i < klen; i += 256) {
    int32_t oa, ob;
    int64_t orr;
    float mu;
    cls_decode(g.c[CL_K], (uint32_t)(kb + i), g.Nb, oa, ob, orr, mu);
    koA[i] = oa;
    koB[i] = ob;
  }
  __syncthreads();

  const int lane = tid & 63, wave = tid >> 6, r16 = lane & 15, gq = lane >> 4;
  const int wm = wave % WGM, wn = wave / WGM;
  f4 t1[FM][FN], t2[FM][FN], t3[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) t1[i][j] = t2[i][j] = t3[i][j] = f4zero();

  TileLoader<TM, TK> la;
  TileLoader<TN, TK> lb;
  const bool akf = g.a_kfast != 0, bkf = g.b_kfast != 0;
  const int nst = (klen + TK - 1) / TK;
  const bool avc = g.a_vec != 0, bvc = g.b_vec != 0;
  la.load(g.a, g.a_elem, g.conj_a, akf, avc, baA, moA, koA, 0, klen);
  lb.load(g.b, g.b_elem, g.conj_b, bkf, bvc, baB, noB, koB, 0, klen);
  for (int st = 0; st < nst; ++st) {
    la.store(akf, As[0], As[1]);
    lb.store(bkf, Bs[0], Bs[1]);
    __syncthreads();
    if (st + 1 < nst) {  // next stage in flight during this one's products
      la.load(g.a, g.a_elem, g.conj_a, akf, avc, baA, moA, koA, (st + 1) * TK, klen);
      lb.load(g.b, g.b_elem, g.conj_b, bkf, bvc, baB, noB, koB, (st + 1) * TK, klen);
    }
    if constexpr (H) {
      // lane (r16, gq) holds k = 16 ks + 4 gq .. + 3 of k-step ks (A and B
      // alike), one v_mfma_f32_16x16x16_f16 per real product:
      // t1 = Re = ar br + (-ai) bi, t2 = Im = ar bi + ai br.
#pragma unroll
      for (int ks = 0; ks < TK / 16; ++ks) {
        h4 ar[FM], ai[FM], nai[FM], br[FN], bi[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const int row = wm * WM + i * 16 + r16;
          ar[i] = *reinterpret_cast<const h4*>(&As[0][row * LS + 16 * ks + 4 * gq]);
          ai[i] = *reinterpret_cast<const h4*>(&As[1][row * LS + 16 * ks + 4 * gq]);
          nai[i] = -ai[i];
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = wn * WN + j * 16 + r16;
          br[j] = *reinterpret_cast<const h4*>(&Bs[0][col * LS + 16 * ks + 4 * gq]);
          bi[j] = *reinterpret_cast<const h4*>(&Bs[1][col * LS + 16 * ks + 4 * gq]);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            t1[i][j] = __builtin_amdgcn_mfma_f32_16x16x16f16(ar[i], br[j], t1[i][j], 0, 0, 0);
            t1[i][j] = __builtin_amdgcn_mfma_f32_16x16x16f16(nai[i], bi[j], t1[i][j], 0, 0, 0);
            t2[i][j] = __builtin_amdgcn_mfma_f32_16x16x16f16(ar[i], bi[j], t2[i][j], 0, 0, 0);
            t2[i][j] = __builtin_amdgcn_mfma_f32_16x16x16f16(ai[i], br[j], t2[i][j], 0, 0, 0);
          }
      }
      __syncthreads();
      continue;
    }
    // lane (r16, gq) holds k = 4 gq + s of MFMA k-step s (A and B alike).
    // Complex product with three real products (Gauss): t1 = ar br,
    // t2 = ai bi, t3 = (ar + ai)(br + bi); Re = t1 - t2, Im = t3 - t1 - t2.
    f4 ar[FM], ai[FM], as[FM], br[FN], bi[FN], bs[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = wm * WM + i * 16 + r16;
      ar[i] = *reinterpret_cast<const f4*>(&As[0][row * LS + 4 * gq]);
      ai[i] = *reinterpret_cast<const f4*>(&As[1][row * LS + 4 * gq]);
      as[i] = ar[i] + ai[i];
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = wn * WN + j * 16 + r16;
      br[j] = *reinterpret_cast<const f4*>(&Bs[0][col * LS + 4 * gq]);
      bi[j] = *reinterpret_cast<const f4*>(&Bs[1][col * LS + 4 * gq]);
      bs[j] = br[j] + bi[j];
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          t1[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ar[i][s], br[j][s], t1[i][j], 0, 0, 0);
          t2[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ai[i][s], bi[j][s], t2[i][j], 0, 0, 0);
          t3[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(as[i][s], bs[j][s], t3[i][j], 0, 0, 0);
        }
    __syncthreads();
  }
  f4 cr[FM][FN], ci[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      if constexpr (H) {
        cr[i][j] = t1[i][j];
        ci[i][j] = t2[i][j];
      } else {
        cr[i][j] = t1[i][j] - t2[i][j];
        ci[i][j] = t3[i][j] - t1[i][j] - t2[i][j];
      }
    }

  // D: lane holds rows 4 gq + v, column r16 of each 16 x 16 tile
  const int64_t total = (int64_t)g.c[CL_BT].size * M * N;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int rr = wm * WM + i * 16 + 4 * gq + v;
        const int cc = wn * WN + j * 16 + r16;
        if (m0 + rr >= M || n0 + cc >= N) continue;
        if (g.splits > 1) {
          const int64_t e = ((int64_t)bt * M + m0 + rr) * N + n0 + cc;
          reinterpret_cast<f2*>(g.part)[(int64_t)sp * total + e] = f2{cr[i][j][v], ci[i][j][v]};
        } else {
          const float sc = g.scale * bmul * mmul[rr] * nmul[cc];
          store_c(g.out, g.out_elem, baR + moR[rr] + noR[cc], cr[i][j][v] * sc, ci[i][j][v] * sc);
        }
      }
}

// Split-K: result = scale * sum of the partial sums.  A work-group of up to
// GR_WAVES waves takes 64 results (one per lane); wave w adds its contiguous
// run of splits in order, then the wave sums are added in wave order, so the
// result does not depend on scheduling.
constexpr int GR_WAVES = 16;

__global__ __launch_bounds__(GR_WAVES * 64) void pair_gemm_reduce_kernel(GemmArgs g) {
  __shared__ f2 red[GR_WAVES][64];
  const int64_t M = g.c[CL_M].size, N = g.c[CL_N].size;
  const int64_t total = (int64_t)g.c[CL_BT].size * M * N;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int64_t e = (int64_t)blockIdx.x * 64 + lane;
  const int per = (g.splits + nw - 1) / nw;
  const int s0 = wave * per, s1 = min(g.splits, s0 + per);
  const f2* part = reinterpret_cast<const f2*>(g.part);
  float sr = 0.0f, si = 0.0f;
  if (e < total) {
    int s = s0;
    for (; s + 4 <= s1; s += 4) {  // four loads in flight, added in order
      f2 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = part[(int64_t)(s + u) * total + e];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        sr += v[u][0];
        si += v[u][1];
      }
    }
    for (; s < s1; ++s) {
      const f2 v = part[(int64_t)s * total + e];
      sr += v[0];
      si += v[1];
    }
  }
  red[wave][lane] = f2{sr, si};
  __syncthreads();
  if (wave != 0 || e >= total) return;
  sr = 0.0f;
  si = 0.0f;
  for (int w = 0; w < nw; ++w) {
    sr += red[w][lane][0];
    si += red[w][lane][1];
  }
  const int64_t n = e % N, t = e / N;
  const int64_t m = t % M, bt = t / M;
  int32_t oa, ob;
  int64_t r0, r1, r2;
  float u0, u1, u2;
  cls_decode(g.c[CL_BT], (uint32_t)bt, g.Nb, oa, ob, r0, u0);
  cls_decode(g.c[CL_M], (uint32_t)m, g.Nb, oa, ob, r1, u1);
  cls_decode(g.c[CL_N], (uint32_t)n, g.Nb, oa, ob, r2, u2);
  const float sc = g.scale * u0 * u1 * u2;
  store_c(g.out, g.out_elem, r0 + r1 + r2, sr * sc, si * sc);
}

// Largest element offset an operand reaches through the classes.
int64_t max_offset(const GemmArgs& g, int which) {
  int64_t m = 0;
  for (int c = 0; c < 4; ++c)
    for (int j = 0; j < g.c[c].n; ++j) {
      const int64_t s = which == 0 ? g.c[c].sa[j] : which == 1 ? g.c[c].sb[j] : g.c[c].sr[j];
      m += (int64_t)(g.c[c].ext[j] - 1) * s;
    }
  return m;
}

}  // namespace

// Returns hipErrorNotSupported when the step does not map onto the GEMM
// (an index in the result only, sizes past 32-bit offsets, no room for the
// split-K partial sums) or wastes most of a tile on it; the caller then uses
// the generic kernels.
// ---------------------------------------------------------------------------
// Mode products with a small factor: R(pre, r, post) = s c(t) sum_k
// A(pre, k, post) U(k, r), where the post indices are innermost and
// contiguous in both A and R and U is the small operand (at most 16 columns
// r, indices k and r only); pre, k and r have any strides (pre and k in A,
// pre and r in R).  These are the
// steps that apply u_in or u_out to a spectrum (forward, adjoint and the
// weight gradient's first two).  As a GEMM they have 16 rows at most and a
// long streaming operand; here a work-group takes up to 64 consecutive post
// positions of one pre index, stages the K x 64 block of A in LDS with all
// of its loads issued at once, and each thread forms four consecutive
// positions of one column r in fp32 (VALU).
constexpr int MP_T = 64;
constexpr int MP_PRE = 6;

struct ModeProdArgs {
  const void* a;
  const void* u;
  void* out;
  int a_elem, u_elem, out_elem, conj_a, conj_u;
  int K, R;
  int64_t T, P;              // post positions, pre positions
  int tt;                    // post positions per work-group (T, or 64)
  int n_pre;                 // pre indices (innermost last)
  int64_t pre_ext[MP_PRE], pre_sa[MP_PRE], pre_so[MP_PRE];  // extents, strides in A and R
  int64_t sa_k;              // stride of k in A
  int64_t so_r;              // stride of r in R
  int64_t su_k, su_r;        // element strides of U
  int vec;                   // 16-byte loads of A rows
  float scale;
  int c_ext;                 // extent of the innermost post index carrying c(t) (0: none)
  int Nb;
};

template <typename TA>
__global__ __launch_bounds__(256) void pair_modeprod_kernel(ModeProdArgs m) {
  extern __shared__ __align__(16) unsigned char smem[];
  typedef typename std::conditional<std::is_same<TA, _Float16>::value, h2, f2>::type CA;
  CA* As = reinterpret_cast<CA*>(smem);                   // [K][MP_T]
  f2* Us = reinterpret_cast<f2*>(As + (size_t)m.K * MP_T);  // [K][16]
  const int tid = threadIdx.x;
  const int tt = m.tt;
  const int64_t t0 = (int64_t)blockIdx.x * tt;
  const int64_t p = blockIdx.y;
  int64_t aoff = 0, ooff = 0;
  {
    int64_t q = p;
    for (int j = m.n_pre - 1; j >= 0; --j) {
      const int64_t dgt = q % m.pre_ext[j];
      q /= m.pre_ext[j];
      aoff += dgt * m.pre_sa[j];
      ooff += dgt * m.pre_so[j];
    }
  }
  const CA* a = reinterpret_cast<const CA*>(m.a) + aoff;
  // A block: all loads in flight at once
  constexpr int CPV = 16 / (int)sizeof(CA);  // complex values per 16-byte vector
  if (m.vec) {
    const int vpr = tt / CPV;  // vectors per row
    for (int v = tid; v < m.K * vpr; v += 256) {
      const int k = v / vpr, c = v - (v / vpr) * vpr;
      const int64_t t = t0 + (int64_t)c * CPV;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (t < m.T) val = *reinterpret_cast<const u32x4*>(a + k * m.sa_k + t);
      *reinterpret_cast<u32x4*>(As + k * MP_T + c * CPV) = val;
    }
  } else {
    for (int v = tid; v < m.K * tt; v += 256) {
      const int k = v / tt, c = v - (v / tt) * tt;
      const int64_t t = t0 + c;
      CA val{};
      if (t < m.T) val = a[k * m.sa_k + t];
      As[k * MP_T + c] = val;
    }
  }
  for (int e = tid; e < m.K * 16; e += 256) {
    const int k = e >> 4, r = e & 15;
    f2 uv = f2{0.0f, 0.0f};
    if (r < m.R) {
      const int64_t off = k * m.su_k + r * m.su_r;
      if (m.u_elem == ELEM_F16) {
        const h2 h = reinterpret_cast<const h2*>(m.u)[off];
        uv = f2{(float)h[0], (float)h[1]};
      } else {
        uv = reinterpret_cast<const f2*>(m.u)[off];
      }
      if (m.conj_u) uv[1] = -uv[1];
    }
    Us[e] = uv;
  }
  __syncthreads();
  const int tq = tid & 15, r = tid >> 4;
  if (r >= m.R || 4 * tq >= tt) return;
  float ar[4] = {0.0f, 0.0f, 0.0f, 0.0f}, ai[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  const float sa = m.conj_a ? -1.0f : 1.0f;
  for (int k = 0; k < m.K; ++k) {
    const f2 uv = Us[k * 16 + r];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const CA av = As[k * MP_T + 4 * tq + i];
      const float xr = (float)av[0], xi = sa * (float)av[1];
      ar[i] = __builtin_fmaf(xr, uv[0], __builtin_fmaf(-xi, uv[1], ar[i]));
      ai[i] = __builtin_fmaf(xr, uv[1], __builtin_fmaf(xi, uv[0], ai[i]));
    }
  }
  const int64_t obase = ooff + r * m.so_r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t t = t0 + 4 * tq + i;
    if (t >= m.T || 4 * tq + i >= tt) continue;
    float sc = m.scale;
    if (m.c_ext) {
      const int64_t ci = t % m.c_ext;
      sc *= (ci == 0 || 2 * ci == m.Nb) ? 1.0f : 2.0f;
    }
    if (m.out_elem == ELEM_F16)
      reinterpret_cast<h2*>(m.out)[obase + t] = h2{to_h(ar[i] * sc), to_h(ai[i] * sc)};
    else
      reinterpret_cast<f2*>(m.out)[obase + t] = f2{ar[i] * sc, ai[i] * sc};
  }
}

// Both operands in fp16: the products on the matrix cores, four real
// v_mfma_f32_16x16x16_f16 per complex product (M = r, N = post positions,
// K = k).  The block of A is staged transposed (position-major, k
// contiguous) and split into real and imaginary planes, so that a lane's
// four consecutive k are one 8-byte LDS read; wave w takes positions
// 16 w .. 16 w + 15 of the tile.
__host__ __device__ inline int mp_kp(int K) { return ((K + 15) / 16) * 16 + 4; }

__global__ __launch_bounds__(256) void pair_modeprod_h_kernel(ModeProdArgs m) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int KP = mp_kp(m.K), Kp = KP - 4;
  _Float16* Ar = reinterpret_cast<_Float16*>(smem);  // [MP_T][KP]
  _Float16* Ai = Ar + MP_T * KP;
  _Float16* Ur = Ai + MP_T * KP;                     // [16][KP]
  _Float16* Ui = Ur + 16 * KP;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int tt = m.tt;
  const int64_t t0 = (int64_t)blockIdx.x * tt;
  const int64_t p = blockIdx.y;
  int64_t aoff = 0, ooff = 0;
  {
    int64_t q = p;
    for (int j = m.n_pre - 1; j >= 0; --j) {
      const int64_t dgt = q % m.pre_ext[j];
      q /= m.pre_ext[j];
      aoff += dgt * m.pre_sa[j];
      ooff += dgt * m.pre_so[j];
    }
  }
  const h2* a = reinterpret_cast<const h2*>(m.a) + aoff;
  const _Float16 sa = m.conj_a ? (_Float16)-1.0f : (_Float16)1.0f;
  // zero the padding rows k in [K, Kp) of the A planes
  for (int e = tid; e < MP_T * (Kp - m.K); e += 256) {
    const int t = e / (Kp - m.K), k = m.K + e % (Kp - m.K);
    Ar[t * KP + k] = Ai[t * KP + k] = (_Float16)0.0f;
  }
  if (m.vec) {
    const int vpr = tt / 4;  // 16-byte pieces (four complex values) per row
    for (int v = tid; v < m.K * vpr; v += 256) {
      const int k = v / vpr, c = v - (v / vpr) * vpr;
      const int64_t t = t0 + (int64_t)c * 4;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (t < m.T) val = *reinterpret_cast<const u32x4*>(a + k * m.sa_k + t);
      const h8 hv = w_as_h8(val);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        Ar[(4 * c + i) * KP + k] = hv[2 * i];
        Ai[(4 * c + i) * KP + k] = hv[2 * i + 1] * sa;
      }
    }
  } else {
    for (int v = tid; v < m.K * tt; v += 256) {
      const int k = v / tt, c = v - (v / tt) * tt;
      const int64_t t = t0 + c;
      h2 val = h2{(_Float16)0.0f, (_Float16)0.0f};
      if (t < m.T) val = a[k * m.sa_k + t];
      Ar[c * KP + k] = val[0];
      Ai[c * KP + k] = val[1] * sa;
    }
  }
  // positions of the tile past tt stay unread (their columns are not stored)
  for (int e = tid; e < 16 * Kp; e += 256) {
    const int r = e / Kp, k = e - (e / Kp) * Kp;
    h2 uv = h2{(_Float16)0.0f, (_Float16)0.0f};
    if (r < m.R && k < m.K) uv = reinterpret_cast<const h2*>(m.u)[k * m.su_k + r * m.su_r];
    Ur[r * KP + k] = uv[0];
    Ui[r * KP + k] = m.conj_u ? -uv[1] : uv[1];
  }
  __syncthreads();
  if (16 * wave >= tt) return;
  f4 re = f4zero(), im = f4zero();
  for (int k0 = 0; k0 < Kp; k0 += 16) {
    const h4 ur = *reinterpret_cast<const h4*>(Ur + r16 * KP + k0 + 4 * g);
    const h4 ui = *reinterpret_cast<const h4*>(Ui + r16 * KP + k0 + 4 * g);
    const h4 br = *reinterpret_cast<const h4*>(Ar + (16 * wave + r16) * KP + k0 + 4 * g);
    const h4 bi = *reinterpret_cast<const h4*>(Ai + (16 * wave + r16) * KP + k0 + 4 * g);
    re = __builtin_amdgcn_mfma_f32_16x16x16f16(ur, br, re, 0, 0, 0);
    re = __builtin_amdgcn_mfma_f32_16x16x16f16(-ui, bi, re, 0, 0, 0);
    im = __builtin_amdgcn_mfma_f32_16x16x16f16(ur, bi, im, 0, 0, 0);
    im = __builtin_amdgcn_mfma_f32_16x16x16f16(ui, br, im, 0, 0, 0);
  }
  // D: lane holds r = 4 g + i, position 16 wave + r16
  const int tl = 16 * wave + r16;
  const int64_t t = t0 + tl;
  if (tl >= tt || t >= m.T) return;
  float sc = m.scale;
  if (m.c_ext) {
    const int64_t ci = t % m.c_ext;
    sc *= (ci == 0 || 2 * ci == m.Nb) ? 1.0f : 2.0f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * g + i;
    if (r >= m.R) continue;
    const int64_t o = ooff + r * m.so_r + t;
    if (m.out_elem == ELEM_F16)
      reinterpret_cast<h2*>(m.out)[o] = h2{to_h(re[i] * sc), to_h(im[i] * sc)};
    else
      reinterpret_cast<f2*>(m.out)[o] = f2{re[i] * sc, im[i] * sc};
  }
}

// ---------------------------------------------------------------------------
// Batches of small products with the batch innermost: R(m, n, t) = s c(t)
// sum_k A(m, k, t) B(n, k, t) with one index each for m (<= 16), n (<= 16)
// and k, and the batch indices t innermost and contiguous in A, B and R (the
// weight-gradient steps R = sum_b P Q, Q conj(S), P S of the factorised
// weights, batched over the modes).  As GEMMs these waste most of a tile or
// run a thread per result with each operand element loaded once per result
// that uses it.  Here a work-group stages the A and B rows of BT_T
// consecutive batch positions in LDS (fp32 complex, every load issued
// before the first is waited for), and thread (t, m, half) forms the n
// results of its half of the row.
constexpr int BT_T = 8;
constexpr int BT_ROWS = 1024;  // (M + N) K rows of BT_T values: 64 KiB of LDS
constexpr int BT_LD = BT_ROWS / (256 / BT_T);

struct BtArgs {
  const void* a;
  const void* b;
  void* out;
  int out_elem, conj_a, conj_b;
  int M, N, K;
  int64_t T;
  int64_t sa_m, sa_k, sb_n, sb_k, so_m, so_n;
  float scale;
  int c_ext, Nb;
};

template <typename TE>
__device__ __forceinline__ f2 bt_load(const void* p, int64_t off) {
  if constexpr (sizeof(TE) == 2) {
    const h2 h = reinterpret_cast<const h2*>(p)[off];
    return f2{(float)h[0], (float)h[1]};
  } else {
    return reinterpret_cast<const f2*>(p)[off];
  }
}

template <typename TE>
__global__ __launch_bounds__(256) void pair_bt_kernel(BtArgs g) {
  extern __shared__ __align__(16) unsigned char smem[];
  f2* S = reinterpret_cast<f2*>(smem);  // rows [A: m K + k][B: M K + n K + k] x BT_T
  const int tid = threadIdx.x;
  const int tl = tid % BT_T;
  const int64_t t = (int64_t)blockIdx.x * BT_T + tl;
  const int64_t tc = t < g.T ? t : g.T - 1;  // in-bounds stand-in past the end
  const int arows = g.M * g.K, rows = (g.M + g.N) * g.K;
  const int nld = (rows + 256 / BT_T - 1) / (256 / BT_T);
  // Every load unconditional (rows clamped into range) so that none waits
  // for another.
  f2 v[BT_LD];
#pragma unroll
  for (int i = 0; i < BT_LD; ++i) {
    if (i < nld) {
      const int r = min(tid / BT_T + i * (256 / BT_T), rows - 1);
      const bool isa = r < arows;
      const int rr = isa ? r : r - arows;
      const int q = rr / g.K, k = rr - q * g.K;
      const int64_t off = (isa ? q * g.sa_m + k * g.sa_k : q * g.sb_n + k * g.sb_k) + tc;
      v[i] = bt_load<TE>(isa ? g.a : g.b, off);
    }
  }
#pragma unroll
  for (int i = 0; i < BT_LD; ++i) {
    if (i < nld) {
      const int r = tid / BT_T + i * (256 / BT_T);
      if (r < rows) {
        const int cj = r < arows ? g.conj_a : g.conj_b;
        S[r * BT_T + tl] = f2{v[i][0], cj ? -v[i][1] : v[i][1]};
      }
    }
  }
  __syncthreads();
  const int m = (tid / BT_T) % 16, n0 = (tid / 128) * 8;
  if (m >= g.M || n0 >= g.N || t >= g.T) return;
  const int nn = min(8, g.N - n0);
  float cr[8], ci[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) cr[j] = ci[j] = 0.0f;
  const f2* Ar = S + (size_t)m * g.K * BT_T + tl;
  const f2* Br = S + ((size_t)arows + (size_t)n0 * g.K) * BT_T + tl;
  for (int k = 0; k < g.K; ++k) {
    const f2 av = Ar[k * BT_T];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < nn) {
        const f2 bv = Br[(j * g.K + k) * BT_T];
        cr[j] = __builtin_fmaf(av[0], bv[0], __builtin_fmaf(-av[1], bv[1], cr[j]));
        ci[j] = __builtin_fmaf(av[0], bv[1], __builtin_fmaf(av[1], bv[0], ci[j]));
      }
    }
  }
  float sc = g.scale;
  if (g.c_ext) {
    const int64_t c = t % g.c_ext;
    sc *= (c == 0 || 2 * c == g.Nb) ? 1.0f : 2.0f;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (j >= nn) continue;
    const int64_t o = m * g.so_m + (n0 + j) * g.so_n + t;
    if (g.out_elem == ELEM_F16)
      reinterpret_cast<h2*>(g.out)[o] = h2{to_h(cr[j] * sc), to_h(ci[j] * sc)};
    else
      reinterpret_cast<f2*>(g.out)[o] = f2{cr[j] * sc, ci[j] * sc};
  }
}

// ---------------------------------------------------------------------------
// The three per-mode products of the Tucker weight gradient in one launch:
// with P[b][a][t], Q[b][e][t], S[a][e][t] (fp32 complex, the mode index t
// innermost),
//   R[a][e][t]  = sum_b P[b][a][t] Q[b][e][t],
//   Z1[b][a][t] = sum_e Q[b][e][t] conj(S[a][e][t]),
//   Z2[b][e][t] = s c(t) sum_a P[b][a][t] conj(S[a][e][t]).
// A work-group stages the three operands of TR_T consecutive modes in LDS
// (every load issued before the first is waited for) and its threads form
// the results of those modes, TR_T consecutive modes per result row.
constexpr int TR_T = 8;
constexpr int TR_ROWS = 1024;  // B A + B E + A E rows of TR_T values: 64 KiB of LDS

__global__ __launch_bounds__(256) void tucker_tri_kernel(TriArgs g) {
  extern __shared__ __align__(16) unsigned char smem[];
  f2* L = reinterpret_cast<f2*>(smem);  // rows [P: b A + a][Q: b E + e][S: a E + e] x TR_T
  const f2* gP = reinterpret_cast<const f2*>(g.P);
  const f2* gQ = reinterpret_cast<const f2*>(g.Q);
  const f2* gS = reinterpret_cast<const f2*>(g.S);
  const int tid = threadIdx.x;
  const int tl = tid % TR_T;
  const int64_t t = (int64_t)blockIdx.x * TR_T + tl;
  const int64_t tc = t < g.T ? t : g.T - 1;  // in-bounds stand-in past the end
  const int np = g.B * g.A, nq = g.B * g.E, ns = g.A * g.E;
  const int rows = np + nq + ns;
  constexpr int RPI = 256 / TR_T;  // rows per pass of the work-group
  for (int r0 = 0; r0 < rows; r0 += 8 * RPI) {
    f2 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = min(r0 + tid / TR_T + i * RPI, rows - 1);
      const f2* src = r < np ? gP + (int64_t)r * g.T
                    : r < np + nq ? gQ + (int64_t)(r - np) * g.T
                                  : gS + (int64_t)(r - np - nq) * g.T;
      v[i] = src[tc];
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = r0 + tid / TR_T + i * RPI;
      if (r < rows) L[r * TR_T + tl] = v[i];
    }
  }
  __syncthreads();
  if (t >= g.T) return;
  const f2* Pl = L + tl;
  const f2* Ql = L + (size_t)np * TR_T + tl;
  const f2* Sl = L + (size_t)(np + nq) * TR_T + tl;
  float cz = g.scale;
  if (g.c_ext) {
    const int64_t c = t % g.c_ext;
    cz *= (c == 0 || 2 * c == g.Nb) ? 1.0f : 2.0f;
  }
  const int nres = ns + np + nq;  // R, then Z1 (B A), then Z2 (B E)
  for (int j = tid / TR_T; j < nres; j += RPI) {
    float sr = 0.0f, si = 0.0f;
    if (j < ns) {
      const int a = j / g.E, e = j - (j / g.E) * g.E;
      for (int b = 0; b < g.B; ++b) {
        const f2 p = Pl[(b * g.A + a) * TR_T], q = Ql[(b * g.E + e) * TR_T];
        sr = __builtin_fmaf(p[0], q[0], __builtin_fmaf(-p[1], q[1], sr));
        si = __builtin_fmaf(p[0], q[1], __builtin_fmaf(p[1], q[0], si));
      }
      reinterpret_cast<f2*>(g.R)[((int64_t)a * g.E + e) * g.T + t] = f2{sr, si};
    } else if (j < ns + np) {
      const int k = j - ns, b = k / g.A, a = k - (k / g.A) * g.A;
      for (int e = 0; e < g.E; ++e) {  // q conj(s)
        const f2 q = Ql[(b * g.E + e) * TR_T], sv = Sl[(a * g.E + e) * TR_T];
        sr = __builtin_fmaf(q[0], sv[0], __builtin_fmaf(q[1], sv[1], sr));
        si = __builtin_fmaf(q[1], sv[0], __builtin_fmaf(-q[0], sv[1], si));
      }
      reinterpret_cast<f2*>(g.Z1)[((int64_t)b * g.A + a) * g.T + t] = f2{sr, si};
    } else {
      const int k = j - ns - np, b = k / g.E, e = k - (k / g.E) * g.E;
      for (int a = 0; a < g.A; ++a) {  // p conj(s)
        const f2 p = Pl[(b * g.A + a) * TR_T], sv = Sl[(a * g.E + e) * TR_T];
        sr = __builtin_fmaf(p[0], sv[0], __builtin_fmaf(p[1], sv[1], sr));
        si = __builtin_fmaf(p[1], sv[0], __builtin_fmaf(-p[0], sv[1], si));
      }
      reinterpret_cast<f2*>(g.Z2)[((int64_t)b * g.E + e) * g.T + t] = f2{sr * cz, si * cz};
    }
  }
}

hipError_t launch_tucker_tri(const TriArgs& g, hipStream_t s) {
  if (g.B < 1 || g.A < 1 || g.E < 1 || g.T < 1) return hipErrorInvalidValue;
  const int64_t rows = (int64_t)g.B * g.A + (int64_t)g.B * g.E + (int64_t)g.A * g.E;
  if (rows > TR_ROWS) return hipErrorNotSupported;
  const int64_t blocks = (g.T + TR_T - 1) / TR_T;
  if (blocks > 0x7fffffff) return hipErrorNotSupported;
  const size_t lds = (size_t)rows * TR_T * sizeof(f2);
  hipLaunchKernelGGL(tucker_tri_kernel, dim3((unsigned)blocks), dim3(256), lds, s, g);
  return hipGetLastError();
}

// The batch-innermost form of a step, if it has one (hipErrorNotSupported
// otherwise): the result's innermost indices are carried by both operands
// with the same dense strides, one other result index by each operand alone,
// one contracted index.
hipError_t launch_pair_bt(const PairArgs& p, hipStream_t s) {
  if (p.n_red != 1 || p.a_stride_red[0] == 0 || p.b_stride_red[0] == 0 || p.a_elem != p.b_elem)
    return hipErrorNotSupported;
  int64_t st = 1, T = 1;
  int bs = p.n_out;
  while (bs > 0 && p.a_stride_out[bs - 1] == st && p.b_stride_out[bs - 1] == st) {
    --bs;
    st *= p.out_ext[bs];
    T *= p.out_ext[bs];
  }
  if (bs == p.n_out || bs != 2) return hipErrorNotSupported;
  // the two outer result indices: one in A only (m), one in B only (n)
  int im = -1, in_ = -1;
  for (int k = 0; k < 2; ++k) {
    const bool ina = p.a_stride_out[k] != 0, inb = p.b_stride_out[k] != 0;
    if (ina && !inb) im = k;
    else if (inb && !ina) in_ = k;
  }
  if (im < 0 || in_ < 0) return hipErrorNotSupported;
  const int64_t M = p.out_ext[im], N = p.out_ext[in_], K = p.red_ext[0];
  if (M > 16 || N > 16) return hipErrorNotSupported;
  int c_ext = 0;
  if (p.scale_c_axis >= 0) {
    if (p.scale_c_axis != p.n_out - 1) return hipErrorNotSupported;
    c_ext = (int)p.out_ext[p.n_out - 1];
  }
  BtArgs g{};
  g.a = p.a;
  g.b = p.b;
  g.out = p.out;
  g.out_elem = p.out_elem;
  g.conj_a = p.conj_a;
  g.conj_b = p.conj_b;
  g.M = (int)M;
  g.N = (int)N;
  g.K = (int)K;
  g.T = T;
  g.sa_m = p.a_stride_out[im];
  g.sa_k = p.a_stride_red[0];
  g.sb_n = p.b_stride_out[in_];
  g.sb_k = p.b_stride_red[0];
  // result strides (dense in result order): the two outer indices
  g.so_m = (im == 0 ? p.out_ext[1] : 1) * T;
  g.so_n = (in_ == 0 ? p.out_ext[1] : 1) * T;
  g.scale = p.scale;
  g.c_ext = c_ext;
  g.Nb = p.Nb;
  if ((M + N) * K > BT_ROWS) return hipErrorNotSupported;
  const size_t lds = (size_t)(M + N) * K * BT_T * sizeof(f2);
  const int64_t blocks = (T + BT_T - 1) / BT_T;
  if (blocks > 0x7fffffff) return hipErrorNotSupported;
  auto kern = p.a_elem == ELEM_F16 ? pair_bt_kernel<_Float16> : pair_bt_kernel<float>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), lds, s, g);
  return hipGetLastError();
}

// The mode-product form of a step, if it has one (hipErrorNotSupported
// otherwise): one contracted index k, one result index r carried by the
// smaller operand only (with k), every other result index carried by the
// larger operand only, which is laid out [pre][k][post] densely with the
// result's order of pre and post.
hipError_t launch_pair_modeprod(const PairArgs& p, hipStream_t s) {
  if (p.n_red != 1 || p.a_stride_red[0] == 0 || p.b_stride_red[0] == 0) return hipErrorNotSupported;
  int rpos = -1;
  for (int k = 0; k < p.n_out; ++k) {
    const bool ina = p.a_stride_out[k] != 0, inb = p.b_stride_out[k] != 0;
    if (ina == inb) return hipErrorNotSupported;  // batch-like or absent index
    if (inb) {
      if (rpos >= 0) return hipErrorNotSupported;
      rpos = k;
    }
  }
  if (rpos < 0) return hipErrorNotSupported;
  const int64_t K = p.red_ext[0], R = p.out_ext[rpos];
  if (R > 16 || K < 1) return hipErrorNotSupported;
  // result strides (dense in result order)
  int64_t os[PW_MAXIDX];
  {
    int64_t st = 1;
    for (int k = p.n_out - 1; k >= 0; --k) {
      os[k] = st;
      st *= p.out_ext[k];
    }
  }
  // post: the longest innermost run of result indices that is also
  // innermost and contiguous in A
  int64_t st = 1, T = 1;
  int ps = p.n_out;
  while (ps > 0 && ps - 1 != rpos && p.a_stride_out[ps - 1] == st) {
    --ps;
    st *= p.out_ext[ps];
    T *= p.out_ext[ps];
  }
  if (ps == p.n_out) return hipErrorNotSupported;
  // pre: every other result index but r
  int n_pre = 0;
  int64_t P = 1;
  int64_t pe[PW_MAXIDX], pa[PW_MAXIDX], po[PW_MAXIDX];
  for (int k = 0; k < ps; ++k) {
    if (k == rpos) continue;
    if (n_pre >= MP_PRE) return hipErrorNotSupported;
    pe[n_pre] = p.out_ext[k];
    pa[n_pre] = p.a_stride_out[k];
    po[n_pre] = os[k];
    P *= p.out_ext[k];
    ++n_pre;
  }
  // c(t) only along the innermost post index
  int c_ext = 0;
  if (p.scale_c_axis >= 0) {
    if (p.scale_c_axis != p.n_out - 1) return hipErrorNotSupported;
    c_ext = (int)p.out_ext[p.n_out - 1];
  }
  const bool ah = p.a_elem == ELEM_F16;
  if (K > (ah ? 256 : 128) || P > 65535 || T / MP_T >= 0x7fffffffll) return hipErrorNotSupported;
  ModeProdArgs m{};
  m.a = p.a;
  m.u = p.b;
  m.out = p.out;
  m.a_elem = p.a_elem;
  m.u_elem = p.b_elem;
  m.out_elem = p.out_elem;
  m.conj_a = p.conj_a;
  m.conj_u = p.conj_b;
  m.K = (int)K;
  m.R = (int)R;
  m.T = T;
  m.P = P;
  m.su_k = p.b_stride_red[0];
  m.su_r = p.b_stride_out[rpos];
  m.sa_k = p.a_stride_red[0];
  m.so_r = os[rpos];
  m.n_pre = n_pre;
  for (int k = 0; k < n_pre; ++k) {
    m.pre_ext[k] = pe[k];
    m.pre_sa[k] = pa[k];
    m.pre_so[k] = po[k];
  }
  m.tt = (int)std::min<int64_t>(T, MP_T);
  const int esz = ah ? 4 : 8;  // bytes per complex value of A
  // 16-byte row pieces: every row start (pre and k strides, the tile
  // starts) a multiple of 16 bytes
  bool vec = ((uintptr_t)p.a & 15u) == 0 && (m.tt * esz) % 16 == 0 && (T * esz) % 16 == 0 &&
             (m.sa_k * esz) % 16 == 0;
  for (int k = 0; k < n_pre; ++k) vec = vec && (m.pre_sa[k] * esz) % 16 == 0;
  m.vec = vec;
  m.scale = p.scale;
  m.c_ext = c_ext;
  m.Nb = p.Nb;
  const size_t lds = (size_t)K * MP_T * esz + (size_t)K * 16 * 8;
  dim3 grid((unsigned)((T + m.tt - 1) / m.tt), (unsigned)P), block(256);
  if (ah && p.b_elem == ELEM_F16) {
    const size_t ldsh = (size_t)(2 * MP_T + 2 * 16) * mp_kp((int)K) * 2;
    if (ldsh > 65536) {
      const hipError_t e = hipFuncSetAttribute(
          reinterpret_cast<const void*>(&pair_modeprod_h_kernel),
          hipFuncAttributeMaxDynamicSharedMemorySize, (int)ldsh);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(pair_modeprod_h_kernel, grid, block, ldsh, s, m);
  } else if (ah) {
    if (lds > 65536) {
      const hipError_t e = hipFuncSetAttribute(
          reinterpret_cast<const void*>(&pair_modeprod_kernel<_Float16>),
          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(pair_modeprod_kernel<_Float16>, grid, block, lds, s, m);
  } else {
    if (lds > 65536) {
      const hipError_t e = hipFuncSetAttribute(
          reinterpret_cast<const void*>(&pair_modeprod_kernel<float>),
          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(pair_modeprod_kernel<float>, grid, block, lds, s, m);
  }
  return hipGetLastError();
}

hipError_t launch_pair_gemm(const PairArgs& p, hipStream_t s) {
  GemmArgs g{};
  g.a = p.a;
  g.b = p.b;
  g.out = p.out;
  g.part = reinterpret_cast<float*>(p.part);
  g.a_elem = p.a_elem;
  g.b_elem = p.b_elem;
  g.out_elem = p.out_elem;
  g.conj_a = p.conj_a;
  g.conj_b = p.conj_b;
  g.scale = p.scale;
  g.Nb = p.Nb;
  struct Sub {
    int64_t ext, sa, sb, sr;
    bool c;
  };
  std::vector<Sub> cls[4];
  int64_t rs = 1;
  std::vector<int64_t> res_stride(p.n_out);
  for (int k = p.n_out - 1; k >= 0; --k) {
    res_stride[k] = rs;
    rs *= p.out_ext[k];
  }
  for (int k = 0; k < p.n_out; ++k) {
    const bool ina = p.a_stride_out[k] != 0, inb = p.b_stride_out[k] != 0;
    if (!ina && !inb) return hipErrorNotSupported;
    const int c = ina && inb ? CL_BT : ina ? CL_M : CL_N;
    cls[c].push_back({p.out_ext[k], p.a_stride_out[k], p.b_stride_out[k], res_stride[k],
                      k == p.scale_c_axis});
  }
  for (int k = 0; k < p.n_red; ++k)
    cls[CL_K].push_back({p.red_ext[k], p.a_stride_red[k], p.b_stride_red[k], 0, false});
  // innermost sub-index = smallest stride of the operand that streams along
  // the class (absent indices, stride 0, go outermost)
  auto key = [](int64_t st) { return st == 0 ? INT64_MAX : st; };
  auto min_stride = [&](const std::vector<Sub>& v, bool a) {
    int64_t m = INT64_MAX;
    for (const Sub& u : v) m = std::min(m, key(a ? u.sa : u.sb));
    return m;
  };
  // The class holding the result's contiguous index goes to N: lanes run
  // along N in the D fragments, so each store instruction then writes
  // consecutive elements.  Otherwise the smaller class goes to N.  (The
  // operands swap roles; the product commutes.)
  auto csize = [&](const std::vector<Sub>& v) {
    int64_t z = 1;
    for (const Sub& u : v) z *= u.ext;
    return z;
  };
  auto has_unit = [&](const std::vector<Sub>& v) {
    for (const Sub& u : v)
      if (u.sr == 1) return true;
    return false;
  };
  const bool swap_mn = has_unit(cls[CL_M])   ? true
                       : has_unit(cls[CL_N]) ? false
                                             : csize(cls[CL_N]) > csize(cls[CL_M]);
  if (swap_mn) {
    std::swap(cls[CL_M], cls[CL_N]);
    for (auto& v : cls)
      for (Sub& u : v) std::swap(u.sa, u.sb);
    std::swap(g.a, g.b);
    std::swap(g.a_elem, g.b_elem);
    std::swap(g.conj_a, g.conj_b);
  }
  g.a_kfast = min_stride(cls[CL_K], true) < min_stride(cls[CL_M], true);
  g.b_kfast = min_stride(cls[CL_K], false) < min_stride(cls[CL_N], false);
  auto sort_by = [&](std::vector<Sub>& v, int which) {
    std::stable_sort(v.begin(), v.end(), [&](const Sub& x, const Sub& y) {
      const int64_t sx = which == 0 ? key(x.sa) : which == 1 ? key(x.sb) : key(x.sr);
      const int64_t sy = which == 0 ? key(y.sa) : which == 1 ? key(y.sb) : key(y.sr);
      return sx > sy;
    });
  };
  sort_by(cls[CL_BT], 2);
  sort_by(cls[CL_M], 0);
  sort_by(cls[CL_N], 1);
  sort_by(cls[CL_K], g.a_kfast || !g.b_kfast ? 0 : 1);
  for (int c = 0; c < 4; ++c) {
    if ((int)cls[c].size() > GM_SUB) return hipErrorNotSupported;
    GemmClass& C = g.c[c];
    C.n = (int)cls[c].size();
    C.csub = -1;
    C.size = 1;
    for (int j = 0; j < C.n; ++j) {
      C.ext[j] = (int32_t)cls[c][j].ext;
      div_magic((uint32_t)cls[c][j].ext, &C.mag[j], &C.shr[j]);
      C.sa[j] = cls[c][j].sa;
      C.sb[j] = cls[c][j].sb;
      C.sr[j] = cls[c][j].sr;
      if (cls[c][j].c) C.csub = j;
      C.size *= cls[c][j].ext;
    }
    if (C.size >= ((int64_t)1 << 31)) return hipErrorNotSupported;
  }
  if (max_offset(g, 0) >= ((int64_t)1 << 31) || max_offset(g, 1) >= ((int64_t)1 << 31))
    return hipErrorNotSupported;
  const int64_t M = g.c[CL_M].size, N = g.c[CL_N].size, K = g.c[CL_K].size;
  const int64_t Bt = g.c[CL_BT].size;
  // 16-byte quad loads for an operand staged along k: the innermost
  // contracted sub-index has unit stride in it and an extent that is a
  // multiple of four, and every other stride of it is a multiple of four (so
  // quads start 16-byte aligned; operands are 16-byte aligned)
  auto quad_vec = [&](bool kfast, int which) {
    const GemmClass& ck = g.c[CL_K];
    if (!kfast || ck.n == 0) return 0;
    const int in = ck.n - 1;
    const int64_t s_in = which == 0 ? ck.sa[in] : ck.sb[in];
    if (s_in != 1 || ck.ext[in] % 4 != 0) return 0;
    for (int c = 0; c < 4; ++c)
      for (int j = 0; j < g.c[c].n; ++j) {
        if (c == CL_K && j == in) continue;
        const int64_t st = which == 0 ? g.c[c].sa[j] : g.c[c].sb[j];
        if (st % 4 != 0) return 0;
      }
    return 1;
  };
  g.a_vec = quad_vec(g.a_kfast != 0, 0);
  g.b_vec = quad_vec(g.b_kfast != 0, 1);
  // Elementwise and outer products (K < 4), large batches of tiny dot
  // products, and large batches of small products with short reductions
  // (at most 16 x 16 results and 64 contracted elements per batch entry:
  // most of a 128 x 16 tile would be padding, one stage per work-group)
  // waste the tile: the generic kernels take those.
  if (K < 4 || (M * N < 16 && Bt * M * N > 4096) ||
      (M <= 16 && N <= 16 && K <= 64 && Bt * M * N > 4096))
    return hipErrorNotSupported;
  int cfg, TM, TN;
  if (N <= 16) {
    cfg = 0, TM = 128, TN = 16;
  } else if (N <= 32) {
    cfg = 1, TM = 128, TN = 32;
  } else if (M <= 16) {
    cfg = 3, TM = 16, TN = 128;
  } else if (M <= 32) {
    cfg = 4, TM = 32, TN = 128;
  } else {
    cfg = 2, TM = 64, TN = 64;
  }
  const bool half = g.a_elem == ELEM_F16 && g.b_elem == ELEM_F16;
  const int tk = half ? GM_TKH : GM_TK;
  g.tiles_m = (int)((M + TM - 1) / TM);
  g.tiles_n = (int)((N + TN - 1) / TN);
  const int64_t tiles = (int64_t)g.tiles_m * g.tiles_n * Bt;
  const int64_t nst = (K + tk - 1) / tk;
  const int64_t total = Bt * M * N;
  // split-K: at least enough splits for the per-work-group offset table,
  // more while the tiles alone leave the chip idle (>= 2 stages a split),
  // as many as the partial-sum area holds
  const int64_t need = (K + GM_KCHUNK - 1) / GM_KCHUNK;
  int64_t want = need;
  if (tiles < 512) want = std::max(want, std::min<int64_t>(nst / 2, (1024 + tiles - 1) / tiles));
  const int64_t cap = p.part ? (int64_t)(p.part_cap / (size_t)(total * 8)) : 0;
  if (need > 1 && cap < need) return hipErrorNotSupported;
  const int64_t splits = want > 1 ? std::max(need, std::min(want, cap)) : 1;
  const int64_t kst = (nst + splits - 1) / splits;
  g.kchunk = (int)(kst * tk);
  g.splits = (int)std::max<int64_t>(1, (K + g.kchunk - 1) / g.kchunk);
  const int64_t blocks = tiles * g.splits;
  if (blocks <= 0 || blocks > 0x7fffffffll) return hipErrorNotSupported;
  dim3 grid((unsigned)blocks), block(256);
  if (half) {
    switch (cfg) {
      case 0: hipLaunchKernelGGL((pair_gemm_kernel<128, 16, 4, true>), grid, block, 0, s, g); break;
      case 1: hipLaunchKernelGGL((pair_gemm_kernel<128, 32, 4, true>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((pair_gemm_kernel<16, 128, 1, true>), grid, block, 0, s, g); break;
      case 4: hipLaunchKernelGGL((pair_gemm_kernel<32, 128, 1, true>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((pair_gemm_kernel<64, 64, 2, true>), grid, block, 0, s, g); break;
    }
  } else {
    switch (cfg) {
      case 0: hipLaunchKernelGGL((pair_gemm_kernel<128, 16, 4, false>), grid, block, 0, s, g); break;
      case 1: hipLaunchKernelGGL((pair_gemm_kernel<128, 32, 4, false>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((pair_gemm_kernel<16, 128, 1, false>), grid, block, 0, s, g); break;
      case 4: hipLaunchKernelGGL((pair_gemm_kernel<32, 128, 1, false>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((pair_gemm_kernel<64, 64, 2, false>), grid, block, 0, s, g); break;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.splits == 1) return e;
  dim3 rgrid((unsigned)((total + 63) / 64)), rblock(64 * std::min(GR_WAVES, g.splits));
  hipLaunchKernelGGL(pair_gemm_reduce_kernel, rgrid, rblock, 0, s, g);
  return hipGetLastError();
}

}  // namespace fno
