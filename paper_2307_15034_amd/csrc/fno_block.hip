// The rest of the FNO block (Sec. 2) after the spectral convolution K:
// out = act(W_skip x + b + y) (+ x), with y = K x, and the two backward
// steps around K's backward.  The channel mix is a dense contraction over
// channels at every grid point, so it runs on the matrix cores
// (v_mfma_f32_16x16x32_f16 in fp16 mode, 16x16x4 f32 in fp32 mode); the
// kernels are bound by HBM traffic (each tensor read or written once).
//
//   epi_mix_kernel      out[b][n][p] = act(sum_k W[n][k] in[b][k][p] + add1 + add2 + bias[n])
//                       (+ in[b][n][p]); the forward (in = x, W = W_skip) and the
//                       data gradient (in = g_z, W = W_skip^T, add1 = gx_spec,
//                       add2 = g_out)
//   epi_wgrad_kernel    g_z = g_out act'(z) (written once), partial sums of
//                       g_W[o][i] = sum g_z[o][p] x[i][p] and g_b[o] per work-group
//   epi_reduce_kernel   the partial sums added in a fixed order
//
// Table-free generic kernels cover what the matrix-core kernels do not
// (points not a multiple of 8, wide channel counts).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "../../include/fno_spectral_conv.h"
#include "fno_device.h"
#include "fno_host.h"

namespace fno {
namespace {

constexpr int kMixP = 128;          // grid points per tile of the channel mix
constexpr int kWaveP = 128;         // grid points per wave and tile of the weight gradient
constexpr int kMaxPartials = 1024;  // work-groups (partial sums) of the weight gradient
constexpr int64_t kPartialBytesCap = (int64_t)256 << 20;

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t rup(int64_t a, int64_t b) { return cdiv(a, b) * b; }

// The normal distribution function Phi(z) = (1 + erf(z / sqrt 2)) / 2 with
// erf from Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.26 (absolute error at most 1.5e-7): for x >= 0,
//   erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2),
//   t = 1 / (1 + p x),
// odd in x.  exp(-x^2) at x = |z| / sqrt 2 is also sqrt(2 pi) phi(z), the
// normal density the derivative needs.
struct NormalCdf {
  float cdf, e;  // Phi(z) and exp(-z^2 / 2)
};
__device__ __forceinline__ NormalCdf normal_cdf(float z) {
  const float x = __builtin_fabsf(z) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, x, 1.0f));
  float poly = __builtin_fmaf(1.061405429f, t, -1.453152027f);
  poly = __builtin_fmaf(poly, t, 1.421413741f);
  poly = __builtin_fmaf(poly, t, -0.284496736f);
  poly = __builtin_fmaf(poly, t, 0.254829592f);
  const float e = __expf(-x * x);
  const float erfc_half = 0.5f * poly * t * e;  // (1 - erf(x)) / 2
  return NormalCdf{z >= 0.0f ? 1.0f - erfc_half : erfc_half, e};
}
__device__ __forceinline__ float gelu_f(float z) {
  if (z != z) return z;
  return z * normal_cdf(z).cdf;
}
// d/dz z Phi(z) = Phi(z) + z phi(z)
__device__ __forceinline__ float gelu_grad_f(float z) {
  if (z != z) return z;
  const NormalCdf n = normal_cdf(z);
  return __builtin_fmaf(z * 0.39894228040143268f, n.e, n.cdf);
}

template <typename T>
struct Vec4;  // four consecutive elements (8 bytes fp16, 16 bytes fp32)
template <>
struct Vec4<_Float16> {
  typedef h4 type;
};
template <>
struct Vec4<float> {
  typedef f4 type;
};

struct EpiMixArgs {
  const void* in;    // [B][K][P]
  const void* w;     // wt = 0: [N][K]; wt = 1: [K][N]
  const void* add1;  // [B][N][P] or null
  const void* add2;  // [B][N][P] or null
  const void* bias;  // [N] or null
  void* out;         // [B][N][P]
  void* zout;        // [B][N][P] or null: the sum before the activation
  int64_t B, P;
  int K, N, Kp, ntt, wt, act, residual;
  int64_t tiles;     // B * ptiles
  int64_t ptiles;    // tiles of kMixP points per channel
};

// LDS of the matrix-core channel mix: W as [ntt*16][Kp + KPL] and the input
// tile transposed to [kMixP][Kp + KPL] (point-major, channels contiguous, so
// that a lane's KPL consecutive channels are one 16-byte read).
template <typename T>
size_t mix_lds_bytes(int ntt, int Kp) {
  const int kpl = 16 / (int)sizeof(T);
  return (size_t)(ntt * 16 + kMixP) * (Kp + kpl) * sizeof(T);
}

// FWD: the forward (activation, z, bias, residual; add2 unused); otherwise
// the data gradient (W transposed, two addends, nothing else).
template <typename T, int NT, bool FWD>
__global__ __launch_bounds__(256) void epi_mix_kernel(EpiMixArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  using V4 = typename Vec4<T>::type;
  constexpr int KPL = M::KPL, KS = M::KSTEP, VE = 16 / (int)sizeof(T);
  extern __shared__ __align__(16) unsigned char smem[];
  const int ld = a.Kp + KPL;
  T* WS = reinterpret_cast<T*>(smem);
  T* XT = WS + (size_t)a.ntt * 16 * ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const T* in = reinterpret_cast<const T*>(a.in);
  const T* w = reinterpret_cast<const T*>(a.w);
  const T* add1 = reinterpret_cast<const T*>(a.add1);
  const T* add2 = FWD ? nullptr : reinterpret_cast<const T*>(a.add2);
  const T* bias = FWD ? reinterpret_cast<const T*>(a.bias) : nullptr;
  T* out = reinterpret_cast<T*>(a.out);
  T* zout = FWD ? reinterpret_cast<T*>(a.zout) : nullptr;
  const bool gelu = FWD && a.act == FNO_EPI_ACT_GELU;
  const bool resid = FWD && a.residual;
  const int wt = FWD ? 0 : 1;

  // W once per work-group, zero beyond N rows and K columns; the input tile's
  // padding columns (k >= K) are zeroed once and never written again
  for (int e = tid; e < a.ntt * 16 * ld; e += 256) {
    const int n = e / ld, k = e - (e / ld) * ld;
    T v = (T)0.0f;
    if (n < a.N && k < a.K) v = wt ? w[(int64_t)k * a.N + n] : w[(int64_t)n * a.K + k];
    WS[e] = v;
  }
  for (int e = tid; e < kMixP * ld; e += 256) XT[e] = (T)0.0f;

  constexpr int vpr = kMixP / VE;  // 16-byte vectors per channel row of a tile
  const int nvec = a.K * vpr;
  for (int64_t t = blockIdx.x; t < a.tiles; t += gridDim.x) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * kMixP;
    __syncthreads();  // the previous tile's readers are done with XT
    for (int v = tid; v < nvec; v += 256) {
      const int k = v / vpr, c = v - (v / vpr) * vpr;
      const int64_t p = p0 + (int64_t)c * VE;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (p < a.P) val = *reinterpret_cast<const u32x4*>(in + ((b * a.K + k) * a.P + p));
      T e8[VE];
      __builtin_memcpy(e8, &val, 16);
#pragma unroll
      for (int e = 0; e < VE; ++e) XT[(c * VE + e) * ld + k] = e8[e];
    }
    __syncthreads();
    const int row0 = 32 * wave;  // this wave's 32 points of the tile
    for (int nc = 0; nc < a.ntt; nc += NT) {
      f4 acc[2][NT];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = (nc + j) * 16 + r16;
          const int64_t p = p0 + row0 + 16 * mt + 4 * g;
          f4 c = f4zero();
          if (nc + j < a.ntt && n < a.N && p < a.P) {
            const int64_t off = (b * a.N + n) * a.P + p;
            const float bv = bias ? (float)bias[n] : 0.0f;
            V4 u1{}, u2{};
            if (add1) u1 = *reinterpret_cast<const V4*>(add1 + off);
            if (add2) u2 = *reinterpret_cast<const V4*>(add2 + off);
#pragma unroll
            for (int i = 0; i < 4; ++i)
              c[i] = bv + (add1 ? (float)u1[i] : 0.0f) + (add2 ? (float)u2[i] : 0.0f);
          }
          acc[mt][j] = c;
        }
      for (int k0 = 0; k0 < a.Kp; k0 += KS) {
        frag af[2];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          af[mt] = M::ld(XT + (row0 + 16 * mt + r16) * ld + k0 + g * KPL);
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if (nc + j >= a.ntt) break;
          const frag bf = M::ld(WS + ((nc + j) * 16 + r16) * ld + k0 + g * KPL);
#pragma unroll
          for (int mt = 0; mt < 2; ++mt) acc[mt][j] = M::mma(af[mt], bf, acc[mt][j]);
        }
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = (nc + j) * 16 + r16;
          const int prow = row0 + 16 * mt + 4 * g;
          const int64_t p = p0 + prow;
          if (nc + j >= a.ntt || n >= a.N || p >= a.P) continue;
          const int64_t off = (b * a.N + n) * a.P + p;
          V4 zv, ov;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float z = acc[mt][j][i];
            zv[i] = (T)z;
            float o = gelu ? gelu_f(z) : z;
            if (resid) o += (float)XT[(prow + i) * ld + n];
            ov[i] = (T)o;
          }
          if (zout) *reinterpret_cast<V4*>(zout + off) = zv;
          *reinterpret_cast<V4*>(out + off) = ov;
        }
    }
  }
}

// Software-pipelined fp16 channel mix for the common shapes (at most NT*16
// output channels, at most 128 input channels), 64-point tiles.  Every
// global access is a 16-byte vector of a channel row, eight lanes covering
// a row's 128 bytes: the input rows are transposed into LDS (channel pairs
// (k, k+1) travel together so that the transposing writes are 32-bit, and
// the 16-byte column blocks of a transposed row are XOR-swizzled by the
// row's 8-row group, when the number of blocks is a power of two, to spread
// those writes over the banks); the addends and the results pass through
// row-major LDS tiles between the row-wise global accesses and the
// matrix-core layout.  The next tile's loads are in flight while the
// current tile is multiplied and stored.
constexpr int kPipeP = 64;  // grid points per tile of the pipelined channel mix

template <int NT>
size_t pipe_lds_bytes(int Kp) {
  const int ld = Kp + 8, lda = kPipeP + 8;
  return (size_t)((NT * 16 + kPipeP) * ld + 2 * NT * 16 * lda) * 2;
}

template <int NT, bool FWD>
__global__ __launch_bounds__(256) void epi_mix_pipe_kernel(EpiMixArgs a) {
  using T = _Float16;
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = 8, KS = 32;
  constexpr int VPR = kPipeP / 8;            // 16-byte vectors per channel row of a tile
  constexpr int XV = 128 / 2 * VPR / 256;    // channel-pair vectors per thread (K <= 128)
  constexpr int AV = NT * 16 * VPR / 256 > 0 ? NT * 16 * VPR / 256 : 1;  // addend vectors
  constexpr int LDA = kPipeP + 8;
  extern __shared__ __align__(16) unsigned char smem[];
  const int ld = a.Kp + KPL;
  const int nkb = a.Kp / KPL;
  const int smask = (nkb & (nkb - 1)) == 0 ? nkb - 1 : 0;
  T* WS = reinterpret_cast<T*>(smem);
  T* XT = WS + (size_t)NT * 16 * ld;
  T* A1 = XT + (size_t)kPipeP * ld;   // addend y / gx_spec, then out / gx
  T* A2 = A1 + (size_t)NT * 16 * LDA; // FWD: z; otherwise the addend g_out
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const T* in = reinterpret_cast<const T*>(a.in);
  const T* w = reinterpret_cast<const T*>(a.w);
  const T* add1 = reinterpret_cast<const T*>(a.add1);
  const T* add2 = FWD ? nullptr : reinterpret_cast<const T*>(a.add2);
  const T* bias = FWD ? reinterpret_cast<const T*>(a.bias) : nullptr;
  T* out = reinterpret_cast<T*>(a.out);
  T* zout = FWD ? reinterpret_cast<T*>(a.zout) : nullptr;
  const bool gelu = FWD && a.act == FNO_EPI_ACT_GELU;
  const bool resid = FWD && a.residual;

  for (int e = tid; e < NT * 16 * ld; e += 256) {
    const int n = e / ld, k = e - (e / ld) * ld;
    T v = (T)0.0f;
    if (n < a.N && k < a.K) v = FWD ? w[(int64_t)n * a.K + k] : w[(int64_t)k * a.N + n];
    WS[e] = v;
  }
  for (int e = tid; e < kPipeP * ld; e += 256) XT[e] = (T)0.0f;
  float bv[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int n = j * 16 + r16;
    bv[j] = (bias && n < a.N) ? (float)bias[n] : 0.0f;
  }
  // swizzled position of channel k in transposed row p
  auto xt_at = [&](int p, int k) {
    return p * ld + ((((k >> 3) ^ ((p >> 3) & smask))) << 3) + (k & 7);
  };

  const int npv = ((a.K + 1) / 2) * VPR;  // channel-pair vectors of a tile
  const int nav = a.N * VPR;              // addend / result vectors of a tile
  u32x4 xr[XV][2], ar1[AV], ar2[AV];
  auto load = [&](int64_t t) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * kPipeP;
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = tid + 256 * i;
      const int kp = v / VPR, c = v - (v / VPR) * VPR;
      const int64_t p = p0 + (int64_t)c * 8;
      xr[i][0] = xr[i][1] = u32x4{0u, 0u, 0u, 0u};
      if (v < npv && p < a.P) {
        const T* src = in + ((b * a.K + 2 * kp) * a.P + p);
        xr[i][0] = *reinterpret_cast<const u32x4*>(src);
        if (2 * kp + 1 < a.K) xr[i][1] = *reinterpret_cast<const u32x4*>(src + a.P);
      }
    }
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + 256 * i;
      const int n = v / VPR, c = v - (v / VPR) * VPR;
      const int64_t p = p0 + (int64_t)c * 8;
      ar1[i] = ar2[i] = u32x4{0u, 0u, 0u, 0u};
      if (v < nav && p < a.P) {
        const int64_t off = (b * a.N + n) * a.P + p;
        if (add1) ar1[i] = *reinterpret_cast<const u32x4*>(add1 + off);
        if (add2) ar2[i] = *reinterpret_cast<const u32x4*>(add2 + off);
      }
    }
  };

  int64_t t = blockIdx.x;
  if (t < a.tiles) load(t);
  const int prow = 16 * wave + 4 * g;  // first of this lane's four points in the tile
  while (t < a.tiles) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * kPipeP;
    __syncthreads();  // the previous tile is out of XT, A1 and A2
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = tid + 256 * i;
      if (v < npv) {
        const int kp = v / VPR, c = v - (v / VPR) * VPR;
        uint16_t lo[8], hi[8];
        __builtin_memcpy(lo, &xr[i][0], 16);
        __builtin_memcpy(hi, &xr[i][1], 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t pr = (uint32_t)lo[e] | ((uint32_t)hi[e] << 16);
          *reinterpret_cast<uint32_t*>(XT + xt_at(c * 8 + e, 2 * kp)) = pr;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + 256 * i;
      if (v < nav) {
        const int n = v / VPR, c = v - (v / VPR) * VPR;
        *reinterpret_cast<u32x4*>(A1 + n * LDA + c * 8) = ar1[i];
        if (!FWD) *reinterpret_cast<u32x4*>(A2 + n * LDA + c * 8) = ar2[i];
      }
    }
    __syncthreads();
    const int64_t tn = t + gridDim.x;
    if (tn < a.tiles) load(tn);  // in flight during this tile's products and stores
    f4 acc[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int n = j * 16 + r16;
      const h4 u1 = *reinterpret_cast<const h4*>(A1 + n * LDA + prow);
      h4 u2 = h4{};
      if (!FWD) u2 = *reinterpret_cast<const h4*>(A2 + n * LDA + prow);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[j][i] = bv[j] + (float)u1[i] + (float)u2[i];
    }
    for (int k0 = 0; k0 < a.Kp; k0 += KS) {
      const frag af = M::ld(XT + xt_at(16 * wave + r16, k0 + g * KPL));
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const frag bf = M::ld(WS + (j * 16 + r16) * ld + k0 + g * KPL);
        acc[j] = M::mma(af, bf, acc[j]);
      }
    }
    // results back into the row-major tiles at this lane's own positions
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int n = j * 16 + r16;
      h4 zv, ov;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float z = acc[j][i];
        zv[i] = (T)z;
        float o = gelu ? gelu_f(z) : z;
        if (resid && n < a.K) o += (float)XT[xt_at(prow + i, n)];
        ov[i] = (T)o;
      }
      *reinterpret_cast<h4*>(A1 + n * LDA + prow) = ov;
      if (FWD) *reinterpret_cast<h4*>(A2 + n * LDA + prow) = zv;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + 256 * i;
      const int n = v / VPR, c = v - (v / VPR) * VPR;
      const int64_t p = p0 + (int64_t)c * 8;
      if (v < nav && p < a.P) {
        const int64_t off = (b * a.N + n) * a.P + p;
        *reinterpret_cast<u32x4*>(out + off) = *reinterpret_cast<const u32x4*>(A1 + n * LDA + c * 8);
        if (zout)
          *reinterpret_cast<u32x4*>(zout + off) =
              *reinterpret_cast<const u32x4*>(A2 + n * LDA + c * 8);
      }
    }
    t = tn;
  }
}

// Any shape: one grid point per thread, eight output channels per
// work-group row of the grid.
template <typename T>
__global__ __launch_bounds__(256) void epi_mix_generic_kernel(EpiMixArgs a) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= a.B * a.P) return;
  const int64_t b = q / a.P, p = q - (q / a.P) * a.P;
  const int n0 = blockIdx.y * 8;
  const T* in = reinterpret_cast<const T*>(a.in);
  const T* w = reinterpret_cast<const T*>(a.w);
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
  for (int k = 0; k < a.K; ++k) {
    const float v = (float)in[(b * a.K + k) * a.P + p];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int n = n0 + j;
      if (n < a.N) {
        const float wv = (float)(a.wt ? w[(int64_t)k * a.N + n] : w[(int64_t)n * a.K + k]);
        acc[j] = __builtin_fmaf(wv, v, acc[j]);
      }
    }
  }
  const T* add1 = reinterpret_cast<const T*>(a.add1);
  const T* add2 = reinterpret_cast<const T*>(a.add2);
  const T* bias = reinterpret_cast<const T*>(a.bias);
  T* out = reinterpret_cast<T*>(a.out);
  T* zout = reinterpret_cast<T*>(a.zout);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int n = n0 + j;
    if (n >= a.N) continue;
    const int64_t off = (b * a.N + n) * a.P + p;
    float z = (bias ? (float)bias[n] : 0.0f) + (add1 ? (float)add1[off] : 0.0f) +
              (add2 ? (float)add2[off] : 0.0f) + acc[j];
    if (zout) zout[off] = (T)z;
    float o = a.act == FNO_EPI_ACT_GELU ? gelu_f(z) : z;
    if (a.residual) o += (float)in[(b * a.K + n) * a.P + p];
    out[off] = (T)o;
  }
}

struct EpiWgradArgs {
  const void* x;     // [B][Cin][P]
  const void* z;     // [B][Cout][P] (act GELU)
  const void* gout;  // [B][Cout][P]
  void* gz;          // [B][Cout][P] (act GELU): written
  float* part;       // [G][Cout*Cin + Cout]
  int64_t B, P;
  int Cin, Cout, act;
  int wpr;           // waves per point range (1, 2 or 4): they split the output channels
  int ranges;        // point ranges per work-group and tile (4 / wpr)
  int64_t tiles, ptiles;
};

template <typename T>
size_t wgrad_lds_bytes(int cout_pad, int cin_pad) {
  return (size_t)(cout_pad * cin_pad + cout_pad) * sizeof(float);
}

// Matrix-core weight gradient: D[o][i] += gz[o][p..] x[i][p..] with the
// contraction over grid points, both operands read straight from HBM as
// KPL consecutive points per lane.  Each wave holds OG output-channel tiles
// by IT input-channel tiles of accumulators; waves of one point range split
// the output channels.  Partial sums leave through LDS in a fixed order.
template <typename T, int OG, int IT>
__global__ __launch_bounds__(256) void epi_wgrad_kernel(EpiWgradArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int og = wave % a.wpr, rg = wave / a.wpr;
  const T* x = reinterpret_cast<const T*>(a.x);
  const T* z = reinterpret_cast<const T*>(a.z);
  const T* gout = reinterpret_cast<const T*>(a.gout);
  T* gz = reinterpret_cast<T*>(a.gz);
  const bool gelu = a.act == FNO_EPI_ACT_GELU;

  f4 acc[OG][IT];
  float bsum[OG];
#pragma unroll
  for (int o = 0; o < OG; ++o) {
    bsum[o] = 0.0f;
#pragma unroll
    for (int it = 0; it < IT; ++it) acc[o][it] = f4zero();
  }
  for (int64_t t = blockIdx.x; t < a.tiles; t += gridDim.x) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * ((int64_t)kWaveP * a.ranges) + (int64_t)rg * kWaveP;
#pragma unroll 2
    for (int k0 = 0; k0 < kWaveP; k0 += KS) {
      const int64_t p = p0 + k0 + g * KPL;
      const bool pin = p < a.P;  // P is a multiple of 8: a lane's KPL points are all in or out
      frag af[OG], bf[IT];
#pragma unroll
      for (int o = 0; o < OG; ++o) {
        const int oc = (og * OG + o) * 16 + r16;
        af[o] = M::zero();
        if (pin && oc < a.Cout) {
          const int64_t off = (b * a.Cout + oc) * a.P + p;
          frag gv = M::ld(gout + off);
          if (gelu) {
            const frag zv = M::ld(z + off);
#pragma unroll
            for (int i = 0; i < KPL; ++i) gv[i] = (T)((float)gv[i] * gelu_grad_f((float)zv[i]));
            *reinterpret_cast<frag*>(gz + off) = gv;
          }
          float s = 0.0f;
#pragma unroll
          for (int i = 0; i < KPL; ++i) s += (float)gv[i];
          bsum[o] += s;
          af[o] = gv;
        }
      }
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int ic = it * 16 + r16;
        bf[it] = M::zero();
        if (pin && ic < a.Cin) bf[it] = M::ld(x + (b * a.Cin + ic) * a.P + p);
      }
#pragma unroll
      for (int o = 0; o < OG; ++o)
#pragma unroll
        for (int it = 0; it < IT; ++it) acc[o][it] = M::mma(af[o], bf[it], acc[o][it]);
    }
  }
  // bias sums: the four lane groups of a row hold parts of the same channel
#pragma unroll
  for (int o = 0; o < OG; ++o) {
    bsum[o] += __shfl_xor(bsum[o], 16);
    bsum[o] += __shfl_xor(bsum[o], 32);
  }
  // fixed-order reduction over the point ranges of the work-group
  const int cin_pad = IT * 16, cout_pad = a.wpr * OG * 16;
  float* red = reinterpret_cast<float*>(smem);
  float* bred = red + cout_pad * cin_pad;
  for (int e = tid; e < cout_pad * cin_pad + cout_pad; e += 256) red[e] = 0.0f;
  __syncthreads();
  for (int r = 0; r < a.ranges; ++r) {
    if (rg == r) {
#pragma unroll
      for (int o = 0; o < OG; ++o) {
        const int orow = (og * OG + o) * 16;
#pragma unroll
        for (int it = 0; it < IT; ++it)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            red[(orow + 4 * g + i) * cin_pad + it * 16 + r16] += acc[o][it][i];
        if (g == 0) bred[orow + r16] += bsum[o];
      }
    }
    __syncthreads();
  }
  const int64_t E = (int64_t)a.Cout * a.Cin + a.Cout;
  float* part = a.part + (int64_t)blockIdx.x * E;
  for (int e = tid; e < a.Cout * a.Cin; e += 256) {
    const int o = e / a.Cin, i = e - (e / a.Cin) * a.Cin;
    part[e] = red[o * cin_pad + i];
  }
  for (int o = tid; o < a.Cout; o += 256) part[(int64_t)a.Cout * a.Cin + o] = bred[o];
}

// Software-pipelined fp16 parameter gradients for up to 128 x 128
// channels, 64-point tiles: g_out, z and x rows arrive as 16-byte vectors
// (eight lanes per 128-byte row segment), g_z is formed and stored in the
// same layout and staged with x in row-major LDS tiles, from which the
// matrix-core fragments (eight consecutive points per lane) are read.  Wave
// w owns output-channel tiles w, w + 4 (OTW of them) by every input-channel
// tile (IT); the next tile's loads are in flight during the products.
constexpr int kWgP = 64;  // grid points per tile of the pipelined weight gradient

template <int OTW, int IT>
size_t wgrad_pipe_lds_bytes() {
  return (size_t)(4 * OTW * 16 + IT * 16) * (kWgP + 8) * 2;
}

template <int OTW, int IT>
__global__ __launch_bounds__(256) void epi_wgrad_pipe_kernel(EpiWgradArgs a) {
  using T = _Float16;
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int VPR = kWgP / 8;          // 16-byte vectors per channel row of a tile
  constexpr int OROWS = 4 * OTW * 16;    // output-channel rows held (padded)
  constexpr int GV = OROWS * VPR / 256;  // g_z vectors per thread
  constexpr int XVN = IT * 16 * VPR / 256 > 0 ? IT * 16 * VPR / 256 : 1;
  constexpr int LDA = kWgP + 8;
  extern __shared__ __align__(16) unsigned char smem[];
  T* GZ = reinterpret_cast<T*>(smem);  // [OROWS][LDA]
  T* XS = GZ + OROWS * LDA;            // [IT*16][LDA]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const T* x = reinterpret_cast<const T*>(a.x);
  const T* z = reinterpret_cast<const T*>(a.z);
  const T* gout = reinterpret_cast<const T*>(a.gout);
  T* gz = reinterpret_cast<T*>(a.gz);
  const bool gelu = a.act == FNO_EPI_ACT_GELU;
  const int ngv = a.Cout * VPR, nxv = a.Cin * VPR;

  u32x4 gr[GV], zr[GV], xr[XVN];
  float bs[GV];
#pragma unroll
  for (int i = 0; i < GV; ++i) bs[i] = 0.0f;
  auto load = [&](int64_t t) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * kWgP;
#pragma unroll
    for (int i = 0; i < GV; ++i) {
      const int v = tid + 256 * i;
      const int o = v / VPR, c = v - (v / VPR) * VPR;
      const int64_t p = p0 + (int64_t)c * 8;
      gr[i] = zr[i] = u32x4{0u, 0u, 0u, 0u};
      if (v < ngv && p < a.P) {
        const int64_t off = (b * a.Cout + o) * a.P + p;
        gr[i] = *reinterpret_cast<const u32x4*>(gout + off);
        if (gelu) zr[i] = *reinterpret_cast<const u32x4*>(z + off);
      }
    }
#pragma unroll
    for (int i = 0; i < XVN; ++i) {
      const int v = tid + 256 * i;
      const int ic = v / VPR, c = v - (v / VPR) * VPR;
      const int64_t p = p0 + (int64_t)c * 8;
      xr[i] = u32x4{0u, 0u, 0u, 0u};
      if (v < nxv && p < a.P) xr[i] = *reinterpret_cast<const u32x4*>(x + (b * a.Cin + ic) * a.P + p);
    }
  };

  f4 acc[OTW][IT];
#pragma unroll
  for (int u = 0; u < OTW; ++u)
#pragma unroll
    for (int it = 0; it < IT; ++it) acc[u][it] = f4zero();
  // rows beyond the channel counts stay zero in LDS
  for (int e = tid; e < (OROWS + IT * 16) * LDA; e += 256) GZ[e] = (T)0.0f;

  int64_t t = blockIdx.x;
  if (t < a.tiles) load(t);
  while (t < a.tiles) {
    const int64_t b = t / a.ptiles;
    const int64_t p0 = (t - b * a.ptiles) * kWgP;
    __syncthreads();  // the previous tile's fragments are read
#pragma unroll
    for (int i = 0; i < GV; ++i) {
      const int v = tid + 256 * i;
      if (v < ngv) {
        const int o = v / VPR, c = v - (v / VPR) * VPR;
        h8 gv = w_as_h8(gr[i]);
        const int64_t p = p0 + (int64_t)c * 8;
        if (gelu) {
          const h8 zv = w_as_h8(zr[i]);
#pragma unroll
          for (int e = 0; e < 8; ++e) gv[e] = (T)((float)gv[e] * gelu_grad_f((float)zv[e]));
          if (p < a.P) *reinterpret_cast<h8*>(gz + (b * a.Cout + o) * a.P + p) = gv;
        }
        float sum = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += (float)gv[e];
        bs[i] += sum;
        *reinterpret_cast<h8*>(GZ + o * LDA + c * 8) = gv;
      }
    }
#pragma unroll
    for (int i = 0; i < XVN; ++i) {
      const int v = tid + 256 * i;
      if (v < nxv) {
        const int ic = v / VPR, c = v - (v / VPR) * VPR;
        *reinterpret_cast<u32x4*>(XS + ic * LDA + c * 8) = xr[i];
      }
    }
    __syncthreads();
    const int64_t tn = t + gridDim.x;
    if (tn < a.tiles) load(tn);  // in flight during the products
#pragma unroll
    for (int k0 = 0; k0 < kWgP; k0 += 32) {
      frag af[OTW], bf[IT];
#pragma unroll
      for (int u = 0; u < OTW; ++u)
        af[u] = M::ld(GZ + ((wave + 4 * u) * 16 + r16) * LDA + k0 + g * 8);
#pragma unroll
      for (int it = 0; it < IT; ++it) bf[it] = M::ld(XS + (it * 16 + r16) * LDA + k0 + g * 8);
#pragma unroll
      for (int u = 0; u < OTW; ++u)
#pragma unroll
        for (int it = 0; it < IT; ++it) acc[u][it] = M::mma(af[u], bf[it], acc[u][it]);
    }
    t = tn;
  }
  // this work-group's partial sums: each (o, i) element belongs to one lane
  const int64_t E = (int64_t)a.Cout * a.Cin + a.Cout;
  float* part = a.part + (int64_t)blockIdx.x * E;
#pragma unroll
  for (int u = 0; u < OTW; ++u)
#pragma unroll
    for (int it = 0; it < IT; ++it)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = (wave + 4 * u) * 16 + 4 * g + q, ic = it * 16 + r16;
        if (o < a.Cout && ic < a.Cin) part[(int64_t)o * a.Cin + ic] = acc[u][it][q];
      }
  // bias sums: the eight lanes of a row segment hold parts of one channel
#pragma unroll
  for (int i = 0; i < GV; ++i) {
    float v = bs[i];
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 4);
    const int vv = tid + 256 * i;
    if ((vv & (VPR - 1)) == 0 && vv < ngv) part[(int64_t)a.Cout * a.Cin + vv / VPR] = v;
  }
}

// Any shape: g_z elementwise (act GELU) ...
template <typename T>
__global__ __launch_bounds__(256) void epi_gz_generic_kernel(const T* gout, const T* z, T* gz,
                                                              int64_t n) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q < n) gz[q] = (T)((float)gout[q] * gelu_grad_f((float)z[q]));
}

// ... then one partial sum per (work-group row of the grid, output element):
// work-group row j sums the grid points [j L, (j + 1) L) of the flattened
// (batch, point) range.
template <typename T>
__global__ __launch_bounds__(256) void epi_wgrad_generic_kernel(const T* x, const T* gz,
                                                                float* part, int64_t B,
                                                                int64_t P, int Cin, int Cout,
                                                                int64_t L) {
  const int64_t E = (int64_t)Cout * Cin + Cout;
  const int64_t e = (int64_t)blockIdx.y * 256 + threadIdx.x;
  if (e >= E) return;
  const int64_t j = blockIdx.x;
  const bool is_bias = e >= (int64_t)Cout * Cin;
  const int o = is_bias ? (int)(e - (int64_t)Cout * Cin) : (int)(e / Cin);
  const int i = is_bias ? 0 : (int)(e - (e / Cin) * Cin);
  const int64_t q0 = j * L, q1 = std::min<int64_t>(q0 + L, B * P);
  float s = 0.0f;
  for (int64_t q = q0; q < q1;) {
    const int64_t b = q / P, p = q - (q / P) * P;
    const int64_t pe = std::min<int64_t>(P, p + (q1 - q));
    const T* gr = gz + (b * Cout + o) * P;
    const T* xr = x + (b * Cin + i) * P;
    for (int64_t pp = p; pp < pe; ++pp)
      s = is_bias ? s + (float)gr[pp] : __builtin_fmaf((float)gr[pp], (float)xr[pp], s);
    q += pe - p;
  }
  part[j * E + e] = s;
}

// 32 elements per work-group; the eight thread rows sum the partials
// j = r, r + 8, ... and are then added in row order (a fixed order).
__global__ __launch_bounds__(256) void epi_reduce_kernel(const float* part, int G, int64_t E,
                                                         int64_t Ew, float* gw, float* gb) {
  __shared__ float red[8][32];
  const int c = threadIdx.x & 31, r = threadIdx.x >> 5;
  const int64_t e = (int64_t)blockIdx.x * 32 + c;
  float s = 0.0f;
  if (e < E)
    for (int j = r; j < G; j += 8) s += part[(int64_t)j * E + e];
  red[r][c] = s;
  __syncthreads();
  if (r == 0 && e < E) {
    float t = red[0][c];
#pragma unroll
    for (int i = 1; i < 8; ++i) t += red[i][c];
    if (e < Ew) gw[e] = t;
    else if (gb) gb[e - Ew] = t;
  }
}

// --------------------------------------------------------------------------
// Host side
// --------------------------------------------------------------------------
struct EpiGeo {
  int es;  // element bytes
  int64_t B, P;
  int Cin, Cout, act, residual;
};

fno_status check_desc(const fno_block_desc* d, EpiGeo* g) {
  if (!d) return FNO_ERR_INVALID_ARGUMENT;
  if (d->precision != FNO_PREC_FP32 && d->precision != FNO_PREC_FP16_TANH)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->batch < 1 || d->points < 1 || d->c_in < 1 || d->c_out < 1 || d->c_in > 65536 ||
      d->c_out > 65536)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->activation != FNO_EPI_ACT_NONE && d->activation != FNO_EPI_ACT_GELU)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->residual != 0 && d->residual != 1) return FNO_ERR_INVALID_ARGUMENT;
  if (d->residual && d->c_in != d->c_out) return FNO_ERR_INVALID_ARGUMENT;
  // element counts within the grid limits of the generic kernels: at most
  // 2^38 elements per tensor, 65535 x 256 parameter-gradient elements
  if (d->batch > ((int64_t)1 << 38) / d->points) return FNO_ERR_INVALID_ARGUMENT;
  const int64_t cmax = std::max(d->c_in, d->c_out);
  if (d->batch * d->points > ((int64_t)1 << 38) / cmax) return FNO_ERR_INVALID_ARGUMENT;
  if (d->c_out * (d->c_in + 1) > (int64_t)65535 * 256) return FNO_ERR_INVALID_ARGUMENT;
  g->es = d->precision == FNO_PREC_FP16_TANH ? 2 : 4;
  g->B = d->batch;
  g->P = d->points;
  g->Cin = (int)d->c_in;
  g->Cout = (int)d->c_out;
  g->act = d->activation;
  g->residual = d->residual;
  return FNO_OK;
}

inline bool ok16(const void* p) { return p && ((uintptr_t)p & 15u) == 0; }
inline bool null_or16(const void* p) { return !p || ((uintptr_t)p & 15u) == 0; }

// The matrix-core channel mix: points a multiple of 8 (16-byte rows), at
// most 128 input channels, W and the tile within 96 KiB of LDS.
bool mix_fast(const EpiGeo& g, int K, int N) {
  if (g.P % 8 != 0 || K > 128) return false;
  const int ks = g.es == 2 ? 32 : 16;
  const int Kp = (int)rup(K, ks), ntt = (int)cdiv(N, 16);
  const size_t lds = g.es == 2 ? mix_lds_bytes<_Float16>(ntt, Kp) : mix_lds_bytes<float>(ntt, Kp);
  return lds <= 96 * 1024;
}

// Weight-gradient layout: input-channel tiles IT (padded to 1, 2, 4, 8),
// output tiles per wave OG (4, or 2 with eight input tiles) and waves per
// point range (1, 2, 4).  False when the shape is outside it.
bool wgrad_fast(const EpiGeo& g, int* it, int* og, int* wpr) {
  if (g.P % 8 != 0 || g.Cin > 128) return false;
  const int cit = (int)cdiv(g.Cin, 16);
  *it = cit <= 1 ? 1 : cit <= 2 ? 2 : cit <= 4 ? 4 : 8;
  *og = *it == 8 ? 2 : 4;
  const int need = (int)cdiv(cdiv(g.Cout, 16), *og);
  if (need > 4) return false;
  *wpr = need <= 1 ? 1 : need <= 2 ? 2 : 4;
  return true;
}

// The pipelined fp16 weight gradient: points a multiple of 8, at most 128
// channels each way.
bool wgrad_pipe(const EpiGeo& g) {
  return g.es == 2 && g.P % 8 == 0 && g.Cin <= 128 && g.Cout <= 128;
}

// Partial sums of the weight gradient: count and bytes.
int wgrad_partials(const EpiGeo& g, int64_t* tiles, int64_t* ptiles) {
  const int64_t E = (int64_t)g.Cout * g.Cin + g.Cout;
  int it, og, wpr;
  int64_t cap = std::max<int64_t>(1, kPartialBytesCap / (E * 4));
  if (wgrad_pipe(g)) {
    *ptiles = cdiv(g.P, kWgP);
    *tiles = g.B * *ptiles;
  } else if (wgrad_fast(g, &it, &og, &wpr)) {
    const int ranges = 4 / wpr;
    *ptiles = cdiv(g.P, (int64_t)kWaveP * ranges);
    *tiles = g.B * *ptiles;
  } else {
    *ptiles = 0;
    *tiles = cdiv(g.B * g.P, 4096);
  }
  return (int)std::min<int64_t>({*tiles, (int64_t)kMaxPartials, cap});
}

size_t wgrad_ws_bytes(const EpiGeo& g) {
  int64_t tiles, ptiles;
  const int G = wgrad_partials(g, &tiles, &ptiles);
  const int64_t E = (int64_t)g.Cout * g.Cin + g.Cout;
  return (size_t)rup((int64_t)G * E * 4, 256);
}

int num_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
    return 256;
  return n;
}

hipError_t allow_lds(const void* kern, size_t lds) {
  if (lds <= 65536) return hipSuccess;
  return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

struct EpiMixLaunch {
  EpiMixArgs a;
  int es;
  hipStream_t s;
  bool fast;
};

template <typename T, int NT, bool FWD>
hipError_t launch_mix_nt(const EpiMixArgs& a, int grid, size_t lds, hipStream_t s) {
  hipError_t e = allow_lds(reinterpret_cast<const void*>(&epi_mix_kernel<T, NT, FWD>), lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((epi_mix_kernel<T, NT, FWD>), dim3(grid), dim3(256), lds, s, a);
  return hipSuccess;
}

template <typename T, bool FWD>
hipError_t launch_mix_fast(const EpiMixArgs& a, int grid, size_t lds, hipStream_t s) {
  if (a.ntt >= 8) return launch_mix_nt<T, 8, FWD>(a, grid, lds, s);
  if (a.ntt >= 4) return launch_mix_nt<T, 4, FWD>(a, grid, lds, s);
  if (a.ntt >= 2) return launch_mix_nt<T, 2, FWD>(a, grid, lds, s);
  return launch_mix_nt<T, 1, FWD>(a, grid, lds, s);
}

template <int NT, bool FWD>
hipError_t launch_pipe_nt(const EpiMixArgs& a, int grid, size_t lds, hipStream_t s) {
  hipError_t e = allow_lds(reinterpret_cast<const void*>(&epi_mix_pipe_kernel<NT, FWD>), lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((epi_mix_pipe_kernel<NT, FWD>), dim3(grid), dim3(256), lds, s, a);
  return hipSuccess;
}

template <bool FWD>
hipError_t launch_pipe(const EpiMixArgs& a, int grid, hipStream_t s) {
  const int nt = a.ntt <= 1 ? 1 : a.ntt <= 2 ? 2 : a.ntt <= 4 ? 4 : 8;
  switch (nt) {
    case 1: return launch_pipe_nt<1, FWD>(a, grid, pipe_lds_bytes<1>(a.Kp), s);
    case 2: return launch_pipe_nt<2, FWD>(a, grid, pipe_lds_bytes<2>(a.Kp), s);
    case 4: return launch_pipe_nt<4, FWD>(a, grid, pipe_lds_bytes<4>(a.Kp), s);
    default: return launch_pipe_nt<8, FWD>(a, grid, pipe_lds_bytes<8>(a.Kp), s);
  }
}

template <typename T>
hipError_t launch_mix_t(EpiMixLaunch* L) {
  EpiMixArgs& a = L->a;
  if (L->fast && sizeof(T) == 2 && a.ntt <= 8 && a.K <= 128) {
    const int64_t tiles = a.B * cdiv(a.P, kPipeP);
    a.ptiles = cdiv(a.P, kPipeP);
    a.tiles = tiles;
    const int grid = (int)std::min<int64_t>(tiles, (int64_t)4 * num_cus());
    const hipError_t e = a.wt ? launch_pipe<false>(a, grid, L->s) : launch_pipe<true>(a, grid, L->s);
    if (e != hipSuccess) return e;
  } else if (L->fast) {
    const size_t lds = mix_lds_bytes<T>(a.ntt, a.Kp);
    const int grid = (int)std::min<int64_t>(a.tiles, (int64_t)4 * num_cus());
    const hipError_t e = a.wt ? launch_mix_fast<T, false>(a, grid, lds, L->s)
                              : launch_mix_fast<T, true>(a, grid, lds, L->s);
    if (e != hipSuccess) return e;
  } else {
    const dim3 grid((unsigned)cdiv(a.B * a.P, 256), (unsigned)cdiv(a.N, 8));
    hipLaunchKernelGGL(epi_mix_generic_kernel<T>, grid, dim3(256), 0, L->s, a);
  }
  return hipGetLastError();
}

hipError_t launch_mix(void* ctx) {
  EpiMixLaunch* L = static_cast<EpiMixLaunch*>(ctx);
  return L->es == 2 ? launch_mix_t<_Float16>(L) : launch_mix_t<float>(L);
}

fno_status run_mix(const EpiGeo& g, const char* name, const void* in, int K, const void* w, int wt,
                   int N, const void* add1, const void* add2, const void* bias, void* out,
                   void* zout, int act, int residual, hipStream_t s) {
  EpiMixLaunch L{};
  EpiMixArgs& a = L.a;
  a.in = in;
  a.w = w;
  a.add1 = add1;
  a.add2 = add2;
  a.bias = bias;
  a.out = out;
  a.zout = zout;
  a.B = g.B;
  a.P = g.P;
  a.K = K;
  a.N = N;
  a.Kp = (int)rup(K, g.es == 2 ? 32 : 16);
  a.ntt = (int)cdiv(N, 16);
  a.wt = wt;
  a.act = act;
  a.residual = residual;
  a.ptiles = cdiv(g.P, kMixP);
  a.tiles = g.B * a.ptiles;
  L.es = g.es;
  L.s = s;
  L.fast = mix_fast(g, K, N);
  const hipError_t e = timed_launch(name, s, launch_mix, &L);
  return e == hipSuccess ? FNO_OK : report_hip_error(e, name);
}

struct EpiWgradLaunch {
  EpiWgradArgs a;
  int es, G, it, og;
  bool fast, pipe;
  const void* gz_src;  // generic path: the gradient the sums read
  float *gw, *gb;
  hipStream_t s;
};

template <typename T>
hipError_t launch_wgrad_t(EpiWgradLaunch* L) {
  EpiWgradArgs& a = L->a;
  const int64_t E = (int64_t)a.Cout * a.Cin + a.Cout;
  if (L->pipe) {
    const int cit = (int)cdiv(a.Cin, 16);
    const int itp = cit <= 1 ? 1 : cit <= 2 ? 2 : cit <= 4 ? 4 : 8;
    const int otw = a.Cout <= 64 ? 1 : 2;
#define FNO_WGP(OTWV, ITV)                                                                     if (otw == OTWV && itp == ITV) {                                                               const size_t lds = wgrad_pipe_lds_bytes<OTWV, ITV>();                                        hipError_t e = allow_lds(reinterpret_cast<const void*>(&epi_wgrad_pipe_kernel<OTWV, ITV>), lds);     if (e != hipSuccess) return e;                                                               hipLaunchKernelGGL((epi_wgrad_pipe_kernel<OTWV, ITV>), dim3(L->G), dim3(256), lds, L->s, a);   }
    FNO_WGP(1, 1) else FNO_WGP(1, 2) else FNO_WGP(1, 4) else FNO_WGP(1, 8)
    else FNO_WGP(2, 1) else FNO_WGP(2, 2) else FNO_WGP(2, 4) else FNO_WGP(2, 8)
    else return hipErrorInvalidValue;
#undef FNO_WGP
  } else if (L->fast) {
    const size_t lds = wgrad_lds_bytes<T>(a.wpr * L->og * 16, L->it * 16);
#define FNO_WG(OGV, ITV)                                                                     \
  if (L->og == OGV && L->it == ITV) {                                                        \
    hipError_t e = allow_lds(reinterpret_cast<const void*>(&epi_wgrad_kernel<T, OGV, ITV>), lds); \
    if (e != hipSuccess) return e;                                                           \
    hipLaunchKernelGGL((epi_wgrad_kernel<T, OGV, ITV>), dim3(L->G), dim3(256), lds, L->s, a); \
  }
    FNO_WG(4, 1) else FNO_WG(4, 2) else FNO_WG(4, 4) else FNO_WG(2, 8) else return hipErrorInvalidValue;
#undef FNO_WG
  } else {
    const T* gzs = reinterpret_cast<const T*>(a.gout);
    if (a.act == FNO_EPI_ACT_GELU) {
      const int64_t n = a.B * a.Cout * a.P;
      hipLaunchKernelGGL(epi_gz_generic_kernel<T>, dim3((unsigned)cdiv(n, 256)), dim3(256), 0,
                         L->s, reinterpret_cast<const T*>(a.gout),
                         reinterpret_cast<const T*>(a.z), reinterpret_cast<T*>(a.gz), n);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      gzs = reinterpret_cast<const T*>(a.gz);
    }
    const int64_t L1 = cdiv(a.B * a.P, L->G);
    hipLaunchKernelGGL(epi_wgrad_generic_kernel<T>, dim3((unsigned)L->G, (unsigned)cdiv(E, 256)),
                       dim3(256), 0, L->s, reinterpret_cast<const T*>(a.x), gzs, a.part, a.B,
                       a.P, a.Cin, a.Cout, L1);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(epi_reduce_kernel, dim3((unsigned)cdiv(E, 32)), dim3(256), 0, L->s, a.part,
                     L->G, E, (int64_t)a.Cout * a.Cin, L->gw, L->gb);
  return hipGetLastError();
}

hipError_t launch_wgrad(void* ctx) {
  EpiWgradLaunch* L = static_cast<EpiWgradLaunch*>(ctx);
  return L->es == 2 ? launch_wgrad_t<_Float16>(L) : launch_wgrad_t<float>(L);
}

}  // namespace
}  // namespace fno

using namespace fno;

extern "C" fno_status fno_block_epilogue_workspace_size(const fno_block_desc* d, fno_op op,
                                                        size_t* bytes) {
  EpiGeo g;
  fno_status st = check_desc(d, &g);
  if (st != FNO_OK) return st;
  if (!bytes) return FNO_ERR_INVALID_ARGUMENT;
  if (op == FNO_OP_FWD || op == FNO_OP_BWD_DATA) {
    *bytes = 0;
  } else if (op == FNO_OP_BWD_WEIGHT) {
    *bytes = wgrad_ws_bytes(g);
  } else {
    return FNO_ERR_INVALID_ARGUMENT;
  }
  return FNO_OK;
}

extern "C" fno_status fno_block_epilogue_fwd(const fno_block_desc* d, const void* x,
                                             const void* y, const void* w_skip, const void* b,
                                             void* out, void* z_out, hipStream_t stream) {
  EpiGeo g;
  fno_status st = check_desc(d, &g);
  if (st != FNO_OK) return st;
  if (!ok16(x) || !ok16(y) || !ok16(w_skip) || !ok16(out) || !null_or16(b) || !null_or16(z_out))
    return FNO_ERR_INVALID_ARGUMENT;
  if (out == x || out == y || (z_out && (z_out == x || z_out == y || z_out == out)))
    return FNO_ERR_INVALID_ARGUMENT;
  return run_mix(g, "block_epilogue_fwd", x, g.Cin, w_skip, 0, g.Cout, y, nullptr, b, out, z_out,
                 g.act, g.residual, stream);
}

extern "C" fno_status fno_block_epilogue_bwd_weight(const fno_block_desc* d, const void* x,
                                                    const void* z, const void* g_out,
                                                    void* g_z, float* g_w_skip, float* g_b,
                                                    void* ws, size_t ws_len,
                                                    hipStream_t stream) {
  EpiGeo g;
  fno_status st = check_desc(d, &g);
  if (st != FNO_OK) return st;
  const bool gelu = g.act == FNO_EPI_ACT_GELU;
  if (!ok16(x) || !ok16(g_out) || !ok16(g_w_skip) || !null_or16(g_b))
    return FNO_ERR_INVALID_ARGUMENT;
  if (gelu && (!ok16(z) || !ok16(g_z) || g_z == g_out || g_z == z || g_z == x))
    return FNO_ERR_INVALID_ARGUMENT;
  if (ws_len < wgrad_ws_bytes(g)) return FNO_ERR_WORKSPACE_TOO_SMALL;
  if (!ok16(ws)) return FNO_ERR_INVALID_ARGUMENT;
  EpiWgradLaunch L{};
  EpiWgradArgs& a = L.a;
  a.x = x;
  a.z = gelu ? z : nullptr;
  a.gout = g_out;
  a.gz = gelu ? g_z : nullptr;
  a.part = reinterpret_cast<float*>(ws);
  a.B = g.B;
  a.P = g.P;
  a.Cin = g.Cin;
  a.Cout = g.Cout;
  a.act = g.act;
  L.es = g.es;
  L.G = wgrad_partials(g, &a.tiles, &a.ptiles);
  L.pipe = wgrad_pipe(g);
  L.fast = !L.pipe && wgrad_fast(g, &L.it, &L.og, &a.wpr);
  a.ranges = L.fast ? 4 / a.wpr : 0;
  L.gw = g_w_skip;
  L.gb = g_b;
  L.s = stream;
  const hipError_t e = timed_launch("block_epilogue_bwd_weight", stream, launch_wgrad, &L);
  return e == hipSuccess ? FNO_OK : report_hip_error(e, "block_epilogue_bwd_weight");
}

extern "C" fno_status fno_block_epilogue_bwd_data(const fno_block_desc* d, const void* g_z,
                                                  const void* w_skip, const void* gx_spec,
                                                  const void* g_out, void* gx,
                                                  hipStream_t stream) {
  EpiGeo g;
  fno_status st = check_desc(d, &g);
  if (st != FNO_OK) return st;
  if (!ok16(g_z) || !ok16(w_skip) || !ok16(gx_spec) || !ok16(gx)) return FNO_ERR_INVALID_ARGUMENT;
  if (g.residual && !ok16(g_out)) return FNO_ERR_INVALID_ARGUMENT;
  if (gx == g_z || (g.residual && gx == g_out)) return FNO_ERR_INVALID_ARGUMENT;
  return run_mix(g, "block_epilogue_bwd_data", g_z, g.Cout, w_skip, 1, g.Cin, gx_spec,
                 g.residual ? g_out : nullptr, nullptr, gx, nullptr, FNO_EPI_ACT_NONE, 0, stream);
}
