// Per-mode channel contraction and weight gradient on slabs of 16 modes
// (fp16 storage, K a multiple of 16).
//
// Spectra and weights keep the mode index innermost, so a row of one
// (batch, channel) or (channel, channel) pair holds consecutive modes.  A
// work-group takes 16 consecutive modes (64-byte row segments: four lanes
// read one segment, one load instruction covers 16 rows) of a tile of
// output rows and columns, and runs the reduction in chunks of 16 complex
// values:
//
//   contract   out[b][p][t] = s c(t) sum_q X[b][q][t] W(q, p, t),
//              W(q, p) = W[q][p] (forward) or conj(W[p][q]) (adjoint)
//   wgrad      gw[q][p][t]  = s c(t) sum_b conj(X[b][q][t]) G[b][p][t]   (fp32)
//
// Each chunk is staged in LDS with the reduction index innermost (a 4 x 4
// register transpose per thread, one 16-byte LDS store per mode), then every
// wave multiplies its two modes with the complex product written as two
// real MFMAs over interleaved (re, im) k-slots: A = (re, im) pairs of the
// rows; B = (Wr, -Wi) for the real part and (Wi, Wr) for the imaginary part
// (and the conjugated/transposed variants), made from one LDS fragment by a
// sign flip and a half swap.  The next chunk is in flight in registers while
// one is multiplied; loads past the operands' ends read zeros (buffer range
// check), so every load is issued.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

namespace {

typedef MM<_Float16> MH;
constexpr int SL_TM = 16;  // modes per slab
constexpr int SL_RC = 16;  // reduction entries per chunk (one MFMA k-step)
constexpr int SL_AR = 16;  // A rows per tile (b for contract, q for wgrad)
constexpr int SL_BC = 32;  // B columns per tile (p)
constexpr int SL_NT = 512;
constexpr int SL_MPW = SL_TM / (SL_NT / 64);  // modes per wave
// LDS strides in dwords (one dword = one fp16 complex)
constexpr int RS = SL_RC + 4;          // row (16 complex + pad)
constexpr int AMS = SL_AR * RS + 4;    // A mode stride
constexpr int BMS = SL_BC * RS + 4;    // B mode stride
constexpr int A_DW = SL_TM * AMS;
constexpr int B_DW = SL_TM * BMS;

enum SlabOp { SLAB_FWD = 0, SLAB_ADJ = 1, SLAB_WGRAD = 2 };

__device__ __forceinline__ u32 swap_halves(u32 v) { return (v >> 16) | (v << 16); }

__device__ __forceinline__ h8 as_frag(const u32x4& v) {
  h8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// out-type staging strides (dwords)
template <SlabOp OP>
struct SlabOut;
template <>
struct SlabOut<SLAB_FWD> {
  static constexpr int DPM = 1;                 // dwords per mode value
  static constexpr int PS = SL_TM * 1 + 4;      // (row, col) stride
  static constexpr int RSO = SL_BC * PS + 4;    // row stride
};
template <>
struct SlabOut<SLAB_ADJ> : SlabOut<SLAB_FWD> {};
template <>
struct SlabOut<SLAB_WGRAD> {
  static constexpr int DPM = 2;
  static constexpr int PS = SL_TM * 2 + 4;
  static constexpr int RSO = SL_BC * PS + 4;
};

}  // namespace

struct SlabArgs {
  const void* a;      // contract: X [B][Q][K]; wgrad: X [B][Cin][K]
  const void* b;      // contract: W [wrows][wcols][K]; wgrad: G [B][Cout][K]
  void* out;          // contract: [B][P][K] fp16 complex; wgrad: [Cin][Cout][K] fp32 complex
  int a_bytes, b_bytes;  // operand sizes (< 2^30)
  int nrow, ncol, nred;  // A rows (B or Cin), B columns (P or Cout), reduction (Q or B)
  int K;
  int a_ld;           // contract: Q (X row = b * Q + q); wgrad: Cin (X row = b * Cin + q)
  int b_ld;           // contract: wcols; wgrad: Cout
  int Kb, Nb;
  float scale;
};

// One work-group's tile: block `bid` of `nblocks` blocks of this operation.
template <SlabOp OP>
__device__ __forceinline__ void slab_body(const SlabArgs& s, int bid, int nblocks,
                                          unsigned char* smem) {
  using OT = SlabOut<OP>;
  u32* sA = reinterpret_cast<u32*>(smem);  // [mode][A row][reduction]
  u32* sB = sA + A_DW;                      // [mode][B col][reduction]
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int nrt = (s.nrow + SL_AR - 1) / SL_AR, nct = (s.ncol + SL_BC - 1) / SL_BC;
  const int lid = xcd_logical_block(bid, nblocks);
  const int t0 = (lid / (nrt * nct)) * SL_TM;
  const int row0 = ((lid / nct) % nrt) * SL_AR;
  const int col0 = (lid % nct) * SL_BC;
  // Buffer loads.  The byte offset of each load is a per-lane part (row or
  // column, mode quad, the lane's reduction sub-index) plus a uniform part
  // (chunk and load index) passed as the scalar offset, so the loads need no
  // per-load address registers.  Per-lane offsets past an operand's size
  // read zeros: lanes of out-of-range rows or columns carry a large per-lane
  // part, and so do reduction entries past the end (partial or empty chunks).
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(s.a), (short)0, s.a_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(s.b), (short)0, s.b_bytes, 0x00020000);
  constexpr int BIG = 0x40000000;  // beyond every operand (sizes < 2^30 bytes)

  // load tasks, one of each per thread: A: (row 16) x (reduction pair 8) x
  // (mode quad 4) = 512, two loads; B: (col 32) x (reduction quad 4) x (mode
  // quad 4) = 512, four loads.  Lanes take the four mode quads of a row
  // segment, then reduction groups, then rows.
  const int a_mq = tid & 3, a_rp = (tid >> 2) & 7, a_row = tid >> 5;
  const int b_mq = tid & 3, b_rq = (tid >> 2) & 3, b_col = tid >> 4;
  const int K4 = s.K * 4;
  // bytes per reduction step of each operand
  const int a_rstep = OP == SLAB_WGRAD ? s.a_ld * K4 : K4;
  const int b_rstep = OP == SLAB_ADJ ? K4 : s.b_ld * K4;
  int a_lane, b_lane;
  {
    const int row = row0 + a_row, col = col0 + b_col;
    if constexpr (OP == SLAB_WGRAD) a_lane = row * K4;            // X[b][q = row]
    else a_lane = row * s.a_ld * K4;                              // X[b = row][q]
    a_lane += 2 * a_rp * a_rstep + (t0 + 4 * a_mq) * 4;
    if constexpr (OP == SLAB_ADJ) b_lane = col * s.b_ld * K4;     // W[p = col][q]
    else b_lane = col * K4;                                       // W[q][p], G[b][p]
    b_lane += 4 * b_rq * b_rstep + (t0 + 4 * b_mq) * 4;
    if (row >= s.nrow) a_lane = BIG;
    if (col >= s.ncol) b_lane = BIG;
  }

  struct Chunk {
    u32x4 a[2], b[4];
  };
  // The range check covers the per-lane offset only, so every out-of-range
  // case is expressed there (the scalar part is 0 for them).
  auto load = [&](int c, Chunk& ch) {
    const int rbase = c * SL_RC;
    const bool part = rbase + SL_RC > s.nred;  // uniform: partial or empty chunk
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bool out = part && rbase + 2 * a_rp + j >= s.nred;
      const int vo = out ? BIG : a_lane;
      const int so = rbase >= s.nred ? 0 : (rbase + j) * a_rstep;
      ch.a[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, vo, so, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool out = part && rbase + 4 * b_rq + j >= s.nred;
      const int vo = out ? BIG : b_lane;
      const int so = rbase >= s.nred ? 0 : (rbase + j) * b_rstep;
      ch.b[j] = __builtin_amdgcn_raw_buffer_load_b128(rb, vo, so, 0);
    }
  };
  // register transposes: word e of load j is reduction entry j of mode e
  auto stage = [&](const Chunk& ch) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const u32x2 v = {ch.a[0][e], ch.a[1][e]};
      *reinterpret_cast<u32x2*>(sA + (4 * a_mq + e) * AMS + a_row * RS + 2 * a_rp) = v;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const u32x4 v = {ch.b[0][e], ch.b[1][e], ch.b[2][e], ch.b[3][e]};
      *reinterpret_cast<u32x4*>(sB + (4 * b_mq + e) * BMS + b_col * RS + 4 * b_rq) = v;
    }
  };

  f4 accR[SL_MPW][2], accI[SL_MPW][2];
#pragma unroll
  for (int m = 0; m < SL_MPW; ++m)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) accR[m][ct] = accI[m][ct] = f4zero();

  auto multiply = [&]() {
#pragma unroll
    for (int mm = 0; mm < SL_MPW; ++mm) {
      const int m = SL_MPW * wave + mm;
      const h8 af = as_frag(*reinterpret_cast<const u32x4*>(sA + m * AMS + r16 * RS + 4 * g));
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const u32x4 raw =
            *reinterpret_cast<const u32x4*>(sB + m * BMS + (16 * ct + r16) * RS + 4 * g);
        u32x4 br, bi;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (OP == SLAB_FWD) {        // (Wr, -Wi), (Wi, Wr)
            br[w] = raw[w] ^ 0x80000000u;
            bi[w] = swap_halves(raw[w]);
          } else if constexpr (OP == SLAB_ADJ) { // (Wr, Wi), (-Wi, Wr)
            br[w] = raw[w];
            bi[w] = swap_halves(raw[w]) ^ 0x00008000u;
          } else {                               // (Gr, Gi), (Gi, -Gr)
            br[w] = raw[w];
            bi[w] = swap_halves(raw[w]) ^ 0x80000000u;
          }
        }
        accR[mm][ct] = MH::mma(af, as_frag(br), accR[mm][ct]);
        accI[mm][ct] = MH::mma(af, as_frag(bi), accI[mm][ct]);
      }
    }
  };

  // The next chunk is in flight in registers while one is multiplied (two
  // chunks ahead would not fit the 128 registers that let two work-groups
  // share a CU); loads past the last chunk read zeros.
  const int nchunk = (s.nred + SL_RC - 1) / SL_RC;
  Chunk c0;
  load(0, c0);
  for (int c = 0; c < nchunk; ++c) {
    stage(c0);
    block_sync_lds();
    load(c + 1, c0);
    multiply();
    block_sync_lds();
  }

  // ---- epilogue: scale, stage [row][col][mode], write 16-byte row pieces ----
  u32* so = reinterpret_cast<u32*>(smem);
#pragma unroll
  for (int mm = 0; mm < SL_MPW; ++mm) {
    const int m = SL_MPW * wave + mm;
    const float sc = s.scale * cmult(t0 + m, s.Kb, s.Nb);
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rr = 4 * g + i, cc = 16 * ct + r16;
        u32* d = so + rr * OT::RSO + cc * OT::PS + m * OT::DPM;
        if constexpr (OP == SLAB_WGRAD) {
          *reinterpret_cast<f2*>(d) = f2{accR[mm][ct][i] * sc, accI[mm][ct][i] * sc};
        } else {
          *reinterpret_cast<h2*>(d) = h2{to_h(accR[mm][ct][i] * sc), to_h(accI[mm][ct][i] * sc)};
        }
      }
  }
  block_sync_lds();
  constexpr int PPR = SL_TM * OT::DPM / 4;  // 16-byte pieces per (row, col)
  constexpr int NPIECE = SL_AR * SL_BC * PPR;
#pragma unroll
  for (int k = 0; k < NPIECE / SL_NT; ++k) {
    const int idx = tid + SL_NT * k;
    const int v = idx % PPR, rc = idx / PPR;
    const int rr = rc / SL_BC, cc = rc % SL_BC;
    const int row = row0 + rr, col = col0 + cc;
    if (row < s.nrow && col < s.ncol) {
      const u32x4 val = *reinterpret_cast<const u32x4*>(so + rr * OT::RSO + cc * OT::PS + 4 * v);
      if constexpr (OP == SLAB_WGRAD) {
        // streaming store: the weight gradient is not read again here
        float* d = reinterpret_cast<float*>(s.out) + (((int64_t)row * s.ncol + col) * s.K + t0) * 2;
        __builtin_nontemporal_store(val, reinterpret_cast<u32x4*>(d) + v);
      } else {
        _Float16* d =
            reinterpret_cast<_Float16*>(s.out) + (((int64_t)row * s.ncol + col) * s.K + t0) * 2;
        reinterpret_cast<u32x4*>(d)[v] = val;
      }
    }
  }
}

template <SlabOp OP>
__global__ __launch_bounds__(SL_NT, 4) void slab_kernel(SlabArgs s) {
  extern __shared__ __align__(16) unsigned char smem[];
  slab_body<OP>(s, blockIdx.x, gridDim.x, smem);
}

// The adjoint contraction and the weight gradient of the backward pass in
// one launch: blocks [0, n1) are adjoint-contraction tiles, the rest weight-
// gradient tiles (both read the gradient spectrum; one launch instead of two,
// and each operation's waits are covered by the other's work).
__global__ __launch_bounds__(SL_NT, 4) void slab_adj_wgrad_kernel(SlabArgs s1, SlabArgs s2,
                                                                  int n1) {
  extern __shared__ __align__(16) unsigned char smem[];
  if ((int)blockIdx.x < n1) slab_body<SLAB_ADJ>(s1, blockIdx.x, n1, smem);
  else slab_body<SLAB_WGRAD>(s2, blockIdx.x - n1, gridDim.x - n1, smem);
}

size_t slab_lds_bytes(int op) {
  const int stage_dw = A_DW + B_DW;
  const int out_dw = op == SLAB_WGRAD ? SL_AR * SlabOut<SLAB_WGRAD>::RSO
                                      : SL_AR * SlabOut<SLAB_FWD>::RSO;
  return 4 * (size_t)(stage_dw > out_dw ? stage_dw : out_dw);
}

static hipError_t slab_launch(int op, const SlabArgs& s, hipStream_t st) {
  if (s.K % SL_TM != 0) return hipErrorNotSupported;
  const int64_t nblk = (int64_t)(s.K / SL_TM) * ((s.nrow + SL_AR - 1) / SL_AR) *
                       ((s.ncol + SL_BC - 1) / SL_BC);
  if (nblk > 0x7fffffff || nblk == 0) return hipErrorInvalidValue;
  const size_t lds = slab_lds_bytes(op);
  auto go = [&](auto kern) -> hipError_t {
    if (lds > 64 * 1024) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)nblk), dim3(SL_NT), lds, st, s);
    return hipGetLastError();
  };
  if (op == SLAB_FWD) return go(slab_kernel<SLAB_FWD>);
  if (op == SLAB_ADJ) return go(slab_kernel<SLAB_ADJ>);
  return go(slab_kernel<SLAB_WGRAD>);
}

static bool make_contract_slab(const ContractArgs& a, SlabArgs* out) {
  if ((int64_t)a.B * a.Q * a.K * 4 >= (1ll << 30) - 64 ||
      (int64_t)a.wrows * a.wcols * a.K * 4 >= (1ll << 30) - 64 ||
      (int64_t)a.B * a.P * a.K * 2 >= (1ll << 31) || a.K % SL_TM != 0)
    return false;
  SlabArgs s{};
  s.a = a.in;
  s.b = a.w;
  s.out = a.out;
  s.a_bytes = (int)((int64_t)a.B * a.Q * a.K * 4);
  s.b_bytes = (int)((int64_t)a.wrows * a.wcols * a.K * 4);
  s.nrow = a.B;
  s.ncol = a.P;
  s.nred = a.Q;
  s.K = a.K;
  s.a_ld = a.Q;
  s.b_ld = a.wcols;
  s.Kb = a.Kb;
  s.Nb = a.Nb;
  s.scale = a.scale;
  *out = s;
  return true;
}

static bool make_wgrad_slab(const WgradArgs& a, SlabArgs* out) {
  if ((int64_t)a.B * a.Cin * a.K * 4 >= (1ll << 30) - 64 ||
      (int64_t)a.B * a.Cout * a.K * 4 >= (1ll << 30) - 64 || a.K % SL_TM != 0)
    return false;
  SlabArgs s{};
  s.a = a.xh;
  s.b = a.gh;
  s.out = a.gw;
  s.a_bytes = (int)((int64_t)a.B * a.Cin * a.K * 4);
  s.b_bytes = (int)((int64_t)a.B * a.Cout * a.K * 4);
  s.nrow = a.Cin;
  s.ncol = a.Cout;
  s.nred = a.B;
  s.K = a.K;
  s.a_ld = a.Cin;
  s.b_ld = a.Cout;
  s.Kb = a.Kb;
  s.Nb = a.Nb;
  s.scale = a.scale;
  *out = s;
  return true;
}

static int64_t slab_blocks(const SlabArgs& s) {
  return (int64_t)(s.K / SL_TM) * ((s.nrow + SL_AR - 1) / SL_AR) *
         ((s.ncol + SL_BC - 1) / SL_BC);
}

hipError_t launch_contract_slab(const ContractArgs& a, hipStream_t st) {
  SlabArgs s;
  if (!make_contract_slab(a, &s)) return hipErrorNotSupported;
  return slab_launch(a.adjoint ? SLAB_ADJ : SLAB_FWD, s, st);
}

hipError_t launch_wgrad_slab(const WgradArgs& a, hipStream_t st) {
  SlabArgs s;
  if (!make_wgrad_slab(a, &s)) return hipErrorNotSupported;
  return slab_launch(SLAB_WGRAD, s, st);
}

bool contract_slab_supported(const ContractArgs& a) {
  SlabArgs s;
  return make_contract_slab(a, &s) && slab_blocks(s) > 0 && slab_blocks(s) <= 0x7fffffff;
}

bool wgrad_slab_supported(const WgradArgs& a) {
  SlabArgs s;
  return make_wgrad_slab(a, &s) && slab_blocks(s) > 0 && slab_blocks(s) <= 0x7fffffff;
}

bool adj_wgrad_slab_supported(const ContractArgs& adj, const WgradArgs& wg) {
  SlabArgs s1, s2;
  return adj.adjoint && make_contract_slab(adj, &s1) && make_wgrad_slab(wg, &s2) &&
         slab_blocks(s1) > 0 && slab_blocks(s2) > 0 &&
         slab_blocks(s1) + slab_blocks(s2) <= 0x7fffffff;
}

hipError_t launch_adj_wgrad_slab(const ContractArgs& adj, const WgradArgs& wg, hipStream_t st) {
  if (!adj_wgrad_slab_supported(adj, wg)) return hipErrorNotSupported;
  SlabArgs s1, s2;
  make_contract_slab(adj, &s1);
  make_wgrad_slab(wg, &s2);
  const int64_t n1 = slab_blocks(s1), n2 = slab_blocks(s2);
  const size_t lds = slab_lds_bytes(SLAB_WGRAD);  // the larger of the two
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(slab_adj_wgrad_kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(slab_adj_wgrad_kernel, dim3((unsigned)(n1 + n2)), dim3(SL_NT), lds, st, s1,
                     s2, (int)n1);
  return hipGetLastError();
}

}  // namespace fno
