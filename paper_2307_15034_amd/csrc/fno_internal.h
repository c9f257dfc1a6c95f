// Internal interfaces between the host planner (fno_plan.cpp) and the HIP
// kernels (fno_kernels.hip).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fno {

enum Elem { ELEM_F32 = 0, ELEM_F16 = 1 };
// Pre-activation of a plan (the `act` codes of the kernel arguments).
enum Act { ACT_NONE = 0, ACT_TANH = 1, ACT_CLIP = 2, ACT_SIGMA = 3 };

// Truncated real-to-complex transform of the last two axes of every plane
// [planes][Na][Nb] -> spectrum [planes][Ka][Kb] (complex).  Step A runs the
// last axis (Nb reals -> Kb complex, scaled by sA), step B the other axis
// (Na -> Ka complex, scaled by sB), both as DFT-by-MFMA with twiddle tables.
struct R2CArgs {
  const void* in;
  void* out;
  const void* zeros;  // >= 256 zero bytes: target of out-of-range lanes' loads
  const void* twA;  // [2*Kbp][Nbp]: rows t < Kbp: cos(2 pi t n / Nb), rows Kbp+t: -sin
  const void* cB;   // [Kap16][Nap]: cos(2 pi k_a(t) n / Na)
  const void* sB;   // [Kap16][Nap]: sin(2 pi k_a(t) n / Na)
  int64_t planes;
  int Na, Nb, Ka, Kb;
  int Kbp;          // Kb padded: 16 * NCT / 2
  int Nbp;          // Nb padded to 32
  int Nap;          // Na padded to a multiple of R
  int Kap16;        // Ka padded to 16
  int R;            // rows per chunk (multiple of 32)
  float scaleA, scaleB;
  int do_tanh;      // 1 if the pre-activation u = f(x) is applied (any act)
  int act;          // arithmetic kernels: 0 none, 1 tanh, 2 hard clip to [-clip, clip]
  float clip;
  int vec;          // 1 if Nb allows 16-byte row loads
  // chained fast path (fp16): permuted copies of the tables
  const void* twAc; // [2*Kbp][Nbp]: row 16 ct + r: part ct / (Kbp/16) of t = (Kbp/16) r + ct % (Kbp/16)
  const void* cBc;  // [Kap16][NaC]: column 32 j + 8 q + e holds row n = 32 j + 4 q + e (e < 4)
  const void* sBc;  //   or 32 j + 16 + 4 q + e - 4 (e >= 4)
  int NaC;          // Na padded to 32
  const void* lut;  // fp16 f(x) of every non-negative fp16 code (32768 entries; f odd)
  int lut_sat;      // first code from which f stays at its +inf value
  // ACT_SIGMA (table-free kernels only): per statistics group (batch x
  // channel) the clip bounds (lo, hi) in double; plane p uses group p / bgroup
  const double* bounds;
  int bgroup;
  // radix-2 wide-plane forward, narrow variant: 1 requests a work item's
  // step-B tables at its start and the next item's rows during its last two
  // slices (more registers held per wave)
  int early;
};

// Inverse of the above: spectrum [planes][Ka][Kb] -> y [planes][Na][Nb],
// y = scale * sum_t Re(Z e^{+i theta}) (no multiplicity), optional epilogue
// y *= f'(x), the derivative of the pre-activation.
struct C2RArgs {
  const void* in;
  void* out;
  const void* zeros;  // >= 256 zero bytes: target of out-of-range lanes' loads
  const void* x;    // epilogue input or null
  const void* cI;   // [Nap][Kap]: cos(2 pi k_a(t) n / Na)   (row n, col t)
  const void* sI;   // [Nap][Kap]: sin(2 pi k_a(t) n / Na)
  const void* twI;  // [Nbp16][2*Kbp]: cols t < Kbp: cos(2 pi t n / Nb), Kbp+t: -sin
  int64_t planes;
  int Na, Nb, Ka, Kb;
  int Kbp, Kap;     // Kap = Ka padded to 32
  int Nap;          // Na padded to a multiple of R
  int R;            // rows per chunk (multiple of 64)
  float scale;
  int epilogue;     // 0: none, 1: multiply by f'(x)
  int act;          // arithmetic kernels: 1 tanh, 2 hard clip to [-clip, clip]
  float clip;
  int vec;
  // chained fast path (fp16): [Nb64][2*Kbp], row 16 T + R holds column
  // n = 64 (T/4) + 16 (R/4) + 4 (T%4) + R%4; column 32 ks + 8 q + e holds
  // part/tile pair 2 ks + e/4 (Re tiles first) at t = 16 tile + 4 q + e%4
  const void* twIc;
  const void* cIc;  // [Nap][Kap] like cI, sI with column 32 ks + 8 q + e holding
  const void* sIc;  //   t = 32 ks + 4 q + e (e < 4) or 32 ks + 16 + 4 q + e - 4
  const void* lut;  // fp16 f'(x) of every non-negative fp16 code (32768 entries; f' even)
  int lut_sat;      // first code from which f' stays at its +inf value
  const double* bounds;  // ACT_SIGMA: as in R2CArgs
  int bgroup;
};

// Clip bounds of the statistics-based pre-activation: for each of `groups`
// contiguous groups of n values of x (fp16 or fp32), mean -/+ k population
// standard deviations, in double (NaN when not finite).
hipError_t launch_sigma_stats(int elem, const void* x, int64_t groups, int64_t n, double k,
                              double* bounds, hipStream_t s);

// Complex DFT along a middle axis: in [outer][Lin][inner] -> out
// [outer][Lout][inner], out[o][t][j] = scale * sum_l E[t][l] in[o][l][j].
struct AxisArgs {
  const void* in;
  void* out;
  const void* er;   // [Lout16][Linp] Re E
  const void* ei;   // [Lout16][Linp] Im E
  int64_t outer;
  int Lin, Lout, inner;
  int Linp;         // Lin padded to 32
  int Lout16;
  float scale;
};

// Per-mode channel contraction:
//   out[b][p][t] = scale * c(t) * sum_q in[b][q][t] * Wop(q, p, t)
//   Wop = W[q][p][t] (forward) or conj(W[p][q][t]) (adjoint).
struct ContractArgs {
  const void* in;
  const void* w;
  void* out;
  const void* zeros;  // >= 256 zero bytes: target of out-of-range lanes' loads
  int B, Q, P, K;
  int wrows, wcols;  // W is [wrows][wcols][K]
  int adjoint;
  int Kb, Nb;        // last-axis retained count and length (for c(t))
  float scale;
};

// Batch-reduced weight gradient:
//   gw[q][p][t] = scale * c(t) * sum_b conj(xh[b][q][t]) * gh[b][p][t]   (fp32)
struct WgradArgs {
  const void* xh;
  const void* gh;
  float* gw;
  const void* zeros;  // >= 256 zero bytes: target of out-of-range lanes' loads
  int B, Cin, Cout, K;
  int Kb, Nb;
  float scale;
};

// Generic pairwise complex contraction for the Tucker path (fp32 or fp16 complex
// intermediates; operand element type given per operand).
//   out[m, n, ...] (batch, free-A, free-B index groups, row-major in the
//   result's own index order) = sum_k A * B, with optional conjugation.
constexpr int PW_MAXIDX = 8;
struct PairArgs {
  const void* a;
  const void* b;
  void* out;           // complex of out_elem
  int a_elem, b_elem;  // Elem of each operand
  int out_elem;
  int conj_a, conj_b;
  int64_t out_size;
  int n_out;           // number of result indices
  int64_t out_ext[PW_MAXIDX];     // extents in result order
  int64_t a_stride_out[PW_MAXIDX];// stride of A per result index (0 if absent)
  int64_t b_stride_out[PW_MAXIDX];
  int n_red;           // contracted indices
  int64_t red_ext[PW_MAXIDX];
  int64_t a_stride_red[PW_MAXIDX];
  int64_t b_stride_red[PW_MAXIDX];
  int64_t red_size;
  float scale;
  int scale_c_axis;    // result index position of the last spatial axis for c(t), -1 none
  int Nb;              // last-axis length for c(t)
  // Register blocking (set by launch_pair): result index blk_k, absent from
  // A, is covered PB_NB values per thread so each A element loaded serves
  // them all; -1 for one result per thread.  res_stride: the result's own
  // strides.
  int blk_k;
  int64_t res_stride[PW_MAXIDX];
  // Room for split-K partial sums of the GEMM form (null: no split-K).
  void* part;
  size_t part_cap;
  // Division by out_ext[k] (and by the blocked index's block count) as a
  // multiply-high and shift (set by launch_pair; see div_magic).
  uint32_t out_mag[PW_MAXIDX], out_shr[PW_MAXIDX];
  uint32_t blk_mag, blk_shr;
};

// Division by an invariant integer (Granlund and Montgomery, "Division by
// invariant integers using multiplication", 1994): for 1 <= d < 2^32 with
// s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1, every 32-bit n has
// n / d = (n + mulhi(n, m)) >> s, the sum taken in 64 bits.
inline void div_magic(uint32_t d, uint32_t* m, uint32_t* s) {
  uint32_t l = 0;
  while (l < 32 && ((uint64_t)1 << l) < d) ++l;
  *s = l;
  *m = (uint32_t)((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d + 1);
}

// Bytes of every factorised-weight scratch area reserved for the split-K
// partial sums of one pairwise step.
constexpr size_t kPairPartBytes = (size_t)8 << 20;

hipError_t launch_r2c(int elem, int nct, const R2CArgs& a, size_t lds, hipStream_t s);
hipError_t launch_c2r(int elem, int nct, const C2RArgs& a, size_t lds, hipStream_t s);
hipError_t launch_axis(int elem, const AxisArgs& a, size_t lds, hipStream_t s);
hipError_t launch_contract(int elem, const ContractArgs& a, hipStream_t s);
hipError_t launch_wgrad(int elem, const WgradArgs& a, hipStream_t s);
hipError_t launch_pair(const PairArgs& a, hipStream_t s);
hipError_t launch_pair_gemm(const PairArgs& a, hipStream_t s);
// The mode-product form (a small factor applied along one index of a large
// dense operand); hipErrorNotSupported when the step is not of that form.
hipError_t launch_pair_modeprod(const PairArgs& a, hipStream_t s);
// The batch-innermost form (small products batched over the modes);
// hipErrorNotSupported when the step is not of that form.
hipError_t launch_pair_bt(const PairArgs& a, hipStream_t s);

// The Tucker weight gradient's three per-mode products in one launch (all
// fp32 complex, mode index t innermost, T modes):
//   R[a][e][t] = sum_b P[b][a][t] Q[b][e][t],
//   Z1[b][a][t] = sum_e Q[b][e][t] conj(S[a][e][t]),
//   Z2[b][e][t] = scale c(t) sum_a P[b][a][t] conj(S[a][e][t]),
// c(t) of the last axis index t % c_ext (1 at 0 and Nb/2, else 2; c_ext 0:
// none).  hipErrorNotSupported when B A + B E + A E > 1024.
struct TriArgs {
  const void* P;  // fp32 complex
  const void* Q;
  const void* S;
  void* R;
  void* Z1;
  void* Z2;
  int B, A, E;
  int64_t T;
  float scale;
  int c_ext, Nb;
};
hipError_t launch_tucker_tri(const TriArgs& g, hipStream_t s);
size_t r2c_wide_lds_bytes(int nct, bool pre, int lut_sat);
size_t c2r_wide_lds_bytes(int nct, int Kap, bool epi, int lut_sat);
hipError_t launch_r2c_wide(const R2CArgs& a, int nct, int grid, size_t lds, hipStream_t s);
hipError_t launch_c2r_wide(const C2RArgs& a, int nct, int grid, size_t lds, hipStream_t s);
hipError_t launch_scale_complex(float* p, int64_t n, float s, hipStream_t st);

// Persistent fp16 fast paths (planes up to 128 x 256); hipErrorNotSupported
// when no instantiation matches the shape.
// nw: waves per work-group, one per 16-row tile of the plane.
hipError_t launch_r2c_fast(const R2CArgs& a, int nct, int nka, int nw, int grid, size_t lds,
                           hipStream_t s);
hipError_t launch_c2r_fast(const C2RArgs& a, int nct, int nw, int nbt, int nkz, int grid,
                           size_t lds, hipStream_t s);
size_t r2c_fast_lds_bytes(int nct, int nka, int nw, int Kap16, int Nap);
size_t c2r_fast_lds_bytes(int nct, int nw, int nbt, int nkz);

// Chained fp16 transforms, one wavefront per plane (Na <= 128, Nb <= 256):
// nka = Nbp/32, ntb = Kbp/16, nta = Kap16/16 (forward); ng = Nb64/64,
// nkz = Kap/32 (inverse).  hipErrorNotSupported when not instantiated.
hipError_t launch_r2c_chain(const R2CArgs& a, int nka, int ntb, int nta, int grid, size_t lds,
                            hipStream_t s);
hipError_t launch_c2r_chain(const C2RArgs& a, int ng, int ntb, int nkz, int grid, size_t lds,
                            hipStream_t s);
bool r2c_chain_has(int nka, int ntb, int nta);
bool c2r_chain_has(int ng, int ntb, int nkz);
// dynamic LDS only; a lookup table adds 64 KiB of static LDS
size_t r2c_chain_lds_bytes(int nka, int ntb, int nta, int NaC, bool pre_lut);
size_t c2r_chain_lds_bytes(int ng, int ntb, int Kap, int Na, bool grad_lut);
constexpr int kChainWaves = 8;  // waves per work-group of the chained kernels

// fp16 contraction / weight gradient on slabs of 16 modes (K % 16 == 0,
// operands under 1 GiB: 32-bit buffer offsets); hipErrorNotSupported
// otherwise.  The *_supported predicates say beforehand whether a launch
// would be taken, so that callers pick the generic kernels instead.
bool contract_slab_supported(const ContractArgs& a);
bool wgrad_slab_supported(const WgradArgs& a);
hipError_t launch_contract_slab(const ContractArgs& a, hipStream_t s);
hipError_t launch_wgrad_slab(const WgradArgs& a, hipStream_t s);
// Adjoint contraction and weight gradient in one launch (fp16 slab path).
bool adj_wgrad_slab_supported(const ContractArgs& adj, const WgradArgs& wg);
hipError_t launch_adj_wgrad_slab(const ContractArgs& adj, const WgradArgs& wg, hipStream_t s);

// Radix-2 wide-plane transforms (fno_wide2.hip): the radix-2 tables in the
// table fields; hipErrorNotSupported when the shape is not one of the path's.
size_t r2c_wide2_lds_bytes(int nctc, bool pre, int lut_sat);
size_t c2r_wide2_lds_bytes(int nctc, int nkzh, bool epi, int lut_sat);
hipError_t launch_r2c_wide2(const R2CArgs& a, int nctc, int grid, size_t lds, hipStream_t s);
hipError_t launch_c2r_wide2(const C2RArgs& a, int nctc, int grid, size_t lds, hipStream_t s);

size_t r2c_lds_bytes(int elem, int Kbp, int R);
size_t c2r_lds_bytes(int elem, int Kbp, int Kap, int R);
size_t axis_lds_bytes(int elem, int Linp);

}  // namespace fno
