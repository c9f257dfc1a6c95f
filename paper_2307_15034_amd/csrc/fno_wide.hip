// Truncated transforms of large fp16 planes: Na a multiple of 256, Nb a
// multiple of 128, 2*Kbp in {64, 128} real last-axis columns, up to 128
// retained leading-axis modes (the 256^2 and 1024^2 workloads).  Same
// arithmetic as the generic plane kernels (DFT-by-MFMA with the twiddle
// tables of the plan, v_mfma_f32_16x16x32_f16, fp32 accumulation), laid out
// for bandwidth:
//   - persistent work-groups of eight waves walk (plane, 256-row chunk)
//     items; each wave owns two 16-row tiles, so each twiddle fragment it
//     loads serves two products;
//   - the next k-step's (forward) or the next column tiles' (inverse) global
//     data is in flight while the current one is multiplied (register double
//     buffering, loads issued unconditionally so the waits stay exact); rows
//     are read with buffer loads, rows past the plane reading zero;
//   - the pre-activation f (tanh or the hard clip, forward) and its
//     derivative f' (backward epilogue) come from a table in LDS of the fp16 codes up to the code where the function
//     saturates, plus one NaN entry (three packed 16-bit operations pick the
//     entry), instead of fp32 arithmetic per element.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

namespace {

constexpr int WD_WAVES = 8;
constexpr int WD_R = 256;   // rows per chunk: 8 waves x 2 tiles x 16
constexpr int WD_PAD = 8;   // LDS row padding in halves
constexpr int WD_BIG = 0x40000000;  // buffer offset past every plane
constexpr int WD_NT = 2;    // cache policy of the inverse's stores: streaming
constexpr int WD_XD = 8;    // column tiles of x in flight (inverse epilogue)
constexpr int WD_AD = 4;    // k-steps of row data in flight (forward)

}  // namespace

// ---------------------------------------------------------------------------
// Forward: plane [Na][Nb] -> spectrum [Ka][Kb].  Step A (last axis) per
// chunk: Y[row][c] = sum_n u[row][n] twA[c][n] (c < Kbp: cos, else -sin),
// into LDS (transposed, fp16); step B (leading axis) accumulates
// X[t_a][t_b] += sum_rows (cB - i sB)[t_a][row] Y[row][t_b] over the chunks.
//
// The twiddles of step A go through LDS in slices of two k-steps (all 2 Kbp
// rows x 64 columns), double buffered: the whole work-group loads slice
// g + 2 into registers while slice g is multiplied, and writes slice g + 1
// to LDS before the barrier that ends slice g.  The slice sequence is the
// same for every item, so it simply wraps around at the item boundary.  The
// per-wave global loads are then the row stream (four k-steps ahead) and,
// once per chunk, the step-B tables; every load is waited for about four
// k-steps after its request (outstanding loads complete in order, so a
// short-latency load waited for early would also wait for the rows).
// ---------------------------------------------------------------------------
constexpr int WD_SK = 64;             // columns (n) per twiddle slice
constexpr int WD_LDT = WD_SK + WD_PAD;

template <int NCT, bool PRE>
__global__ __launch_bounds__(WD_WAVES * 64, 1) void r2c_wide_kernel(R2CArgs a) {
  typedef MM<_Float16> M;
  constexpr int KS = 32, NTB = NCT / 2, KBP = NCT * 8;
  constexpr int LDA = WD_R + WD_PAD;
  constexpr int TWP = 2 * KBP * WD_SK / 8 / (WD_WAVES * 64);  // 16-byte pieces per thread
  static_assert(TWP >= 1, "slice pieces");
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* ATr = reinterpret_cast<_Float16*>(smem);
  _Float16* ATi = ATr + KBP * LDA;
  _Float16* TWb = ATi + KBP * LDA;                  // [2][2 KBP][WD_LDT]
  _Float16* lut = TWb + 2 * 2 * KBP * WD_LDT;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const _Float16* twA = reinterpret_cast<const _Float16*>(a.twA);
  const _Float16* cB = reinterpret_cast<const _Float16*>(a.cB);
  const _Float16* sB = reinterpret_cast<const _Float16*>(a.sB);
  const us2 sat = {(unsigned short)a.lut_sat, (unsigned short)a.lut_sat};
  if (PRE) stage_lut<WD_WAVES * 64>(lut, a.lut, a.lut_sat);

  const int64_t plane_bytes = (int64_t)a.Na * a.Nb * 2;
  const int nks = a.Nb / KS;        // a multiple of 4 on this path
  const int ngr = nks / 2;          // twiddle slices per item (even)
  const int nch = a.Na / WD_R;
  // step-B share of this wave: spectrum row tile ta, column tiles tb0 + j*tbs
  const int nta = a.Kap16 >> 4;
  const int ta = wave % nta, tb0 = wave / nta, tbs = WD_WAVES / nta;

  // work items (plane, chunk) of this work-group, in order
  const int64_t nitems = a.planes > (int64_t)blockIdx.x
                             ? ((a.planes - 1 - blockIdx.x) / gridDim.x + 1) * nch
                             : 0;
  auto item_plane = [&](int64_t it) { return (int64_t)blockIdx.x + (it / nch) * gridDim.x; };
  auto item_chunk = [&](int64_t it) { return (int)(it % nch) * WD_R; };

  // Lane part of the row-data offset (the second row tile, 128 rows on, in
  // the scalar offset), formed from an opaque copy of the thread index where
  // it is used, so it is recomputed rather than held through the loops.
  auto row_lane = [&](int c0) {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return (c0 + wave * 16 + (t & 15)) * a.Nb * 2 + ((t >> 4) & 3) * 16;
  };
  const int rstep = WD_WAVES * 16 * a.Nb * 2;
  auto ldA = [&](const __amdgpu_buffer_rsrc_t& rs, int rb, int s, u32x4 (&v)[2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
      v[u] = __builtin_amdgcn_raw_buffer_load_b128(rs, rb + s * KS * 2, u * rstep, 0);
  };
  // twiddle slice gs: rows c < 2 KBP, columns gs * 64 + [0, 64); thread t
  // takes pieces t + 512 e (row piece / 8, 8 halves at (piece % 8) * 8)
  const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<_Float16*>(twA), (short)0, 2 * KBP * a.Nbp * 2, 0x00020000);
  auto ldTW = [&](int gs, u32x4 (&v)[TWP]) {
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * WD_WAVES * 64;
      v[e] = __builtin_amdgcn_raw_buffer_load_b128(rt, ((pc >> 3) * a.Nbp + (pc & 7) * 8) * 2,
                                                   gs * WD_SK * 2, 0);
    }
  };
  auto stTW = [&](const u32x4 (&v)[TWP], int buf) {
    _Float16* d = TWb + buf * (2 * KBP * WD_LDT);
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * WD_WAVES * 64;
      *reinterpret_cast<u32x4*>(d + (pc >> 3) * WD_LDT + (pc & 7) * 8) = v[e];
    }
  };

  f4 accR[NTB], accI[NTB];
  // row fragments of k-steps s .. s+3 (slot s % 4), each requested four
  // k-steps before it is multiplied; twiddle slices g + 1, g + 2 in flight
  u32x4 va[WD_AD][2];
  u32x4 twr[2][TWP];
  __amdgpu_buffer_rsrc_t rs = plane_rsrc(a.in, nitems > 0 ? item_plane(0) : 0, plane_bytes);
  if (nitems > 0) {
    ldTW(0, twr[0]);
    ldTW(1, twr[1]);
    const int rb = row_lane(0);
#pragma unroll
    for (int d = 0; d < WD_AD; ++d) ldA(rs, rb, d, va[d]);
    stTW(twr[0], 0);
  }
  __syncthreads();  // table and first slice staged

  for (int64_t it = 0; it < nitems; ++it) {
    const int64_t p = item_plane(it);
    const int c0 = item_chunk(it);
    if (c0 == 0) {
#pragma unroll
      for (int j = 0; j < NTB; ++j) accR[j] = accI[j] = f4zero();
    }
    const bool more = it + 1 < nitems;
    const __amdgpu_buffer_rsrc_t rsn = more ? plane_rsrc(a.in, item_plane(it + 1), plane_bytes) : rs;
    const int cn = more ? item_chunk(it + 1) : c0;

    // ---- step A ------------------------------------------------------------
    f4 acc[2][NCT];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[u][ct] = f4zero();
    // k-step k of the slice in LDS buffer buf
    auto mul = [&](const u32x4 (&v)[2], int buf, int k) {
      h8 af[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 w = v[u];
        if (PRE) {
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = lut2<true>(lut, w[e], sat);
        }
        af[u] = w_as_h8(w);
      }
      const _Float16* tb = TWb + buf * (2 * KBP * WD_LDT) + r16 * WD_LDT + k * KS + g * 8;
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const h8 bf = M::ld(tb + ct * 16 * WD_LDT);
#pragma unroll
        for (int u = 0; u < 2; ++u) acc[u][ct] = M::mma(af[u], bf, acc[u][ct]);
      }
    };
    // one slice: its two k-steps, then the next slice into LDS and a barrier
    auto slice = [&](int gs, int par, int rb, bool rows) {
      ldTW(gs + 2 < ngr ? gs + 2 : gs + 2 - ngr, twr[par]);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int s = 2 * gs + k;
        mul(va[(2 * par + k) % WD_AD], par, k);
        if (rows) ldA(rs, rb, s + WD_AD, va[(2 * par + k) % WD_AD]);
      }
      stTW(twr[1 - par], 1 - par);
      __syncthreads();
    };
#pragma nounroll
    for (int gs = 0; gs < ngr - 2; gs += 2) {
      const int rb = row_lane(c0);
      slice(gs, 0, rb, true);
      slice(gs + 1, 1, rb, true);
    }
    // last two slices: the next item's rows are requested after the step-B
    // tables
    slice(ngr - 2, 0, 0, false);
    slice(ngr - 1, 1, 0, false);
    {
      // LDS offsets formed here, not hoisted out of the item loop (registers)
      int lb = r16 * LDA + wave * 16 + 4 * g;
      asm volatile("" : "+v"(lb));
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          // column ct * 16 + r16: rows ct * 16 of [ATr | ATi] (ATi = ATr + KBP * LDA)
          _Float16* dst = ATr + lb + ct * 16 * LDA + WD_WAVES * 16 * u;
#pragma unroll
          for (int i = 0; i < 4; ++i) dst[i] = to_h(acc[u][ct][i] * a.scaleA);
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // accumulators dead before the tables load
    // step-B tables of this chunk, then the next item's first row fragments
    // (operands selected, not branched on: one load sequence, exact waits)
    constexpr int NKB = WD_R / KS;
    h8 cfs[NKB], sfs[NKB];
#pragma unroll
    for (int k = 0; k < NKB; ++k) {
      const int64_t toff = (int64_t)(ta * 16 + r16) * a.Nap + c0 + k * KS + g * 8;
      cfs[k] = M::ld(cB + toff);
      sfs[k] = M::ld(sB + toff);
    }
    {
      const int rb = row_lane(cn);
#pragma unroll
      for (int d = 0; d < WD_AD; ++d) ldA(more ? rsn : rs, rb, more ? d : nks - 1, va[d]);
    }
    __syncthreads();

    // ---- step B ------------------------------------------------------------
#pragma unroll
    for (int k = 0; k < NKB; ++k) {
      const int k0 = k * KS;
      const h8 nsf = M::neg(sfs[k]);
#pragma unroll
      for (int j = 0; j < NTB; ++j) {
        // (column tiles past NTB are computed from a clamped tile and never
        // stored: no branch, so no copies of the accumulators)
        const int tb = min(tb0 + j * tbs, NTB - 1);
        const h8 ar = M::ld(ATr + (tb * 16 + r16) * LDA + k0 + g * 8);
        const h8 ai = M::ld(ATi + (tb * 16 + r16) * LDA + k0 + g * 8);
        accR[j] = M::mma(cfs[k], ar, accR[j]);
        accR[j] = M::mma(sfs[k], ai, accR[j]);
        accI[j] = M::mma(cfs[k], ai, accI[j]);
        accI[j] = M::mma(nsf, ar, accI[j]);
      }
      __builtin_amdgcn_sched_barrier(0);  // bound the hoisting of LDS reads
    }
    __syncthreads();

    if (c0 + WD_R >= a.Na) {  // last chunk of the plane: store its spectrum
      const __amdgpu_buffer_rsrc_t ro = plane_rsrc(a.out, p, (int64_t)a.Ka * a.Kb * 4);
      // offsets formed here, not hoisted out of the item loop (registers)
      int ta0 = ta * 16 + 4 * g;
      asm volatile("" : "+v"(ta0));
#pragma unroll
      for (int j = 0; j < NTB; ++j) {
        const int tb = tb0 + j * tbs;
        if (tb >= NTB) continue;
        const int t_b = tb * 16 + r16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t_a = ta0 + i;
          if (t_a < a.Ka && t_b < a.Kb) {
            h2 v = {to_h(accR[j][i] * a.scaleB), to_h(accI[j][i] * a.scaleB)};
            uint32_t w;
            __builtin_memcpy(&w, &v, 4);
            __builtin_amdgcn_raw_buffer_store_b32(w, ro, (t_a * a.Kb + t_b) * 4, 0, 0);
          }
        }
      }
    }
    rs = rsn;
  }
}

// ---------------------------------------------------------------------------
// Inverse: spectrum [Ka][Kb] -> plane [Na][Nb], y = scale * sum Re(Z e^{+i
// theta}), optional epilogue y *= f'(x).  Per plane the spectrum is
// staged transposed in LDS (ZT[kb][ka]: real rows, then imaginary); per
// chunk step B' gives V[row][kb] = sum_ka (cI + i sI)[row][ka] Z[ka][kb] into
// LDS as [Re V | Im V] (each wave two 16-row tiles), and each wave then holds
// its rows of V in registers for step A', y[row][m] = sum_k V[row][k]
// twI[m][k], over blocks of 64 columns m.  The twiddles of a block go
// through LDS (double buffered, in the space V used: the whole work-group
// loads block b + 2 into registers while block b is multiplied and writes
// block b + 1 before the barrier that ends block b).  Each wave's 16 x 64
// result of a row tile passes through a per-wave fp32 LDS buffer so that
// every 16-byte store instruction writes eight whole 128-byte lines (a lane
// takes 8 consecutive outputs of two rows), and x of the epilogue is read in
// the same layout two blocks ahead.  The next item's step-B' table rows and spectrum are
// requested before this item's blocks (outstanding loads complete in
// order).
// ---------------------------------------------------------------------------
constexpr int WD_MB = 64;      // output columns per block of step A'
constexpr int WD_LDO = 68;     // transpose buffer row stride (floats)

template <int NCT, int NKZ>
struct C2RWide {
  static constexpr int KBP = NCT * 8;
  static constexpr int LDV = 2 * KBP + WD_PAD;
  static constexpr int LDZ = NKZ * 32 + WD_PAD;
  static constexpr int LDT = 2 * KBP + WD_PAD;
  static constexpr size_t zt_bytes = (size_t)2 * KBP * LDZ * 2;
  static constexpr size_t vl_bytes = (size_t)WD_R * LDV * 2;
  static constexpr size_t tw_bytes = (size_t)2 * WD_MB * LDT * 2;
  static constexpr size_t ob_bytes = (size_t)WD_WAVES * 16 * WD_LDO * 4;
  static constexpr size_t reg_bytes = vl_bytes > tw_bytes + ob_bytes ? vl_bytes : tw_bytes + ob_bytes;
};

template <int NCT, int NKZ, bool EPI>
__global__ __launch_bounds__(WD_WAVES * 64, 1) void c2r_wide_kernel(C2RArgs a) {
  typedef MM<_Float16> M;
  typedef C2RWide<NCT, NKZ> L;
  constexpr int KS = 32, NTB = NCT / 2, KBP = NCT * 8;
  constexpr int NKV = NCT / 2;          // k-steps of step A' (2 Kbp / 32)
  constexpr int LDV = L::LDV, LDZ = L::LDZ, LDT = L::LDT;
  constexpr int ZQ = 4;                 // 16-byte spectrum pieces per thread
  constexpr int TWP = 2 * KBP * WD_MB / 8 / (WD_WAVES * 64);  // twiddle pieces per thread
  static_assert(TWP >= 1, "block pieces");
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* ZT = reinterpret_cast<_Float16*>(smem);                      // [2 KBP][LDZ]
  unsigned char* reg = smem + L::zt_bytes;
  _Float16* VL = reinterpret_cast<_Float16*>(reg);                       // [WD_R][LDV]
  _Float16* TW = reinterpret_cast<_Float16*>(reg);                       // [2][WD_MB][LDT]
  float* OB = reinterpret_cast<float*>(reg + L::tw_bytes);               // [8][16][WD_LDO]
  _Float16* lut = reinterpret_cast<_Float16*>(reg + L::reg_bytes);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const _Float16* cI = reinterpret_cast<const _Float16*>(a.cI);
  const _Float16* sI = reinterpret_cast<const _Float16*>(a.sI);
  const _Float16* twI = reinterpret_cast<const _Float16*>(a.twI);
  const us2 sat = {(unsigned short)a.lut_sat, (unsigned short)a.lut_sat};
  float* ob = OB + wave * 16 * WD_LDO;

  const int64_t plane_bytes = (int64_t)a.Na * a.Nb * 2;
  const int spec_bytes = a.Ka * a.Kb * 4;
  const int nch = a.Na / WD_R;
  const int nmb = a.Nb / WD_MB;          // even on this path
  const int nq = a.Ka * a.Kb / 4;        // 16-byte spectrum pieces
  const int64_t nitems = a.planes > (int64_t)blockIdx.x
                             ? ((a.planes - 1 - blockIdx.x) / gridDim.x + 1) * nch
                             : 0;
  auto item_plane = [&](int64_t it) { return (int64_t)blockIdx.x + (it / nch) * gridDim.x; };
  auto item_chunk = [&](int64_t it) { return (int)(it % nch) * WD_R; };

  // the padding of ZT stays zero: every plane writes the same positions
  for (int i = tid; i < 2 * KBP * LDZ; i += WD_WAVES * 64) ZT[i] = (_Float16)0.0f;
  if (EPI) stage_lut<WD_WAVES * 64>(lut, a.lut, a.lut_sat);

  auto ldZ = [&](int64_t p, u32x4 (&zq)[ZQ]) {
    const __amdgpu_buffer_rsrc_t rz = plane_rsrc(a.in, p, spec_bytes);
#pragma unroll
    for (int q = 0; q < ZQ; ++q) {
      const int i = tid + q * WD_WAVES * 64;
      zq[q] = __builtin_amdgcn_raw_buffer_load_b128(rz, i < nq ? i * 16 : WD_BIG, 0, 0);
    }
  };
  auto stZ = [&](const u32x4 (&zq)[ZQ]) {
    const int qpr = a.Kb / 4;
#pragma unroll
    for (int q = 0; q < ZQ; ++q) {
      const int i = tid + q * WD_WAVES * 64;
      if (i < nq) {
        const int ka = i / qpr, kb0 = (i - ka * qpr) * 4;
        const h8 v = w_as_h8(zq[q]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ZT[(kb0 + e) * LDZ + ka] = v[2 * e];
          ZT[(KBP + kb0 + e) * LDZ + ka] = v[2 * e + 1];
        }
      }
    }
  };
  auto ldC = [&](int c0, h8 (&cf)[2][NKZ], h8 (&sf)[2][NKZ]) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t row = c0 + (wave + WD_WAVES * u) * 16 + r16;
#pragma unroll
      for (int k = 0; k < NKZ; ++k) {
        cf[u][k] = M::ld(cI + row * a.Kap + k * KS + g * 8);
        sf[u][k] = M::ld(sI + row * a.Kap + k * KS + g * 8);
      }
    }
  };
  // twiddle block b: rows m = b * 64 + [0, 64), all 2 KBP columns; thread t
  // takes pieces t + 512 e (row piece / (KBP / 4), 8 halves at the rest * 8)
  const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<_Float16*>(twI), (short)0, a.Nb * 2 * KBP * 2, 0x00020000);
  constexpr int PPR = 2 * KBP / 8;  // pieces per twiddle row
  auto ldTW = [&](int b, u32x4 (&v)[TWP]) {
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * WD_WAVES * 64;
      v[e] = __builtin_amdgcn_raw_buffer_load_b128(rt, ((pc / PPR) * 2 * KBP + (pc % PPR) * 8) * 2,
                                                   b * WD_MB * 2 * KBP * 2, 0);
    }
  };
  auto stTW = [&](const u32x4 (&v)[TWP], int buf) {
    _Float16* d = TW + buf * (WD_MB * LDT);
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * WD_WAVES * 64;
      *reinterpret_cast<u32x4*>(d + (pc / PPR) * LDT + (pc % PPR) * 8) = v[e];
    }
  };
  // x (or y) offset of this lane in the transposed layout: row
  // lane / 8 + 8 h of row tile u, 8 columns at (lane % 8) * 8 of block b, so
  // that each 16-byte access instruction covers eight whole 128-byte lines
  auto xoff = [&](int c0, int u, int b, int h) {
    return (c0 + (wave + WD_WAVES * u) * 16 + (lane >> 3) + 8 * h) * a.Nb * 2 +
           (b * WD_MB + (lane & 7) * 8) * 2;
  };
  auto ldX = [&](const __amdgpu_buffer_rsrc_t& rx, int c0, int b, u32x4 (&v)[2][2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        v[u][h] = __builtin_amdgcn_raw_buffer_load_b128(rx, xoff(c0, u, b, h), 0, 0);
  };

  u32x4 zq[ZQ];
  h8 cf[2][NKZ], sf[2][NKZ];
  u32x4 twr[2][TWP];   // twiddle blocks b + 1, b + 2 in flight
  u32x4 xr[2][2][2];   // x of blocks b + 1, b + 2 (slot b % 2)
  if (nitems > 0) {
    ldZ(item_plane(0), zq);
    ldC(0, cf, sf);
    ldTW(0, twr[0]);
    ldTW(1, twr[1]);
    if (EPI) {
      const __amdgpu_buffer_rsrc_t rx = plane_rsrc(a.x, item_plane(0), plane_bytes);
      ldX(rx, 0, 0, xr[0]);
      ldX(rx, 0, 1, xr[1]);
    }
  }
  __syncthreads();  // ZT cleared, table staged

  for (int64_t it = 0; it < nitems; ++it) {
    const int64_t p = item_plane(it);
    const int c0 = item_chunk(it);
    const bool more = it + 1 < nitems;
    const int64_t pn = more ? item_plane(it + 1) : p;
    const int cn = more ? item_chunk(it + 1) : c0;
    if (c0 == 0) {
      stZ(zq);
      __syncthreads();
    }

    // ---- step B': V for rows c0 + (wave + 8u) * 16 + [0, 16), two column
    // tiles of kb at a time (register pressure) ------------------------------
    constexpr int TBH = NTB < 2 ? NTB : 2;
#pragma unroll
    for (int tbh = 0; tbh < NTB; tbh += TBH) {
      f4 vr[2][TBH], vi[2][TBH];
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int t = 0; t < TBH; ++t) vr[u][t] = vi[u][t] = f4zero();
#pragma unroll
      for (int ks = 0; ks < NKZ; ++ks) {
        h8 nsf[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) nsf[u] = M::neg(sf[u][ks]);
#pragma unroll
        for (int t = 0; t < TBH; ++t) {
          const int tb = tbh + t;
          const h8 zr = M::ld(ZT + (tb * 16 + r16) * LDZ + ks * KS + g * 8);
          const h8 zi = M::ld(ZT + (KBP + tb * 16 + r16) * LDZ + ks * KS + g * 8);
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            vr[u][t] = M::mma(cf[u][ks], zr, vr[u][t]);
            vr[u][t] = M::mma(nsf[u], zi, vr[u][t]);
            vi[u][t] = M::mma(cf[u][ks], zi, vi[u][t]);
            vi[u][t] = M::mma(sf[u][ks], zr, vi[u][t]);
          }
        }
      }
      // D: lane holds rows 4 g + i, column kb = tb * 16 + r16
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int t = 0; t < TBH; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int rl = (wave + WD_WAVES * u) * 16 + 4 * g + i;
            const int kb = (tbh + t) * 16 + r16;
            VL[rl * LDV + kb] = to_h(vr[u][t][i]);
            VL[rl * LDV + KBP + kb] = to_h(vi[u][t][i]);
          }
    }
    __syncthreads();

    // this wave's rows of V, as B operands of step A'
    h8 vf[2][NKV];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int k = 0; k < NKV; ++k)
        vf[u][k] = M::ld(VL + ((wave + WD_WAVES * u) * 16 + r16) * LDV + k * KS + g * 8);
    // next item's step-B' table rows and (new plane) spectrum, before this
    // item's block requests
    ldC(cn, cf, sf);
    if (more && cn == 0) ldZ(pn, zq);
    __syncthreads();  // V read: its space takes the twiddle blocks
    stTW(twr[0], 0);
    __syncthreads();

    // ---- step A' ---------------------------------------------------------------
    const __amdgpu_buffer_rsrc_t ry = plane_rsrc(a.out, p, plane_bytes);
    const __amdgpu_buffer_rsrc_t rx = plane_rsrc(EPI ? a.x : a.out, p, plane_bytes);
    const __amdgpu_buffer_rsrc_t rxn = plane_rsrc(EPI ? a.x : a.out, pn, plane_bytes);
    auto block = [&](int b, int par) {
      // requests two blocks ahead (the next item's first ones at the end);
      // operands selected, not branched on: one load sequence, exact waits
      ldTW(b + 2 < nmb ? b + 2 : b + 2 - nmb, twr[par]);
      u32x4 xs[2][2];
      if (EPI) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          xs[u][0] = xr[par][u][0];
          xs[u][1] = xr[par][u][1];
        }
        const bool nxt = b + 2 >= nmb;
        ldX(nxt ? rxn : rx, nxt ? cn : c0, nxt ? b + 2 - nmb : b + 2, xr[par]);
      }
      const _Float16* tb = TW + par * (WD_MB * LDT) + r16 * LDT + g * 8;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f4 acc[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          acc[c] = f4zero();
#pragma unroll
          for (int k = 0; k < NKV; ++k)
            acc[c] = M::mma(M::ld(tb + c * 16 * LDT + k * KS), vf[u][k], acc[c]);
        }
        // D: lane holds column n = r16 (row of y), rows m = c * 16 + 4 g + i
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) ob[r16 * WD_LDO + c * 16 + 4 * g + i] = acc[c][i] * a.scale;
        wave_lds_sync();
        float v[16];  // v[8 h + e]: row lane / 8 + 8 h, column (lane % 8) * 8 + e
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int h = q >> 1, e0 = (q & 1) * 4;
          const f4 t = *reinterpret_cast<const f4*>(ob + ((lane >> 3) + 8 * h) * WD_LDO +
                                                    (lane & 7) * 8 + e0);
          v[4 * q] = t[0];
          v[4 * q + 1] = t[1];
          v[4 * q + 2] = t[2];
          v[4 * q + 3] = t[3];
        }
        wave_lds_sync();
        if (EPI) {
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t sw = lut2<false>(lut, xs[u][h][e], sat);
              h2 s2;
              __builtin_memcpy(&s2, &sw, 4);
              v[8 * h + 2 * e] *= (float)s2[0];
              v[8 * h + 2 * e + 1] *= (float)s2[1];
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          h8 w;
#pragma unroll
          for (int e = 0; e < 8; ++e) w[e] = to_h(v[8 * h + e]);
          u32x4 wv;
          __builtin_memcpy(&wv, &w, 16);
          __builtin_amdgcn_raw_buffer_store_b128(wv, ry, xoff(c0, u, b, h), 0, WD_NT);
        }
      }
      stTW(twr[1 - par], 1 - par);
      __syncthreads();
    };
#pragma nounroll
    for (int b = 0; b < nmb; b += 2) {
      block(b, 0);
      block(b + 1, 1);
    }
  }
}

// ---------------------------------------------------------------------------
// Launchers (hipErrorNotSupported: the shape is not one of this path's)
// ---------------------------------------------------------------------------
size_t r2c_wide_lds_bytes(int nct, bool pre, int lut_sat) {
  const size_t at = (size_t)2 * (nct * 8) * (WD_R + WD_PAD) * 2;
  const size_t tw = (size_t)2 * 2 * (nct * 8) * WD_LDT * 2;
  return at + tw + (pre ? (size_t)(lut_sat + 2) * 2 : 0);
}

size_t c2r_wide_lds_bytes(int nct, int Kap, bool epi, int lut_sat) {
  size_t base = 0;
  const int nkz = Kap / 32;
#define FNO_C2RW_BYTES(N, K) \
  if (nct == N && nkz == K) base = C2RWide<N, K>::zt_bytes + C2RWide<N, K>::reg_bytes;
  FNO_C2RW_BYTES(4, 1) FNO_C2RW_BYTES(4, 2) FNO_C2RW_BYTES(4, 4)
  FNO_C2RW_BYTES(8, 1) FNO_C2RW_BYTES(8, 2) FNO_C2RW_BYTES(8, 4)
#undef FNO_C2RW_BYTES
  if (base == 0) return (size_t)1 << 30;  // not a shape of this path
  return base + (epi ? (size_t)(lut_sat + 2) * 2 : 0);
}

hipError_t launch_r2c_wide(const R2CArgs& a, int nct, int grid, size_t lds, hipStream_t s) {
  const bool t = a.do_tanh != 0;
  const void* k = nullptr;
  if (nct == 4) k = t ? (const void*)&r2c_wide_kernel<4, true> : (const void*)&r2c_wide_kernel<4, false>;
  if (nct == 8) k = t ? (const void*)&r2c_wide_kernel<8, true> : (const void*)&r2c_wide_kernel<8, false>;
  if (!k || lds > 160 * 1024) return hipErrorNotSupported;
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 gr(grid), bl(WD_WAVES * 64);
  if (nct == 4) {
    if (t) hipLaunchKernelGGL((r2c_wide_kernel<4, true>), gr, bl, lds, s, a);
    else hipLaunchKernelGGL((r2c_wide_kernel<4, false>), gr, bl, lds, s, a);
  } else {
    if (t) hipLaunchKernelGGL((r2c_wide_kernel<8, true>), gr, bl, lds, s, a);
    else hipLaunchKernelGGL((r2c_wide_kernel<8, false>), gr, bl, lds, s, a);
  }
  return hipGetLastError();
}

template <int NCT, int NKZ>
static hipError_t c2r_wide_go(const C2RArgs& a, int grid, size_t lds, hipStream_t s) {
  const void* k = a.epilogue ? (const void*)&c2r_wide_kernel<NCT, NKZ, true>
                             : (const void*)&c2r_wide_kernel<NCT, NKZ, false>;
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 gr(grid), bl(WD_WAVES * 64);
  if (a.epilogue) hipLaunchKernelGGL((c2r_wide_kernel<NCT, NKZ, true>), gr, bl, lds, s, a);
  else hipLaunchKernelGGL((c2r_wide_kernel<NCT, NKZ, false>), gr, bl, lds, s, a);
  return hipGetLastError();
}

// Shapes: nct in {4, 8}, Kap in {32, 64, 128}, Ka * Kb <= 8192, Nb a multiple
// of 128, Na a multiple of 256.
hipError_t launch_c2r_wide(const C2RArgs& a, int nct, int grid, size_t lds, hipStream_t s) {
  if (lds > 160 * 1024 || a.Ka * a.Kb > 8192 || a.Nb % (2 * WD_MB) != 0 || a.Na % WD_R != 0 ||
      a.Kb % 4 != 0)
    return hipErrorNotSupported;
  const int nkz = a.Kap / 32;
  if (nct == 4 && nkz == 1) return c2r_wide_go<4, 1>(a, grid, lds, s);
  if (nct == 4 && nkz == 2) return c2r_wide_go<4, 2>(a, grid, lds, s);
  if (nct == 4 && nkz == 4) return c2r_wide_go<4, 4>(a, grid, lds, s);
  if (nct == 8 && nkz == 1) return c2r_wide_go<8, 1>(a, grid, lds, s);
  if (nct == 8 && nkz == 2) return c2r_wide_go<8, 2>(a, grid, lds, s);
  if (nct == 8 && nkz == 4) return c2r_wide_go<8, 4>(a, grid, lds, s);
  return hipErrorNotSupported;
}

}  // namespace fno
