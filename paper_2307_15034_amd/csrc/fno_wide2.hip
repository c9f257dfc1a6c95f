// Truncated transforms of large fp16 planes with one radix-2 stage on each
// axis ahead of (forward) or behind (inverse) the DFT-by-MFMA stages: planes
// with Na and Nb multiples of 256, at most 64 retained modes on the last axis
// and 128 on the leading one (the 256^2 and 1024^2 workloads).
//
// The radix-2 split (decimation in frequency) follows from e^{-2 pi i k (n +
// N/2) / N} = (-1)^k e^{-2 pi i k n / N}:
//   X[k] = sum_{n < N/2} (u[n] + (-1)^k u[n + N/2]) e^{-2 pi i k n / N},
// so the even retained frequencies need only the sums u[n] + u[n + N/2] and
// the odd ones only the differences, each over half the length.  Applied to
// the last axis (sums and differences of the two halves of each row, in
// fp16, before the MFMA stage) and to the leading one (sums and differences
// of rows r and r + Na/2, in fp32, on the step-A accumulators) it halves the
// matrix-core work and the twiddle traffic through LDS of both stages.  The
// inverse runs the mirror image: V[r] = E[r] + O[r], V[r + Na/2] = E[r] -
// O[r] with E, O the sums over even and odd leading frequencies, and y[m] =
// E'[m] + O'[m], y[m + Nb/2] = E'[m] - O'[m] on the last axis.  Retained
// frequencies keep their parity under the mode map (k(t) = t or N - 2m + t,
// N even), so the classes are the even and odd slots t.
//
// A work item is (plane, chunk): rows c0 + [0, 128) and c0 + Na/2 + [0, 128);
// each of the eight waves owns the 16-row tiles c0 + 16 w + [0, 16) and
// c0 + Na/2 + 16 w + [0, 16), so the leading-axis butterfly pairs registers
// of the same lane.  Persistent work-groups (one per compute unit) walk the
// items; the twiddle staging through LDS and the tanh' lookup of the
// inverse are as in the one-stage wide kernels, the forward's tanh lookup
// batches eight table reads per wait.  The padded LDS layouts below give
// 16-byte accesses without bank conflicts beyond the half rate that gfx950
// applies to any 16-byte read whose 16-lane groups do not each cover one
// aligned 256-byte block (measured: such reads take twice the cycles of
// block-aligned ones, with or without padding).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

namespace {

constexpr int W2_WAVES = 8;
constexpr int W2_NT = W2_WAVES * 64;
constexpr int W2_H = 128;          // rows of an item in each half of the plane
constexpr int W2_KS = 32;          // MFMA k-step
constexpr int W2_SK = 64;          // n per twiddle slice (two k-steps)
constexpr int W2_LDT = W2_SK + 8;  // slice row stride (halves): 36 dwords
constexpr int W2_LDR = W2_H + 8;   // step-A result row stride (halves): 68 dwords
constexpr int W2_BIG = 0x40000000; // buffer offset past every plane
constexpr int W2_NTS = 2;          // cache policy of the inverse's stores: streaming
constexpr int W2_MB = 64;          // output columns per block of the inverse's last stage
constexpr int W2_LDO = 68;         // transpose buffer row stride (floats)


// column x of a 64-wide row of the transpose buffer, stored with the two
// 4-float halves of each 8-float group swapped in the upper 32 columns: the
// eight lanes that read one row (8 floats each) then hit 32 distinct banks
__device__ __forceinline__ int ob_col(int x) { return x ^ ((x & 32) >> 3); }

}  // namespace

// ---------------------------------------------------------------------------
// Forward.  Tables (radix-2 forms, built by the planner):
//   twA [4 KBPC][Nb/2]: row cls 2 KBPC + c:  cos(2 pi k n / Nb), k = 2c + cls,
//                       row cls 2 KBPC + KBPC + c: -sin(...)  (zero past Kb)
//   cB, sB [2][nta 16][Na/2]: row rc nta16 + t: cos / sin(2 pi k_a(2t + rc) r / Na)
// Step A per item: Y_cls[row][c] = sum_{n < Nb/2} y_cls[row][n] twA[cls][c][n]
// with y_e = (u[n] + u[n + Nb/2]) / 2, y_o = (u[n] - u[n + Nb/2]) / 2 (each
// rounded once to fp16; the factor 2 returns with the scale); then the row
// butterfly Ye = Y(r) + Y(r + Na/2), Yo = Y(r) - Y(r + Na/2) into LDS
// AT[rc][cls][col][row] (transposed, fp16); step B accumulates
// X[t_a][t_b] += sum_r (cB - i sB)[rc][t][r] Y_rc[r][t_b] over the items of
// the plane, t_a = 2t + rc, t_b = 2 t' + cls.
// ---------------------------------------------------------------------------
template <int NCTC, bool PRE, bool EARLY>
__global__ __launch_bounds__(W2_NT, 1) void r2c_wide2_kernel(R2CArgs a) {
  typedef MM<_Float16> M;
  constexpr int KBPC = NCTC * 8;               // complex columns per class (padded)
  constexpr int NROW = 4 * KBPC;               // twiddle rows (both classes)
  constexpr int NTBC = NCTC / 2;               // step-B column tiles per class
  constexpr int NTBW = NCTC;                   // step-B column tiles, both classes
  constexpr int TWP = NROW * W2_SK / 8 / W2_NT;  // 16-byte slice pieces per thread
  constexpr int NKB = W2_H / W2_KS;            // step-B k-steps per item
  static_assert(TWP >= 1, "slice pieces");
  // The next item's first four k-steps are requested during this item's
  // last two slices.  Its step-B tables then complete behind them (loads
  // complete in order), unless EARLY requests them at the item's start,
  // which holds their 32 registers through step A: for short items (one
  // chunk per plane) waiting for the rows at step B costs more than that.
  static_assert(!EARLY || NCTC == 2, "early requests: narrow variant only");
  extern __shared__ __align__(16) unsigned char smem[];
  // the lookup table first, so that a lookup address is the byte offset of
  // the code itself (no base to add)
  _Float16* lut = reinterpret_cast<_Float16*>(smem);
  _Float16* AT = reinterpret_cast<_Float16*>(smem + (PRE ? lutn_bytes(a.lut_sat) : 0));
  // [2 rc][2 cls][2 KBPC][LDR]
  _Float16* TWb = AT + 4 * 2 * KBPC * W2_LDR;           // [2][NROW][LDT]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const _Float16* cB = reinterpret_cast<const _Float16*>(a.cB);
  const _Float16* sB = reinterpret_cast<const _Float16*>(a.sB);
  const uint32_t sat2 = (uint32_t)(2 * a.lut_sat) * 0x10001u;
  if (PRE) stage_lutn<W2_NT>(lut, a.lut, a.lut_sat);

  const int Nh = a.Nb >> 1, NhA = a.Na >> 1;
  const int64_t plane_bytes = (int64_t)a.Na * a.Nb * 2;
  const int nks = Nh / W2_KS;      // a multiple of 4 on this path
  const int ngr = nks / 2;         // twiddle slices per item (even)
  const int nch = NhA / W2_H;
  // step-B share of this wave: row tile q = (class rc, tile ta), column tiles
  // tb0 + j tbs over both column classes
  const int nta = a.Kap16 >> 4;    // leading-axis tiles per class (1, 2 or 4)
  const int nq = 2 * nta;
  const int q = wave % nq, tb0 = wave / nq, tbs = W2_WAVES / nq;
  const int rc = q / nta, ta = q % nta;

  const int64_t nitems = a.planes > (int64_t)blockIdx.x
                             ? ((a.planes - 1 - blockIdx.x) / gridDim.x + 1) * nch
                             : 0;
  auto item_plane = [&](int64_t it) { return (int64_t)blockIdx.x + (it / nch) * gridDim.x; };
  auto item_chunk = [&](int64_t it) { return (int)(it % nch) * W2_H; };

  // lane part of the row offset (the upper half's rows and the row's second
  // half go in the scalar offset), formed where it is used
  auto row_lane = [&](int c0) {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return (c0 + wave * 16 + (t & 15)) * a.Nb * 2 + ((t >> 4) & 3) * 16;
  };
  const int hiA = NhA * a.Nb * 2;  // bytes from row r to row r + Na/2
  const int hiB = Nh * 2;          // bytes from column n to n + Nb/2
  // k-step s of both row tiles (u: r, r + Na/2) and both column halves (h)
  auto ldA = [&](const __amdgpu_buffer_rsrc_t& rs, int rb, int s, u32x4 (&v)[2][2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        v[u][h] = __builtin_amdgcn_raw_buffer_load_b128(rs, rb + s * W2_KS * 2,
                                                        u * hiA + h * hiB, 0);
  };
  const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.twA), (short)0, NROW * Nh * 2, 0x00020000);
  // twiddle slice gs: all NROW rows, columns gs 64 + [0, 64); thread t takes
  // pieces t + 512 e (row piece / 8, 8 halves at (piece % 8) 8)
  auto ldTW = [&](int gs, u32x4 (&v)[TWP]) {
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * W2_NT;
      v[e] = __builtin_amdgcn_raw_buffer_load_b128(rt, ((pc >> 3) * Nh + (pc & 7) * 8) * 2,
                                                   gs * W2_SK * 2, 0);
    }
  };
  auto stTW = [&](const u32x4 (&v)[TWP], int buf) {
    _Float16* d = TWb + buf * (NROW * W2_LDT);
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * W2_NT;
      *reinterpret_cast<u32x4*>(d + (pc >> 3) * W2_LDT + (pc & 7) * 8) = v[e];
    }
  };

  f4 accR[NTBW], accI[NTBW];
  u32x4 va[4][2][2];   // row fragments of k-steps s .. s + 3 (slot s % 4)
  u32x4 twr[2][TWP];   // twiddle slices g + 1, g + 2 in flight
  __amdgpu_buffer_rsrc_t rs = plane_rsrc(a.in, nitems > 0 ? item_plane(0) : 0, plane_bytes);
  if (nitems > 0) {
    ldTW(0, twr[0]);
    ldTW(1, twr[1]);
    const int rb = row_lane(0);
#pragma unroll
    for (int d = 0; d < 4; ++d) ldA(rs, rb, d, va[d]);
    stTW(twr[0], 0);
  }
  __syncthreads();  // table and first slice staged

  for (int64_t it = 0; it < nitems; ++it) {
    const int64_t p = item_plane(it);
    const int c0 = item_chunk(it);
    if (c0 == 0) {
#pragma unroll
      for (int j = 0; j < NTBW; ++j) accR[j] = accI[j] = f4zero();
    }
    const bool more = it + 1 < nitems;
    const __amdgpu_buffer_rsrc_t rsn = more ? plane_rsrc(a.in, item_plane(it + 1), plane_bytes) : rs;
    const int cn = more ? item_chunk(it + 1) : c0;
    h8 cfs[NKB], sfs[NKB];
    auto ld_tables = [&] {
#pragma unroll
      for (int k = 0; k < NKB; ++k) {
        const int64_t toff = (int64_t)(rc * nta * 16 + ta * 16 + r16) * NhA + c0 + k * W2_KS + g * 8;
        cfs[k] = M::ld(cB + toff);
        sfs[k] = M::ld(sB + toff);
      }
    };
    if (EARLY) ld_tables();

    // ---- step A (last axis, radix-2) ----------------------------------------
    f4 accE[2][NCTC], accO[2][NCTC];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int ct = 0; ct < NCTC; ++ct) accE[u][ct] = accO[u][ct] = f4zero();
    const h8 half8 = {(_Float16)0.5f, (_Float16)0.5f, (_Float16)0.5f, (_Float16)0.5f,
                      (_Float16)0.5f, (_Float16)0.5f, (_Float16)0.5f, (_Float16)0.5f};
    auto mul = [&](const u32x4 (&v)[2][2], int buf, int k) {
      h8 ye[2], yo[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 lo = v[u][0], hi = v[u][1];
        if (PRE) {
          lutn_odd4(lo, sat2);
          lutn_odd4(hi, sat2);
        }
        // half sums and half differences: fp16 cannot overflow here (large
        // pre-activation bounds reach 65504), and halving is exact; the
        // factor 2 is restored in fp32 after the products
        const h8 L = w_as_h8(lo), H = w_as_h8(hi) * (_Float16)0.5f;
        ye[u] = __builtin_elementwise_fma(L, half8, H);
        yo[u] = __builtin_elementwise_fma(L, half8, -H);
      }
      const _Float16* tb = TWb + buf * (NROW * W2_LDT) + r16 * W2_LDT + k * W2_KS + g * 8;
#pragma unroll
      for (int ct = 0; ct < NCTC; ++ct) {
        const h8 be = M::ld(tb + ct * 16 * W2_LDT);
        const h8 bo = M::ld(tb + (2 * KBPC + ct * 16) * W2_LDT);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          accE[u][ct] = M::mma(ye[u], be, accE[u][ct]);
          accO[u][ct] = M::mma(yo[u], bo, accO[u][ct]);
        }
      }
    };
    // one slice: its two k-steps (the rows two slices on requested as each
    // k-step's registers free up), then the next slice into LDS and a barrier
    auto slice = [&](int gs, int par, int rb, bool rows) {
      ldTW(gs + 2 < ngr ? gs + 2 : gs + 2 - ngr, twr[par]);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        mul(va[2 * par + k], par, k);
        if (rows) ldA(rs, rb, 2 * gs + k + 4, va[2 * par + k]);
        // the last two slices request the next item's k-steps into the
        // slots they free (operands selected, not branched on: the last
        // k-step of this plane, in range, when there is no next item)
        if (!rows)
          ldA(more ? rsn : rs, row_lane(cn), more ? 2 * gs + k + 4 - nks : nks - 1, va[2 * par + k]);
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
    // last two slices: the next item's rows
    slice(ngr - 2, 0, 0, false);
    slice(ngr - 1, 1, 0, false);
    {
      // row butterfly, scale (twice the step-A scale: the last-axis stage
      // took half sums), fp16: AT[rc][cls][col][row] for this wave's 16 rows
      // (four consecutive rows per lane: one 8-byte store)
      const float scaleA2 = 2.0f * a.scaleA;
      int lb = r16 * W2_LDR + wave * 16 + 4 * g;
      asm volatile("" : "+v"(lb));
#pragma unroll
      for (int cls = 0; cls < 2; ++cls)
#pragma unroll
        for (int ct = 0; ct < NCTC; ++ct) {
          const f4 lo = cls == 0 ? accE[0][ct] : accO[0][ct];
          const f4 hi = cls == 0 ? accE[1][ct] : accO[1][ct];
          h4 se, so;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            se[i] = to_h((lo[i] + hi[i]) * scaleA2);
            so[i] = to_h((lo[i] - hi[i]) * scaleA2);
          }
          _Float16* d = AT + lb + (cls * 2 * KBPC + ct * 16) * W2_LDR;
          *reinterpret_cast<h4*>(d) = se;                              // rc = 0
          *reinterpret_cast<h4*>(d + 4 * KBPC * W2_LDR) = so;          // rc = 1
        }
    }
    __builtin_amdgcn_sched_barrier(0);  // accumulators dead before the tables load
    if (!EARLY) ld_tables();  // this item's step-B tables
    __syncthreads();

    // ---- step B (leading axis, the rc class of this wave's tile) -------------
    const _Float16* atb = AT + rc * 2 * (2 * KBPC) * W2_LDR;
#pragma unroll
    for (int k = 0; k < NKB; ++k) {
      const int k0 = k * W2_KS;
      const h8 nsf = M::neg(sfs[k]);
#pragma unroll
      for (int j = 0; j < NTBW; ++j) {
        // (tiles past NTBW are computed from a clamped tile and never stored)
        const int jt = min(tb0 + j * tbs, NTBW - 1);
        const int cls = jt / NTBC, tb = jt % NTBC;
        const _Float16* col = atb + (cls * 2 * KBPC + tb * 16 + r16) * W2_LDR + k0 + g * 8;
        const h8 ar = M::ld(col);
        const h8 ai = M::ld(col + KBPC * W2_LDR);
        accR[j] = M::mma(cfs[k], ar, accR[j]);
        accR[j] = M::mma(sfs[k], ai, accR[j]);
        accI[j] = M::mma(cfs[k], ai, accI[j]);
        accI[j] = M::mma(nsf, ar, accI[j]);
      }
      __builtin_amdgcn_sched_barrier(0);  // bound the hoisting of LDS reads
    }
    __syncthreads();

    if (c0 + W2_H >= NhA) {  // last item of the plane: store its spectrum
      const __amdgpu_buffer_rsrc_t ro = plane_rsrc(a.out, p, (int64_t)a.Ka * a.Kb * 4);
      int tq = ta * 16 + 4 * g;
      asm volatile("" : "+v"(tq));
#pragma unroll
      for (int j = 0; j < NTBW; ++j) {
        const int jt = tb0 + j * tbs;
        if (jt >= NTBW) continue;
        const int cls = jt / NTBC, tb = jt % NTBC;
        const int t_b = 2 * (tb * 16 + r16) + cls;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t_a = 2 * (tq + i) + rc;
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
// Inverse.  Tables (radix-2 forms):
//   cI, sI [2][Na/2][KAH]: [cls][r][t]: cos / sin(2 pi k_a(2t + cls) r / Na)
//   twI [Nb/2][4 KBPC]: row m: [cls 0: cos | -sin][cls 1: cos | -sin] of
//                       2 pi k m / Nb, k = 2c + cls (zero past Kb)
// Per plane the spectrum is staged transposed in LDS, split by the parity
// of t_a (the step-B' class) and ordered by the parity of t_b (the step-A'
// class): ZT[cls_a][re|im][p][t'] with t_a = 2t' + cls_a and p = cls_b KBPC
// + t_b' (t_b = 2 t_b' + cls_b).  Per item step B' gives E (even t_a) and O
// (odd t_a) for the wave's 16 rows r and writes V(r) = E + O and V(r + Na/2)
// = E - O to LDS as [Re V | Im V] per class; each wave then holds its rows
// of V as B operands of step A', which sweeps blocks of 64 columns m < Nb/2
// giving E' and O' and stores y[m] = E' + O' and y[m + Nb/2] = E' - O'
// through a per-wave transpose buffer (whole 128-byte lines per store
// instruction).  The epilogue multiplies by f'(x); each output segment
// (16 rows x 64 columns) requests its x at its start, after the previous
// segment's stores, and uses it after its transpose.
// ---------------------------------------------------------------------------
constexpr int W2_LDOH = 72;        // fp16 transpose buffer row stride (halves)

// LDS bytes of the inverse's table of codes 0..sat plus one NaN entry (its
// lookups index at most sat + 1), rounded up to 256 (the regions after it
// stay aligned)
__host__ __device__ __forceinline__ int w2_lut_bytes(int sat) { return ((sat + 2) * 2 + 255) & ~255; }

template <int NCTC, int NKZH, int MB = W2_MB, bool OB16 = false>
struct C2RWide2 {
  static constexpr int KBPC = NCTC * 8;
  static constexpr int LDZ = NKZH * 32 + 8;
  static constexpr int LDV = 4 * KBPC + 8;
  static constexpr int LDT = 4 * KBPC + 8;
  static constexpr size_t zt_bytes = (size_t)2 * 2 * (2 * KBPC) * LDZ * 2;
  static constexpr size_t vl_bytes = (size_t)2 * W2_H * LDV * 2;
  static constexpr size_t tw_bytes = (size_t)2 * MB * LDT * 2;
  static constexpr size_t ob_bytes =
      OB16 ? (size_t)W2_WAVES * 16 * W2_LDOH * 2 : (size_t)W2_WAVES * 16 * W2_LDO * 4;
  static constexpr size_t reg_bytes =
      vl_bytes > tw_bytes + ob_bytes ? vl_bytes : tw_bytes + ob_bytes;
};

template <int NCTC, int NKZH, bool EPI, int MB = W2_MB>
__global__ __launch_bounds__(W2_NT, 1) void c2r_wide2_kernel(C2RArgs a) {
  typedef MM<_Float16> M;
  // MB 128 (the wide variant on planes with Nb / 2 a multiple of 256): half
  // the blocks per item, so half the block barriers and twiddle stagings;
  // each block's results still go out through the transpose buffer one
  // 64-column chunk at a time.  With the epilogue the buffer then holds fp16
  // (the table leaves no room for fp32): the products are rounded to fp16
  // before the multiplication by f'(x), as an unfused epilogue would read
  // them.
  constexpr bool OB16 = EPI && MB == 128;
  typedef C2RWide2<NCTC, NKZH, MB, OB16> L;
  constexpr int NQ = MB / 64;          // 64-column chunks per block
  constexpr int KBPC = L::KBPC;
  constexpr int NTB = NCTC;            // p tiles (both step-A' classes)
  constexpr int NTBC = NCTC / 2;
  constexpr int NKVC = NCTC / 2;       // step-A' k-steps per class (2 KBPC / 32)
  constexpr int LDZ = L::LDZ, LDV = L::LDV, LDT = L::LDT;
  constexpr int KAH = NKZH * 32;
  constexpr int ZQ = 4;                // 16-byte spectrum pieces per thread
  constexpr int TWP = MB * 4 * KBPC / 8 / W2_NT;  // twiddle pieces per thread
  constexpr int PPR = 4 * KBPC / 8;    // pieces per twiddle row
  static_assert(TWP >= 1, "block pieces");
  extern __shared__ __align__(16) unsigned char smem[];
  // the lookup table first (a lookup address is the code's byte offset)
  _Float16* lut = reinterpret_cast<_Float16*>(smem);
  _Float16* ZT = reinterpret_cast<_Float16*>(smem + (EPI ? w2_lut_bytes(a.lut_sat) : 0));
  // [2][2][2 KBPC][LDZ]
  unsigned char* reg = reinterpret_cast<unsigned char*>(ZT) + L::zt_bytes;
  _Float16* VL = reinterpret_cast<_Float16*>(reg);       // [2 W2_H][LDV]
  _Float16* TW = reinterpret_cast<_Float16*>(reg);       // [2][W2_MB][LDT]
  float* OB = reinterpret_cast<float*>(reg + L::tw_bytes);  // [8][16][W2_LDO]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const _Float16* cI = reinterpret_cast<const _Float16*>(a.cI);
  const _Float16* sI = reinterpret_cast<const _Float16*>(a.sI);
  const us2 sat = {(unsigned short)a.lut_sat, (unsigned short)a.lut_sat};
  float* ob = OB + wave * 16 * W2_LDO;
  _Float16* obh = reinterpret_cast<_Float16*>(OB) + wave * 16 * W2_LDOH;

  const int Nh = a.Nb >> 1, NhA = a.Na >> 1;
  const int64_t plane_bytes = (int64_t)a.Na * a.Nb * 2;
  const int spec_bytes = a.Ka * a.Kb * 4;
  const int nch = NhA / W2_H;
  const int nmb = Nh / MB;             // even on this path
  const int nq = a.Ka * a.Kb / 4;      // 16-byte spectrum pieces
  const int64_t nitems = a.planes > (int64_t)blockIdx.x
                             ? ((a.planes - 1 - blockIdx.x) / gridDim.x + 1) * nch
                             : 0;
  auto item_plane = [&](int64_t it) { return (int64_t)blockIdx.x + (it / nch) * gridDim.x; };
  auto item_chunk = [&](int64_t it) { return (int)(it % nch) * W2_H; };

  // the padding of ZT stays zero: every plane writes the same positions
  for (int i = tid; i < 2 * 2 * 2 * KBPC * LDZ; i += W2_NT) ZT[i] = (_Float16)0.0f;
  if (EPI) stage_lut<W2_NT>(lut, a.lut, a.lut_sat);

  auto ldZ = [&](int64_t p, u32x4 (&zq)[ZQ]) {
    const __amdgpu_buffer_rsrc_t rz = plane_rsrc(a.in, p, spec_bytes);
#pragma unroll
    for (int q = 0; q < ZQ; ++q) {
      const int i = tid + q * W2_NT;
      zq[q] = __builtin_amdgcn_raw_buffer_load_b128(rz, i < nq ? i * 16 : W2_BIG, 0, 0);
    }
  };
  auto stZ = [&](const u32x4 (&zq)[ZQ]) {
    const int qpr = a.Kb / 4;
#pragma unroll
    for (int q = 0; q < ZQ; ++q) {
      const int i = tid + q * W2_NT;
      if (i < nq) {
        // kb0 is a multiple of 4: slot kb0 + e sits in column (e & 1) KBPC +
        // kb0 / 2 + e / 2 of its class, a constant step from the first (one
        // address per piece, formed per item rather than held live)
        int t_a = i / qpr;
        asm volatile("" : "+v"(t_a));
        const int kb0 = (i - t_a * qpr) * 4;
        const int ca = t_a & 1, tq = t_a >> 1;
        _Float16* z0 = ZT + (ca * 2 * 2 * KBPC + (kb0 >> 1)) * LDZ + tq;
        const h8 v = w_as_h8(zq[q]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int pc = ((e & 1) * KBPC + (e >> 1)) * LDZ;
          z0[pc] = v[2 * e];                       // real part
          z0[2 * KBPC * LDZ + pc] = v[2 * e + 1];  // imaginary part
        }
      }
    }
  };
  // step-B' table rows of this wave's rows r = c0 + 16 w + r16, both classes
  auto ldC = [&](int c0, h8 (&cf)[2][NKZH], h8 (&sf)[2][NKZH]) {
    const int64_t row = c0 + wave * 16 + r16;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int k = 0; k < NKZH; ++k) {
        cf[c][k] = M::ld(cI + ((int64_t)c * NhA + row) * KAH + k * W2_KS + g * 8);
        sf[c][k] = M::ld(sI + ((int64_t)c * NhA + row) * KAH + k * W2_KS + g * 8);
      }
  };
  // twiddle block b: rows m = b 64 + [0, 64), all 4 KBPC columns
  const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.twI), (short)0, Nh * 4 * KBPC * 2, 0x00020000);
  auto ldTW = [&](int b, u32x4 (&v)[TWP]) {
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * W2_NT;
      v[e] = __builtin_amdgcn_raw_buffer_load_b128(
          rt, ((pc / PPR) * 4 * KBPC + (pc % PPR) * 8) * 2, b * MB * 4 * KBPC * 2, 0);
    }
  };
  auto stTW = [&](const u32x4 (&v)[TWP], int buf) {
    _Float16* d = TW + buf * (MB * LDT);
#pragma unroll
    for (int e = 0; e < TWP; ++e) {
      const int pc = tid + e * W2_NT;
      *reinterpret_cast<u32x4*>(d + (pc / PPR) * LDT + (pc % PPR) * 8) = v[e];
    }
  };
  // offset of this lane's 8 outputs in the transposed layout: row lane / 8 +
  // 8 h of the tile (rows r; the scalar offset adds Na/2 rows for the upper
  // tile), columns half Nb/2 + b 64 + (lane % 8) 8: each 16-byte access
  // instruction covers eight whole 128-byte lines
  const int hiA = NhA * a.Nb * 2;
  auto xoff = [&](int c0, int b, int half, int h) {
    return (c0 + wave * 16 + (lane >> 3) + 8 * h) * a.Nb * 2 +
           (half * Nh + b * MB + (lane & 7) * 8) * 2;
  };
  // x of unit (u, q) of block b: 64-column chunk q of the rows of tile u,
  // both halves hf and both row groups h
  auto ldX = [&](const __amdgpu_buffer_rsrc_t& rx, int c0, int b, int u, int q,
                 u32x4 (&v)[2][2]) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        v[hf][h] = __builtin_amdgcn_raw_buffer_load_b128(rx, xoff(c0, b, hf, h) + q * 128, u * hiA, 0);
  };

  u32x4 zq[ZQ];
  h8 cf[2][NKZH], sf[2][NKZH];
  // twiddle blocks in flight: b + 1 and b + 2, or, with 128-column blocks
  // (each as long as two 64-column ones), b + 1
  constexpr int TWA = MB == 128 ? 1 : 2;
  u32x4 twr[TWA][TWP];
  // x of the epilogue, one unit ahead: a block's units are (u, q), u the
  // row tile and q the 64-column chunk, in that order; unit t of a block
  // (t = u NQ + q) sits in slot t % 2.  Each unit's x is requested before
  // the products of the unit before it, the next block's first unit before
  // those of the last one, and the next item's first during this item's
  // last block (the first item's before the loop)
  u32x4 xr[2][2][2];
  if (nitems > 0) {
    ldZ(item_plane(0), zq);
    ldC(0, cf, sf);
    ldTW(0, twr[0]);
    if (TWA == 2) ldTW(1, twr[TWA - 1]);
    if (EPI) {
      const __amdgpu_buffer_rsrc_t rx0 = plane_rsrc(a.x, item_plane(0), plane_bytes);
      ldX(rx0, item_chunk(0), 0, 0, 0, xr[0]);
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

    // ---- step B' (leading axis, radix-2): V for rows r and r + Na/2 ----------
#pragma unroll
    for (int t = 0; t < NTB; ++t) {
      f4 er = f4zero(), ei = f4zero(), orr = f4zero(), oi = f4zero();
#pragma unroll
      for (int ks = 0; ks < NKZH; ++ks) {
        const _Float16* z0 = ZT + (t * 16 + r16) * LDZ + ks * W2_KS + g * 8;
        const h8 zr0 = M::ld(z0), zi0 = M::ld(z0 + 2 * KBPC * LDZ);
        const h8 zr1 = M::ld(z0 + 4 * KBPC * LDZ), zi1 = M::ld(z0 + 6 * KBPC * LDZ);
        er = M::mma(cf[0][ks], zr0, er);
        er = M::mma(M::neg(sf[0][ks]), zi0, er);
        ei = M::mma(cf[0][ks], zi0, ei);
        ei = M::mma(sf[0][ks], zr0, ei);
        orr = M::mma(cf[1][ks], zr1, orr);
        orr = M::mma(M::neg(sf[1][ks]), zi1, orr);
        oi = M::mma(cf[1][ks], zi1, oi);
        oi = M::mma(sf[1][ks], zr1, oi);
      }
      // lane: rows 4 g + i of the wave's tile, column p = t 16 + r16
      const int cb = t / NTBC, kb = (t % NTBC) * 16 + r16;
      const int cre = cb * 2 * KBPC + kb, cim = cre + KBPC;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = wave * 16 + 4 * g + i;
        VL[rl * LDV + cre] = to_h(er[i] + orr[i]);
        VL[rl * LDV + cim] = to_h(ei[i] + oi[i]);
        VL[(W2_H + rl) * LDV + cre] = to_h(er[i] - orr[i]);
        VL[(W2_H + rl) * LDV + cim] = to_h(ei[i] - oi[i]);
      }
      __builtin_amdgcn_sched_barrier(0);  // bound the hoisting of LDS reads
    }
    __syncthreads();

    // this wave's rows of V (tiles u: r, r + Na/2), per class, as B operands
    h8 vf[2][2][NKVC];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int k = 0; k < NKVC; ++k)
          vf[u][c][k] = M::ld(VL + (u * W2_H + wave * 16 + r16) * LDV + c * 2 * KBPC +
                              k * W2_KS + g * 8);
    __syncthreads();  // V read: its space takes the twiddle blocks
    stTW(twr[0], 0);
    __syncthreads();

    // ---- step A' (last axis, radix-2) ------------------------------------------
    const __amdgpu_buffer_rsrc_t ry = plane_rsrc(a.out, p, plane_bytes);
    const __amdgpu_buffer_rsrc_t rx = plane_rsrc(EPI ? a.x : a.out, p, plane_bytes);
    const __amdgpu_buffer_rsrc_t rxn = more ? plane_rsrc(EPI ? a.x : a.out, pn, plane_bytes) : rx;
    // planes of one item (narrow variant): the next plane's spectrum is
    // requested a whole item before it is staged (zq is free: this plane's
    // staging has read it)
    const bool z_early = NCTC == 2 && nch == 1;
    if (more && z_early) ldZ(pn, zq);
    // request the unit after unit t of block b (operands selected where
    // there is no next item: this item's first unit again, in range)
    auto req = [&](int b, int t) {
      const int t1 = t + 1;
      if (t1 < 2 * NQ) ldX(rx, c0, b, t1 / NQ, t1 % NQ, xr[t1 & 1]);
      else if (b + 1 < nmb) ldX(rx, c0, b + 1, 0, 0, xr[0]);
      else ldX(rxn, more ? cn : c0, 0, 0, 0, xr[0]);
    };
    auto block = [&](int b, int par) {
      // twiddles requested two blocks (one 128-column block) ahead; the
      // sequence wraps at the item boundary: every item walks the same blocks
      if (TWA == 2) ldTW(b + 2 < nmb ? b + 2 : b + 2 - nmb, twr[par & (TWA - 1)]);
      else ldTW(b + 1 < nmb ? b + 1 : 0, twr[0]);
      const _Float16* tb = TW + par * (MB * LDT) + r16 * LDT + g * 8;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int t = u * NQ + q;
          if (EPI) req(b, t);  // before this unit's products
          // the unit's four 16-column tiles
          f4 ae[4], ao[4];
#pragma unroll
          for (int c4 = 0; c4 < 4; ++c4) {
            const int c = q * 4 + c4;
            ae[c4] = ao[c4] = f4zero();
#pragma unroll
            for (int k = 0; k < NKVC; ++k) {
              ae[c4] = M::mma(M::ld(tb + c * 16 * LDT + k * W2_KS), vf[u][0][k], ae[c4]);
              ao[c4] = M::mma(M::ld(tb + c * 16 * LDT + 2 * KBPC + k * W2_KS), vf[u][1][k], ao[c4]);
            }
          }
          const u32x4 (&xs2)[2][2] = xr[t & 1];
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const u32x4 (&xs)[2] = xs2[hf];
            // D: lane holds row r16 of the tile, columns m = c 16 + 4 g + i
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) {
              f4 v;
#pragma unroll
              for (int i = 0; i < 4; ++i)
                v[i] = (hf == 0 ? ae[c4][i] + ao[c4][i] : ae[c4][i] - ao[c4][i]) * a.scale;
              if (OB16) {
                const h4 hv = {to_h(v[0]), to_h(v[1]), to_h(v[2]), to_h(v[3])};
                *reinterpret_cast<h4*>(obh + r16 * W2_LDOH + c4 * 16 + 4 * g) = hv;
              } else {
                *reinterpret_cast<f4*>(ob + r16 * W2_LDO + ob_col(c4 * 16 + 4 * g)) = v;
              }
            }
            wave_lds_sync();
            // one row group h (row lane / 8 + 8 h, columns (lane % 8) 8 + e) at
            // a time: read, epilogue, store
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              float v[8];
              if (OB16) {
                const h8 t8 = *reinterpret_cast<const h8*>(obh + ((lane >> 3) + 8 * h) * W2_LDOH +
                                                           (lane & 7) * 8);
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = (float)t8[e];
              } else {
#pragma unroll
                for (int e0 = 0; e0 < 8; e0 += 4) {
                  const f4 t4 = *reinterpret_cast<const f4*>(
                      ob + ((lane >> 3) + 8 * h) * W2_LDO + ob_col((lane & 7) * 8 + e0));
#pragma unroll
                  for (int i = 0; i < 4; ++i) v[e0 + i] = t4[i];
                }
              }
              if (EPI) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const uint32_t sw = lut2<false>(lut, xs[h][e], sat);
                  h2 s2;
                  __builtin_memcpy(&s2, &sw, 4);
                  v[2 * e] *= (float)s2[0];
                  v[2 * e + 1] *= (float)s2[1];
                }
              }
              h8 w;
#pragma unroll
              for (int e = 0; e < 8; ++e) w[e] = to_h(v[e]);
              u32x4 wv;
              __builtin_memcpy(&wv, &w, 16);
              // the whole offset in the vector operand: with an SGPR offset
              // the compiler leaves no wait states between this store and a
              // VALU write of its data registers, and the store has then
              // been seen to take the new values of some lanes
              __builtin_amdgcn_raw_buffer_store_b128(wv, ry, xoff(c0, b, hf, h) + q * 128 + u * hiA,
                                                     0, W2_NTS);
            }
            wave_lds_sync();  // the buffer is written again by the next segment
          }
        }
      }
      stTW(twr[(1 - par) & (TWA - 1)], 1 - par);
      __syncthreads();
    };
#pragma nounroll
    for (int b = 0; b < nmb - 2; b += 2) {
      block(b, 0);
      block(b + 1, 1);
    }
    block(nmb - 2, 0);
    // next item's step-B' table rows, one block before they are needed
    // (registers free during the other blocks)
    ldC(cn, cf, sf);
    block(nmb - 1, 1);
    // otherwise after the plane's last block
    if (more && cn == 0 && !z_early) ldZ(pn, zq);
  }
}

// ---------------------------------------------------------------------------
// Launchers (hipErrorNotSupported: the shape is not one of this path's)
// ---------------------------------------------------------------------------
size_t r2c_wide2_lds_bytes(int nctc, bool pre, int lut_sat) {
  const int kbpc = nctc * 8;
  const size_t at = (size_t)4 * 2 * kbpc * W2_LDR * 2;
  const size_t tw = (size_t)2 * 4 * kbpc * W2_LDT * 2;
  return at + tw + (pre ? (size_t)lutn_bytes(lut_sat) : 0);
}

size_t c2r_wide2_lds_bytes(int nctc, int nkzh, bool epi, int lut_sat) {
  size_t base = 0;
#define FNO_C2RW2_BYTES(N, K) \
  if (nctc == N && nkzh == K) base = C2RWide2<N, K>::zt_bytes + C2RWide2<N, K>::reg_bytes;
  // the wide variant may take 128-column blocks (enough for both)
  if (nctc == 4 && nkzh == 2)
    return epi ? C2RWide2<4, 2, 128, true>::zt_bytes + C2RWide2<4, 2, 128, true>::reg_bytes +
                     (size_t)w2_lut_bytes(lut_sat)
               : C2RWide2<4, 2, 128>::zt_bytes + C2RWide2<4, 2, 128>::reg_bytes;
  FNO_C2RW2_BYTES(2, 1) FNO_C2RW2_BYTES(2, 2) FNO_C2RW2_BYTES(4, 1) FNO_C2RW2_BYTES(4, 2)
#undef FNO_C2RW2_BYTES
  if (base == 0) return (size_t)1 << 30;  // not a shape of this path
  return base + (epi ? (size_t)w2_lut_bytes(lut_sat) : 0);
}

template <int NCTC, bool PRE, bool EARLY>
static hipError_t r2c_wide2_go(const R2CArgs& a, int grid, size_t lds, hipStream_t s) {
  const void* k = (const void*)&r2c_wide2_kernel<NCTC, PRE, EARLY>;
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((r2c_wide2_kernel<NCTC, PRE, EARLY>), dim3(grid), dim3(W2_NT), lds, s, a);
  return hipGetLastError();
}

// a.twA, a.cB, a.sB: the radix-2 tables; a.Kap16: leading-axis rows per
// class padded to a tile count of 1, 2 or 4; a.early: the early requests of
// the narrow variant (ignored for nctc 4).  Shapes: nctc in {2, 4}, Na and Nb
// multiples of 256.
hipError_t launch_r2c_wide2(const R2CArgs& a, int nctc, int grid, size_t lds, hipStream_t s) {
  const int nta = a.Kap16 / 16;
  if (lds > 160 * 1024 || a.Na % 256 != 0 || a.Nb % 256 != 0 || a.Kap16 % 16 != 0 ||
      (nta != 1 && nta != 2 && nta != 4) || grid <= 0)
    return hipErrorNotSupported;
  const bool t = a.do_tanh != 0;
  if (nctc == 2 && a.early)
    return t ? r2c_wide2_go<2, true, true>(a, grid, lds, s) : r2c_wide2_go<2, false, true>(a, grid, lds, s);
  if (nctc == 2)
    return t ? r2c_wide2_go<2, true, false>(a, grid, lds, s) : r2c_wide2_go<2, false, false>(a, grid, lds, s);
  if (nctc == 4)
    return t ? r2c_wide2_go<4, true, false>(a, grid, lds, s) : r2c_wide2_go<4, false, false>(a, grid, lds, s);
  return hipErrorNotSupported;
}

template <int NCTC, int NKZH>
static hipError_t c2r_wide2_go(const C2RArgs& a, int grid, size_t lds, hipStream_t s) {
  const void* k = a.epilogue ? (const void*)&c2r_wide2_kernel<NCTC, NKZH, true>
                             : (const void*)&c2r_wide2_kernel<NCTC, NKZH, false>;
  hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 gr(grid), bl(W2_NT);
  if (a.epilogue) hipLaunchKernelGGL((c2r_wide2_kernel<NCTC, NKZH, true>), gr, bl, lds, s, a);
  else hipLaunchKernelGGL((c2r_wide2_kernel<NCTC, NKZH, false>), gr, bl, lds, s, a);
  return hipGetLastError();
}

// a.cI, a.sI, a.twI: the radix-2 tables; a.Kap: leading-axis slots per class
// padded to 32 (nkzh = a.Kap / 32).  Shapes: nctc in {2, 4}, nkzh in {1, 2},
// Ka Kb <= 8192 and Kb a multiple of 4, Na and Nb multiples of 256.
hipError_t launch_c2r_wide2(const C2RArgs& a, int nctc, int grid, size_t lds, hipStream_t s) {
  if (lds > 160 * 1024 || a.Ka * a.Kb > 8192 || a.Nb % 256 != 0 || a.Na % 256 != 0 ||
      a.Kb % 4 != 0 || grid <= 0)
    return hipErrorNotSupported;
  const int nkzh = a.Kap / 32;
  if (nctc == 2 && nkzh == 1) return c2r_wide2_go<2, 1>(a, grid, lds, s);
  if (nctc == 2 && nkzh == 2) return c2r_wide2_go<2, 2>(a, grid, lds, s);
  if (nctc == 4 && nkzh == 1) return c2r_wide2_go<4, 1>(a, grid, lds, s);
  // wide variant, Nb / 2 a multiple of 256 (an even count of 128-column
  // blocks): 128-column blocks
  if (nctc == 4 && nkzh == 2 && (a.Nb / 2) % 256 == 0) {
    const void* k = a.epilogue ? (const void*)&c2r_wide2_kernel<4, 2, true, 128>
                               : (const void*)&c2r_wide2_kernel<4, 2, false, 128>;
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (a.epilogue)
      hipLaunchKernelGGL((c2r_wide2_kernel<4, 2, true, 128>), dim3(grid), dim3(W2_NT), lds, s, a);
    else
      hipLaunchKernelGGL((c2r_wide2_kernel<4, 2, false, 128>), dim3(grid), dim3(W2_NT), lds, s, a);
    return hipGetLastError();
  }
  if (nctc == 4 && nkzh == 2) return c2r_wide2_go<4, 2>(a, grid, lds, s);
  return hipErrorNotSupported;
}

}  // namespace fno
