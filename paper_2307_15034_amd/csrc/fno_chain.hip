// Chained fp16 truncated transforms: one wavefront per plane, no block
// barriers after the one-time table staging, no LDS round trip for data.
//
// Both axes of a plane transform are DFT-by-MFMA products.  The contraction
// index of an MFMA may be ordered arbitrarily inside a k-step as long as the
// two operands agree, so the k-slots of the second product are chosen to be
// exactly the (row, column) positions that the lane already holds in the
// result registers of the first product (D lane: rows 4g..4g+3 of a 16x16
// tile).  The constant twiddle operand is stored with the matching
// permutation; the data operand never leaves the registers.
//
//   forward  (per plane): x[Na][Nb] -> step A (last axis, x . [cos | -sin])
//            -> step B (leading axis, complex, accumulated over 32-row blocks)
//            -> spectrum [Ka][Kb]
//   inverse  (per plane): spectrum -> step B' (leading axis, per 16-row tile
//            of the output) -> step A' (last axis, real part) -> y[Na][Nb]
//
// Output rows of the last products are also permuted so that every lane
// ends up with contiguous output elements (16-byte stores).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

namespace {

typedef MM<_Float16> MH;
constexpr int KS = 32;   // k per MFMA step (v_mfma_f32_16x16x32_f16)
constexpr int PADH = 8;  // LDS row padding in halves
constexpr int CH_NW = kChainWaves;  // waves per work-group, one plane each at a time

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h8 u_as_h8(const u32x4& v) {
  h8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ u32x4 h8_as_u4(const h8& v) {
  u32x4 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// -v for eight fp16 values: one sign-bit XOR per register
__device__ __forceinline__ h8 neg_h8(const h8& v) {
  u32x4 r = h8_as_u4(v);
#pragma unroll
  for (int w = 0; w < 4; ++w) r[w] ^= 0x80008000u;
  return u_as_h8(r);
}

// Copy of a [rows][cols] fp16 table (row stride gstride) into LDS rows of
// stride lstride (cols, strides multiples of 8), at most MAXP 16-byte pieces
// per thread.  All loads are issued before any store, so staging costs one
// memory latency rather than one per piece.
template <int MAXP>
struct Stager {
  u32x4 v[MAXP];
  __device__ __forceinline__ void load(const _Float16* src, int gstride, int rows, int cols,
                                       const _Float16* zeros) {
    const int cpr = cols / 8;
#pragma unroll
    for (int k = 0; k < MAXP; ++k) {
      const int i = threadIdx.x + k * CH_NW * 64;
      const int r = i / cpr, c = (i - r * cpr) * 8;
      const bool ok = i < rows * cpr;
      v[k] = *reinterpret_cast<const u32x4*>(ok ? src + (int64_t)r * gstride + c : zeros);
    }
  }
  __device__ __forceinline__ void store(_Float16* dst, int lstride, int rows, int cols) const {
    const int cpr = cols / 8;
#pragma unroll
    for (int k = 0; k < MAXP; ++k) {
      const int i = threadIdx.x + k * CH_NW * 64;
      const int r = i / cpr, c = (i - r * cpr) * 8;
      if (i < rows * cpr) *reinterpret_cast<u32x4*>(dst + r * lstride + c) = v[k];
    }
  }
};

// Table lookup of two fp16 values packed in w: the LDS table holds f(|x|)
// for the 32768 non-negative codes; `odd` restores the sign (f odd).
// 2 * code of the low half is (w << 1) & 0xfffe, of the high half
// (w >> 15) & 0xfffe.
template <bool ODD>
__device__ __forceinline__ unsigned lut_pair(const _Float16* tab, unsigned w) {
  const unsigned lo = (w << 1) & 0xfffeu, hi = (w >> 15) & 0xfffeu;
  const char* t = reinterpret_cast<const char*>(tab);
  h2 r;
  r[0] = *reinterpret_cast<const _Float16*>(t + lo);
  r[1] = *reinterpret_cast<const _Float16*>(t + hi);
  unsigned u;
  __builtin_memcpy(&u, &r, 4);
  return ODD ? (u | (w & 0x80008000u)) : u;
}

template <bool ODD>
__device__ __forceinline__ u32x4 lut_u4(const _Float16* tab, const u32x4& w) {
  return u32x4{lut_pair<ODD>(tab, w[0]), lut_pair<ODD>(tab, w[1]), lut_pair<ODD>(tab, w[2]),
               lut_pair<ODD>(tab, w[3])};
}

constexpr int LUT_HALVES = 32768;  // one entry per non-negative fp16 code

// cache-policy operand of buffer stores: non-temporal (streaming) store
constexpr int CPOL_NT = 2;

// Position in a wave's flattened sequence of (plane, block) work items.
struct Pos {
  int64_t p;
  int j;
};

}  // namespace

// ---------------------------------------------------------------------------
// Forward.  Template: NKA = ceil(Nb / 32) k-steps of step A, NTB = Kbp / 16
// spectrum column tiles, NTA = Kap16 / 16 spectrum row tiles.
//
// Step A of a 32-row block (two 16-row tiles, rt = 0, 1) gives, per column
// tile ct, D registers holding Y[32 j + 16 rt + 4 g + i][col(ct, l % 16)].
// Column tile ct is part ct / NTB (0: cos -> Re, 1: -sin -> Im) of the
// spectrum columns tb = NTB * (l % 16) + ct % NTB.  Step B takes those eight
// values (rt = 0, 1; i = 0..3) as the B operand of one k-step; the leading-
// axis table column 32 j + 8 g + e holds the matching row n_a.
// ---------------------------------------------------------------------------
template <int NKA, int NTB, int NTA, bool PRE>
__global__ __launch_bounds__(CH_NW * 64, 2) void r2c_chain_kernel(R2CArgs a) {
  constexpr int NCT = 2 * NTB;
  constexpr int LDT = NKA * KS + PADH;
  extern __shared__ __align__(16) unsigned char smem[];
  // the wave index is the same on every lane: keep it (and the loop control
  // derived from it) in scalar registers
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int LDE = a.NaC + PADH;
  // the lookup table is a static LDS array (at a known address, so lookups
  // need no base add); the twiddle tables are dynamic LDS after it
  __shared__ __align__(16) _Float16 sLut[PRE ? LUT_HALVES : 8];  // f(x) of each fp16 code
  _Float16* sT = reinterpret_cast<_Float16*>(smem);    // [NCT * 16][LDT]
  _Float16* sEc = sT + NCT * 16 * LDT;                // [NTA * 16][LDE]
  _Float16* sEs = sEc + NTA * 16 * LDE;
  const _Float16* x = reinterpret_cast<const _Float16*>(a.in);
  const _Float16* zr = reinterpret_cast<const _Float16*>(a.zeros);
  _Float16* out = reinterpret_cast<_Float16*>(a.out);

  // tables: 16 NCT rows x 4 NKA pieces, and 16 NTA rows x NaC / 8 <= 16 pieces
  constexpr int PT = (NCT * 16 * NKA * 4 + CH_NW * 64 - 1) / (CH_NW * 64);
  constexpr int PE = (NTA * 16 * 16 + CH_NW * 64 - 1) / (CH_NW * 64);
  Stager<PT> st;
  Stager<PE> sc, ss;
  Stager<PRE ? LUT_HALVES / 8 / (CH_NW * 64) : 1> sl;

  const int NJ = a.NaC / 32;
  const int64_t plane = (int64_t)a.Na * a.Nb;
  const int64_t W = (int64_t)gridDim.x * CH_NW;
  auto next = [&](Pos q) -> Pos { return q.j + 1 < NJ ? Pos{q.p, q.j + 1} : Pos{q.p + W, 0}; };

  // Row block (p, j): lane holds rows 32 j + 16 rt + r16, columns 32 s + 8 g.
  // Buffer loads through a per-plane resource (scalar registers); lanes past
  // the plane's rows or columns, and every lane past the last plane (an empty
  // resource), read zeros.  All loads are issued, so the wait before each use
  // counts exactly the loads issued after it.
  // beyond every plane (planes < 2^29 bytes); a row and a column offset that
  // are both BIG still add up to less than 2^31
  constexpr int BIG = 0x20000000;
  int colo[NKA];
#pragma unroll
  for (int s = 0; s < NKA; ++s) {
    const int col = s * KS + g * 8;
    colo[s] = col < a.Nb ? col * 2 : BIG;
  }
  auto load = [&](Pos q, u32x4 (&buf)[2][NKA]) {
    const bool pok = q.p < a.planes;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<_Float16*>(x + (pok ? q.p : 0) * plane), (short)0, pok ? (int)(plane * 2) : 0,
        0x00020000);
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int row = 32 * q.j + 16 * rt + r16;
      const int rowo = row < a.Na ? row * a.Nb * 2 : BIG;
#pragma unroll
      for (int s = 0; s < NKA; ++s) buf[rt][s] = __builtin_amdgcn_raw_buffer_load_b128(rs, rowo + colo[s], 0, 0);
    }
  };

  f4 zre[NTA][NTB], zim[NTA][NTB];

  // ---- step A: 32 rows x [cos | -sin]; returns the step-B operands ------------
  auto step_a = [&](const u32x4 (&buf)[2][NKA], h8 (&yf)[NCT]) {
    f4 acc[2][NCT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[rt][ct] = f4zero();
#pragma unroll
    for (int s = 0; s < NKA; ++s) {
      h8 v0, v1;
      if constexpr (PRE) {
        // the pre-activation f (odd: tanh or the hard clip) rounded to fp16,
        // looked up per fp16 code
        v0 = u_as_h8(lut_u4<true>(sLut, buf[0][s]));
        v1 = u_as_h8(lut_u4<true>(sLut, buf[1][s]));
      } else {
        v0 = u_as_h8(buf[0][s]);
        v1 = u_as_h8(buf[1][s]);
      }
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const h8 bf = MH::ld(sT + (ct * 16 + r16) * LDT + s * KS + g * 8);
        acc[0][ct] = MH::mma(v0, bf, acc[0][ct]);
        acc[1][ct] = MH::mma(v1, bf, acc[1][ct]);
      }
    }
    // fp16, scaled: slots 0..3 rows 32 j + 4 g + i, slots 4..7 rows + 16
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        yf[ct][i] = to_h(acc[0][ct][i] * a.scaleA);
        yf[ct][4 + i] = to_h(acc[1][ct][i] * a.scaleA);
      }
  };

  // ---- step B: Z[t_a][t_b] += (c - i s)[t_a][rows] (Yr + i Yi)[rows][t_b] -----
  auto step_b = [&](Pos q, const h8 (&yf)[NCT]) {
    if (q.j == 0) {
#pragma unroll
      for (int ta = 0; ta < NTA; ++ta)
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) zre[ta][tb] = zim[ta][tb] = f4zero();
    }
#pragma unroll
    for (int ta = 0; ta < NTA; ++ta) {
      const int eo = (ta * 16 + r16) * LDE + 32 * q.j + g * 8;
      const h8 cf = MH::ld(sEc + eo), sf = MH::ld(sEs + eo);
      const h8 nsf = neg_h8(sf);
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        zre[ta][tb] = MH::mma(cf, yf[tb], zre[ta][tb]);
        zre[ta][tb] = MH::mma(sf, yf[NTB + tb], zre[ta][tb]);
        zim[ta][tb] = MH::mma(cf, yf[NTB + tb], zim[ta][tb]);
        zim[ta][tb] = MH::mma(nsf, yf[tb], zim[ta][tb]);
      }
    }
    if (q.j == NJ - 1) {
      // lane holds Z[16 ta + 4 g + i][NTB r16 + tb]: NTB consecutive complex.
      // Buffer stores through the output plane's resource; lanes past Ka or
      // Kb carry an offset beyond it (the store is dropped), so no branch.
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          out + q.p * (int64_t)a.Ka * a.Kb * 2, (short)0, a.Ka * a.Kb * 4, 0x00020000);
      // Kb % 4 == 0 (dispatcher) and NTB <= 4: a lane's NTB columns are
      // either all below Kb or all past it.  Row t_a = 16 ta + i + 4 g is
      // valid iff 16 ta + i < Ka - 4 g.  (The empty asm keeps the compiler
      // from hoisting the sixteen offsets out of the plane loop.)
      const int tb0 = NTB * r16;
      int sb = tb0 < a.Kb ? (4 * g * a.Kb + tb0) * 4 : BIG;
      int glim = a.Ka - 4 * g;
      asm volatile("" : "+v"(sb), "+v"(glim));
#pragma unroll
      for (int ta = 0; ta < NTA; ++ta)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 16 * ta + i;
          const int vo = r < glim ? sb + r * a.Kb * 4 : BIG;
          _Float16 v[2 * NTB];
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb) {
            v[2 * tb] = to_h(zre[ta][tb][i] * a.scaleB);
            v[2 * tb + 1] = to_h(zim[ta][tb][i] * a.scaleB);
          }
          if constexpr (NTB == 1) {
            u32 w;
            __builtin_memcpy(&w, v, 4);
            __builtin_amdgcn_raw_buffer_store_b32(w, rs, vo, 0, 0);
          } else if constexpr (NTB == 2) {
            u32x2 w;
            __builtin_memcpy(&w, v, 8);
            __builtin_amdgcn_raw_buffer_store_b64(w, rs, vo, 0, 0);
          } else {
            u32x4 w;
            __builtin_memcpy(&w, v, 16);
            __builtin_amdgcn_raw_buffer_store_b128(w, rs, vo, 0, 0);
          }
        }
    }
  };

  // Each wave walks its planes p = wave_id, wave_id + W, ... in 32-row blocks
  // (nitems blocks in all, a wave-uniform count).  Two register buffers in
  // fixed roles (loop unrolled by two): a buffer is refilled with the block
  // two ahead as soon as step A has consumed it, so those loads overlap this
  // block's step B and the next block's step A.  The loop has one exit test
  // per pair, so every pass through the loop head has the same loads in
  // flight and the wait before each step A covers that block only.
  const int64_t pw = (int64_t)blockIdx.x * CH_NW + wave;
  const int64_t nitems = pw < a.planes ? ((a.planes - 1 - pw) / W + 1) * NJ : 0;
  Pos q0{pw, 0};
  Pos q1 = next(q0);
  u32x4 b0[2][NKA], b1[2][NKA];
  h8 yf[NCT];
  // Load order: the first row block, the tables, and (after the barrier) the
  // second row block.  The first block and the tables are what the first
  // step needs; requesting the second block only once they have arrived
  // lets them arrive sooner (all waves start at once, and the memory system
  // does not serve requests in order).
  load(q0, b0);
  __builtin_amdgcn_sched_barrier(0);
  st.load(reinterpret_cast<const _Float16*>(a.twAc), a.Nbp, NCT * 16, NKA * KS, zr);
  sc.load(reinterpret_cast<const _Float16*>(a.cBc), a.NaC, NTA * 16, a.NaC, zr);
  ss.load(reinterpret_cast<const _Float16*>(a.sBc), a.NaC, NTA * 16, a.NaC, zr);
  if constexpr (PRE) sl.load(reinterpret_cast<const _Float16*>(a.lut), 0, 1, LUT_HALVES, zr);
  __builtin_amdgcn_sched_barrier(0);
  st.store(sT, LDT, NCT * 16, NKA * KS);
  sc.store(sEc, LDE, NTA * 16, a.NaC);
  ss.store(sEs, LDE, NTA * 16, a.NaC);
  if constexpr (PRE) sl.store(sLut, 0, 1, LUT_HALVES);
  __syncthreads();  // tables staged
  load(q1, b1);
  int64_t it = 0;
  for (; it + 2 <= nitems; it += 2) {
    step_a(b0, yf);
    const Pos c0 = q0;
    q0 = next(q1);
    load(q0, b0);
    step_b(c0, yf);
    step_a(b1, yf);
    const Pos c1 = q1;
    q1 = next(q0);
    load(q1, b1);
    step_b(c1, yf);
  }
  if (it < nitems) {
    step_a(b0, yf);
    step_b(q0, yf);
  }
}

// ---------------------------------------------------------------------------
// Inverse.  Template: NG = Nb64 / 64 output column groups, NTB = Kbp / 16,
// NKZ = Kap / 32 k-steps of step B'.  EPI multiplies by f'(x), the
// derivative of the pre-activation.
//
// Step B' for one 16-row output tile computes V^T[t_b][n_a] (complex) with
// Z^T as the A operand (gathered from global memory, k = t_a) and the
// leading-axis table as B.  Its D registers hold V^T rows t_b = 16 tt + 4 g
// + i, which are the k-slots of step A' (y^T = T'^T V'^T); the last-axis
// table column 32 ks + 8 g + e names (part, t_b) to match.  Row R of output
// tile T covers n_b = 64 (T / 4) + 16 (R / 4) + 4 (T % 4) + R % 4, so a lane
// holds 16 consecutive n_b of its row per group of four tiles.
// ---------------------------------------------------------------------------
template <int NG, int NTB, int NKZ, bool EPI>
__global__ __launch_bounds__(CH_NW * 64, 2) void c2r_chain_kernel(C2RArgs a) {
  constexpr int NYT = 4 * NG;  // output tiles (16 columns each) per row tile
  constexpr int LDI = 2 * NTB * 16 + PADH;
  extern __shared__ __align__(16) unsigned char smem[];
  // the wave index is the same on every lane: keep it (and the loop control
  // derived from it) in scalar registers
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int LDK = a.Kap + PADH;
  const int NAT = (a.Na + 15) / 16;
  // static LDS lookup table (see the forward kernel), dynamic tables after
  __shared__ __align__(16) _Float16 sLut[EPI ? LUT_HALVES : 8];  // f'(x) per fp16 code
  _Float16* sTI = reinterpret_cast<_Float16*>(smem);   // [NG * 64][LDI]
  _Float16* sCI = sTI + NG * 64 * LDI;                 // [NAT * 16][LDK]
  _Float16* sSI = sCI + NAT * 16 * LDK;
  // per-wave output staging: 16 rows x 64 columns (one column group)
  constexpr int LDO = 64 + PADH;
  _Float16* sOut = sSI + NAT * 16 * LDK + wave * 16 * LDO;
  const _Float16* zin = reinterpret_cast<const _Float16*>(a.in);
  const _Float16* xin = reinterpret_cast<const _Float16*>(a.x);
  const _Float16* zr = reinterpret_cast<const _Float16*>(a.zeros);
  _Float16* yout = reinterpret_cast<_Float16*>(a.out);

  // tables: 64 NG rows x 4 NTB pieces, and <= 128 rows x 4 NKZ pieces
  constexpr int PT = (NG * 64 * NTB * 4 + CH_NW * 64 - 1) / (CH_NW * 64);
  constexpr int PE = (128 * NKZ * 4 + CH_NW * 64 - 1) / (CH_NW * 64);
  Stager<PT> st;
  Stager<PE> sc, ss;
  Stager<EPI ? LUT_HALVES / 8 / (CH_NW * 64) : 1> sl;

  const int64_t plane = (int64_t)a.Na * a.Nb;
  const int64_t zplane = (int64_t)a.Ka * a.Kb * 2;
  const int64_t W = (int64_t)gridDim.x * CH_NW;
  auto next = [&](Pos q) -> Pos { return q.j + 1 < NAT ? Pos{q.p, q.j + 1} : Pos{q.p + W, 0}; };

  // Buffer loads and stores through per-plane resources (scalar registers):
  // lanes past a plane's rows or columns carry an offset beyond it (loads
  // read zeros, stores are dropped), and a plane past the last has an empty
  // resource, so every load is issued and no store needs a branch.
  // beyond every plane (planes < 2^29 bytes); a row and a column offset that
  // are both BIG still add up to less than 2^31
  constexpr int BIG = 0x20000000;
  auto rsrc = [&](const _Float16* base, int64_t p, int64_t halves) {
    const bool pok = p < a.planes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<_Float16*>(base + (pok ? p : 0) * halves),
                                             (short)0, pok ? (int)(halves * 2) : 0, 0x00020000);
  };
  // Spectrum plane as MFMA A operands, natural layout: lane (r16, g) holds
  // row t_a = 16 rt + r16, complex t_b = 16 kz + 4 g .. + 4 (16-byte loads).
  auto load_z = [&](int64_t p, u32x4 (&buf)[2 * NKZ][NTB]) {
    const __amdgpu_buffer_rsrc_t rs = rsrc(zin, p, zplane);
#pragma unroll
    for (int rt = 0; rt < 2 * NKZ; ++rt)
#pragma unroll
      for (int kz = 0; kz < NTB; ++kz) {
        const int ta = 16 * rt + r16, tb = 16 * kz + 4 * g;
        const int vo = (ta < a.Ka && tb < a.Kb) ? (ta * a.Kb + tb) * 4 : BIG;
        buf[rt][kz] = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, 0, 0);
      }
  };
  // epilogue input of row tile (p, j): row 16 j + r16, columns 64 G + 16 g + 8 h
  constexpr int XG = EPI ? NG : 1;
  int colx[XG][2];
#pragma unroll
  for (int G = 0; G < XG; ++G)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int col = 64 * G + 16 * g + 8 * h;
      colx[G][h] = col < a.Nb ? col * 2 : BIG;
    }
  auto load_x = [&](Pos q, u32x4 (&buf)[XG][2]) {
    if constexpr (EPI) {
      const __amdgpu_buffer_rsrc_t rs = rsrc(xin, q.p, plane);
      const int row = 16 * q.j + r16;
      const int rowo = row < a.Na ? row * a.Nb * 2 : BIG;
#pragma unroll
      for (int G = 0; G < NG; ++G)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          buf[G][h] = __builtin_amdgcn_raw_buffer_load_b128(rs, rowo + colx[G][h], 0, 0);
    }
  };

  h8 zfr[NTB][NKZ], zfi[NTB][NKZ];
  // Selection operands that move (re, im) of a 16x32 block of Z into a D
  // tile of its transpose: B[k][j] = 1 where k = 2 j (re) or 2 j + 1 (im).
  h8 selr, seli;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    selr[e] = (_Float16)(8 * g + e == 2 * r16 ? 1.0f : 0.0f);
    seli[e] = (_Float16)(8 * g + e == 2 * r16 + 1 ? 1.0f : 0.0f);
  }

  // A spectrum plane, transposed by the selection products (exact): D lane
  // (r16, g) gets Re/Im Z[16 rt + 4 g + i][16 kz + r16]; the step-B' k-step
  // ks takes row tiles 2 ks (slots 0..3) and 2 ks + 1 (4..7).
  auto transpose_z = [&](const u32x4 (&zraw)[2 * NKZ][NTB]) {
#pragma unroll
    for (int kz = 0; kz < NTB; ++kz)
#pragma unroll
      for (int ks = 0; ks < NKZ; ++ks)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const h8 av = u_as_h8(zraw[2 * ks + hh][kz]);
          const f4 dr = MH::mma(av, selr, f4zero());
          const f4 di = MH::mma(av, seli, f4zero());
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            zfr[kz][ks][4 * hh + i] = to_h(dr[i]);
            zfi[kz][ks][4 * hh + i] = to_h(di[i]);
          }
        }
  };
  const int64_t first_plane = (int64_t)blockIdx.x * CH_NW + wave;

  auto process = [&](Pos q, const u32x4 (&xb)[XG][2]) {
    if (q.j == 0 && q.p != first_plane) {
      // a later plane of this wave (the first one is loaded up front)
      u32x4 zraw[2 * NKZ][NTB];
      load_z(q.p, zraw);
      transpose_z(zraw);
    }
    // ---- step B': V^T[t_b][n_a] = sum_t_a Z^T[t_b][t_a] (c + i s)[t_a][n_a] -----
    f4 vr[NTB], vi[NTB];
#pragma unroll
    for (int tt = 0; tt < NTB; ++tt) vr[tt] = vi[tt] = f4zero();
#pragma unroll
    for (int ks = 0; ks < NKZ; ++ks) {
      const int eo = (16 * q.j + r16) * LDK + 32 * ks + 8 * g;
      const h8 cf = MH::ld(sCI + eo), sf = MH::ld(sSI + eo);
      const h8 nsf = neg_h8(sf);
#pragma unroll
      for (int tt = 0; tt < NTB; ++tt) {
        vr[tt] = MH::mma(zfr[tt][ks], cf, vr[tt]);
        vr[tt] = MH::mma(zfi[tt][ks], nsf, vr[tt]);
        vi[tt] = MH::mma(zfr[tt][ks], sf, vi[tt]);
        vi[tt] = MH::mma(zfi[tt][ks], cf, vi[tt]);
      }
    }
    // pairs (part, tile) in the order Re tiles, then Im tiles; k-step ks of
    // step A' takes pairs 2 ks (slots 0..3) and 2 ks + 1 (slots 4..7)
    h8 vf[NTB];
#pragma unroll
    for (int ks = 0; ks < NTB; ++ks)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int pi = 2 * ks + hh;
        const f4& src = pi < NTB ? vr[pi] : vi[pi - NTB];
#pragma unroll
        for (int i = 0; i < 4; ++i) vf[ks][4 * hh + i] = to_h(src[i]);
      }
    // ---- step A': y^T[n_b][n_a] = sum_k T'^T[n_b][k] V'^T[k][n_a] --------------
    f4 yacc[NYT];
#pragma unroll
    for (int t = 0; t < NYT; ++t) yacc[t] = f4zero();
#pragma unroll
    for (int ks = 0; ks < NTB; ++ks)
#pragma unroll
      for (int t = 0; t < NYT; ++t) {
        const h8 tf = MH::ld(sTI + (16 * t + r16) * LDI + 32 * ks + 8 * g);
        yacc[t] = MH::mma(tf, vf[ks], yacc[t]);
      }
    // ---- epilogue: lane holds y[16 j + r16][64 G + 16 g .. + 16] ---------------
    const __amdgpu_buffer_rsrc_t ry = rsrc(yout, q.p, plane);
#pragma unroll
    for (int G = 0; G < NG; ++G) {
      float v[16];
#pragma unroll
      for (int tq = 0; tq < 4; ++tq)
#pragma unroll
        for (int i = 0; i < 4; ++i) v[4 * tq + i] = yacc[4 * G + tq][i] * a.scale;
      if constexpr (EPI) {
        // f'(x) (even), rounded to fp16, looked up per fp16 code
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const h8 fv = u_as_h8(lut_u4<false>(sLut, xb[G][h]));
#pragma unroll
          for (int e = 0; e < 8; ++e) v[8 * h + e] *= (float)fv[e];
        }
      }
      // Restage the 16 x 64 block through this wave's LDS so that each
      // store instruction writes whole 128-byte rows (8 lanes per row):
      // the streaming stores below bypass the caches that would otherwise
      // merge partial lines.
      h8 o0, o1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        o0[e] = to_h(v[e]);
        o1[e] = to_h(v[8 + e]);
      }
      *reinterpret_cast<h8*>(sOut + r16 * LDO + 16 * g) = o0;
      *reinterpret_cast<h8*>(sOut + r16 * LDO + 16 * g + 8) = o1;
      wave_lds_sync();
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int rr = (lane >> 3) + 8 * k, c8 = (lane & 7) * 8;
        const u32x4 val = *reinterpret_cast<const u32x4*>(sOut + rr * LDO + c8);
        const int row = 16 * q.j + rr, col = 64 * G + c8;
        // Nb % 16 == 0 (dispatcher): a 16-byte piece is all in range or out.
        // Streaming (non-temporal) stores: the layer does not read y again.
        const int vo = (row < a.Na && col < a.Nb) ? (row * a.Nb + col) * 2 : BIG;
        __builtin_amdgcn_raw_buffer_store_b128(val, ry, vo, 0, CPOL_NT);
      }
      wave_lds_sync();  // staging reads done before the next group's writes
    }
  };

  // Each wave walks its planes in 16-row tiles (nitems tiles in all, a
  // wave-uniform count), with the epilogue inputs of three tiles in flight
  // (loop unrolled by three, one exit test per pass, so every pass through
  // the loop head has the same loads in flight).
  const int64_t nitems =
      first_plane < a.planes ? ((a.planes - 1 - first_plane) / W + 1) * NAT : 0;
  Pos q0{first_plane, 0};
  Pos q1 = next(q0), q2 = next(q1);
  u32x4 x0[XG][2], x1[XG][2], x2[XG][2];
  // Load order: the tables (cache hits, all work-groups read the same
  // ones), the first plane's spectrum, then the epilogue inputs of the first
  // two row tiles.  Waits count loads in issue order, so staging the tables
  // waits for the tables only, and the first transposition for the spectrum
  // but not the epilogue inputs.
  {
    u32x4 zraw[2 * NKZ][NTB];
    st.load(reinterpret_cast<const _Float16*>(a.twIc), 2 * NTB * 16, NG * 64, 2 * NTB * 16, zr);
    sc.load(reinterpret_cast<const _Float16*>(a.cIc), a.Kap, NAT * 16, a.Kap, zr);
    ss.load(reinterpret_cast<const _Float16*>(a.sIc), a.Kap, NAT * 16, a.Kap, zr);
    if constexpr (EPI) sl.load(reinterpret_cast<const _Float16*>(a.lut), 0, 1, LUT_HALVES, zr);
    __builtin_amdgcn_sched_barrier(0);
    load_z(q0.p, zraw);
    __builtin_amdgcn_sched_barrier(0);
    load_x(q0, x0);
    __builtin_amdgcn_sched_barrier(0);
    load_x(q1, x1);
    __builtin_amdgcn_sched_barrier(0);
    st.store(sTI, LDI, NG * 64, 2 * NTB * 16);
    sc.store(sCI, LDK, NAT * 16, a.Kap);
    ss.store(sSI, LDK, NAT * 16, a.Kap);
    if constexpr (EPI) sl.store(sLut, 0, 1, LUT_HALVES);
    transpose_z(zraw);
  }
  __syncthreads();  // tables staged
  int64_t it = 0;
  for (; it + 3 <= nitems; it += 3) {
    load_x(q2, x2);
    process(q0, x0);
    q0 = next(q2);
    load_x(q0, x0);
    process(q1, x1);
    q1 = next(q0);
    load_x(q1, x1);
    process(q2, x2);
    q2 = next(q1);
  }
  if (it < nitems) process(q0, x0);
  if (it + 1 < nitems) process(q1, x1);
}

// ---------------------------------------------------------------------------
// Dispatch
// ---------------------------------------------------------------------------
// Dynamic LDS bytes; the lookup table (64 KiB when used) is static LDS.
size_t r2c_chain_lds_bytes(int nka, int ntb, int nta, int NaC, bool pre_lut) {
  (void)pre_lut;
  return sizeof(_Float16) * ((size_t)2 * ntb * 16 * (nka * KS + PADH) +
                             (size_t)2 * nta * 16 * (NaC + PADH));
}

size_t c2r_chain_lds_bytes(int ng, int ntb, int Kap, int Na, bool grad_lut) {
  const int nat = (Na + 15) / 16;
  (void)grad_lut;
  return sizeof(_Float16) * ((size_t)ng * 64 * (2 * ntb * 16 + PADH) +
                             (size_t)2 * nat * 16 * (Kap + PADH) +
                             (size_t)CH_NW * 16 * (64 + PADH));
}

// Kernels above 64 KiB of LDS must raise their dynamic-LDS limit first.
template <typename K>
static hipError_t allow_lds(K kern, size_t lds) {
  if (lds <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

#define R2C_CHAIN_SHAPES(X) X(2, 1, 1) X(2, 1, 2) X(2, 2, 2) X(4, 1, 1) X(4, 1, 2) X(4, 2, 2) \
  X(4, 2, 4)
#define C2R_CHAIN_SHAPES(X) X(1, 1, 1) X(1, 1, 2) X(2, 1, 1) X(2, 1, 2) X(2, 2, 1) X(2, 2, 2)

bool r2c_chain_has(int nka, int ntb, int nta) {
#define HAS(A, B, C) if (nka == A && ntb == B && nta == C) return true;
  R2C_CHAIN_SHAPES(HAS)
#undef HAS
  return false;
}

bool c2r_chain_has(int ng, int ntb, int nkz) {
#define HAS(A, B, C) if (ng == A && ntb == B && nkz == C) return true;
  C2R_CHAIN_SHAPES(HAS)
#undef HAS
  return false;
}

hipError_t launch_r2c_chain(const R2CArgs& a, int nka, int ntb, int nta, int grid, size_t lds,
                            hipStream_t s) {
#define R2C_CH(NKA_, NTB_, NTA_)                                                      \
  if (nka == NKA_ && ntb == NTB_ && nta == NTA_) {                                    \
    auto kern = a.do_tanh ? r2c_chain_kernel<NKA_, NTB_, NTA_, true>                  \
                          : r2c_chain_kernel<NKA_, NTB_, NTA_, false>;                \
    hipError_t e = allow_lds(kern, lds);                                              \
    if (e != hipSuccess) return e;                                                    \
    hipLaunchKernelGGL(kern, dim3(grid), dim3(CH_NW * 64), lds, s, a);                \
    return hipGetLastError();                                                         \
  }
  R2C_CHAIN_SHAPES(R2C_CH)
#undef R2C_CH
  return hipErrorNotSupported;
}

hipError_t launch_c2r_chain(const C2RArgs& a, int ng, int ntb, int nkz, int grid, size_t lds,
                            hipStream_t s) {
#define C2R_CH(NG_, NTB_, NKZ_)                                                       \
  if (ng == NG_ && ntb == NTB_ && nkz == NKZ_) {                                      \
    auto kern = a.epilogue ? c2r_chain_kernel<NG_, NTB_, NKZ_, true>                  \
                           : c2r_chain_kernel<NG_, NTB_, NKZ_, false>;                \
    hipError_t e = allow_lds(kern, lds);                                              \
    if (e != hipSuccess) return e;                                                    \
    hipLaunchKernelGGL(kern, dim3(grid), dim3(CH_NW * 64), lds, s, a);                \
    return hipGetLastError();                                                         \
  }
  C2R_CHAIN_SHAPES(C2R_CH)
#undef C2R_CH
  return hipErrorNotSupported;
}

}  // namespace fno
