// Device-side helpers shared by the HIP kernels of the FNO spectral
// convolution (gfx950): MFMA operand types, conversions, LDS synchronisation,
// and the staging helpers of the mode-indexed tensors.
//
// MFMA 16x16 operand layout used throughout (wave64, lane l, g = l / 16):
//   A (16 x KSTEP): lane holds A[l % 16][g*KPL .. g*KPL+KPL-1]
//   B (KSTEP x 16): lane holds B[g*KPL .. g*KPL+KPL-1][l % 16]
//   D (16 x 16)   : lane holds D[4*g + i][l % 16], i = 0..3
// The k-ordering within a step only has to agree between A and B.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_internal.h"

namespace fno {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));

template <typename T>
struct MM;

template <>
struct MM<_Float16> {
  static constexpr int KPL = 8;
  static constexpr int KSTEP = 32;
  typedef h8 frag;
  static __device__ __forceinline__ f4 mma(const frag& a, const frag& b, const f4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() {
    frag z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (_Float16)0.0f;
    return z;
  }
  static __device__ __forceinline__ frag ld(const _Float16* p) {
    return *reinterpret_cast<const frag*>(p);
  }
  static __device__ __forceinline__ frag neg(const frag& a) { return -a; }
};

// fp32: one fragment is four k-steps of v_mfma_f32_16x16x4_f32 over a
// 16-wide k-block, lane group g holding k = 4 g + s at sub-step s (A and B
// agree, so the four steps sum the whole block).  Each lane then reads its
// four k-values of a row with one 16-byte load.
template <>
struct MM<float> {
  static constexpr int KPL = 4;
  static constexpr int KSTEP = 16;
  typedef f4 frag;
  static __device__ __forceinline__ f4 mma(const frag& a, const frag& b, const f4& c) {
    f4 d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], d, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], d, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() { return f4{0.0f, 0.0f, 0.0f, 0.0f}; }
  static __device__ __forceinline__ frag ld(const float* p) {
    return *reinterpret_cast<const f4*>(p);
  }
  static __device__ __forceinline__ frag neg(const frag& a) { return -a; }
};

__device__ __forceinline__ f4 f4zero() { return f4{0.0f, 0.0f, 0.0f, 0.0f}; }

// n / d for a 32-bit n, with (m, s) from div_magic(d).
__device__ __forceinline__ uint32_t fast_div(uint32_t n, uint32_t m, uint32_t s) {
  return (uint32_t)(((uint64_t)__umulhi(n, m) + n) >> s);
}

// tanh in fp32 without branches (lanes of one wave see mixed magnitudes, and
// a branchy tanh runs both paths): for |x| < 1/16 the odd series
// x (1 - x^2/3 + 2 x^4/15) (truncation < 3e-9 relative there), otherwise
// sign(x) (1 - e) / (1 + e) with e = exp(-2|x|) (no cancellation for
// |x| >= 1/16).  Both are evaluated and one is selected.  Rounds to the
// correctly rounded fp16 value for every fp16 input; +-inf -> +-1, NaN -> NaN.
__device__ __forceinline__ float tanh_f32(float x) {
  const float ax = __builtin_fabsf(x);
  const float e = __builtin_amdgcn_exp2f(ax * -2.8853900817779268f);  // exp(-2|x|)
  const float big = (1.0f - e) * __builtin_amdgcn_rcpf(1.0f + e);
  const float x2 = x * x;
  const float small = x * __builtin_fmaf(x2, __builtin_fmaf(x2, 0.13333333333f, -0.33333333333f),
                                         1.0f);
  return ax < 0.0625f ? small : __builtin_copysignf(big, x);
}

// Pre-activation u = f(x) of the arithmetic (table-free) kernels and its
// derivative f'(x) for the data gradient.  act 1: tanh, f' = 1 - tanh^2;
// act 2: the hard clip to [-clip, clip], f' = 1 for |x| <= clip and 0
// beyond.  NaN stays NaN in both (the clip's comparisons are false for it).
__device__ __forceinline__ float preact_f32(float x, int act, float clip) {
  if (act == 2) return __builtin_fabsf(x) > clip ? __builtin_copysignf(clip, x) : x;
  return tanh_f32(x);
}

__device__ __forceinline__ float preact_grad_f32(float x, int act, float clip) {
  if (act == 2) {
    const float ax = __builtin_fabsf(x);
    return ax <= clip ? 1.0f : (ax > clip ? 0.0f : x);
  }
  const float t = tanh_f32(x);
  return 1.0f - t * t;
}

// The statistics-based clip (act 3) with its plane's bounds [lo, hi],
// compared in double; NaN bounds (a plane with a non-finite value) give NaN.
__device__ __forceinline__ float preact_sigma_f32(float x, double lo, double hi) {
  const double xd = (double)x;
  if (lo != lo) return __builtin_nanf("");
  return xd < lo ? (float)lo : (xd > hi ? (float)hi : x);
}

__device__ __forceinline__ float preact_sigma_grad_f32(float x, double lo, double hi) {
  const double xd = (double)x;
  if (lo != lo || x != x) return __builtin_nanf("");
  return (xd >= lo && xd <= hi) ? 1.0f : 0.0f;
}

// Round-to-nearest-even conversions to the storage type.
__device__ __forceinline__ _Float16 to_h(float v) { return (_Float16)v; }

template <typename T>
__device__ __forceinline__ T from_f(float v);
template <>
__device__ __forceinline__ _Float16 from_f<_Float16>(float v) { return (_Float16)v; }
template <>
__device__ __forceinline__ float from_f<float>(float v) { return v; }

// One complex value written as a single 4-byte (fp16) or 8-byte (fp32) store.
template <typename T>
__device__ __forceinline__ void store_pair(T* d, float re, float im);
template <>
__device__ __forceinline__ void store_pair<_Float16>(_Float16* d, float re, float im) {
  *reinterpret_cast<h2*>(d) = h2{to_h(re), to_h(im)};
}
template <>
__device__ __forceinline__ void store_pair<float>(float* d, float re, float im) {
  *reinterpret_cast<f2*>(d) = f2{re, im};
}

// Work-groups are dispatched round-robin over the 8 XCDs (each with its own
// L2): physical block b runs on XCD b % 8.  Returns a logical block id such
// that consecutive logical ids sit on the same XCD and are dispatched one
// after the other, so neighbouring tiles that share cache lines share an L2.
__device__ __forceinline__ int xcd_logical_block(int b, int nblocks) {
  constexpr int NX = 8;
  const int full = nblocks - nblocks % NX;
  if (b >= full) return b;
  return (b % NX) * (full / NX) + b / NX;
}

// Make LDS writes of one lane visible to the other lanes of its wavefront.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// Input fragment of step A: KPL consecutive row elements, optional
// pre-activation (act as for preact_f32, 0: none).
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ typename MM<T>::frag load_row_frag(const T* row, int n0, int Nb,
                                                              bool vrow, int act,
                                                              float clip, int vec,
                                                              double lo, double hi);

template <>
__device__ __forceinline__ h8 load_row_frag<_Float16>(const _Float16* row, int n0, int Nb,
                                                      bool vrow, int act, float clip,
                                                      int vec, double lo, double hi) {
  h8 v = MM<_Float16>::zero();
  if (vrow) {
    if (vec) {
      if (n0 < Nb) v = *reinterpret_cast<const h8*>(row + n0);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (n0 + i < Nb) v[i] = row[n0 + i];
    }
    if (act == 3) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = to_h(preact_sigma_f32((float)v[i], lo, hi));
    } else if (act) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = to_h(preact_f32((float)v[i], act, clip));
    }
  }
  return v;
}

template <>
__device__ __forceinline__ f4 load_row_frag<float>(const float* row, int n0, int Nb,
                                                   bool vrow, int act, float clip, int vec,
                                                   double lo, double hi) {
  f4 v = f4{0.0f, 0.0f, 0.0f, 0.0f};
  if (vrow) {
    if (vec) {
      if (n0 < Nb) v = *reinterpret_cast<const f4*>(row + n0);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (n0 + i < Nb) v[i] = row[n0 + i];
    }
    if (act == 3) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = preact_sigma_f32(v[i], lo, hi);
    } else if (act) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = preact_f32(v[i], act, clip);
    }
  }
  return v;
}

// ---------------------------------------------------------------------------
// Shared pieces of the per-mode contraction and the weight gradient.
//
// Spectra and weights keep the mode index t innermost, so a 16-byte load
// holds CPL consecutive modes of one (row, channel) pair.  The MFMA reduction
// runs over a channel (or batch) index, so tiles are staged in LDS with that
// index innermost: each thread loads 4 rows x CPL modes and writes, per mode,
// the real and the imaginary parts of the 4 rows as one 8- or 16-byte LDS
// store (a 4 x CPL transpose done with register moves only).
// ---------------------------------------------------------------------------
constexpr int CT_TM = 8;   // modes per tile
constexpr int CT_PB = 32;  // output channels per tile
constexpr int CT_BB = 32;  // batch rows per tile

__device__ __forceinline__ float cmult(int t, int Kb, int Nb) {
  const int tb = t % Kb;
  return (tb == 0 || 2 * tb == Nb) ? 1.0f : 2.0f;
}

typedef unsigned int u32;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef u32 u32x2 __attribute__((ext_vector_type(2)));

template <typename T>
struct CplxIO {
  static constexpr int CPL = 16 / (2 * (int)sizeof(T));  // complex values per 16 bytes
};

// 16 bytes of one row starting at mode t (CPL complex values); modes past K
// (or a row outside the tile) read as zero.  VEC: K is a multiple of CPL, so a
// full 16-byte load stays inside the row; the load is then issued
// unconditionally, out-of-range lanes reading from `zeros` (a zero block), so
// the loaded value needs no fix-up and the wait can sit at its first use.
template <typename T, bool VEC>
__device__ __forceinline__ u32x4 load_modes16(const T* zeros, const T* row, int t, int K,
                                              bool valid) {
  constexpr int CPL = CplxIO<T>::CPL;
  if constexpr (VEC) {
    const bool ok = valid && t < K;
    const T* p = ok ? row + 2 * t : zeros;
    return *reinterpret_cast<const u32x4*>(p);
  } else {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (!valid) return v;
    const u32* r = reinterpret_cast<const u32*>(row);
    constexpr int WPC = 2 * sizeof(T) / 4;  // 32-bit words per complex value
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      if (t + c < K)
#pragma unroll
        for (int w = 0; w < WPC; ++w) v[c * WPC + w] = r[(size_t)(t + c) * WPC + w];
    return v;
  }
}

// From four 16-byte loads (rows r..r+3, modes m0..m0+CPL-1) write, for every
// mode m, re(rows r..r+3) to dre + m*mstride and im(...) to dim + m*mstride.
// neg_im flips the sign of the imaginary parts (conjugation).
template <typename T>
__device__ __forceinline__ void scatter4(const u32x4 (&L)[4], T* dre, T* dim, int mstride,
                                         bool neg_im);

template <>
__device__ __forceinline__ void scatter4<_Float16>(const u32x4 (&L)[4], _Float16* dre,
                                                   _Float16* dim, int mstride, bool neg_im) {
  const u32 sign = neg_im ? 0x80008000u : 0u;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    // dword = (re lo | im hi) of one complex; gather the low / high halves
    u32x2 re, im;
    re[0] = __builtin_amdgcn_perm(L[1][m], L[0][m], 0x05040100u);
    re[1] = __builtin_amdgcn_perm(L[3][m], L[2][m], 0x05040100u);
    im[0] = __builtin_amdgcn_perm(L[1][m], L[0][m], 0x07060302u) ^ sign;
    im[1] = __builtin_amdgcn_perm(L[3][m], L[2][m], 0x07060302u) ^ sign;
    *reinterpret_cast<u32x2*>(dre + m * mstride) = re;
    *reinterpret_cast<u32x2*>(dim + m * mstride) = im;
  }
}

template <>
__device__ __forceinline__ void scatter4<float>(const u32x4 (&L)[4], float* dre, float* dim,
                                                int mstride, bool neg_im) {
  const u32 sign = neg_im ? 0x80000000u : 0u;
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    u32x4 re, im;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      re[j] = L[j][2 * m];
      im[j] = L[j][2 * m + 1] ^ sign;
    }
    *reinterpret_cast<u32x4*>(dre + m * mstride) = re;
    *reinterpret_cast<u32x4*>(dim + m * mstride) = im;
  }
}

// Asynchronous-friendly block barrier for LDS only: waits for this wave's
// LDS operations, not for outstanding global loads (prefetches stay in flight).
__device__ __forceinline__ void block_sync_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}



// ---------------------------------------------------------------------------
// Wide-plane transform helpers (fp16 planes, persistent work-groups)
// ---------------------------------------------------------------------------
typedef unsigned short us2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h8 w_as_h8(const u32x4& v) {
  h8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// f(|x|) of the two fp16 values packed in w, from the LDS table tab:
// tab[0..sat] holds f of the non-negative codes (every code from sat up to
// +inf has the value tab[sat]) and tab[sat + 1] is NaN.  ODD: f odd, the
// sign of x is restored.
template <bool ODD>
__device__ __forceinline__ uint32_t lut2(const _Float16* tab, uint32_t w, us2 sat) {
  const uint32_t aw = w & 0x7fff7fffu;
  us2 ax;
  __builtin_memcpy(&ax, &aw, 4);
  // 1 for the NaN codes (above 0x7c00): bit 15 of ax + 0x3ff (no overflow,
  // ax <= 0x7fff); all on packed 16-bit operations
  const us2 nan = (ax + (us2){0x3ff, 0x3ff}) >> (us2){15, 15};
  const us2 off = (__builtin_elementwise_min(ax, sat) + nan) << (us2){1, 1};  // byte offsets
  uint32_t o;
  __builtin_memcpy(&o, &off, 4);
  const unsigned char* base = reinterpret_cast<const unsigned char*>(tab);
  const uint32_t r0 = *reinterpret_cast<const uint16_t*>(base + (o & 0xffffu));
  const uint32_t r1 = *reinterpret_cast<const uint16_t*>(base + (o >> 16));
  const uint32_t u = r0 | (r1 << 16);
  return ODD ? (u | (w & 0x80008000u)) : u;
}

// A second table layout for kernels whose dynamic LDS starts with the table
// (LDS byte address 0, no static LDS in the kernel): f of the codes 0..sat
// followed by LUTN_NANS NaN entries.  With o = 2 |code| (the sign shifted out
// of each 16-bit half) the byte address of a code's entry is
//   min(o, 2 sat) + max(o - 0xf800, 0),
// whose second term is 0 for every finite code and for inf (o <= 0xf800)
// and 2..0x7fe for the NaN codes, which land in the NaN entries: three
// packed 16-bit operations and two zero-extending adds form both addresses
// of a word, with no base to add.  Entry sat + 1 is NaN as in the first
// layout, so lut2 reads this layout too.
constexpr int LUTN_NANS = 1023;

// f(|x|) with the sign of x restored (odd f) for the four words of v
// through such a table, in one asm block: the eight addresses, the eight LDS
// reads in flight together, one wait, then the halves joined and the signs
// put back.  The block waits for every LDS read of the wave (lgkmcnt(0)), so
// the compiler's own outstanding LDS reads are complete after it too.
// s2 holds 2 sat in both halves.
__device__ __forceinline__ void lutn_odd4(u32x4& v, uint32_t s2) {
  uint32_t w0 = v[0], w1 = v[1], w2 = v[2], w3 = v[3];
  uint32_t a0, a1, a2, a3, t0, t1, t2, t3, r0, r1, r2, r3;
#define FNO_LUTN_ADDR(W, A, T, R)                                                        \
  "v_pk_lshlrev_b16 " R ", 1, " W " op_sel_hi:[0,1]\n\t"                                \
  "v_pk_sub_u16 " A ", " R ", %[cn] clamp\n\t"                                          \
  "v_pk_min_u16 " R ", " R ", %[s2]\n\t"                                                \
  "v_add_u32_sdwa " T ", " R ", " A                                                     \
  " dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:WORD_1\n\t"            \
  "v_add_u32_sdwa " A ", " R ", " A                                                     \
  " dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_0\n\t"
#define FNO_LUTN_READ(A, T) "ds_read_u16 " A ", " A "\n\tds_read_u16 " T ", " T "\n\t"
#define FNO_LUTN_JOIN(W, A, T) \
  "v_lshl_or_b32 " T ", " T ", 16, " A "\n\tv_and_or_b32 " W ", " W ", %[sm], " T "\n\t"
  asm volatile(
      FNO_LUTN_ADDR("%[w0]", "%[a0]", "%[t0]", "%[r0]")
      FNO_LUTN_ADDR("%[w1]", "%[a1]", "%[t1]", "%[r1]")
      FNO_LUTN_ADDR("%[w2]", "%[a2]", "%[t2]", "%[r2]")
      FNO_LUTN_ADDR("%[w3]", "%[a3]", "%[t3]", "%[r3]")
      FNO_LUTN_READ("%[a0]", "%[t0]") FNO_LUTN_READ("%[a1]", "%[t1]")
      FNO_LUTN_READ("%[a2]", "%[t2]") FNO_LUTN_READ("%[a3]", "%[t3]")
      "s_waitcnt lgkmcnt(0)\n\t"
      FNO_LUTN_JOIN("%[w0]", "%[a0]", "%[t0]") FNO_LUTN_JOIN("%[w1]", "%[a1]", "%[t1]")
      FNO_LUTN_JOIN("%[w2]", "%[a2]", "%[t2]") FNO_LUTN_JOIN("%[w3]", "%[a3]", "%[t3]")
      : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3),
        [a0] "=&v"(a0), [a1] "=&v"(a1), [a2] "=&v"(a2), [a3] "=&v"(a3),
        [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3),
        [r0] "=&v"(r0), [r1] "=&v"(r1), [r2] "=&v"(r2), [r3] "=&v"(r3)
      : [cn] "s"(0xf800f800u), [s2] "s"(s2), [sm] "s"(0x80008000u));
#undef FNO_LUTN_ADDR
#undef FNO_LUTN_READ
#undef FNO_LUTN_JOIN
  v[0] = w0;
  v[1] = w1;
  v[2] = w2;
  v[3] = w3;
}

// LDS bytes of such a table (codes 0..sat, the NaN entries), rounded up to
// 256 so that the regions after it stay aligned.
__host__ __device__ __forceinline__ int lutn_bytes(int sat) {
  return ((sat + 1 + LUTN_NANS) * 2 + 255) & ~255;
}

// Stage tab[0..sat] of a global table and the NaN entries (NT threads).
template <int NT>
__device__ __forceinline__ void stage_lutn(_Float16* dst, const void* src, int sat) {
  const _Float16* s = reinterpret_cast<const _Float16*>(src);
  for (int i = threadIdx.x; i <= sat; i += NT) dst[i] = s[i];
  const uint16_t qnan = 0x7e00;
  for (int i = threadIdx.x; i < LUTN_NANS; i += NT) __builtin_memcpy(&dst[sat + 1 + i], &qnan, 2);
}

// Stage tab[0..sat] of a global table and the NaN entry (NT threads).
template <int NT>
__device__ __forceinline__ void stage_lut(_Float16* dst, const void* src, int sat) {
  const _Float16* s = reinterpret_cast<const _Float16*>(src);
  for (int i = threadIdx.x; i <= sat; i += NT) dst[i] = s[i];
  if (threadIdx.x == 0) {
    const uint16_t qnan = 0x7e00;
    __builtin_memcpy(&dst[sat + 1], &qnan, 2);
  }
}

// Buffer resource of plane p of a tensor of planes of plane_bytes each:
// accesses past the plane read zero and write nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc(const void* base, int64_t p,
                                                             int64_t plane_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(reinterpret_cast<const char*>(base) + p * plane_bytes), (short)0,
      (int)plane_bytes, 0x00020000);
}

}  // namespace fno
