// HIP kernels (gfx950 / CDNA4) of the FNO spectral-convolution layer.
//
// Every transform step is a small dense contraction with a table of unit
// twiddles, so it runs on the matrix cores: v_mfma_f32_16x16x32_f16 for fp16
// storage (fp32 accumulation) and v_mfma_f32_16x16x4_f32 for fp32 storage.
// Only retained modes are computed (output-pruned forward transform,
// input-pruned inverse), which is the truncation T_K of the Fourier
// convolution operator (Sec. 2) folded into the transform.
//
// MFMA 16x16 operand layout used throughout (wave64, lane l, g = l / 16):
//   A (16 x KSTEP): lane holds A[l % 16][g*KPL .. g*KPL+KPL-1]
//   B (KSTEP x 16): lane holds B[g*KPL .. g*KPL+KPL-1][l % 16]
//   D (16 x 16)   : lane holds D[4*g + i][l % 16], i = 0..3
// The k-ordering within a step only has to agree between A and B.
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

template <>
struct MM<float> {
  static constexpr int KPL = 1;
  static constexpr int KSTEP = 4;
  typedef float frag;
  static __device__ __forceinline__ f4 mma(const frag& a, const frag& b, const f4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() { return 0.0f; }
  static __device__ __forceinline__ frag ld(const float* p) { return *p; }
  static __device__ __forceinline__ frag neg(const frag& a) { return -a; }
};

__device__ __forceinline__ f4 f4zero() { return f4{0.0f, 0.0f, 0.0f, 0.0f}; }

// tanh(x) = 1 - 2 / (1 + e^{2x}); exact limits at +-inf, NaN propagates.
__device__ __forceinline__ float tanh_f32(float x) {
  float e = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);  // e^{2x}
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + e);
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

// Make LDS writes of one lane visible to the other lanes of its wavefront.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// Input fragment of step A: KPL consecutive row elements, optional tanh.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ typename MM<T>::frag load_row_frag(const T* row, int n0, int Nb,
                                                              bool vrow, int do_tanh,
                                                              int vec);

template <>
__device__ __forceinline__ h8 load_row_frag<_Float16>(const _Float16* row, int n0, int Nb,
                                                      bool vrow, int do_tanh, int vec) {
  h8 v = MM<_Float16>::zero();
  if (vrow) {
    if (vec) {
      if (n0 < Nb) v = *reinterpret_cast<const h8*>(row + n0);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (n0 + i < Nb) v[i] = row[n0 + i];
    }
    if (do_tanh) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = to_h(tanh_f32((float)v[i]));
    }
  }
  return v;
}

template <>
__device__ __forceinline__ float load_row_frag<float>(const float* row, int n0, int Nb,
                                                      bool vrow, int do_tanh, int vec) {
  float v = 0.0f;
  if (vrow && n0 < Nb) {
    v = row[n0];
    if (do_tanh) v = tanh_f32(v);
  }
  return v;
}

// ---------------------------------------------------------------------------
// r2c: truncated forward transform of the last two axes.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ int lds_pad() { return 16 / (int)sizeof(T); }

size_t r2c_lds_bytes(int elem, int Kbp, int R) {
  int es = elem == ELEM_F16 ? 2 : 4;
  int pad = 16 / es;
  return (size_t)2 * Kbp * (R + pad) * es;
}

template <typename T, int NCT>
__global__ __launch_bounds__(256) void r2c_plane_kernel(R2CArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int NTB = NCT / 2;  // step-B column tiles (t_b)
  constexpr int Kbp = NCT * 8;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ldA = a.R + lds_pad<T>();
  T* ATr = reinterpret_cast<T*>(smem);
  T* ATi = ATr + Kbp * ldA;
  const int64_t p = blockIdx.x;
  const T* in = reinterpret_cast<const T*>(a.in) + p * (int64_t)a.Na * a.Nb;
  const T* twA = reinterpret_cast<const T*>(a.twA);
  const T* cB = reinterpret_cast<const T*>(a.cB);
  const T* sB = reinterpret_cast<const T*>(a.sB);
  const int nta = a.Kap16 >> 4;

  f4 accR[2][NTB], accI[2][NTB];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) accR[q][tb] = accI[q][tb] = f4zero();

  for (int c0 = 0; c0 < a.Na; c0 += a.R) {
    // ---- step A: rows c0 .. c0+R-1, last axis -> 2*Kbp real columns -------
    const int nrt = a.R >> 4;
    for (int rt = wave; rt < nrt; rt += 4) {
      f4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f4zero();
      const int row = c0 + rt * 16 + r16;
      const bool vrow = row < a.Na;
      const T* rp = in + (int64_t)(vrow ? row : 0) * a.Nb;
      for (int k0 = 0; k0 < a.Nbp; k0 += KS) {
        frag af = load_row_frag<T>(rp, k0 + g * KPL, a.Nb, vrow, a.do_tanh, a.vec);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          frag bf = M::ld(twA + (int64_t)(ct * 16 + r16) * a.Nbp + k0 + g * KPL);
          acc[ct] = M::mma(af, bf, acc[ct]);
        }
      }
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int col = ct * 16 + r16;
        T* dst = (col < Kbp ? ATr + col * ldA : ATi + (col - Kbp) * ldA) + rt * 16 + 4 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[i] = from_f<T>(acc[ct][i] * a.scaleA);
      }
    }
    __syncthreads();
    // ---- step B: accumulate the other axis over this chunk ----------------
    for (int k0 = 0; k0 < a.R; k0 += KS) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int ta = wave + 4 * q;
        if (ta < nta) {
          const int64_t toff = (int64_t)(ta * 16 + r16) * a.Nap + c0 + k0 + g * KPL;
          frag cf = M::ld(cB + toff);
          frag sf = M::ld(sB + toff);
          frag nsf = M::neg(sf);
#pragma unroll
          for (int tb = 0; tb < NTB; ++tb) {
            frag ar = M::ld(ATr + (tb * 16 + r16) * ldA + k0 + g * KPL);
            frag ai = M::ld(ATi + (tb * 16 + r16) * ldA + k0 + g * KPL);
            accR[q][tb] = M::mma(cf, ar, accR[q][tb]);
            accR[q][tb] = M::mma(sf, ai, accR[q][tb]);
            accI[q][tb] = M::mma(cf, ai, accI[q][tb]);
            accI[q][tb] = M::mma(nsf, ar, accI[q][tb]);
          }
        }
      }
    }
    __syncthreads();
  }
  // ---- store the retained spectrum -----------------------------------------
  T* out = reinterpret_cast<T*>(a.out) + p * (int64_t)a.Ka * a.Kb * 2;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int ta = wave + 4 * q;
    if (ta < nta) {
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        const int t_b = tb * 16 + r16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t_a = ta * 16 + 4 * g + i;
          if (t_a < a.Ka && t_b < a.Kb) {
            store_pair<T>(out + ((int64_t)t_a * a.Kb + t_b) * 2, accR[q][tb][i] * a.scaleB,
                          accI[q][tb][i] * a.scaleB);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// c2r: input-pruned inverse of the last two axes.
// ---------------------------------------------------------------------------
size_t c2r_lds_bytes(int elem, int Kbp, int Kap, int R) {
  int es = elem == ELEM_F16 ? 2 : 4;
  int pad = 16 / es;
  size_t zt = (size_t)2 * Kbp * (Kap + pad) * es;
  size_t vl = (size_t)R * (2 * Kbp + pad) * es;
  size_t ob = (size_t)4 * 16 * 68 * 4;
  return zt + vl + ob;
}

template <typename T>
__device__ __forceinline__ void load16(const T* src, float* v, int n, bool vec);

template <>
__device__ __forceinline__ void load16<_Float16>(const _Float16* src, float* v, int n,
                                                 bool vec) {
  if (vec && n >= 16) {
    h8 a0 = *reinterpret_cast<const h8*>(src);
    h8 a1 = *reinterpret_cast<const h8*>(src + 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[i] = (float)a0[i];
      v[8 + i] = (float)a1[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n ? (float)src[i] : 0.0f;
  }
}

template <>
__device__ __forceinline__ void load16<float>(const float* src, float* v, int n, bool vec) {
  if (vec && n >= 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f4 t = *reinterpret_cast<const f4*>(src + 4 * i);
      v[4 * i + 0] = t[0];
      v[4 * i + 1] = t[1];
      v[4 * i + 2] = t[2];
      v[4 * i + 3] = t[3];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n ? src[i] : 0.0f;
  }
}

template <typename T>
__device__ __forceinline__ void store16(T* dst, const float* v, int n, bool vec);

template <>
__device__ __forceinline__ void store16<_Float16>(_Float16* dst, const float* v, int n,
                                                  bool vec) {
  if (vec && n >= 16) {
    h8 a0, a1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a0[i] = to_h(v[i]);
      a1[i] = to_h(v[8 + i]);
    }
    *reinterpret_cast<h8*>(dst) = a0;
    *reinterpret_cast<h8*>(dst + 8) = a1;
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < n) dst[i] = to_h(v[i]);
  }
}

template <>
__device__ __forceinline__ void store16<float>(float* dst, const float* v, int n, bool vec) {
  if (vec && n >= 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<f4*>(dst + 4 * i) = f4{v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < n) dst[i] = v[i];
  }
}

template <typename T, int NCT>
__global__ __launch_bounds__(256) void c2r_plane_kernel(C2RArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int NTB = NCT / 2;
  constexpr int Kbp = NCT * 8;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int pad = lds_pad<T>();
  const int ldZ = a.Kap + pad;
  const int ldV = 2 * Kbp + pad;
  T* ZTr = reinterpret_cast<T*>(smem);
  T* ZTi = ZTr + Kbp * ldZ;
  T* VL = ZTi + Kbp * ldZ;
  float* obuf = reinterpret_cast<float*>(VL + a.R * ldV) + wave * (16 * 68);
  const int64_t p = blockIdx.x;
  const T* zin = reinterpret_cast<const T*>(a.in) + p * (int64_t)a.Ka * a.Kb * 2;
  const T* cI = reinterpret_cast<const T*>(a.cI);
  const T* sI = reinterpret_cast<const T*>(a.sI);
  const T* twI = reinterpret_cast<const T*>(a.twI);
  T* yout = reinterpret_cast<T*>(a.out) + p * (int64_t)a.Na * a.Nb;
  const T* xin = a.x ? reinterpret_cast<const T*>(a.x) + p * (int64_t)a.Na * a.Nb : nullptr;

  // ---- stage the spectrum transposed: ZT[t_b][t_a] ------------------------
  for (int idx = threadIdx.x; idx < a.Kap * Kbp; idx += 256) {
    const int t_a = idx / Kbp, t_b = idx - t_a * Kbp;
    T re = from_f<T>(0.0f), im = from_f<T>(0.0f);
    if (t_a < a.Ka && t_b < a.Kb) {
      const T* z = zin + ((int64_t)t_a * a.Kb + t_b) * 2;
      re = z[0];
      im = z[1];
    }
    ZTr[t_b * ldZ + t_a] = re;
    ZTi[t_b * ldZ + t_a] = im;
  }
  __syncthreads();

  const int nnt = a.R >> 4;
  const int ncg = (a.Nb + 63) >> 6;
  for (int c0 = 0; c0 < a.Na; c0 += a.R) {
    // ---- step B': V^T[t_b][n] = sum_t Z^T[t_b][t] E[t][n] ------------------
    for (int nt = wave; nt < nnt; nt += 4) {
      f4 vr[NTB], vi[NTB];
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) vr[tb] = vi[tb] = f4zero();
      const int64_t roff = (int64_t)(c0 + nt * 16 + r16) * a.Kap;
      for (int k0 = 0; k0 < a.Kap; k0 += KS) {
        frag cf = M::ld(cI + roff + k0 + g * KPL);
        frag sf = M::ld(sI + roff + k0 + g * KPL);
        frag nsf = M::neg(sf);
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          frag zr = M::ld(ZTr + (tb * 16 + r16) * ldZ + k0 + g * KPL);
          frag zi = M::ld(ZTi + (tb * 16 + r16) * ldZ + k0 + g * KPL);
          vr[tb] = M::mma(zr, cf, vr[tb]);
          vr[tb] = M::mma(zi, nsf, vr[tb]);
          vi[tb] = M::mma(zr, sf, vi[tb]);
          vi[tb] = M::mma(zi, cf, vi[tb]);
        }
      }
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        T* dst = VL + (nt * 16 + r16) * ldV + tb * 16 + 4 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dst[i] = from_f<T>(vr[tb][i]);
          dst[Kbp + i] = from_f<T>(vi[tb][i]);
        }
      }
    }
    __syncthreads();
    // ---- step A': y[n][m] = sum_k VL[n][k] twI[m][k] ------------------------
    for (int rt = wave; rt < nnt; rt += 4) {
      const int row0 = c0 + rt * 16;
      for (int cg = 0; cg < ncg; ++cg) {
        f4 acc[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = f4zero();
        // D = y^T tile: row n_b (4 consecutive per lane), column n_a
        for (int k0 = 0; k0 < 2 * Kbp; k0 += KS) {
          frag vf = M::ld(VL + (rt * 16 + r16) * ldV + k0 + g * KPL);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int ct = cg * 4 + c;
            frag tf = M::ld(twI + (int64_t)(ct * 16 + r16) * (2 * Kbp) + k0 + g * KPL);
            acc[c] = M::mma(tf, vf, acc[c]);
          }
        }
        // one 16-byte store per tile: obuf[n_a][n_b .. n_b + 3]
#pragma unroll
        for (int c = 0; c < 4; ++c)
          *reinterpret_cast<f4*>(obuf + r16 * 68 + c * 16 + 4 * g) = acc[c];
        wave_lds_sync();
        const int orow = lane >> 2;
        const int ocol = (lane & 3) * 16;
        const int n_a = row0 + orow;
        const int n_b = cg * 64 + ocol;
        float v[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f4 t = *reinterpret_cast<const f4*>(obuf + orow * 68 + ocol + 4 * i);
          v[4 * i] = t[0] * a.scale;
          v[4 * i + 1] = t[1] * a.scale;
          v[4 * i + 2] = t[2] * a.scale;
          v[4 * i + 3] = t[3] * a.scale;
        }
        wave_lds_sync();
        if (n_a < a.Na && n_b < a.Nb) {
          const int nval = min(16, a.Nb - n_b);
          const int64_t off = (int64_t)n_a * a.Nb + n_b;
          if (a.epilogue) {
            float xv[16];
            load16<T>(xin + off, xv, nval, a.vec);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              const float t = tanh_f32(xv[i]);
              v[i] *= (1.0f - t * t);
            }
          }
          store16<T>(yout + off, v, nval, a.vec);
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Complex DFT along a middle axis (3-D leading axis).
// ---------------------------------------------------------------------------
size_t axis_lds_bytes(int elem, int Linp) {
  int es = elem == ELEM_F16 ? 2 : 4;
  int pad = 16 / es;
  return (size_t)2 * 64 * (Linp + pad) * es;
}

template <typename T>
__global__ __launch_bounds__(256) void axis_kernel(AxisArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ld = a.Linp + lds_pad<T>();
  T* Ir = reinterpret_cast<T*>(smem);
  T* Ii = Ir + 64 * ld;
  const int j0 = blockIdx.x * 64;
  const int64_t o = blockIdx.y;
  const T* in = reinterpret_cast<const T*>(a.in) + o * (int64_t)a.Lin * a.inner * 2;
  T* out = reinterpret_cast<T*>(a.out) + o * (int64_t)a.Lout * a.inner * 2;
  const T* er = reinterpret_cast<const T*>(a.er);
  const T* ei = reinterpret_cast<const T*>(a.ei);

  for (int idx = threadIdx.x; idx < a.Linp * 64; idx += 256) {
    const int l = idx >> 6, jj = idx & 63;
    T re = from_f<T>(0.0f), im = from_f<T>(0.0f);
    if (l < a.Lin && j0 + jj < a.inner) {
      const T* s = in + ((int64_t)l * a.inner + j0 + jj) * 2;
      re = s[0];
      im = s[1];
    }
    Ir[jj * ld + l] = re;
    Ii[jj * ld + l] = im;
  }
  __syncthreads();
  const int jt = wave;  // each wave owns 16 of the 64 columns
  const int ntt = a.Lout16 >> 4;
  for (int tg = 0; tg < ntt; tg += 4) {
    f4 accR[4], accI[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) accR[u] = accI[u] = f4zero();
    for (int k0 = 0; k0 < a.Linp; k0 += KS) {
      frag br = M::ld(Ir + (jt * 16 + r16) * ld + k0 + g * KPL);
      frag bi = M::ld(Ii + (jt * 16 + r16) * ld + k0 + g * KPL);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int tt = tg + u;
        if (tt < ntt) {
          const int64_t eoff = (int64_t)(tt * 16 + r16) * a.Linp + k0 + g * KPL;
          frag xr = M::ld(er + eoff);
          frag xi = M::ld(ei + eoff);
          frag nxi = M::neg(xi);
          accR[u] = M::mma(xr, br, accR[u]);
          accR[u] = M::mma(nxi, bi, accR[u]);
          accI[u] = M::mma(xr, bi, accI[u]);
          accI[u] = M::mma(xi, br, accI[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int tt = tg + u;
      if (tt < ntt) {
        const int j = j0 + jt * 16 + r16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = tt * 16 + 4 * g + i;
          if (t < a.Lout && j < a.inner) {
            store_pair<T>(out + ((int64_t)t * a.inner + j) * 2, accR[u][i] * a.scale,
                          accI[u][i] * a.scale);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Per-mode channel contraction (forward and adjoint).
// Work-group: 8 consecutive modes x 32 output channels x 32 batch rows.
// ---------------------------------------------------------------------------
constexpr int CT_TM = 8;
constexpr int CT_PB = 32;
constexpr int CT_BB = 32;

__device__ __forceinline__ float cmult(int t, int Kb, int Nb) {
  const int tb = t % Kb;
  return (tb == 0 || 2 * tb == Nb) ? 1.0f : 2.0f;
}

template <typename T>
__device__ __forceinline__ void load_cplx(const T* src, int n, bool vec, float* re, float* im);

// Loads n (<= 4) consecutive complex values.
template <>
__device__ __forceinline__ void load_cplx<_Float16>(const _Float16* src, int n, bool vec,
                                                    float* re, float* im) {
  if (vec && n == 4) {
    h8 v = *reinterpret_cast<const h8*>(src);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      re[i] = (float)v[2 * i];
      im[i] = (float)v[2 * i + 1];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      re[i] = i < n ? (float)src[2 * i] : 0.0f;
      im[i] = i < n ? (float)src[2 * i + 1] : 0.0f;
    }
  }
}

template <>
__device__ __forceinline__ void load_cplx<float>(const float* src, int n, bool vec, float* re,
                                                 float* im) {
  if (vec && n == 4) {
    f4 v0 = *reinterpret_cast<const f4*>(src);
    f4 v1 = *reinterpret_cast<const f4*>(src + 4);
    re[0] = v0[0]; im[0] = v0[1]; re[1] = v0[2]; im[1] = v0[3];
    re[2] = v1[0]; im[2] = v1[1]; re[3] = v1[2]; im[3] = v1[3];
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      re[i] = i < n ? src[2 * i] : 0.0f;
      im[i] = i < n ? src[2 * i + 1] : 0.0f;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void contract_kernel(ContractArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int QC = (sizeof(T) == 2) ? 32 : 16;  // q per staged chunk
  constexpr int LDQ = QC + 16 / (int)sizeof(T);
  constexpr size_t STAGE = sizeof(T) * 2 * CT_TM * (CT_BB + CT_PB) * LDQ;
  constexpr size_t OUTB = sizeof(T) * 2 * CT_BB * CT_PB * CT_TM;
  __shared__ __align__(16) unsigned char smem[STAGE > OUTB ? STAGE : OUTB];
  T(*sIn)[CT_TM][CT_BB][LDQ] = reinterpret_cast<T(*)[CT_TM][CT_BB][LDQ]>(smem);
  T(*sW)[CT_TM][CT_PB][LDQ] =
      reinterpret_cast<T(*)[CT_TM][CT_PB][LDQ]>(smem + sizeof(T) * 2 * CT_TM * CT_BB * LDQ);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int t0 = blockIdx.x * CT_TM;
  const int p0 = blockIdx.y * CT_PB;
  const int b0 = blockIdx.z * CT_BB;
  const T* in = reinterpret_cast<const T*>(a.in);
  const T* w = reinterpret_cast<const T*>(a.w);
  const bool vec = (a.K % 4) == 0;
  // wave -> (b tile, p tile)
  const int bt = wave >> 1, pt = wave & 1;
  f4 accR[CT_TM], accI[CT_TM];
#pragma unroll
  for (int m = 0; m < CT_TM; ++m) accR[m] = accI[m] = f4zero();

  for (int q0 = 0; q0 < a.Q; q0 += QC) {
    // stage in[b][q][t0..t0+8) -> sIn[.][t][b][q]
    for (int idx = threadIdx.x; idx < CT_BB * QC * 2; idx += 256) {
      const int half = idx & 1, rest = idx >> 1;
      const int qq = rest % QC, bb = rest / QC;
      const int b = b0 + bb, q = q0 + qq;
      const int tt = t0 + half * 4;
      float re[4], im[4];
      const int n = (b < a.B && q < a.Q) ? max(0, min(4, a.K - tt)) : 0;
      load_cplx<T>(in + (((int64_t)b * a.Q + q) * a.K + tt) * 2, n, vec, re, im);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sIn[0][half * 4 + i][bb][qq] = from_f<T>(re[i]);
        sIn[1][half * 4 + i][bb][qq] = from_f<T>(im[i]);
      }
    }
    // stage Wop(q, p, t) -> sW[.][t][p][q]
    for (int idx = threadIdx.x; idx < CT_PB * QC * 2; idx += 256) {
      const int half = idx & 1, rest = idx >> 1;
      int qq, pp;
      if (a.adjoint) {  // W[p][q][t]: q fastest
        qq = rest % QC;
        pp = rest / QC;
      } else {          // W[q][p][t]: p fastest
        pp = rest % CT_PB;
        qq = rest / CT_PB;
      }
      const int q = q0 + qq, pc = p0 + pp;
      const int tt = t0 + half * 4;
      float re[4], im[4];
      const int n = (q < a.Q && pc < a.P) ? max(0, min(4, a.K - tt)) : 0;
      const int64_t row = a.adjoint ? ((int64_t)pc * a.wcols + q) : ((int64_t)q * a.wcols + pc);
      load_cplx<T>(w + (row * a.K + tt) * 2, n, vec, re, im);
      const float sgn = a.adjoint ? -1.0f : 1.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sW[0][half * 4 + i][pp][qq] = from_f<T>(re[i]);
        sW[1][half * 4 + i][pp][qq] = from_f<T>(sgn * im[i]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < CT_TM; ++m) {
#pragma unroll
      for (int k0 = 0; k0 < QC; k0 += KS) {
        frag ar = M::ld(&sIn[0][m][bt * 16 + r16][k0 + g * KPL]);
        frag ai = M::ld(&sIn[1][m][bt * 16 + r16][k0 + g * KPL]);
        frag br = M::ld(&sW[0][m][pt * 16 + r16][k0 + g * KPL]);
        frag bi = M::ld(&sW[1][m][pt * 16 + r16][k0 + g * KPL]);
        frag nai = M::neg(ai);
        accR[m] = M::mma(ar, br, accR[m]);
        accR[m] = M::mma(nai, bi, accR[m]);
        accI[m] = M::mma(ar, bi, accI[m]);
        accI[m] = M::mma(ai, br, accI[m]);
      }
    }
    __syncthreads();
  }
  // epilogue: stage [b][p][t] complex in LDS (reuse sIn), then 8-mode rows
  T* so = reinterpret_cast<T*>(smem);  // [b][p][t] complex
#pragma unroll
  for (int m = 0; m < CT_TM; ++m) {
    const int t = t0 + m;
    const float s = (t < a.K) ? a.scale * cmult(t, a.Kb, a.Nb) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int bb = bt * 16 + 4 * g + i, pp = pt * 16 + r16;
      store_pair<T>(so + ((bb * CT_PB + pp) * CT_TM + m) * 2, accR[m][i] * s, accI[m][i] * s);
    }
  }
  __syncthreads();
  T* out = reinterpret_cast<T*>(a.out);
  for (int idx = threadIdx.x; idx < CT_BB * CT_PB; idx += 256) {
    const int bb = idx / CT_PB, pp = idx % CT_PB;
    const int b = b0 + bb, pc = p0 + pp;
    if (b < a.B && pc < a.P) {
      T* d = out + (((int64_t)b * a.P + pc) * a.K + t0) * 2;
      const T* s = so + (bb * CT_PB + pp) * CT_TM * 2;
      const int n = min(CT_TM, a.K - t0);
      if (n == CT_TM && vec) {
        if (sizeof(T) == 2) {
          *reinterpret_cast<h8*>(d) = *reinterpret_cast<const h8*>(s);
          *reinterpret_cast<h8*>(d + 8) = *reinterpret_cast<const h8*>(s + 8);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            reinterpret_cast<f4*>(d)[i] = reinterpret_cast<const f4*>(s)[i];
        }
      } else {
        for (int i = 0; i < 2 * n; ++i) d[i] = s[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Weight gradient: gw[q][p][t] = scale c(t) sum_b conj(xh[b][q][t]) gh[b][p][t]
// Work-group: 8 modes x 32 (q) x 32 (p); fixed-order reduction over b.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int BC = (sizeof(T) == 2) ? 32 : 16;  // batch rows per chunk
  constexpr int LDB = BC + 16 / (int)sizeof(T);
  constexpr int TM = 8, QB = 32, PB = 32;
  constexpr size_t STAGE = sizeof(T) * 2 * TM * (QB + PB) * LDB;
  constexpr size_t OUTB = sizeof(float) * 2 * QB * PB * TM;
  __shared__ __align__(16) unsigned char smem[STAGE > OUTB ? STAGE : OUTB];
  T(*sX)[TM][QB][LDB] = reinterpret_cast<T(*)[TM][QB][LDB]>(smem);
  T(*sG)[TM][PB][LDB] = reinterpret_cast<T(*)[TM][PB][LDB]>(smem + sizeof(T) * 2 * TM * QB * LDB);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int t0 = blockIdx.x * TM;
  const int q0 = blockIdx.y * QB;
  const int p0 = blockIdx.z * PB;
  const T* xh = reinterpret_cast<const T*>(a.xh);
  const T* gh = reinterpret_cast<const T*>(a.gh);
  const bool vec = (a.K % 4) == 0;
  const int qt = wave >> 1, pt = wave & 1;
  f4 accR[TM], accI[TM];
#pragma unroll
  for (int m = 0; m < TM; ++m) accR[m] = accI[m] = f4zero();

  for (int bs = 0; bs < a.B; bs += BC) {
    for (int idx = threadIdx.x; idx < BC * QB * 2; idx += 256) {
      const int half = idx & 1, rest = idx >> 1;
      const int qq = rest % QB, bb = rest / QB;
      const int b = bs + bb, q = q0 + qq, tt = t0 + half * 4;
      float re[4], im[4];
      const int n = (b < a.B && q < a.Cin) ? max(0, min(4, a.K - tt)) : 0;
      load_cplx<T>(xh + (((int64_t)b * a.Cin + q) * a.K + tt) * 2, n, vec, re, im);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sX[0][half * 4 + i][qq][bb] = from_f<T>(re[i]);
        sX[1][half * 4 + i][qq][bb] = from_f<T>(im[i]);
      }
    }
    for (int idx = threadIdx.x; idx < BC * PB * 2; idx += 256) {
      const int half = idx & 1, rest = idx >> 1;
      const int pp = rest % PB, bb = rest / PB;
      const int b = bs + bb, pc = p0 + pp, tt = t0 + half * 4;
      float re[4], im[4];
      const int n = (b < a.B && pc < a.Cout) ? max(0, min(4, a.K - tt)) : 0;
      load_cplx<T>(gh + (((int64_t)b * a.Cout + pc) * a.K + tt) * 2, n, vec, re, im);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sG[0][half * 4 + i][pp][bb] = from_f<T>(re[i]);
        sG[1][half * 4 + i][pp][bb] = from_f<T>(im[i]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < TM; ++m) {
#pragma unroll
      for (int k0 = 0; k0 < BC; k0 += KS) {
        frag xr = M::ld(&sX[0][m][qt * 16 + r16][k0 + g * KPL]);
        frag xi = M::ld(&sX[1][m][qt * 16 + r16][k0 + g * KPL]);
        frag gr = M::ld(&sG[0][m][pt * 16 + r16][k0 + g * KPL]);
        frag gi = M::ld(&sG[1][m][pt * 16 + r16][k0 + g * KPL]);
        frag nxi = M::neg(xi);
        // conj(x) * g = (xr gr + xi gi) + i (xr gi - xi gr)
        accR[m] = M::mma(xr, gr, accR[m]);
        accR[m] = M::mma(xi, gi, accR[m]);
        accI[m] = M::mma(xr, gi, accI[m]);
        accI[m] = M::mma(nxi, gr, accI[m]);
      }
    }
    __syncthreads();
  }
  float* so = reinterpret_cast<float*>(smem);  // [QB][PB][TM] complex
#pragma unroll
  for (int m = 0; m < TM; ++m) {
    const int t = t0 + m;
    const float s = (t < a.K) ? a.scale * cmult(t, a.Kb, a.Nb) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qq = qt * 16 + 4 * g + i, pp = pt * 16 + r16;
      store_pair<float>(so + ((qq * PB + pp) * TM + m) * 2, accR[m][i] * s, accI[m][i] * s);
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < QB * PB; idx += 256) {
    const int qq = idx / PB, pp = idx % PB;
    const int q = q0 + qq, pc = p0 + pp;
    if (q < a.Cin && pc < a.Cout) {
      float* d = a.gw + (((int64_t)q * a.Cout + pc) * a.K + t0) * 2;
      const float* s = so + (qq * PB + pp) * TM * 2;
      const int n = min(TM, a.K - t0);
      if (n == TM && vec) {
#pragma unroll
        for (int i = 0; i < 4; ++i) reinterpret_cast<f4*>(d)[i] = reinterpret_cast<const f4*>(s)[i];
      } else {
        for (int i = 0; i < 2 * n; ++i) d[i] = s[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Generic pairwise complex contraction (Tucker path steps), fp32 accumulate.
// One thread per result element; strides decode the index groups.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f2 load_elem(const void* p, int elem, int64_t off) {
  if (elem == ELEM_F16) {
    h2 v = reinterpret_cast<const h2*>(p)[off];
    return f2{(float)v[0], (float)v[1]};
  }
  return reinterpret_cast<const f2*>(p)[off];
}

__global__ __launch_bounds__(256) void pair_kernel(PairArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.out_size) return;
  int64_t rem = idx;
  int64_t aoff = 0, boff = 0;
  int64_t cidx = 0;
  for (int k = a.n_out - 1; k >= 0; --k) {
    const int64_t e = a.out_ext[k];
    const int64_t v = rem % e;
    rem /= e;
    aoff += v * a.a_stride_out[k];
    boff += v * a.b_stride_out[k];
    if (k == a.scale_c_axis) cidx = v;
  }
  float sr = 0.0f, si = 0.0f;
  for (int64_t r = 0; r < a.red_size; ++r) {
    int64_t rr = r, ao = aoff, bo = boff;
    for (int k = a.n_red - 1; k >= 0; --k) {
      const int64_t e = a.red_ext[k];
      const int64_t v = rr % e;
      rr /= e;
      ao += v * a.a_stride_red[k];
      bo += v * a.b_stride_red[k];
    }
    f2 x = load_elem(a.a, a.a_elem, ao);
    f2 y = load_elem(a.b, a.b_elem, bo);
    if (a.conj_a) x[1] = -x[1];
    if (a.conj_b) y[1] = -y[1];
    sr = fmaf(x[0], y[0], sr);
    sr = fmaf(-x[1], y[1], sr);
    si = fmaf(x[0], y[1], si);
    si = fmaf(x[1], y[0], si);
  }
  float s = a.scale;
  if (a.scale_c_axis >= 0) s *= (cidx == 0 || 2 * cidx == a.Nb) ? 1.0f : 2.0f;
  if (a.out_elem == ELEM_F16) {
    reinterpret_cast<h2*>(a.out)[idx] = h2{to_h(sr * s), to_h(si * s)};
  } else {
    reinterpret_cast<f2*>(a.out)[idx] = f2{sr * s, si * s};
  }
}

__global__ void scale_kernel(float* p, int64_t n, float s) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] *= s;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
// Dynamic LDS above 64 KiB has to be opted into per kernel.
static hipError_t allow_lds(const void* kern, size_t lds) {
  if (lds <= 65536) return hipSuccess;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

#define FNO_LAUNCH(kern, grid, block, lds, s, args)                              \
  do {                                                                           \
    hipError_t e_ = allow_lds(reinterpret_cast<const void*>(&kern), lds);        \
    if (e_ != hipSuccess) return e_;                                             \
    hipLaunchKernelGGL(kern, grid, block, lds, s, args);                         \
  } while (0)
template <typename T>
static hipError_t r2c_dispatch(int nct, const R2CArgs& a, size_t lds, hipStream_t s) {
  dim3 grid((unsigned)a.planes), block(256);
  switch (nct) {
    case 2: FNO_LAUNCH((r2c_plane_kernel<T, 2>), grid, block, lds, s, a); break;
    case 4: FNO_LAUNCH((r2c_plane_kernel<T, 4>), grid, block, lds, s, a); break;
    case 8: FNO_LAUNCH((r2c_plane_kernel<T, 8>), grid, block, lds, s, a); break;
    case 16: FNO_LAUNCH((r2c_plane_kernel<T, 16>), grid, block, lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_r2c(int elem, int nct, const R2CArgs& a, size_t lds, hipStream_t s) {
  return elem == ELEM_F16 ? r2c_dispatch<_Float16>(nct, a, lds, s)
                          : r2c_dispatch<float>(nct, a, lds, s);
}

template <typename T>
static hipError_t c2r_dispatch(int nct, const C2RArgs& a, size_t lds, hipStream_t s) {
  dim3 grid((unsigned)a.planes), block(256);
  switch (nct) {
    case 2: FNO_LAUNCH((c2r_plane_kernel<T, 2>), grid, block, lds, s, a); break;
    case 4: FNO_LAUNCH((c2r_plane_kernel<T, 4>), grid, block, lds, s, a); break;
    case 8: FNO_LAUNCH((c2r_plane_kernel<T, 8>), grid, block, lds, s, a); break;
    case 16: FNO_LAUNCH((c2r_plane_kernel<T, 16>), grid, block, lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_c2r(int elem, int nct, const C2RArgs& a, size_t lds, hipStream_t s) {
  return elem == ELEM_F16 ? c2r_dispatch<_Float16>(nct, a, lds, s)
                          : c2r_dispatch<float>(nct, a, lds, s);
}

hipError_t launch_axis(int elem, const AxisArgs& a, size_t lds, hipStream_t s) {
  dim3 grid((unsigned)((a.inner + 63) / 64), (unsigned)a.outer), block(256);
  if (elem == ELEM_F16)
    FNO_LAUNCH((axis_kernel<_Float16>), grid, block, lds, s, a);
  else
    FNO_LAUNCH((axis_kernel<float>), grid, block, lds, s, a);
  return hipGetLastError();
}

hipError_t launch_contract(int elem, const ContractArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.K + CT_TM - 1) / CT_TM), (unsigned)((a.P + CT_PB - 1) / CT_PB),
            (unsigned)((a.B + CT_BB - 1) / CT_BB));
  dim3 block(256);
  if (elem == ELEM_F16)
    hipLaunchKernelGGL((contract_kernel<_Float16>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((contract_kernel<float>), grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_wgrad(int elem, const WgradArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.K + 7) / 8), (unsigned)((a.Cin + 31) / 32),
            (unsigned)((a.Cout + 31) / 32));
  dim3 block(256);
  if (elem == ELEM_F16)
    hipLaunchKernelGGL((wgrad_kernel<_Float16>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((wgrad_kernel<float>), grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pair(const PairArgs& a, hipStream_t s) {
  if (a.out_size <= 0) return hipSuccess;
  dim3 grid((unsigned)((a.out_size + 255) / 256)), block(256);
  hipLaunchKernelGGL(pair_kernel, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_scale_complex(float* p, int64_t n, float sc, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  dim3 grid((unsigned)((n + 255) / 256)), block(256);
  hipLaunchKernelGGL(scale_kernel, grid, block, 0, st, p, n, sc);
  return hipGetLastError();
}

}  // namespace fno
