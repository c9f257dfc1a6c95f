// HIP kernels (gfx950 / CDNA4) of the FNO spectral-convolution layer.
//
// Every transform step is a small dense contraction with a table of unit
// twiddles, so it runs on the matrix cores: v_mfma_f32_16x16x32_f16 for fp16
// storage (fp32 accumulation) and v_mfma_f32_16x16x4_f32 for fp32 storage.
// Only retained modes are computed (output-pruned forward transform,
// input-pruned inverse), which is the truncation T_K of the Fourier
// convolution operator (Sec. 2) folded into the transform.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

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

// row tiles per wave and pass in the generic transforms' last-axis products
constexpr int R2C_NRT = 2;
constexpr int C2R_NRT = 2;

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
  // statistics-based clip: this plane's bounds
  double slo = 0.0, shi = 0.0;
  if (a.act == ACT_SIGMA) {
    slo = a.bounds[2 * (p / a.bgroup)];
    shi = a.bounds[2 * (p / a.bgroup) + 1];
  }

  f4 accR[2][NTB], accI[2][NTB];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) accR[q][tb] = accI[q][tb] = f4zero();

  for (int c0 = 0; c0 < a.Na; c0 += a.R) {
    // ---- step A: rows c0 .. c0+R-1, last axis -> 2*Kbp real columns -------
    // A wave takes NRT row tiles (rt, rt + 4, ...) at once, so each twiddle
    // fragment it loads serves NRT products.
    const int nrt = a.R >> 4;
    for (int rt0 = wave; rt0 < nrt; rt0 += 4 * R2C_NRT) {
      f4 acc[R2C_NRT][NCT];
      const T* rp[R2C_NRT];
      bool vrow[R2C_NRT];
#pragma unroll
      for (int u = 0; u < R2C_NRT; ++u) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) acc[u][ct] = f4zero();
        const int row = c0 + (rt0 + 4 * u) * 16 + r16;
        vrow[u] = rt0 + 4 * u < nrt && row < a.Na;
        rp[u] = in + (int64_t)(vrow[u] ? row : 0) * a.Nb;
      }
      for (int k0 = 0; k0 < a.Nbp; k0 += KS) {
        frag af[R2C_NRT];
#pragma unroll
        for (int u = 0; u < R2C_NRT; ++u)
          if (rt0 + 4 * u < nrt)
            af[u] = load_row_frag<T>(rp[u], k0 + g * KPL, a.Nb, vrow[u], a.act, a.clip,
                                    a.vec, slo, shi);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          frag bf = M::ld(twA + (int64_t)(ct * 16 + r16) * a.Nbp + k0 + g * KPL);
#pragma unroll
          for (int u = 0; u < R2C_NRT; ++u)
            if (rt0 + 4 * u < nrt) acc[u][ct] = M::mma(af[u], bf, acc[u][ct]);
        }
      }
#pragma unroll
      for (int u = 0; u < R2C_NRT; ++u) {
        if (rt0 + 4 * u >= nrt) continue;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          const int col = ct * 16 + r16;
          T* dst = (col < Kbp ? ATr + col * ldA : ATi + (col - Kbp) * ldA) +
                   (rt0 + 4 * u) * 16 + 4 * g;
#pragma unroll
          for (int i = 0; i < 4; ++i) dst[i] = from_f<T>(acc[u][ct][i] * a.scaleA);
        }
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
    // A wave takes C2R_NRT row tiles (rt, rt + 4, ...) per column group, so
    // each twiddle fragment it loads serves C2R_NRT products.
    for (int rt0 = wave; rt0 < nnt; rt0 += 4 * C2R_NRT) {
      for (int cg = 0; cg < ncg; ++cg) {
        f4 acc[C2R_NRT][4];
#pragma unroll
        for (int u = 0; u < C2R_NRT; ++u)
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[u][c] = f4zero();
        // D = y^T tile: row n_b (4 consecutive per lane), column n_a
        for (int k0 = 0; k0 < 2 * Kbp; k0 += KS) {
          frag vf[C2R_NRT];
#pragma unroll
          for (int u = 0; u < C2R_NRT; ++u)
            if (rt0 + 4 * u < nnt)
              vf[u] = M::ld(VL + ((rt0 + 4 * u) * 16 + r16) * ldV + k0 + g * KPL);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int ct = cg * 4 + c;
            frag tf = M::ld(twI + (int64_t)(ct * 16 + r16) * (2 * Kbp) + k0 + g * KPL);
#pragma unroll
            for (int u = 0; u < C2R_NRT; ++u)
              if (rt0 + 4 * u < nnt) acc[u][c] = M::mma(tf, vf[u], acc[u][c]);
          }
        }
#pragma unroll
        for (int u = 0; u < C2R_NRT; ++u) {
          if (rt0 + 4 * u >= nnt) continue;
          const int row0 = c0 + (rt0 + 4 * u) * 16;
          // one 16-byte store per tile: obuf[n_a][n_b .. n_b + 3]
#pragma unroll
          for (int c = 0; c < 4; ++c)
            *reinterpret_cast<f4*>(obuf + r16 * 68 + c * 16 + 4 * g) = acc[u][c];
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
              if (a.act == ACT_SIGMA) {
                const int64_t grp = p / a.bgroup;
                const double lo = a.bounds[2 * grp], hi = a.bounds[2 * grp + 1];
#pragma unroll
                for (int i = 0; i < 16; ++i) v[i] *= preact_sigma_grad_f32(xv[i], lo, hi);
              } else {
#pragma unroll
                for (int i = 0; i < 16; ++i) v[i] *= preact_grad_f32(xv[i], a.act, a.clip);
              }
            }
            store16<T>(yout + off, v, nval, a.vec);
          }
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

template <typename T, bool VEC>
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

  if constexpr (VEC) {
    // fp16 with inner % 4 == 0: 16-byte loads of four consecutive columns
    for (int idx = threadIdx.x; idx < a.Linp * 16; idx += 256) {
      const int l = idx >> 4, jj = (idx & 15) * 4;
      h8 v = MM<_Float16>::zero();
      if (l < a.Lin && j0 + jj < a.inner)
        v = *reinterpret_cast<const h8*>(in + ((int64_t)l * a.inner + j0 + jj) * 2);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Ir[(jj + e) * ld + l] = v[2 * e];
        Ii[(jj + e) * ld + l] = v[2 * e + 1];
      }
    }
  } else {
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

// fp16 variant for small tables (Lout padded to 16 <= 128, Lin padded to 32
// <= 128, inner a multiple of 4): the twiddle table is staged in LDS next to
// the data (no global loads between the products), and the 16-row x 64-column
// result tiles are staged in LDS too, so that every store instruction writes
// whole 256-byte row segments (consecutive lanes, consecutive 16 bytes).
size_t axis_f16_lds_bytes(int Linp, int Lout16) {
  const int ldl = Linp + 8;
  return (size_t)2 * 64 * ldl * 2 + (size_t)2 * Lout16 * ldl * 2 + (size_t)Lout16 * 68 * 4;
}

template <int NTT>
__global__ __launch_bounds__(256) void axis_f16_kernel(AxisArgs a) {
  typedef MM<_Float16> M;
  constexpr int KS = 32;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ldl = a.Linp + 8;
  _Float16* Ir = reinterpret_cast<_Float16*>(smem);
  _Float16* Ii = Ir + 64 * ldl;
  _Float16* Er = Ii + 64 * ldl;
  _Float16* Ei = Er + NTT * 16 * ldl;
  uint32_t* Ob = reinterpret_cast<uint32_t*>(Ei + NTT * 16 * ldl);  // [NTT*16][68]
  const int j0 = blockIdx.x * 64;
  const int64_t o = blockIdx.y;
  const _Float16* in = reinterpret_cast<const _Float16*>(a.in) + o * (int64_t)a.Lin * a.inner * 2;
  _Float16* out = reinterpret_cast<_Float16*>(a.out) + o * (int64_t)a.Lout * a.inner * 2;
  const _Float16* er = reinterpret_cast<const _Float16*>(a.er);
  const _Float16* ei = reinterpret_cast<const _Float16*>(a.ei);

  // table: [NTT*16][Linp] twice, 16-byte pieces; data: Linp rows x 16 quads
  const int tpr = a.Linp / 8;
  for (int i = tid; i < 2 * NTT * 16 * tpr; i += 256) {
    const int tab = i / (NTT * 16 * tpr), rem = i - tab * (NTT * 16 * tpr);
    const int t = rem / tpr, c = (rem - t * tpr) * 8;
    const h8 v = *reinterpret_cast<const h8*>((tab ? ei : er) + (int64_t)t * a.Linp + c);
    *reinterpret_cast<h8*>((tab ? Ei : Er) + t * ldl + c) = v;
  }
  for (int idx = tid; idx < a.Linp * 16; idx += 256) {
    const int l = idx >> 4, jj = (idx & 15) * 4;
    h8 v = M::zero();
    if (l < a.Lin && j0 + jj < a.inner)
      v = *reinterpret_cast<const h8*>(in + ((int64_t)l * a.inner + j0 + jj) * 2);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      Ir[(jj + e) * ldl + l] = v[2 * e];
      Ii[(jj + e) * ldl + l] = v[2 * e + 1];
    }
  }
  __syncthreads();
  // D[t][j] = sum_l E[t][l] X[l][j]; wave owns columns 16 wave .. + 16
  f4 accR[NTT], accI[NTT];
#pragma unroll
  for (int u = 0; u < NTT; ++u) accR[u] = accI[u] = f4zero();
  for (int k0 = 0; k0 < a.Linp; k0 += KS) {
    const h8 br = M::ld(Ir + (wave * 16 + r16) * ldl + k0 + g * 8);
    const h8 bi = M::ld(Ii + (wave * 16 + r16) * ldl + k0 + g * 8);
#pragma unroll
    for (int u = 0; u < NTT; ++u) {
      const h8 xr = M::ld(Er + (u * 16 + r16) * ldl + k0 + g * 8);
      const h8 xi = M::ld(Ei + (u * 16 + r16) * ldl + k0 + g * 8);
      const h8 nxi = M::neg(xi);
      accR[u] = M::mma(xr, br, accR[u]);
      accR[u] = M::mma(nxi, bi, accR[u]);
      accI[u] = M::mma(xr, bi, accI[u]);
      accI[u] = M::mma(xi, br, accI[u]);
    }
  }
  // D: lane holds rows t = 16 u + 4 g + i, column j = 16 wave + r16
#pragma unroll
  for (int u = 0; u < NTT; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      h2 v = {to_h(accR[u][i] * a.scale), to_h(accI[u][i] * a.scale)};
      uint32_t w;
      __builtin_memcpy(&w, &v, 4);
      Ob[(u * 16 + 4 * g + i) * 68 + wave * 16 + r16] = w;
    }
  __syncthreads();
  // rows t < Lout, 64 complex (256 bytes) each: 16 pieces of 16 bytes
  for (int i = tid; i < a.Lout * 16; i += 256) {
    const int t = i >> 4, q = i & 15;
    if (j0 + 4 * q < a.inner) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(Ob + t * 68 + 4 * q);
      *reinterpret_cast<u32x4*>(out + ((int64_t)t * a.inner + j0 + 4 * q) * 2) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Per-mode channel contraction (forward and adjoint):
//   out[b][p][t] = scale c(t) sum_q in[b][q][t] Wop(q, p, t)
// Tile: 8 modes x 32 batch rows x 32 output channels per work-group; the
// reduction runs over chunks of QC input channels, the next chunk's loads in
// flight while the current one is multiplied.
// ---------------------------------------------------------------------------
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void contract_kernel(ContractArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int CPL = CplxIO<T>::CPL;
  constexpr int TM = CT_TM, BB = CT_BB, PB = CT_PB;
  constexpr int QC = (sizeof(T) == 2) ? 32 : 16;
  constexpr int LDQ = QC + 16 / (int)sizeof(T);
  constexpr int NG = BB * (QC / 4) * (TM / CPL);  // 4-row groups per tile (= 512)
  constexpr int GPT = NG / 256;                   // groups per thread
  constexpr size_t SA = (size_t)2 * TM * BB * LDQ, SB = (size_t)2 * TM * PB * LDQ;
  constexpr size_t STAGE = sizeof(T) * (SA + SB);
  constexpr size_t OUTB = sizeof(T) * 2 * BB * PB * TM;
  static_assert(NG % 256 == 0, "staging groups must divide over 256 threads");
  __shared__ __align__(16) unsigned char smem[STAGE > OUTB ? STAGE : OUTB];
  T* sA = reinterpret_cast<T*>(smem);   // [re/im][TM][BB][LDQ]
  T* sB = sA + SA;                      // [re/im][TM][PB][LDQ]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int npb = (a.P + PB - 1) / PB, nbb = (a.B + BB - 1) / BB;
  const int lid = xcd_logical_block(blockIdx.x, gridDim.x);
  const int t0 = (lid / (npb * nbb)) * TM;
  const int p0 = (lid % npb) * PB;
  const int b0 = ((lid / npb) % nbb) * BB;
  const T* in = reinterpret_cast<const T*>(a.in);
  const T* w = reinterpret_cast<const T*>(a.w);
  const T* zr = reinterpret_cast<const T*>(a.zeros);
  const bool vec = VEC;
  const int bt = wave >> 1, pt = wave & 1;

  u32x4 LA[GPT][4], LB[GPT][4];
  auto load_chunk = [&](int q0) {
#pragma unroll
    for (int gi = 0; gi < GPT; ++gi) {
      const int gidx = threadIdx.x + 256 * gi;
      const int mg = gidx % (TM / CPL);
      const int q4 = (gidx / (TM / CPL)) % (QC / 4);
      const int rr = gidx / ((TM / CPL) * (QC / 4));   // b (A) or p (B) within the tile
      const int tt = t0 + mg * CPL;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int q = q0 + q4 * 4 + j;
        const int b = b0 + rr;
        LA[gi][j] = load_modes16<T, VEC>(zr, in + ((int64_t)b * a.Q + q) * a.K * 2, tt, a.K,
                                         b < a.B && q < a.Q);
        const int pc = p0 + rr;
        const int64_t wrow = a.adjoint ? ((int64_t)pc * a.wcols + q) : ((int64_t)q * a.wcols + pc);
        LB[gi][j] = load_modes16<T, VEC>(zr, w + wrow * a.K * 2, tt, a.K, pc < a.P && q < a.Q);
      }
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int gi = 0; gi < GPT; ++gi) {
      const int gidx = threadIdx.x + 256 * gi;
      const int mg = gidx % (TM / CPL);
      const int q4 = (gidx / (TM / CPL)) % (QC / 4);
      const int rr = gidx / ((TM / CPL) * (QC / 4));
      T* da = sA + ((size_t)(mg * CPL) * BB + rr) * LDQ + q4 * 4;
      scatter4<T>(LA[gi], da, da + TM * BB * LDQ, BB * LDQ, false);
      T* db = sB + ((size_t)(mg * CPL) * PB + rr) * LDQ + q4 * 4;
      scatter4<T>(LB[gi], db, db + TM * PB * LDQ, PB * LDQ, a.adjoint != 0);
    }
  };

  f4 accR[TM], accI[TM];
#pragma unroll
  for (int m = 0; m < TM; ++m) accR[m] = accI[m] = f4zero();

  load_chunk(0);
  for (int q0 = 0; q0 < a.Q; q0 += QC) {
    store_chunk();
    block_sync_lds();
    if (q0 + QC < a.Q) load_chunk(q0 + QC);
#pragma unroll
    for (int m = 0; m < TM; ++m) {
#pragma unroll
      for (int k0 = 0; k0 < QC; k0 += KS) {
        const T* pa = sA + ((size_t)m * BB + bt * 16 + r16) * LDQ + k0 + g * KPL;
        const T* pb = sB + ((size_t)m * PB + pt * 16 + r16) * LDQ + k0 + g * KPL;
        frag ar = M::ld(pa), ai = M::ld(pa + TM * BB * LDQ);
        frag br = M::ld(pb), bi = M::ld(pb + TM * PB * LDQ);
        frag nai = M::neg(ai);
        accR[m] = M::mma(ar, br, accR[m]);
        accR[m] = M::mma(nai, bi, accR[m]);
        accI[m] = M::mma(ar, bi, accI[m]);
        accI[m] = M::mma(ai, br, accI[m]);
      }
    }
    block_sync_lds();
  }
  // epilogue: [b][p][t] complex staged in LDS, written as rows of 8 modes
  T* so = reinterpret_cast<T*>(smem);
#pragma unroll
  for (int m = 0; m < TM; ++m) {
    const int t = t0 + m;
    const float sc = (t < a.K) ? a.scale * cmult(t, a.Kb, a.Nb) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int bb = bt * 16 + 4 * g + i, pp = pt * 16 + r16;
      store_pair<T>(so + ((bb * PB + pp) * TM + m) * 2, accR[m][i] * sc, accI[m][i] * sc);
    }
  }
  block_sync_lds();
  T* out = reinterpret_cast<T*>(a.out);
  constexpr int V16 = TM * 2 * (int)sizeof(T) / 16;  // 16-byte pieces per (b, p) row
  const int nmodes = min(TM, a.K - t0);
  for (int idx = threadIdx.x; idx < BB * PB * V16; idx += 256) {
    const int v = idx % V16, bp = idx / V16;
    const int bb = bp / PB, pp = bp % PB;
    const int b = b0 + bb, pc = p0 + pp;
    if (b < a.B && pc < a.P) {
      T* d = out + (((int64_t)b * a.P + pc) * a.K + t0) * 2;
      const T* sv = so + (size_t)bp * TM * 2;
      if (nmodes == TM && vec) {
        reinterpret_cast<u32x4*>(d)[v] = reinterpret_cast<const u32x4*>(sv)[v];
      } else if (v == 0) {
        for (int i = 0; i < 2 * nmodes; ++i) d[i] = sv[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Weight gradient: gw[q][p][t] = scale c(t) sum_b conj(xh[b][q][t]) gh[b][p][t]
// Tile: 8 modes x 32 (q) x 32 (p); fixed-order reduction over batch chunks.
// ---------------------------------------------------------------------------
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a) {
  using M = MM<T>;
  using frag = typename M::frag;
  constexpr int KPL = M::KPL, KS = M::KSTEP;
  constexpr int CPL = CplxIO<T>::CPL;
  constexpr int TM = CT_TM, QB = 32, PB = 32;
  constexpr int BC = (sizeof(T) == 2) ? 32 : 16;  // batch rows per chunk (MFMA K)
  constexpr int LDB = BC + 16 / (int)sizeof(T);
  constexpr int NG = QB * (BC / 4) * (TM / CPL);
  constexpr int GPT = NG / 256;
  constexpr size_t SX = (size_t)2 * TM * QB * LDB, SG = (size_t)2 * TM * PB * LDB;
  constexpr size_t STAGE = sizeof(T) * (SX + SG);
  constexpr size_t OUTB = sizeof(float) * 2 * QB * PB * TM;
  static_assert(NG % 256 == 0, "staging groups must divide over 256 threads");
  __shared__ __align__(16) unsigned char smem[STAGE > OUTB ? STAGE : OUTB];
  T* sX = reinterpret_cast<T*>(smem);   // [re/im][TM][QB][LDB]
  T* sG = sX + SX;                      // [re/im][TM][PB][LDB]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int nqb = (a.Cin + QB - 1) / QB, npb = (a.Cout + PB - 1) / PB;
  const int lid = xcd_logical_block(blockIdx.x, gridDim.x);
  const int t0 = (lid / (nqb * npb)) * TM;
  const int q0 = ((lid / npb) % nqb) * QB;
  const int p0 = (lid % npb) * PB;
  const T* xh = reinterpret_cast<const T*>(a.xh);
  const T* gh = reinterpret_cast<const T*>(a.gh);
  const T* zr = reinterpret_cast<const T*>(a.zeros);
  const int qt = wave >> 1, pt = wave & 1;

  u32x4 LX[GPT][4], LG[GPT][4];
  auto load_chunk = [&](int bs) {
#pragma unroll
    for (int gi = 0; gi < GPT; ++gi) {
      const int gidx = threadIdx.x + 256 * gi;
      const int mg = gidx % (TM / CPL);
      const int b4 = (gidx / (TM / CPL)) % (BC / 4);
      const int rr = gidx / ((TM / CPL) * (BC / 4));   // q (X) or p (G) within the tile
      const int tt = t0 + mg * CPL;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int b = bs + b4 * 4 + j;
        const int q = q0 + rr, pc = p0 + rr;
        LX[gi][j] = load_modes16<T, VEC>(zr, xh + ((int64_t)b * a.Cin + q) * a.K * 2, tt,
                                         a.K, b < a.B && q < a.Cin);
        LG[gi][j] = load_modes16<T, VEC>(zr, gh + ((int64_t)b * a.Cout + pc) * a.K * 2, tt,
                                         a.K, b < a.B && pc < a.Cout);
      }
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int gi = 0; gi < GPT; ++gi) {
      const int gidx = threadIdx.x + 256 * gi;
      const int mg = gidx % (TM / CPL);
      const int b4 = (gidx / (TM / CPL)) % (BC / 4);
      const int rr = gidx / ((TM / CPL) * (BC / 4));
      T* dx = sX + ((size_t)(mg * CPL) * QB + rr) * LDB + b4 * 4;
      scatter4<T>(LX[gi], dx, dx + TM * QB * LDB, QB * LDB, false);
      T* dg = sG + ((size_t)(mg * CPL) * PB + rr) * LDB + b4 * 4;
      scatter4<T>(LG[gi], dg, dg + TM * PB * LDB, PB * LDB, false);
    }
  };

  f4 accR[TM], accI[TM];
#pragma unroll
  for (int m = 0; m < TM; ++m) accR[m] = accI[m] = f4zero();

  load_chunk(0);
  for (int bs = 0; bs < a.B; bs += BC) {
    store_chunk();
    block_sync_lds();
    if (bs + BC < a.B) load_chunk(bs + BC);
#pragma unroll
    for (int m = 0; m < TM; ++m) {
#pragma unroll
      for (int k0 = 0; k0 < BC; k0 += KS) {
        const T* px = sX + ((size_t)m * QB + qt * 16 + r16) * LDB + k0 + g * KPL;
        const T* pg = sG + ((size_t)m * PB + pt * 16 + r16) * LDB + k0 + g * KPL;
        frag xr = M::ld(px), xi = M::ld(px + TM * QB * LDB);
        frag gr = M::ld(pg), gi_ = M::ld(pg + TM * PB * LDB);
        frag nxi = M::neg(xi);
        // conj(x) g = (xr gr + xi gi) + i (xr gi - xi gr)
        accR[m] = M::mma(xr, gr, accR[m]);
        accR[m] = M::mma(xi, gi_, accR[m]);
        accI[m] = M::mma(xr, gi_, accI[m]);
        accI[m] = M::mma(nxi, gr, accI[m]);
      }
    }
    block_sync_lds();
  }
  float* so = reinterpret_cast<float*>(smem);  // [QB][PB][TM] complex
#pragma unroll
  for (int m = 0; m < TM; ++m) {
    const int t = t0 + m;
    const float sc = (t < a.K) ? a.scale * cmult(t, a.Kb, a.Nb) : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qq = qt * 16 + 4 * g + i, pp = pt * 16 + r16;
      store_pair<float>(so + ((qq * PB + pp) * TM + m) * 2, accR[m][i] * sc, accI[m][i] * sc);
    }
  }
  block_sync_lds();
  constexpr int V16 = TM * 8 / 16;  // 16-byte pieces per (q, p) row of fp32 complex
  const int nmodes = min(TM, a.K - t0);
  const bool vout = (a.K % 2) == 0;
  for (int idx = threadIdx.x; idx < QB * PB * V16; idx += 256) {
    const int v = idx % V16, qp = idx / V16;
    const int qq = qp / PB, pp = qp % PB;
    const int q = q0 + qq, pc = p0 + pp;
    if (q < a.Cin && pc < a.Cout) {
      float* d = a.gw + (((int64_t)q * a.Cout + pc) * a.K + t0) * 2;
      const float* sv = so + (size_t)qp * TM * 2;
      if (nmodes == TM && vout) {
        reinterpret_cast<f4*>(d)[v] = reinterpret_cast<const f4*>(sv)[v];
      } else if (v == 0) {
        for (int i = 0; i < 2 * nmodes; ++i) d[i] = sv[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Generic pairwise complex contraction (Tucker and CP path steps), fp32
// accumulate.  The result index is decoded once into the two operands'
// offsets; the contracted indices are walked with an odometer (counters and
// offsets stepped in place by a mixed-radix addition, no division per
// element).  Two launch shapes: one thread per result element, or, for few
// results with long reductions, one work-group per result element.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f2 load_elem(const void* p, int elem, int64_t off) {
  if (elem == ELEM_F16) {
    h2 v = reinterpret_cast<const h2*>(p)[off];
    return f2{(float)v[0], (float)v[1]};
  }
  return reinterpret_cast<const f2*>(p)[off];
}

// Offsets of result element idx in A and B, and its last-spatial-axis slot.
// (while the result has fewer than 2^32 elements, 32-bit division by
// multiply-high: a true divide costs tens of instructions and runs once per
// index per element)
__device__ __forceinline__ void pair_decode(const PairArgs& a, int64_t idx, int64_t& aoff,
                                            int64_t& boff, int64_t& cidx) {
  aoff = 0;
  boff = 0;
  cidx = 0;
  if (a.out_size <= 0xffffffffll) {
    uint32_t rem = (uint32_t)idx;
    for (int k = a.n_out - 1; k >= 0; --k) {
      const uint32_t q = fast_div(rem, a.out_mag[k], a.out_shr[k]);
      const uint32_t v = rem - q * (uint32_t)a.out_ext[k];
      rem = q;
      aoff += (int64_t)v * a.a_stride_out[k];
      boff += (int64_t)v * a.b_stride_out[k];
      if (k == a.scale_c_axis) cidx = v;
    }
    return;
  }
  int64_t rem = idx;
  for (int k = a.n_out - 1; k >= 0; --k) {
    const int64_t e = a.out_ext[k];
    const int64_t v = rem % e;
    rem /= e;
    aoff += v * a.a_stride_out[k];
    boff += v * a.b_stride_out[k];
    if (k == a.scale_c_axis) cidx = v;
  }
}

// Advance the contracted-index counters by `dig` (digits of the step in the
// radix of the contracted extents, innermost last), carrying outwards, and
// move the two offsets along.
__device__ __forceinline__ void pair_step(const PairArgs& a, const int64_t (&dig)[PW_MAXIDX],
                                          int64_t (&cnt)[PW_MAXIDX], int64_t& ao,
                                          int64_t& bo) {
  int64_t carry = 0;
#pragma unroll
  for (int k = PW_MAXIDX - 1; k >= 0; --k) {
    if (k < a.n_red) {
      const int64_t add = dig[k] + carry;
      cnt[k] += add;
      ao += add * a.a_stride_red[k];
      bo += add * a.b_stride_red[k];
      carry = 0;
      if (cnt[k] >= a.red_ext[k]) {
        cnt[k] -= a.red_ext[k];
        ao -= a.red_ext[k] * a.a_stride_red[k];
        bo -= a.red_ext[k] * a.b_stride_red[k];
        carry = 1;
      }
    }
  }
}

// Counters of contracted element r0 and the digits of `step`; offsets move
// to element r0.
__device__ __forceinline__ void pair_start(const PairArgs& a, int64_t r0, int64_t step,
                                           int64_t (&dig)[PW_MAXIDX], int64_t (&cnt)[PW_MAXIDX],
                                           int64_t& ao, int64_t& bo) {
  int64_t q = step, rr = r0;
#pragma unroll
  for (int k = PW_MAXIDX - 1; k >= 0; --k) {
    dig[k] = 0;
    cnt[k] = 0;
    if (k < a.n_red) {
      const int64_t e = a.red_ext[k];
      dig[k] = q % e;
      q /= e;
      cnt[k] = rr % e;
      rr /= e;
      ao += cnt[k] * a.a_stride_red[k];
      bo += cnt[k] * a.b_stride_red[k];
    }
  }
}

__device__ __forceinline__ void pair_fma(const PairArgs& a, f2 x, f2 y, float& sr, float& si) {
  if (a.conj_a) x[1] = -x[1];
  if (a.conj_b) y[1] = -y[1];
  sr = fmaf(x[0], y[0], sr);
  sr = fmaf(-x[1], y[1], sr);
  si = fmaf(x[0], y[1], si);
  si = fmaf(x[1], y[0], si);
}

// Sum over contracted elements r0, r0 + step, ... below r1, starting from
// the result element's offsets.  Eight elements' loads are issued before
// their products (in the same order, so the sum is the plain sequential one).
__device__ __forceinline__ void pair_reduce(const PairArgs& a, int64_t r0, int64_t r1,
                                            int64_t step, int64_t ao, int64_t bo, float& sr,
                                            float& si) {
  if (r0 >= r1) return;
  int64_t dig[PW_MAXIDX], cnt[PW_MAXIDX];
  pair_start(a, r0, step, dig, cnt, ao, bo);
  constexpr int UN = 8;
  int64_t r = r0;
  for (; r + (UN - 1) * step < r1; r += UN * step) {
    f2 xs[UN], ys[UN];
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      xs[u] = load_elem(a.a, a.a_elem, ao);
      ys[u] = load_elem(a.b, a.b_elem, bo);
      pair_step(a, dig, cnt, ao, bo);
    }
#pragma unroll
    for (int u = 0; u < UN; ++u) pair_fma(a, xs[u], ys[u], sr, si);
  }
  for (; r < r1; r += step) {
    pair_fma(a, load_elem(a.a, a.a_elem, ao), load_elem(a.b, a.b_elem, bo), sr, si);
    pair_step(a, dig, cnt, ao, bo);
  }
}

__device__ __forceinline__ void pair_store(const PairArgs& a, int64_t idx, int64_t cidx,
                                           float sr, float si) {
  float s = a.scale;
  if (a.scale_c_axis >= 0) s *= (cidx == 0 || 2 * cidx == a.Nb) ? 1.0f : 2.0f;
  if (a.out_elem == ELEM_F16) {
    reinterpret_cast<h2*>(a.out)[idx] = h2{to_h(sr * s), to_h(si * s)};
  } else {
    reinterpret_cast<f2*>(a.out)[idx] = f2{sr * s, si * s};
  }
}

__global__ __launch_bounds__(256) void pair_kernel(PairArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.out_size) return;
  int64_t aoff, boff, cidx;
  pair_decode(a, idx, aoff, boff, cidx);
  float sr = 0.0f, si = 0.0f;
  pair_reduce(a, 0, a.red_size, 1, aoff, boff, sr, si);
  pair_store(a, idx, cidx, sr, si);
}

// Products without a contracted index (elementwise and outer products):
// PE_NV consecutive results along the innermost result index per thread,
// decoded once; each is the same single product as in pair_kernel.  The
// two results of a thread are stored with one access (16 bytes fp32, 8 bytes
// fp16), so consecutive lanes write consecutive bytes and every store
// instruction covers whole cache lines.
constexpr int PE_NV = 2;

__global__ __launch_bounds__(256) void pair_ew_kernel(PairArgs a, int64_t items) {
  const int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (it >= items) return;
  const int64_t idx = it * PE_NV;
  int64_t ao, bo, cidx;
  pair_decode(a, idx, ao, bo, cidx);
  const int kin = a.n_out - 1;
  const int64_t sa = a.a_stride_out[kin], sb = a.b_stride_out[kin];
  f2 x[PE_NV], y[PE_NV];
#pragma unroll
  for (int j = 0; j < PE_NV; ++j) {
    x[j] = load_elem(a.a, a.a_elem, ao + j * sa);
    y[j] = load_elem(a.b, a.b_elem, bo + j * sb);
  }
  float r[2 * PE_NV];
#pragma unroll
  for (int j = 0; j < PE_NV; ++j) {
    float sr = 0.0f, si = 0.0f;
    pair_fma(a, x[j], y[j], sr, si);
    float s = a.scale;
    if (a.scale_c_axis >= 0) {
      const int64_t ci = kin == a.scale_c_axis ? cidx + j : cidx;
      s *= (ci == 0 || 2 * ci == a.Nb) ? 1.0f : 2.0f;
    }
    r[2 * j] = sr * s;
    r[2 * j + 1] = si * s;
  }
  if (a.out_elem == ELEM_F16) {
    h4 v = {to_h(r[0]), to_h(r[1]), to_h(r[2]), to_h(r[3])};
    reinterpret_cast<h4*>(a.out)[it] = v;
  } else {
    reinterpret_cast<f4*>(a.out)[it] = f4{r[0], r[1], r[2], r[3]};
  }
}

// PB_NB results per thread along result index blk_k (absent from A): the
// thread walks the contraction once, loads each A element once and the PB_NB
// matching B elements, and keeps PB_NB sums.  Each sum runs over the
// contracted elements in the same order as in pair_kernel, so the results
// are the same bits.
constexpr int PB_NB = 16;

__global__ __launch_bounds__(256) void pair_blocked_kernel(PairArgs a, int64_t items) {
  const int64_t it = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (it >= items) return;
  const int kb = a.blk_k;
  // decode the item over the result indices with blk_k in blocks of PB_NB
  // (items < 2^32: launch_pair checks; 32-bit division as in pair_decode)
  uint32_t rem = (uint32_t)it;
  int64_t ao = 0, bo = 0, oo = 0, cidx = 0, j0 = 0;
  for (int k = a.n_out - 1; k >= 0; --k) {
    const bool blk = k == kb;
    const uint32_t e =
        (uint32_t)(blk ? (a.out_ext[k] + PB_NB - 1) / PB_NB : a.out_ext[k]);
    const uint32_t q = fast_div(rem, blk ? a.blk_mag : a.out_mag[k], blk ? a.blk_shr : a.out_shr[k]);
    int64_t v = rem - q * e;
    rem = q;
    if (k == kb) {
      v *= PB_NB;
      j0 = v;
    }
    ao += v * a.a_stride_out[k];
    bo += v * a.b_stride_out[k];
    oo += v * a.res_stride[k];
    if (k == a.scale_c_axis) cidx = v;
  }
  const int nj = (int)min((int64_t)PB_NB, a.out_ext[kb] - j0);
  const int64_t bstep = a.b_stride_out[kb];
  float sr[PB_NB], si[PB_NB];
#pragma unroll
  for (int j = 0; j < PB_NB; ++j) sr[j] = si[j] = 0.0f;
  int64_t dig[PW_MAXIDX], cnt[PW_MAXIDX];
  pair_start(a, 0, 1, dig, cnt, ao, bo);
  for (int64_t r = 0; r < a.red_size; ++r) {
    f2 x = load_elem(a.a, a.a_elem, ao);
    if (a.conj_a) x[1] = -x[1];
#pragma unroll
    for (int j = 0; j < PB_NB; ++j) {
      if (j < nj) {
        f2 y = load_elem(a.b, a.b_elem, bo + j * bstep);
        if (a.conj_b) y[1] = -y[1];
        sr[j] = fmaf(x[0], y[0], sr[j]);
        sr[j] = fmaf(-x[1], y[1], sr[j]);
        si[j] = fmaf(x[0], y[1], si[j]);
        si[j] = fmaf(x[1], y[0], si[j]);
      }
    }
    pair_step(a, dig, cnt, ao, bo);
  }
  const int64_t ostep = a.res_stride[kb];
#pragma unroll
  for (int j = 0; j < PB_NB; ++j) {
    if (j < nj) {
      const int64_t ci = kb == a.scale_c_axis ? j0 + j : cidx;
      pair_store(a, oo + j * ostep, ci, sr[j], si[j]);
    }
  }
}

// One work-group per result element: thread t takes the contracted elements
// t, t + 256, ... (consecutive threads read consecutive elements of the
// innermost contracted index); the 256 partial sums are added in a fixed
// order (bit-reproducible).
__global__ __launch_bounds__(256) void pair_block_kernel(PairArgs a) {
  __shared__ float red[2][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t idx = blockIdx.x;
  int64_t aoff, boff, cidx;
  pair_decode(a, idx, aoff, boff, cidx);
  float sr = 0.0f, si = 0.0f;
  pair_reduce(a, tid, a.red_size, 256, aoff, boff, sr, si);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    sr += __shfl_xor(sr, off, 64);
    si += __shfl_xor(si, off, 64);
  }
  if (lane == 0) {
    red[0][wave] = sr;
    red[1][wave] = si;
  }
  __syncthreads();
  if (tid == 0) {
    const float tr = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const float ti = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    pair_store(a, idx, cidx, tr, ti);
  }
}

__global__ void scale_kernel(float* p, int64_t n, float s) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] *= s;
}

// Clip bounds of the statistics-based pre-activation, one work-group per
// group of n contiguous values.  The sums run in double over the values
// shifted by the group's first one (which keeps the sum of squares from
// cancelling when the mean is large against the spread); a non-finite value
// anywhere in the group makes both bounds NaN.
template <typename T>
__global__ __launch_bounds__(256) void sigma_stats_kernel(const T* x, int64_t n, double k,
                                                          double* bounds) {
  __shared__ double red[2][4];
  __shared__ int redb[4];
  const int64_t gi = blockIdx.x;
  const T* xg = x + gi * n;
  const double shift = (double)xg[0];
  double s1 = 0.0, s2 = 0.0;
  int bad = 0;
  constexpr int V = 16 / (int)sizeof(T);
  if (((n * (int64_t)sizeof(T)) & 15) == 0) {
    using vec = u32x4;
    const vec* xv = reinterpret_cast<const vec*>(xg);
    const int64_t nv = n / V;
    for (int64_t i = threadIdx.x; i < nv; i += 256) {
      const vec w = xv[i];
      const T* e = reinterpret_cast<const T*>(&w);
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const double v = (double)e[j];
        bad |= !__builtin_isfinite(v);
        const double dv = v - shift;
        s1 += dv;
        s2 = __builtin_fma(dv, dv, s2);
      }
    }
  } else {
    for (int64_t i = threadIdx.x; i < n; i += 256) {
      const double v = (double)xg[i];
      bad |= !__builtin_isfinite(v);
      const double dv = v - shift;
      s1 += dv;
      s2 = __builtin_fma(dv, dv, s2);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    s1 += __shfl_xor(s1, o);
    s2 += __shfl_xor(s2, o);
    bad |= __shfl_xor(bad, o);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = s1;
    red[1][wave] = s2;
    redb[wave] = bad;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double t1 = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const double t2 = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    const int b = redb[0] | redb[1] | redb[2] | redb[3];
    const double m1 = t1 / (double)n;
    const double var = t2 / (double)n - m1 * m1;
    const double sd = __builtin_sqrt(var > 0.0 ? var : 0.0);
    const double mu = shift + m1;
    double lo = mu - k * sd, hi = mu + k * sd;
    if (b || !__builtin_isfinite(lo) || !__builtin_isfinite(hi)) lo = hi = __builtin_nan("");
    bounds[2 * gi] = lo;
    bounds[2 * gi + 1] = hi;
  }
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

hipError_t launch_sigma_stats(int elem, const void* x, int64_t groups, int64_t n, double k,
                              double* bounds, hipStream_t s) {
  if (groups == 0) return hipSuccess;
  if (groups < 0 || groups > 0x7fffffff || n < 1) return hipErrorInvalidValue;
  dim3 grid((unsigned)groups), block(256);
  if (elem == ELEM_F16)
    hipLaunchKernelGGL(sigma_stats_kernel<_Float16>, grid, block, 0, s,
                       reinterpret_cast<const _Float16*>(x), n, k, bounds);
  else
    hipLaunchKernelGGL(sigma_stats_kernel<float>, grid, block, 0, s,
                       reinterpret_cast<const float*>(x), n, k, bounds);
  return hipGetLastError();
}

hipError_t launch_axis(int elem, const AxisArgs& a, size_t lds, hipStream_t s) {
  dim3 grid((unsigned)((a.inner + 63) / 64), (unsigned)a.outer), block(256);
  if (elem == ELEM_F16 && a.inner % 4 == 0 && a.Linp <= 128 && a.Lout16 <= 128) {
    const size_t l2 = axis_f16_lds_bytes(a.Linp, a.Lout16);
    switch (a.Lout16 / 16) {
#define FNO_AXIS_F16(N)                                                            \
  case N:                                                                          \
    FNO_LAUNCH((axis_f16_kernel<N>), grid, block, l2, s, a);                       \
    return hipGetLastError();
      FNO_AXIS_F16(1) FNO_AXIS_F16(2) FNO_AXIS_F16(3) FNO_AXIS_F16(4)
      FNO_AXIS_F16(5) FNO_AXIS_F16(6) FNO_AXIS_F16(7) FNO_AXIS_F16(8)
#undef FNO_AXIS_F16
      default: break;
    }
  }
  if (elem == ELEM_F16 && a.inner % 4 == 0)
    FNO_LAUNCH((axis_kernel<_Float16, true>), grid, block, lds, s, a);
  else if (elem == ELEM_F16)
    FNO_LAUNCH((axis_kernel<_Float16, false>), grid, block, lds, s, a);
  else
    FNO_LAUNCH((axis_kernel<float, false>), grid, block, lds, s, a);
  return hipGetLastError();
}

hipError_t launch_contract(int elem, const ContractArgs& a, hipStream_t s) {
  const int64_t nblk = (int64_t)((a.K + CT_TM - 1) / CT_TM) * ((a.P + CT_PB - 1) / CT_PB) *
                       ((a.B + CT_BB - 1) / CT_BB);
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  dim3 grid((unsigned)nblk);
  dim3 block(256);
  if (elem == ELEM_F16) {
    if (a.K % 4 == 0)
      hipLaunchKernelGGL((contract_kernel<_Float16, true>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((contract_kernel<_Float16, false>), grid, block, 0, s, a);
  } else {
    if (a.K % 2 == 0)
      hipLaunchKernelGGL((contract_kernel<float, true>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((contract_kernel<float, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_wgrad(int elem, const WgradArgs& a, hipStream_t s) {
  const int64_t nblk = (int64_t)((a.K + 7) / 8) * ((a.Cin + 31) / 32) * ((a.Cout + 31) / 32);
  if (nblk > 0x7fffffff) return hipErrorInvalidValue;
  dim3 grid((unsigned)nblk);
  dim3 block(256);
  if (elem == ELEM_F16) {
    if (a.K % 4 == 0)
      hipLaunchKernelGGL((wgrad_kernel<_Float16, true>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((wgrad_kernel<_Float16, false>), grid, block, 0, s, a);
  } else {
    if (a.K % 2 == 0)
      hipLaunchKernelGGL((wgrad_kernel<float, true>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((wgrad_kernel<float, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_pair(const PairArgs& a_in, hipStream_t s) {
  PairArgs a = a_in;
  if (a.out_size <= 0) return hipSuccess;
  {
    const hipError_t e = launch_pair_modeprod(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  {
    const hipError_t e = launch_pair_bt(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  {
    const hipError_t e = launch_pair_gemm(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  int64_t st = 1;
  for (int k = a.n_out - 1; k >= 0; --k) {
    a.res_stride[k] = st;
    st *= a.out_ext[k];
    div_magic((uint32_t)std::min<int64_t>(a.out_ext[k], 0xffffffffll), &a.out_mag[k],
              &a.out_shr[k]);
  }
  // Register blocking: the widest result index that A (the larger operand)
  // does not carry, if at least 4 wide.
  a.blk_k = -1;
  int64_t best = 3;
  for (int k = 0; k < a.n_out; ++k)
    if (a.a_stride_out[k] == 0 && a.out_ext[k] > best) {
      best = a.out_ext[k];
      a.blk_k = k;
    }
  if (a.blk_k >= 0)
    div_magic((uint32_t)((a.out_ext[a.blk_k] + PB_NB - 1) / PB_NB), &a.blk_mag, &a.blk_shr);
  // Few results with long reductions (weight-gradient steps): a work-group
  // per result.  Otherwise a thread per PB_NB results or per result.
  if (a.red_size == 1 && a.n_out > 0 && a.out_ext[a.n_out - 1] % PE_NV == 0 &&
      a.out_size / PE_NV <= 0xffffffffll * 256) {
    const int64_t items = a.out_size / PE_NV;
    dim3 grid((unsigned)((items + 255) / 256)), block(256);
    hipLaunchKernelGGL(pair_ew_kernel, grid, block, 0, s, a, items);
  } else if (a.red_size >= 2048 && a.out_size <= (int64_t)1 << 20) {
    dim3 grid((unsigned)a.out_size), block(256);
    hipLaunchKernelGGL(pair_block_kernel, grid, block, 0, s, a);
  } else if (a.blk_k >= 0 &&
             a.out_size / a.out_ext[a.blk_k] * ((a.out_ext[a.blk_k] + PB_NB - 1) / PB_NB) >=
                 ((int64_t)1 << 17)) {
    // (only with enough blocked items left to fill the chip: >= 2048 waves)
    const int64_t items = a.out_size / a.out_ext[a.blk_k] *
                          ((a.out_ext[a.blk_k] + PB_NB - 1) / PB_NB);
    if (items > 0xffffffffll) return hipErrorInvalidValue;
    dim3 grid((unsigned)((items + 255) / 256)), block(256);
    hipLaunchKernelGGL(pair_blocked_kernel, grid, block, 0, s, a, items);
  } else {
    dim3 grid((unsigned)((a.out_size + 255) / 256)), block(256);
    hipLaunchKernelGGL(pair_kernel, grid, block, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_scale_complex(float* p, int64_t n, float sc, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  dim3 grid((unsigned)((n + 255) / 256)), block(256);
  hipLaunchKernelGGL(scale_kernel, grid, block, 0, st, p, n, sc);
  return hipGetLastError();
}

}  // namespace fno
