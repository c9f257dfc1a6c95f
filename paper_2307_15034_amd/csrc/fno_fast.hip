// Persistent fast-path truncated transforms for fp16 planes of up to 128 rows
// x 256 columns (the 64^2, 128^2 and 3-D 64^2-slice workloads).
//
// Each work-group stays resident and walks planes p = blockIdx.x,
// blockIdx.x + gridDim.x, ...; the twiddle tables are staged once per
// work-group (LDS, or registers for the inverse's leading-axis factors), the
// next plane's input is loaded into registers while the current plane is
// transformed, and block barriers wait for LDS traffic only, so those
// prefetches stay in flight across them.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fno_device.h"

namespace fno {

namespace {

typedef MM<_Float16> MH;
constexpr int KS = 32;   // k per MFMA step (v_mfma_f32_16x16x32_f16)
constexpr int PADH = 8;  // LDS row padding in halves (rows then start 4 banks apart)

__device__ __forceinline__ h8 as_h8(const u32x4& v) {
  h8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ u32x4 h8_as_u(const h8& v) {
  u32x4 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// Cooperative copy of a [rows][cols] fp16 table (global, row stride gstride)
// into LDS with row stride lstride; columns past `cols` are zero-filled up to
// lcols.  cols, lcols, gstride multiples of 8.
template <int NT>
__device__ __forceinline__ void stage_table(_Float16* dst, int lstride, int lcols,
                                            const _Float16* src, int gstride, int rows,
                                            int cols) {
  const int cpr = lcols / 8;  // 16-byte pieces per row
  for (int i = threadIdx.x; i < rows * cpr; i += NT) {
    const int r = i / cpr, c = (i - r * cpr) * 8;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (c < cols) v = *reinterpret_cast<const u32x4*>(src + (int64_t)r * gstride + c);
    *reinterpret_cast<u32x4*>(dst + r * lstride + c) = v;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// Forward: plane [Na][Nb] -> spectrum [Ka][Kb]; one wave per 16-row tile
// (Na <= 16*NW), Nb <= 32*NKA, Kb <= 8*NCT.  Step A (last axis): rows x
// [cos | -sin] table on MFMA; step B (leading axis): complex multiply-
// accumulate with cos/sin of k_a(t) n, one 16x16 output tile per wave at a time.
// ---------------------------------------------------------------------------
template <int NCT, int NKA, int NW>
__global__ __launch_bounds__(NW * 64, 2) void r2c_fast_kernel(R2CArgs a) {
  constexpr int NT = NW * 64;
  constexpr int Kbp = NCT * 8, NTB = NCT / 2;
  constexpr int R = 16 * NW;
  constexpr int LDT = NKA * KS + PADH;  // twA row stride
  constexpr int LDA = R + PADH;         // AT row stride
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int LDC = a.Nap + PADH;         // cB / sB row stride
  _Float16* sTw = reinterpret_cast<_Float16*>(smem);   // [2 Kbp][LDT]
  _Float16* sC = sTw + 2 * Kbp * LDT;                   // [Kap16][LDC]
  _Float16* sS = sC + a.Kap16 * LDC;
  _Float16* ATr = sS + a.Kap16 * LDC;                   // [Kbp][LDA]
  _Float16* ATi = ATr + Kbp * LDA;
  const _Float16* x = reinterpret_cast<const _Float16*>(a.in);
  const _Float16* zr = reinterpret_cast<const _Float16*>(a.zeros);
  _Float16* out = reinterpret_cast<_Float16*>(a.out);

  stage_table<NT>(sTw, LDT, NKA * KS, reinterpret_cast<const _Float16*>(a.twA), a.Nbp,
                  2 * Kbp, a.Nbp);
  stage_table<NT>(sC, LDC, a.Nap, reinterpret_cast<const _Float16*>(a.cB), a.Nap, a.Kap16,
                  a.Nap);
  stage_table<NT>(sS, LDC, a.Nap, reinterpret_cast<const _Float16*>(a.sB), a.Nap, a.Kap16,
                  a.Nap);

  const int nta = a.Kap16 >> 4;
  const int ntiles = nta * NTB;          // step-B output tiles
  const int nkb = (a.Na + KS - 1) / KS;  // step-B k-steps
  const int64_t plane = (int64_t)a.Na * a.Nb;
  const int row = wave * 16 + r16;       // this lane's row in step A

  // Loads are issued unconditionally (past the last plane they read the zero
  // block) so that the wait before a plane's use counts every load issued
  // after it; a skipped load would make the compiler wait for all of them.
  auto load_plane = [&](int64_t p, u32x4 (&buf)[NKA]) {
    const bool pok = p < a.planes;
    const _Float16* base = x + (pok ? p : 0) * plane;
#pragma unroll
    for (int s = 0; s < NKA; ++s) {
      const int col = s * KS + g * 8;
      const bool ok = pok && row < a.Na && col < a.Nb;
      buf[s] = *reinterpret_cast<const u32x4*>(ok ? base + (int64_t)row * a.Nb + col : zr);
    }
  };

  auto process = [&](int64_t p, const u32x4 (&cur)[NKA]) {
    // ---- step A: this wave's 16 rows -> 2 Kbp columns ---------------------------
    {
      f4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f4zero();
#pragma unroll
      for (int s = 0; s < NKA; ++s) {
        h8 v = as_h8(cur[s]);
        if (a.act) {
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = to_h(preact_f32((float)v[i], a.act, a.clip));
        }
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          h8 bf = MH::ld(sTw + (ct * 16 + r16) * LDT + s * KS + g * 8);
          acc[ct] = MH::mma(v, bf, acc[ct]);
        }
      }
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int col = ct * 16 + r16;
        _Float16* dst = (col < Kbp ? ATr + col * LDA : ATi + (col - Kbp) * LDA) + wave * 16 + 4 * g;
        h4 w4;
#pragma unroll
        for (int i = 0; i < 4; ++i) w4[i] = to_h(acc[ct][i] * a.scaleA);
        *reinterpret_cast<h4*>(dst) = w4;
      }
    }
    block_sync_lds();
    // ---- step B: output tiles (t_a tile, t_b tile) round-robin over waves ------
    _Float16* o = out + p * (int64_t)a.Ka * a.Kb * 2;
    for (int tile = wave; tile < ntiles; tile += NW) {
      const int ta = tile / NTB, tb = tile - ta * NTB;
      f4 accR = f4zero(), accI = f4zero();
      for (int ks = 0; ks < nkb; ++ks) {
        const int toff = (ta * 16 + r16) * LDC + ks * KS + g * 8;
        const int aoff = (tb * 16 + r16) * LDA + ks * KS + g * 8;
        h8 cf = MH::ld(sC + toff), sf = MH::ld(sS + toff);
        h8 ar = MH::ld(ATr + aoff), ai = MH::ld(ATi + aoff);
        h8 nsf = -sf;
        accR = MH::mma(cf, ar, accR);
        accR = MH::mma(sf, ai, accR);
        accI = MH::mma(cf, ai, accI);
        accI = MH::mma(nsf, ar, accI);
      }
      const int t_b = tb * 16 + r16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t_a = ta * 16 + 4 * g + i;
        if (t_a < a.Ka && t_b < a.Kb)
          store_pair<_Float16>(o + ((int64_t)t_a * a.Kb + t_b) * 2, accR[i] * a.scaleB,
                               accI[i] * a.scaleB);
      }
    }
    block_sync_lds();  // AT free for the next plane
  };

  // Planes p, p + G, p + 2G, ... with the input two planes ahead in flight:
  // three register buffers in fixed roles per unrolled step (no register
  // copies, so a wait happens only where a buffer is consumed).
  const int64_t G = gridDim.x;
  u32x4 b0[NKA], b1[NKA], b2[NKA];
  int64_t p = blockIdx.x;
  load_plane(p, b0);
  load_plane(p + G, b1);
  block_sync_lds();  // tables staged
  for (; p < a.planes; p += 3 * G) {
    load_plane(p + 2 * G, b2);
    process(p, b0);
    if (p + G >= a.planes) break;
    load_plane(p + 3 * G, b0);
    process(p + G, b1);
    if (p + 2 * G >= a.planes) break;
    load_plane(p + 4 * G, b1);
    process(p + 2 * G, b2);
  }
}

// ---------------------------------------------------------------------------
// Inverse: spectrum [Ka][Kb] -> plane [Na][Nb]; one wave per 16-row tile
// (Na <= 16*NW), Nb <= 64*NBT, Ka <= 32*NKZ, Kb <= 8*NCT.  EPI multiplies by
// the pre-activation's derivative f'(x).
// ---------------------------------------------------------------------------
template <int NCT, int NW, int NBT, int NKZ, bool EPI>
__global__ __launch_bounds__(NW * 64, 2) void c2r_fast_kernel(C2RArgs a) {
  constexpr int NT = NW * 64;
  constexpr int Kbp = NCT * 8, NTB = NCT / 2;
  constexpr int Kap = NKZ * KS;
  constexpr int LDZ = Kap + PADH;        // ZT row stride
  constexpr int LDV = 2 * Kbp + PADH;    // VL / twI row stride
  constexpr int NB64 = NBT * 64;
  constexpr int ZGROUPS = (Kap / 4) * (Kbp / 4);         // 4 t_a rows x 4 t_b columns
  constexpr int ZG = (ZGROUPS + NT - 1) / NT;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  _Float16* ZTr = reinterpret_cast<_Float16*>(smem);   // [Kbp][LDZ]
  _Float16* ZTi = ZTr + Kbp * LDZ;
  _Float16* VL = ZTi + Kbp * LDZ;                       // [16 NW][LDV]
  _Float16* sTw = VL + 16 * NW * LDV;                   // [NB64][LDV]
  float* obuf = reinterpret_cast<float*>(sTw + NB64 * LDV) + wave * (16 * 68);
  const _Float16* zin = reinterpret_cast<const _Float16*>(a.in);
  const _Float16* xin = reinterpret_cast<const _Float16*>(a.x);
  const _Float16* zr = reinterpret_cast<const _Float16*>(a.zeros);
  _Float16* yout = reinterpret_cast<_Float16*>(a.out);
  const _Float16* cI = reinterpret_cast<const _Float16*>(a.cI);
  const _Float16* sI = reinterpret_cast<const _Float16*>(a.sI);

  stage_table<NT>(sTw, LDV, 2 * Kbp, reinterpret_cast<const _Float16*>(a.twI), 2 * Kbp, NB64,
                  2 * Kbp);
  // leading-axis inverse factors for this wave's 16 rows, kept in registers
  h8 cf[NKZ], sf[NKZ];
  {
    const int row = wave * 16 + r16;
#pragma unroll
    for (int s = 0; s < NKZ; ++s) {
      const int col = s * KS + g * 8;
      const bool okc = row < a.Nap && col < a.Kap;
      cf[s] = MH::ld(okc ? cI + (int64_t)row * a.Kap + col : zr);
      sf[s] = MH::ld(okc ? sI + (int64_t)row * a.Kap + col : zr);
    }
  }

  const int64_t plane = (int64_t)a.Na * a.Nb;
  const int64_t zplane = (int64_t)a.Ka * a.Kb * 2;
  // the dispatcher guarantees Kb % 4 == 0: whole 16-byte groups of modes
  auto load_z = [&](int64_t p, u32x4 (&buf)[ZG][4]) {
    const bool pok = p < a.planes;  // unconditional loads, as in r2c
    const _Float16* base = zin + (pok ? p : 0) * zplane;
#pragma unroll
    for (int gi = 0; gi < ZG; ++gi) {
      const int gidx = threadIdx.x + NT * gi;
      const int tb4 = gidx % (Kbp / 4), ta4 = gidx / (Kbp / 4);
      const bool gok = gidx < ZGROUPS;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ta = ta4 * 4 + j;
        buf[gi][j] = load_modes16<_Float16, true>(zr, base + (int64_t)ta * a.Kb * 2, tb4 * 4,
                                                  a.Kb, pok && gok && ta < a.Ka);
      }
    }
  };
  // epilogue prefetch: row (lane >> 2) of this wave's tile, 16 columns of
  // every 64-column group
  constexpr int XR = EPI ? NBT : 1;
  const int orow = lane >> 2, ocol = (lane & 3) * 16;
  auto load_x = [&](int64_t p, u32x4 (&buf)[XR][2]) {
    if constexpr (EPI) {
      const bool pok = p < a.planes;
      const _Float16* base = xin + (pok ? p : 0) * plane;
      const int rr = wave * 16 + orow;
#pragma unroll
      for (int c = 0; c < NBT; ++c) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int col = c * 64 + ocol + h * 8;
          const bool ok = pok && rr < a.Na && col < a.Nb;
          buf[c][h] = *reinterpret_cast<const u32x4*>(ok ? base + (int64_t)rr * a.Nb + col : zr);
        }
      }
    }
  };

  auto process = [&](int64_t p, const u32x4 (&zc)[ZG][4], const u32x4 (&xc)[XR][2]) {
#pragma unroll
    for (int gi = 0; gi < ZG; ++gi) {
      const int gidx = threadIdx.x + NT * gi;
      if (gidx < ZGROUPS) {
        const int tb4 = gidx % (Kbp / 4), ta4 = gidx / (Kbp / 4);
        _Float16* d = ZTr + (tb4 * 4) * LDZ + ta4 * 4;
        scatter4<_Float16>(zc[gi], d, d + Kbp * LDZ, LDZ, false);
      }
    }
    block_sync_lds();
    // ---- step B': V^T[t_b][n] = sum_t Z^T[t_b][t] E[t][n], this wave's rows ----
    {
      f4 vr[NTB], vi[NTB];
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) vr[tb] = vi[tb] = f4zero();
#pragma unroll
      for (int s2 = 0; s2 < NKZ; ++s2) {
        h8 nsf = -sf[s2];
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
          const int zoff = (tb * 16 + r16) * LDZ + s2 * KS + g * 8;
          h8 zr_ = MH::ld(ZTr + zoff), zi_ = MH::ld(ZTi + zoff);
          vr[tb] = MH::mma(zr_, cf[s2], vr[tb]);
          vr[tb] = MH::mma(zi_, nsf, vr[tb]);
          vi[tb] = MH::mma(zr_, sf[s2], vi[tb]);
          vi[tb] = MH::mma(zi_, cf[s2], vi[tb]);
        }
      }
      // V rows are private to this wave: written and read back by it only
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        _Float16* dst = VL + (wave * 16 + r16) * LDV + tb * 16 + 4 * g;
        h4 wr, wi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          wr[i] = to_h(vr[tb][i]);
          wi[i] = to_h(vi[tb][i]);
        }
        *reinterpret_cast<h4*>(dst) = wr;
        *reinterpret_cast<h4*>(dst + Kbp) = wi;
      }
    }
    block_sync_lds();  // ZT reads done (the next plane may overwrite it); VL visible
    // ---- step A': y^T tiles = twI x VL^T, staged through obuf --------------------
    _Float16* yp = yout + p * plane;
#pragma unroll
    for (int c = 0; c < NBT; ++c) {
      f4 acc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] = f4zero();
#pragma unroll
      for (int k0 = 0; k0 < 2 * Kbp; k0 += KS) {
        h8 vf = MH::ld(VL + (wave * 16 + r16) * LDV + k0 + g * 8);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          h8 tf = MH::ld(sTw + ((c * 4 + u) * 16 + r16) * LDV + k0 + g * 8);
          acc[u] = MH::mma(tf, vf, acc[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        *reinterpret_cast<f4*>(obuf + r16 * 68 + u * 16 + 4 * g) = acc[u];
      wave_lds_sync();
      float v[16];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f4 t = *reinterpret_cast<const f4*>(obuf + orow * 68 + ocol + 4 * i);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[4 * i + e] = t[e] * a.scale;
      }
      wave_lds_sync();
      if constexpr (EPI) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          h8 xv = as_h8(xc[c][h]);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[8 * h + e] *= preact_grad_f32((float)xv[e], a.act, a.clip);
        }
      }
      const int n_a = wave * 16 + orow, n_b = c * 64 + ocol;
      if (n_a < a.Na && n_b < a.Nb) {
        const int nval = min(16, a.Nb - n_b);
        _Float16* dst = yp + (int64_t)n_a * a.Nb + n_b;
        if (nval == 16) {
          h8 o0, o1;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            o0[e] = to_h(v[e]);
            o1[e] = to_h(v[8 + e]);
          }
          *reinterpret_cast<h8*>(dst) = o0;
          *reinterpret_cast<h8*>(dst + 8) = o1;
        } else {
          for (int e = 0; e < nval; ++e) dst[e] = to_h(v[e]);
        }
      }
    }
  };

  // two planes ahead in flight, three buffer sets in fixed roles (see r2c)
  const int64_t G = gridDim.x;
  u32x4 z0[ZG][4], z1[ZG][4], z2[ZG][4];
  u32x4 x0[XR][2], x1[XR][2], x2[XR][2];
  int64_t p = blockIdx.x;
  load_z(p, z0);
  load_x(p, x0);
  load_z(p + G, z1);
  load_x(p + G, x1);
  block_sync_lds();  // tables staged
  for (; p < a.planes; p += 3 * G) {
    load_z(p + 2 * G, z2);
    load_x(p + 2 * G, x2);
    process(p, z0, x0);
    if (p + G >= a.planes) break;
    load_z(p + 3 * G, z0);
    load_x(p + 3 * G, x0);
    process(p + G, z1, x1);
    if (p + 2 * G >= a.planes) break;
    load_z(p + 4 * G, z1);
    load_x(p + 4 * G, x1);
    process(p + 2 * G, z2, x2);
  }
}

// ---------------------------------------------------------------------------
// Dispatch over the instantiated shapes.
// ---------------------------------------------------------------------------
size_t r2c_fast_lds_bytes(int nct, int nka, int nw, int Kap16, int Nap) {
  const int Kbp = nct * 8;
  return (size_t)2 * (2 * Kbp * (nka * KS + PADH) + 2 * Kap16 * (Nap + PADH) +
                      2 * Kbp * (16 * nw + PADH));
}

size_t c2r_fast_lds_bytes(int nct, int nw, int nbt, int nkz) {
  const int Kbp = nct * 8;
  const int LDV = 2 * Kbp + PADH;
  return (size_t)2 * (2 * Kbp * (nkz * KS + PADH) + 16 * nw * LDV + nbt * 64 * LDV) +
         (size_t)nw * 16 * 68 * 4;
}

#define FAST_LAUNCH(K)                                                                    \
  do {                                                                                    \
    auto k = K;                                                                           \
    if (lds > 65536) {                                                                    \
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),                \
                                         hipFuncAttributeMaxDynamicSharedMemorySize,      \
                                         (int)lds);                                       \
      if (e != hipSuccess) return e;                                                      \
    }                                                                                     \
    hipLaunchKernelGGL(k, dim3(grid), dim3(nw * 64), lds, s, a);                          \
    return hipGetLastError();                                                             \
  } while (0)

#define R2C_CASE(NCT_, NKA_, NW_) \
  if (nct == NCT_ && nka == NKA_ && nw == NW_) FAST_LAUNCH((r2c_fast_kernel<NCT_, NKA_, NW_>));

hipError_t launch_r2c_fast(const R2CArgs& a, int nct, int nka, int nw, int grid, size_t lds,
                           hipStream_t s) {
  R2C_CASE(2, 1, 4)
  R2C_CASE(2, 2, 4)
  R2C_CASE(2, 4, 4)
  R2C_CASE(2, 4, 8)
  R2C_CASE(4, 2, 4)
  R2C_CASE(4, 4, 4)
  R2C_CASE(4, 4, 8)
  R2C_CASE(4, 8, 4)
  R2C_CASE(8, 2, 4)
  R2C_CASE(8, 4, 8)
  return hipErrorNotSupported;
}

#define C2R_CASE(NCT_, NW_, NBT_, NKZ_)                                                  \
  if (nct == NCT_ && nw == NW_ && nbt == NBT_ && nkz == NKZ_) {                         \
    if (a.epilogue) FAST_LAUNCH((c2r_fast_kernel<NCT_, NW_, NBT_, NKZ_, true>));         \
    FAST_LAUNCH((c2r_fast_kernel<NCT_, NW_, NBT_, NKZ_, false>));                        \
  }

hipError_t launch_c2r_fast(const C2RArgs& a, int nct, int nw, int nbt, int nkz, int grid,
                           size_t lds, hipStream_t s) {
  C2R_CASE(2, 4, 1, 1)
  C2R_CASE(2, 4, 2, 1)
  C2R_CASE(2, 8, 2, 1)
  C2R_CASE(4, 4, 1, 1)
  C2R_CASE(4, 4, 2, 1)
  C2R_CASE(4, 8, 2, 2)
  C2R_CASE(4, 8, 2, 1)
  C2R_CASE(8, 4, 1, 2)
  C2R_CASE(8, 8, 2, 2)
  C2R_CASE(8, 8, 4, 2)
  return hipErrorNotSupported;
}

}  // namespace fno
