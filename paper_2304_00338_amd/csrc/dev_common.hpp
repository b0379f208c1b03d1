// Device helpers shared by the gfx950 kernels: MFMA operand traits, tile
// staging, row LayerNorm statistics and deterministic in-wave reductions.
//
// Every kernel works on tiles of TM = 32 rows (edges or nodes) with one
// wave64 per 16 latent columns: 8 waves (512 threads) for the latent width
// 128, 10 waves (640 threads) for the latent width 150 padded to 160.  Wave
// w owns output columns [16w, 16w+16) of every latent-wide layer.  MFMA 16x16xK operand layout (lane l, i = l & 15,
// q = l >> 4):
//   A fragment: A[i][k0 + q*KQ + j]   (KQ = 1 for fp32, 8 for bf16)
//   B fragment: B[k0 + q*KQ + j][i]
//   C/D:        c[r] = C[q*4 + r][i]
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mgn.h"

namespace mgn {
namespace dev {

constexpr int D = 128;     // latent width
constexpr int NT = 512;    // threads per block
constexpr int NW = 8;      // waves per block
constexpr int TM = 32;     // rows per tile
constexpr int NRB = TM / 16;

// Real latent width of a kernel width LD: the 3D model's latent 150 runs
// padded to 160 columns.  Padded weight rows and columns, biases, gains and
// offsets are zero, so padded feature columns stay exactly zero; only the
// LayerNorm statistics need the real width (and a mask on the padding).
template <int LD>
struct Width {
  static constexpr int DR = LD == 160 ? 150 : LD;
  static constexpr int NW = LD / 16;
  static constexpr int NT = NW * 64;
  static_assert(LD == 128 || LD == 160, "supported kernel widths: 128, 160");
};

// Host-side dispatch on the kernel width lat (128, or 160 for the latent
// 150): F(LD) expands to the launch of the width-LD instantiation.
#define MGN_BY_WIDTH(lat, F) \
  do {                       \
    if ((lat) == 160)        \
      F(160);                \
    else                     \
      F(128);                \
  } while (0)

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int PREC>
struct Tr;

template <>
struct Tr<MGN_FP32> {
  typedef float T;
  typedef float Frag;
  static constexpr int KS = 4;   // K per MFMA
  static constexpr int PAD = 4;  // LDS row padding (elements)
  static __device__ __forceinline__ f32x4 mma(Frag a, Frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // A[row0 + i][k0 + q] from a row-major LDS tile
  static __device__ __forceinline__ Frag lda(const T* t, int ld, int row0, int k0, int i, int q) {
    return t[(row0 + i) * ld + k0 + q];
  }
  // B[k][n] = W[n0 + n][k] from a row-major [n][k] matrix
  static __device__ __forceinline__ Frag ldb(const T* W, int ldw, int n0, int k0, int i, int q) {
    return W[(size_t)(n0 + i) * ldw + k0 + q];
  }
  static __device__ __forceinline__ T cvt(float x) { return x; }
};

template <>
struct Tr<MGN_BF16> {
  typedef bf16 T;
  typedef bf16x8 Frag;
  static constexpr int KS = 32;
  static constexpr int PAD = 8;
  static __device__ __forceinline__ f32x4 mma(Frag a, Frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Frag lda(const T* t, int ld, int row0, int k0, int i, int q) {
    return *reinterpret_cast<const bf16x8*>(t + (row0 + i) * ld + k0 + q * 8);
  }
  static __device__ __forceinline__ Frag ldb(const T* W, int ldw, int n0, int k0, int i, int q) {
    return *reinterpret_cast<const bf16x8*>(W + (size_t)(n0 + i) * ldw + k0 + q * 8);
  }
  static __device__ __forceinline__ T cvt(float x) { return (bf16)x; }
};

__device__ __forceinline__ float tof(float x) { return x; }
__device__ __forceinline__ float tof(bf16 x) { return (float)x; }

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

// acc[rb] += A[rb*16 .. +16][0..K) * B, B[k][n] = W[n0 + n][kofs + k].
template <int PREC, int K>
__device__ __forceinline__ void gemm_tile(f32x4 (&acc)[NRB], const typename Tr<PREC>::T* A, int lda,
                                          const typename Tr<PREC>::T* W, int ldw, int n0, int kofs,
                                          int i, int q) {
  typedef Tr<PREC> P;
#pragma unroll 4
  for (int k0 = 0; k0 < K; k0 += P::KS) {
    const typename P::Frag b = P::ldb(W, ldw, n0, kofs + k0, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = P::mma(P::lda(A, lda, rb * 16, k0, i, q), b, acc[rb]);
  }
}

// acc[cb] += sum over the tile's rows of G[row][o] * X[row][xcol0 + cb*16 + n]
// where G arrives in C layout (g[rb][r] = G[rb*16 + q*4 + r][o = 16w + i]).
// The MFMA's K dimension runs over tile rows; the row order inside K is a
// fixed permutation applied to both operands.
template <int NCB>
__device__ __forceinline__ void gtx_f32(f32x4 (&acc)[NCB], const f32x4 (&g)[NRB], const float* X, int ldx, int xcol0,
                                        int i, int q) {
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = g[rb][r];
      const float* xr = X + (rb * 16 + q * 4 + r) * ldx + xcol0 + i;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, xr[cb * 16], acc[cb], 0, 0, 0);
    }
}

template <int NCB>
__device__ __forceinline__ void gtx_bf16(f32x4 (&acc)[NCB], const f32x4 (&g)[NRB], const bf16* X, int ldx,
                                         int xcol0, int i, int q) {
#pragma unroll
  for (int t = 0; t < NRB / 2; ++t) {
    bf16x8 a;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      a[j] = (bf16)g[2 * t][j];
      a[4 + j] = (bf16)g[2 * t + 1][j];
    }
    const bf16* x0 = X + ((2 * t) * 16 + q * 4) * ldx + xcol0 + i;
    const bf16* x1 = X + ((2 * t + 1) * 16 + q * 4) * ldx + xcol0 + i;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      bf16x8 b;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        b[j] = x0[j * ldx + cb * 16];
        b[4 + j] = x1[j * ldx + cb * 16];
      }
      acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[cb], 0, 0, 0);
    }
  }
}

template <int PREC, int NCB>
__device__ __forceinline__ void gtx(f32x4 (&acc)[NCB], const f32x4 (&g)[NRB], const typename Tr<PREC>::T* X, int ldx,
                                    int xcol0, int i, int q) {
  if constexpr (PREC == MGN_BF16)
    gtx_bf16<NCB>(acc, g, X, ldx, xcol0, i, q);
  else
    gtx_f32<NCB>(acc, g, X, ldx, xcol0, i, q);
}

// Sum over the 16 lanes that share q (one DPP row = one row of a 16-column
// block): rotate-and-add within the row by 8, 4, 2, 1 lanes, so every lane
// ends with the same total, formed in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float sum16(float s) {
  s += dpp_f<0x128>(s);  // row_ror:8
  s += dpp_f<0x124>(s);  // row_ror:4
  s += dpp_f<0x122>(s);  // row_ror:2
  s += dpp_f<0x121>(s);  // row_ror:1
  return s;
}
// sum16 of all 4*NRB values of a C-layout tile, one rotation step at a time
// so that independent DPP operations fill each other's wait states.  Same
// order of additions per value as sum16.
__device__ __forceinline__ void sum16x(f32x4 (&v)[NRB]) {
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[rb][r] += dpp_f<0x128>(v[rb][r]);
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[rb][r] += dpp_f<0x124>(v[rb][r]);
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[rb][r] += dpp_f<0x122>(v[rb][r]);
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[rb][r] += dpp_f<0x121>(v[rb][r]);
}

// Sum over the four q groups (lanes i, i+16, i+32, i+48): the pair sums of
// lanes l, l ^ 16 and then l, l ^ 32 with gfx950's row swaps
// (v_permlane16_swap / v_permlane32_swap of a value with itself hand every
// lane both members of its pair, lower row first), on the VALU instead of
// an LDS permute.  Each pair sum adds the same two values as s + s[l ^ k].
__device__ __forceinline__ float sum_q(float s) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(s), __float_as_uint(s), false, false);
  s = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// LDS scratch of the row LayerNorm helpers for NWV waves.  red/red2/red2x
// hold one partial per (row, wave); fin holds, per wave, the 32 row totals
// that wave formed itself (so reading them back needs no block barrier).
template <int NWV>
struct alignas(16) LnScratch {
  float red[TM][NWV];
  float red2[TM][NWV];
  float red2x[TM][NWV][2];
  float fin[NWV][2 * TM];
};

// Orders this wave's LDS writes before its later LDS reads of other lanes'
// data (LDS requests of one wave are served in issue order).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sum of the NWV per-wave partials of one row in wave order.
template <int NWV>
__device__ __forceinline__ float row_total(const float* p) {
  if constexpr (NWV == 8) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
    return ((((((a[0] + a[1]) + a[2]) + a[3]) + b[0]) + b[1]) + b[2]) + b[3];
  } else {
    float t = p[0];
#pragma unroll
    for (int u = 1; u < NWV; ++u) t += p[u];
    return t;
  }
}

// Per-row mean and 1/sqrt(var + eps) over the real latent columns held by
// the NWV waves (biased variance, two passes; padded columns are left out).
// Each wave reduces its 16 columns with DPP, the wave partials of a row are
// summed once per wave by lane row (lanes 0..31) and handed back through the
// wave's own LDS slot.  Contains two block barriers; every thread of the
// block must call it.
template <int NWV>
__device__ __forceinline__ void ln_stats(const f32x4 (&v)[NRB], LnScratch<NWV>& S, float eps, int w, int i, int q,
                                         f32x4 (&mean)[NRB], f32x4 (&rstd)[NRB]) {
  constexpr int LD = NWV * 16, DR = Width<LD>::DR;
  const int lane = threadIdx.x & 63;
  float* fin = S.fin[w];
  {
    f32x4 s[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) s[rb] = v[rb];
    sum16x(s);
    if (i == 0)
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) S.red[rb * 16 + q * 4 + r][w] = s[rb][r];
  }
  __syncthreads();
  if (lane < TM) fin[lane] = row_total<NWV>(S.red[lane]) * (1.0f / DR);
  wave_lds_sync();
  {
    const bool live = DR == LD || w * 16 + i < DR;
    f32x4 s[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      mean[rb] = *reinterpret_cast<const f32x4*>(fin + rb * 16 + q * 4);
      const f32x4 d = v[rb] - mean[rb];
      s[rb] = live ? d * d : zero4();
    }
    sum16x(s);
    if (i == 0)
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) S.red2[rb * 16 + q * 4 + r][w] = s[rb][r];
  }
  __syncthreads();
  if (lane < TM) fin[TM + lane] = __builtin_amdgcn_rsqf(row_total<NWV>(S.red2[lane]) * (1.0f / DR) + eps);
  wave_lds_sync();
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) rstd[rb] = *reinterpret_cast<const f32x4*>(fin + TM + rb * 16 + q * 4);
}

// LayerNorm backward for one tile: given dy (C layout), xhat, rstd and this
// lane's gain, returns dz = rstd * (dxh - mean(dxh) - xhat * mean(dxh*xhat))
// with dxh = dy * gamma, the means over the real columns (a padded column's
// gain is zero) and dz = 0 on padded columns.  One block barrier.
template <int NWV>
__device__ __forceinline__ void ln_bwd(f32x4 (&dz)[NRB], const f32x4 (&dy)[NRB], const f32x4 (&xhat)[NRB],
                                       const f32x4 (&rstd)[NRB], float gam, LnScratch<NWV>& S, int w, int i, int q) {
  constexpr int LD = NWV * 16, DR = Width<LD>::DR;
  const int lane = threadIdx.x & 63;
  float* fin = S.fin[w];
  {
    f32x4 s1[NRB], s2[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      s1[rb] = dy[rb] * gam;
      s2[rb] = s1[rb] * xhat[rb];
    }
    sum16x(s1);
    sum16x(s2);
    if (i == 0)
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          S.red2x[rb * 16 + q * 4 + r][w][0] = s1[rb][r];
          S.red2x[rb * 16 + q * 4 + r][w][1] = s2[rb][r];
        }
  }
  __syncthreads();
  if (lane < TM) {
    const f32x4* p = reinterpret_cast<const f32x4*>(S.red2x[lane]);
    float t1 = 0.f, t2 = 0.f;
#pragma unroll
    for (int u = 0; u < NWV / 2; ++u) {
      const f32x4 x = p[u];
      t1 += x[0];
      t2 += x[1];
      t1 += x[2];
      t2 += x[3];
    }
    fin[lane] = t1 * (1.0f / DR);
    fin[TM + lane] = t2 * (1.0f / DR);
  }
  wave_lds_sync();
  const bool live = DR == LD || w * 16 + i < DR;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const f32x4 m1 = *reinterpret_cast<const f32x4*>(fin + rb * 16 + q * 4);
    const f32x4 m2 = *reinterpret_cast<const f32x4*>(fin + TM + rb * 16 + q * 4);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float dxh = dy[rb][r] * gam;
      dz[rb][r] = live ? rstd[rb][r] * (dxh - m1[r] - xhat[rb][r] * m2[r]) : 0.f;
    }
  }
}

// Copy rows [0, nrows) of a row-major global [.][LD] array (element type S)
// into an LDS tile of T with row stride ld, zero-filling rows nrows..TM-1.
// Each thread moves 8 consecutive elements per step.
template <int LD, typename T, typename S>
__device__ __forceinline__ void stage_rows(T* lds, int ld, const S* src, int nrows, int tid) {
  constexpr int CPR = LD / 8, NTH = Width<LD>::NT;
  for (int idx = tid; idx < TM * CPR; idx += NTH) {
    const int row = idx / CPR, c = (idx % CPR) * 8;
    T* dst = lds + row * ld + c;
    float v[8];
    if (row < nrows) {
      const S* s = src + (size_t)row * LD + c;
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = tof(s[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[j] = (T)v[j];
  }
}

}  // namespace dev
}  // namespace mgn
