// Fused edge-phase kernels of one MGN message-passing step on gfx950, forward
// and reverse (Sec. 2.1: every edge is updated from its incident nodes, then
// every node from the sum of its incident edge messages), in the
// feature-split layout, fp32 at the latent widths 128 and 160 (bf16 runs on
// the row-per-wave kernels).
//
// Both kernels are persistent: block b handles the receiver-aligned tiles
// b, b+G, b+2G, ...  While a tile is computed, the block already has the
// next tile's streams in flight in registers (edge latents, gathered node
// products, and in reverse mode the incoming edge gradient and the gathered
// aggregate gradient); the tile after that has its sender/receiver ids in
// flight, and the one after that its descriptor.  Weight fragments are read
// from the cache per use.
//
// The first edge-MLP layer is evaluated as W1e e + P_s[s] + P_r[r] with the
// node products P = [W1s h, W1r h] computed per node (same linear map as
// W1 [e, h_s, h_r]; only the fp32 summation order differs).
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

// A zero the compiler cannot see through: weight-fragment reads offset by a
// fresh one per tile are not loop-invariant, so they are not hoisted out of
// the tile loop into registers (which spills at width 160, where a 10-wave
// block leaves a wave 168 registers).
__device__ __forceinline__ int tile_opaque_zero() {
  int z = 0;
  asm volatile("" : "+v"(z));
  return z;
}

// B fragments of one 16-column weight slice with K = LD (the kernel width),
// B[k][n] = W[n0 + n][kofs + k], read from the cache per use; refresh()
// starts a tile.
template <int PREC, int LD>
struct WSlice {
  typedef Tr<PREC> P;
  static constexpr int NK = LD / P::KS;
  const typename P::T* W;
  int ldw, n0, kofs, i, q, z = 0;
  __device__ __forceinline__ void init(const typename P::T* W_, int ldw_, int n0_, int kofs_, int i_, int q_) {
    W = W_;
    ldw = ldw_;
    n0 = n0_;
    kofs = kofs_;
    i = i_;
    q = q_;
  }
  __device__ __forceinline__ typename P::Frag get(int kk) const {
    return P::ldb(W, ldw, n0, kofs + z + kk * P::KS, i, q);
  }
  __device__ __forceinline__ void refresh() { z = tile_opaque_zero(); }
};

template <int PREC, class WSL>
__device__ __forceinline__ void gemm_w(f32x4 (&acc)[NRB], const typename Tr<PREC>::T* A, int lda, const WSL& w,
                                       int i, int q) {
  typedef Tr<PREC> P;
#pragma unroll
  for (int kk = 0; kk < WSL::NK; ++kk) {
    const typename P::Frag b = w.get(kk);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = P::mma(P::lda(A, lda, rb * 16, kk * P::KS, i, q), b, acc[rb]);
  }
}

// Row-chunk geometry: 16-byte chunks of LD-wide rows of element type T,
// split over the LD * 4 threads of a block.
template <typename T, int LD>
struct Rows {
  static constexpr int NTH = Width<LD>::NT;
  static constexpr int EPC = 16 / sizeof(T);          // elements per chunk
  static constexpr int CPR = LD / EPC;                // chunks per row
  static constexpr int CPT = TM * CPR / NTH;          // chunks per thread per tile
  static_assert(CPT >= 1 && TM * CPR == CPT * NTH, "tile must split evenly");
  __device__ __forceinline__ static int row(int tid, int k) { return (tid + k * NTH) / CPR; }
  __device__ __forceinline__ static int col(int tid, int k) { return ((tid + k * NTH) % CPR) * EPC; }
};

__device__ __forceinline__ void unpack(const uint4& u, float (&f)[4]) {
  f[0] = __uint_as_float(u.x);
  f[1] = __uint_as_float(u.y);
  f[2] = __uint_as_float(u.z);
  f[3] = __uint_as_float(u.w);
}
__device__ __forceinline__ void unpack(const uint4& u, float (&f)[8]) {
  const bf16* b = reinterpret_cast<const bf16*>(&u);
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)b[j];
}

// Position of the first row of the tile whose receiver is >= v (rows are
// receiver-sorted).
__device__ __forceinline__ int first_row(const int2* sr, int n, int v) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (sr[mid].y < v)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// Sum of in-tile rows per receiver (ascending in-segment order), or of all
// rows into a slot for a chunk of a long segment.
template <int LD, typename S>
__device__ __forceinline__ void segment_sums(const S* rows, int ld, const int2* sr, int4 td, float* __restrict__ out,
                                             float* __restrict__ slots, int tid) {
  constexpr int D = LD, NT = Width<LD>::NT;
  const int c = tid % D, vg = tid / D;
  const int nb = td.x, ne_ = td.w - td.z;
  if (td.y >= 0) {
    const int nv = td.y - nb;
    for (int j = vg; j < nv; j += NT / D) {
      const int a = first_row(sr, ne_, nb + j), b = first_row(sr, ne_, nb + j + 1);
      float s = 0.f;
      for (int u = a; u < b; ++u) s += tof(rows[u * ld + c]);
      out[(size_t)(nb + j) * D + c] = s;
    }
  } else if (vg == 0) {
    float s = 0.f;
    for (int u = 0; u < ne_; ++u) s += tof(rows[u * ld + c]);
    slots[(size_t)(-1 - td.y) * D + c] = s;
  }
}

__device__ __forceinline__ int4 tile_or_zero(const int4* tiles, int64_t t, int64_t n) {
  const int4 z = {0, 0, 0, 0};
  return t < n ? tiles[t] : z;
}

__device__ __forceinline__ int2 sr_of(const EdgeTiles& tl, int4 d, int row) {
  int2 v = {0, 0};
  if (row < d.w - d.z) {
    v.x = tl.senders[d.z + row];
    v.y = tl.receivers[d.z + row];
  }
  return v;
}

// ===================================================================== forward
template <int PREC, int LD>
struct FwdLoads {
  typedef Rows<typename Tr<PREC>::T, LD> RT;
  uint4 e[RT::CPT], ps[RT::CPT], pr[RT::CPT];
};

template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) __attribute__((amdgpu_waves_per_eu(LD == 128 ? 2 : 3, LD == 128 ? 2 : 3)))
k_edge_fwd(EdgeTiles tl, const typename Tr<PREC>::T* __restrict__ e_in,
                                                 typename Tr<PREC>::T* __restrict__ e_out, int write_e,
                                                 const typename Tr<PREC>::T* __restrict__ Pn, MlpW w, float eps,
                                                 float* __restrict__ agg, float* __restrict__ slots) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  typedef Rows<T, LD> RT;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;
  constexpr int LDT = D + P::PAD;
  constexpr int LDM = D + 4;
  constexpr int A1B = TM * LDT * (int)sizeof(T);
  constexpr int MB = TM * LDM * 4;
  __shared__ __align__(16) T sE[TM * LDT];
  __shared__ __align__(16) float sP[TM * LDM];
  __shared__ __align__(16) char sU[A1B > MB ? A1B : MB];  // a1 tile, then m tile
  __shared__ LnScratch<NW> ln;
  __shared__ int2 sSR[2][TM];
  T* sA1 = reinterpret_cast<T*>(sU);
  float* sM = reinterpret_cast<float*>(sU);

  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n], b2 = w.b2[n], gam = w.gamma[n], bet = w.beta[n];
  WSlice<PREC, LD> w1, w2;
  w1.init((const T*)w.W1, 3 * D, w8 * 16, 0, i, q);
  w2.init((const T*)w.W2, D, w8 * 16, 0, i, q);

  const int64_t G = gridDim.x, NTL = tl.n_tiles;
  int64_t t = blockIdx.x;
  if (t >= NTL) return;
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  int4 d0 = tiles[t];
  int4 d1 = tile_or_zero(tiles, t + G, NTL);
  int4 d2 = tile_or_zero(tiles, t + 2 * G, NTL);
  if (tid < TM) sSR[0][tid] = sr_of(tl, d0, tid);
  int2 srn = {0, 0};
  if (tid < TM) srn = sr_of(tl, d1, tid);
  __syncthreads();

  FwdLoads<PREC, LD> L;
  auto issue = [&](int4 d, const int2* sr) {
    const int ne_ = d.w - d.z;
    const uint4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) L.e[k] = L.ps[k] = L.pr[k] = z;
    if (ne_ <= 0) return;
    const T* et = e_in + (size_t)d.z * D;
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      const int rc = min(row, ne_ - 1);
      const int2 v = sr[rc];
      const uint4 a = *reinterpret_cast<const uint4*>(et + (uint32_t)(rc * D + col));
      const uint4 b = *reinterpret_cast<const uint4*>(Pn + (uint32_t)(v.x * (2 * D) + col));
      const uint4 c = *reinterpret_cast<const uint4*>(Pn + (uint32_t)(v.y * (2 * D) + D + col));
      const bool ok = row < ne_;
      L.e[k] = ok ? a : z;
      L.ps[k] = ok ? b : z;
      L.pr[k] = ok ? c : z;
    }
  };
  issue(d0, sSR[0]);
  int buf = 0;
  for (; t < NTL; t += G) {
    if constexpr (LD == 160) {
      w1.refresh();
      w2.refresh();
    }
    // ---- commit the prefetched streams of tile t to LDS
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      *reinterpret_cast<uint4*>(sE + row * LDT + col) = L.e[k];
      float a[RT::EPC], b[RT::EPC];
      unpack(L.ps[k], a);
      unpack(L.pr[k], b);
#pragma unroll
      for (int j = 0; j < RT::EPC; ++j) sP[row * LDM + col + j] = a[j] + b[j];
    }
    if (tid < TM) sSR[buf ^ 1][tid] = srn;
    __syncthreads();
    // ---- put the next tiles in flight
    const int4 d3 = tile_or_zero(tiles, t + 3 * G, NTL);
    if (t + G < NTL) issue(d1, sSR[buf ^ 1]);
    srn = tid < TM ? sr_of(tl, d2, tid) : int2{0, 0};

    // ---- compute tile t
    const int ne_ = d0.w - d0.z, eb = d0.z;
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[rb][r] = b1 + sP[(rb * 16 + q * 4 + r) * LDM + n];
    gemm_w<PREC>(acc, sE, LDT, w1, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) sA1[(rb * 16 + q * 4 + r) * LDT + n] = P::cvt(fmaxf(acc[rb][r], 0.f));
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b2, b2, b2, b2};
    gemm_w<PREC>(acc, sA1, LDT, w2, i, q);
    f32x4 mean[NRB], rstd[NRB];
    ln_stats(acc, ln, eps, w8, i, q, mean, rstd);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sM[(rb * 16 + q * 4 + r) * LDM + n] = gam * ((acc[rb][r] - mean[rb][r]) * rstd[rb][r]) + bet;
    __syncthreads();
    if (write_e) {
      for (int idx = tid; idx < ne_ * RT::CPR; idx += NT) {
        const int row = idx / RT::CPR, col = (idx % RT::CPR) * RT::EPC;
        float a[RT::EPC];
        unpack(*reinterpret_cast<const uint4*>(sE + row * LDT + col), a);
        uint4 o;
        T* ot = reinterpret_cast<T*>(&o);
#pragma unroll
        for (int j = 0; j < RT::EPC; ++j) ot[j] = P::cvt(a[j] + sM[row * LDM + col + j]);
        *reinterpret_cast<uint4*>(e_out + (size_t)(eb + row) * D + col) = o;
      }
    }
    segment_sums<LD>(sM, LDM, sSR[buf], d0, agg, slots, tid);
    __syncthreads();
    d0 = d1;
    d1 = d2;
    d2 = d3;
    buf ^= 1;
  }
}

// ===================================================================== reverse
template <int PREC, int LD>
struct BwdLoads {
  typedef Rows<typename Tr<PREC>::T, LD> RT;
  uint4 e[RT::CPT], ps[RT::CPT], pr[RT::CPT];
};

// Given ebar_in = dL/de_out (absent for the last block) and aggbar:
// mbar = ebar_in + aggbar[receiver]; back through LayerNorm and the MLP to
// zbar = dL/dz1 (written out; the sender sums and dW1e = sum zbar e^T are
// taken by later kernels) and its per-receiver sums R; ebar_out = ebar_in +
// W1e^T zbar; per-block partials of db1, dW2, db2, dgamma, dbeta.
// No global load is waited on inside a tile's compute apart from this
// tile's own gradient rows, which are issued before the next tile's prefetch
// (vector-memory loads retire in issue order): the forward weights sit in
// registers and, in bf16, the transposed ones in LDS.
template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) __attribute__((amdgpu_waves_per_eu(LD == 128 ? 2 : 3, LD == 128 ? 2 : 3)))
k_edge_bwd(EdgeTiles tl, const typename Tr<PREC>::T* __restrict__ e, const float* __restrict__ ebar_in,
           int have_ebar, float* __restrict__ ebar_out, const typename Tr<PREC>::T* __restrict__ Pn,
           const float* __restrict__ aggbar, MlpW w, float eps, typename Tr<PREC>::T* __restrict__ zbar,
           float* __restrict__ R, float* __restrict__ slots, Partials part) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  typedef Rows<T, LD> RT;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;
  constexpr int LDT = D + P::PAD;
  constexpr int LDM = D + 4;
  __shared__ __align__(16) T sE[TM * LDT];
  __shared__ __align__(16) float sP[TM * LDM];
  __shared__ __align__(16) T sA1[TM * LDT];
  __shared__ __align__(16) T sG[TM * LDT];
  __shared__ __align__(16) T sZ[TM * LDT];
  __shared__ LnScratch<NW> ln;
  __shared__ int2 sSR[2][TM];

  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n], b2 = w.b2[n], gam = w.gamma[n];
  WSlice<PREC, LD> w1, w2;
  w1.init((const T*)w.W1, 3 * D, w8 * 16, 0, i, q);
  w2.init((const T*)w.W2, D, w8 * 16, 0, i, q);
  WSlice<PREC, LD> g2t, g1t;
  g2t.init((const T*)w.W2t, D, w8 * 16, 0, i, q);
  g1t.init((const T*)w.W1t, D, w8 * 16, 0, i, q);
  f32x4 dW2[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dW2[cb] = zero4();
  float db1 = 0.f, db2 = 0.f, dg = 0.f, dbt = 0.f;

  const int64_t G = gridDim.x, NTL = tl.n_tiles;
  int64_t t = blockIdx.x;
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  int4 d0 = tile_or_zero(tiles, t, NTL);
  int4 d1 = tile_or_zero(tiles, t + G, NTL);
  int4 d2 = tile_or_zero(tiles, t + 2 * G, NTL);
  if (tid < TM) sSR[0][tid] = sr_of(tl, d0, tid);
  int2 srn = {0, 0};
  if (tid < TM) srn = sr_of(tl, d1, tid);
  __syncthreads();

  // Prefetch of one tile's edge latents and node products: 32-bit element
  // offsets from uniform bases; rows past the tile's end are clamped to its
  // last row and zeroed afterwards.
  BwdLoads<PREC, LD> L;
  auto issue = [&](int4 d, const int2* sr) {
    const int ne_ = d.w - d.z;
    const uint4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) L.e[k] = L.ps[k] = L.pr[k] = z;
    if (ne_ <= 0) return;
    const T* et = e + (size_t)d.z * D;
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      const int rc = min(row, ne_ - 1);
      const int2 v = sr[rc];
      const uint4 a = *reinterpret_cast<const uint4*>(et + (uint32_t)(rc * D + col));
      const uint4 b = *reinterpret_cast<const uint4*>(Pn + (uint32_t)(v.x * (2 * D) + col));
      const uint4 c = *reinterpret_cast<const uint4*>(Pn + (uint32_t)(v.y * (2 * D) + D + col));
      const bool ok = row < ne_;
      L.e[k] = ok ? a : z;
      L.ps[k] = ok ? b : z;
      L.pr[k] = ok ? c : z;
    }
  };
  if (t < NTL) issue(d0, sSR[0]);
  int buf = 0;
  for (; t < NTL; t += G) {
    if constexpr (LD == 160) {
      w1.refresh();
      w2.refresh();
      g1t.refresh();
      g2t.refresh();
    }
    // ---- commit tile t
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      *reinterpret_cast<uint4*>(sE + row * LDT + col) = L.e[k];
      float a[RT::EPC], b[RT::EPC];
      unpack(L.ps[k], a);
      unpack(L.pr[k], b);
#pragma unroll
      for (int j = 0; j < RT::EPC; ++j) sP[row * LDM + col + j] = a[j] + b[j];
    }
    if (tid < TM) sSR[buf ^ 1][tid] = srn;
    __syncthreads();
    // this tile's incoming edge gradient and gathered aggregate gradient (C layout)
    const int ne_ = d0.w - d0.z, eb = d0.z;
    f32x4 eb_in[NRB], mb[NRB];
    {
      const float* ebt = ebar_in + (size_t)eb * D;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rb * 16 + q * 4 + r;
          const int rc = max(0, min(row, ne_ - 1));
          const bool ok = row < ne_;
          float ag = 0.f, eo = 0.f;
          if (ne_ > 0) ag = aggbar[(uint32_t)(sSR[buf][rc].y * D + n)];
          if (have_ebar && ne_ > 0) eo = ebt[(uint32_t)(rc * D + n)];
          eb_in[rb][r] = ok ? eo : 0.f;
          mb[rb][r] = ok ? eo + ag : 0.f;
        }
    }
    const int4 d3 = tile_or_zero(tiles, t + 3 * G, NTL);
    if (t + G < NTL) issue(d1, sSR[buf ^ 1]);
    srn = tid < TM ? sr_of(tl, d2, tid) : int2{0, 0};

    // ---- recompute the forward edge MLP
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[rb][r] = b1 + sP[(rb * 16 + q * 4 + r) * LDM + n];
    gemm_w<PREC>(acc, sE, LDT, w1, i, q);
    uint32_t mask = 0;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (acc[rb][r] > 0.f) mask |= 1u << (rb * 4 + r);
        sA1[(rb * 16 + q * 4 + r) * LDT + n] = P::cvt(fmaxf(acc[rb][r], 0.f));
      }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b2, b2, b2, b2};
    gemm_w<PREC>(acc, sA1, LDT, w2, i, q);
    f32x4 rstd[NRB];
    {
      f32x4 mean[NRB];
      ln_stats(acc, ln, eps, w8, i, q, mean, rstd);
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) acc[rb] = (acc[rb] - mean[rb]) * rstd[rb];  // xhat
    }
    // ---- LayerNorm backward
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dg += mb[rb][r] * acc[rb][r];
        dbt += mb[rb][r];
      }
    f32x4 g[NRB];
    ln_bwd(g, mb, acc, rstd, gam, ln, w8, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        db2 += g[rb][r];
        sG[(rb * 16 + q * 4 + r) * LDT + n] = P::cvt(g[rb][r]);
      }
    gtx<PREC, NCB>(dW2, g, sA1, LDT, 0, i, q);
    __syncthreads();
    // ---- back through W2 and the ReLU
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = zero4();
    gemm_w<PREC>(acc, sG, LDT, g2t, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float z = (mask >> (rb * 4 + r)) & 1u ? acc[rb][r] : 0.f;
        db1 += z;
        sZ[(rb * 16 + q * 4 + r) * LDT + n] = P::cvt(z);
      }
    __syncthreads();
    // ---- back through W1e: ebar_out = ebar_in + W1e^T zbar
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = eb_in[rb];
    gemm_w<PREC>(acc, sZ, LDT, g1t, i, q);
    float* ebo = ebar_out + (size_t)eb * D;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        if (row < ne_) ebo[(uint32_t)(row * D + n)] = acc[rb][r];
      }
    for (int idx = tid; idx < ne_ * RT::CPR; idx += NT) {
      const int row = idx / RT::CPR, col = (idx % RT::CPR) * RT::EPC;
      *reinterpret_cast<uint4*>(zbar + (size_t)(eb + row) * D + col) =
          *reinterpret_cast<const uint4*>(sZ + row * LDT + col);
    }
    segment_sums<LD>(sZ, LDT, sSR[buf], d0, R, slots, tid);
    __syncthreads();
    d0 = d1;
    d1 = d2;
    d2 = d3;
    buf ^= 1;
  }
  // partial layout: the edge-MLP parameters after W1 (b1, W2, b2, gamma,
  // beta) at offset D * D
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) base[D * D + D + (size_t)(w8 * 16 + q * 4 + r) * D + cb * 16 + i] = dW2[cb][r];
  db1 = sum_q(db1);
  db2 = sum_q(db2);
  dg = sum_q(dg);
  dbt = sum_q(dbt);
  if (q == 0) {
    base[D * D + n] = db1;
    base[2 * D * D + D + n] = db2;
    base[2 * D * D + 2 * D + n] = dg;
    base[2 * D * D + 3 * D + n] = dbt;
  }
}

// Weight gradient of a linear map over edges: dW[o][i] = sum over rows of
// G[row][o] X[row][i] for two row-major [M][128] operand-precision streams
// (here G = zbar, X = the block input edge latents, so dW is the gradient of
// the edge MLP's first layer with respect to its edge-latent part).  Rows
// are taken 32 at a time in order; both chunks are staged feature-major in
// LDS so each MFMA operand fragment is one 16-byte (bf16) read, and the next
// chunk is in flight in registers while the current one is multiplied.
template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) __attribute__((amdgpu_waves_per_eu(LD == 128 ? 2 : 3, LD == 128 ? 2 : 3)))
k_wgrad(int64_t M, const typename Tr<PREC>::T* __restrict__ Gm, const typename Tr<PREC>::T* __restrict__ Xm,
        Partials part) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  typedef Rows<T, LD> RT;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;

  constexpr int LDF = TM + 8;  // feature-major row stride (elements)
  __shared__ __align__(16) T sGT[D * LDF];
  __shared__ __align__(16) T sXT[D * LDF];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  f32x4 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = zero4();
  const int64_t nch = (M + TM - 1) / TM, G = gridDim.x;
  uint4 lg[RT::CPT], lx[RT::CPT];
  auto issue = [&](int64_t c) {
    const int64_t r0 = c * TM;
    const int nr = (int)min((int64_t)TM, M - r0);
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      const int rc = min(row, nr - 1);
      const uint4 z = {0u, 0u, 0u, 0u};
      const uint4 a = *reinterpret_cast<const uint4*>(Gm + (size_t)(r0 + rc) * D + col);
      const uint4 b = *reinterpret_cast<const uint4*>(Xm + (size_t)(r0 + rc) * D + col);
      lg[k] = row < nr ? a : z;
      lx[k] = row < nr ? b : z;
    }
  };
  int64_t c = blockIdx.x;
  if (c < nch) issue(c);
  for (; c < nch; c += G) {
#pragma unroll
    for (int k = 0; k < RT::CPT; ++k) {
      const int row = RT::row(tid, k), col = RT::col(tid, k);
      const T* gv = reinterpret_cast<const T*>(&lg[k]);
      const T* xv = reinterpret_cast<const T*>(&lx[k]);
#pragma unroll
      for (int j = 0; j < RT::EPC; ++j) {
        sGT[(col + j) * LDF + row] = gv[j];
        sXT[(col + j) * LDF + row] = xv[j];
      }
    }
    __syncthreads();
    if (c + G < nch) issue(c + G);
    // A[o][k] = G[row k][o], B[k][n] = X[row k][n], K = the chunk's 32 rows
#pragma unroll
    for (int k0 = 0; k0 < TM; k0 += P::KS) {
      const typename P::Frag a = P::ldb(sGT, LDF, w8 * 16, k0, i, q);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[cb] = P::mma(a, P::ldb(sXT, LDF, cb * 16, k0, i, q), acc[cb]);
    }
    __syncthreads();
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) base[(size_t)(w8 * 16 + q * 4 + r) * D + cb * 16 + i] = acc[cb][r];
}

}  // namespace dev

// ============================================================ launchers
using namespace dev;

static constexpr int kEdgeFwdBlocks = 512;
static constexpr int kEdgeBwdBlocks = 256;
static constexpr int kWgradBlocks = 512;

hipError_t launch_edge_fwd(int prec, int lat, const EdgeTiles& t, const void* e_in, void* e_out, int write_e,
                           const void* Pn, const MlpW& w, float eps, float* agg, float* slots, void* a1_out,
                           hipStream_t s) {
  // bf16: the row-per-wave kernels
  if (prec == MGN_BF16 && lat == 128)
    return launch_edge_fwd_rows(t, e_in, e_out, write_e, Pn, w, eps, agg, slots, a1_out, s);
  if (prec == MGN_BF16) return launch_edge_fwd_w160(t, e_in, e_out, write_e, Pn, w, eps, agg, slots, a1_out, s);
  const int g = grid_for(t.n_tiles, kEdgeFwdBlocks);
  if (!g) return hipSuccess;
#define F(LD)                                                                                                     \
  hipLaunchKernelGGL((k_edge_fwd<MGN_FP32, LD>), dim3(g), dim3(LD * 4), 0, s, t, (const float*)e_in,              \
                     (float*)e_out, write_e, (const float*)Pn, w, eps, agg, slots)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_edge_bwd(int prec, int lat, const EdgeTiles& t, const void* e, const float* ebar_in, int have_ebar,
                           float* ebar_out, const void* Pn, const float* aggbar, const MlpW& w, float eps, void* zbar,
                           float* R, float* slots, const Partials& part, int* nblocks, hipStream_t s) {
  const int g = grid_for(t.n_tiles, std::min(kEdgeBwdBlocks, part.max_blocks));
  *nblocks = g;
  if (!g) return hipSuccess;
  // bf16 runs on the row-per-wave kernels (k_edge_bwd_fused at width 128,
  // k_edge_bwd_w160 at 160)
  if (prec == MGN_BF16) return hipErrorInvalidValue;
#define F(LD)                                                                                                      \
  hipLaunchKernelGGL((k_edge_bwd<MGN_FP32, LD>), dim3(g), dim3(LD * 4), 0, s, t, (const float*)e, ebar_in,         \
                     have_ebar, ebar_out, (const float*)Pn, aggbar, w, eps, (float*)zbar, R, slots, part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_wgrad(int prec, int lat, int64_t M, const void* Gm, const void* Xm, const Partials& part,
                        int* nblocks, hipStream_t s) {
  const int g = grid_for((M + TM - 1) / TM, std::min(kWgradBlocks, part.max_blocks));
  *nblocks = g;
  if (!g) return hipSuccess;
  // bf16 runs on k_wgrad2 (width 128) and k_wgrad2_w160
  if (prec == MGN_BF16) return hipErrorInvalidValue;
#define F(LD)                                                                                                     \
  hipLaunchKernelGGL((k_wgrad<MGN_FP32, LD>), dim3(g), dim3(LD * 4), 0, s, M, (const float*)Gm, (const float*)Xm, \
                     part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

}  // namespace mgn
