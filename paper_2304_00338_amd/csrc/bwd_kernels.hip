// Reverse-mode kernels of one MGN call on gfx950 in the feature-split
// layout, bf16 only (fp32 runs on the row-layout kernels): the decoder, and
// at width 128 the sender-side sums and the node encoder; and the
// reduction of the per-block partials (both precisions).  Activations inside each MLP are
// recomputed from the saved block inputs (edge latents, node latents,
// aggregates and node products).  Weight gradients are accumulated per
// persistent block in registers and written as per-block partials, which
// k_reduce sums in block order: no atomics anywhere, so gradients are
// bitwise reproducible.
//
// Sender-side sums use the reverse-edge index: the out-edges of node v are
// the reverses of its in-edges, so sum_{e: s(e)=v} x_e is a gather over the
// in-segment of v through rev[], in a fixed order.
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

// Column partial: sum over q groups, lane q == 0 holds the result.
__device__ __forceinline__ void put_col(float* dst, float v, int q) {
  v = sum_q(v);
  if (q == 0) *dst = v;
}

// Write an [o: 16w + q*4 + r][cb*16 + i] accumulator block set.
template <int NCB>
__device__ __forceinline__ void put_w(float* base, int ld, const f32x4 (&acc)[NCB], int w8, int i, int q) {
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) base[(size_t)(w8 * 16 + q * 4 + r) * ld + cb * 16 + i] = acc[cb][r];
}

// ------------------------------------------------------------ decoder
template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) k_decoder_bwd(int64_t N, const float* __restrict__ h,
                                                    const float* __restrict__ gout, MlpW w,
                                                    float* __restrict__ hbar, Partials part) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;
  constexpr int LDT = D + P::PAD;
  __shared__ __align__(16) T sX[TM * LDT];
  __shared__ __align__(16) T sG[TM * LDT];
  __shared__ float sO[TM][4];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n];
  float w2c[4];
#pragma unroll
  for (int o = 0; o < 4; ++o) w2c[o] = w.W2f[o * D + n];
  f32x4 dW1[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dW1[cb] = zero4();
  float db1 = 0.f, dW2[4] = {0.f, 0.f, 0.f, 0.f}, db2 = 0.f;
  const int64_t ntiles = (N + TM - 1) / TM;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * TM;
    const int nr = (int)min((int64_t)TM, N - r0);
    stage_rows<D>(sX, LDT, h + (size_t)r0 * D, nr, tid);
    if (tid < TM * 4) {
      const int row = tid >> 2, o = tid & 3;
      sO[row][o] = row < nr ? gout[(r0 + row) * 4 + o] : 0.f;
    }
    __syncthreads();
    if (tid < 4)
      for (int row = 0; row < nr; ++row) db2 += sO[row][tid];
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b1, b1, b1, b1};
    gemm_tile<PREC, D>(acc, sX, LDT, (const T*)w.W1, D, w8 * 16, 0, i, q);
    f32x4 g[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        const float a1 = fmaxf(acc[rb][r], 0.f);
        float ab = 0.f;
#pragma unroll
        for (int o = 0; o < 4; ++o) {
          const float go = sO[row][o];
          dW2[o] += go * a1;
          ab += go * w2c[o];
        }
        const float zb = acc[rb][r] > 0.f ? ab : 0.f;
        db1 += zb;
        g[rb][r] = zb;
        sG[row * LDT + n] = P::cvt(zb);
      }
    gtx<PREC, NCB>(dW1, g, sX, LDT, 0, i, q);
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = zero4();
    gemm_tile<PREC, D>(acc, sG, LDT, (const T*)w.W1t, D, w8 * 16, 0, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        if (row < nr) hbar[(size_t)(r0 + row) * D + n] = acc[rb][r];
      }
    __syncthreads();
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  // decoder parameter order: W1 [D][D], b1, W2 [4][D], b2
  put_w<NCB>(base, D, dW1, w8, i, q);
  put_col(base + D * D + n, db1, q);
#pragma unroll
  for (int o = 0; o < 4; ++o) put_col(base + D * D + D + o * D + n, dW2[o], q);
  if (tid < 4) base[D * D + 5 * D + tid] = db2;
}

// 8 consecutive elements of a row as one (bf16) or two (fp32) 16-byte loads.
template <typename T>
struct RowChunk;
template <>
struct RowChunk<bf16> {
  struct V {
    uint4 a;
  };
  static __device__ __forceinline__ V load(const bf16* p) { return V{*reinterpret_cast<const uint4*>(p)}; }
  static __device__ __forceinline__ void add(float (&s)[8], const V& v) {
    const bf16x8 b = __builtin_bit_cast(bf16x8, v.a);
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u] += (float)b[u];
  }
};
template <>
struct RowChunk<float> {
  struct V {
    float4 a, b;
  };
  static __device__ __forceinline__ V load(const float* p) {
    return V{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  static __device__ __forceinline__ void add(float (&s)[8], const V& v) {
    s[0] += v.a.x;
    s[1] += v.a.y;
    s[2] += v.a.z;
    s[3] += v.a.w;
    s[4] += v.b.x;
    s[5] += v.b.y;
    s[6] += v.b.z;
    s[7] += v.b.w;
  }
};

// ------------------------------------------------- sender-side sums
// S[v] = sum over in-edges e of v of zbar[rev[e]] (= sum over out-edges of v),
// then hbar_out = hbar_part + W1s^T S + W1r^T R and the weight gradients of
// the sender / receiver parts of the edge MLP's first layer.
template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) k_node_srcsum(int64_t N, const int32_t* __restrict__ rowptr,
                                                    const int32_t* __restrict__ rev,
                                                    const typename Tr<PREC>::T* __restrict__ zbar,
                                                    const float* __restrict__ R, const float* __restrict__ h,
                                                    const float* __restrict__ hbar_part, MlpW w,
                                                    float* __restrict__ hbar_out, Partials part) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;
  constexpr int LDT = D + P::PAD;
  constexpr int LDX = 2 * D + P::PAD;
  __shared__ __align__(16) T sSR[TM * LDX];
  __shared__ __align__(16) T sH[TM * LDT];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  f32x4 dWs[NCB], dWr[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dWs[cb] = dWr[cb] = zero4();
  const int64_t ntiles = (N + TM - 1) / TM;
  // D/8 lanes per node, 8 features per lane; the node's reversed in-edges
  // are gathered 8 at a time (independent loads) and added in edge order.
  // The first 8 of the next tile's node go through their three dependent
  // loads (rowptr, then rev, then zbar) one step at a time around this
  // tile's staging and products, so each has work to hide behind.
  const int j = tid / (D / 8), c8 = (tid % (D / 8)) * 8;
  struct First {
    int e, e1;
    int rv[8];
    typename RowChunk<T>::V x[8];
  };
  auto f_rowptr = [&](int64_t t, First& F) {
    F.e = F.e1 = 0;
    if (t < ntiles && t * TM + j < N) {
      const int v = (int)(t * TM + j);
      F.e = rowptr[v];
      F.e1 = rowptr[v + 1];
    }
  };
  auto f_rev = [&](First& F) {
#pragma unroll
    for (int k = 0; k < 8; ++k) F.rv[k] = F.e + k < F.e1 ? rev[F.e + k] : -1;
  };
  auto f_z = [&](First& F) {
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (F.rv[k] >= 0) F.x[k] = RowChunk<T>::load(zbar + (size_t)F.rv[k] * D + c8);
  };
  First F, Fn;
  f_rowptr(blockIdx.x, F);
  f_rev(F);
  f_z(F);
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * TM;
    const int nr = (int)min((int64_t)TM, N - r0);
    {
      float acc8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc8[u] = 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (F.rv[k] >= 0) RowChunk<T>::add(acc8, F.x[k]);
      for (int e = F.e + 8; e < F.e1; e += 8) {
        int rv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) rv[k] = e + k < F.e1 ? rev[e + k] : -1;
        typename RowChunk<T>::V x[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (rv[k] >= 0) x[k] = RowChunk<T>::load(zbar + (size_t)rv[k] * D + c8);
#pragma unroll
        for (int k = 0; k < 8; ++k)
          if (rv[k] >= 0) RowChunk<T>::add(acc8, x[k]);
      }
      T o[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) o[u] = P::cvt(acc8[u]);
      // rows past the tile's end get zeros (their rv are all -1)
#pragma unroll
      for (int u = 0; u < (int)(8 * sizeof(T)) / 16; ++u)
        reinterpret_cast<uint4*>(sSR + j * LDX + c8)[u] = reinterpret_cast<const uint4*>(o)[u];
    }
    f_rowptr(t + gridDim.x, Fn);
    stage_rows<D>(sSR + D, LDX, R + (size_t)r0 * D, nr, tid);
    stage_rows<D>(sH, LDT, h + (size_t)r0 * D, nr, tid);
    __syncthreads();
    f_rev(Fn);
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        acc[rb][r] = row < nr ? hbar_part[(size_t)(r0 + row) * D + n] : 0.f;
      }
    gemm_tile<PREC, D>(acc, sSR, LDX, (const T*)w.W1t, D, D + w8 * 16, 0, i, q);
    gemm_tile<PREC, D>(acc, sSR + D, LDX, (const T*)w.W1t, D, 2 * D + w8 * 16, 0, i, q);
    f_z(Fn);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        if (row < nr) hbar_out[(size_t)(r0 + row) * D + n] = acc[rb][r];
      }
    f32x4 g[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) g[rb][r] = tof(sSR[(rb * 16 + q * 4 + r) * LDX + n]);
    gtx<PREC, NCB>(dWs, g, sH, LDT, 0, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) g[rb][r] = tof(sSR[(rb * 16 + q * 4 + r) * LDX + D + n]);
    gtx<PREC, NCB>(dWr, g, sH, LDT, 0, i, q);
    __syncthreads();
    F = Fn;
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  put_w<NCB>(base, D, dWs, w8, i, q);
  put_w<NCB>(base + D * D, D, dWr, w8, i, q);
}

// ------------------------------------------------------- node encoder
// ybar: dL/d(encoder output), fp32; KIN inputs per row (the node encoder's 8).
template <int PREC, int LD, int KIN>
__global__ void __launch_bounds__(LD * 4) k_enc_bwd(int64_t M, const float* __restrict__ x_in,
                                                const float* __restrict__ ybar, MlpW w, float eps,
                                                float* __restrict__ gin, Partials part) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int NCB = D / 16;
  constexpr int LDT = D + P::PAD;
  constexpr int LDM = D + 4;
  __shared__ float sX[TM][KIN];
  __shared__ __align__(16) T sA[TM * LDT];
  __shared__ __align__(16) T sG[TM * LDT];
  __shared__ float sZ[KIN == 8 ? TM * LDM : 1];
  __shared__ LnScratch<NW> ln;
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n], b2 = w.b2[n], gam = w.gamma[n];
  float w1[KIN];
#pragma unroll
  for (int k = 0; k < KIN; ++k) w1[k] = w.W1f[n * KIN + k];
  f32x4 dW2[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dW2[cb] = zero4();
  float dW1[KIN];
#pragma unroll
  for (int k = 0; k < KIN; ++k) dW1[k] = 0.f;
  float db1 = 0.f, db2 = 0.f, dg = 0.f, dbt = 0.f;
  const int64_t ntiles = (M + TM - 1) / TM;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * TM;
    const int nr = (int)min((int64_t)TM, M - r0);
    for (int idx = tid; idx < TM * KIN; idx += NT) {
      const int row = idx / KIN, k = idx % KIN;
      sX[row][k] = row < nr ? x_in[(r0 + row) * KIN + k] : 0.f;
    }
    __syncthreads();
    uint32_t mask = 0;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        float z = b1;
#pragma unroll
        for (int k = 0; k < KIN; ++k) z += w1[k] * sX[row][k];
        if (z > 0.f) mask |= 1u << (rb * 4 + r);
        sA[row * LDT + n] = P::cvt(fmaxf(z, 0.f));
      }
    __syncthreads();
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b2, b2, b2, b2};
    gemm_tile<PREC, D>(acc, sA, LDT, (const T*)w.W2, D, w8 * 16, 0, i, q);
    f32x4 mean[NRB], rstd[NRB], xh[NRB], yb[NRB];
    ln_stats(acc, ln, eps, w8, i, q, mean, rstd);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        xh[rb][r] = (acc[rb][r] - mean[rb][r]) * rstd[rb][r];
        yb[rb][r] = row < nr ? ybar[(size_t)(r0 + row) * D + n] : 0.f;
        dg += yb[rb][r] * xh[rb][r];
        dbt += yb[rb][r];
      }
    f32x4 g[NRB];
    ln_bwd(g, yb, xh, rstd, gam, ln, w8, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        db2 += g[rb][r];
        sG[(rb * 16 + q * 4 + r) * LDT + n] = P::cvt(g[rb][r]);
      }
    gtx<PREC, NCB>(dW2, g, sA, LDT, 0, i, q);
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = zero4();
    gemm_tile<PREC, D>(acc, sG, LDT, (const T*)w.W2t, D, w8 * 16, 0, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        const float zb = (mask >> (rb * 4 + r)) & 1u ? acc[rb][r] : 0.f;
        db1 += zb;
#pragma unroll
        for (int k = 0; k < KIN; ++k) dW1[k] += zb * sX[row][k];
        if (KIN == 8) sZ[row * LDM + n] = zb;
      }
    if (KIN == 8 && gin) {
      __syncthreads();
      const int row = tid >> 3, k = tid & 7;
      if (row < nr) {
        float s = 0.f;
        for (int c = 0; c < D; ++c) s += sZ[row * LDM + c] * w.W1f[c * KIN + k];
        gin[(r0 + row) * KIN + k] = s;
      }
    }
    __syncthreads();
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int k = 0; k < KIN; ++k) put_col(base + n * KIN + k, dW1[k], q);
  const int o1 = D * KIN;
  put_col(base + o1 + n, db1, q);
  put_w<NCB>(base + o1 + D, D, dW2, w8, i, q);
  put_col(base + o1 + D + D * D + n, db2, q);
  put_col(base + o1 + 2 * D + D * D + n, dg, q);
  put_col(base + o1 + 3 * D + D * D + n, dbt, q);
}

// ----------------------------------------------------------- reduce
// grad[...] += sum over the nblocks partial rows.  A block takes 16
// consecutive entries; its 16 lane groups each sum every 16th partial row
// (group g: rows g, g+16, ...) in row order, 8 loads in flight, and the 16
// group sums are added in group order: a fixed order for any launch.
constexpr int kRedCols = 16, kRedGroups = 16;
__global__ void __launch_bounds__(256) k_reduce(Partials part, int nblocks, int64_t src, int32_t rows, int32_t cols,
                                                float* __restrict__ grad, int64_t dst, int64_t dst_ld) {
  __shared__ float red[kRedGroups][kRedCols];
  const int64_t total = (int64_t)rows * cols;
  const int c = threadIdx.x % kRedCols, gr = threadIdx.x / kRedCols;
  const int64_t idx = (int64_t)blockIdx.x * kRedCols + c;
  float s = 0.f;
  if (idx < total) {
    const float* p = part.buf + src + idx;
    int b = gr;
    for (; b + 7 * kRedGroups < nblocks; b += 8 * kRedGroups) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(size_t)(b + u * kRedGroups) * part.stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; b < nblocks; b += kRedGroups) s += p[(size_t)b * part.stride];
  }
  red[gr][c] = s;
  __syncthreads();
  if (gr == 0 && idx < total) {
    float t = 0.f;
#pragma unroll
    for (int g = 0; g < kRedGroups; ++g) t += red[g][c];
    const int64_t r = idx / cols, cc = idx % cols;
    grad[dst + r * dst_ld + cc] += t;
  }
}

// The jobs of a batch one after the other over the launch's blocks; each
// entry is summed exactly as in k_reduce.
__global__ void __launch_bounds__(256) k_reduce_batch(Partials part, int64_t region_floats, ReduceBatch b,
                                                      float* __restrict__ grad) {
  __shared__ float red[kRedGroups][kRedCols];
  int k = 0;
  while (k + 1 < b.n && (int64_t)blockIdx.x >= b.j[k + 1].blk0) ++k;
  const ReduceJob& J = b.j[k];
  const int64_t total = (int64_t)J.rows * J.cols;
  const int c = threadIdx.x % kRedCols, gr = threadIdx.x / kRedCols;
  const int64_t idx = ((int64_t)blockIdx.x - J.blk0) * kRedCols + c;
  float s = 0.f;
  if (idx < total) {
    const float* p = part.buf + J.region * region_floats + J.src + idx;
    int bl = gr;
    for (; bl + 7 * kRedGroups < J.nblocks; bl += 8 * kRedGroups) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(size_t)(bl + u * kRedGroups) * part.stride];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; bl < J.nblocks; bl += kRedGroups) s += p[(size_t)bl * part.stride];
  }
  red[gr][c] = s;
  __syncthreads();
  if (gr == 0 && idx < total) {
    float t = 0.f;
#pragma unroll
    for (int g = 0; g < kRedGroups; ++g) t += red[g][c];
    const int64_t r = idx / J.cols, cc = idx % J.cols;
    grad[J.dst + r * J.ld + cc] += t;
  }
}

}  // namespace dev

// ============================================================ launchers
using namespace dev;

static constexpr int kBwdBlocks = 256;

static int bwd_grid(int64_t n_tiles, const Partials& p) {
  return part_grid(n_tiles, std::min(kBwdBlocks, p.max_blocks));
}

hipError_t launch_decoder_bwd(int prec, int lat, int64_t N, const float* h, const float* gout, const MlpW& w,
                              float* hbar, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  // bf16 (fp32 runs on launch_decoder_bwd_r32)
  if (prec != MGN_BF16) return hipErrorInvalidValue;
  const int g = bwd_grid((N + TM - 1) / TM, part);
  *nblocks = g;
  if (!g) return hipSuccess;
#define F(LD) hipLaunchKernelGGL((k_decoder_bwd<MGN_BF16, LD>), dim3(g), dim3(LD * 4), 0, s, N, h, gout, w, hbar, part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_node_srcsum(int prec, int lat, int64_t N, const int32_t* rowptr, const int32_t* rev,
                              const void* zbar, const float* R, const float* h, const float* hbar_part, const MlpW& w,
                              float* hbar_out, const Partials& part, int* nblocks, hipStream_t s) {
  // bf16 at width 128 (fp32 runs on launch_node_srcsum_r32, bf16 at width
  // 160 on launch_srcsum_w160)
  *nblocks = 0;
  if (prec != MGN_BF16 || lat != 128) return hipErrorInvalidValue;
  const int g = bwd_grid((N + TM - 1) / TM, part);
  *nblocks = g;
  if (!g) return hipSuccess;
  hipLaunchKernelGGL((k_node_srcsum<MGN_BF16, 128>), dim3(g), dim3(128 * 4), 0, s, N, rowptr, rev, (const bf16*)zbar,
                     R, h, hbar_part, w, hbar_out, part);
  return hipGetLastError();
}

hipError_t launch_node_enc_bwd(int prec, int lat, int64_t N, const float* node_in, const float* hbar, const MlpW& w,
                               float eps, float* gin, const Partials& part, int* nblocks, hipStream_t s) {
  if (prec == MGN_BF16 && lat == 160) return launch_node_enc_bwd_w160(N, node_in, hbar, w, eps, gin, part, nblocks, s);
  *nblocks = 0;
  // bf16 at width 128 (fp32 runs on launch_node_enc_bwd_r32)
  if (prec != MGN_BF16 || lat != 128) return hipErrorInvalidValue;
  const int g = bwd_grid((N + TM - 1) / TM, part);
  *nblocks = g;
  if (!g) return hipSuccess;
  hipLaunchKernelGGL((k_enc_bwd<MGN_BF16, 128, 8>), dim3(g), dim3(128 * 4), 0, s, N, node_in, hbar, w, eps, gin, part);
  return hipGetLastError();
}

hipError_t launch_reduce(const Partials& part, int nblocks, int64_t src, int32_t rows, int32_t cols, float* grad,
                         int64_t dst, int64_t dst_ld, hipStream_t s) {
  if (nblocks <= 0 || rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t total = (int64_t)rows * cols;
  const int64_t g = (total + kRedCols - 1) / kRedCols;
  hipLaunchKernelGGL(k_reduce, dim3((unsigned)g), dim3(256), 0, s, part, nblocks, src, rows, cols, grad, dst, dst_ld);
  return hipGetLastError();
}

hipError_t launch_reduce_batch(const Partials& part, int64_t region_floats, ReduceBatch b, float* grad,
                               hipStream_t s) {
  if (b.n <= 0) return hipSuccess;
  if (b.n > kMaxReduceJobs) return hipErrorInvalidValue;
  int64_t blocks = 0;
  for (int k = 0; k < b.n; ++k) {
    b.j[k].blk0 = blocks;
    blocks += ((int64_t)b.j[k].rows * b.j[k].cols + kRedCols - 1) / kRedCols;
  }
  hipLaunchKernelGGL(k_reduce_batch, dim3((unsigned)blocks), dim3(256), 0, s, part, region_floats, b, grad);
  return hipGetLastError();
}

}  // namespace mgn
