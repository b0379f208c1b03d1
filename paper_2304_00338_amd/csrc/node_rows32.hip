// Node phase of one MGN message-passing step in fp32 (Sec. 2.1: every node
// latent is updated by the node MLP from itself and the sum of its incoming
// edge messages, with LayerNorm and a residual), in the fp32 row layout of
// rows32_common.hpp at kernel width LD = 128 or 160 (latent 150 padded with
// zero columns): one wave per 16-node unit, the four lanes of a node holding
// its contiguous row, every product on gemm32 from fragment-major weights.
//
// The first layer acts on the concatenation [h, agg]; it is evaluated as
// (b1 + W1h h) + W1a agg with the two column blocks of W1 (the same linear
// map, in this summation order in the forward and the reverse's recompute).
#include "rows32_common.hpp"

namespace mgn {
namespace dev {

// z1 = (b1 + W1h h) + W1a agg for the lane's features (the C layout of
// gemm32: acc[ob][r] is feature f0 + 4 ob + r).  Shared by the forward and
// the reverse, so the reverse's recompute equals the forward bitwise.
template <int LD>
__device__ __forceinline__ void node_z1_r32(f32x4 (&acc)[R32<LD>::NOB], const float (&h)[R32<LD>::KL],
                                            const float (&a)[R32<LD>::KL], const MlpW& w, int f0, int lane,
                                            int oz) {
#pragma unroll
  for (int ob = 0; ob < R32<LD>::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b1 + f0 + 4 * ob);
  gemm32<LD>(acc, h, w.F1 + oz, lane);
  gemm32<LD>(acc, a, w.F1a + oz, lane);
}

// LayerNorm statistics of a row over its DR real features (padded features
// hold 0 and are left out of the variance): acc becomes acc - mean.
template <int LD>
__device__ __forceinline__ float ln_center_r32(f32x4 (&acc)[R32<LD>::NOB], int f0, float eps) {
  typedef R32<LD> Z;
  float sm = 0.f;
#pragma unroll
  for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm += acc[ob][r];
  const float mean = sum_q(sm) * (1.0f / Z::DR);
  float sq = 0.f;
#pragma unroll
  for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float dlt = acc[ob][r] - mean;
      acc[ob][r] = dlt;
      if (Z::DR == LD || f0 + 4 * ob + r < Z::DR) sq += dlt * dlt;
    }
  return __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / Z::DR) + eps);
}

// Forward: h_out = h + LN(W2 relu(z1) + b2); with EMIT, also the next
// block's node products P_out = [W1s h_out, W1r h_out] ([N][2 LD]) from the
// next edge MLP nx.  The next unit's agg row is requested after the first
// layer, its h row after the residual (single buffers: each is dead by
// then); rows past N read row N - 1 and store nothing.
template <int LD, bool EMIT>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_node_fwd_r32(int64_t N, const float* __restrict__ h_in, const float* __restrict__ agg, MlpW w, MlpW nx, float eps,
               float* __restrict__ h_out, float* __restrict__ P_out) {
  typedef R32<LD> Z;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  if (ur.t >= ur.end) return;
  const int f0 = Z::KL * g;
  auto rowp = [&](int64_t u) { return (size_t)min(u * 16 + i, N - 1) * LD + f0; };
  float h[Z::KL], a[Z::KL];
  load_row32<LD>(h, h_in + rowp(ur.t));
  load_row32<LD>(a, agg + rowp(ur.t));
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const int64_t un = u + ur.stride;
    const bool live = u * 16 + i < N;
    // the weight addresses are opaque per unit: otherwise the loop-invariant
    // fragment loads are hoisted out of the loop into registers
    const int oz = opaque_zero();
    f32x4 acc[Z::NOB];
    node_z1_r32<LD>(acc, h, a, w, f0, lane, oz);
    load_row32<LD>(a, agg + rowp(un));
    float a1[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) a1[4 * ob + r] = relu(acc[ob][r]);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, w.F2 + oz, lane);
    const float rstd = ln_center_r32<LD>(acc, f0, eps);
    float y[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      const f32x4 ga = *reinterpret_cast<const f32x4*>(w.gamma + f0 + 4 * ob);
      const f32x4 be = *reinterpret_cast<const f32x4*>(w.beta + f0 + 4 * ob);
      const f32x4 m = ga * (acc[ob] * rstd) + be;
#pragma unroll
      for (int r = 0; r < 4; ++r) y[4 * ob + r] = m[r] + h[4 * ob + r];
    }
    if (live) {
      float* p = h_out + (size_t)(u * 16 + i) * LD + f0;
#pragma unroll
      for (int c = 0; c < Z::KC; ++c)
        *reinterpret_cast<f32x4*>(p + 4 * c) = f32x4{y[4 * c], y[4 * c + 1], y[4 * c + 2], y[4 * c + 3]};
    }
    load_row32<LD>(h, h_in + rowp(un));
    if (EMIT) {
      f32x4 ps[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = ps[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      gemm32<LD>(ps, y, nx.F1s + oz, lane);
      gemm32<LD>(acc, y, nx.F1r + oz, lane);
      if (live) {
        float* p = P_out + (size_t)(u * 16 + i) * (2 * LD) + f0;
        store_row32<LD>(p, ps);
        store_row32<LD>(p + LD, acc);
      }
    }
  }
}

// Reverse of the node phase for the rows of hbar_in = dL/dh_out: the
// forward recomputed (z1 bitwise as in the forward), the LayerNorm reverse
// (padded features of dz2 zeroed), da1 = W2^T dz2, dz1 = da1 where z1 > 0,
// hbar_part = hbar_in + W1h^T dz1 and aggbar = W1a^T dz1.  The rows of a1,
// dz2 and dz1 go to the streams (fp32 [N][LD] each) for the weight-gradient
// passes (dW1 = sum dz1^T [h, agg], dW2 = sum dz2^T a1); db1, db2, dgamma
// and dbeta are DPP column sums, written per block as [4][LD] partials (db1,
// db2, dgamma, dbeta).  Each input row is requested again for the next unit
// once its last use is issued.
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_node_bwd_r32(int64_t N, const float* __restrict__ h_in, const float* __restrict__ agg,
               const float* __restrict__ hbar_in, MlpW w, float eps, float* __restrict__ hbar_part,
               float* __restrict__ aggbar, float* __restrict__ a1s, float* __restrict__ dz2s,
               float* __restrict__ dz1s, Partials part) {
  typedef R32<LD> Z;
  __shared__ __align__(16) float red[4][R32_NW][LD];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  ColSum32<LD> cs[4];  // db1, db2, dgamma, dbeta
  if (ur.t < ur.end) {
    auto rowp = [&](int64_t u) { return (size_t)min(u * 16 + i, N - 1) * LD + f0; };
    float h[Z::KL], a[Z::KL], yb[Z::KL];
    load_row32<LD>(h, h_in + rowp(ur.t));
    load_row32<LD>(a, agg + rowp(ur.t));
    load_row32<LD>(yb, hbar_in + rowp(ur.t));
    for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
      const int64_t un = u + ur.stride;
      const bool live = u * 16 + i < N;
      const size_t orow = (size_t)(u * 16 + i) * LD + f0;
      const int oz = opaque_zero();
      // ---- the forward: z1, its ReLU mask, a1, z2 and its LayerNorm
      f32x4 acc[Z::NOB];
      node_z1_r32<LD>(acc, h, a, w, f0, lane, oz);
      load_row32<LD>(h, h_in + rowp(un));
      load_row32<LD>(a, agg + rowp(un));
      float a1[Z::KL];
      uint64_t mask = 0;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          a1[4 * ob + r] = relu(acc[ob][r]);
          if (acc[ob][r] > 0.f) mask |= 1ull << (4 * ob + r);
        }
      if (live) {
        float* p = a1s + orow;
#pragma unroll
        for (int c = 0; c < Z::KC; ++c)
          *reinterpret_cast<f32x4*>(p + 4 * c) = f32x4{a1[4 * c], a1[4 * c + 1], a1[4 * c + 2], a1[4 * c + 3]};
      }
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b2 + f0 + 4 * ob);
      gemm32<LD>(acc, a1, w.F2 + oz, lane);
      const float rstd = ln_center_r32<LD>(acc, f0, eps);
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] *= rstd;  // xhat
      // ---- dbeta, dgamma (live rows); the LayerNorm reverse
      f32x4 t[Z::NOB];
      {
        f32x4 p[Z::NOB];
#pragma unroll
        for (int ob = 0; ob < Z::NOB; ++ob) {
          t[ob] = f32x4{yb[4 * ob], yb[4 * ob + 1], yb[4 * ob + 2], yb[4 * ob + 3]};
          p[ob] = live ? t[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        cs[3].add(p, i);
#pragma unroll
        for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = live ? t[ob] * acc[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
        cs[2].add(p, i);
      }
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        t[ob] *= *reinterpret_cast<const f32x4*>(w.gamma + f0 + 4 * ob);  // dxh
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          s1 += t[ob][r];
          s2 += t[ob][r] * acc[ob][r];
        }
      }
      const float m1 = sum_q(s1) * (1.0f / Z::DR), m2 = sum_q(s2) * (1.0f / Z::DR);
      float dz[Z::KL];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          dz[4 * ob + r] = (Z::DR == LD || f0 + 4 * ob + r < Z::DR) ? rstd * (t[ob][r] - m1 - acc[ob][r] * m2) : 0.f;
      {
        f32x4 p[Z::NOB];
#pragma unroll
        for (int ob = 0; ob < Z::NOB; ++ob)
          p[ob] = live ? f32x4{dz[4 * ob], dz[4 * ob + 1], dz[4 * ob + 2], dz[4 * ob + 3]} : f32x4{0.f, 0.f, 0.f, 0.f};
        cs[1].add(p, i);
        if (live) store_row32<LD>(dz2s + orow, p);
      }
      // ---- da1 = W2^T dz2, dz1 = da1 where z1 > 0
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      gemm32<LD>(acc, dz, w.F2t + oz, lane);
      float d1[Z::KL];
      {
        f32x4 p[Z::NOB];
#pragma unroll
        for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = (mask >> (4 * ob + r)) & 1ull ? acc[ob][r] : 0.f;
            d1[4 * ob + r] = v;
            p[ob][r] = live ? v : 0.f;
          }
        cs[0].add(p, i);
        if (live) store_row32<LD>(dz1s + orow, p);
      }
      // ---- hbar_part = hbar_in + W1h^T dz1, aggbar = W1a^T dz1
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
        acc[ob] = f32x4{yb[4 * ob], yb[4 * ob + 1], yb[4 * ob + 2], yb[4 * ob + 3]};
      gemm32<LD>(acc, d1, w.F1t + oz, lane);
      if (live) store_row32<LD>(hbar_part + orow, acc);
      load_row32<LD>(yb, hbar_in + rowp(un));
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      gemm32<LD>(acc, d1, w.F1at + oz, lane);
      if (live) store_row32<LD>(aggbar + orow, acc);
    }
  }
  // ---- block partials [4][LD]: the waves' column sums added in wave order
#pragma unroll
  for (int k = 0; k < 4; ++k) cs[k].put(red[k][wv], f0, i);
  __syncthreads();
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  for (int idx = tid; idx < 4 * LD; idx += R32_NT) {
    const int k = idx / LD, c = idx % LD;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) v += red[k][u][c];
    base[idx] = v;
  }
}


// Sender-side sums and the node gradient through the edge MLP's sender and
// receiver blocks: S_v = sum of zbar over the reverses of v's in-edges (the
// out-edges of v), added in edge order; hbar_out = hbar_part + W1s^T S +
// W1r^T R.  The rows of S go to S_out (fp32 [N][LD]) for the weight
// gradients dW1s = sum S h^T, dW1r = sum R h^T.  Each lane gathers its KL
// features of four edges' rows at a time; rows of an edge-less or a dead
// node add nothing.
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_node_srcsum_r32(int64_t N, const int32_t* __restrict__ rowptr, const int32_t* __restrict__ rev,
                  const float* __restrict__ zbar, const float* __restrict__ R, const float* __restrict__ hbar_part,
                  MlpW w, float* __restrict__ hbar_out, float* __restrict__ S_out) {
  typedef R32<LD> Z;
  constexpr int GE = 4;  // edges gathered at a time
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  // The reversed edge ids of a gather round are requested one round ahead
  // (with the zbar rows of the current round), and the next unit's segment
  // bounds and first ids during this unit's products, so each round waits
  // for one load latency instead of two.
  struct Seg {
    int e0, e1;
    int r[GE];
  };
  auto seg = [&](int64_t uu, Seg& q) {
    q.e0 = q.e1 = 0;
    if (uu < ur.end && uu * 16 + i < N) {
      q.e0 = rowptr[uu * 16 + i];
      q.e1 = rowptr[uu * 16 + i + 1];
    }
  };
  auto ids = [&](const Seg& q, int k0, int (&r)[GE]) {
#pragma unroll
    for (int k = 0; k < GE; ++k) r[k] = q.e0 + k0 + k < q.e1 ? rev[q.e0 + k0 + k] : 0;
  };
  Seg sg;
  if (ur.t < ur.end) {
    seg(ur.t, sg);
    ids(sg, 0, sg.r);
  }
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const bool live = u * 16 + i < N;
    const int64_t v = min(u * 16 + i, N - 1);
    const size_t orow = (size_t)v * LD + f0;
    const int e0 = sg.e0, e1 = sg.e1;
    float hb[Z::KL], rr[Z::KL];
    load_row32<LD>(hb, hbar_part + orow);
    load_row32<LD>(rr, R + orow);
    int md = e1 - e0;  // the unit's largest in-degree
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) md = max(md, __shfl_xor(md, o));
    float S[Z::KL];
#pragma unroll
    for (int c = 0; c < Z::KL; ++c) S[c] = 0.f;
    int rc[GE];
#pragma unroll
    for (int k = 0; k < GE; ++k) rc[k] = sg.r[k];
    for (int k0 = 0; k0 < md; k0 += GE) {
      int rn[GE];
      ids(sg, k0 + GE, rn);
      f32x4 x[GE][Z::KC];
#pragma unroll
      for (int k = 0; k < GE; ++k) {
        const int e = e0 + k0 + k;
        if (e < e1) {
          const float* zp = zbar + (size_t)rc[k] * LD + f0;
#pragma unroll
          for (int c = 0; c < Z::KC; ++c) x[k][c] = *reinterpret_cast<const f32x4*>(zp + 4 * c);
        }
      }
#pragma unroll
      for (int k = 0; k < GE; ++k)
        if (e0 + k0 + k < e1)
#pragma unroll
          for (int c = 0; c < Z::KC; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) S[4 * c + r] += x[k][c][r];
#pragma unroll
      for (int k = 0; k < GE; ++k) rc[k] = rn[k];
    }
    if (live) {
      float* p = S_out + orow;
#pragma unroll
      for (int c = 0; c < Z::KC; ++c)
        *reinterpret_cast<f32x4*>(p + 4 * c) = f32x4{S[4 * c], S[4 * c + 1], S[4 * c + 2], S[4 * c + 3]};
    }
    const int oz = opaque_zero();
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
      acc[ob] = f32x4{hb[4 * ob], hb[4 * ob + 1], hb[4 * ob + 2], hb[4 * ob + 3]};
    seg(u + ur.stride, sg);
    gemm32<LD>(acc, S, w.F1st + oz, lane);
    ids(sg, 0, sg.r);
    gemm32<LD>(acc, rr, w.F1rt + oz, lane);
    if (live) store_row32<LD>(hbar_out + orow, acc);
  }
}


// Decoder (Sec. 2.1: the last node latents are decoded by an MLP without
// LayerNorm to the output fields): out = W2 relu(W1 h + b1) + b2 with W2
// [4][LD] on VALU from LDS, one wave per 16-node unit.
constexpr int DEC_OUT = 4;

template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_decoder_r32(int64_t N, const float* __restrict__ h_in, MlpW w, float* __restrict__ out) {
  typedef R32<LD> Z;
  __shared__ __align__(16) float w2[DEC_OUT][LD];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int idx = tid; idx < DEC_OUT * LD; idx += R32_NT) w2[idx / LD][idx % LD] = w.W2f[idx];
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const bool live = u * 16 + i < N;
    const int64_t v = min(u * 16 + i, N - 1);
    float h[Z::KL];
    load_row32<LD>(h, h_in + (size_t)v * LD + f0);
    const int oz = opaque_zero();
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b1 + f0 + 4 * ob);
    gemm32<LD>(acc, h, w.F1 + oz, lane);
    float o[DEC_OUT] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float a1 = relu(acc[ob][r]);
#pragma unroll
        for (int k = 0; k < DEC_OUT; ++k) o[k] += w2[k][f0 + 4 * ob + r] * a1;
      }
#pragma unroll
    for (int k = 0; k < DEC_OUT; ++k) o[k] = sum_q(o[k]) + w.b2[k];
    if (live && g == 0) *reinterpret_cast<f32x4*>(out + (size_t)v * DEC_OUT) = f32x4{o[0], o[1], o[2], o[3]};
  }
}

// Decoder reverse from gout = dL/dout [N][4]: hbar = W1^T dz1 (written),
// dz1 = (W2^T gout) where z1 > 0; the dz1 rows go to dz1s for dW1 = sum
// dz1^T h (launch_wgrad_r32); db1, dW2 = sum gout a1^T and db2 = sum gout
// as column sums, written per block in the decoder's parameter order after
// W1: [LD] db1, [4][LD] dW2, [4] db2.
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_decoder_bwd_r32(int64_t N, const float* __restrict__ h_in, const float* __restrict__ gout, MlpW w,
                  float* __restrict__ hbar, float* __restrict__ dz1s, Partials part) {
  typedef R32<LD> Z;
  __shared__ __align__(16) float w2[DEC_OUT][LD];
  __shared__ __align__(16) float red[1 + DEC_OUT][R32_NW][LD];
  __shared__ float rb2[R32_NW][16][DEC_OUT];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int idx = tid; idx < DEC_OUT * LD; idx += R32_NT) w2[idx / LD][idx % LD] = w.W2f[idx];
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  ColSum32<LD> cb1, cw2[DEC_OUT];
  float db2[DEC_OUT] = {0.f, 0.f, 0.f, 0.f};
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const bool live = u * 16 + i < N;
    const int64_t v = min(u * 16 + i, N - 1);
    const size_t orow = (size_t)v * LD + f0;
    float h[Z::KL];
    load_row32<LD>(h, h_in + orow);
    const f32x4 go = *reinterpret_cast<const f32x4*>(gout + (size_t)v * DEC_OUT);
    const int oz = opaque_zero();
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b1 + f0 + 4 * ob);
    gemm32<LD>(acc, h, w.F1 + oz, lane);
#pragma unroll
    for (int k = 0; k < DEC_OUT; ++k) {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) p[ob][r] = live ? go[k] * relu(acc[ob][r]) : 0.f;
      cw2[k].add(p, i);
      if (live && g == 0) db2[k] += go[k];
    }
    float d1[Z::KL];
    {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int f = f0 + 4 * ob + r;
          float ab = 0.f;
#pragma unroll
          for (int k = 0; k < DEC_OUT; ++k) ab += go[k] * w2[k][f];
          const float z = acc[ob][r] > 0.f ? ab : 0.f;
          d1[4 * ob + r] = z;
          p[ob][r] = live ? z : 0.f;
        }
      cb1.add(p, i);
      if (live) store_row32<LD>(dz1s + orow, p);
    }
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    gemm32<LD>(acc, d1, w.F1t + oz, lane);
    if (live) store_row32<LD>(hbar + orow, acc);
  }
  cb1.put(red[0][wv], f0, i);
#pragma unroll
  for (int k = 0; k < DEC_OUT; ++k) cw2[k].put(red[1 + k][wv], f0, i);
  if (g == 0)
#pragma unroll
    for (int k = 0; k < DEC_OUT; ++k) rb2[wv][i][k] = db2[k];
  __syncthreads();
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  for (int idx = tid; idx < (1 + DEC_OUT) * LD; idx += R32_NT) {
    const int k = idx / LD, c = idx % LD;
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) s += red[k][u][c];
    base[idx] = s;
  }
  if (tid < DEC_OUT) {
    float s = 0.f;
    for (int u = 0; u < R32_NW; ++u)
      for (int r = 0; r < 16; ++r) s += rb2[u][r][tid];
    base[(1 + DEC_OUT) * LD + tid] = s;
  }
}


// Node encoder (Sec. 2.1: the node features are encoded to the latent width
// by an MLP with LayerNorm): h0 = LN(W2 relu(W1 x + b1) + b2), x the 8 node
// inputs; the first layer (K = 8) as one fp32 fma chain per feature from LDS,
// written once for the forward and the reverse's recompute.
constexpr int NK = 8;  // node inputs

template <int LD>
struct NodeEncVec {
  __attribute__((aligned(16))) float4 w1[LD][2];  // W1 [LD][8]
  __attribute__((aligned(16))) float b1[LD];
  __attribute__((aligned(16))) float b2[LD];
  __attribute__((aligned(16))) float g[LD];
  __attribute__((aligned(16))) float bt[LD];
};
template <int LD>
__device__ __forceinline__ void stage_node_enc_vec(NodeEncVec<LD>& V, const MlpW& w, int tid) {
  for (int idx = tid; idx < LD * NK; idx += R32_NT) reinterpret_cast<float*>(V.w1)[idx] = w.W1f[idx];
  for (int idx = tid; idx < LD; idx += R32_NT) {
    V.b1[idx] = w.b1[idx];
    V.b2[idx] = w.b2[idx];
    V.g[idx] = w.gamma[idx];
    V.bt[idx] = w.beta[idx];
  }
}
// z[s] = b1[f0 + s] + sum over k of W1[f0 + s][k] x[k], k ascending
template <int LD>
__device__ __forceinline__ void node_enc_z1(const NodeEncVec<LD>& V, float4 xa, float4 xb, int f0,
                                            float (&z)[R32<LD>::KL]) {
#pragma unroll
  for (int s = 0; s < R32<LD>::KL; ++s) {
    const float4 wa = V.w1[f0 + s][0], wb = V.w1[f0 + s][1];
    float t = V.b1[f0 + s];
    t = __builtin_fmaf(wa.x, xa.x, t);
    t = __builtin_fmaf(wa.y, xa.y, t);
    t = __builtin_fmaf(wa.z, xa.z, t);
    t = __builtin_fmaf(wa.w, xa.w, t);
    t = __builtin_fmaf(wb.x, xb.x, t);
    t = __builtin_fmaf(wb.y, xb.y, t);
    t = __builtin_fmaf(wb.z, xb.z, t);
    t = __builtin_fmaf(wb.w, xb.w, t);
    z[s] = t;
  }
}

template <int LD>
struct __attribute__((aligned(16))) NodeEncFwdLds {
  NodeEncVec<LD> V;
  __attribute__((aligned(16))) float w2[LD * LD];  // fragment-major W2
};

// Forward (with EMIT the node products of the first MP block from the
// first edge MLP nx, as the node phase does).
template <int LD, bool EMIT>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_node_enc_r32(int64_t N, const float* __restrict__ x_in, MlpW w, MlpW nx, float eps, float* __restrict__ h_out,
               float* __restrict__ P_out) {
  typedef R32<LD> Z;
  __shared__ __align__(16) NodeEncFwdLds<LD> S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int idx = tid; idx < LD * LD / 4; idx += R32_NT)
    reinterpret_cast<f32x4*>(S.w2)[idx] = reinterpret_cast<const f32x4*>(w.F2)[idx];
  stage_node_enc_vec<LD>(S.V, w, tid);
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const bool live = u * 16 + i < N;
    const int64_t v = min(u * 16 + i, N - 1);
    const float4 xa = *reinterpret_cast<const float4*>(x_in + v * NK);
    const float4 xb = *reinterpret_cast<const float4*>(x_in + v * NK + 4);
    // LDS reads through an opaque reference: otherwise the loop-invariant
    // weight reads are hoisted out of the loop into registers
    const NodeEncFwdLds<LD>& L = fresh(S);
    float a1[Z::KL];
    node_enc_z1<LD>(L.V, xa, xb, f0, a1);
#pragma unroll
    for (int s2 = 0; s2 < Z::KL; ++s2) a1[s2] = relu(a1[s2]);
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(L.V.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, L.w2, lane);
    const float rstd = ln_center_r32<LD>(acc, f0, eps);
    float y[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      const f32x4 m = *reinterpret_cast<const f32x4*>(L.V.g + f0 + 4 * ob) * (acc[ob] * rstd) +
                      *reinterpret_cast<const f32x4*>(L.V.bt + f0 + 4 * ob);
#pragma unroll
      for (int r = 0; r < 4; ++r) y[4 * ob + r] = m[r];
      acc[ob] = m;
    }
    if (live) store_row32<LD>(h_out + (size_t)v * LD + f0, acc);
    if (EMIT) {
      const int oz = opaque_zero();
      f32x4 ps[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = ps[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      gemm32<LD>(ps, y, nx.F1s + oz, lane);
      gemm32<LD>(acc, y, nx.F1r + oz, lane);
      if (live) {
        float* p = P_out + (size_t)v * (2 * LD) + f0;
        store_row32<LD>(p, ps);
        store_row32<LD>(p + LD, acc);
      }
    }
  }
}

// Reverse from ybar = dL/dh0: the forward recomputed (z1 bitwise), the
// LayerNorm reverse, dz1 = (W2^T dz2) where z1 > 0, gin = W1^T dz1 (when gin
// is given, [N][8]); the a1 and dz2 rows go to a1s / dz2s for dW2 (by
// launch_wgrad_r32); dW1 = sum dz1 x^T, db1, db2, dgamma, dbeta as column
// sums, written per block in the encoder's parameter order with W2 left out:
// [LD][8] dW1, [LD] db1, then [LD] db2, dgamma, dbeta.
template <int LD>
struct __attribute__((aligned(16))) NodeEncBwdLds {
  NodeEncVec<LD> V;
  __attribute__((aligned(16))) float red[NK + 4][R32_NW][LD];  // dW1 columns k, db1, db2, dgamma, dbeta
};

template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_node_enc_bwd_r32(int64_t N, const float* __restrict__ x_in, const float* __restrict__ ybar, MlpW w, float eps,
                   float* __restrict__ gin, float* __restrict__ a1s, float* __restrict__ dz2s, Partials part) {
  typedef R32<LD> Z;
  __shared__ __align__(16) NodeEncBwdLds<LD> S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_node_enc_vec<LD>(S.V, w, tid);
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  const int f0 = Z::KL * g;
  ColSum32<LD> cw1[NK], cb1, cb2, cg, cbt;
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const bool live = u * 16 + i < N;
    const int64_t v = min(u * 16 + i, N - 1);
    const size_t orow = (size_t)v * LD + f0;
    const float4 xa = *reinterpret_cast<const float4*>(x_in + v * NK);
    const float4 xb = *reinterpret_cast<const float4*>(x_in + v * NK + 4);
    float yb[Z::KL];
    load_row32<LD>(yb, ybar + orow);
    const NodeEncBwdLds<LD>& L = fresh(S);
    const int oz = opaque_zero();
    float a1[Z::KL];
    node_enc_z1<LD>(L.V, xa, xb, f0, a1);
    uint64_t mask = 0;
#pragma unroll
    for (int s2 = 0; s2 < Z::KL; ++s2) {
      if (a1[s2] > 0.f) mask |= 1ull << s2;
      a1[s2] = relu(a1[s2]);
    }
    if (live) {
      float* p = a1s + orow;
#pragma unroll
      for (int c = 0; c < Z::KC; ++c)
        *reinterpret_cast<f32x4*>(p + 4 * c) = f32x4{a1[4 * c], a1[4 * c + 1], a1[4 * c + 2], a1[4 * c + 3]};
    }
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(L.V.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, w.F2 + oz, lane);
    const float rstd = ln_center_r32<LD>(acc, f0, eps);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] *= rstd;  // xhat
    f32x4 t[Z::NOB];
    {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        t[ob] = f32x4{yb[4 * ob], yb[4 * ob + 1], yb[4 * ob + 2], yb[4 * ob + 3]};
        p[ob] = live ? t[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      cbt.add(p, i);
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = live ? t[ob] * acc[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      cg.add(p, i);
    }
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      t[ob] *= *reinterpret_cast<const f32x4*>(L.V.g + f0 + 4 * ob);  // dxh
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s1 += t[ob][r];
        s2 += t[ob][r] * acc[ob][r];
      }
    }
    const float m1 = sum_q(s1) * (1.0f / Z::DR), m2 = sum_q(s2) * (1.0f / Z::DR);
    float dz[Z::KL];
    {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = (Z::DR == LD || f0 + 4 * ob + r < Z::DR) ? rstd * (t[ob][r] - m1 - acc[ob][r] * m2) : 0.f;
          dz[4 * ob + r] = d;
          p[ob][r] = live ? d : 0.f;
        }
      cb2.add(p, i);
      if (live) store_row32<LD>(dz2s + orow, p);
    }
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    gemm32<LD>(acc, dz, w.F2t + oz, lane);
    f32x4 d1[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) d1[ob][r] = (mask >> (4 * ob + r)) & 1ull && live ? acc[ob][r] : 0.f;
    cb1.add(d1, i);
    const float xs[NK] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
    float gi[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = d1[ob] * xs[k];
      cw1[k].add(p, i);
      gi[k] = 0.f;
    }
    if (gin) {
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float4 wa = L.V.w1[f0 + 4 * ob + r][0], wb = L.V.w1[f0 + 4 * ob + r][1];
          const float d = d1[ob][r];
          gi[0] += wa.x * d;
          gi[1] += wa.y * d;
          gi[2] += wa.z * d;
          gi[3] += wa.w * d;
          gi[4] += wb.x * d;
          gi[5] += wb.y * d;
          gi[6] += wb.z * d;
          gi[7] += wb.w * d;
        }
#pragma unroll
      for (int k = 0; k < NK; ++k) gi[k] = sum_q(gi[k]);
      if (live && g == 0) {
        *reinterpret_cast<f32x4*>(gin + v * NK) = f32x4{gi[0], gi[1], gi[2], gi[3]};
        *reinterpret_cast<f32x4*>(gin + v * NK + 4) = f32x4{gi[4], gi[5], gi[6], gi[7]};
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NK; ++k) cw1[k].put(S.red[k][wv], f0, i);
  cb1.put(S.red[NK][wv], f0, i);
  cb2.put(S.red[NK + 1][wv], f0, i);
  cg.put(S.red[NK + 2][wv], f0, i);
  cbt.put(S.red[NK + 3][wv], f0, i);
  __syncthreads();
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  for (int idx = tid; idx < (NK + 4) * LD; idx += R32_NT) {
    // [LD][8] dW1 (feature-major), then the four vectors
    const int k = idx < NK * LD ? idx % NK : NK + (idx - NK * LD) / LD;
    const int c = idx < NK * LD ? idx / NK : (idx - NK * LD) % LD;
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) s += S.red[k][u][c];
    base[idx] = s;
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kNodeRows32Blocks = 256;

hipError_t launch_node_fwd_r32(int lat, int64_t N, const float* h_in, const float* agg, const MlpW& w,
                               const MlpW* nx, float eps, float* h_out, float* P_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F1 || !w.F1a || !w.F2 || (nx && (!nx->F1s || !nx->F1r || !P_out)))
    return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kNodeRows32Blocks);
  if (g >= 8) g &= ~7;
  const MlpW nn = nx ? *nx : w;
#define F(L)                                                                                                     \
  if (nx)                                                                                                        \
    hipLaunchKernelGGL((k_node_fwd_r32<L, true>), dim3(g), dim3(R32_NT), 0, s, N, h_in, agg, w, nn, eps, h_out, \
                       P_out);                                                                                   \
  else                                                                                                           \
    hipLaunchKernelGGL((k_node_fwd_r32<L, false>), dim3(g), dim3(R32_NT), 0, s, N, h_in, agg, w, nn, eps, h_out, \
                       P_out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_node_bwd_r32(int lat, int64_t N, const float* h, const float* agg, const float* hbar_in,
                               const MlpW& w, float eps, float* hbar_part, float* aggbar, float* streams,
                               const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F1 || !w.F1a || !w.F2 || !w.F1t || !w.F1at || !w.F2t ||
      part.stride < 4LL * lat)
    return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, std::min(kNodeRows32Blocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  float* a1s = streams;
  float* dz2s = streams + (size_t)N * lat;
  float* dz1s = streams + (size_t)2 * N * lat;
#define F(L)                                                                                                    \
  hipLaunchKernelGGL(k_node_bwd_r32<L>, dim3(g), dim3(R32_NT), 0, s, N, h, agg, hbar_in, w, eps, hbar_part,     \
                     aggbar, a1s, dz2s, dz1s, part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_node_srcsum_r32(int lat, int64_t N, const int32_t* rowptr, const int32_t* rev, const float* zbar,
                                  const float* R, const float* hbar_part, const MlpW& w, float* hbar_out,
                                  float* S_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F1st || !w.F1rt) return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kNodeRows32Blocks);
  if (g >= 8) g &= ~7;
#define F(L)                                                                                                    \
  hipLaunchKernelGGL(k_node_srcsum_r32<L>, dim3(g), dim3(R32_NT), 0, s, N, rowptr, rev, zbar, R, hbar_part, w, \
                     hbar_out, S_out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_decoder_r32(int lat, int64_t N, const float* h, const MlpW& w, float* out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F1) return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kNodeRows32Blocks);
  if (g >= 8) g &= ~7;
#define F(L) hipLaunchKernelGGL(k_decoder_r32<L>, dim3(g), dim3(R32_NT), 0, s, N, h, w, out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_decoder_bwd_r32(int lat, int64_t N, const float* h, const float* gout, const MlpW& w, float* hbar,
                                  float* dz1s, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F1 || !w.F1t || part.stride < 5LL * lat + 4) return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, std::min(kNodeRows32Blocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
#define F(L) hipLaunchKernelGGL(k_decoder_bwd_r32<L>, dim3(g), dim3(R32_NT), 0, s, N, h, gout, w, hbar, dz1s, part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_node_enc_r32(int lat, int64_t N, const float* x, const MlpW& w, const MlpW* nx, float eps,
                               float* h_out, float* P_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F2 || (nx && (!nx->F1s || !nx->F1r || !P_out))) return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kNodeRows32Blocks);
  if (g >= 8) g &= ~7;
  const MlpW nn = nx ? *nx : w;
#define F(L)                                                                                                  \
  if (nx)                                                                                                     \
    hipLaunchKernelGGL((k_node_enc_r32<L, true>), dim3(g), dim3(R32_NT), 0, s, N, x, w, nn, eps, h_out, P_out); \
  else                                                                                                        \
    hipLaunchKernelGGL((k_node_enc_r32<L, false>), dim3(g), dim3(R32_NT), 0, s, N, x, w, nn, eps, h_out, P_out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_node_enc_bwd_r32(int lat, int64_t N, const float* x, const float* ybar, const MlpW& w, float eps,
                                   float* gin, float* streams, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if ((lat != 128 && lat != 160) || !w.F2 || !w.F2t || part.stride < (int64_t)(NK + 4) * lat)
    return hipErrorInvalidValue;
  const int64_t need = ((N + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, std::min(kNodeRows32Blocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  float* a1s = streams;
  float* dz2s = streams + (size_t)N * lat;
#define F(L)                                                                                                   \
  hipLaunchKernelGGL(k_node_enc_bwd_r32<L>, dim3(g), dim3(R32_NT), 0, s, N, x, ybar, w, eps, gin, a1s, dz2s, \
                     part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

}  // namespace mgn
