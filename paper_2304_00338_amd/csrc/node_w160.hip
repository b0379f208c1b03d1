// Node phase of one MGN message-passing step, bf16 operands, at the
// latent width 150 computed 160 wide (App. C: the 3D model; padded features
// are exactly zero), in the lane layout of w160_common.hpp (Sec. 2.1: every
// node latent is updated by the node MLP from itself and the sum of its
// incoming messages, with a residual connection; the first layer of the next
// edge MLP is split into per-node products).
//
//   k_node_bwd_w160    one wave per 16-node unit: recomputes the MLP from h
//                      and agg, writes a1 = relu(z1), dz2 = dL/dz2 and
//                      dz1 = dL/dz1 (bf16 streams for the weight gradients),
//                      hbar_part = hbar_in + W1h^T dz1 (the residual
//                      included), aggbar = W1a^T dz1, and per-block partials
//                      of dgamma, dbeta
//   k_wgrad_node_w160  dW1 = sum dz1^T [h; agg], db1 (pass 0) and
//                      dW2 = sum dz2^T a1, db2 (pass 1) from those streams
//   k_node_fwd_w160    the forward: h_out = h + LN(W2 relu(W1 [h; agg] + b1)
//                      + b2) over the 150 real features
//   k_emit_w160        P = [W1s h; W1r h] of the next edge layer
//   k_srcsum_w160      per-sender sums S of the edge MLP's zbar (over the
//                      reversed in-edges, in edge order) and hbar_out =
//                      hbar_part + W1s^T S + W1r^T R; writes S for pass 2
//                      of k_wgrad_node_w160 (dW1s = sum S h^T, dW1r =
//                      sum R h^T)
//
// W1 = [W1h W1a] (the columns acting on h and on agg), each block and W2
// staged row-permuted in the rotated layout (153.6 KB of LDS).
#include "w160_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

namespace w160 {
struct __attribute__((aligned(16))) NodeLds {
  __attribute__((aligned(16))) bf16 W1h[L * L];
  __attribute__((aligned(16))) bf16 W1a[L * L];
  __attribute__((aligned(16))) bf16 W2[L * L];
  __attribute__((aligned(16))) float b1[L];
  __attribute__((aligned(16))) float b2[L];
  __attribute__((aligned(16))) float g[L];
  __attribute__((aligned(16))) float bt[L];
};

__device__ __forceinline__ void stage_node(NodeLds& S, const MlpW& w, int tid, bool beta) {
  stage_rot(S.W1h, (const bf16*)w.W1p, tid);
  stage_rot(S.W1a, (const bf16*)w.W1ap, tid);
  stage_rot(S.W2, (const bf16*)w.W2p, tid);
  if (tid < L) {
    S.b1[tid] = w.b1[tid];
    S.b2[tid] = w.b2[tid];
    S.g[tid] = w.gamma[tid];
    S.bt[tid] = beta ? w.beta[tid] : 0.f;
  }
}

// The ten C-layout fragments of one fp32 [.][160] row (p: the row plus the
// lane's 8q).
__device__ __forceinline__ void load_row10(const float* p, f32x4 (&v)[NOB]) {
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) v[ob] = *reinterpret_cast<const f32x4*>(p + fo0(ob));
}
__device__ __forceinline__ void store_row10(float* p, const f32x4 (&v)[NOB]) {
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) *reinterpret_cast<f32x4*>(p + fo0(ob)) = v[ob];
}
// Five bf16 runs of one [.][160] row (p: the row plus the lane's 8q).
__device__ __forceinline__ void store_runs5(bf16* p, const bf16x8 (&v)[NS]) {
#pragma unroll
  for (int s = 0; s < NS; ++s) *reinterpret_cast<uint4*>(p + 32 * s) = __builtin_bit_cast(uint4, v[s]);
}

// z1 = b1 + W1h x_h + W1a x_a (x[s]: run s of h for s < 5, of agg for s >= 5).
__device__ __forceinline__ void node_z1(const NodeLds& S, const bf16* W1h, const bf16* W1a, const RotOff& RO,
                                        const bf16x8 (&x)[2 * NS], int q, f32x4 (&acc)[NOB]) {
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b1 + 8 * q + fo0(ob));
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W1h, ob, s), x[s], acc[ob], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W1a, ob, s), x[NS + s], acc[ob], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// z2 = b2 + W2 a1.
__device__ __forceinline__ void node_z2(const NodeLds& S, const bf16* W2, const RotOff& RO, const bf16x8 (&a1)[NS],
                                        int q, f32x4 (&acc)[NOB]) {
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + 8 * q + fo0(ob));
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W2, ob, s), a1[s], acc[ob], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// acc += W^T v for the lane's five runs v (W: a staged [160][160] block).
__device__ __forceinline__ void prod_t(const bf16* W, const RotOff& RO, const bf16x8 (&v)[NS], f32x4 (&acc)[NOB]) {
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.t_frag(W, ob, s), v[s], acc[ob], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// LayerNorm statistics of the row over the 150 real features (padded
// features of z2 are exactly 0); acc becomes xhat.  Returns rstd.
__device__ __forceinline__ float ln_xhat150(f32x4 (&acc)[NOB], const int (&lv)[2], float eps) {
  float sm = 0.f;
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm += acc[ob][r];
  const float mean = sum_rowlanes(sm) * (1.0f / LR);
  float sq = 0.f;
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) {
    acc[ob] -= mean;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool live = ob < 8 || ((lv[ob - 8] >> r) & 1);
      sq += live ? acc[ob][r] * acc[ob][r] : 0.f;
    }
  }
  const float rstd = __builtin_amdgcn_rsqf(sum_rowlanes(sq) * (1.0f / LR) + eps);
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] *= rstd;
  return rstd;
}
}  // namespace w160

// ===================================================================== reverse
// Per-block partials of dgamma (at 3 L^2 + 2 L) and dbeta (at 3 L^2 + 3 L),
// the parameter order of the node MLP.  hbar_part may alias hbar_in.
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_node_bwd_w160(int64_t N, const float* __restrict__ h, const float* __restrict__ agg, const float* hbar_in, MlpW w,
                float eps, float* hbar_part, float* __restrict__ aggbar, bf16* __restrict__ a1_out,
                bf16* __restrict__ dz2_out, bf16* __restrict__ dz1_out, Partials part) {
  using namespace w160;
  __shared__ __align__(16) NodeLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_node(S, w, tid, false);
  const int lv[2] = {live_bits(8, q), live_bits(9, q)};
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range(nu, wv);
  // column sums: main part (lane i: features fo(i/2, q) + 2 (i%2) + {0, 1})
  // and tail (lane i: feature tail_feature(i, q))
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  float tga = 0.f, tbe = 0.f;
  // the lane's row of unit u clamped into [0, N), plus its 8q
  auto rowp = [&](int64_t u) -> int64_t { return min(u * 16 + i, N - 1) * L + 8 * q; };
  // x[s]: the bf16 runs of h (s < 5) and agg (s >= 5) of the unit; the next
  // unit's h is in flight from the first product to the W1^T products, its
  // agg from there to the next unit (the registers do not hold both in fp32
  // beside a unit's working set)
  auto pack5 = [&](const f32x4 (&v)[NOB], bf16x8* x) {
#pragma unroll
    for (int s = 0; s < NS; ++s) x[s] = pack_run(v[2 * s], v[2 * s + 1]);
  };
  if (ur.t < ur.end) {
    bf16x8 x[2 * NS];
    f32x4 an[NOB];
    {
      f32x4 hn[NOB];
      load_row10(h + rowp(ur.t), hn);
      load_row10(agg + rowp(ur.t), an);
      pack5(hn, x);
    }
    for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
      pack5(an, x + NS);
      const bool ok = u * 16 + i < N;
      const int64_t p = rowp(u);
      // per-unit opaque offsets: staged-weight reads are not hoisted out of the loop
      const int oz = opaque_zero();
      const bf16* W1h = S.W1h + oz;
      const bf16* W1a = S.W1a + oz;
      const bf16* W2s = S.W2 + oz;
      f32x4 hb[NOB];
      load_row10(hbar_in + p, hb);
      // ---- z1, the mask z1 > 0 (bit 4 ob + r of mlo / mhi), a1 = relu(z1)
      f32x4 acc[NOB];
      node_z1(S, W1h, W1a, RotOff(i + oz, q), x, q, acc);
      f32x4 hn[NOB];
      load_row10(h + rowp(u + ur.stride), hn);
      uint32_t mlo = 0, mhi = 0;
      bf16x8 a1[NS];
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t b = acc[ob][r] > 0.f ? 1u : 0u;
          if (ob < 8)
            mlo |= b << (4 * ob + r);
          else
            mhi |= b << (4 * (ob - 8) + r);
        }
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          a1[s][r] = (bf16)relu(acc[2 * s][r]);
          a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
        }
      if (ok) store_runs5(a1_out + p, a1);
      // ---- z2 and its LayerNorm over the 150 real features
      node_z2(S, W2s, RotOff(i + oz, q), a1, q, acc);
      const float rstd = ln_xhat150(acc, lv, eps);  // acc = xhat
      // rows past N contribute nothing
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) hb[ob][r] = ok ? hb[ob][r] : 0.f;
      // ---- dbeta += sum_rows hbar_in
      {
        const float2 d = colsum16(reinterpret_cast<const f32x4(&)[8]>(hb), i);
        dbe.x += d.x;
        dbe.y += d.y;
        tbe += colsum16_tail(hb, i);
      }
      // ---- dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = hbar_in gamma,
      // 0 on padded features
      bf16x8 dz2[NS];
      {
        const float* gq = S.g + 8 * q;
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          const f32x4 dxh = hb[ob] * *reinterpret_cast<const f32x4*>(gq + fo0(ob));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            s1 += dxh[r];
            s2 += dxh[r] * acc[ob][r];
          }
        }
        const float m1 = sum_rowlanes(s1) * (1.0f / LR), m2 = sum_rowlanes(s2) * (1.0f / LR);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          f32x4 v[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int ob = 2 * s + hh;
            const f32x4 dxh = hb[ob] * *reinterpret_cast<const f32x4*>(gq + fo0(ob));
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = ob < 8 || ((lv[ob - 8] >> r) & 1);
              v[hh][r] = live ? rstd * (dxh[r] - m1 - acc[ob][r] * m2) : 0.f;
            }
          }
          dz2[s] = pack_run(v[0], v[1]);
        }
      }
      if (ok) store_runs5(dz2_out + p, dz2);
      // ---- dgamma += sum_rows hbar_in xhat (in place: xhat is not used again)
      {
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) acc[ob] *= hb[ob];
        const float2 c = colsum16(reinterpret_cast<const f32x4(&)[8]>(acc), i);
        dga.x += c.x;
        dga.y += c.y;
        tga += colsum16_tail(acc, i);
      }
      // ---- dz1 = (W2^T dz2) where z1 > 0
      const RotOff RO(i + oz, q);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      prod_t(W2s, RO, dz2, acc);
      bf16x8 dz1[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ob = 2 * s + hh;
            const bool on = ob < 8 ? (mlo >> (4 * ob + r)) & 1u : (mhi >> (4 * (ob - 8) + r)) & 1u;
            dz1[s][4 * hh + r] = on ? (bf16)acc[ob][r] : (bf16)0.f;
          }
      if (ok) store_runs5(dz1_out + p, dz1);
      // ---- the next unit's operands
      pack5(hn, x);
      load_row10(agg + rowp(u + ur.stride), an);
      // ---- hbar_part = hbar_in + W1h^T dz1, aggbar = W1a^T dz1
      prod_t(W1h, RO, dz1, hb);
      if (ok) store_row10(hbar_part + p, hb);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      prod_t(W1a, RO, dz1, acc);
      if (ok) store_row10(aggbar + p, acc);
    }
  }
  // ---- block partials of dgamma, dbeta: the 8 waves' sums in wave order
  __syncthreads();
  float* red = reinterpret_cast<float*>(S.W1h);  // [2][NW][L]
  {
    const int fm = fo(i >> 1, q) + 2 * (i & 1), ft = tail_feature(i, q);
    float* r0 = red + wv * L;
    float* r1 = red + (NW + wv) * L;
    *reinterpret_cast<float2*>(r0 + fm) = dga;
    *reinterpret_cast<float2*>(r1 + fm) = dbe;
    if ((i & 1) == 0) {  // lanes i and i ^ 1 hold the same tail sums
      r0[ft] = tga;
      r1[ft] = tbe;
    }
  }
  __syncthreads();
  float* base = part.buf + (size_t)blockIdx.x * part.stride + 3 * L * L + 2 * L;
  for (int idx = tid; idx < 2 * L; idx += NT) {
    const int k = idx / L, f = idx % L;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * L + f];
    base[idx] = v;
  }
}

// Weight gradients of the node MLP from the streams of k_node_bwd_w160, as
// per-block partials in the parameter order of the node MLP: pass 0 dW1
// [160][320] at 0 (dz1^T [h; agg], h and agg rounded to bf16 as in the
// forward product) and db1 at 2 L^2; pass 1 dW2 at 2 L^2 + L and db2 at
// 3 L^2 + L.  32-row chunks of the streams are staged row-major in
// LDS (rows 176 elements apart: the transposing reads are free of bank
// conflicts) while the next chunk is in flight in registers; wave w owns
// output rows [16w, 16w + 16).  Both passes use the same grid.
namespace w160 {
constexpr int WN_NT = 640;
}  // namespace w160

// Pass 2 (the edge MLP's sender / receiver blocks): dW1s = sum S h^T at 0 and
// dW1r = sum R h^T at L^2 (S: bf16 stream in dz, R: fp32 in agg, rounded to
// bf16 as operands), wave w owning output rows [16w, 16w + 16) of both.
template <int PASS>
__global__ void __launch_bounds__(w160::WN_NT) k_wgrad_node_w160(int64_t N, const float* __restrict__ h,
                                                                const float* __restrict__ agg,
                                                                const bf16* __restrict__ dz,
                                                                const bf16* __restrict__ a1, Partials part) {
  using namespace w160;
  // staged streams: dz1, h, agg / dz2, a1 / S, R, h
  constexpr int NSTR = PASS == 1 ? 2 : 3;
  constexpr int NCB = PASS == 1 ? NOB : 2 * NOB;
  __shared__ __align__(16) bf16 Sg[2][NSTR][TM * WG_LD];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int jp = i >> 2, c4 = i & 3;
  f32x4 acc[NCB], ab = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 ones;
#pragma unroll
  for (int j = 0; j < 8; ++j) ones[j] = (bf16)1.f;
  const int64_t nch = (N + TM - 1) / TM, G = gridDim.x;
  // staging: thread tid moves 8 elements of row srow of every stream
  const int srow = tid / (L / 8), scol = (tid % (L / 8)) * 8;
  uint4 Ld[NSTR];
  auto cvt8 = [](float4 a, float4 b) -> uint4 {
    bf16x8 v;
    v[0] = (bf16)a.x;
    v[1] = (bf16)a.y;
    v[2] = (bf16)a.z;
    v[3] = (bf16)a.w;
    v[4] = (bf16)b.x;
    v[5] = (bf16)b.y;
    v[6] = (bf16)b.z;
    v[7] = (bf16)b.w;
    return __builtin_bit_cast(uint4, v);
  };
  // rows past N read row N - 1 with zero gradients (so they add nothing);
  // the zeroing is per component
  auto issue = [&](int64_t ch) {
    const int64_t r = ch * TM + srow;
    const bool ok = r < N;
    const int64_t rc = ok ? r : N - 1;
    const uint4 v = ld_stream(dz + rc * L + scol);
    Ld[0].x = ok ? v.x : 0u;
    Ld[0].y = ok ? v.y : 0u;
    Ld[0].z = ok ? v.z : 0u;
    Ld[0].w = ok ? v.w : 0u;
    if constexpr (PASS == 0) {
      const float* hp = h + rc * L + scol;
      const float* gp = agg + rc * L + scol;
      Ld[1] = cvt8(*reinterpret_cast<const float4*>(hp), *reinterpret_cast<const float4*>(hp + 4));
      Ld[2] = cvt8(*reinterpret_cast<const float4*>(gp), *reinterpret_cast<const float4*>(gp + 4));
    } else if constexpr (PASS == 1) {
      Ld[1] = ld_stream(a1 + rc * L + scol);
    } else {
      // R rows past N are zeroed like S; h rows are then multiplied by zero
      const float* gp = agg + rc * L + scol;
      const float* hp = h + rc * L + scol;
      const uint4 v = cvt8(*reinterpret_cast<const float4*>(gp), *reinterpret_cast<const float4*>(gp + 4));
      Ld[1].x = ok ? v.x : 0u;
      Ld[1].y = ok ? v.y : 0u;
      Ld[1].z = ok ? v.z : 0u;
      Ld[1].w = ok ? v.w : 0u;
      Ld[2] = cvt8(*reinterpret_cast<const float4*>(hp), *reinterpret_cast<const float4*>(hp + 4));
    }
  };
  // operand of 16 columns col0.. with K = the chunk's rows q*8 + j
  auto frag = [&](const bf16* X, int col0) -> bf16x8 {
    const bf16* p = X + (q * 8 + jp) * WG_LD + col0 + 4 * c4;
    return cat8(lds_tr(p), lds_tr(p + 4 * WG_LD));
  };
  int64_t c = blockIdx.x;
  int buf = 0;
  if (c < nch) issue(c);
  for (; c < nch; c += G) {
#pragma unroll
    for (int k = 0; k < NSTR; ++k) *reinterpret_cast<uint4*>(&Sg[buf][k][srow * WG_LD + scol]) = Ld[k];
    __syncthreads();
    if (c + G < nch) issue(c + G);
    if constexpr (PASS == 2) {
      const bf16x8 as = frag(Sg[buf][0], 16 * w), ar = frag(Sg[buf][1], 16 * w);
#pragma unroll
      for (int cb = 0; cb < NOB; ++cb) {
        const bf16x8 bh = frag(Sg[buf][2], 16 * cb);
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as, bh, acc[cb], 0, 0, 0);
        acc[NOB + cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar, bh, acc[NOB + cb], 0, 0, 0);
      }
    } else {
      const bf16x8 az = frag(Sg[buf][0], 16 * w);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az, frag(Sg[buf][1 + cb / NOB], 16 * (cb % NOB)), acc[cb],
                                                          0, 0, 0);
      ab = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az, ones, ab, 0, 0, 0);
    }
    buf ^= 1;
  }
  float* blk = part.buf + (size_t)blockIdx.x * part.stride;
  if constexpr (PASS == 2) {
    // dW1s [160][160] at 0, dW1r at L^2
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = w * 16 + q * 4 + r;
#pragma unroll
      for (int cb = 0; cb < NOB; ++cb) {
        blk[(size_t)o * L + cb * 16 + i] = acc[cb][r];
        blk[L * L + (size_t)o * L + cb * 16 + i] = acc[NOB + cb][r];
      }
    }
  } else {
    // dW1: columns cb * 16 (cb < 10: the h block, else the agg block at 160 +);
    // dW2: columns cb * 16
    constexpr int ld = PASS == 0 ? 2 * L : L;
    float* base = blk + (PASS == 0 ? 0 : 2 * L * L + L);
    float* bias = blk + (PASS == 0 ? 2 * L * L : 3 * L * L + L);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = w * 16 + q * 4 + r;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) base[(size_t)o * ld + cb * 16 + i] = acc[cb][r];
      if (i == 0) bias[o] = ab[r];
    }
  }
}


// ===================================================================== forward
// h_out = h_in + LN(MLP([h_in, agg])); h_out may alias h_in (each row is
// read before it is written, by the same lane).
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_node_fwd_w160(int64_t N, const float* h_in, const float* __restrict__ agg, MlpW w, float eps, float* h_out) {
  using namespace w160;
  __shared__ __align__(16) NodeLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_node(S, w, tid, true);
  const int lv[2] = {live_bits(8, q), live_bits(9, q)};
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range(nu, wv);
  if (ur.t >= ur.end) return;
  auto rowp = [&](int64_t u) -> int64_t { return min(u * 16 + i, N - 1) * L + 8 * q; };
  auto pack5 = [&](const f32x4 (&v)[NOB], bf16x8* x) {
#pragma unroll
    for (int s = 0; s < NS; ++s) x[s] = pack_run(v[2 * s], v[2 * s + 1]);
  };
  // hr: the unit's h rows in fp32 (the residual); the next unit's h is in
  // flight from the first product on, its agg from the LayerNorm on
  f32x4 hr[NOB], an[NOB];
  load_row10(h_in + rowp(ur.t), hr);
  load_row10(agg + rowp(ur.t), an);
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const int64_t p = rowp(u);
    const int oz = opaque_zero();
    bf16x8 x[2 * NS];
    pack5(hr, x);
    pack5(an, x + NS);
    f32x4 acc[NOB];
    node_z1(S, S.W1h + oz, S.W1a + oz, RotOff(i + oz, q), x, q, acc);
    f32x4 hn[NOB];
    load_row10(h_in + rowp(u + ur.stride), hn);
    bf16x8 a1[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        a1[s][r] = (bf16)relu(acc[2 * s][r]);
        a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
      }
    node_z2(S, S.W2 + oz, RotOff(i + oz, q), a1, q, acc);
    ln_xhat150(acc, lv, eps);
    load_row10(agg + rowp(u + ur.stride), an);
    const float* gq = S.g + 8 * q;
    const float* bq = S.bt + 8 * q;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = hr[ob] + (*reinterpret_cast<const f32x4*>(gq + fo0(ob)) * acc[ob] +
                          *reinterpret_cast<const f32x4*>(bq + fo0(ob)));
    if (u * 16 + i < N) store_row10(h_out + p, acc);
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) hr[ob] = hn[ob];
  }
}

// P[v] = [W1s h[v]; W1r h[v]] in bf16 for the next edge layer (W1s, W1r:
// its row-permuted sender / receiver column blocks, rotated in LDS).
namespace w160 {
struct __attribute__((aligned(16))) EmitLds {
  __attribute__((aligned(16))) bf16 Ws[L * L];
  __attribute__((aligned(16))) bf16 Wr[L * L];
};
}  // namespace w160

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_emit_w160(int64_t N, const float* __restrict__ h, MlpW nx, bf16* __restrict__ P) {
  using namespace w160;
  __shared__ __align__(16) EmitLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_rot(S.Ws, (const bf16*)nx.W1sp, tid);
  stage_rot(S.Wr, (const bf16*)nx.W1rp, tid);
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range(nu, wv);
  if (ur.t >= ur.end) return;
  auto rowp = [&](int64_t u) -> int64_t { return min(u * 16 + i, N - 1) * L + 8 * q; };
  f32x4 hv[NOB];
  load_row10(h + rowp(ur.t), hv);
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const int oz = opaque_zero();
    const RotOff RO(i + oz, q);
    bf16x8 x[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) x[s] = pack_run(hv[2 * s], hv[2 * s + 1]);
    load_row10(h + rowp(u + ur.stride), hv);
    const bool ok = u * 16 + i < N;
    bf16* out = P + min(u * 16 + i, N - 1) * (2 * L) + 8 * q;
#pragma unroll
    for (int part = 0; part < 2; ++part) {
      const bf16* W = (part == 0 ? S.Ws : S.Wr) + oz;
      f32x4 acc[NOB];
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W, ob, s), x[s], acc[ob], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      bf16x8 o[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s) o[s] = pack_run(acc[2 * s], acc[2 * s + 1]);
      if (ok) store_runs5(out + part * L, o);
    }
  }
}


// Per-sender sums of the edge MLP's zbar and the node gradient they feed:
// S[v] = sum of zbar over the reversed in-edges of v (the out-edges of v in
// a graph whose every edge has its reverse), in edge order from 0.0 in fp32;
// hbar_out = hbar_part + W1s^T S + W1r^T R (S and R rounded to bf16 as
// operands).  S is written in bf16 for the weight-gradient pass.
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_srcsum_w160(int64_t N, const int32_t* __restrict__ rowptr, const int32_t* __restrict__ rev,
              const bf16* __restrict__ zbar, const float* __restrict__ R, const float* __restrict__ hbar_part,
              MlpW w, float* __restrict__ hbar_out, bf16* __restrict__ S_out) {
  using namespace w160;
  __shared__ __align__(16) EmitLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_rot(S.Ws, (const bf16*)w.W1sp, tid);
  stage_rot(S.Wr, (const bf16*)w.W1rp, tid);
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const UnitRange ur = unit_range(nu, wv);
  constexpr int UE = 4;  // in-edges gathered per step
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const int64_t v = u * 16 + i;
    const bool ok = v < N;
    const int64_t vc = ok ? v : N - 1;
    const int e0 = rowptr[vc], deg = ok ? rowptr[vc + 1] - e0 : 0;
    int md = deg;  // the unit's largest in-degree (the 4 lane groups hold the same nodes)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) md = max(md, __shfl_xor(md, off, 16));
    f32x4 sacc[NOB];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) sacc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < md; k0 += UE) {
      uint4 zr[UE][NS];
#pragma unroll
      for (int k = 0; k < UE; ++k) {
        // past the node's in-degree: the node's first reversed edge (or edge
        // 0 for a node without in-edges), not added
        const int kk = k0 + k < deg ? k0 + k : 0;
        const int e = deg > 0 ? rev[e0 + kk] : 0;
        const bf16* zp = zbar + (size_t)e * L + 8 * q;
#pragma unroll
        for (int s = 0; s < NS; ++s) zr[k][s] = *reinterpret_cast<const uint4*>(zp + 32 * s);
      }
#pragma unroll
      for (int k = 0; k < UE; ++k)
        if (k0 + k < deg) {
#pragma unroll
          for (int ob = 0; ob < NOB; ++ob) sacc[ob] += run_block5(zr[k], ob);
        }
    }
    const int64_t p = vc * L + 8 * q;
    bf16x8 sr[NS], rr[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) sr[s] = pack_run(sacc[2 * s], sacc[2 * s + 1]);
    if (ok) store_runs5(S_out + p, sr);
    {
      f32x4 rv[NOB];
      load_row10(R + p, rv);
#pragma unroll
      for (int s = 0; s < NS; ++s) rr[s] = pack_run(rv[2 * s], rv[2 * s + 1]);
    }
    f32x4 hb[NOB];
    load_row10(hbar_part + p, hb);
    const int oz = opaque_zero();
    const RotOff RO(i + oz, q);
    prod_t(S.Ws + oz, RO, sr, hb);
    prod_t(S.Wr + oz, RO, rr, hb);
    if (ok) store_row10(hbar_out + p, hb);
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kNodeBlocks160 = 256;

hipError_t launch_node_bwd_w160(int64_t N, const float* h, const float* agg, const float* hbar_in, const MlpW& w,
                                float eps, float* hbar_part, float* aggbar, void* a1, void* dz2, void* dz1,
                                const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if (!w.W1p || !w.W1ap || !w.W2p || part.stride < 3 * 160 * 160 + 4 * 160) return hipErrorInvalidValue;
  const int64_t need = (((N + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, std::min(kNodeBlocks160, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  hipLaunchKernelGGL(k_node_bwd_w160, dim3(g), dim3(NT), 0, s, N, h, agg, hbar_in, w, eps, hbar_part, aggbar,
                     (bf16*)a1, (bf16*)dz2, (bf16*)dz1, part);
  return hipGetLastError();
}

hipError_t launch_wgrad_node_w160(int64_t N, const float* h, const float* agg, const void* dz1, const void* dz2,
                                  const void* a1, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if (part.stride < 3 * 160 * 160 + 2 * 160) return hipErrorInvalidValue;
  const int g = grid_for((N + TM - 1) / TM, std::min(512, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_wgrad_node_w160<0>, dim3(g), dim3(w160::WN_NT), 0, s, N, h, agg, (const bf16*)dz1,
                     (const bf16*)nullptr, part);
  hipLaunchKernelGGL(k_wgrad_node_w160<1>, dim3(g), dim3(w160::WN_NT), 0, s, N, h, agg, (const bf16*)dz2,
                     (const bf16*)a1, part);
  return hipGetLastError();
}

hipError_t launch_node_fwd_w160(int64_t N, const float* h_in, const float* agg, const MlpW& w, float eps,
                                float* h_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (!w.W1p || !w.W1ap || !w.W2p) return hipErrorInvalidValue;
  const int64_t need = (((N + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kNodeBlocks160);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_node_fwd_w160, dim3(g), dim3(NT), 0, s, N, h_in, agg, w, eps, h_out);
  return hipGetLastError();
}

hipError_t launch_emit_w160(int64_t N, const float* h, const MlpW& next_edge, void* P, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (!next_edge.W1sp || !next_edge.W1rp) return hipErrorInvalidValue;
  const int64_t need = (((N + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kNodeBlocks160);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_emit_w160, dim3(g), dim3(NT), 0, s, N, h, next_edge, (bf16*)P);
  return hipGetLastError();
}

hipError_t launch_srcsum_w160(int64_t N, const int32_t* rowptr, const int32_t* rev, const void* zbar, const float* R,
                              const float* h, const float* hbar_part, const MlpW& w, float* hbar_out, void* S_buf,
                              const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if (!w.W1sp || !w.W1rp || part.stride < 2 * 160 * 160) return hipErrorInvalidValue;
  const int64_t need = (((N + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kNodeBlocks160);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_srcsum_w160, dim3(g), dim3(NT), 0, s, N, rowptr, rev, (const bf16*)zbar, R, hbar_part, w,
                     hbar_out, (bf16*)S_buf);
  const int gw = grid_for((N + TM - 1) / TM, std::min(512, part.max_blocks));
  *nblocks = gw;
  hipLaunchKernelGGL(k_wgrad_node_w160<2>, dim3(gw), dim3(w160::WN_NT), 0, s, N, h, R, (const bf16*)S_buf,
                     (const bf16*)nullptr, part);
  return hipGetLastError();
}

}  // namespace mgn
