// Edge phase of one MGN message-passing step, reverse, bf16 operands, at the
// latent width 150 computed 160 wide (App. C: the 3D model; padded features
// are exactly zero), with one wave per 16-row half of a receiver-aligned
// tile (Sec. 2.1: every edge latent is updated from itself and its two end
// nodes, every node from the sum of its in-edge messages; this is the
// reverse of that update).
//
// Lane layout and weight staging as in w160_common.hpp.  The forward stages
// its weights in padded rows, the backward W2 and W1e in the rotated layout.
//
// Per half: z2 = b2 + W2 a1 from the saved first-layer activations,
// LayerNorm statistics over the 150 real features, mbar = ebar_in +
// aggbar[receiver], dgamma / dbeta / db2 column sums (DPP butterflies),
// dz2 (written for the weight-gradient pass), zbar = (W2^T dz2) where
// a1 > 0 (written), per-receiver sums of zbar in ascending row order (from a
// per-wave bf16 stage; also db1), ebar_out = ebar_in + W1e^T zbar.  The only
// block barriers stage the weights before the loop and combine the column
// sums after it.
#include "w160_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

namespace w160 {
struct __attribute__((aligned(16))) Lds {
  __attribute__((aligned(16))) bf16 W1[L * L];  // row-permuted W1e, rotated chunks
  __attribute__((aligned(16))) bf16 W2[L * L];  // row-permuted W2, rotated chunks
  __attribute__((aligned(16))) float b2[L];
  __attribute__((aligned(16))) float g[L];
  __attribute__((aligned(16))) bf16 stage[NW][16 * L];
};
}  // namespace w160

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_bwd_w160(EdgeTiles tl, const bf16* __restrict__ a1_in, const bf16* ebar_in, int have_ebar, bf16* ebar_out,
                const float* __restrict__ aggbar, const bf16* __restrict__ W1p, const bf16* __restrict__ W2p,
                const float* __restrict__ b2, const float* __restrict__ gamma,
                float eps, bf16* __restrict__ zbar, bf16* __restrict__ dz_out, float* __restrict__ R,
                float* __restrict__ slots, Partials part) {
  using namespace w160;
  __shared__ __align__(16) Lds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_rot(S.W1, W1p, tid);
  stage_rot(S.W2, W2p, tid);
  if (tid < L) {
    S.b2[tid] = b2[tid];
    S.g[tid] = gamma[tid];
  }
  __syncthreads();

  const UnitRange ur = unit_range(tl.n_tiles, wv);
  int64_t t = ur.t;
  const int64_t stride = ur.stride, tend = ur.end;
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tend - 1];
    int4 r;  // per-component selects (an aggregate select goes through scratch)
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  // the a1 runs of a half are prefetched one half ahead; the incoming edge
  // gradient of a half is loaded when the half starts (first used after the
  // z2 product)
  struct HalfLoads {
    uint4 a[NS];
  };
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto nrows = [](int4 d) { return d.w - d.z; };
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, nrows(d) - 1), 0), lastE); };
  auto load_half = [&](int4 d, int rb, HalfLoads& H, int& recv) {
    const size_t row = (size_t)erow(d, rb);
    recv = tl.receivers[row];
    const bf16* ap = a1_in + row * L + 8 * q;
#pragma unroll
    for (int k = 0; k < NS; ++k) H.a[k] = *reinterpret_cast<const uint4*>(ap + 32 * k);
  };
  auto load_eb = [&](int4 d, int rb, uint4 (&eb)[NS]) {
    const bf16* ep = ebar_in + (size_t)erow(d, rb) * L + 8 * q;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const uint4 v = *reinterpret_cast<const uint4*>(ep + 32 * k);
      eb[k].x = have_ebar ? v.x : 0u;
      eb[k].y = have_ebar ? v.y : 0u;
      eb[k].z = have_ebar ? v.z : 0u;
      eb[k].w = have_ebar ? v.w : 0u;
    }
  };

  // column-sum accumulators: main part (lane i: features fo(i/2, q) + 2 (i%2)
  // + {0, 1}) and tail (lane i: feature tail_feature(i, q))
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f}, db2 = {0.f, 0.f};
  float tga = 0.f, tbe = 0.f, tb2 = 0.f;
  // db1 from the receiver sums: lane: features 2 lane, 2 lane + 1 and, for
  // lanes < 16, 128 + 2 lane, 128 + 2 lane + 1
  float2 db1 = {0.f, 0.f}, db1t = {0.f, 0.f};
  bf16* stage = S.stage[wv];
  const int lv[2] = {w160::live_bits(8, q), w160::live_bits(9, q)};
  const RotOff RO(i, q);

  auto half = [&](const HalfLoads& H, int recv, int4 d0, int rb, int segraw, bool chunk, int nv, int& j,
                  float2& carry, float2& carryt) {
    const int n = nrows(d0);
    const int row = rb * 16 + i;
    const bool ok = row < n;
    // staged weights at an opaque offset: reads of them are not loop-invariant,
    // so they are not hoisted into registers
    const int oz = opaque_zero();
    const bf16* W1s = S.W1 + oz;
    const bf16* W2s = S.W2 + oz;
    // the receiver's aggregate gradient (a gather, mostly from the cache) is
    // in flight during the z2 product: it is first needed after it
    f32x4 ag0[NOB];
    {
      const float* gp = aggbar + (size_t)recv * L;
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) ag0[ob] = *reinterpret_cast<const f32x4*>(gp + fo(ob, q));
    }
    // ---- z2 = b2 + W2 a1 and its LayerNorm statistics (150 real features)
    f32x4 acc[NOB];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + fo(ob, q));
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W2s, ob, s), as_frag(H.a[s]), acc[ob], 0, 0, 0);
      }
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
    // ---- mbar = ebar_in + aggbar[receiver] (zero on rows past the tile)
    f32x4 mb[NOB];
    {
      uint4 eb[NS];
      load_eb(d0, rb, eb);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        const f32x4 ag = ag0[ob];
        mb[ob] = ok ? ag + run_block5(eb, ob) : f32x4{0.f, 0.f, 0.f, 0.f};
        acc[ob] *= rstd;  // xhat
      }
    }
    // ---- dgamma += sum_rows mbar xhat, dbeta += sum_rows mbar
    {
      const float2 d = colsum16(reinterpret_cast<const f32x4(&)[8]>(mb), i);
      dbe.x += d.x;
      dbe.y += d.y;
      tbe += w160::colsum16_tail(mb, i);
      f32x4 p[NOB];
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) p[ob] = mb[ob] * acc[ob];
      const float2 c = colsum16(reinterpret_cast<const f32x4(&)[8]>(p), i);
      dga.x += c.x;
      dga.y += c.y;
      tga += w160::colsum16_tail(p, i);
    }
    // ---- LayerNorm backward: dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)),
    // dxh = mbar gamma (zero on padded features), dz2 = 0 on padded features
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) {
      mb[ob] *= *reinterpret_cast<const f32x4*>(S.g + fo(ob, q));  // dxh
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s1 += mb[ob][r];
        s2 += mb[ob][r] * acc[ob][r];
      }
    }
    const float m1 = sum_rowlanes(s1) * (1.0f / LR), m2 = sum_rowlanes(s2) * (1.0f / LR);
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool live = ob < 8 || ((lv[ob - 8] >> r) & 1);
        acc[ob][r] = live ? rstd * (mb[ob][r] - m1 - acc[ob][r] * m2) : 0.f;
      }
    bf16x8 dzf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) dzf[s] = pack_run(acc[2 * s], acc[2 * s + 1]);
    if (ok) {
      bf16* dp = dz_out + ((size_t)d0.z + row) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s) *reinterpret_cast<uint4*>(dp + 32 * s) = __builtin_bit_cast(uint4, dzf[s]);
    }
    // ---- db2 += sum_rows dz2 (as stored)
    {
      f32x4 v[NOB];
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[2 * s][r] = (float)dzf[s][r];
          v[2 * s + 1][r] = (float)dzf[s][4 + r];
        }
      const float2 c = colsum16(reinterpret_cast<const f32x4(&)[8]>(v), i);
      db2.x += c.x;
      db2.y += c.y;
      tb2 += w160::colsum16_tail(v, i);
    }
    // ---- da1 = W2^T dz2, zbar = da1 where a1 > 0
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.t_frag(W2s, ob, s), dzf[s], acc[ob], 0, 0, 0);
      }
    bf16x8 zf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 a = as_frag(H.a[s]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        zf[s][r] = (float)a[r] > 0.f ? (bf16)acc[2 * s][r] : (bf16)0.f;
        zf[s][4 + r] = (float)a[4 + r] > 0.f ? (bf16)acc[2 * s + 1][r] : (bf16)0.f;
      }
    }
    if (ok) {
      bf16* zp = zbar + ((size_t)d0.z + row) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s) *reinterpret_cast<uint4*>(zp + 32 * s) = __builtin_bit_cast(uint4, zf[s]);
    }
    // ---- per-receiver sums of zbar (as stored) in ascending row order, and db1
    wave_lds_sync();
#pragma unroll
    for (int s = 0; s < NS; ++s) *reinterpret_cast<uint4*>(stage + i * L + 32 * s + 8 * q) = __builtin_bit_cast(uint4, zf[s]);
    wave_lds_sync();
    {
      const int lo_row = rb * 16, hi_row = lo_row + 16;
      const bool tl16 = lane < 16;
      while (j < nv) {
        const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - d0.z;
        const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - d0.z;
        const int u0 = max(a, lo_row), u1 = min(b, hi_row);
        for (int u = u0; u < u1; ++u) {
          const bf16* sr = stage + (u - lo_row) * L;
          typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
          const bf16x2 v = *reinterpret_cast<const bf16x2*>(sr + 2 * lane);
          carry.x += (float)v[0];
          carry.y += (float)v[1];
          if (tl16) {
            const bf16x2 w = *reinterpret_cast<const bf16x2*>(sr + 128 + 2 * lane);
            carryt.x += (float)w[0];
            carryt.y += (float)w[1];
          }
        }
        if (b > hi_row) break;
        float* dst = !chunk ? R + (size_t)(d0.x + j) * L : slots + (size_t)(-1 - d0.y) * L;
        *reinterpret_cast<float2*>(dst + 2 * lane) = carry;
        if (tl16) *reinterpret_cast<float2*>(dst + 128 + 2 * lane) = carryt;
        db1.x += carry.x;
        db1.y += carry.y;
        db1t.x += carryt.x;
        db1t.y += carryt.y;
        carry = float2{0.f, 0.f};
        carryt = float2{0.f, 0.f};
        ++j;
      }
    }
    // ---- ebar_out = ebar_in + W1e^T zbar (the incoming rows again, from the cache)
    {
      uint4 eb[NS];
      load_eb(d0, rb, eb);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = run_block5(eb, ob);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.t_frag(W1s, ob, s), zf[s], acc[ob], 0, 0, 0);
    if (ok) {
      bf16* op = ebar_out + ((size_t)d0.z + row) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(acc[2 * s], acc[2 * s + 1]));
    }
    wave_lds_sync();
  };

  if (t < tend) {
    int4 d0 = desc(t);
    HalfLoads A, B;
    int rA, rB;
    load_half(d0, 0, A, rA);
    for (; t < tend; t += stride) {
      const bool chunk = d0.y < 0;
      const int nv = chunk ? 1 : d0.y - d0.x;
      const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
      const int4 d1 = desc(t + stride);
      load_half(d0, 1, B, rB);
      float2 carry = {0.f, 0.f}, carryt = {0.f, 0.f};
      int j = 0;  // next node whose sum is open
      half(A, rA, d0, 0, segraw, chunk, nv, j, carry, carryt);
      load_half(d1, 0, A, rA);
      half(B, rB, d0, 1, segraw, chunk, nv, j, carry, carryt);
      d0 = d1;
    }
  }
  // ---- block partials [db1 | db2 | dgamma | dbeta], the 8 waves' sums in wave order
  __syncthreads();
  float* red = reinterpret_cast<float*>(S.W2);  // [4][NW][L]
  {
    const int fm = fo(i >> 1, q) + 2 * (i & 1), ft = w160::tail_feature(i, q);
    float* r0 = red + (0 * NW + wv) * L;
    float* r1 = red + (1 * NW + wv) * L;
    float* r2 = red + (2 * NW + wv) * L;
    float* r3 = red + (3 * NW + wv) * L;
    *reinterpret_cast<float2*>(r0 + 2 * lane) = db1;
    if (lane < 16) *reinterpret_cast<float2*>(r0 + 128 + 2 * lane) = db1t;
    *reinterpret_cast<float2*>(r1 + fm) = db2;
    *reinterpret_cast<float2*>(r2 + fm) = dga;
    *reinterpret_cast<float2*>(r3 + fm) = dbe;
    if ((i & 1) == 0) {  // lanes i and i ^ 1 hold the same tail sums
      r1[ft] = tb2;
      r2[ft] = tga;
      r3[ft] = tbe;
    }
  }
  __syncthreads();
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  for (int idx = tid; idx < 4 * L; idx += NT) {
    const int k = idx / L, f = idx % L;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * L + f];
    base[idx] = v;
  }
}

// Forward edge phase at width 160 (bf16), one wave per 16-row half of a
// tile: z1 = b1 + P_s[s] + P_r[r] + W1e e, a1 = relu(z1) (written when the
// caller saves it), z2 = b2 + W2 a1, message m = gamma xhat + beta over the
// 150 real features (padded ones are exactly 0), e_out = e + m, and the
// receiver sums of m in ascending row order from 0.0 (in three slices of
// features, runs {0, 1}, {2, 3}, {4}, staged per wave in fp32).  Row-permuted
// W1e and W2 are staged in LDS with padded rows.
namespace w160 {
constexpr int FS = 68;  // stage row stride (floats) of a 64-feature slice
struct __attribute__((aligned(16))) FwdLds {
  __attribute__((aligned(16))) bf16 W1[L * LW];
  __attribute__((aligned(16))) bf16 W2[L * LW];
  __attribute__((aligned(16))) float b1[L];
  __attribute__((aligned(16))) float b2[L];
  __attribute__((aligned(16))) float g[L];
  __attribute__((aligned(16))) float bt[L];
  __attribute__((aligned(16))) float stage[NW][16 * FS];
};
}  // namespace w160

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_fwd_w160(EdgeTiles tl, const bf16* __restrict__ e_in, bf16* __restrict__ e_out, int write_e,
                const bf16* __restrict__ Pn, const bf16* __restrict__ W1p, const bf16* __restrict__ W2p,
                const float* __restrict__ b1, const float* __restrict__ b2, const float* __restrict__ gamma,
                const float* __restrict__ beta, float eps, float* __restrict__ agg, float* __restrict__ slots,
                bf16* __restrict__ a1_out) {
  using namespace w160;
  __shared__ __align__(16) FwdLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_w(S.W1, W1p, tid);
  stage_w(S.W2, W2p, tid);
  if (tid < L) {
    S.b1[tid] = b1[tid];
    S.b2[tid] = b2[tid];
    S.g[tid] = gamma[tid];
    S.bt[tid] = beta[tid];
  }
  __syncthreads();

  const UnitRange ur = unit_range(tl.n_tiles, wv);
  int64_t t = ur.t;
  const int64_t stride = ur.stride, tend = ur.end;
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tend - 1];
    int4 r;  // per-component selects (an aggregate select goes through scratch)
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto nrows = [](int4 d) { return d.w - d.z; };
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, nrows(d) - 1), 0), lastE); };
  // the streams of one half for this lane's row (prefetched one half ahead):
  // the five runs of the edge latent and of the two gathered node products
  struct HalfF {
    uint4 e[NS], ps[NS], pr[NS];
  };
  auto issue_half = [&](int4 d, int rb, HalfF& H) {
    const size_t row = (size_t)erow(d, rb);
    const int snd = tl.senders[row], rcv = tl.receivers[row];
    const bf16* ep = e_in + row * L + 8 * q;
    const bf16* sp = Pn + (size_t)snd * (2 * L) + 8 * q;
    const bf16* rp = Pn + (size_t)rcv * (2 * L) + L + 8 * q;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      H.e[k] = *reinterpret_cast<const uint4*>(ep + 32 * k);
      H.ps[k] = *reinterpret_cast<const uint4*>(sp + 32 * k);
      H.pr[k] = *reinterpret_cast<const uint4*>(rp + 32 * k);
    }
  };
  float* stage = S.stage[wv];
  const int lv[2] = {w160::live_bits(8, q), w160::live_bits(9, q)};

  auto half = [&](const HalfF& H, int4 d0, int rb, int segraw, bool chunk, int nv, int (&js)[3], float (&carry)[3]) {
    const int n = nrows(d0);
    const int row = rb * 16 + i;
    const bool ok = row < n;
    const int oz = opaque_zero();
    const bf16* W1s = S.W1 + oz;
    const bf16* W2s = S.W2 + oz;
    // ---- z1 = (b1 + P_s) + P_r + W1e e
    f32x4 acc[NOB];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = (*reinterpret_cast<const f32x4*>(S.b1 + fo(ob, q)) + run_block5(H.ps, ob)) + run_block5(H.pr, ob);
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(W1s + (ob * 16 + i) * LW + 32 * s + 8 * q);
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_frag(H.e[s]), acc[ob], 0, 0, 0);
      }
    // ---- a1 = relu(z1), the B operand of the second layer
    bf16x8 a1[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        a1[s][r] = (bf16)relu(acc[2 * s][r]);
        a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
      }
    if (a1_out != nullptr && ok) {
      bf16* ap = a1_out + ((size_t)d0.z + row) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s) *reinterpret_cast<uint4*>(ap + 32 * s) = __builtin_bit_cast(uint4, a1[s]);
    }
    // ---- z2 = b2 + W2 a1
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + fo(ob, q));
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(W2s + (ob * 16 + i) * LW + 32 * s + 8 * q);
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, a1[s], acc[ob], 0, 0, 0);
      }
    // ---- LayerNorm over the 150 real features; message m = gamma xhat + beta
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
    for (int ob = 0; ob < NOB; ++ob) {
      const f32x4 ga = *reinterpret_cast<const f32x4*>(S.g + fo(ob, q));
      const f32x4 be = *reinterpret_cast<const f32x4*>(S.bt + fo(ob, q));
      acc[ob] = ga * (acc[ob] * rstd) + be;  // message m (exactly 0 on padded features)
    }
    // ---- e_out = e + m
    if (write_e && ok) {
      bf16* op = e_out + ((size_t)d0.z + row) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const f32x4 lo = run_block5(H.e, 2 * s) + acc[2 * s], hi = run_block5(H.e, 2 * s + 1) + acc[2 * s + 1];
        *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(lo, hi));
      }
    }
    // ---- receiver sums of m, slice by slice (rows past the tile's end are
    // never inside a segment)
    const int lo_row = rb * 16, hi_row = lo_row + 16;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const int width = k < 2 ? 64 : 32;
      wave_lds_sync();
#pragma unroll
      for (int ob = 4 * k; ob < (k < 2 ? 4 * k + 4 : NOB); ++ob)
        *reinterpret_cast<f32x4*>(stage + i * FS + fo(ob, q) - 64 * k) = acc[ob];
      wave_lds_sync();
      int& j = js[k];
      while (j < nv) {
        const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - d0.z;
        const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - d0.z;
        const int u0 = max(a, lo_row), u1 = min(b, hi_row);
        if (lane < width)
          for (int u = u0; u < u1; ++u) carry[k] += stage[(u - lo_row) * FS + lane];
        if (b > hi_row) break;
        float* dst = !chunk ? agg + (size_t)(d0.x + j) * L : slots + (size_t)(-1 - d0.y) * L;
        if (lane < width) dst[64 * k + lane] = carry[k];
        carry[k] = 0.f;
        ++j;
      }
    }
    wave_lds_sync();
  };

  if (t < tend) {
    int4 d0 = desc(t);
    HalfF A, B;
    issue_half(d0, 0, A);
    for (; t < tend; t += stride) {
      const bool chunk = d0.y < 0;
      const int nv = chunk ? 1 : d0.y - d0.x;
      const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
      const int4 d1 = desc(t + stride);
      issue_half(d0, 1, B);
      int js[3] = {0, 0, 0};  // next node whose sum is open, per slice
      float carry[3] = {0.f, 0.f, 0.f};
      half(A, d0, 0, segraw, chunk, nv, js, carry);
      issue_half(d1, 0, A);
      half(B, d0, 1, segraw, chunk, nv, js, carry);
      d0 = d1;
    }
  }
}

// Weight gradients of the edge MLP at width 160 from the saved bf16 streams,
// one pass: dW1e = sum_rows zbar^T e (partials at 0) and dW2 = sum_rows
// dz2^T a1 (at 160 * 160).  Each 32-row chunk of the four streams is staged
// row-major in LDS (rows 176 elements apart: 88 dwords, so the 4-row x
// 4-piece transposing reads below hit distinct banks) while the next chunk
// is in flight in registers; wave w (10 waves) owns output rows [16w, 16w +
// 16) of both matrices and reads its MFMA operands with K = the chunk's rows
// through ds_read_b64_tr_b16.
namespace w160 {
constexpr int WG_NT = 640;
}  // namespace w160

__global__ void __launch_bounds__(w160::WG_NT) k_wgrad2_w160(int64_t M, const bf16* __restrict__ zb,
                                                           const bf16* __restrict__ e, const bf16* __restrict__ dz,
                                                           const bf16* __restrict__ a1, Partials part) {
  using namespace w160;
  __shared__ __align__(16) bf16 Sg[2][4][TM * WG_LD];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int jp = i >> 2, c4 = i & 3;
  f32x4 acc1[NOB], acc2[NOB];
#pragma unroll
  for (int cb = 0; cb < NOB; ++cb) acc1[cb] = acc2[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int64_t nch = (M + TM - 1) / TM, G = gridDim.x;
  const int srow = tid / (L / 8), scol = (tid % (L / 8)) * 8;
  const bf16* src[4] = {zb, e, dz, a1};
  uint4 Ld[4];
  auto issue = [&](int64_t ch) {
    const int64_t r = ch * TM + srow;
    const int64_t rc = r < M ? r : M - 1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint4 v = ld_stream(src[k] + rc * L + scol);
      Ld[k].x = r < M ? v.x : 0u;
      Ld[k].y = r < M ? v.y : 0u;
      Ld[k].z = r < M ? v.z : 0u;
      Ld[k].w = r < M ? v.w : 0u;
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
    for (int k = 0; k < 4; ++k) *reinterpret_cast<uint4*>(&Sg[buf][k][srow * WG_LD + scol]) = Ld[k];
    __syncthreads();
    if (c + G < nch) issue(c + G);
    const bf16x8 az = frag(Sg[buf][0], 16 * w);
    const bf16x8 ad = frag(Sg[buf][2], 16 * w);
#pragma unroll
    for (int cb = 0; cb < NOB; ++cb) {
      acc1[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az, frag(Sg[buf][1], 16 * cb), acc1[cb], 0, 0, 0);
      acc2[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad, frag(Sg[buf][3], 16 * cb), acc2[cb], 0, 0, 0);
    }
    buf ^= 1;
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int cb = 0; cb < NOB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = w * 16 + q * 4 + r;
      base[(size_t)o * L + cb * 16 + i] = acc1[cb][r];
      base[L * L + (size_t)o * L + cb * 16 + i] = acc2[cb][r];
    }
}

}  // namespace dev

using namespace dev;

hipError_t launch_edge_bwd_w160(const EdgeTiles& t, const void* a1, const void* ebar_in, int have_ebar,
                                void* ebar_out, const float* aggbar, const MlpW& w, float eps, void* zbar, void* dz,
                                float* R, float* slots, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (t.n_tiles <= 0) return hipSuccess;
  if (!w.W1p || !w.W2p || part.stride < 4 * 160) return hipErrorInvalidValue;
  const int64_t need = (t.n_tiles + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, std::min(256, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  hipLaunchKernelGGL(k_edge_bwd_w160, dim3(g), dim3(NT), 0, s, t, (const bf16*)a1, (const bf16*)ebar_in, have_ebar,
                     (bf16*)ebar_out, aggbar, (const bf16*)w.W1p, (const bf16*)w.W2p, w.b2,
                     w.gamma, eps, (bf16*)zbar, (bf16*)dz, R, slots, part);
  return hipGetLastError();
}

hipError_t launch_wgrad2_w160(int64_t M, const void* zbar, const void* e, const void* dz, const void* a1,
                              const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (M <= 0) return hipSuccess;
  if (part.stride < 2 * 160 * 160) return hipErrorInvalidValue;
  const int g = grid_for((M + TM - 1) / TM, std::min(512, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_wgrad2_w160, dim3(g), dim3(w160::WG_NT), 0, s, M, (const bf16*)zbar, (const bf16*)e,
                     (const bf16*)dz, (const bf16*)a1, part);
  return hipGetLastError();
}

hipError_t launch_edge_fwd_w160(const EdgeTiles& t, const void* e_in, void* e_out, int write_e, const void* Pn,
                                const MlpW& w, float eps, float* agg, float* slots, void* a1_out, hipStream_t s) {
  if (t.n_tiles <= 0) return hipSuccess;
  if (!w.W1p || !w.W2p) return hipErrorInvalidValue;
  const int64_t need = (t.n_tiles + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, 512);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_edge_fwd_w160, dim3(g), dim3(NT), 0, s, t, (const bf16*)e_in, (bf16*)e_out, write_e,
                     (const bf16*)Pn, (const bf16*)w.W1p, (const bf16*)w.W2p, w.b1, w.b2, w.gamma, w.beta, eps, agg,
                     slots, (bf16*)a1_out);
  return hipGetLastError();
}

}  // namespace mgn
