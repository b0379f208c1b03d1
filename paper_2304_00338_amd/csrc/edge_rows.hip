// Edge phase of one MGN message-passing step, forward, bf16 operands, with
// one wave per receiver-aligned tile (Sec. 2.1: every edge latent is updated
// by the edge MLP from itself and its two end nodes, then each node sums the
// new messages of its in-edges).
//
// Work split.  Each of the 8 waves of a block runs its own persistent loop
// over tiles; the only block barrier is the one after the weights are
// staged in LDS.  A tile is two 16-row blocks in the lane layout of
// rows_common.hpp.
//
// Adds of bf16 inputs into fp32 accumulators (the node products P_s + P_r
// and the residual e + m) are MFMAs with a 0/1 selection operand: one
// product per output, so each is a single fp32 rounding, as a VALU add.
//
// Node sums: the wave stages each 16-row half of the messages in its own
// LDS area and sums every in-segment in ascending row order from 0.0, so a
// node's aggregate does not depend on where its segment sits in a tile.
#include "rows_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

constexpr int RW_LDM = D + 4;  // LDS row stride of a wave's message half-tile (fp32)

struct __attribute__((aligned(16))) RowsLds {
  __attribute__((aligned(16))) bf16 W1[D * D];
  __attribute__((aligned(16))) bf16 W2[D * D];
  __attribute__((aligned(16))) float b1[D];
  __attribute__((aligned(16))) float b2[D];
  __attribute__((aligned(16))) float g[D];
  __attribute__((aligned(16))) float bt[D];
  __attribute__((aligned(16))) float stage[NW][16 * RW_LDM];
};

__device__ __forceinline__ int tile_rows(int4 d) { return d.w - d.z; }

// In-segment node sums over one staged 16-row half [lo_row, lo_row + 16) of
// a tile (rows past the tile's end are never inside a segment).  For a tile
// of whole segments node j's rows are [rp(j) - base, rp(j+1) - base) with
// rp(j) held by lane j of segraw; a chunk tile (chunk) is the single segment
// [0, n).  j is the first node whose sum is still open and carry its partial
// sum (features 2*lane, 2*lane+1), added in ascending row order; close(j,
// sum) is called for every node whose segment ends inside this half.
template <class F>
__device__ __forceinline__ void seg_pass(const float* stage, int lane, int segraw, int base, bool chunk, int n,
                                         int nv, int lo_row, int& j, float2& carry, F&& close) {
  const int hi_row = lo_row + 16;
  while (j < nv) {
    const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - base;
    const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - base;
    const int u0 = max(a, lo_row), u1 = min(b, hi_row);
    for (int u = u0; u < u1; ++u) {
      const float2 v = *reinterpret_cast<const float2*>(stage + (u - lo_row) * RW_LDM + 2 * lane);
      carry.x += v.x;
      carry.y += v.y;
    }
    if (b > hi_row) break;
    close(j, carry);
    carry = float2{0.f, 0.f};
    ++j;
  }
}

// Sum over the first nr staged rows of features 2*lane, 2*lane+1.
__device__ __forceinline__ float2 col_pass(const float* stage, int lane, int nr) {
  float2 c = {0.f, 0.f};
  for (int u = 0; u < nr; ++u) {
    const float2 v = *reinterpret_cast<const float2*>(stage + u * RW_LDM + 2 * lane);
    c.x += v.x;
    c.y += v.y;
  }
  return c;
}

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_fwd_rows(EdgeTiles tl, const bf16* __restrict__ e_in, bf16* __restrict__ e_out, int write_e,
                const bf16* __restrict__ Pn, MlpW w, float eps, float* __restrict__ agg,
                float* __restrict__ slots, bf16* __restrict__ a1_out) {
  __shared__ __align__(16) RowsLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  {
    stage_weights<D>(S.W1, (const bf16*)w.W1p, tid);
    stage_weights<D>(S.W2, (const bf16*)w.W2p, tid);
    if (tid < D) {
      S.b1[tid] = w.b1[tid];
      S.b2[tid] = w.b2[tid];
      S.g[tid] = w.gamma[tid];
      S.bt[tid] = w.beta[tid];
    }
  }
  __syncthreads();

  // XCD-contiguous tile ranges: the node products gathered by one XCD's
  // waves then mostly share that XCD's L2.
  const UnitRange ur = unit_range(tl.n_tiles, wv);
  int64_t t = ur.t;
  const int64_t stride = ur.stride, tend = ur.end;
  if (t >= tend) return;

  const bf16x8 sel0 = select_frag(0, i, q), sel1 = select_frag(1, i, q);
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tend - 1];
    int4 r;
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  // Every global load below is unconditional, from an index clamped into
  // its array (so the compiler's in-order wait counts stay exact and a wait
  // never covers a later prefetch): rows past a tile's end, and the tiles
  // of edge-less nodes, read a valid row whose values are never stored or
  // summed (rows never mix inside the products or the LayerNorm).
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  auto load_sr = [&](int4 d, int (&s)[2], int (&r)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      s[rb] = tl.senders[erow(d, rb)];
      r[rb] = tl.receivers[erow(d, rb)];
    }
  };
  // The streams of one 16-row half of a tile for this lane's row: its four
  // 8-feature runs of the edge latent and of the two gathered node products.
  // The next half's streams are in flight while a half is computed.
  struct HalfF {
    uint4 e[4], ps[4], pr[4];
  };
  auto issue_half = [&](int4 d, int rb, int snd, int rcv, HalfF& H) {
    const bf16* ep = e_in + (size_t)erow(d, rb) * D + 8 * q;
    const bf16* sp = Pn + (size_t)snd * (2 * D) + 8 * q;
    const bf16* rp = Pn + (size_t)rcv * (2 * D) + D + 8 * q;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      H.e[k] = *reinterpret_cast<const uint4*>(ep + 32 * k);
      H.ps[k] = *reinterpret_cast<const uint4*>(sp + 32 * k);
      H.pr[k] = *reinterpret_cast<const uint4*>(rp + 32 * k);
    }
  };
  float* stage = S.stage[wv];

  // One half (rows rb*16 .. +16) of tile d0 with its streams in H.
  auto half = [&](HalfF& H, int4 d0, int rb, int segraw, bool chunk, int nv, int& j, float2& carry) {
    const int n = tile_rows(d0);
    // ---- z1 = b1 + P_s + P_r + W1e e
    f32x4 acc[8];
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      acc[ob] = *reinterpret_cast<const f32x4*>(S.b1 + fo(ob, q));
      const bf16x8 sel = (ob & 1) ? sel1 : sel0;
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, as_frag(H.ps[ob >> 1]), acc[ob], 0, 0, 0);
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, as_frag(H.pr[ob >> 1]), acc[ob], 0, 0, 0);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(wchunk(S.W1, ob * 16 + i, 4 * s + q));
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_frag(H.e[s]), acc[ob], 0, 0, 0);
      }
    // ---- a1 = relu(z1) as the B operand of the second layer
    bf16x8 a1[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        a1[s][r] = (bf16)relu(acc[2 * s][r]);
        a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
      }
    const int row = rb * 16 + i;
    if (a1_out != nullptr && row < n) {
      bf16* ap = a1_out + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(ap + 32 * s) = __builtin_bit_cast(uint4, a1[s]);
    }
    // ---- z2 = b2 + W2 a1
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + fo(ob, q));
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(wchunk(S.W2, ob * 16 + i, 4 * s + q));
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, a1[s], acc[ob], 0, 0, 0);
      }
    // ---- LayerNorm over the row's 128 features (4 lanes x 32)
    float sm = 0.f;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm += acc[ob][r];
    const float mean = sum_rowlanes(sm) * (1.0f / D);
    float sq = 0.f;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      acc[ob] -= mean;
#pragma unroll
      for (int r = 0; r < 4; ++r) sq += acc[ob][r] * acc[ob][r];
    }
    const float rstd = __builtin_amdgcn_rsqf(sum_rowlanes(sq) * (1.0f / D) + eps);
    float* srow = stage + i * RW_LDM;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      const f32x4 ga = *reinterpret_cast<const f32x4*>(S.g + fo(ob, q));
      const f32x4 be = *reinterpret_cast<const f32x4*>(S.bt + fo(ob, q));
      acc[ob] = ga * (acc[ob] * rstd) + be;  // message m
      *reinterpret_cast<f32x4*>(srow + fo(ob, q)) = acc[ob];
    }
    // ---- e_out = e + m
    if (write_e) {
      uint4 o[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        f32x4 lo = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel0, as_frag(H.e[s]), acc[2 * s], 0, 0, 0);
        f32x4 hi = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel1, as_frag(H.e[s]), acc[2 * s + 1], 0, 0, 0);
        bf16x8 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = (bf16)lo[r];
          v[4 + r] = (bf16)hi[r];
        }
        o[s] = __builtin_bit_cast(uint4, v);
      }
      if (row < n) {
        bf16* op = e_out + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
        for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(op + 32 * s) = o[s];
      }
    }
    wave_lds_sync();
    seg_pass(stage, lane, segraw, d0.z, chunk, n, nv, rb * 16, j, carry, [&](int jj, float2 v) {
      float* dst = !chunk ? agg + (size_t)(d0.x + jj) * D : slots + (size_t)(-1 - d0.y) * D;
      *reinterpret_cast<float2*>(dst + 2 * lane) = v;
    });
    wave_lds_sync();
  };

  // issue order = use order, so each wait covers only older requests
  int4 d0 = desc(t), d1 = desc(t + stride);
  int sc[2], rc[2], sn[2], rn[2];
  load_sr(d0, sc, rc);
  HalfF A, B;
  issue_half(d0, 0, sc[0], rc[0], A);
  for (; t < tend; t += stride) {
    const bool chunk = d0.y < 0;
    const int nv = chunk ? 1 : d0.y - d0.x;
    // in-segment starts of the tile's nodes (lane j: rowptr of node j)
    const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
    const int4 d2 = desc(t + 2 * stride);
    load_sr(d1, sn, rn);
    issue_half(d0, 1, sc[1], rc[1], B);
    float2 carry = {0.f, 0.f};
    int j = 0;  // next node whose sum is open
    half(A, d0, 0, segraw, chunk, nv, j, carry);
    issue_half(d1, 0, sn[0], rn[0], A);
    half(B, d0, 1, segraw, chunk, nv, j, carry);
    d0 = d1;
    d1 = d2;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      sc[rb] = sn[rb];
      rc[rb] = rn[rb];
    }
  }
}

// ===================================================================== reverse
// Given ebar_in = dL/de_out (absent for the last block), aggbar, and the
// saved first-layer activations a1 of the edge MLP: mbar = ebar_in +
// aggbar[receiver]; back through the LayerNorm and the MLP to zbar = dL/dz1
// (written out, with dz2 = dL/dz2 for the weight-gradient kernel), the
// per-receiver sums R of zbar, ebar_out = ebar_in + W1e^T zbar, and
// per-block partials of db1, dgamma, dbeta.  The edge-gradient stream is
// bf16 like the edge latents it belongs to: ebar_out is formed in fp32 and
// rounded once.
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_bwd_rows(EdgeTiles tl, const bf16* __restrict__ a1_in, const bf16* ebar_in, int have_ebar,
                bf16* ebar_out, const float* __restrict__ aggbar, MlpW w, float eps,
                bf16* __restrict__ zbar, bf16* __restrict__ dz_out, float* __restrict__ R,
                float* __restrict__ slots, Partials part) {
  __shared__ __align__(16) RowsLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  {
    stage_weights<D>(S.W1, (const bf16*)w.W1p, tid);
    stage_weights<D>(S.W2, (const bf16*)w.W2p, tid);
    if (tid < D) {
      S.b2[tid] = w.b2[tid];
      S.g[tid] = w.gamma[tid];
    }
  }
  __syncthreads();

  const UnitRange ur = unit_range(tl.n_tiles, wv);
  int64_t t = ur.t;
  const int64_t stride = ur.stride, tend = ur.end;

  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tend - 1];
    int4 r;
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  // The streamed inputs of one 16-row half of a tile for this lane's row:
  // the four runs of a1 and of the incoming edge gradient.  The next half's streams are in flight while a half is computed;
  // the receiver's aggregate gradient (shared by the ~14 consecutive rows of
  // a receiver, so mostly a cache hit) is loaded when the half starts.
  struct HalfLoads {
    uint4 a[4], eb[4];
  };
  // All global loads are unconditional from clamped indices (see the
  // forward kernel); without an incoming edge gradient the loaded values are
  // replaced by zeros.
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  auto load_recv = [&](int4 d, int (&rv)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) rv[rb] = tl.receivers[erow(d, rb)];
  };
  auto load_half = [&](int4 d, int rb, HalfLoads& H) {
    const size_t row = (size_t)erow(d, rb);
    const bf16* ap = a1_in + row * D + 8 * q;
#pragma unroll
    for (int k = 0; k < 4; ++k) H.a[k] = *reinterpret_cast<const uint4*>(ap + 32 * k);
    const bf16* ep = ebar_in + row * D + 8 * q;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint4 v = *reinterpret_cast<const uint4*>(ep + 32 * k);
      H.eb[k].x = have_ebar ? v.x : 0u;
      H.eb[k].y = have_ebar ? v.y : 0u;
      H.eb[k].z = have_ebar ? v.z : 0u;
      H.eb[k].w = have_ebar ? v.w : 0u;
    }
  };
  auto load_ag = [&](int recv, f32x4 (&ag)[8]) {
    const float* gp = aggbar + (size_t)recv * D;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) ag[ob] = *reinterpret_cast<const f32x4*>(gp + fo(ob, q));
  };

  float2 db1 = {0.f, 0.f}, dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  float* stage = S.stage[wv];
  float* srow = stage + i * RW_LDM;

  // One half (rows rb*16 .. +16) of tile d0 with its streams in H.
  auto half = [&](HalfLoads& H, f32x4 (&ag)[8], int4 d0, int rb, int segraw, bool chunk, int nv, int& j,
                  float2& carry) {
    const int n = tile_rows(d0);
    const int row = rb * 16 + i;
    const int nh = max(0, min(16, n - rb * 16));  // valid rows of this half
    // ---- z2 = b2 + W2 a1 and its LayerNorm statistics
    f32x4 acc[8];
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + fo(ob, q));
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(wchunk(S.W2, ob * 16 + i, 4 * s + q));
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_frag(H.a[s]), acc[ob], 0, 0, 0);
      }
    }
    float sm = 0.f;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm += acc[ob][r];
    const float mean = sum_rowlanes(sm) * (1.0f / D);
    float sq = 0.f;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      acc[ob] -= mean;
#pragma unroll
      for (int r = 0; r < 4; ++r) sq += acc[ob][r] * acc[ob][r];
    }
    const float rstd = __builtin_amdgcn_rsqf(sum_rowlanes(sq) * (1.0f / D) + eps);
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      acc[ob] *= rstd;          // xhat
      ag[ob] += run_block(H.eb, ob);  // mbar = ebar_in + aggbar[receiver]
    }
    // ---- dgamma += sum_rows mbar * xhat, dbeta += sum_rows mbar
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) *reinterpret_cast<f32x4*>(srow + fo(ob, q)) = ag[ob] * acc[ob];
    wave_lds_sync();
    {
      const float2 c = col_pass(stage, lane, nh);
      dga.x += c.x;
      dga.y += c.y;
    }
    wave_lds_sync();
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) *reinterpret_cast<f32x4*>(srow + fo(ob, q)) = ag[ob];
    wave_lds_sync();
    {
      const float2 c = col_pass(stage, lane, nh);
      dbe.x += c.x;
      dbe.y += c.y;
    }
    // ---- LayerNorm backward: dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = mbar gamma
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      ag[ob] *= *reinterpret_cast<const f32x4*>(S.g + fo(ob, q));  // dxh
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s1 += ag[ob][r];
        s2 += ag[ob][r] * acc[ob][r];
      }
    }
    const float m1 = sum_rowlanes(s1) * (1.0f / D), m2 = sum_rowlanes(s2) * (1.0f / D);
    bf16x8 dzf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dzf[s][r] = (bf16)(rstd * (ag[2 * s][r] - m1 - acc[2 * s][r] * m2));
        dzf[s][4 + r] = (bf16)(rstd * (ag[2 * s + 1][r] - m1 - acc[2 * s + 1][r] * m2));
      }
    if (row < n) {
      bf16* dp = dz_out + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(dp + 32 * s) = __builtin_bit_cast(uint4, dzf[s]);
    }
    // ---- da1 = W2^T dz2, zbar = da1 where a1 > 0
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wt_frag(S.W2, ob, s, i, q), dzf[s], acc[ob], 0, 0, 0);
    }
    bf16x8 zf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bf16x8 a = as_frag(H.a[s]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        zf[s][r] = (float)a[r] > 0.f ? (bf16)acc[2 * s][r] : (bf16)0.f;
        zf[s][4 + r] = (float)a[4 + r] > 0.f ? (bf16)acc[2 * s + 1][r] : (bf16)0.f;
      }
    }
    if (row < n) {
      bf16* zp = zbar + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(zp + 32 * s) = __builtin_bit_cast(uint4, zf[s]);
    }
    // ---- per-receiver sums of zbar (as stored) and db1
    wave_lds_sync();
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      f32x4 lo, hi;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        lo[r] = (float)zf[s][r];
        hi[r] = (float)zf[s][4 + r];
      }
      *reinterpret_cast<f32x4*>(srow + 32 * s + 8 * q) = lo;
      *reinterpret_cast<f32x4*>(srow + 32 * s + 8 * q + 4) = hi;
    }
    wave_lds_sync();
    seg_pass(stage, lane, segraw, d0.z, chunk, n, nv, rb * 16, j, carry, [&](int jj, float2 v) {
      float* dst = !chunk ? R + (size_t)(d0.x + jj) * D : slots + (size_t)(-1 - d0.y) * D;
      *reinterpret_cast<float2*>(dst + 2 * lane) = v;
      db1.x += v.x;
      db1.y += v.y;
    });
    // ---- ebar_out = ebar_in + W1e^T zbar
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = run_block(H.eb, ob);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wt_frag(S.W1, ob, s, i, q), zf[s], acc[ob], 0, 0, 0);
    }
    if (row < n) {
      bf16* op = ebar_out + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(acc[2 * s], acc[2 * s + 1]));
    }
    wave_lds_sync();
  };

  if (t < tend) {
    int4 d0 = desc(t), d1 = desc(t + stride);
    int rc0[2], rn[2];
    load_recv(d0, rc0);
    HalfLoads A, B;
    load_half(d0, 0, A);
    for (; t < tend; t += stride) {
      // issue order = use order, so each wait covers only older requests
      const bool chunk = d0.y < 0;
      const int nv = chunk ? 1 : d0.y - d0.x;
      const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
      const int4 d2 = desc(t + 2 * stride);
      load_recv(d1, rn);
      f32x4 ag[8];
      load_ag(rc0[0], ag);
      load_half(d0, 1, B);
      float2 carry = {0.f, 0.f};
      int j = 0;
      half(A, ag, d0, 0, segraw, chunk, nv, j, carry);
      load_ag(rc0[1], ag);
      load_half(d1, 0, A);
      half(B, ag, d0, 1, segraw, chunk, nv, j, carry);
      d0 = d1;
      d1 = d2;
      rc0[0] = rn[0];
      rc0[1] = rn[1];
    }
  }
  // ---- block partials: the 8 waves' column sums in wave order
  __syncthreads();
  float* red = &S.stage[0][0];  // [3][NW][D]
  *reinterpret_cast<float2*>(red + (0 * NW + wv) * D + 2 * lane) = db1;
  *reinterpret_cast<float2*>(red + (1 * NW + wv) * D + 2 * lane) = dga;
  *reinterpret_cast<float2*>(red + (2 * NW + wv) * D + 2 * lane) = dbe;
  __syncthreads();
  if (tid < 3 * D) {
    const int k = tid >> 7, f = tid & (D - 1);
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * D + f];
    float* base = part.buf + (size_t)blockIdx.x * part.stride;
    const int off = k == 0 ? 16384 : (k == 1 ? 33024 : 33152);
    base[off + f] = v;
  }
}

// Weight gradients of the edge MLP from the saved streams, one pass:
// dW1e = sum_rows zbar^T e, dW2 = sum_rows dz2^T a1, db2 = sum_rows dz2.
// Each 32-row chunk of the four bf16 streams is staged row-major in LDS
// (rows 144 elements apart, so the transposing reads below are free of bank
// conflicts) while the next chunk is in flight in registers; wave w owns
// output rows [16w, 16w + 16) of both matrices and reads its MFMA operands
// with K = the chunk's rows through ds_read_b64_tr_b16.
constexpr int WG_LD = D + 16;

__global__ void __launch_bounds__(NT) k_wgrad2(int64_t M, const bf16* __restrict__ zb, const bf16* __restrict__ e,
                                               const bf16* __restrict__ dz, const bf16* __restrict__ a1,
                                               Partials part) {
  __shared__ __align__(16) bf16 Sg[2][4][TM * WG_LD];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int jp = i >> 2, c4 = i & 3;
  f32x4 acc1[8], acc2[8], accb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc1[cb] = acc2[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 ones;
#pragma unroll
  for (int j = 0; j < 8; ++j) ones[j] = (bf16)1.f;
  const int64_t nch = (M + TM - 1) / TM, G = gridDim.x;
  const int srow = tid >> 4, scol = (tid & 15) * 8;
  const bf16* src[4] = {zb, e, dz, a1};
  uint4 L[4];
  auto issue = [&](int64_t ch) {
    const int64_t r = ch * TM + srow;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (r < M)
        L[k] = ld_stream(src[k] + r * D + scol);
      else
        L[k] = uint4{0u, 0u, 0u, 0u};
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
    for (int k = 0; k < 4; ++k) *reinterpret_cast<uint4*>(&Sg[buf][k][srow * WG_LD + scol]) = L[k];
    __syncthreads();
    if (c + G < nch) issue(c + G);
    const bf16x8 az = frag(Sg[buf][0], 16 * w8);
    const bf16x8 ad = frag(Sg[buf][2], 16 * w8);
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      acc1[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az, frag(Sg[buf][1], 16 * cb), acc1[cb], 0, 0, 0);
      acc2[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad, frag(Sg[buf][3], 16 * cb), acc2[cb], 0, 0, 0);
    }
    accb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad, ones, accb, 0, 0, 0);
    buf ^= 1;
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = w8 * 16 + q * 4 + r;
      base[(size_t)o * D + cb * 16 + i] = acc1[cb][r];
      base[16512 + (size_t)o * D + cb * 16 + i] = acc2[cb][r];
    }
  if (i == 0)
#pragma unroll
    for (int r = 0; r < 4; ++r) base[32896 + w8 * 16 + q * 4 + r] = accb[r];
}

}  // namespace dev

using namespace dev;

static constexpr int kRowsBlocks = 256;

static int rows_grid(int64_t n_tiles, int max_blocks) {
  const int64_t need = (n_tiles + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, max_blocks);
  if (g >= 8) g &= ~7;
  return g;
}

hipError_t launch_edge_fwd_rows(const EdgeTiles& t, const void* e_in, void* e_out, int write_e, const void* Pn,
                                const MlpW& w, float eps, float* agg, float* slots, void* a1_out, hipStream_t s) {
  if (t.n_tiles <= 0) return hipSuccess;
  if (t.n_edges <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_edge_fwd_rows, dim3(rows_grid(t.n_tiles, kRowsBlocks)), dim3(NT), 0, s, t, (const bf16*)e_in,
                     (bf16*)e_out, write_e, (const bf16*)Pn, w, eps, agg, slots, (bf16*)a1_out);
  return hipGetLastError();
}

hipError_t launch_edge_bwd_rows(const EdgeTiles& t, const void* a1, const void* ebar_in, int have_ebar,
                                void* ebar_out, const float* aggbar, const MlpW& w, float eps, void* zbar, void* dz,
                                float* R, float* slots, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (t.n_tiles <= 0) return hipSuccess;
  if (t.n_edges <= 0) return hipErrorInvalidValue;
  const int g = rows_grid(t.n_tiles, std::min(kRowsBlocks, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_edge_bwd_rows, dim3(g), dim3(NT), 0, s, t, (const bf16*)a1, (const bf16*)ebar_in, have_ebar, (bf16*)ebar_out,
                     aggbar, w, eps, (bf16*)zbar, (bf16*)dz, R, slots, part);
  return hipGetLastError();
}

static constexpr int kWgrad2Blocks = 512;

hipError_t launch_wgrad2(int64_t M, const void* zbar, const void* e, const void* dz, const void* a1,
                         const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (M <= 0) return hipSuccess;
  const int g = (int)std::min<int64_t>((M + TM - 1) / TM, std::min(kWgrad2Blocks, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_wgrad2, dim3(g), dim3(NT), 0, s, M, (const bf16*)zbar, (const bf16*)e, (const bf16*)dz,
                     (const bf16*)a1, part);
  return hipGetLastError();
}

}  // namespace mgn
