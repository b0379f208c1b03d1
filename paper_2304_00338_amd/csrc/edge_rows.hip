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
// product per output and one rounding, though not always to nearest (on
// random operands about 4% of these sums come out one ulp below the
// round-to-nearest VALU add, as if the aligned addend were truncated).
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
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tile_desc(tl.tiles, ok ? tt : tend - 1);
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

// ============================================================ fused reverse
// The edge phase's reverse with its weight gradients in the same pass: per
// 16-row half of a tile, from the saved a1, the block's input edge latents
// e and the incoming gradients (ebar_in, aggbar at the receiver), it writes
// zbar = dL/dz1 (for the sender sums), the receiver sums R of zbar and
// ebar_out = ebar_in + W1e^T zbar, and accumulates dW2 = sum dz2^T a1,
// dW1e = sum zbar^T e, db2 = sum dz2, db1 = sum zbar, dgamma, dbeta.
//
// Work split: eight waves per block, two per SIMD, in two roles.  Row
// waves 0..3 run the reverse of one 16-row half per round (the layout and
// products of the forward kernel) and stage its rows of dz2, zbar and a1
// in LDS (row-major; dz2 and zbar are zero past the tile's end); gradient
// waves 4..7 load the matching rows of e into the staging and, while the
// row waves compute the next round, form the receiver sums of the staged
// zbar rows and add the staged 64 rows into the weight gradients: wave
// 4 + k owns the rows [64 (k % 2), + 64) of dW2 (k < 2: A = dz2^T, B = a1)
// or of dW1e (A = zbar^T, B = e), with the row index as the MFMA's K
// dimension (transposing LDS reads) and the column sums db2 / db1 through a
// ones operand.  So each SIMD runs one row wave and one gradient wave, the
// accumulators never share a wave with the row work, and the row waves
// carry only the work that needs their registers.  Two block barriers per
// round order the staging: after the first it is free (the gradient waves
// have read the previous round), after the second it is full.  dgamma and
// dbeta are column sums of each half on MFMA (its rows, rounded to bf16,
// through the wave's own LDS rows), accumulated per lane of the row waves.  Every sum runs in a fixed order, so results are reproducible.
constexpr int FB_RW = 4;             // row waves per block (= gradient waves)
constexpr int FB_NT = 128 * FB_RW;   // threads per block
constexpr int FB_ROWS = 16 * FB_RW;  // rows staged per round
constexpr int FB_LD = D + 16;        // staged row stride (elements)

struct __attribute__((aligned(16))) FusedLds {
  __attribute__((aligned(16))) bf16 W1[D * D];
  __attribute__((aligned(16))) bf16 W2[D * D];
  __attribute__((aligned(16))) float b2[D];
  __attribute__((aligned(16))) float g[D];
  // staged streams of a round: 0 dz2, 1 zbar, 2 a1, 3 e
  __attribute__((aligned(16))) bf16 st[4][FB_ROWS * FB_LD];
  // each row wave's own 16 rows of a column-sum operand (mbar xhat, mbar)
  __attribute__((aligned(16))) bf16 cs[FB_RW][16 * FB_LD];
};

// Column sums of a row wave's 16 staged rows (bf16, row stride FB_LD) on
// MFMA: for each 16-feature block ob, the transposing read gives lane
// (i, q) rows 4q .. 4q + 3 of feature 16 ob + i (the A operand, M = feature,
// K = row) and a 0/1 operand that is 1 only in column ob routes the block's
// sums there, so one accumulator collects all eight blocks: lane (i, q)
// with i < 8 ends with the sums of features 16 i + 4 q + r (r < 4); lanes
// with i >= 8 hold zeros.
__device__ __forceinline__ f32x4 colsum_mfma(const bf16* rows, f32x4 acc, int i, int q) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  const bf16* p = rows + (4 * q + (i >> 2)) * FB_LD + 4 * (i & 3);
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) {
    const bf16x4 a = lds_tr(p + 16 * ob);
    const uint32_t w = i == ob ? 0x3F803F80u : 0u;  // bf16 pair (1, 1) or (0, 0)
    const bf16x4 b = __builtin_bit_cast(bf16x4, uint2{w, w});
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
  }
  return acc;
}

// operand of 16 columns col0.. with K = the 32 staged rows r0 .. r0 + 31
// (lane (i, q) gets rows r0 + 8q .. + 8 of column col0 + i)
__device__ __forceinline__ bf16x8 staged_frag(const bf16* X, int r0, int col0, int i, int q) {
  const bf16* p = X + (r0 + q * 8 + (i >> 2)) * FB_LD + col0 + 4 * (i & 3);
  return cat8(lds_tr(p), lds_tr(p + 4 * FB_LD));
}

// A pair of bf16 values w with each half cleared unless the matching half of
// a (bf16 bits) is a positive number: the ReLU mask a > 0 on the bit
// patterns as signed 16-bit integers (+0 and negative values have no
// positive pattern), in three packed integer operations.
__device__ __forceinline__ uint32_t relu_mask_pair(uint32_t w, uint32_t a) {
  typedef short s16x2 __attribute__((ext_vector_type(2)));
  const s16x2 zero = {0, 0}, one = {1, 1};
  const s16x2 pos = __builtin_elementwise_min(__builtin_elementwise_max(__builtin_bit_cast(s16x2, a), zero), one);
  return w & __builtin_bit_cast(uint32_t, zero - pos);
}

template <bool HAVE_EBAR>
__global__ void __launch_bounds__(FB_NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_bwd_fused(EdgeTiles tl, const bf16* __restrict__ a1_in, const bf16* __restrict__ e_in, const bf16* ebar_in,
                 bf16* ebar_out, const float* __restrict__ aggbar, MlpW w, float eps, bf16* __restrict__ zbar,
                 float* __restrict__ R, float* __restrict__ slots, Partials part) {
  __shared__ __align__(16) FusedLds S;
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

  // The block's tiles: XCD-contiguous ranges (see unit_range); row wave k
  // (and gradient wave 4 + k for the e rows and the receiver sums) takes
  // tile tb + k of every round pair; all waves run the same number of
  // rounds (a row wave past the range runs empty tiles).
  const int G = gridDim.x;
  int64_t tb, stride, tend;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (tl.n_tiles + 7) >> 3;
    const int64_t lo = x * chunk;
    tend = min(tl.n_tiles, lo + chunk);
    tb = lo + (int64_t)(blockIdx.x >> 3) * FB_RW;
    stride = (int64_t)per * FB_RW;
  } else {
    tb = (int64_t)blockIdx.x * FB_RW;
    stride = (int64_t)G * FB_RW;
    tend = tl.n_tiles;
  }
  const bool row_wave = wv < FB_RW;
  const int k = row_wave ? wv : wv - FB_RW;  // the tile slot this wave follows

  const int64_t tlast = max(tend - 1, (int64_t)0);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tile_desc(tl.tiles, ok ? tt : tlast);
    int4 r;
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  // Every global load is unconditional from a clamped index (see the
  // forward kernel); rows past a tile's end (and the rows of an empty tile)
  // read row 0 or the tile's last row, and are never stored or summed.
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  const int srow = 16 * k + i;  // this lane's staged row
  auto stage_runs = [&](bf16* X, const uint4 (&v)[4], bool live) {
    bf16* p = X + srow * FB_LD + 8 * q;
#pragma unroll
    for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(p + 32 * s) = live ? v[s] : uint4{0u, 0u, 0u, 0u};
  };
  float* base = part.buf + (size_t)blockIdx.x * part.stride;

  if (!row_wave) {
    // ================================ gradient waves
    const int mat = k >> 1, oh = k & 1;
    const bf16* Ast = S.st[mat];      // dz2 or zbar
    const bf16* Bst = S.st[2 + mat];  // a1 or e
    f32x4 acc_w[4][8], acc_b[4];
#pragma unroll
    for (int ob = 0; ob < 4; ++ob) {
      acc_b[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) acc_w[ob][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    bf16x8 ones;
#pragma unroll
    for (int j = 0; j < 8; ++j) ones[j] = (bf16)1.f;
    auto products = [&]() {
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        bf16x8 af[4];
#pragma unroll
        for (int ob = 0; ob < 4; ++ob) {
          af[ob] = staged_frag(Ast, 32 * kc, 64 * oh + 16 * ob, i, q);
          acc_b[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[ob], ones, acc_b[ob], 0, 0, 0);
        }
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
          const bf16x8 bfr = staged_frag(Bst, 32 * kc, 16 * nb, i, q);
#pragma unroll
          for (int ob = 0; ob < 4; ++ob)
            acc_w[ob][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[ob], bfr, acc_w[ob][nb], 0, 0, 0);
        }
      }
    };
    // Per-receiver sums of zbar (as stored) over the staged rows of row
    // wave k's half rb of tile d, each in ascending row order from 0.0 and
    // carried into the next half while its segment is open: nodes d.x + j
    // of a tile of whole segments (rp(j) in lane j of segraw), or the single
    // segment of a chunk tile, summed into its slot.
    auto recv_sums = [&](int4 d, int rb, int segraw, bool chunk, int nv, int& j, float2& carry) {
      const bf16* zs = S.st[1] + 16 * k * FB_LD;
      uint32_t zr[16];  // the 16 rows' values of this lane's two features, read at once
#pragma unroll
      for (int r = 0; r < 16; ++r) zr[r] = *reinterpret_cast<const uint32_t*>(zs + r * FB_LD + 2 * lane);
      const int n = tile_rows(d);
      const int lo_row = rb * 16, hi_row = lo_row + 16;
      while (j < nv) {
        const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - d.z;
        const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - d.z;
        const int u0 = max(a, lo_row), u1 = min(b, hi_row);
        for (int u = u0; u < u1; ++u) {
          const uint32_t v = zr[u - lo_row];
          carry.x += __uint_as_float(v << 16);
          carry.y += __uint_as_float(v & 0xffff0000u);
        }
        if (b > hi_row) break;
        float* dst = !chunk ? R + (size_t)(d.x + j) * D : slots + (size_t)(-1 - d.y) * D;
        *reinterpret_cast<float2*>(dst + 2 * lane) = carry;
        carry = float2{0.f, 0.f};
        ++j;
      }
    };
    auto load_e = [&](int4 d, int rb, uint4 (&v)[4]) {
      const bf16* xp = e_in + (size_t)erow(d, rb) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) v[s] = *reinterpret_cast<const uint4*>(xp + 32 * s);
    };
    if (tb < tend) {
      int4 d0 = desc(tb + k), d1 = desc(tb + k + stride);
      uint4 ev[4];
      load_e(d0, 0, ev);
      for (; tb < tend; tb += stride) {
        const bool chunk = d0.y < 0;
        const int nv = chunk ? 1 : d0.y - d0.x;
        // in-segment starts of the tile's nodes (lane j: rowptr of node j)
        const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
        float2 carry = {0.f, 0.f};
        int j = 0;  // next node whose sum is open
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          __syncthreads();  // staging free
          stage_runs(S.st[3], ev, rb * 16 + i < tile_rows(d0));
          __syncthreads();  // staging full
          recv_sums(d0, rb, segraw, chunk, nv, j, carry);
          products();
          // the next round's e rows, in flight while the row waves finish it
          if (rb == 0)
            load_e(d0, 1, ev);
          else
            load_e(d1, 0, ev);
        }
        d0 = d1;
        d1 = desc(tb + k + 2 * stride);
      }
    }
    // weight gradients straight from the owning wave; db1 / db2 from the
    // ones column
    const int wofs = mat == 0 ? 16512 : 0, bofs = mat == 0 ? 32896 : 16384;
#pragma unroll
    for (int ob = 0; ob < 4; ++ob) {
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int o = 64 * oh + 16 * ob + 4 * q + r;
          base[wofs + (size_t)o * D + 16 * nb + i] = acc_w[ob][nb][r];
        }
      if (i == 0)
#pragma unroll
        for (int r = 0; r < 4; ++r) base[bofs + 64 * oh + 16 * ob + 4 * q + r] = acc_b[ob][r];
    }
    __syncthreads();
    __syncthreads();
    return;
  }

  // ==================================== row waves
  struct HalfLoads {
    uint4 a[4], eb[4];
  };
  auto load_recv = [&](int4 d, int (&rv)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) rv[rb] = tl.receivers[erow(d, rb)];
  };
  auto load_half = [&](int4 d, int rb, HalfLoads& H) {
    const size_t row = (size_t)erow(d, rb);
    const bf16* ap = a1_in + row * D + 8 * q;
#pragma unroll
    for (int s = 0; s < 4; ++s) H.a[s] = *reinterpret_cast<const uint4*>(ap + 32 * s);
    if (HAVE_EBAR) {
      const bf16* ep = ebar_in + row * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) H.eb[s] = *reinterpret_cast<const uint4*>(ep + 32 * s);
    }
  };
  auto load_ag = [&](int recv, f32x4 (&ag)[8]) {
    const float* gp = aggbar + (size_t)recv * D;
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) ag[ob] = *reinterpret_cast<const f32x4*>(gp + fo(ob, q));
  };
  const bf16x8 sel0 = select_frag(0, i, q), sel1 = select_frag(1, i, q);
  f32x4 dga = {0.f, 0.f, 0.f, 0.f}, dbe = {0.f, 0.f, 0.f, 0.f};
  bf16* csw = S.cs[k];  // this wave's column-sum rows

  // One round: the reverse of half rb of tile d0 (streams in H), its rows staged.
  auto round = [&](HalfLoads& H, f32x4 (&ag)[8], int next_recv, int4 d0, int rb) {
    const int n = tile_rows(d0);
    const int row = rb * 16 + i;
    const bool live = row < n;
    // ---- z2 = b2 + W2 a1 and its LayerNorm statistics
    f32x4 acc[8];
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + fo(ob, q));
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(wchunk(S.W2, ob * 16 + i, 4 * s + q));
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_frag(H.a[s]), acc[ob], 0, 0, 0);
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
    // mbar = aggbar[receiver] + ebar_in (the bf16 ebar entered by a
    // selection MFMA: one product per output, within an ulp of the VALU
    // add), zero on rows past the tile's end
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) {
      acc[ob] *= rstd;  // xhat
      if (HAVE_EBAR)
        ag[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16((ob & 1) ? sel1 : sel0, as_frag(H.eb[ob >> 1]), ag[ob], 0,
                                                         0, 0);
    }
    if (n < rb * 16 + 16) {  // a partial half (uniform)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) ag[ob] = live ? ag[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // ---- dgamma += sum_rows mbar * xhat, dbeta += sum_rows mbar: the
    // half's rows (bf16) through this wave's own LDS rows into MFMA column
    // sums (the second write follows the first operand's reads in the
    // wave's LDS order)
    {
      bf16* cp = csw + i * FB_LD + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        *reinterpret_cast<bf16x8*>(cp + 32 * s) = pack_run(ag[2 * s] * acc[2 * s], ag[2 * s + 1] * acc[2 * s + 1]);
      dga = colsum_mfma(csw, dga, i, q);
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<bf16x8*>(cp + 32 * s) = pack_run(ag[2 * s], ag[2 * s + 1]);
      dbe = colsum_mfma(csw, dbe, i, q);
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
    // dz2 = rstd dxh - rstd m1 - xhat (rstd m2), two fused multiply-adds per value
    const float m1 = sum_rowlanes(s1) * (1.0f / D), m2 = sum_rowlanes(s2) * (1.0f / D);
    const float c0 = -rstd * m1, c1 = -rstd * m2;
    bf16x8 dzf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dzf[s][r] = (bf16)__builtin_fmaf(acc[2 * s][r], c1, __builtin_fmaf(rstd, ag[2 * s][r], c0));
        dzf[s][4 + r] = (bf16)__builtin_fmaf(acc[2 * s + 1][r], c1, __builtin_fmaf(rstd, ag[2 * s + 1][r], c0));
      }
    // the next half's receiver gradients, in flight for the rest of the round
    load_ag(next_recv, ag);
    // ---- da1 = W2^T dz2, zbar = da1 where a1 > 0
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wt_frag(S.W2, ob, s, i, q), dzf[s],
                                                          s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[ob], 0, 0, 0);
    uint4 zw[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint4 z = __builtin_bit_cast(uint4, pack_run(acc[2 * s], acc[2 * s + 1]));
      zw[s].x = relu_mask_pair(z.x, H.a[s].x);
      zw[s].y = relu_mask_pair(z.y, H.a[s].y);
      zw[s].z = relu_mask_pair(z.z, H.a[s].z);
      zw[s].w = relu_mask_pair(z.w, H.a[s].w);
    }
    if (live) {
      bf16* zp = zbar + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(zp + 32 * s) = zw[s];
    }
    // ---- ebar_out = ebar_in + W1e^T zbar (ebar_in entered exactly by a
    // selection MFMA, then the products in the same order)
#pragma unroll
    for (int ob = 0; ob < 8; ++ob)
      acc[ob] = HAVE_EBAR ? __builtin_amdgcn_mfma_f32_16x16x32_bf16((ob & 1) ? sel1 : sel0, as_frag(H.eb[ob >> 1]),
                                                                    f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(wt_frag(S.W1, ob, s, i, q), as_frag(zw[s]), acc[ob], 0, 0, 0);
    if (live) {
      bf16* op = ebar_out + ((size_t)d0.z + row) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(acc[2 * s], acc[2 * s + 1]));
    }
    // ---- stage the round's rows of dz2, zbar, a1.  Past the tile's end
    // mbar is zero, so dz2 and zbar are zero there too (a row's LayerNorm
    // statistics are its own) and those rows add nothing to the weight
    // gradients; their a1 is a copy of a valid row, finite.
    __syncthreads();  // staging free
    {
      uint4 v[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) v[s] = __builtin_bit_cast(uint4, dzf[s]);
      stage_runs(S.st[0], v, true);
      stage_runs(S.st[1], zw, true);
      stage_runs(S.st[2], H.a, true);
    }
    __syncthreads();  // staging full
  };

  if (tb < tend) {
    int4 d0 = desc(tb + k), d1 = desc(tb + k + stride);
    int rc0[2], rn[2];
    load_recv(d0, rc0);
    load_recv(d1, rn);
    HalfLoads A, B;
    load_half(d0, 0, A);
    f32x4 ag[8];
    load_ag(rc0[0], ag);
    for (; tb < tend; tb += stride) {
      // issue order = use order, so each wait covers only older requests
      const int4 d2 = desc(tb + k + 2 * stride);
      load_half(d0, 1, B);
      round(A, ag, rc0[1], d0, 0);
      load_half(d1, 0, A);
      round(B, ag, rn[0], d0, 1);
      rc0[0] = rn[0];
      rc0[1] = rn[1];
      load_recv(d2, rn);
      d0 = d1;
      d1 = d2;
    }
  }
  // ---- dgamma, dbeta: the row waves' sums in wave order
  __syncthreads();  // the gradient waves have read the last round
  float* red = reinterpret_cast<float*>(&S.st[0][0]);  // [2][FB_RW][D]
  if (i < 8) {
    const int f = 16 * i + 4 * q;
    *reinterpret_cast<f32x4*>(red + k * D + f) = dga;
    *reinterpret_cast<f32x4*>(red + (FB_RW + k) * D + f) = dbe;
  }
  __syncthreads();
  if (tid < 2 * D) {
    const int c2 = tid >> 7, c = tid & (D - 1);
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < FB_RW; ++u) v += red[(c2 * FB_RW + u) * D + c];
    base[33024 + c2 * D + c] = v;
  }
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



static constexpr int kFusedBlocks = 256;

hipError_t launch_edge_bwd_fused(const EdgeTiles& t, const void* a1, const void* e, const void* ebar_in,
                                 int have_ebar, void* ebar_out, const float* aggbar, const MlpW& w, float eps,
                                 void* zbar, float* R, float* slots, const Partials& part, int* nblocks,
                                 hipStream_t s) {
  *nblocks = 0;
  if (t.n_tiles <= 0) return hipSuccess;
  if (t.n_edges <= 0 || part.stride < 33280) return hipErrorInvalidValue;
  const int64_t need = (t.n_tiles + FB_RW - 1) / FB_RW;
  int g = (int)std::min<int64_t>(need, std::min(kFusedBlocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  if (have_ebar)
    hipLaunchKernelGGL(k_edge_bwd_fused<true>, dim3(g), dim3(FB_NT), 0, s, t, (const bf16*)a1, (const bf16*)e,
                       (const bf16*)ebar_in, (bf16*)ebar_out, aggbar, w, eps, (bf16*)zbar, R, slots, part);
  else
    hipLaunchKernelGGL(k_edge_bwd_fused<false>, dim3(g), dim3(FB_NT), 0, s, t, (const bf16*)a1, (const bf16*)e,
                       (const bf16*)ebar_in, (bf16*)ebar_out, aggbar, w, eps, (bf16*)zbar, R, slots, part);
  return hipGetLastError();
}


}  // namespace mgn
