// Edge phase of one MGN message-passing step in fp32 (Sec. 2.1: every edge
// latent is updated by the edge MLP from itself and its two end nodes, then
// each node sums the new messages of its in-edges), with one wave per
// receiver-aligned tile, at kernel width LD = 128 or 160 (latent 150 padded
// with zero columns).
//
// The lane layout and the product routine (gemm32) are those of
// rows32_common.hpp.
#include "rows32_common.hpp"
#include "w160_common.hpp"

namespace mgn {
namespace dev {


template <int LD>
struct __attribute__((aligned(16))) Fwd32Lds {
  // At width 128 both products' fragment-major weights fit in LDS (64 KB
  // each) beside an unpadded message staging (exactly 160 KiB); at 160 only
  // W2 (100 KB) does, and the staging rows are padded.
  static constexpr bool W1L = LD == 128;
  static constexpr int SS = W1L ? LD : R32<LD>::SLD;  // staging row stride
  __attribute__((aligned(16))) float stage[R32_NW][16 * SS];
  __attribute__((aligned(16))) float w2[LD * LD];
  __attribute__((aligned(16))) float w1[W1L ? LD * LD : 4];
};

// In-segment node sums over one staged 16-row half [lo_row, lo_row + 16) of
// a tile (as in the bf16 forward): node j's rows are [rp(j) - base,
// rp(j + 1) - base), rp(j) held by lane j of segraw; a chunk tile is the
// single segment [0, n).  Each lane sums the LD / 2 feature pairs p = lane,
// lane + 64 (p < LD / 2) of every row in ascending row order from 0.0;
// close(j, pair index, sum) stores a finished node sum.
template <int LD, class F>
__device__ __forceinline__ void seg_pass32(const float* stage, int lane, int segraw, int base, bool chunk, int n,
                                           int nv, int lo_row, int& j, float2 (&carry)[2], F&& close,
                                           int SLD = R32<LD>::SLD) {
  constexpr int NP = LD / 2;
  const int hi_row = lo_row + 16;
  while (j < nv) {
    const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - base;
    const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - base;
    const int u0 = max(a, lo_row), u1 = min(b, hi_row);
    for (int u = u0; u < u1; ++u) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int p = lane + 64 * h;
        if (h == 0 || p < NP) {
          const float2 v = *reinterpret_cast<const float2*>(stage + (u - lo_row) * SLD + 2 * p);
          carry[h].x += v.x;
          carry[h].y += v.y;
        }
      }
    }
    if (b > hi_row) break;
    close(j, carry);
    carry[0] = carry[1] = float2{0.f, 0.f};
    ++j;
  }
}

// Forward: e' = e + m (when write_e), agg = receiver sums of m, with
// m = LN(W2 relu(b1 + P_s + P_r + W1e e) + b2) (the node products P = [W1s
// h, W1r h] of the block come from the node kernels).  The next half's rows
// are in flight while a half is computed; all global loads are
// unconditional from clamped indices (rows past a tile's end read a valid
// row that is never stored or summed).
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_edge_fwd_r32(EdgeTiles tl, const float* __restrict__ e_in, float* __restrict__ e_out, int write_e,
               const float* __restrict__ Pn, MlpW w, float eps, float* __restrict__ agg, float* __restrict__ slots) {
  typedef R32<LD> Z;
  __shared__ __align__(16) Fwd32Lds<LD> S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  typedef Fwd32Lds<LD> L;
  for (int idx = tid; idx < LD * LD / 4; idx += R32_NT) {
    reinterpret_cast<f32x4*>(S.w2)[idx] = reinterpret_cast<const f32x4*>(w.F2)[idx];
    if (L::W1L) reinterpret_cast<f32x4*>(S.w1)[idx] = reinterpret_cast<const f32x4*>(w.F1)[idx];
  }
  __syncthreads();
  const UnitRange ur = unit_range<R32_NW>(tl.n_tiles, wv);
  int64_t t = ur.t;
  const int64_t stride = ur.stride, tend = ur.end;
  if (t >= tend) return;
  const int f0 = Z::KL * g;  // first feature of the lane

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
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  struct Half {
    float e[Z::KL];
    f32x4 p[Z::NOB];  // b1 + P_s + P_r in the C layout
  };
  auto load_half = [&](int4 d, int rb, Half& H) {
    const int row = erow(d, rb);
    const int snd = tl.senders[row], rcv = tl.receivers[row];
    load_row32<LD>(H.e, e_in + (size_t)row * LD + f0);
    const float* ps = Pn + (size_t)snd * (2 * LD) + f0;
    const float* pr = Pn + (size_t)rcv * (2 * LD) + LD + f0;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(w.b1 + f0 + 4 * ob);
      const f32x4 a = *reinterpret_cast<const f32x4*>(ps + 4 * ob);
      const f32x4 b = *reinterpret_cast<const f32x4*>(pr + 4 * ob);
      H.p[ob] = (b1 + a) + b;
    }
  };
  float* stage = S.stage[wv];

  auto half = [&](Half& H, int4 d0, int rb, int segraw, bool chunk, int nv, int& j, float2 (&carry)[2]) {
    const int n = tile_rows(d0);
    const int row = rb * 16 + i;
    // ---- z1 = b1 + P_s + P_r + W1e e, a1 = relu(z1)
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = H.p[ob];
    // the weight addresses are opaque per half: otherwise the loop-invariant
    // fragment loads are hoisted out of the tile loop into registers
    const int oz = opaque_zero();
    gemm32<LD>(acc, H.e, (L::W1L ? S.w1 : w.F1) + oz, lane);
    float a1[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) a1[4 * ob + r] = relu(acc[ob][r]);
    // ---- z2 = b2 + W2 a1
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(w.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, S.w2 + oz, lane);
    // ---- LayerNorm over the row's DR real features (padded ones are 0)
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
    const float rstd = __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / Z::DR) + eps);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      const f32x4 ga = *reinterpret_cast<const f32x4*>(w.gamma + f0 + 4 * ob);
      const f32x4 be = *reinterpret_cast<const f32x4*>(w.beta + f0 + 4 * ob);
      acc[ob] = ga * (acc[ob] * rstd) + be;  // message m
    }
    store_row32<LD>(stage + i * L::SS + f0, acc);
    // ---- e_out = e + m
    if (write_e && row < n) {
      f32x4 o[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[ob][r] = H.e[4 * ob + r] + acc[ob][r];
      store_row32<LD>(e_out + ((size_t)d0.z + row) * LD + f0, o);
    }
    wave_lds_sync();
    seg_pass32<LD>(stage, lane, segraw, d0.z, chunk, n, nv, rb * 16, j, carry, [&](int jj, float2 (&v)[2]) {
      float* dst = !chunk ? agg + (size_t)(d0.x + jj) * LD : slots + (size_t)(-1 - d0.y) * LD;
      *reinterpret_cast<float2*>(dst + 2 * lane) = v[0];
      if (LD / 2 > 64 && lane + 64 < LD / 2) *reinterpret_cast<float2*>(dst + 2 * (lane + 64)) = v[1];
    }, L::SS);
    wave_lds_sync();
  };

  int4 d0 = desc(t), d1 = desc(t + stride);
  Half A, B;
  load_half(d0, 0, A);
  for (; t < tend; t += stride) {
    const bool chunk = d0.y < 0;
    const int nv = chunk ? 1 : d0.y - d0.x;
    const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
    const int4 d2 = desc(t + 2 * stride);
    load_half(d0, 1, B);
    float2 carry[2] = {{0.f, 0.f}, {0.f, 0.f}};
    int j = 0;
    half(A, d0, 0, segraw, chunk, nv, j, carry);
    load_half(d1, 0, A);
    half(B, d0, 1, segraw, chunk, nv, j, carry);
    d0 = d1;
    d1 = d2;
  }
}


// ================================================================= reverse
// fp32 edge reverse with its weight gradients in one pass (width 128): per
// 16-row half of a tile, from the block's input edge latents e, the node
// products P (the first layer is recomputed: z1 = b1 + P_s + P_r + W1e e)
// and the incoming gradients (ebar_in, aggbar at the receiver), it writes
// zbar = dL/dz1 (for the sender sums), the receiver sums R of zbar and
// ebar_out = ebar_in + W1e^T zbar, and accumulates dW2 = sum dz2^T a1,
// dW1e = sum zbar^T e, db2, db1 (ones columns), dgamma, dbeta (DPP column
// sums).  Four waves per block, one per SIMD (512 registers: the weight
// gradient accumulators, a quarter of dW2 and dW1e per wave, live in
// AGPRs), in lockstep rounds: each wave computes one half and stages its
// rows of dz2, a1, e and zbar in LDS, then after a block barrier adds the
// round's 64 rows into its 32 output rows of dW2 and dW1e with the row
// index as the K dimension.  In fp32 the MFMA work (four 128 x 128 products
// per row plus the weight gradients) dominates each round, so one wave per
// SIMD keeps the MFMA pipe busy with its own independent chains.
constexpr int B32_LD = 128;
constexpr int B32_SLD = B32_LD + 16;  // staged row stride: lane groups 0, 1 hit distinct banks
constexpr int B32_ROWS = 16 * R32_NW;

struct __attribute__((aligned(16))) Bwd32Lds {
  // staged streams of a round: 0 dz2, 1 a1, 2 e, 3 zbar
  __attribute__((aligned(16))) float st[4][B32_ROWS * B32_SLD];
  // b1, b2, gamma: read per half from LDS, not L2 (the L2 reads, issued
  // where they are used, left their latency exposed)
  __attribute__((aligned(16))) float vec[3][B32_LD];
};

// in-segment sums of the staged zbar rows (as in seg_pass32, stride B32_SLD)
template <class F>
__device__ __forceinline__ void seg_pass_b32(const float* stage, int lane, int segraw, int base, bool chunk, int n,
                                             int nv, int lo_row, int& j, float2& carry, F&& close) {
  const int hi_row = lo_row + 16;
  while (j < nv) {
    const int a = chunk ? 0 : __builtin_amdgcn_readlane(segraw, j) - base;
    const int b = chunk ? n : __builtin_amdgcn_readlane(segraw, j + 1) - base;
    const int u0 = max(a, lo_row), u1 = min(b, hi_row);
    for (int u = u0; u < u1; ++u) {
      const float2 v = *reinterpret_cast<const float2*>(stage + (u - lo_row) * B32_SLD + 2 * lane);
      carry.x += v.x;
      carry.y += v.y;
    }
    if (b > hi_row) break;
    close(j, carry);
    carry = float2{0.f, 0.f};
    ++j;
  }
}

__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_edge_bwd_r32(EdgeTiles tl, const float* __restrict__ e_in, const float* ebar_in, int have_ebar, float* ebar_out,
               const float* __restrict__ Pn, const float* __restrict__ aggbar, MlpW w, float eps,
               float* __restrict__ zbar, float* __restrict__ R, float* __restrict__ slots, Partials part) {
  constexpr int LD = B32_LD;
  typedef R32<LD> Z;
  __shared__ __align__(16) Bwd32Lds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int f0 = Z::KL * g;
  for (int idx = tid; idx < LD; idx += R32_NT) {
    S.vec[0][idx] = w.b1[idx];
    S.vec[1][idx] = w.b2[idx];
    S.vec[2][idx] = w.gamma[idx];
  }
  __syncthreads();

  // The block's tiles: XCD-contiguous ranges, wave wv takes tile tb + wv of
  // every round pair; all four waves run the same number of rounds.
  const int G = gridDim.x;
  int64_t tb, stride, tend;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (tl.n_tiles + 7) >> 3;
    const int64_t lo = x * chunk;
    tend = min(tl.n_tiles, lo + chunk);
    tb = lo + (int64_t)(blockIdx.x >> 3) * R32_NW;
    stride = (int64_t)per * R32_NW;
  } else {
    tb = (int64_t)blockIdx.x * R32_NW;
    stride = (int64_t)G * R32_NW;
    tend = tl.n_tiles;
  }
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  const int64_t tlast = max(tend - 1, (int64_t)0);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tlast];
    int4 r;
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  struct Half {
    float e[Z::KL];
  };
  auto load_half = [&](int4 d, int rb, Half& H) {
    load_row32<LD>(H.e, e_in + (size_t)erow(d, rb) * LD + f0);
  };

  // this wave's share of the weight gradients: output rows [32 wv, 32 wv + 32)
  f32x4 aw2[2][8], aw1[2][8], ab2[2], ab1[2];
#pragma unroll
  for (int ob = 0; ob < 2; ++ob) {
    ab2[ob] = ab1[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) aw2[ob][nb] = aw1[ob][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // dgamma, dbeta: per half, the column sums over its 16 rows by the DPP
  // butterfly (lane i ends with 2 of lane group g's 32 column sums),
  // accumulated per lane
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  const int srow = 16 * wv + i;
  auto stage_row = [&](float* X, const float (&v)[Z::KL], bool live) {
    float* p = X + srow * B32_SLD + f0;
#pragma unroll
    for (int c = 0; c < Z::KC; ++c)
      *reinterpret_cast<f32x4*>(p + 4 * c) =
          live ? f32x4{v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]} : f32x4{0.f, 0.f, 0.f, 0.f};
  };

  // H holds the half's e rows (the first product's operand, then staged);
  // after the last product the next half's rows (tile dn, half rbn) are
  // requested into the same registers.
  auto round = [&](Half& H, int4 d0, int rb, int4 dn, int rbn, int segraw, bool chunk, int nv, int& j,
                   float2& carry) {
    const int n = tile_rows(d0);
    const int row = rb * 16 + i;
    const bool live = row < n;
    const size_t grow = (size_t)erow(d0, rb);
    const int snd = tl.senders[grow], rcv = tl.receivers[grow];
    const int oz = opaque_zero();
    // the incoming edge gradient of the half (needed after the forward
    // recompute: in flight during its two products)
    float eb[Z::KL];
    load_row32<LD>(eb, ebar_in + grow * LD + f0);
    if (!have_ebar)
#pragma unroll
      for (int s = 0; s < Z::KL; ++s) eb[s] = 0.f;
    // ---- z1 = W1e e + (b1 + P_s + P_r), a1 = relu(z1); e is staged right
    // after its product (the staging is free: every wave has finished the
    // previous round's products)
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    __syncthreads();
    // the gathered node products are requested halfway through the product
    f32x4 pa[Z::NOB], pb[Z::NOB];
    gemm32<LD>(acc, H.e, w.F1 + oz, lane, [&] {
      const float* ps = Pn + (size_t)snd * (2 * LD) + f0;
      const float* pr = Pn + (size_t)rcv * (2 * LD) + LD + f0;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        pa[ob] = *reinterpret_cast<const f32x4*>(ps + 4 * ob);
        pb[ob] = *reinterpret_cast<const f32x4*>(pr + 4 * ob);
      }
    });
    stage_row(S.st[2], H.e, live);
    float a1[Z::KL];
    uint32_t mask = 0;
    {
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(S.vec[0] + f0 + 4 * ob);
        const f32x4 z = acc[ob] + ((b1 + pa[ob]) + pb[ob]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          a1[4 * ob + r] = relu(z[r]);
          if (z[r] > 0.f) mask |= 1u << (4 * ob + r);
        }
      }
    }
    // ---- z2 = b2 + W2 a1 and its LayerNorm statistics
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.vec[1] + f0 + 4 * ob);
    // the receiver's aggregate gradient, requested halfway through the product
    f32x4 ag[Z::NOB];
    gemm32<LD>(acc, a1, w.F2 + oz, lane, [&] {
      const float* gp = aggbar + (size_t)rcv * LD + f0;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) ag[ob] = *reinterpret_cast<const f32x4*>(gp + 4 * ob);
    });
    float sm = 0.f;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm += acc[ob][r];
    const float mean = sum_q(sm) * (1.0f / LD);
    float sq = 0.f;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      acc[ob] -= mean;
#pragma unroll
      for (int r = 0; r < 4; ++r) sq += acc[ob][r] * acc[ob][r];
    }
    const float rstd = __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / LD) + eps);
    // ---- mbar = ebar_in + aggbar[receiver]; dgamma, dbeta; LayerNorm reverse
    float dz[Z::KL];
    {
      float s1 = 0.f, s2 = 0.f;
      f32x4 pg[Z::NOB], pb[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        const f32x4 ga = *reinterpret_cast<const f32x4*>(S.vec[2] + f0 + 4 * ob);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 4 * ob + r;
          const float xh = acc[ob][r] * rstd;
          acc[ob][r] = xh;
          const float mb = eb[s] + ag[ob][r];
          pg[ob][r] = live ? mb * xh : 0.f;
          pb[ob][r] = live ? mb : 0.f;
          const float dxh = mb * ga[r];
          dz[s] = dxh;
          s1 += dxh;
          s2 += dxh * xh;
        }
      }
      const float2 cg = colsum16(pg, i), cb = colsum16(pb, i);
      dga.x += cg.x;
      dga.y += cg.y;
      dbe.x += cb.x;
      dbe.y += cb.y;
      const float m1 = sum_q(s1) * (1.0f / LD), m2 = sum_q(s2) * (1.0f / LD);
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) dz[4 * ob + r] = rstd * (dz[4 * ob + r] - m1 - acc[ob][r] * m2);
    }
    // ---- stage dz2, a1
    stage_row(S.st[0], dz, live);
    stage_row(S.st[1], a1, live);
    // ---- da1 = W2^T dz2, zbar = da1 where z1 > 0
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    gemm32<LD>(acc, dz, w.F2t + oz, lane);
    float zb[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) zb[4 * ob + r] = (mask >> (4 * ob + r)) & 1u ? acc[ob][r] : 0.f;
    stage_row(S.st[3], zb, live);
    if (live) {
      float* zp = zbar + ((size_t)d0.z + row) * LD + f0;
#pragma unroll
      for (int c = 0; c < Z::KC; ++c)
        *reinterpret_cast<f32x4*>(zp + 4 * c) = f32x4{zb[4 * c], zb[4 * c + 1], zb[4 * c + 2], zb[4 * c + 3]};
    }
    // ---- ebar_out = ebar_in + W1e^T zbar
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
      acc[ob] = f32x4{eb[4 * ob], eb[4 * ob + 1], eb[4 * ob + 2], eb[4 * ob + 3]};
    gemm32<LD>(acc, zb, w.F1t + oz, lane);
    if (live) store_row32<LD>(ebar_out + ((size_t)d0.z + row) * LD + f0, acc);
    load_half(dn, rbn, H);
    __syncthreads();  // the round's rows are staged
    // ---- receiver sums of zbar over this wave's staged rows
    seg_pass_b32(S.st[3] + 16 * wv * B32_SLD, lane, segraw, d0.z, chunk, n, nv, rb * 16, j, carry,
                 [&](int jj, float2 v) {
                   float* dst = !chunk ? R + (size_t)(d0.x + jj) * LD : slots + (size_t)(-1 - d0.y) * LD;
                   *reinterpret_cast<float2*>(dst + 2 * lane) = v;
                 });
    // ---- the round's 64 rows into this wave's output rows of dW2 and dW1e:
    // A = dz2^T / zbar^T (rows 32 wv + 16 ob + m), B = a1 / e, K = 4 rows
    // (the next 4 rows' operands are read before this step's products)
    struct Ops {
      float a2[2], a1[2], b2[8], b1[8];
    };
    auto rd = [&](int kk, Ops& o) {
      const int r0 = (4 * kk + g) * B32_SLD;
#pragma unroll
      for (int ob = 0; ob < 2; ++ob) {
        o.a2[ob] = S.st[0][r0 + 32 * wv + 16 * ob + i];
        o.a1[ob] = S.st[3][r0 + 32 * wv + 16 * ob + i];
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        o.b2[nb] = S.st[1][r0 + 16 * nb + i];
        o.b1[nb] = S.st[2][r0 + 16 * nb + i];
      }
    };
    auto step = [&](const Ops& o) {
#pragma unroll
      for (int ob = 0; ob < 2; ++ob) {
        ab2[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a2[ob], 1.0f, ab2[ob], 0, 0, 0);
        ab1[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a1[ob], 1.0f, ab1[ob], 0, 0, 0);
      }
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int ob = 0; ob < 2; ++ob) {
          aw2[ob][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a2[ob], o.b2[nb], aw2[ob][nb], 0, 0, 0);
          aw1[ob][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a1[ob], o.b1[nb], aw1[ob][nb], 0, 0, 0);
        }
    };
    Ops o0, o1;
    rd(0, o0);
    for (int kk = 0; kk < B32_ROWS / 4; kk += 2) {
      rd(kk + 1, o1);
      __builtin_amdgcn_sched_barrier(0);
      step(o0);
      if (kk + 2 < B32_ROWS / 4) rd(kk + 2, o0);
      __builtin_amdgcn_sched_barrier(0);
      step(o1);
    }
  };

  if (tb < tend) {
    int4 d0 = desc(tb + wv), d1 = desc(tb + wv + stride);
    Half A;
    load_half(d0, 0, A);
    for (; tb < tend; tb += stride) {
      const bool chunk = d0.y < 0;
      const int nv = chunk ? 1 : d0.y - d0.x;
      const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
      const int4 d2 = desc(tb + wv + 2 * stride);
      float2 carry = {0.f, 0.f};
      int j = 0;
      round(A, d0, 0, d0, 1, segraw, chunk, nv, j, carry);
      round(A, d0, 1, d1, 0, segraw, chunk, nv, j, carry);
      d0 = d1;
      d1 = d2;
    }
  }
  // ---- block partials: weight gradients and db from the owning wave;
  // dgamma, dbeta summed over the 16 rows of each lane group, then over the
  // waves in wave order
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int ob = 0; ob < 2; ++ob) {
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = 32 * wv + 16 * ob + 4 * g + r;
        base[16512 + (size_t)o * LD + 16 * nb + i] = aw2[ob][nb][r];
        base[(size_t)o * LD + 16 * nb + i] = aw1[ob][nb][r];
      }
    if (i == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        base[32896 + 32 * wv + 16 * ob + 4 * g + r] = ab2[ob][r];
        base[16384 + 32 * wv + 16 * ob + 4 * g + r] = ab1[ob][r];
      }
  }
  __syncthreads();
  float* red = &S.st[0][0];  // [2][R32_NW][LD]
  {
    // lane i of group g holds the sums of values 2i, 2i + 1 = features
    // f0 + 4 (i / 2) + 2 (i % 2) + {0, 1}
    const int f = f0 + 4 * (i >> 1) + 2 * (i & 1);
    *reinterpret_cast<float2*>(red + (0 * R32_NW + wv) * LD + f) = dga;
    *reinterpret_cast<float2*>(red + (1 * R32_NW + wv) * LD + f) = dbe;
  }
  __syncthreads();
  {
    const int k2 = tid >> 7, c = tid & (LD - 1);  // 256 threads: dgamma (k2 = 0), dbeta (1)
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) v += red[(k2 * R32_NW + u) * LD + c];
    base[33024 + k2 * LD + c] = v;
  }
}


// ======================================================= reverse, width 160
// The reverse at width 160 (latent 150 padded with zero columns): as the
// width-128 pass, but only dW2 (with db2, db1, dgamma, dbeta) accumulates
// in the kernel; dW1e = sum zbar^T e is left to the weight-gradient pass
// over the zbar and e streams (at this width both quarters of the two
// 160 x 160 products would need 224 accumulator registers per wave, and
// four staged fp32 streams 180 KB of LDS).  Buffers: X (dz2) and Y (a1) of
// the round's 64 rows, Zs (each wave's own zbar rows, for its receiver
// sums).  Each wave owns a 5 x 5 block of the 100 16 x 16 tiles of dW2
// (output blocks 5 (wv / 2) .., input blocks 5 (wv % 2) ..) and the ones
// columns of three or two of its five output blocks.  The LayerNorm runs
// over the 150 real features (padded features of dz2 are zeroed); db1 is a
// DPP column sum of zbar per half.
constexpr int C32_LD = 160;
constexpr int C32_SLD = C32_LD + 16;  // staged row stride: lane groups 0, 1 hit distinct banks
constexpr int C32_HB = 5;             // a wave's dW2 tiles: a 5 x 5 block of the 10 x 10
constexpr int C32_TILES = C32_HB * C32_HB;

struct __attribute__((aligned(16))) Bwd32wLds {
  __attribute__((aligned(16))) float st[3][B32_ROWS * C32_SLD];  // X, Y, Zs
  __attribute__((aligned(16))) float vec[3][C32_LD];              // b1, b2, gamma (as at width 128)
};

// column sums over a half's 16 rows of 40 C-layout values (blocks 0..7 by
// colsum16, blocks 8, 9 by the tail butterfly), accumulated
__device__ __forceinline__ void colsum40(const f32x4 (&v)[10], int i, float2& acc8, float& tail) {
  f32x4 p8[8];
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) p8[ob] = v[ob];
  const float2 c = colsum16(p8, i);
  acc8.x += c.x;
  acc8.y += c.y;
  tail += w160::colsum16_tail(v, i);
}

__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_edge_bwd_r32w(EdgeTiles tl, const float* __restrict__ e_in, const float* ebar_in, int have_ebar, float* ebar_out,
                const float* __restrict__ Pn, const float* __restrict__ aggbar, MlpW w, float eps,
                float* __restrict__ zbar, float* __restrict__ R, float* __restrict__ slots, Partials part) {
  constexpr int LD = C32_LD;
  typedef R32<LD> Z;
  __shared__ __align__(16) Bwd32wLds S;
  float* X = S.st[0];
  float* Y = S.st[1];
  float* Zs = S.st[2];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int f0 = Z::KL * g;
  for (int idx = tid; idx < LD; idx += R32_NT) {
    S.vec[0][idx] = w.b1[idx];
    S.vec[1][idx] = w.b2[idx];
    S.vec[2][idx] = w.gamma[idx];
  }
  __syncthreads();
  // this wave's block of dW2 tiles and the output blocks of its db2 ones
  // columns (the two waves of a block row split its five output blocks)
  const int ob0 = C32_HB * (wv >> 1), nb0 = C32_HB * (wv & 1);
  const int uones = (wv & 1) ? 3 : 0, nones = (wv & 1) ? 2 : 3;

  const int G = gridDim.x;
  int64_t tb, stride, tend;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (tl.n_tiles + 7) >> 3;
    const int64_t lo = x * chunk;
    tend = min(tl.n_tiles, lo + chunk);
    tb = lo + (int64_t)(blockIdx.x >> 3) * R32_NW;
    stride = (int64_t)per * R32_NW;
  } else {
    tb = (int64_t)blockIdx.x * R32_NW;
    stride = (int64_t)G * R32_NW;
    tend = tl.n_tiles;
  }
  const int4* tiles = reinterpret_cast<const int4*>(tl.tiles);
  const int64_t tlast = max(tend - 1, (int64_t)0);
  auto desc = [&](int64_t tt) -> int4 {
    const bool ok = tt < tend;
    const int4 v = tiles[ok ? tt : tlast];
    int4 r;
    r.x = ok ? v.x : 0;
    r.y = ok ? v.y : 0;
    r.z = ok ? v.z : 0;
    r.w = ok ? v.w : 0;
    return r;
  };
  const int lastE = (int)max(tl.n_edges - 1, (int64_t)0);
  auto erow = [&](int4 d, int rb) { return min(max(d.z + min(rb * 16 + i, tile_rows(d) - 1), 0), lastE); };
  struct Half {
    float e[Z::KL];
  };
  auto load_half = [&](int4 d, int rb, Half& H) { load_row32<LD>(H.e, e_in + (size_t)erow(d, rb) * LD + f0); };

  f32x4 aw2[C32_TILES], ab2[3];
#pragma unroll
  for (int t = 0; t < C32_TILES; ++t) aw2[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < 3; ++t) ab2[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  // column sums: dgamma, dbeta, db1 (blocks 0..7 pairwise, blocks 8, 9 tail)
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f}, db1 = {0.f, 0.f};
  float tga = 0.f, tbe = 0.f, tb1 = 0.f;
  const int srow = 16 * wv + i;
  auto stage_row = [&](float* B, const float (&v)[Z::KL], bool live) {
    float* p = B + srow * C32_SLD + f0;
#pragma unroll
    for (int c = 0; c < Z::KC; ++c)
      *reinterpret_cast<f32x4*>(p + 4 * c) =
          live ? f32x4{v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]} : f32x4{0.f, 0.f, 0.f, 0.f};
  };

  // H holds the half's e rows, used by the first product only; after the
  // last product the next half's rows (tile dn, half rbn) are requested into
  // the same registers and arrive behind the receiver sums and dW2 products.
  auto round = [&](Half& H, int4 d0, int rb, int4 dn, int rbn, int segraw, bool chunk, int nv, int& j,
                   float2 (&carry)[2]) {
    const int n = tile_rows(d0);
    const int row = rb * 16 + i;
    const bool live = row < n;
    const size_t grow = (size_t)erow(d0, rb);
    const int snd = tl.senders[grow], rcv = tl.receivers[grow];
    const int oz = opaque_zero();
    // ---- z1 = W1e e + (b1 + P_s + P_r), a1 = relu(z1)
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the gathered node products are requested halfway through the product
    f32x4 pa[Z::NOB], pb[Z::NOB];
    gemm32<LD>(acc, H.e, w.F1 + oz, lane, [&] {
      const float* ps = Pn + (size_t)snd * (2 * LD) + f0;
      const float* pr = Pn + (size_t)rcv * (2 * LD) + LD + f0;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        pa[ob] = *reinterpret_cast<const f32x4*>(ps + 4 * ob);
        pb[ob] = *reinterpret_cast<const f32x4*>(pr + 4 * ob);
      }
    });
    float a1[Z::KL];
    uint64_t mask = 0;
    {
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) {
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(S.vec[0] + f0 + 4 * ob);
        const f32x4 z = acc[ob] + ((b1 + pa[ob]) + pb[ob]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          a1[4 * ob + r] = relu(z[r]);
          if (z[r] > 0.f) mask |= 1ull << (4 * ob + r);
        }
      }
    }
    __syncthreads();  // the previous round's products are done
    stage_row(Y, a1, live);
    // ---- z2 = b2 + W2 a1; LayerNorm statistics over the 150 real features
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.vec[1] + f0 + 4 * ob);
    float eb[Z::KL];
    f32x4 ag[Z::NOB];
    gemm32<LD>(acc, a1, w.F2 + oz, lane, [&] {
      const float* gp = aggbar + (size_t)rcv * LD + f0;
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) ag[ob] = *reinterpret_cast<const f32x4*>(gp + 4 * ob);
    });
    load_row32<LD>(eb, ebar_in + grow * LD + f0);
    if (!have_ebar)
#pragma unroll
      for (int s = 0; s < Z::KL; ++s) eb[s] = 0.f;
    f32x4 t[Z::NOB];  // mbar, then dxh, then dz2
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) t[ob][r] = eb[4 * ob + r] + ag[ob][r];
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
        acc[ob][r] -= mean;
        if (f0 + 4 * ob + r < Z::DR) sq += acc[ob][r] * acc[ob][r];
      }
    const float rstd = __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / Z::DR) + eps);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] *= rstd;  // xhat
    // ---- dbeta, dgamma (live rows); LayerNorm reverse (padded features:
    // dxh = 0 from gamma = 0, dz2 zeroed)
    {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = live ? t[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      colsum40(p, i, dbe, tbe);
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = live ? t[ob] * acc[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      colsum40(p, i, dga, tga);
    }
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      t[ob] *= *reinterpret_cast<const f32x4*>(S.vec[2] + f0 + 4 * ob);  // dxh
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
        dz[4 * ob + r] = f0 + 4 * ob + r < Z::DR ? rstd * (t[ob][r] - m1 - acc[ob][r] * m2) : 0.f;
    stage_row(X, dz, live);
    // ---- da1 = W2^T dz2, zbar = da1 where z1 > 0 (db1: its column sums)
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    gemm32<LD>(acc, dz, w.F2t + oz, lane);
    float zb[Z::KL];
    {
      f32x4 pz[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float z = (mask >> (4 * ob + r)) & 1ull ? acc[ob][r] : 0.f;
          zb[4 * ob + r] = z;
          pz[ob][r] = live ? z : 0.f;
        }
      colsum40(pz, i, db1, tb1);
    }
    stage_row(Zs, zb, live);
    if (live) {
      float* zp = zbar + ((size_t)d0.z + row) * LD + f0;
#pragma unroll
      for (int c = 0; c < Z::KC; ++c)
        *reinterpret_cast<f32x4*>(zp + 4 * c) = f32x4{zb[4 * c], zb[4 * c + 1], zb[4 * c + 2], zb[4 * c + 3]};
    }
    // ---- ebar_out = ebar_in + W1e^T zbar
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
      acc[ob] = f32x4{eb[4 * ob], eb[4 * ob + 1], eb[4 * ob + 2], eb[4 * ob + 3]};
    gemm32<LD>(acc, zb, w.F1t + oz, lane);
    if (live) store_row32<LD>(ebar_out + ((size_t)d0.z + row) * LD + f0, acc);
    load_half(dn, rbn, H);
    __syncthreads();  // X = dz2, Y = a1, Zs = zbar staged
    // ---- receiver sums of this wave's zbar rows
    seg_pass32<LD>(Zs + 16 * wv * C32_SLD, lane, segraw, d0.z, chunk, n, nv, rb * 16, j, carry,
                   [&](int jj, float2 (&v)[2]) {
                     float* dst = !chunk ? R + (size_t)(d0.x + jj) * LD : slots + (size_t)(-1 - d0.y) * LD;
                     *reinterpret_cast<float2*>(dst + 2 * lane) = v[0];
                     if (lane + 64 < LD / 2) *reinterpret_cast<float2*>(dst + 2 * (lane + 64)) = v[1];
                   },
                   C32_SLD);
    // ---- the round's 64 rows into this wave's block of dW2 = dz2^T a1
    // (per 4 rows: 10 LDS reads, 25 products and the db2 ones columns)
    {
      const float* pa = X + g * C32_SLD + 16 * ob0 + i;
      const float* pb = Y + g * C32_SLD + 16 * nb0 + i;
#pragma unroll 2
      for (int kk = 0; kk < B32_ROWS / 4; ++kk) {
        float A[C32_HB], B[C32_HB];
#pragma unroll
        for (int u = 0; u < C32_HB; ++u) {
          A[u] = pa[4 * kk * C32_SLD + 16 * u];
          B[u] = pb[4 * kk * C32_SLD + 16 * u];
        }
#pragma unroll
        for (int t3 = 0; t3 < 3; ++t3)
          if (t3 < nones) ab2[t3] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[uones + t3], 1.0f, ab2[t3], 0, 0, 0);
#pragma unroll
        for (int u = 0; u < C32_HB; ++u)
#pragma unroll
          for (int v = 0; v < C32_HB; ++v)
            aw2[u * C32_HB + v] =
                __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], B[v], aw2[u * C32_HB + v], 0, 0, 0);
      }
    }
  };

  if (tb < tend) {
    int4 d0 = desc(tb + wv), d1 = desc(tb + wv + stride);
    Half A;
    load_half(d0, 0, A);
    for (; tb < tend; tb += stride) {
      const bool chunk = d0.y < 0;
      const int nv = chunk ? 1 : d0.y - d0.x;
      const int segraw = tl.rowptr[min(d0.x + lane, max(d0.x, d0.y))];
      const int4 d2 = desc(tb + wv + 2 * stride);
      float2 carry[2] = {{0.f, 0.f}, {0.f, 0.f}};
      int j = 0;
      round(A, d0, 0, d0, 1, segraw, chunk, nv, j, carry);
      round(A, d0, 1, d1, 0, segraw, chunk, nv, j, carry);
      d0 = d1;
      d1 = d2;
    }
  }
  // ---- block partials in the layout of the edge MLP's parameters after W1
  // (offset LD^2): db1, dW2, db2, dgamma, dbeta
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  constexpr int ob1 = LD * LD, oW2 = LD * LD + LD, ob2 = 2 * LD * LD + LD, og = 2 * LD * LD + 2 * LD;
#pragma unroll
  for (int u = 0; u < C32_HB; ++u)
#pragma unroll
    for (int v = 0; v < C32_HB; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        base[oW2 + (size_t)(16 * (ob0 + u) + 4 * g + r) * LD + 16 * (nb0 + v) + i] = aw2[u * C32_HB + v][r];
  if (i == 0)
#pragma unroll
    for (int t = 0; t < 3; ++t)
      if (t < nones)
#pragma unroll
        for (int r = 0; r < 4; ++r) base[ob2 + 16 * (ob0 + uones + t) + 4 * g + r] = ab2[t][r];
  __syncthreads();
  float* red = S.st[0];  // [3][R32_NW][LD]: dgamma, dbeta, db1
  {
    // colsum16: lane i holds features f0 + 4 (i / 2) + 2 (i % 2) + {0, 1};
    // colsum16_tail: lanes i, i ^ 1 hold value k of blocks 8, 9
    const int f = f0 + 4 * (i >> 1) + 2 * (i & 1);
    *reinterpret_cast<float2*>(red + (0 * R32_NW + wv) * LD + f) = dga;
    *reinterpret_cast<float2*>(red + (1 * R32_NW + wv) * LD + f) = dbe;
    *reinterpret_cast<float2*>(red + (2 * R32_NW + wv) * LD + f) = db1;
    if ((i & 1) == 0) {
      const int k = (((i >> 3) & 1) << 2) | (((i >> 2) & 1) << 1) | ((i >> 1) & 1);
      const int ft = f0 + 4 * (8 + (k >> 2)) + (k & 3);
      red[(0 * R32_NW + wv) * LD + ft] = tga;
      red[(1 * R32_NW + wv) * LD + ft] = tbe;
      red[(2 * R32_NW + wv) * LD + ft] = tb1;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < 3 * LD; idx += R32_NT) {
    const int k2 = idx / LD, c = idx % LD;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) v += red[(k2 * R32_NW + u) * LD + c];
    base[k2 == 2 ? ob1 + c : og + k2 * LD + c] = v;
  }
}

// ======================================================= weight gradient
// dW[o][n] = sum over rows of G[row][o] X[row][n] for two row-major fp32
// [M][LD] streams (the width-160 reverse leaves dW1e = sum zbar^T e to this
// pass).  Rounds of 64 rows: each wave loads 16 rows of both streams in the
// row layout, stages them in LDS, and after a block barrier adds the round
// into its quarter of dW, a block of (NOB / 2)^2 16 x 16 tiles, with the
// rows as K (accumulators in AGPRs; per 4 rows NOB LDS reads feed
// (NOB / 2)^2 MFMAs); the next round's rows are requested before the
// round's MFMAs.  Rows are added in ascending order within a block.
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_wgrad_r32(int64_t M, const float* __restrict__ Gm, const float* __restrict__ Xm, Partials part) {
  typedef R32<LD> Z;
  constexpr int SLD = LD + 16;  // lane groups 0, 1 of a staging write hit distinct banks
  // wave wv owns the HB x HB block of 16 x 16 tiles (ob0 + u, nb0 + v)
  constexpr int HB = Z::NOB / 2, TPW = HB * HB;
  __shared__ __align__(16) float st[2][B32_ROWS * SLD];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int f0 = Z::KL * g;
  const int ob0 = HB * (wv >> 1), nb0 = HB * (wv & 1);
  const int64_t nr = (M + B32_ROWS - 1) / B32_ROWS;
  f32x4 aw[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) aw[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float xg[Z::KL], xx[Z::KL];
  auto load = [&](int64_t r) {
    const int64_t row = min(r * B32_ROWS + 16 * wv + i, M - 1);
    load_row32<LD>(xg, Gm + (size_t)row * LD + f0);
    load_row32<LD>(xx, Xm + (size_t)row * LD + f0);
  };
  auto stage = [&](float* B, const float (&v)[Z::KL], bool live) {
    float* q = B + (16 * wv + i) * SLD + f0;
#pragma unroll
    for (int c = 0; c < Z::KC; ++c)
      *reinterpret_cast<f32x4*>(q + 4 * c) =
          live ? f32x4{v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]} : f32x4{0.f, 0.f, 0.f, 0.f};
  };
  int64_t r = blockIdx.x;
  if (r < nr) load(r);
  for (; r < nr; r += gridDim.x) {
    const bool live = r * B32_ROWS + 16 * wv + i < M;
    stage(st[0], xg, live);
    stage(st[1], xx, live);
    __syncthreads();
    if (r + gridDim.x < nr) load(r + gridDim.x);
    __builtin_amdgcn_sched_barrier(0);
    // A[m][k] = G[row k][16 ob + m], B[k][n] = X[row k][16 nb + n], K = 4
    // rows; the next 4 rows' operands are read from LDS before this step's
    // products (the scheduling barrier keeps them there), so their latency
    // lies under the MFMAs
    const float* pa = st[0] + g * SLD + 16 * ob0 + i;
    const float* pb = st[1] + g * SLD + 16 * nb0 + i;
    float A[2][HB], B[2][HB];
    auto rd = [&](int kk, float (&a)[HB], float (&b)[HB]) {
#pragma unroll
      for (int u = 0; u < HB; ++u) {
        a[u] = pa[4 * kk * SLD + 16 * u];
        b[u] = pb[4 * kk * SLD + 16 * u];
      }
    };
    rd(0, A[0], B[0]);
#pragma unroll
    for (int kk = 0; kk < B32_ROWS / 4; ++kk) {
      const int c = kk & 1;
      if (kk + 1 < B32_ROWS / 4) rd(kk + 1, A[c ^ 1], B[c ^ 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < HB; ++u)
#pragma unroll
        for (int v = 0; v < HB; ++v)
          aw[u * HB + v] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[c][u], B[c][v], aw[u * HB + v], 0, 0, 0);
    }
    __syncthreads();
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int u = 0; u < HB; ++u)
#pragma unroll
    for (int v = 0; v < HB; ++v)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        base[(size_t)(16 * (ob0 + u) + 4 * g + q) * LD + 16 * (nb0 + v) + i] = aw[u * HB + v][q];
}

// ========================================================= edge encoder
// The edge encoder e = LN(W2 relu(W1 f + b1) + b2) (Sec. 2.1: the edge
// features are encoded to the latent width by an MLP with LayerNorm) in this
// row layout, forward and reverse.  The first layer (K = 4) runs on VALU as
// one fma chain per feature from b1, k = 0..3, identical in both kernels, so
// the reverse recomputes the forward's values bitwise; the second layer is
// gemm32 on the fragment-major W2 (in LDS in the forward, from L2 in the
// reverse, whose LDS holds the staged rows).
constexpr int EK = 4;  // edge input features

// z[s] = b1[f0 + s] + W1[f0 + s] . x, the lane's KL features (w1 holds each
// feature's four input weights).
template <int LD>
__device__ __forceinline__ void enc_z1_r32(const float4* w1, const float* b1, float4 x, int f0,
                                           float (&z)[R32<LD>::KL]) {
#pragma unroll
  for (int s = 0; s < R32<LD>::KL; ++s) {
    const float4 wr = w1[f0 + s];
    float v = b1[f0 + s];
    v = __builtin_fmaf(wr.x, x.x, v);
    v = __builtin_fmaf(wr.y, x.y, v);
    v = __builtin_fmaf(wr.z, x.z, v);
    v = __builtin_fmaf(wr.w, x.w, v);
    z[s] = v;
  }
}

template <int LD>
struct __attribute__((aligned(16))) EncVec32 {
  __attribute__((aligned(16))) float4 w1[LD];  // W1 by output feature
  __attribute__((aligned(16))) float b1[LD];
  __attribute__((aligned(16))) float b2[LD];
  __attribute__((aligned(16))) float g[LD];
  __attribute__((aligned(16))) float bt[LD];
};
template <int LD>
__device__ __forceinline__ void stage_enc_vec(EncVec32<LD>& V, const MlpW& w, int tid) {
  for (int f = tid; f < LD; f += R32_NT) {
    V.w1[f] = float4{w.W1f[f * EK], w.W1f[f * EK + 1], w.W1f[f * EK + 2], w.W1f[f * EK + 3]};
    V.b1[f] = w.b1[f];
    V.b2[f] = w.b2[f];
    V.g[f] = w.gamma[f];
    V.bt[f] = w.beta[f];
  }
}

template <int LD>
struct __attribute__((aligned(16))) EncFwd32Lds {
  EncVec32<LD> V;
  __attribute__((aligned(16))) float w2[LD * LD];  // fragment-major W2
};

// Forward: one wave per 16-edge unit, no block barrier in the loop; the
// next unit's inputs are in flight while one is computed.
template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_edge_enc_r32(int64_t E, const float* __restrict__ f_in, MlpW w, float eps, float* __restrict__ e_out) {
  typedef R32<LD> Z;
  __shared__ __align__(16) EncFwd32Lds<LD> S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int idx = tid; idx < LD * LD / 4; idx += R32_NT)
    reinterpret_cast<f32x4*>(S.w2)[idx] = reinterpret_cast<const f32x4*>(w.F2)[idx];
  stage_enc_vec<LD>(S.V, w, tid);
  __syncthreads();
  const int64_t nu = (E + 15) >> 4;
  const UnitRange ur = unit_range<R32_NW>(nu, wv);
  if (ur.t >= ur.end) return;
  const int f0 = Z::KL * g;
  // rows clamped into [0, E): rows past E read row E - 1 and store nothing
  auto load = [&](int64_t u) { return *reinterpret_cast<const float4*>(f_in + min(u * 16 + i, E - 1) * EK); };
  float4 fa = load(ur.t);
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const float4 fn = load(u + ur.stride);
    // LDS reads through an opaque reference: otherwise the loop-invariant
    // weight reads are hoisted out of the loop into (far too many) registers
    const EncFwd32Lds<LD>& L = fresh(S);
    float a1[Z::KL];
    enc_z1_r32<LD>(L.V.w1, L.V.b1, fa, f0, a1);
#pragma unroll
    for (int s = 0; s < Z::KL; ++s) a1[s] = relu(a1[s]);
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(L.V.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, L.w2, lane);
    // ---- LayerNorm over the row's DR real features (padded ones are 0)
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
    const float rstd = __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / Z::DR) + eps);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
      acc[ob] = *reinterpret_cast<const f32x4*>(L.V.g + f0 + 4 * ob) * (acc[ob] * rstd) +
                *reinterpret_cast<const f32x4*>(L.V.bt + f0 + 4 * ob);
    if (u * 16 + i < E) store_row32<LD>(e_out + (size_t)(u * 16 + i) * LD + f0, acc);
    fa = fn;
  }
}

// Reverse: every parameter gradient of the encoder from dL/de in one pass.
// Four waves per block, each the reverse of one 16-edge unit per round (the
// forward recomputed bitwise, the LayerNorm reverse, da1 = W2^T dz2, the
// ReLU mask), staging its rows of dz2, a1, dz1 and the inputs [f, 1] in LDS;
// after the round's second barrier each wave adds the round's 64 rows into
// its tiles of dW2 = sum dz2^T a1 (NOB^2 / 4 tiles, row-major), its blocks
// of dW1 | db1 = sum dz1^T [f, 1] and the ones column db2 = sum dz2 (output
// blocks wv, wv + 4, wv + 8), with K = the rows.  dgamma and dbeta are DPP
// column sums per unit.  Per-block partials in the encoder's parameter
// order: W1 [LD][4], b1, W2 [LD][LD], b2, gamma, beta.
template <int LD>
struct __attribute__((aligned(16))) EncBwd32Lds {
  EncVec32<LD> V;
  __attribute__((aligned(16))) float st[3][B32_ROWS * (LD + 16)];  // dz2, a1, dz1
  __attribute__((aligned(16))) float fx[B32_ROWS * 8];             // [f0..f3, 1, 0, 0, 0] per row
};

template <int LD>
__global__ void __launch_bounds__(R32_NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_edge_enc_bwd_r32(int64_t E, const float* __restrict__ f_in, const float* __restrict__ ebar, MlpW w, float eps,
                   Partials part) {
  typedef R32<LD> Z;
  constexpr int SL = LD + 16;                 // staged row stride (floats)
  // wave wv owns the HB x HB block of dW2 tiles (ob0 + u, nb0 + v) and the
  // db2 / dW1 | db1 columns of nones of its block row's HB output blocks
  constexpr int HB = Z::NOB / 2, TPW = HB * HB;
  __shared__ __align__(16) EncBwd32Lds<LD> S;
  float* X = S.st[0];
  float* Y = S.st[1];
  float* Z1 = S.st[2];
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int f0 = Z::KL * g;
  const int ob0 = HB * (wv >> 1), nb0 = HB * (wv & 1);
  const int uones = (wv & 1) ? HB - HB / 2 : 0, nones = (wv & 1) ? HB / 2 : HB - HB / 2;
  stage_enc_vec<LD>(S.V, w, tid);
  __syncthreads();

  // The block's units: XCD-contiguous ranges; wave wv takes unit tb + wv of
  // every round; all four waves run the same number of rounds.
  const int64_t nu = (E + 15) >> 4;
  const int G = gridDim.x;
  int64_t tb, stride, tend;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (nu + 7) >> 3;
    const int64_t lo = x * chunk;
    tend = min(nu, lo + chunk);
    tb = lo + (int64_t)(blockIdx.x >> 3) * R32_NW;
    stride = (int64_t)per * R32_NW;
  } else {
    tb = (int64_t)blockIdx.x * R32_NW;
    stride = (int64_t)G * R32_NW;
    tend = nu;
  }
  const int64_t lastE = max(E - 1, (int64_t)0);
  auto grow = [&](int64_t u) { return min(u * 16 + i, lastE); };
  struct In {
    float4 x;
    float yb[Z::KL];
  };
  auto load_in = [&](int64_t u, In& I) {
    I.x = *reinterpret_cast<const float4*>(f_in + grow(u) * EK);
    load_row32<LD>(I.yb, ebar + (size_t)grow(u) * LD + f0);
  };

  f32x4 aw2[TPW], ab2[3], aw1[3];
#pragma unroll
  for (int t = 0; t < TPW; ++t) aw2[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < 3; ++t) ab2[t] = aw1[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  float tga = 0.f, tbe = 0.f;  // width 160: blocks 8, 9 (tail butterfly)
  const int srow = 16 * wv + i;
  auto stage_row = [&](float* B, const float (&v)[Z::KL], bool live) {
    float* p = B + srow * SL + f0;
#pragma unroll
    for (int c = 0; c < Z::KC; ++c)
      *reinterpret_cast<f32x4*>(p + 4 * c) =
          live ? f32x4{v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]} : f32x4{0.f, 0.f, 0.f, 0.f};
  };
  auto colsum = [&](const f32x4 (&v)[Z::NOB], float2& acc8, float& tail) {
    f32x4 p8[8];
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) p8[ob] = v[ob];
    const float2 c = colsum16(p8, i);
    acc8.x += c.x;
    acc8.y += c.y;
    if constexpr (Z::NOB == 10) tail += w160::colsum16_tail(reinterpret_cast<const f32x4(&)[10]>(v), i);
  };

  // units past the block's range (the last round's) are empty: their rows
  // are never staged as live or stored
  auto round = [&](In& I, int64_t u) {
    const bool live = u < tend && u * 16 + i < E;
    const int oz = opaque_zero();
    const EncVec32<LD>& V = fresh(S.V);
    // ---- z1, a1 = relu(z1), the mask z1 > 0 (the forward's values)
    float a1[Z::KL];
    enc_z1_r32<LD>(V.w1, V.b1, I.x, f0, a1);
    uint64_t mask = 0;
#pragma unroll
    for (int s = 0; s < Z::KL; ++s) {
      if (a1[s] > 0.f) mask |= 1ull << s;
      a1[s] = relu(a1[s]);
    }
    __syncthreads();  // every wave's products of the previous round are done
    stage_row(Y, a1, live);
    if (g == 0) {
      float* fp = S.fx + srow * 8;
      *reinterpret_cast<float4*>(fp) = I.x;
      *reinterpret_cast<float4*>(fp + 4) = float4{1.f, 0.f, 0.f, 0.f};
    }
    // ---- z2 = b2 + W2 a1 and its LayerNorm (DR real features)
    f32x4 acc[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(V.b2 + f0 + 4 * ob);
    gemm32<LD>(acc, a1, w.F2 + oz, lane);
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
        acc[ob][r] -= mean;
        if (Z::DR == LD || f0 + 4 * ob + r < Z::DR) sq += acc[ob][r] * acc[ob][r];
      }
    const float rstd = __builtin_amdgcn_rsqf(sum_q(sq) * (1.0f / Z::DR) + eps);
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] *= rstd;  // xhat
    // ---- dgamma += sum_rows ybar xhat, dbeta += sum_rows ybar (live rows)
    f32x4 t[Z::NOB];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
      t[ob] = live ? f32x4{I.yb[4 * ob], I.yb[4 * ob + 1], I.yb[4 * ob + 2], I.yb[4 * ob + 3]}
                   : f32x4{0.f, 0.f, 0.f, 0.f};
    colsum(t, dbe, tbe);
    {
      f32x4 p[Z::NOB];
#pragma unroll
      for (int ob = 0; ob < Z::NOB; ++ob) p[ob] = t[ob] * acc[ob];
      colsum(p, dga, tga);
    }
    // ---- dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = ybar gamma
    // (padded features: gamma = 0, dz2 zeroed)
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) {
      t[ob] *= *reinterpret_cast<const f32x4*>(V.g + f0 + 4 * ob);
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
        dz[4 * ob + r] = Z::DR == LD || f0 + 4 * ob + r < Z::DR ? rstd * (t[ob][r] - m1 - acc[ob][r] * m2) : 0.f;
    stage_row(X, dz, live);
    // ---- da1 = W2^T dz2, dz1 = da1 where z1 > 0
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    gemm32<LD>(acc, dz, w.F2t + oz, lane);
    float d1[Z::KL];
#pragma unroll
    for (int ob = 0; ob < Z::NOB; ++ob)
#pragma unroll
      for (int r = 0; r < 4; ++r) d1[4 * ob + r] = (mask >> (4 * ob + r)) & 1ull ? acc[ob][r] : 0.f;
    stage_row(Z1, d1, live);
    __syncthreads();  // the round's rows are staged
    // ---- the round's 64 rows into this wave's gradient tiles
#pragma unroll 2
    for (int kk = 0; kk < B32_ROWS / 4; ++kk) {
      const int rr = 4 * kk + g, r0 = rr * SL;
      const float fb = i < 8 ? S.fx[rr * 8 + i] : 0.f;  // [f, 1, 0...] of row rr, column i
      float A[HB], B[HB];
#pragma unroll
      for (int u = 0; u < HB; ++u) {
        A[u] = X[r0 + 16 * (ob0 + u) + i];
        B[u] = Y[r0 + 16 * (nb0 + u) + i];
      }
#pragma unroll
      for (int t3 = 0; t3 < 3; ++t3)
        if (t3 < nones) {
          ab2[t3] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[uones + t3], 1.0f, ab2[t3], 0, 0, 0);
          aw1[t3] = __builtin_amdgcn_mfma_f32_16x16x4f32(Z1[r0 + 16 * (ob0 + uones + t3) + i], fb, aw1[t3], 0, 0, 0);
        }
#pragma unroll
      for (int u = 0; u < HB; ++u)
#pragma unroll
        for (int v = 0; v < HB; ++v)
          aw2[u * HB + v] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], B[v], aw2[u * HB + v], 0, 0, 0);
    }
  };

  if (tb < tend) {
    In A, B;
    load_in(tb + wv, A);
    for (; tb < tend; tb += 2 * stride) {
      load_in(tb + wv + stride, B);
      round(A, tb + wv);
      load_in(tb + wv + 2 * stride, A);
      if (tb + stride < tend) round(B, tb + wv + stride);
    }
  }
  // ---- block partials in the encoder's parameter order
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  constexpr int oW1 = 0, ob1 = EK * LD, oW2 = (EK + 1) * LD, ob2 = (EK + 1) * LD + LD * LD;
  constexpr int og = ob2 + LD, obt = og + LD;
#pragma unroll
  for (int u = 0; u < HB; ++u)
#pragma unroll
    for (int v = 0; v < HB; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        base[oW2 + (size_t)(16 * (ob0 + u) + 4 * g + r) * LD + 16 * (nb0 + v) + i] = aw2[u * HB + v][r];
#pragma unroll
  for (int t3 = 0; t3 < 3; ++t3) {
    const int ob = ob0 + uones + t3;
    if (t3 < nones)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int f = 16 * ob + 4 * g + r;
        if (i == 0) base[ob2 + f] = ab2[t3][r];
        if (i < EK) base[oW1 + f * EK + i] = aw1[t3][r];
        if (i == EK) base[ob1 + f] = aw1[t3][r];
      }
  }
  __syncthreads();
  float* red = S.st[0];  // [2][R32_NW][LD]: dgamma, dbeta
  {
    // colsum16: lane i holds features f0 + 4 (i / 2) + 2 (i % 2) + {0, 1};
    // colsum16_tail (width 160): lanes i, i ^ 1 hold value k of blocks 8, 9
    const int f = f0 + 4 * (i >> 1) + 2 * (i & 1);
    *reinterpret_cast<float2*>(red + (0 * R32_NW + wv) * LD + f) = dga;
    *reinterpret_cast<float2*>(red + (1 * R32_NW + wv) * LD + f) = dbe;
    if (Z::NOB == 10 && (i & 1) == 0) {
      const int k = (((i >> 3) & 1) << 2) | (((i >> 2) & 1) << 1) | ((i >> 1) & 1);
      const int ft = f0 + 4 * (8 + (k >> 2)) + (k & 3);
      red[(0 * R32_NW + wv) * LD + ft] = tga;
      red[(1 * R32_NW + wv) * LD + ft] = tbe;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < 2 * LD; idx += R32_NT) {
    const int k2 = idx / LD, c = idx % LD;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < R32_NW; ++u) v += red[(k2 * R32_NW + u) * LD + c];
    base[(k2 == 0 ? og : obt) + c] = v;
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kRows32Blocks = 256;

hipError_t launch_edge_fwd_r32(int lat, const EdgeTiles& t, const void* e_in, void* e_out, int write_e,
                               const void* Pn, const MlpW& w, float eps, float* agg, float* slots, hipStream_t s) {
  if (t.n_tiles <= 0) return hipSuccess;
  if (t.n_edges <= 0 || !w.F1 || !w.F2) return hipErrorInvalidValue;
  const int64_t need = (t.n_tiles + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kRows32Blocks);
  if (g >= 8) g &= ~7;
#define F(LD)                                                                                                      \
  hipLaunchKernelGGL(k_edge_fwd_r32<LD>, dim3(g), dim3(R32_NT), 0, s, t, (const float*)e_in, (float*)e_out, write_e, \
                     (const float*)Pn, w, eps, agg, slots)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_edge_bwd_r32(int lat, const EdgeTiles& t, const void* e, const float* ebar_in, int have_ebar,
                               float* ebar_out, const void* Pn, const float* aggbar, const MlpW& w, float eps,
                               void* zbar, float* R, float* slots, const Partials& part, int* nblocks,
                               hipStream_t s) {
  *nblocks = 0;
  if (t.n_tiles <= 0) return hipSuccess;
  if ((lat != B32_LD && lat != C32_LD) || t.n_edges <= 0 || part.stride < 2LL * lat * lat + 4 * lat || !w.F1 ||
      !w.F2 || !w.F1t || !w.F2t)
    return hipErrorInvalidValue;
  const int64_t need = (t.n_tiles + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, std::min(kRows32Blocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
  if (lat == C32_LD)
    hipLaunchKernelGGL(k_edge_bwd_r32w, dim3(g), dim3(R32_NT), 0, s, t, (const float*)e, ebar_in, have_ebar,
                       ebar_out, (const float*)Pn, aggbar, w, eps, (float*)zbar, R, slots, part);
  else
    hipLaunchKernelGGL(k_edge_bwd_r32, dim3(g), dim3(R32_NT), 0, s, t, (const float*)e, ebar_in, have_ebar,
                       ebar_out, (const float*)Pn, aggbar, w, eps, (float*)zbar, R, slots, part);
  return hipGetLastError();
}

hipError_t launch_wgrad_r32(int lat, int64_t M, const float* G, const float* X, const Partials& part, int* nblocks,
                            hipStream_t s) {
  *nblocks = 0;
  if (M <= 0) return hipSuccess;
  if ((lat != B32_LD && lat != C32_LD) || part.stride < (int64_t)lat * lat) return hipErrorInvalidValue;
  const int64_t need = (M + B32_ROWS - 1) / B32_ROWS;
  const int g = (int)std::min<int64_t>(need, std::min(kRows32Blocks, part.max_blocks));
  *nblocks = g;
  if (lat == C32_LD)
    hipLaunchKernelGGL(k_wgrad_r32<C32_LD>, dim3(g), dim3(R32_NT), 0, s, M, G, X, part);
  else
    hipLaunchKernelGGL(k_wgrad_r32<B32_LD>, dim3(g), dim3(R32_NT), 0, s, M, G, X, part);
  return hipGetLastError();
}

hipError_t launch_edge_enc_r32(int lat, int64_t E, const float* f, const MlpW& w, float eps, void* e_out,
                               hipStream_t s) {
  if (E <= 0) return hipSuccess;
  if (!w.F2) return hipErrorInvalidValue;
  const int64_t need = ((E + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, kRows32Blocks);
  if (g >= 8) g &= ~7;
#define F(LD) \
  hipLaunchKernelGGL(k_edge_enc_r32<LD>, dim3(g), dim3(R32_NT), 0, s, E, f, w, eps, (float*)e_out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_edge_enc_bwd_r32(int lat, int64_t E, const float* f, const void* ebar, const MlpW& w, float eps,
                                   const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (E <= 0) return hipSuccess;
  if (!w.F2 || !w.F2t || part.stride < (int64_t)lat * lat + (EK + 4) * lat) return hipErrorInvalidValue;
  const int64_t need = ((E + 15) / 16 + R32_NW - 1) / R32_NW;
  int g = (int)std::min<int64_t>(need, std::min(kRows32Blocks, part.max_blocks));
  if (g >= 8) g &= ~7;
  *nblocks = g;
#define F(LD)                                                                                                 \
  hipLaunchKernelGGL(k_edge_enc_bwd_r32<LD>, dim3(g), dim3(R32_NT), 0, s, E, f, (const float*)ebar, w, eps, \
                     part)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

}  // namespace mgn
