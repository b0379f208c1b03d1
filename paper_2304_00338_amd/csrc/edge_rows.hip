// Edge phase of one MGN message-passing step, forward, bf16 operands, with
// one wave per receiver-aligned tile (Sec. 2.1: every edge latent is updated
// by the edge MLP from itself and its two end nodes, then each node sums the
// new messages of its in-edges).
//
// Work split.  Each of the 8 waves of a block runs its own persistent loop
// over tiles; the only block barrier is the one after the weights are
// staged in LDS.  Lane l (i = l & 15, q = l >> 4) holds rows i and 16 + i of
// the wave's tile and the 32 contiguous features [32q, 32q + 32) of each
// row.  The GEMMs run transposed (C[feature][row] = W x^T): the A operand is
// a 16-row block of the row-permuted weights (perm_row) read from LDS, the B
// operand is the lane's own 8-feature runs of x, and the C fragment of
// output block ob gives the lane features 32q + 4ob + r.  So GEMM outputs
// are already the next GEMM's B operand, and every LayerNorm statistic is a
// sum over the lane's 32 values plus two cross-lane steps (the four lanes
// that share a row).
//
// Adds of bf16 inputs into fp32 accumulators (the node products P_s + P_r
// and the residual e + m) are MFMAs with a 0/1 selection operand: one
// product per output, so each is a single fp32 rounding, as a VALU add.
//
// Node sums: the wave stages each 16-row half of the messages in its own
// LDS area and sums every in-segment in ascending row order from 0.0, so a
// node's aggregate does not depend on where its segment sits in a tile.
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

constexpr int RW_LDW = D + 8;  // LDS row stride of the staged weights (bf16)
constexpr int RW_LDM = D + 4;  // LDS row stride of a wave's message half-tile (fp32)

struct __attribute__((aligned(16))) RowsLds {
  __attribute__((aligned(16))) bf16 W1[D * RW_LDW];
  __attribute__((aligned(16))) bf16 W2[D * RW_LDW];
  __attribute__((aligned(16))) float b1[D];
  __attribute__((aligned(16))) float b2[D];
  __attribute__((aligned(16))) float g[D];
  __attribute__((aligned(16))) float bt[D];
  __attribute__((aligned(16))) float stage[NW][16 * RW_LDM];
};

typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// The 0/1 operand that adds a B fragment (features 32q + 8s + j) into the C
// fragment of output block ob = 2s + h: A[m][k] = 1 iff k = (m/4)*8 + 4h + m%4.
__device__ __forceinline__ bf16x8 select_frag(int h, int i, int q) {
  bf16x8 a;
#pragma unroll
  for (int j = 0; j < 8; ++j) a[j] = (bf16)(((i >> 2) == q && j == 4 * h + (i & 3)) ? 1.f : 0.f);
  return a;
}

__device__ __forceinline__ bf16x8 as_frag(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

// The streams of one tile row pair a lane needs: its 32-feature run of the
// edge latent and of the two gathered node products, for rows i and 16 + i.
struct RowLoads {
  uint4 e[2][4], ps[2][4], pr[2][4];
};

__device__ __forceinline__ int tile_rows(int4 d) { return d.w - d.z; }

// max(x, 0) as one integer max on the bit pattern (negative floats have the
// sign bit set, so they compare below +0.0 as signed integers).
__device__ __forceinline__ float relu(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

template <int CTRL>
__device__ __forceinline__ float xlane(float v) {
  return __shfl_xor(v, CTRL, 64);
}
// Sum over the four lanes that hold the same row (q = 0..3).
__device__ __forceinline__ float sum_rowlanes(float s) {
  s += xlane<16>(s);
  s += xlane<32>(s);
  return s;
}

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_fwd_rows(EdgeTiles tl, const bf16* __restrict__ e_in, bf16* __restrict__ e_out, int write_e,
                const bf16* __restrict__ Pn, MlpW w, float eps, float* __restrict__ agg,
                float* __restrict__ slots) {
  __shared__ __align__(16) RowsLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  {
    const bf16* W1p = (const bf16*)w.W1p;
    const bf16* W2p = (const bf16*)w.W2p;
    for (int idx = tid; idx < D * D / 8; idx += NT) {
      const int row = idx >> 4, c = (idx & 15) * 8;
      *reinterpret_cast<uint4*>(S.W1 + row * RW_LDW + c) = *reinterpret_cast<const uint4*>(W1p + row * D + c);
      *reinterpret_cast<uint4*>(S.W2 + row * RW_LDW + c) = *reinterpret_cast<const uint4*>(W2p + row * D + c);
    }
    if (tid < D) {
      S.b1[tid] = w.b1[tid];
      S.b2[tid] = w.b2[tid];
      S.g[tid] = w.gamma[tid];
      S.bt[tid] = w.beta[tid];
    }
  }
  __syncthreads();

  // Tile order: blocks are dealt to the 8 XCDs round-robin, so the waves of
  // the blocks of one XCD walk one contiguous eighth of the tiles (their
  // node products then mostly share that XCD's L2).
  const int64_t NTL = tl.n_tiles;
  const int G = gridDim.x;
  int64_t t, stride, tend;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (NTL + 7) >> 3;
    const int64_t lo = x * chunk;
    tend = min(NTL, lo + chunk);
    t = lo + (int64_t)(blockIdx.x >> 3) * NW + wv;
    stride = (int64_t)per * NW;
  } else {
    t = (int64_t)blockIdx.x * NW + wv;
    stride = (int64_t)G * NW;
    tend = NTL;
  }
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
  // sender / receiver of rows i and 16 + i of a tile (0 past its end)
  auto load_sr = [&](int4 d, int (&s)[2], int (&r)[2]) {
    const int n = tile_rows(d);
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = rb * 16 + i;
      s[rb] = row < n ? tl.senders[d.z + row] : 0;
      r[rb] = row < n ? tl.receivers[d.z + row] : 0;
    }
  };
  // Rows past the tile's end load a copy of its last edge row and node 0's
  // products: rows never mix inside the products or the LayerNorm, and such
  // rows are neither stored nor summed.
  auto issue = [&](int4 d, const int (&s)[2], const int (&r)[2], RowLoads& L) {
    const int n = tile_rows(d);
    if (n <= 0) return;  // a tile of edge-less nodes: nothing to load
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int rc = max(0, min(rb * 16 + i, n - 1));
      const bf16* ep = e_in + ((size_t)d.z + rc) * D + 32 * q;
      const bf16* sp = Pn + (size_t)s[rb] * (2 * D) + 32 * q;
      const bf16* rp = Pn + (size_t)r[rb] * (2 * D) + D + 32 * q;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        L.e[rb][k] = *reinterpret_cast<const uint4*>(ep + 8 * k);
        L.ps[rb][k] = *reinterpret_cast<const uint4*>(sp + 8 * k);
        L.pr[rb][k] = *reinterpret_cast<const uint4*>(rp + 8 * k);
      }
    }
  };

  int4 d0 = desc(t), d1 = desc(t + stride), d2 = desc(t + 2 * stride);
  int s0[2], r0[2], s1[2], r1[2];
  load_sr(d0, s0, r0);
  load_sr(d1, s1, r1);
  RowLoads cur;
  issue(d0, s0, r0, cur);
  float* stage = S.stage[wv];

  for (; t < tend; t += stride) {
    const int n = tile_rows(d0);
    const int4 d3 = desc(t + 3 * stride);
    int s2[2], r2[2];
    load_sr(d2, s2, r2);
    // in-segment starts of the tile's nodes (lane j holds the start of node j)
    const int nv = d0.y >= 0 ? d0.y - d0.x : 1;
    int segv = 0;
    if (d0.y >= 0) {
      if (lane <= nv) segv = tl.rowptr[d0.x + lane] - d0.z;
    } else {
      segv = lane == 0 ? 0 : n;
    }

    RowLoads nxt;
    bool issued = false;
    float2 carry = {0.f, 0.f};
    int j = 0;  // next node whose sum is open
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      // ---- z1 = b1 + P_s + P_r + W1e e
      f32x4 acc[8];
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        acc[ob] = *reinterpret_cast<const f32x4*>(S.b1 + 32 * q + 4 * ob);
        const bf16x8 sel = (ob & 1) ? sel1 : sel0;
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, as_frag(cur.ps[rb][ob >> 1]), acc[ob], 0, 0, 0);
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, as_frag(cur.pr[rb][ob >> 1]), acc[ob], 0, 0, 0);
      }
      if (rb == 1 && t + stride < tend) {
        // the node products of this tile are consumed: put the next tile in flight
        issue(d1, s1, r1, nxt);
        issued = true;
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(S.W1 + (ob * 16 + i) * RW_LDW + 32 * q + 8 * s);
          acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, as_frag(cur.e[rb][s]), acc[ob], 0, 0, 0);
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
      // ---- z2 = b2 + W2 a1
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + 32 * q + 4 * ob);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(S.W2 + (ob * 16 + i) * RW_LDW + 32 * q + 8 * s);
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
      float* srow = stage + i * RW_LDM + 32 * q;
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        const f32x4 ga = *reinterpret_cast<const f32x4*>(S.g + 32 * q + 4 * ob);
        const f32x4 be = *reinterpret_cast<const f32x4*>(S.bt + 32 * q + 4 * ob);
        acc[ob] = ga * (acc[ob] * rstd) + be;  // message m
        *reinterpret_cast<f32x4*>(srow + 4 * ob) = acc[ob];
      }
      // ---- e_out = e + m
      const int row = rb * 16 + i;
      if (write_e) {
        uint4 o[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          f32x4 lo = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel0, as_frag(cur.e[rb][s]), acc[2 * s], 0, 0, 0);
          f32x4 hi = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel1, as_frag(cur.e[rb][s]), acc[2 * s + 1], 0, 0, 0);
          bf16x8 v;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[r] = (bf16)lo[r];
            v[4 + r] = (bf16)hi[r];
          }
          o[s] = __builtin_bit_cast(uint4, v);
        }
        if (row < n) {
          bf16* op = e_out + ((size_t)d0.z + row) * D + 32 * q;
#pragma unroll
          for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(op + 8 * s) = o[s];
        }
      }
      wave_lds_sync();
      // ---- in-segment sums over this half's rows; lane owns features 2l, 2l+1
      const int lo_row = rb * 16, hi_row = rb * 16 + 16;
      while (j < nv) {
        const int a = __builtin_amdgcn_readlane(segv, j), b = __builtin_amdgcn_readlane(segv, j + 1);
        const int u0 = max(a, lo_row), u1 = min(b, hi_row);
        for (int u = u0; u < u1; ++u) {
          const float2 v = *reinterpret_cast<const float2*>(stage + (u - lo_row) * RW_LDM + 2 * lane);
          carry.x += v.x;
          carry.y += v.y;
        }
        if (b > hi_row) break;
        float* dst = d0.y >= 0 ? agg + (size_t)(d0.x + j) * D : slots + (size_t)(-1 - d0.y) * D;
        *reinterpret_cast<float2*>(dst + 2 * lane) = carry;
        carry = float2{0.f, 0.f};
        ++j;
      }
      wave_lds_sync();
    }
    if (!issued && t + stride < tend) issue(d1, s1, r1, nxt);
    cur = nxt;
    d0 = d1;
    d1 = d2;
    d2 = d3;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      s1[rb] = s2[rb];
      r1[rb] = r2[rb];
    }
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kRowsBlocks = 256;

hipError_t launch_edge_fwd_rows(const EdgeTiles& t, const void* e_in, void* e_out, int write_e, const void* Pn,
                                const MlpW& w, float eps, float* agg, float* slots, hipStream_t s) {
  if (t.n_tiles <= 0) return hipSuccess;
  const int64_t need = (t.n_tiles + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kRowsBlocks);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_edge_fwd_rows, dim3(g), dim3(NT), 0, s, t, (const bf16*)e_in, (bf16*)e_out, write_e,
                     (const bf16*)Pn, w, eps, agg, slots);
  return hipGetLastError();
}

}  // namespace mgn
