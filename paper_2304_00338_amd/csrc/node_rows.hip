// Node phase of one MGN message-passing step, bf16 operands, one wave per
// 16-node block (Sec. 2.1: every node latent is updated by the node MLP from
// itself and the sum of its incoming messages, with a residual connection;
// the first layer of the next edge MLP is split into per-node products).
//
// Each of the 8 waves of a block runs its own persistent loop over 16-row
// units in the lane layout of rows_common.hpp; the only block barriers stage
// the weights before the loop and combine the column sums after it.  Inputs
// of the next unit are in flight while a unit is computed.
//
//   k_node_fwd_rows  h_out = h + LN(W2 relu(W1 [h; agg] + b1) + b2)
//   k_emit_rows      P = [W1s h; W1r h] of the next edge layer
//   k_node_bwd_rows  back through the node MLP from dL/dh_out: dL/dh (residual
//                    included), dL/dagg, the streams a1, dz2, dz1 and block
//                    partials of dgamma, dbeta
//   k_wgrad_node     dW1 = sum dz1^T [h; agg], db1, dW2 = sum dz2^T a1, db2
#include "rows_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

constexpr int D2 = 2 * D;

struct __attribute__((aligned(16))) NodeLds {
  __attribute__((aligned(16))) bf16 W1[D * D2];  // [128][256], rows permuted, swizzled
  __attribute__((aligned(16))) bf16 W2[D * D];
  __attribute__((aligned(16))) float b1[D];
  __attribute__((aligned(16))) float b2[D];
  __attribute__((aligned(16))) float g[D];
  __attribute__((aligned(16))) float bt[D];
};

__device__ __forceinline__ void stage_node_mlp(NodeLds& S, const MlpW& w, int tid, bool beta) {
  stage_weights<D2>(S.W1, (const bf16*)w.W1p, tid);
  stage_weights<D>(S.W2, (const bf16*)w.W2p, tid);
  if (tid < D) {
    S.b1[tid] = w.b1[tid];
    S.b2[tid] = w.b2[tid];
    S.g[tid] = w.gamma[tid];
    S.bt[tid] = beta ? w.beta[tid] : 0.f;
  }
}

__device__ __forceinline__ f32x4 lds4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

// Row addressing: a unit's 16 rows are contiguous, so every access is a
// wave-uniform base (unit u's first row, kept in scalar registers) plus the
// lane's element offset lo = i * D + 8q (one register shared by all streams).
// Loads clamp the lane's row into [0, N) and the unit into [0, n_units), so
// the rows past N and the prefetches past a wave's last unit read row N - 1.
struct Rows {
  int64_t N, nu;
  int i, q;
  __device__ __forceinline__ int64_t base(int64_t u) const { return min(u, nu - 1) * 16 * D; }
  __device__ __forceinline__ int lo(int64_t u) const {
    return (int)min((int64_t)i, N - 1 - min(u, nu - 1) * 16) * D + 8 * q;
  }
  __device__ __forceinline__ bool valid(int64_t u) const { return u * 16 + i < N; }
};

// The 8 C-layout fragments of one fp32 [.][128] row at p + lo: v[ob] =
// features fo(ob, q) .. + 4 (lo includes the 8q).
__device__ __forceinline__ int fo0(int ob) { return 32 * (ob >> 1) + 4 * (ob & 1); }
__device__ __forceinline__ void load_row(const float* p, int lo, f32x4 (&v)[8]) {
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) v[ob] = *reinterpret_cast<const f32x4*>(p + lo + fo0(ob));
}
__device__ __forceinline__ void store_row(float* p, int lo, const f32x4 (&v)[8]) {
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) *reinterpret_cast<f32x4*>(p + lo + fo0(ob)) = v[ob];
}
// Four bf16 runs of one [.][128] row: run s = features 32s + 8q .. + 8.
__device__ __forceinline__ void store_runs(bf16* p, int lo, const bf16x8 (&v)[4]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(p + lo + 32 * s) = __builtin_bit_cast(uint4, v[s]);
}

// z1 = b1 + W1 [h; agg] for one unit (x[s]: run s of h for s < 4, of agg
// for s >= 4).
__device__ __forceinline__ void node_gemm1(const NodeLds& S, const AOff<D2>& A1, const bf16x8 (&x)[8], int q,
                                           f32x4 (&acc)[8]) {
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) acc[ob] = lds4(S.b1 + fo(ob, q));
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1.a(S.W1, ob, s), x[s], acc[ob], 0, 0, 0);
}

// z2 = b2 + W2 a1.
__device__ __forceinline__ void node_gemm2(const NodeLds& S, const AOff<D>& A2, const bf16x8 (&a1)[4], int q,
                                           f32x4 (&acc)[8]) {
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) acc[ob] = lds4(S.b2 + fo(ob, q));
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A2.a(S.W2, ob, s), a1[s], acc[ob], 0, 0, 0);
}

// ===================================================================== forward
// h_out = h_in + LN(MLP([h_in, agg])); h_out may alias h_in (each row is
// read before it is written, by the same lane).
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_node_fwd_rows(int64_t N, const float* h_in, const float* __restrict__ agg, MlpW w, float eps, float* h_out) {
  __shared__ NodeLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_node_mlp(S, w, tid, true);
  const AOff<D2> A1(i, q);
  const AOff<D> A2(i, q);
  __syncthreads();
  const Rows rw{N, (N + 15) >> 4, i, q};
  const UnitRange ur = unit_range(rw.nu, wv);
  if (ur.t >= ur.end) return;
  struct In {
    f32x4 h[8], a[8];
  };
  auto load = [&](int64_t u, In& X) {
    const int64_t b = rw.base(u);
    const int lo = rw.lo(u);
    load_row(h_in + b, lo, X.h);
    load_row(agg + b, lo, X.a);
  };
  auto unit = [&](In& X, int64_t u) {
    const NodeLds& L = fresh(S);
    bf16x8 x[8];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      x[s] = pack_run(X.h[2 * s], X.h[2 * s + 1]);
      x[4 + s] = pack_run(X.a[2 * s], X.a[2 * s + 1]);
    }
    f32x4 acc[8];
    node_gemm1(L, A1, x, q, acc);
    bf16x8 a1[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        a1[s][r] = (bf16)relu(acc[2 * s][r]);
        a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
      }
    node_gemm2(L, A2, a1, q, acc);
    ln_normalize(acc, eps);
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = X.h[ob] + (lds4(L.g + fo(ob, q)) * acc[ob] + lds4(L.bt + fo(ob, q)));
    if (rw.valid(u)) store_row(h_out + u * 16 * D, i * D + 8 * q, acc);
  };
  In A, B;
  int64_t u = ur.t;
  load(u, A);
  for (;;) {
    load(u + ur.stride, B);
    unit(A, u);
    u += ur.stride;
    if (u >= ur.end) break;
    load(u + ur.stride, A);
    unit(B, u);
    u += ur.stride;
    if (u >= ur.end) break;
  }
}

// P[v] = [W1s h[v]; W1r h[v]] in bf16 for the next edge layer.
struct __attribute__((aligned(16))) EmitLds {
  __attribute__((aligned(16))) bf16 Ws[D * D];
  __attribute__((aligned(16))) bf16 Wr[D * D];
};

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_emit_rows(int64_t N, const float* __restrict__ h, MlpW nx, bf16* __restrict__ P) {
  __shared__ EmitLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_weights<D>(S.Ws, (const bf16*)nx.W1sp, tid);
  stage_weights<D>(S.Wr, (const bf16*)nx.W1rp, tid);
  const AOff<D> AW(i, q);
  __syncthreads();
  const Rows rw{N, (N + 15) >> 4, i, q};
  const UnitRange ur = unit_range(rw.nu, wv);
  if (ur.t >= ur.end) return;
  struct In {
    f32x4 h[8];
  };
  auto load = [&](int64_t u, In& X) { load_row(h + rw.base(u), rw.lo(u), X.h); };
  auto unit = [&](In& X, int64_t u) {
    const EmitLds& L = fresh(S);
    bf16x8 x[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) x[s] = pack_run(X.h[2 * s], X.h[2 * s + 1]);
    const bool ok = rw.valid(u);
    bf16* out = P + u * 16 * D2;
    const int lo = i * D2 + 8 * q;
#pragma unroll
    for (int part = 0; part < 2; ++part) {
      const bf16* W = part == 0 ? L.Ws : L.Wr;
      f32x4 acc[8];
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) {
          acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AW.a(W, ob, s), x[s], acc[ob], 0, 0, 0);
        }
      bf16x8 o[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) o[s] = pack_run(acc[2 * s], acc[2 * s + 1]);
      if (ok) store_runs(out + part * D, lo, o);
    }
  };
  In A, B;
  int64_t u = ur.t;
  load(u, A);
  for (;;) {
    load(u + ur.stride, B);
    unit(A, u);
    u += ur.stride;
    if (u >= ur.end) break;
    load(u + ur.stride, A);
    unit(B, u);
    u += ur.stride;
    if (u >= ur.end) break;
  }
}

// ===================================================================== reverse
// Given hbar_in = dL/dh_out for h_out = h + LN(MLP([h, agg])): recomputes
// the MLP, writes a1 = relu(z1), dz2 = dL/dz2 and dz1 = dL/dz1 (bf16
// streams for k_wgrad_node), hbar_part = hbar_in + dL/dh through the MLP,
// aggbar = dL/dagg, and per-block partials of dgamma (at 49408) and dbeta
// (at 49536).  hbar_part may alias hbar_in.
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_node_bwd_rows(int64_t N, const float* __restrict__ h, const float* __restrict__ agg, const float* hbar_in,
                MlpW w, float eps, float* hbar_part, float* __restrict__ aggbar, bf16* __restrict__ a1_out,
                bf16* __restrict__ dz2_out, bf16* __restrict__ dz1_out, Partials part) {
  __shared__ NodeLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_node_mlp(S, w, tid, false);
  const AOff<D2> A1(i, q);
  const AOff<D> A2(i, q);
  __syncthreads();
  const Rows rw{N, (N + 15) >> 4, i, q};
  const UnitRange ur = unit_range(rw.nu, wv);
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  struct In {
    f32x4 h[8], a[8];
  };
  auto load = [&](int64_t u, In& X) {
    const int64_t b = rw.base(u);
    const int lo = rw.lo(u);
    load_row(h + b, lo, X.h);
    load_row(agg + b, lo, X.a);
  };
  // hbar_in of unit u is issued before the next unit's inputs (so waiting
  // for it never waits for them) and used after the two recomputed products.
  auto unit = [&](In& X, In& Xn, int64_t u, int64_t un) {
    const NodeLds& L = fresh(S);
    bf16x8 x[8];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      x[s] = pack_run(X.h[2 * s], X.h[2 * s + 1]);
      x[4 + s] = pack_run(X.a[2 * s], X.a[2 * s + 1]);
    }
    f32x4 hb[8];
    load_row(hbar_in + rw.base(u), rw.lo(u), hb);
    load(un, Xn);
    const bool ok = rw.valid(u);
    const int64_t b = u * 16 * D;
    const int lo = i * D + 8 * q;
    // ---- z1, a1 = relu(z1), the mask z1 > 0
    f32x4 acc[8];
    node_gemm1(L, A1, x, q, acc);
    uint32_t mask = 0;
    bf16x8 a1[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        mask |= (acc[2 * s][r] > 0.f ? 1u : 0u) << (8 * s + r);
        mask |= (acc[2 * s + 1][r] > 0.f ? 1u : 0u) << (8 * s + 4 + r);
        a1[s][r] = (bf16)relu(acc[2 * s][r]);
        a1[s][4 + r] = (bf16)relu(acc[2 * s + 1][r]);
      }
    if (ok) store_runs(a1_out + b, lo, a1);
    // ---- z2 and its LayerNorm
    node_gemm2(L, A2, a1, q, acc);
    const float rstd = ln_normalize(acc, eps);  // acc = xhat
    // ---- dgamma += sum_rows hbar_in * xhat, dbeta += sum_rows hbar_in
    {
      f32x4 p[8];
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) p[ob] = ok ? hb[ob] * acc[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      const float2 c = colsum16(p, i);
      dga.x += c.x;
      dga.y += c.y;
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) p[ob] = ok ? hb[ob] : f32x4{0.f, 0.f, 0.f, 0.f};
      const float2 d = colsum16(p, i);
      dbe.x += d.x;
      dbe.y += d.y;
    }
    // ---- dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = hbar_in gamma
    bf16x8 dz2[4];
    {
      f32x4 dxh[8];
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) {
        dxh[ob] = hb[ob] * lds4(L.g + fo(ob, q));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          s1 += dxh[ob][r];
          s2 += dxh[ob][r] * acc[ob][r];
        }
      }
      const float m1 = sum_rowlanes(s1) * (1.0f / D), m2 = sum_rowlanes(s2) * (1.0f / D);
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) dxh[ob] = rstd * (dxh[ob] - m1 - acc[ob] * m2);
#pragma unroll
      for (int s = 0; s < 4; ++s) dz2[s] = pack_run(dxh[2 * s], dxh[2 * s + 1]);
    }
    if (ok) store_runs(dz2_out + b, lo, dz2);
    // ---- dz1 = (W2^T dz2) where z1 > 0
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A2.t(L.W2, ob, s), dz2[s], acc[ob], 0, 0, 0);
    bf16x8 dz1[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        dz1[s][r] = (mask >> (8 * s + r)) & 1u ? (bf16)acc[2 * s][r] : (bf16)0.f;
        dz1[s][4 + r] = (mask >> (8 * s + 4 + r)) & 1u ? (bf16)acc[2 * s + 1][r] : (bf16)0.f;
      }
    if (ok) store_runs(dz1_out + b, lo, dz1);
    // ---- [hbar_part, aggbar] = [hbar_in, 0] + W1^T dz1
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        hb[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1.t(L.W1, ob, s), dz1[s], hb[ob], 0, 0, 0);
    if (ok) store_row(hbar_part + b, lo, hb);
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ob = 0; ob < 8; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1.t(L.W1, 8 + ob, s), dz1[s], acc[ob], 0, 0,
                                                          0);
    if (ok) store_row(aggbar + b, lo, acc);
  };
  if (ur.t < ur.end) {
    In A, B;
    int64_t u = ur.t;
    load(u, A);
    for (;;) {
      unit(A, B, u, u + ur.stride);
      u += ur.stride;
      if (u >= ur.end) break;
      unit(B, A, u, u + ur.stride);
      u += ur.stride;
      if (u >= ur.end) break;
    }
  }
  // ---- block partials of dgamma, dbeta: the 8 waves' sums in wave order
  __syncthreads();
  float* red = reinterpret_cast<float*>(S.W1);  // [2][NW][D]
  const int f = fo(i >> 1, q) + 2 * (i & 1);
  *reinterpret_cast<float2*>(red + wv * D + f) = dga;
  *reinterpret_cast<float2*>(red + (NW + wv) * D + f) = dbe;
  __syncthreads();
  if (tid < 2 * D) {
    const int k = tid >> 7, c = tid & (D - 1);
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * D + c];
    part.buf[(size_t)blockIdx.x * part.stride + 49408 + k * D + c] = v;
  }
}

// Weight gradients of the node MLP from the streams of k_node_bwd_rows:
// dW1 = sum_rows dz1^T [h; agg] (h, agg rounded to bf16 as in the forward
// product), db1 = sum dz1, dW2 = sum dz2^T a1, db2 = sum dz2, as per-block
// partials at 0, 32768, 32896 and 49280 (the parameter order of the node
// MLP).  32-row chunks are staged row-major in LDS while the next chunk is
// in flight in registers; wave w owns output rows [16w, 16w + 16).
constexpr int WN_LD = D + 16;
constexpr int WX_LD = D2 + 16;

__global__ void __launch_bounds__(NT) k_wgrad_node(int64_t N, const float* __restrict__ h,
                                                   const float* __restrict__ agg, const bf16* __restrict__ dz1,
                                                   const bf16* __restrict__ dz2, const bf16* __restrict__ a1,
                                                   Partials part) {
  __shared__ __align__(16) bf16 Sz1[2][TM * WN_LD];
  __shared__ __align__(16) bf16 Sz2[2][TM * WN_LD];
  __shared__ __align__(16) bf16 Sa[2][TM * WN_LD];
  __shared__ __align__(16) bf16 Sx[2][TM * WX_LD];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int jp = i >> 2, c4 = i & 3;
  f32x4 acc1[16], acc2[8], ab1 = {0.f, 0.f, 0.f, 0.f}, ab2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cb = 0; cb < 16; ++cb) acc1[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc2[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 ones;
#pragma unroll
  for (int j = 0; j < 8; ++j) ones[j] = (bf16)1.f;
  const int64_t nch = (N + TM - 1) / TM, G = gridDim.x;
  // staging: thread tid moves 8 elements of row srow of every stream
  const int srow = tid >> 4, scol = (tid & 15) * 8;
  struct Ld {
    uint4 z1, z2, a;
    float4 h0, h1, g0, g1;
  } L;
  // rows past N read row N - 1 with zero gradients (so they add nothing);
  // the zeroing is per component (a select of whole vectors goes through
  // scratch memory)
  auto issue = [&](int64_t ch) {
    const int64_t r = ch * TM + srow;
    const bool ok = r < N;
    const int64_t rr = ok ? r : N - 1;
    const uint4 v1 = ld_stream(dz1 + rr * D + scol);
    const uint4 v2 = ld_stream(dz2 + rr * D + scol);
    L.a = ld_stream(a1 + rr * D + scol);
    L.h0 = *reinterpret_cast<const float4*>(h + rr * D + scol);
    L.h1 = *reinterpret_cast<const float4*>(h + rr * D + scol + 4);
    L.g0 = *reinterpret_cast<const float4*>(agg + rr * D + scol);
    L.g1 = *reinterpret_cast<const float4*>(agg + rr * D + scol + 4);
    L.z1.x = ok ? v1.x : 0u;
    L.z1.y = ok ? v1.y : 0u;
    L.z1.z = ok ? v1.z : 0u;
    L.z1.w = ok ? v1.w : 0u;
    L.z2.x = ok ? v2.x : 0u;
    L.z2.y = ok ? v2.y : 0u;
    L.z2.z = ok ? v2.z : 0u;
    L.z2.w = ok ? v2.w : 0u;
  };
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
  // operand of 16 columns col0.. with K = the chunk's rows q*8 + j
  auto frag = [&](const bf16* X, int ld, int col0) -> bf16x8 {
    const bf16* p = X + (q * 8 + jp) * ld + col0 + 4 * c4;
    return cat8(lds_tr(p), lds_tr(p + 4 * ld));
  };
  int64_t c = blockIdx.x;
  int buf = 0;
  if (c < nch) issue(c);
  for (; c < nch; c += G) {
    *reinterpret_cast<uint4*>(&Sz1[buf][srow * WN_LD + scol]) = L.z1;
    *reinterpret_cast<uint4*>(&Sz2[buf][srow * WN_LD + scol]) = L.z2;
    *reinterpret_cast<uint4*>(&Sa[buf][srow * WN_LD + scol]) = L.a;
    *reinterpret_cast<uint4*>(&Sx[buf][srow * WX_LD + scol]) = cvt8(L.h0, L.h1);
    *reinterpret_cast<uint4*>(&Sx[buf][srow * WX_LD + D + scol]) = cvt8(L.g0, L.g1);
    __syncthreads();
    if (c + G < nch) issue(c + G);
    const bf16x8 az1 = frag(Sz1[buf], WN_LD, 16 * w8);
    const bf16x8 az2 = frag(Sz2[buf], WN_LD, 16 * w8);
#pragma unroll
    for (int cb = 0; cb < 16; ++cb)
      acc1[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az1, frag(Sx[buf], WX_LD, 16 * cb), acc1[cb], 0, 0, 0);
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
      acc2[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, frag(Sa[buf], WN_LD, 16 * cb), acc2[cb], 0, 0, 0);
    ab1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az1, ones, ab1, 0, 0, 0);
    ab2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, ones, ab2, 0, 0, 0);
    buf ^= 1;
  }
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int o = w8 * 16 + q * 4 + r;
#pragma unroll
    for (int cb = 0; cb < 16; ++cb) base[(size_t)o * D2 + cb * 16 + i] = acc1[cb][r];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) base[32896 + (size_t)o * D + cb * 16 + i] = acc2[cb][r];
  }
  if (i == 0)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      base[32768 + w8 * 16 + q * 4 + r] = ab1[r];
      base[49280 + w8 * 16 + q * 4 + r] = ab2[r];
    }
}

}  // namespace dev

using namespace dev;

static constexpr int kNodeBlocks = 256;

static int node_grid(int64_t N, int max_blocks) {
  const int64_t units = (N + 15) >> 4;
  const int64_t need = (units + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, max_blocks);
  if (g >= 8) g &= ~7;
  return g;
}

hipError_t launch_node_fwd_rows(int64_t N, const float* h_in, const float* agg, const MlpW& w, float eps,
                                float* h_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_node_fwd_rows, dim3(node_grid(N, kNodeBlocks)), dim3(NT), 0, s, N, h_in, agg, w, eps, h_out);
  return hipGetLastError();
}

hipError_t launch_emit_rows(int64_t N, const float* h, const MlpW& next_edge, void* P, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_emit_rows, dim3(node_grid(N, kNodeBlocks)), dim3(NT), 0, s, N, h, next_edge, (bf16*)P);
  return hipGetLastError();
}

hipError_t launch_node_bwd_rows(int64_t N, const float* h, const float* agg, const float* hbar_in, const MlpW& w,
                                float eps, float* hbar_part, float* aggbar, void* a1, void* dz2, void* dz1,
                                const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  const int g = node_grid(N, std::min(kNodeBlocks, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_node_bwd_rows, dim3(g), dim3(NT), 0, s, N, h, agg, hbar_in, w, eps, hbar_part, aggbar,
                     (bf16*)a1, (bf16*)dz2, (bf16*)dz1, part);
  return hipGetLastError();
}

static constexpr int kWgradNodeBlocks = 256;

hipError_t launch_wgrad_node(int64_t N, const float* h, const float* agg, const void* dz1, const void* dz2,
                             const void* a1, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  const int g = part_grid((N + TM - 1) / TM, std::min(kWgradNodeBlocks, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_wgrad_node, dim3(g), dim3(NT), 0, s, N, h, agg, (const bf16*)dz1, (const bf16*)dz2,
                     (const bf16*)a1, part);
  return hipGetLastError();
}

}  // namespace mgn
