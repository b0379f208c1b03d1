// Edge and node encoders of the MGN (Sec. 2.1: every edge's and node's input
// features are mapped to the latent by an MLP with LayerNorm) at the latent
// width 150 computed
// 160 wide (App. C: the 3D model; padded features are exactly zero), bf16
// operands, in the lane layout of w160_common.hpp.
//
//   k_edge_enc_w160      e = LN(W2 relu(W1 f + b1) + b2) over the 150 real
//                        features, one wave per 16-edge unit, no block
//                        barrier in the loop
//   k_edge_enc_bwd_w160  all encoder parameter gradients from dL/de in one
//                        pass: block rounds of 8 units (one per wave); each
//                        wave takes its unit back to dz2 and dz1, then in two
//                        sub-rounds of 4 units the units' bf16 dz2, dz1, a1
//                        and inputs are staged in LDS and every wave adds its
//                        15 of the 120 output tiles over the staged rows
//                        (K = rows)
//
//   k_node_enc_bwd_w160  the node encoder's reverse (8 inputs) in the same
//                        rounds, with dL/d(node input) = W1^T dz1 per unit
//
// The first layer (K = 4) runs on VALU in fp32 as one fma chain per
// feature, k = 0..3 from b1, identical in both edge-encoder kernels, as is
// the second product (W2 staged in the rotated layout in both), so the
// backward recomputes the forward's values bitwise.
#include "w160_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

namespace w160 {
constexpr int KE = 4;      // edge input features
constexpr int ESL = WG_LD;  // LDS row stride of the staged [rows][160] bf16 tiles
constexpr int SUB = 64;    // rows staged per sub-round (4 units)
constexpr int PCOL = 160;  // a1 tile columns 160..175: the input pieces

struct __attribute__((aligned(16))) EncLds {
  __attribute__((aligned(16))) bf16 W2[L * L];  // row-permuted W2, rotated chunks
  __attribute__((aligned(16))) float4 W1[L];    // W1 rows by feature
  __attribute__((aligned(16))) float b1[L];
  __attribute__((aligned(16))) float b2[L];
  __attribute__((aligned(16))) float g[L];
  __attribute__((aligned(16))) float bt[L];
};

__device__ __forceinline__ void stage_enc(EncLds& S, const MlpW& w, int tid) {
  stage_rot(S.W2, (const bf16*)w.W2p, tid);
  if (tid < L) {
    S.W1[tid] = float4{w.W1f[tid * KE], w.W1f[tid * KE + 1], w.W1f[tid * KE + 2], w.W1f[tid * KE + 3]};
    S.b1[tid] = w.b1[tid];
    S.b2[tid] = w.b2[tid];
    S.g[tid] = w.gamma[tid];
    S.bt[tid] = w.beta[tid];
  }
}

// z1 = b1 + W1 f for the lane's 40 features (fo(ob, q) + r).
__device__ __forceinline__ void enc_z1(const EncLds& S, float4 f, int q, f32x4 (&z)[NOB]) {
  const float4* W1q = S.W1 + 8 * q;
  const float* b1q = S.b1 + 8 * q;
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float4 wr = W1q[fo0(ob) + r];
      float v = b1q[fo0(ob) + r];
      v = __builtin_fmaf(wr.x, f.x, v);
      v = __builtin_fmaf(wr.y, f.y, v);
      v = __builtin_fmaf(wr.z, f.z, v);
      v = __builtin_fmaf(wr.w, f.w, v);
      z[ob][r] = v;
    }
}

// a1 = relu(z1) as bf16 runs, then z2 = b2 + W2 a1 (W2s: the staged W2).
__device__ __forceinline__ void enc_z2(const EncLds& S, const bf16* W2s, const RotOff& RO, const f32x4 (&z1)[NOB],
                                       int q, bf16x8 (&a1)[NS], f32x4 (&acc)[NOB]) {
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      a1[s][r] = (bf16)relu(z1[2 * s][r]);
      a1[s][4 + r] = (bf16)relu(z1[2 * s + 1][r]);
    }
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + 8 * q + fo0(ob));
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W2s, ob, s), a1[s], acc[ob], 0, 0, 0);
}

// LayerNorm statistics of the row over the 150 real features (padded
// features of z2 are exactly 0, so the plain sum is the real one); acc
// becomes xhat on the real features.  Returns rstd.
__device__ __forceinline__ float ln_xhat(f32x4 (&acc)[NOB], const int (&lv)[2], float eps) {
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

// ===================================================================== forward
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_enc_w160(int64_t E, const float* __restrict__ f_in, MlpW w, float eps, bf16* __restrict__ e_out) {
  using namespace w160;
  __shared__ __align__(16) EncLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_enc(S, w, tid);
  const RotOff RO(i, q);
  const int lv[2] = {live_bits(8, q), live_bits(9, q)};
  __syncthreads();
  const int64_t nu = (E + 15) >> 4;
  const UnitRange ur = unit_range(nu, wv);
  if (ur.t >= ur.end) return;
  // rows clamped into [0, E): rows past E and prefetches past the wave's
  // last unit read row E - 1 and store nothing
  auto load = [&](int64_t u) { return *reinterpret_cast<const float4*>(f_in + min(u * 16 + i, E - 1) * KE); };
  float4 fa = load(ur.t);
  for (int64_t u = ur.t; u < ur.end; u += ur.stride) {
    const float4 fn = load(u + ur.stride);
    // staged W2 at an opaque offset: its fragments are not hoisted out of the loop
    const bf16* W2s = S.W2 + opaque_zero();
    f32x4 z[NOB], acc[NOB];
    enc_z1(S, fa, q, z);
    bf16x8 a1[NS];
    enc_z2(S, W2s, RO, z, q, a1, acc);
    ln_xhat(acc, lv, eps);
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      acc[ob] = *reinterpret_cast<const f32x4*>(S.g + 8 * q + fo0(ob)) * acc[ob] +
                *reinterpret_cast<const f32x4*>(S.bt + 8 * q + fo0(ob));
    if (u * 16 + i < E) {
      bf16* op = e_out + (u * 16 + i) * L + 8 * q;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(acc[2 * s], acc[2 * s + 1]));
    }
    fa = fn;
  }
}

// ===================================================================== reverse
// Per-block partials in the parameter order of the encoder at width 160:
// dW1 [160][4] at 0, db1 at 640, dW2 [160][160] at 800, db2 at 26400, dgamma
// at 26560, dbeta at 26720.  Output tiles (16 x 16, K = the staged rows):
// row block rb, kind c: c < 10: dW2 columns 16c.. (dz2^T a1); c = 10: dz2^T
// against the input pieces, whose column 8 (all ones) gives db2; c = 11: dz1^T
// against the input pieces: dW1 (columns f_hi 0..3 plus f_lo 4..7; f = f_hi +
// f_lo, both bf16: the input features keep 16 significant bits) and db1
// (column 8).  Wave w owns row block w (kinds 0..11) and kinds 3 (w % 4) ..
// + 2 of row block 8 + w / 4.
namespace w160 {
struct __attribute__((aligned(16))) EncBwdLds {
  EncLds P;
  __attribute__((aligned(16))) bf16 z2[SUB * ESL];
  __attribute__((aligned(16))) bf16 z1[SUB * ESL];
  __attribute__((aligned(16))) bf16 a1[SUB * ESL];
};
}  // namespace w160

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_enc_bwd_w160(int64_t E, const float* __restrict__ f_in, const bf16* __restrict__ ebar, MlpW w, float eps,
                    Partials part) {
  using namespace w160;
  __shared__ __align__(16) EncBwdLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_enc(S.P, w, tid);
  const int lv[2] = {live_bits(8, q), live_bits(9, q)};
  const int jp = i >> 2, c4 = i & 3;
  __syncthreads();
  const int64_t nu = (E + 15) >> 4;
  const int64_t nrounds = (nu + NW - 1) / NW;
  const int G = gridDim.x;
  // shared row block and its first kind
  const int rx = 8 + (wv >> 2), cx0 = 3 * (wv & 3);
  f32x4 acc_t[15];
#pragma unroll
  for (int k = 0; k < 15; ++k) acc_t[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  // column sums: main part (lane i: features fo(i/2, q) + 2 (i%2) + {0, 1})
  // and tail (lane i: feature tail_feature(i, q))
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  float tga = 0.f, tbe = 0.f;
  struct In {
    float4 f;
    uint4 eb[NS];
  };
  // unit u = round * 8 + wave; rows clamped into [0, E)
  auto load = [&](int64_t R, In& X) {
    const int64_t row = min((R * NW + wv) * 16 + i, E - 1);
    X.f = *reinterpret_cast<const float4*>(f_in + row * KE);
    const bf16* ep = ebar + row * L + 8 * q;
#pragma unroll
    for (int k = 0; k < NS; ++k) X.eb[k] = *reinterpret_cast<const uint4*>(ep + 32 * k);
  };
  // operand of 16 columns col0.. with K = staged rows r0 + q*8 + j; lb: the
  // lane's part of the address, rebuilt per sub-round from an opaque zero so
  // that the per-operand addresses are not hoisted out of the loop
  const int lb0 = (q * 8 + jp) * ESL + 4 * c4;
  auto frag = [&](const bf16* X, int lb, int r0, int col0) -> bf16x8 {
    const bf16* p = X + lb + r0 * ESL + col0;
    return cat8(lds_tr(p), lds_tr(p + 4 * ESL));
  };
  In X;
  int64_t R = blockIdx.x;
  if (R < nrounds) load(R, X);
  for (; R < nrounds; R += G) {
    const bool ok = (R * NW + wv) * 16 + i < E;
    // input pieces: q = 0: f_hi, 1: f_lo, 2: [1, 0, 0, 0], 3: zeros
    uint2 piece;
    {
      const float fv[4] = {X.f.x, X.f.y, X.f.z, X.f.w};
      uint32_t hb[4], lb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bf16 hi = (bf16)fv[k];
        const bf16 lo = (bf16)(fv[k] - (float)hi);
        hb[k] = __builtin_bit_cast(uint16_t, hi);
        lb[k] = __builtin_bit_cast(uint16_t, lo);
      }
      const uint32_t one = 0x3F80u;  // bf16 1.0
      const uint32_t h0 = hb[0] | (hb[1] << 16), h1 = hb[2] | (hb[3] << 16);
      const uint32_t l0 = lb[0] | (lb[1] << 16), l1 = lb[2] | (lb[3] << 16);
      piece.x = q == 0 ? h0 : (q == 1 ? l0 : (q == 2 ? one : 0u));
      piece.y = q == 0 ? h1 : (q == 1 ? l1 : 0u);
    }
    bf16x8 a1[NS], dz2[NS], dz1[NS];
    {
      // the per-lane fragment offsets are rebuilt where they are used (from
      // an opaque zero), so they are not live across the unit
      const bf16* W2s = S.P.W2 + opaque_zero();
      f32x4 acc[NOB];
      // mask bits of z1 > 0: bit 4 ob + r of mlo (ob < 8) / mhi (ob >= 8)
      uint32_t mlo = 0, mhi = 0;
      {
        f32x4 z[NOB];
        enc_z1(S.P, X.f, q, z);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const uint32_t b = z[ob][r] > 0.f ? 1u : 0u;
            if (ob < 8)
              mlo |= b << (4 * ob + r);
            else
              mhi |= b << (4 * (ob - 8) + r);
          }
        enc_z2(S.P, W2s, RotOff(i + opaque_zero(), q), z, q, a1, acc);
      }
      const float rstd = ln_xhat(acc, lv, eps);  // acc = xhat
      // ybar (the bf16 edge-gradient runs; zero on rows past E) is unpacked
      // where it is used
      if (!ok) {
#pragma unroll
        for (int k = 0; k < NS; ++k) X.eb[k] = uint4{0u, 0u, 0u, 0u};
      }
      auto yb = [&](int ob) { return run_block5(X.eb, ob); };
      // dbeta += sum_rows ybar
      {
        f32x4 v[NOB];
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) v[ob] = yb(ob);
        const float2 d = colsum16(reinterpret_cast<const f32x4(&)[8]>(v), i);
        dbe.x += d.x;
        dbe.y += d.y;
        tbe += colsum16_tail(v, i);
      }
      // dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = ybar gamma,
      // 0 on padded features
      {
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          const f32x4 dxh = yb(ob) * *reinterpret_cast<const f32x4*>(S.P.g + 8 * q + fo0(ob));
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
          for (int h = 0; h < 2; ++h) {
            const int ob = 2 * s + h;
            const f32x4 dxh = yb(ob) * *reinterpret_cast<const f32x4*>(S.P.g + 8 * q + fo0(ob));
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = ob < 8 || ((lv[ob - 8] >> r) & 1);
              v[h][r] = live ? rstd * (dxh[r] - m1 - acc[ob][r] * m2) : 0.f;
            }
          }
          dz2[s] = pack_run(v[0], v[1]);
        }
      }
      // dgamma += sum_rows ybar xhat (in place: xhat is not used again)
      {
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) acc[ob] *= yb(ob);
        const float2 c = colsum16(reinterpret_cast<const f32x4(&)[8]>(acc), i);
        dga.x += c.x;
        dga.y += c.y;
        tga += colsum16_tail(acc, i);
      }
      // dz1 = (W2^T dz2) where z1 > 0
      const RotOff RO(i + opaque_zero(), q);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.t_frag(W2s, ob, s), dz2[s], acc[ob], 0, 0, 0);
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ob = 2 * s + h;
            const bool on = ob < 8 ? (mlo >> (4 * ob + r)) & 1u : (mhi >> (4 * (ob - 8) + r)) & 1u;
            dz1[s][4 * h + r] = on ? (bf16)acc[ob][r] : (bf16)0.f;
          }
    }
    // two sub-rounds: waves 4h .. 4h + 3 stage their units (rows past E have
    // dz2 = dz1 = 0), then every wave adds its tiles over the 64 staged rows
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if ((wv >> 2) == h) {
        const int srow = 16 * (wv & 3) + i;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          *reinterpret_cast<uint4*>(S.z2 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz2[s]);
          *reinterpret_cast<uint4*>(S.z1 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz1[s]);
          *reinterpret_cast<uint4*>(S.a1 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, a1[s]);
        }
        *reinterpret_cast<uint2*>(S.a1 + srow * ESL + PCOL + 4 * q) = piece;
      }
      __syncthreads();
      // the next round's inputs are in flight while the last tiles are added
      if (h == 1) load(R + G, X);
      const int lb = lb0 + opaque_zero();
#pragma unroll
      for (int kk = 0; kk < SUB / 32; ++kk) {
        const int r0 = 32 * kk;
        const bf16x8 az2 = frag(S.z2, lb, r0, 16 * wv), az1 = frag(S.z1, lb, r0, 16 * wv);
        const bf16x8 bp = frag(S.a1, lb, r0, PCOL);
#pragma unroll
        for (int c = 0; c < NOB; ++c)
          acc_t[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, frag(S.a1, lb, r0, 16 * c), acc_t[c], 0, 0, 0);
        acc_t[10] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, bp, acc_t[10], 0, 0, 0);
        acc_t[11] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az1, bp, acc_t[11], 0, 0, 0);
        const bf16x8 ax2 = frag(S.z2, lb, r0, 16 * rx), ax1 = frag(S.z1, lb, r0, 16 * rx);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          const int c = cx0 + k;
          const bf16x8 b = frag(S.a1, lb, r0, c < NOB ? 16 * c : PCOL);
          acc_t[12 + k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c == 11 ? ax1 : ax2, b, acc_t[12 + k], 0, 0, 0);
        }
      }
      __syncthreads();
    }
  }
  // ---- partials
  constexpr int oW1 = 0, oB1 = KE * L, oW2 = oB1 + L, oB2 = oW2 + L * L, oG = oB2 + L, oBt = oG + L;
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  auto put = [&](const f32x4& a, int rb, int c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = 16 * rb + 4 * q + r;
      if (c < NOB) {
        base[oW2 + o * L + 16 * c + i] = a[r];
      } else if (c == NOB) {
        if (i == 8) base[oB2 + o] = a[r];
      } else {
        // column i < 4: sum dz1 f_hi[i], 4 + i: the f_lo part, 8: the sum of dz1
        const float lo = __shfl_down(a[r], 4, 16);
        if (i < 4) base[oW1 + o * KE + i] = a[r] + lo;
        if (i == 8) base[oB1 + o] = a[r];
      }
    }
  };
#pragma unroll
  for (int c = 0; c < 12; ++c) put(acc_t[c], wv, c);
#pragma unroll
  for (int k = 0; k < 3; ++k) put(acc_t[12 + k], rx, cx0 + k);
  // dgamma, dbeta: the 8 waves' column sums in wave order
  float* red = reinterpret_cast<float*>(S.z2);  // [2][NW][L] fp32
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
  for (int idx = tid; idx < 2 * L; idx += NT) {
    const int k = idx / L, f = idx % L;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * L + f];
    base[oG + idx] = v;
  }
}


// Node encoder, reverse (8 inputs: z1 = b1 + W1 x as one fma chain per
// feature, k = 0..7).  Per-block partials in the parameter order of the
// encoder at width 160: dW1 [160][8] at 0, db1 at 1280, dW2 at 1440, db2 at
// 27040, dgamma at 27200, dbeta at 27360.  Output tiles (K = the staged
// rows): row block rb, kind c < 10: dW2 columns 16c.. (dz2^T a1); c = 10:
// dz1^T against the input pieces [x_hi (8), x_lo (8)] (x = x_hi + x_lo, both
// bf16).  Wave w owns row block w (11 kinds) and kinds 3 (w % 4) .. + 2 (up
// to 10) of row block 8 + w / 4.  db1, db2, dgamma, dbeta are column sums
// (DPP butterflies) per unit; gin = W1^T dz1 (when gin is not null) is one
// product per unit with the bf16 W1^T staged as a [16][160] A operand (rows
// 8..15 zero).  The incoming gradient dL/dh is rounded to bf16 like the
// other MLP operands.
namespace w160 {
struct __attribute__((aligned(16))) NodeEncLds {
  __attribute__((aligned(16))) bf16 W2[L * L];  // row-permuted W2, rotated chunks
  __attribute__((aligned(16))) float4 W1[2][L];  // W1 rows by feature: inputs 0..3, 4..7
  __attribute__((aligned(16))) float b1[L];
  __attribute__((aligned(16))) float b2[L];
  __attribute__((aligned(16))) float g[L];
  __attribute__((aligned(16))) bf16 W1t[16 * L];  // W1^T, rows 8..15 zero
  __attribute__((aligned(16))) bf16 z2[SUB * ESL];
  __attribute__((aligned(16))) bf16 z1[SUB * ESL];
  __attribute__((aligned(16))) bf16 a1[SUB * ESL];
};
}  // namespace w160

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_node_enc_bwd_w160(int64_t N, const float* __restrict__ x_in, const float* __restrict__ hbar, MlpW w, float eps,
                    float* __restrict__ gin, Partials part) {
  using namespace w160;
  constexpr int KN = 8;
  __shared__ __align__(16) NodeEncLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_rot(S.W2, (const bf16*)w.W2p, tid);
  if (tid < L) {
    const float* wr = w.W1f + tid * KN;
    S.W1[0][tid] = float4{wr[0], wr[1], wr[2], wr[3]};
    S.W1[1][tid] = float4{wr[4], wr[5], wr[6], wr[7]};
    S.b1[tid] = w.b1[tid];
    S.b2[tid] = w.b2[tid];
    S.g[tid] = w.gamma[tid];
  }
  for (int idx = tid; idx < 16 * L; idx += NT) {
    const int k = idx / L, f = idx % L;
    S.W1t[idx] = k < KN ? (bf16)w.W1f[f * KN + k] : (bf16)0.f;
  }
  const int lv[2] = {live_bits(8, q), live_bits(9, q)};
  const int jp = i >> 2, c4 = i & 3;
  __syncthreads();
  const int64_t nu = (N + 15) >> 4;
  const int64_t nrounds = (nu + NW - 1) / NW;
  const int G = gridDim.x;
  const int rx = 8 + (wv >> 2), cx0 = 3 * (wv & 3);
  constexpr int NT_ = 14;  // tiles per wave
  f32x4 acc_t[NT_];
#pragma unroll
  for (int k = 0; k < NT_; ++k) acc_t[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  // column sums (main part: lane i features fo(i/2, q) + 2 (i%2) + {0, 1};
  // tail: feature tail_feature(i, q)) of dgamma, dbeta, db1, db2
  float2 cs[4] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
  float ct[4] = {0.f, 0.f, 0.f, 0.f};
  auto colsums = [&](const f32x4 (&v)[NOB], int k) {
    const float2 c = colsum16(reinterpret_cast<const f32x4(&)[8]>(v), i);
    cs[k].x += c.x;
    cs[k].y += c.y;
    ct[k] += colsum16_tail(v, i);
  };
  // the inputs of the round's unit are prefetched one round ahead; its
  // incoming gradient is loaded when the unit starts (first used after the
  // recomputed forward)
  struct In {
    float4 x0, x1;
  };
  // unit u = round * 8 + wave; rows clamped into [0, N)
  auto clamp_row = [&](int64_t R) { return min((R * NW + wv) * 16 + i, N - 1); };
  auto load = [&](int64_t R, In& X) {
    const int64_t row = clamp_row(R);
    X.x0 = *reinterpret_cast<const float4*>(x_in + row * KN);
    X.x1 = *reinterpret_cast<const float4*>(x_in + row * KN + 4);
  };
  const int lb0 = (q * 8 + jp) * ESL + 4 * c4;
  auto frag = [&](const bf16* X, int lb, int r0, int col0) -> bf16x8 {
    const bf16* p = X + lb + r0 * ESL + col0;
    return cat8(lds_tr(p), lds_tr(p + 4 * ESL));
  };
  In X;
  int64_t R = blockIdx.x;
  if (R < nrounds) load(R, X);
  for (; R < nrounds; R += G) {
    const int64_t row = (R * NW + wv) * 16 + i;
    const bool ok = row < N;
    // input pieces: q = 0: x_hi 0..3, 1: x_hi 4..7, 2: x_lo 0..3, 3: x_lo 4..7
    uint2 piece;
    {
      const float xv[4] = {q & 1 ? X.x1.x : X.x0.x, q & 1 ? X.x1.y : X.x0.y, q & 1 ? X.x1.z : X.x0.z,
                           q & 1 ? X.x1.w : X.x0.w};
      uint32_t pb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bf16 hi = (bf16)xv[k];
        const bf16 lo = (bf16)(xv[k] - (float)hi);
        pb[k] = __builtin_bit_cast(uint16_t, q < 2 ? hi : lo);
      }
      piece.x = pb[0] | (pb[1] << 16);
      piece.y = pb[2] | (pb[3] << 16);
    }
    f32x4 ybf[NOB];
    {
      const float* yp = hbar + clamp_row(R) * L + 8 * q;
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) ybf[ob] = *reinterpret_cast<const f32x4*>(yp + fo0(ob));
    }
    // ybar as bf16 runs (rows past N: zero), unpacked where it is used
    uint4 ybr[NS];
    auto yb = [&](int ob) { return run_block5(ybr, ob); };
    bf16x8 a1[NS], dz2[NS], dz1[NS];
    {
      const bf16* W2s = S.W2 + opaque_zero();
      f32x4 acc[NOB];
      uint32_t mlo = 0, mhi = 0;
      {
        f32x4 z[NOB];
        const float4* W0 = S.W1[0] + 8 * q;
        const float4* W1q = S.W1[1] + 8 * q;
        const float* b1q = S.b1 + 8 * q;
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float4 wa = W0[fo0(ob) + r], wb = W1q[fo0(ob) + r];
            float v = b1q[fo0(ob) + r];
            v = __builtin_fmaf(wa.x, X.x0.x, v);
            v = __builtin_fmaf(wa.y, X.x0.y, v);
            v = __builtin_fmaf(wa.z, X.x0.z, v);
            v = __builtin_fmaf(wa.w, X.x0.w, v);
            v = __builtin_fmaf(wb.x, X.x1.x, v);
            v = __builtin_fmaf(wb.y, X.x1.y, v);
            v = __builtin_fmaf(wb.z, X.x1.z, v);
            v = __builtin_fmaf(wb.w, X.x1.w, v);
            z[ob][r] = v;
            const uint32_t b = v > 0.f ? 1u : 0u;
            if (ob < 8)
              mlo |= b << (4 * ob + r);
            else
              mhi |= b << (4 * (ob - 8) + r);
            if (r == 3) __builtin_amdgcn_sched_barrier(0);
          }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            a1[s][r] = (bf16)relu(z[2 * s][r]);
            a1[s][4 + r] = (bf16)relu(z[2 * s + 1][r]);
          }
        const RotOff RO(i + opaque_zero(), q);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + 8 * q + fo0(ob));
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
          for (int ob = 0; ob < NOB; ++ob)
            acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.a_frag(W2s, ob, s), a1[s], acc[ob], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      const float rstd = ln_xhat(acc, lv, eps);  // acc = xhat
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        ybr[s] = __builtin_bit_cast(uint4, pack_run(ybf[2 * s], ybf[2 * s + 1]));
        if (!ok) ybr[s] = uint4{0u, 0u, 0u, 0u};
      }
      {
        f32x4 v[NOB];
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) v[ob] = yb(ob);
        colsums(v, 1);  // dbeta
      }
      // dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = ybar gamma,
      // 0 on padded features
      {
        const float* gq = S.g + 8 * q;
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          const f32x4 dxh = yb(ob) * *reinterpret_cast<const f32x4*>(gq + fo0(ob));
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
            const f32x4 dxh = yb(ob) * *reinterpret_cast<const f32x4*>(gq + fo0(ob));
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool live = ob < 8 || ((lv[ob - 8] >> r) & 1);
              v[hh][r] = live ? rstd * (dxh[r] - m1 - acc[ob][r] * m2) : 0.f;
            }
          }
          dz2[s] = pack_run(v[0], v[1]);
        }
      }
      // dgamma += sum_rows ybar xhat (in place)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] *= yb(ob);
      colsums(acc, 0);
      // db2 += sum_rows dz2 (as stored)
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          acc[2 * s][r] = (float)dz2[s][r];
          acc[2 * s + 1][r] = (float)dz2[s][4 + r];
        }
      colsums(acc, 3);
      // dz1 = (W2^T dz2) where z1 > 0
      const RotOff RO(i + opaque_zero(), q);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(RO.t_frag(W2s, ob, s), dz2[s], acc[ob], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
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
      // db1 += sum_rows dz1 (as stored)
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          acc[2 * s][r] = (float)dz1[s][r];
          acc[2 * s + 1][r] = (float)dz1[s][4 + r];
        }
      colsums(acc, 2);
      // gin = W1^T dz1: C[k][row], lane (i, q < 2) holds inputs 4q .. 4q + 3 of row i
      {
        const bf16* Wt = S.W1t + opaque_zero() + i * L + 8 * q;
        f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s)
          gacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*reinterpret_cast<const bf16x8*>(Wt + 32 * s), dz1[s], gacc,
                                                         0, 0, 0);
        if (gin != nullptr && ok && q < 2) *reinterpret_cast<f32x4*>(gin + row * KN + 4 * q) = gacc;
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if ((wv >> 2) == h) {
        const int srow = 16 * (wv & 3) + i;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          *reinterpret_cast<uint4*>(S.z2 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz2[s]);
          *reinterpret_cast<uint4*>(S.z1 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz1[s]);
          *reinterpret_cast<uint4*>(S.a1 + srow * ESL + 32 * s + 8 * q) = __builtin_bit_cast(uint4, a1[s]);
        }
        *reinterpret_cast<uint2*>(S.a1 + srow * ESL + PCOL + 4 * q) = piece;
      }
      __syncthreads();
      if (h == 1) load(R + G, X);
      const int lb = lb0 + opaque_zero();
#pragma unroll
      for (int kk = 0; kk < SUB / 32; ++kk) {
        const int r0 = 32 * kk;
        const bf16x8 az2 = frag(S.z2, lb, r0, 16 * wv), az1 = frag(S.z1, lb, r0, 16 * wv);
#pragma unroll
        for (int c = 0; c < NOB; ++c)
          acc_t[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, frag(S.a1, lb, r0, 16 * c), acc_t[c], 0, 0, 0);
        acc_t[10] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az1, frag(S.a1, lb, r0, PCOL), acc_t[10], 0, 0, 0);
        const bf16x8 ax2 = frag(S.z2, lb, r0, 16 * rx), ax1 = frag(S.z1, lb, r0, 16 * rx);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          const int c = cx0 + k;
          if (c <= NOB) {
            const bf16x8 b = frag(S.a1, lb, r0, c < NOB ? 16 * c : PCOL);
            acc_t[11 + k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(c == NOB ? ax1 : ax2, b, acc_t[11 + k], 0, 0, 0);
          }
        }
      }
      __syncthreads();
    }
  }
  // ---- partials
  constexpr int oW1 = 0, oB1 = KN * L, oW2 = oB1 + L, oB2 = oW2 + L * L, oG = oB2 + L;
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
  auto put = [&](const f32x4& a, int rb, int c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int o = 16 * rb + 4 * q + r;
      if (c < NOB) {
        base[oW2 + o * L + 16 * c + i] = a[r];
      } else {
        // column i < 8: sum dz1 x_hi[i], 8 + i: the x_lo part
        const float lo = __shfl_down(a[r], 8, 16);
        if (i < KN) base[oW1 + o * KN + i] = a[r] + lo;
      }
    }
  };
#pragma unroll
  for (int c = 0; c <= NOB; ++c) put(acc_t[c], wv, c);
#pragma unroll
  for (int k = 0; k < 3; ++k)
    if (cx0 + k <= NOB) put(acc_t[11 + k], rx, cx0 + k);
  // dgamma, dbeta, db1, db2: the 8 waves' column sums in wave order
  float* red = reinterpret_cast<float*>(S.z2);  // [4][NW][L] fp32
  {
    const int fm = fo(i >> 1, q) + 2 * (i & 1), ft = tail_feature(i, q);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float* rk = red + (k * NW + wv) * L;
      *reinterpret_cast<float2*>(rk + fm) = cs[k];
      if ((i & 1) == 0) rk[ft] = ct[k];  // lanes i and i ^ 1 hold the same tail sums
    }
  }
  __syncthreads();
  // red k: 0 dgamma, 1 dbeta, 2 db1, 3 db2
  for (int idx = tid; idx < 4 * L; idx += NT) {
    const int k = idx / L, f = idx % L;
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * L + f];
    const int dst = k == 0 ? oG : (k == 1 ? oG + L : (k == 2 ? oB1 : oB2));
    base[dst + f] = v;
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kEncBlocks160 = 256;

hipError_t launch_edge_enc_w160(int64_t E, const float* efeat, const MlpW& w, float eps, void* e_out, hipStream_t s) {
  if (E <= 0) return hipSuccess;
  if (!w.W2p) return hipErrorInvalidValue;
  const int64_t need = (((E + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kEncBlocks160);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_edge_enc_w160, dim3(g), dim3(NT), 0, s, E, efeat, w, eps, (bf16*)e_out);
  return hipGetLastError();
}

hipError_t launch_edge_enc_bwd_w160(int64_t E, const float* efeat, const void* ebar, const MlpW& w, float eps,
                                    const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (E <= 0) return hipSuccess;
  if (!w.W2p || part.stride < 8 * 160 + 160 * 160) return hipErrorInvalidValue;
  const int64_t nrounds = (((E + 15) >> 4) + NW - 1) / NW;
  const int g = (int)std::min<int64_t>(nrounds, std::min(kEncBlocks160, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_edge_enc_bwd_w160, dim3(g), dim3(NT), 0, s, E, efeat, (const bf16*)ebar, w, eps, part);
  return hipGetLastError();
}

hipError_t launch_node_enc_bwd_w160(int64_t N, const float* node_in, const float* hbar, const MlpW& w, float eps,
                                    float* gin, const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (N <= 0) return hipSuccess;
  if (!w.W2p || part.stride < 12 * 160 + 160 * 160) return hipErrorInvalidValue;
  const int64_t nrounds = (((N + 15) >> 4) + NW - 1) / NW;
  const int g = (int)std::min<int64_t>(nrounds, std::min(kEncBlocks160, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_node_enc_bwd_w160, dim3(g), dim3(NT), 0, s, N, node_in, hbar, w, eps, gin, part);
  return hipGetLastError();
}

}  // namespace mgn
