// Edge encoder of the MGN (Sec. 2.1: every edge's input features are mapped
// to the 128-wide latent by an MLP with LayerNorm), bf16 operands, in the
// lane layout of rows_common.hpp.
//
//   k_edge_enc_rows      e = LN(W2 relu(W1 f + b1) + b2) for 16-edge units,
//                        one wave per unit, no block barrier in the loop
//   k_edge_enc_bwd_rows  all encoder parameter gradients from dL/de in one
//                        pass: block rounds of 8 units (one per wave); the
//                        waves stage the unit's bf16 dz2, a1, dz1 and inputs
//                        in LDS, then each wave accumulates its 16 output
//                        rows of dW2 and dW1 over the round's 128 rows with
//                        K = rows
//
// The first layer (K = 4) runs on VALU in fp32 as one fma chain per
// feature, k = 0..3 from b1, identical in both kernels, as is the second
// product, so the backward recomputes the forward's values bitwise.
#include "rows_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

constexpr int KE = 4;           // edge input features
constexpr int SLD = D + 16;     // LDS row stride of the staged [128][128] bf16 tiles
constexpr int FLD = 24;         // LDS row stride of the staged [128][16] input tile
constexpr int RROWS = NW * 16;  // rows of one round

struct __attribute__((aligned(16))) EncLds {
  __attribute__((aligned(16))) bf16 W2[D * D];
  __attribute__((aligned(16))) float4 W1[D];  // W1 rows by feature
  __attribute__((aligned(16))) float b1[D];
  __attribute__((aligned(16))) float b2[D];
  __attribute__((aligned(16))) float g[D];
  __attribute__((aligned(16))) float bt[D];
};

__device__ __forceinline__ void stage_enc(EncLds& S, const MlpW& w, int tid) {
  stage_weights<D>(S.W2, (const bf16*)w.W2p, tid);
  if (tid < D) {
    S.W1[tid] = float4{w.W1f[tid * KE], w.W1f[tid * KE + 1], w.W1f[tid * KE + 2], w.W1f[tid * KE + 3]};
    S.b1[tid] = w.b1[tid];
    S.b2[tid] = w.b2[tid];
    S.g[tid] = w.gamma[tid];
    S.bt[tid] = w.beta[tid];
  }
}

// Lane-independent part of fo(ob, q) = 8 q + fo_c(ob): LDS reads at a
// per-lane base plus this constant fold the constant into the instruction's
// offset (one base register instead of one address per feature).
__device__ __forceinline__ constexpr int fo_c(int ob) { return 32 * (ob >> 1) + 4 * (ob & 1); }

// z1 = b1 + W1 f for the lane's 32 features (fo(ob, q) + r).
__device__ __forceinline__ void enc_z1(const EncLds& S, float4 f, int q, f32x4 (&z)[8]) {
  const float4* W1q = S.W1 + 8 * q;
  const float* b1q = S.b1 + 8 * q;
#pragma unroll
  for (int ob = 0; ob < 8; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float4 wr = W1q[fo_c(ob) + r];
      float v = b1q[fo_c(ob) + r];
      v = __builtin_fmaf(wr.x, f.x, v);
      v = __builtin_fmaf(wr.y, f.y, v);
      v = __builtin_fmaf(wr.z, f.z, v);
      v = __builtin_fmaf(wr.w, f.w, v);
      z[ob][r] = v;
    }
}

// a1 = relu(z1) as bf16 runs, then z2 = b2 + W2 a1.
__device__ __forceinline__ void enc_z2(const EncLds& S, const AOff<D>& A2, const f32x4 (&z1)[8], int q,
                                       bf16x8 (&a1)[4], f32x4 (&acc)[8]) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      a1[s][r] = (bf16)relu(z1[2 * s][r]);
      a1[s][4 + r] = (bf16)relu(z1[2 * s + 1][r]);
    }
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) acc[ob] = *reinterpret_cast<const f32x4*>(S.b2 + 8 * q + fo_c(ob));
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) acc[ob] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A2.a(S.W2, ob, s), a1[s], acc[ob], 0, 0, 0);
}

// ===================================================================== forward
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_enc_rows(int64_t E, const float* __restrict__ f_in, MlpW w, float eps, bf16* __restrict__ e_out) {
  __shared__ EncLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_enc(S, w, tid);
  const AOff<D> A2(i, q);
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
    const EncLds& L = fresh(S);
    f32x4 z[8];
    enc_z1(L, fa, q, z);
    bf16x8 a1[4];
    enc_z2(L, A2, z, q, a1, z);
    ln_normalize(z, eps);
#pragma unroll
    for (int ob = 0; ob < 8; ++ob)
      z[ob] = *reinterpret_cast<const f32x4*>(L.g + 8 * q + fo_c(ob)) * z[ob] +
              *reinterpret_cast<const f32x4*>(L.bt + 8 * q + fo_c(ob));
    if (u * 16 + i < E) {
      bf16* op = e_out + (u * 16 + i) * D + 8 * q;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(op + 32 * s) = __builtin_bit_cast(uint4, pack_run(z[2 * s], z[2 * s + 1]));
    }
    fa = fn;
  }
}

// ===================================================================== reverse
// Per-block partials in the parameter order of the encoder: dW1 [128][4] at
// 0, db1 at 512, dW2 [128][128] at 640, db2 at 17024, dgamma at 17152, dbeta
// at 17280.  dW1 and db1 come from one product per K step with the operand
// [f_hi, f_lo, 1, 0..] (f = f_hi + f_lo, both bf16: the input features keep
// 16 significant bits), dW2 and db2 from dz2^T [a1, 1].
struct __attribute__((aligned(16))) EncBwdLds {
  EncLds P;
  __attribute__((aligned(16))) bf16 z2[RROWS * SLD];
  __attribute__((aligned(16))) bf16 a1[RROWS * SLD];
  __attribute__((aligned(16))) bf16 z1[RROWS * SLD];
  __attribute__((aligned(16))) bf16 f[RROWS * FLD];
};

__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_edge_enc_bwd_rows(int64_t E, const float* __restrict__ f_in, const bf16* __restrict__ ebar, MlpW w, float eps,
                    Partials part) {
  __shared__ EncBwdLds S;
  const int tid = threadIdx.x, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  stage_enc(S.P, w, tid);
  const AOff<D> A2(i, q);
  const int jp = i >> 2, c4 = i & 3;
  __syncthreads();
  const int64_t nu = (E + 15) >> 4;
  const int64_t nrounds = (nu + NW - 1) / NW;
  const int G = gridDim.x;
  bf16x8 ones;
#pragma unroll
  for (int j = 0; j < 8; ++j) ones[j] = (bf16)1.f;
  f32x4 aw2[8], ab2 = {0.f, 0.f, 0.f, 0.f}, aw1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) aw2[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float2 dga = {0.f, 0.f}, dbe = {0.f, 0.f};
  struct In {
    float4 f;
    uint4 eb[4];
  };
  // unit u = round * 8 + wave; rows clamped into [0, E)
  auto load = [&](int64_t R, In& X) {
    const int64_t row = min((R * NW + wv) * 16 + i, E - 1);
    X.f = *reinterpret_cast<const float4*>(f_in + row * KE);
    const bf16* ep = ebar + row * D + 8 * q;
#pragma unroll
    for (int k = 0; k < 4; ++k) X.eb[k] = *reinterpret_cast<const uint4*>(ep + 32 * k);
  };
  // operand of 16 columns col0.. with K = staged rows r0 + q*8 + j
  auto frag = [&](const bf16* X, int ld, int r0, int col0) -> bf16x8 {
    const bf16* p = X + (r0 + q * 8 + jp) * ld + col0 + 4 * c4;
    return cat8(lds_tr(p), lds_tr(p + 4 * ld));
  };
  const int srow = 16 * wv + i;
  In X;
  int64_t R = blockIdx.x;
  if (R < nrounds) load(R, X);
  for (; R < nrounds; R += G) {
    In Xn;
    load(R + G, Xn);
    const bool ok = (R * NW + wv) * 16 + i < E;
    {
      const EncLds& L = S.P;
      f32x4 z[8], acc[8];
      enc_z1(L, X.f, q, z);
      uint32_t mask = 0;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          mask |= (z[2 * s][r] > 0.f ? 1u : 0u) << (8 * s + r);
          mask |= (z[2 * s + 1][r] > 0.f ? 1u : 0u) << (8 * s + 4 + r);
        }
      bf16x8 a1[4];
      enc_z2(L, A2, z, q, a1, acc);
      const float rstd = ln_normalize(acc, eps);  // acc = xhat
      f32x4 yb[8];
#pragma unroll
      for (int ob = 0; ob < 8; ++ob) yb[ob] = ok ? run_block(X.eb, ob) : f32x4{0.f, 0.f, 0.f, 0.f};
      // dgamma += sum_rows ybar xhat, dbeta += sum_rows ybar
      {
        f32x4 p[8];
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) p[ob] = yb[ob] * acc[ob];
        const float2 c = colsum16(p, i);
        dga.x += c.x;
        dga.y += c.y;
        const float2 d = colsum16(yb, i);
        dbe.x += d.x;
        dbe.y += d.y;
      }
      // dz2 = rstd (dxh - mean(dxh) - xhat mean(dxh xhat)), dxh = ybar gamma
      bf16x8 dz2[4];
      {
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) {
          yb[ob] *= *reinterpret_cast<const f32x4*>(L.g + 8 * q + fo_c(ob));
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            s1 += yb[ob][r];
            s2 += yb[ob][r] * acc[ob][r];
          }
        }
        const float m1 = sum_rowlanes(s1) * (1.0f / D), m2 = sum_rowlanes(s2) * (1.0f / D);
#pragma unroll
        for (int ob = 0; ob < 8; ++ob) yb[ob] = rstd * (yb[ob] - m1 - acc[ob] * m2);
#pragma unroll
        for (int s = 0; s < 4; ++s) dz2[s] = pack_run(yb[2 * s], yb[2 * s + 1]);
      }
      // dz1 = (W2^T dz2) where z1 > 0
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
      // stage the unit's rows (rows past E have dz2 = dz1 = 0)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        *reinterpret_cast<uint4*>(S.z2 + srow * SLD + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz2[s]);
        *reinterpret_cast<uint4*>(S.a1 + srow * SLD + 32 * s + 8 * q) = __builtin_bit_cast(uint4, a1[s]);
        *reinterpret_cast<uint4*>(S.z1 + srow * SLD + 32 * s + 8 * q) = __builtin_bit_cast(uint4, dz1[s]);
      }
      // input columns: q = 0: f_hi, 1: f_lo, 2: [1, 0, 0, 0], 3: zeros
      {
        const float fv[4] = {X.f.x, X.f.y, X.f.z, X.f.w};
        bf16x4 piece;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bf16 hi = (bf16)fv[k];
          const bf16 lo = (bf16)(fv[k] - (float)hi);
          piece[k] = q == 0 ? hi : (q == 1 ? lo : (bf16)((q == 2 && k == 0) ? 1.f : 0.f));
        }
        *reinterpret_cast<bf16x4*>(S.f + srow * FLD + 4 * q) = piece;
      }
    }
    __syncthreads();
    // wave wv: output rows [16 wv, 16 wv + 16) of dW2 and dW1, K = the round's rows
#pragma unroll
    for (int kk = 0; kk < RROWS / 32; ++kk) {
      const bf16x8 az2 = frag(S.z2, SLD, 32 * kk, 16 * wv);
#pragma unroll
      for (int cb = 0; cb < 8; ++cb)
        aw2[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, frag(S.a1, SLD, 32 * kk, 16 * cb), aw2[cb], 0, 0, 0);
      ab2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(az2, ones, ab2, 0, 0, 0);
      aw1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag(S.z1, SLD, 32 * kk, 16 * wv), frag(S.f, FLD, 32 * kk, 0), aw1,
                                                    0, 0, 0);
    }
    __syncthreads();
    X = Xn;
  }
  // ---- partials
  float* base = part.buf + (size_t)blockIdx.x * part.stride;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int o = 16 * wv + 4 * q + r;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) base[640 + o * D + 16 * cb + i] = aw2[cb][r];
    // aw1: column i < 4 is sum dz1 f_hi[i], 4 + i the f_lo part, 8 the sum of dz1
    const float lo = __shfl_down(aw1[r], 4, 16);
    if (i < 4) base[o * KE + i] = aw1[r] + lo;
    if (i == 8) base[512 + o] = aw1[r];
    if (i == 0) base[17024 + o] = ab2[r];
  }
  float* red = reinterpret_cast<float*>(S.z2);  // [2][NW][D] fp32
  const int f = fo(i >> 1, q) + 2 * (i & 1);
  *reinterpret_cast<float2*>(red + wv * D + f) = dga;
  *reinterpret_cast<float2*>(red + (NW + wv) * D + f) = dbe;
  __syncthreads();
  if (tid < 2 * D) {
    const int k = tid >> 7, c = tid & (D - 1);
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < NW; ++u) v += red[(k * NW + u) * D + c];
    base[17152 + k * D + c] = v;
  }
}

}  // namespace dev

using namespace dev;

static constexpr int kEncBlocks = 256;

hipError_t launch_edge_enc_rows(int64_t E, const float* efeat, const MlpW& w, float eps, void* e_out, hipStream_t s) {
  if (E <= 0) return hipSuccess;
  const int64_t need = (((E + 15) >> 4) + NW - 1) / NW;
  int g = (int)std::min<int64_t>(need, kEncBlocks);
  if (g >= 8) g &= ~7;
  hipLaunchKernelGGL(k_edge_enc_rows, dim3(g), dim3(NT), 0, s, E, efeat, w, eps, (bf16*)e_out);
  return hipGetLastError();
}

hipError_t launch_edge_enc_bwd_rows(int64_t E, const float* efeat, const void* ebar, const MlpW& w, float eps,
                                    const Partials& part, int* nblocks, hipStream_t s) {
  *nblocks = 0;
  if (E <= 0) return hipSuccess;
  const int64_t nrounds = (((E + 15) >> 4) + NW - 1) / NW;
  const int g = (int)std::min<int64_t>(nrounds, std::min(kEncBlocks, part.max_blocks));
  *nblocks = g;
  hipLaunchKernelGGL(k_edge_enc_bwd_rows, dim3(g), dim3(NT), 0, s, E, efeat, (const bf16*)ebar, w, eps, part);
  return hipGetLastError();
}

}  // namespace mgn
