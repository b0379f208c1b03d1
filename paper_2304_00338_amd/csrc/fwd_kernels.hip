// Forward kernels of one MGN call on gfx950 (Sec. 2.1 of the paper) in the
// feature-split layout: weight packing (both precisions), the bf16 node
// encoder and decoder (fp32 runs them on the row layout) and the
// long-segment fixup of the receiver sums.
//
// The first edge-MLP layer acts on the concatenation [e, h_s, h_r]; it is
// evaluated as W1e e + W1s h_s + W1r h_r, where the node products
// P_s = W1s h and P_r = W1r h are computed once per node (by the kernel that
// produced h) and gathered per edge.  This is the same linear map; only the
// fp32 summation order differs.
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

// ------------------------------------------------------------ packing
template <typename T>
__global__ void __launch_bounds__(256) k_pack(const float* __restrict__ params, T* __restrict__ pack, PackList L) {
  const PackEnt pe = L.e[blockIdx.y];
  const int64_t n = (int64_t)pe.rows * pe.cols;
  if (pe.perm >= 2) {
    // fp32 fragment-major copy for the fp32 row-layout kernels (square
    // rows x rows matrix M = W, or W^T when perm == 3): element idx =
    // ((ob * KC + c) * 64 + l) * 4 + t holds M[o][k] with o = KL (m / 4) +
    // 4 ob + m % 4 (output row of A-fragment row m = l % 16 of block ob) and
    // k = KL (l / 16) + 4 c + t (K step 4c + t of lane group l / 16),
    // KL = rows / 4 features per lane, KC = KL / 4.
    const int KL = pe.rows / 4, KC = KL / 4;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * 256) {
      const int t = (int)(idx & 3), l = (int)((idx >> 2) & 63);
      const int rest = (int)(idx >> 8), c = rest % KC, ob = rest / KC;
      const int m = l & 15, g = l >> 4;
      const int64_t o = KL * (m >> 2) + 4 * ob + (m & 3), k = KL * g + 4 * c + t;
      const int64_t src = pe.perm == 2 ? pe.src + o * pe.ld + k : pe.src + k * pe.ld + o;
      pack[pe.dst + idx] = (T)params[src];
    }
    return;
  }
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * 256) {
    const int64_t r = idx / pe.cols, c = idx % pe.cols;
    const int64_t sr = pe.perm ? perm_row((int)r) : r;
    const T v = (T)params[pe.src + sr * pe.ld + c];
    pack[pe.dst + idx] = v;
    if (pe.dstt >= 0) pack[pe.dstt + c * pe.rows + r] = v;
  }
}

// Node products for the next block's edge MLP: P[v] = [W1s h_v, W1r h_v].
template <int PREC, int LD>
__device__ __forceinline__ void emit_P(const typename Tr<PREC>::T* sH, int ld, const MlpW& nx, int64_t r0, int nr,
                                       typename Tr<PREC>::T* __restrict__ P_out, int w8, int i, int q) {
  typedef typename Tr<PREC>::T T;
  constexpr int D = LD;
  const T* W1 = (const T*)nx.W1;
  f32x4 ps[NRB], pr[NRB];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) ps[rb] = pr[rb] = zero4();
  gemm_tile<PREC, D>(ps, sH, ld, W1, 3 * D, w8 * 16, D, i, q);
  gemm_tile<PREC, D>(pr, sH, ld, W1, 3 * D, w8 * 16, 2 * D, i, q);
  const int n = w8 * 16 + i;
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = rb * 16 + q * 4 + r;
      if (row < nr) {
        typename Tr<PREC>::T* p = P_out + (size_t)(r0 + row) * (2 * D);
        p[n] = Tr<PREC>::cvt(ps[rb][r]);
        p[D + n] = Tr<PREC>::cvt(pr[rb][r]);
      }
    }
}

// ------------------------------------------------------- node encoder
template <int PREC, int LD, bool EMIT>
__global__ void __launch_bounds__(LD * 4) k_node_enc(int64_t N, const float* __restrict__ x_in, MlpW w, MlpW nx,
                                                 float eps, float* __restrict__ h_out,
                                                 typename Tr<PREC>::T* __restrict__ P_out) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int LDT = D + P::PAD;
  __shared__ float sX[TM][8];
  __shared__ __align__(16) T sA[TM * LDT];
  __shared__ LnScratch<NW> ln;
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n], b2 = w.b2[n], gam = w.gamma[n], bet = w.beta[n];
  float w1[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) w1[k] = w.W1f[n * 8 + k];
  const int64_t ntiles = (N + TM - 1) / TM;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * TM;
    const int nr = (int)min((int64_t)TM, N - r0);
    for (int idx = tid; idx < TM * 8; idx += NT) {
      const int row = idx >> 3, k = idx & 7;
      sX[row][k] = row < nr ? x_in[(r0 + row) * 8 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        float z = b1;
#pragma unroll
        for (int k = 0; k < 8; ++k) z += w1[k] * sX[row][k];
        sA[row * LDT + n] = P::cvt(fmaxf(z, 0.f));
      }
    __syncthreads();
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b2, b2, b2, b2};
    gemm_tile<PREC, D>(acc, sA, LDT, (const T*)w.W2, D, w8 * 16, 0, i, q);
    f32x4 mean[NRB], rstd[NRB];
    ln_stats(acc, ln, eps, w8, i, q, mean, rstd);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rb * 16 + q * 4 + r;
        const float y = gam * ((acc[rb][r] - mean[rb][r]) * rstd[rb][r]) + bet;
        acc[rb][r] = y;
        if (row < nr) h_out[(size_t)(r0 + row) * D + n] = y;
        if (EMIT) sA[row * LDT + n] = P::cvt(y);
      }
    if (EMIT) {
      __syncthreads();
      emit_P<PREC, LD>(sA, LDT, nx, r0, nr, P_out, w8, i, q);
    }
    __syncthreads();
  }
}

// Long in-segments: dst[v] = sum of the chunk slots in chunk order.
template <int LD>
__global__ void __launch_bounds__(LD) k_slot_fixup(const int32_t* __restrict__ longn, const float* __restrict__ slots,
                                                   float* __restrict__ dst) {
  constexpr int D = LD;
  const int4 L = reinterpret_cast<const int4*>(longn)[blockIdx.x];
  const int c = threadIdx.x;
  float s = 0.f;
  for (int k = 0; k < L.z; ++k) s += slots[(size_t)(L.y + k) * D + c];
  dst[(size_t)L.x * D + c] = s;
}

// ------------------------------------------------------------ decoder
// out = W2 relu(W1 h + b1) + b2 (no LayerNorm); 4 outputs per node.
template <int PREC, int LD>
__global__ void __launch_bounds__(LD * 4) k_decoder(int64_t N, const float* __restrict__ h, MlpW w, float* __restrict__ out) {
  typedef Tr<PREC> P;
  typedef typename P::T T;
  constexpr int D = LD;
  [[maybe_unused]] constexpr int NW = Width<LD>::NW, NT = Width<LD>::NT;
  constexpr int LDT = D + P::PAD;
  constexpr int LDM = D + 4;
  __shared__ __align__(16) T sX[TM * LDT];
  __shared__ float sA[TM * LDM];
  const int tid = threadIdx.x, w8 = tid >> 6, lane = tid & 63, i = lane & 15, q = lane >> 4;
  const int n = w8 * 16 + i;
  const float b1 = w.b1[n];
  const int64_t ntiles = (N + TM - 1) / TM;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * TM;
    const int nr = (int)min((int64_t)TM, N - r0);
    stage_rows<D>(sX, LDT, h + (size_t)r0 * D, nr, tid);
    __syncthreads();
    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{b1, b1, b1, b1};
    gemm_tile<PREC, D>(acc, sX, LDT, (const T*)w.W1, D, w8 * 16, 0, i, q);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) sA[(rb * 16 + q * 4 + r) * LDM + n] = fmaxf(acc[rb][r], 0.f);
    __syncthreads();
    if (tid < TM * 4) {
      const int row = tid >> 2, o = tid & 3;
      if (row < nr) {
        float s = w.b2[o];
        const float* wr = w.W2f + o * D;
        for (int k = 0; k < D; ++k) s += wr[k] * sA[row * LDM + k];
        out[(r0 + row) * 4 + o] = s;
      }
    }
    __syncthreads();
  }
}

}  // namespace dev

// ============================================================ launchers
using namespace dev;

int grid_for(int64_t n_tiles, int max_blocks) {
  if (n_tiles <= 0) return 0;
  return (int)std::min<int64_t>(n_tiles, (int64_t)max_blocks);
}

int part_grid(int64_t n_tiles, int max_blocks) {
  if (n_tiles <= 0) return 0;
  const int64_t cap = std::max<int64_t>(256, n_tiles / 16);
  return (int)std::min<int64_t>(std::min<int64_t>(n_tiles, (int64_t)max_blocks), cap);
}

static constexpr int kFwdBlocks = 1024;

hipError_t launch_pack(int prec, const float* params, void* pack, const PackList& L, hipStream_t s) {
  if (L.n <= 0) return hipSuccess;
  dim3 grid(64, L.n);
  if (prec == MGN_BF16)
    hipLaunchKernelGGL(k_pack<bf16>, grid, dim3(256), 0, s, params, (bf16*)pack, L);
  else
    hipLaunchKernelGGL(k_pack<float>, grid, dim3(256), 0, s, params, (float*)pack, L);
  return hipGetLastError();
}

hipError_t launch_node_enc(int prec, int lat, int64_t N, const float* x, const MlpW& w, const MlpW* nx, float eps,
                           float* h_out, void* P_out, hipStream_t s) {
  const int g = grid_for((N + TM - 1) / TM, kFwdBlocks);
  if (!g) return hipSuccess;
  const MlpW nn = nx ? *nx : w;
  // bf16 (fp32 runs on launch_node_enc_r32)
  if (prec != MGN_BF16) return hipErrorInvalidValue;
#define F(LD)                                                                                                        \
  if (nx)                                                                                                            \
    hipLaunchKernelGGL((k_node_enc<MGN_BF16, LD, true>), dim3(g), dim3(LD * 4), 0, s, N, x, w, nn, eps, h_out,       \
                       (bf16*)P_out);                                                                                \
  else                                                                                                               \
    hipLaunchKernelGGL((k_node_enc<MGN_BF16, LD, false>), dim3(g), dim3(LD * 4), 0, s, N, x, w, nn, eps, h_out,      \
                       (bf16*)P_out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_slot_fixup(int lat, const int32_t* long_nodes, int64_t n_long, const float* slots, float* dst,
                             hipStream_t s) {
  if (n_long <= 0) return hipSuccess;
#define F(LD) hipLaunchKernelGGL(k_slot_fixup<LD>, dim3((unsigned)n_long), dim3(LD), 0, s, long_nodes, slots, dst)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

hipError_t launch_decoder(int prec, int lat, int64_t N, const float* h, const MlpW& w, float* out, hipStream_t s) {
  const int g = grid_for((N + TM - 1) / TM, kFwdBlocks);
  if (!g) return hipSuccess;
  // bf16 (fp32 runs on launch_decoder_r32)
  if (prec != MGN_BF16) return hipErrorInvalidValue;
#define F(LD) hipLaunchKernelGGL((k_decoder<MGN_BF16, LD>), dim3(g), dim3(LD * 4), 0, s, N, h, w, out)
  MGN_BY_WIDTH(lat, F);
#undef F
  return hipGetLastError();
}

}  // namespace mgn
