// Small node-state kernels of the explicit integrators (Sec. 2.1 update
// rule, Sec. 2.3 / App. A Heun forms): stage inputs y + sum_j a_ij K_j and
// the final combination y + sum_i b_i K_i, summed in ascending term order.
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

__global__ void __launch_bounds__(256) k_lincomb(int64_t N, LinComb lc, float* __restrict__ out, int32_t out_ld,
                                                 int32_t out_off) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= N * 4) return;
  const int64_t v = idx >> 2;
  const int c = (int)(idx & 3);
  float s = lc.c[0] * lc.x[0][v * lc.ld[0] + lc.off[0] + c];
  for (int j = 1; j < lc.n; ++j) s += lc.c[j] * lc.x[j][v * lc.ld[j] + lc.off[j] + c];
  out[v * out_ld + out_off + c] = s;
}

__global__ void __launch_bounds__(256) k_copy_static(int64_t N, const float* __restrict__ st, float* __restrict__ node_in) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= N * 4) return;
  const int64_t v = idx >> 2;
  const int c = (int)(idx & 3);
  node_in[v * 8 + c] = st[v * 4 + c];
}

__global__ void __launch_bounds__(256) k_fill(int64_t n, float v, float* __restrict__ p) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx < n) p[idx] = v;
}

// Row moves between a patch's local node order and the global one (4
// floats per row, one thread per float).  Ids outside [0, n) are clamped:
// a caller error gives wrong rows, never an out-of-bounds access.
__global__ void __launch_bounds__(256) k_gather_rows4(int64_t n, const float* __restrict__ src,
                                                      const int32_t* __restrict__ idx, int64_t n_src,
                                                      float* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n * 4) return;
  const int64_t r = t >> 2;
  const int64_t v = min(max((int64_t)idx[r], (int64_t)0), n_src - 1);
  dst[t] = src[v * 4 + (t & 3)];
}

__global__ void __launch_bounds__(256) k_scatter_rows4(int64_t n, const float* __restrict__ src,
                                                       const int32_t* __restrict__ idx,
                                                       const uint8_t* __restrict__ mask, int64_t n_dst,
                                                       float* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n * 4) return;
  const int64_t r = t >> 2;
  if (mask[r] == 0) return;
  const int64_t v = min(max((int64_t)idx[r], (int64_t)0), n_dst - 1);
  dst[v * 4 + (t & 3)] = src[t];
}

// Rectangular block moves between two parameter layouts (the real latent-150
// layout and the kernels' zero-padded latent-160 one): block k moves
// a[a_off + r * a_ld + c] to b[b_off + r * b_ld + c], added to b when
// accumulate is set.  Blocks of one list never overlap in b.
__global__ void __launch_bounds__(256) k_copy_blocks(CopyList L, const float* __restrict__ a, float* __restrict__ b,
                                                     int accumulate) {
  const CopyBlock cb = L.b[blockIdx.y];
  const int64_t n = (int64_t)cb.rows * cb.cols;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * 256) {
    const int64_t r = idx / cb.cols, c = idx % cb.cols;
    const float v = a[cb.a_off + r * cb.a_ld + c];
    float* d = b + cb.b_off + r * cb.b_ld + c;
    *d = accumulate ? *d + v : v;
  }
}

// b = a + b over n values of an edge-latent stream (fp32, or bf16 added in
// fp32 and rounded to nearest even), 8 values per thread; n is a multiple of
// 8 (the latent width is).
__global__ void __launch_bounds__(256) k_add_stream_f32(int64_t n8, const float4* __restrict__ a,
                                                        float4* __restrict__ b) {
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < n8; t += (int64_t)gridDim.x * 256) {
    const float4 x0 = a[2 * t], x1 = a[2 * t + 1];
    float4 y0 = b[2 * t], y1 = b[2 * t + 1];
    y0.x += x0.x; y0.y += x0.y; y0.z += x0.z; y0.w += x0.w;
    y1.x += x1.x; y1.y += x1.y; y1.z += x1.z; y1.w += x1.w;
    b[2 * t] = y0;
    b[2 * t + 1] = y1;
  }
}

__global__ void __launch_bounds__(256) k_add_stream_bf16(int64_t n8, const uint4* __restrict__ a,
                                                         uint4* __restrict__ b) {
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < n8; t += (int64_t)gridDim.x * 256) {
    const bf16x8 x = __builtin_bit_cast(bf16x8, a[t]);
    bf16x8 y = __builtin_bit_cast(bf16x8, b[t]);
#pragma unroll
    for (int u = 0; u < 8; ++u) y[u] = (bf16)((float)y[u] + (float)x[u]);
    b[t] = __builtin_bit_cast(uint4, y);
  }
}

}  // namespace dev

using namespace dev;

hipError_t launch_add_stream(int prec, int64_t n, const void* a, void* b, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 8) return hipErrorInvalidValue;
  const int64_t n8 = n / 8;
  const unsigned g = (unsigned)std::min<int64_t>((n8 + 255) / 256, 8192);
  if (prec == MGN_BF16)
    hipLaunchKernelGGL(k_add_stream_bf16, dim3(g), dim3(256), 0, s, n8, (const uint4*)a, (uint4*)b);
  else
    hipLaunchKernelGGL(k_add_stream_f32, dim3(g), dim3(256), 0, s, n8, (const float4*)a, (float4*)b);
  return hipGetLastError();
}

hipError_t launch_gather_rows4(int64_t n, const float* src, const int32_t* idx, int64_t n_src, float* dst,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n_src <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gather_rows4, dim3((unsigned)((n * 4 + 255) / 256)), dim3(256), 0, s, n, src, idx, n_src, dst);
  return hipGetLastError();
}

hipError_t launch_scatter_rows4(int64_t n, const float* src, const int32_t* idx, const uint8_t* mask, int64_t n_dst,
                                float* dst, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n_dst <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_scatter_rows4, dim3((unsigned)((n * 4 + 255) / 256)), dim3(256), 0, s, n, src, idx, mask,
                     n_dst, dst);
  return hipGetLastError();
}

hipError_t launch_copy_blocks(const CopyList& L, const float* a, float* b, int accumulate, hipStream_t s) {
  if (L.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_blocks, dim3(64, L.n), dim3(256), 0, s, L, a, b, accumulate);
  return hipGetLastError();
}

hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, n, v, p);
  return hipGetLastError();
}

hipError_t launch_lincomb(int64_t N, const LinComb& lc, float* out, int32_t out_ld, int32_t out_off, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const unsigned g = (unsigned)((N * 4 + 255) / 256);
  hipLaunchKernelGGL(k_lincomb, dim3(g), dim3(256), 0, s, N, lc, out, out_ld, out_off);
  return hipGetLastError();
}

hipError_t launch_stage_input(int64_t N, const float* st, const LinComb& lc, float* node_in, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const unsigned g = (unsigned)((N * 4 + 255) / 256);
  hipLaunchKernelGGL(k_copy_static, dim3(g), dim3(256), 0, s, N, st, node_in);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_lincomb(N, lc, node_in, 8, 4, s);
}

}  // namespace mgn
