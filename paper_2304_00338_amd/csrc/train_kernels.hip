// Kernels of the patch training step (Sec. 2.2 conditions 2 and 3; App. C:
// input noise, Adam with an exponentially decaying learning rate): the
// noisy gather of a patch's state rows, the masked squared-error loss and its
// gradient with a fixed-order sum, and the fused Adam update.
#include "dev_common.hpp"
#include "launch.hpp"

namespace mgn {
namespace dev {

constexpr int kLossBlocks = 1024;  // partial sums of the loss (fixed order)

// dst[r][c] = y[v][c] + std[c] * noise[v][c], v = idx[r] clamped into
// [0, n_src); noise may be null (no noise).
__global__ void __launch_bounds__(256) k_gather_noisy(int64_t n, const float* __restrict__ y,
                                                      const float* __restrict__ noise, float4 sd,
                                                      const int32_t* __restrict__ idx, int64_t n_src,
                                                      float* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= n * 4) return;
  const int64_t r = t >> 2;
  const int c = (int)(t & 3);
  const int64_t v = min(max((int64_t)idx[r], (int64_t)0), n_src - 1);
  float out = y[v * 4 + c];
  if (noise != nullptr) {
    const float s = c == 0 ? sd.x : (c == 1 ? sd.y : (c == 2 ? sd.z : sd.w));
    out = __builtin_fmaf(s, noise[v * 4 + c], out);
  }
  dst[t] = out;
}

// Masked squared error of the stepped patch state against the global target
// rows: gout[r][c] = 2 (pred - target) inv for interior rows (0 elsewhere),
// and per-block sums of (pred - target)^2 over interior rows, each block
// summing a contiguous range in index order (one value per thread, then a
// fixed tree).
__global__ void __launch_bounds__(256) k_mse(int64_t n, const float* __restrict__ pred,
                                             const float* __restrict__ target, const int32_t* __restrict__ idx,
                                             const uint8_t* __restrict__ mask, int64_t n_src, float inv,
                                             float* __restrict__ gout, float* __restrict__ part) {
  __shared__ float red[256];
  const int64_t per = (n * 4 + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per, hi = min(lo + per, n * 4);
  float acc = 0.f;
  for (int64_t t = lo + threadIdx.x; t < hi; t += 256) {
    const int64_t r = t >> 2;
    const int64_t v = min(max((int64_t)idx[r], (int64_t)0), n_src - 1);
    const float d = mask[r] ? pred[t] - target[v * 4 + (t & 3)] : 0.f;
    gout[t] = 2.f * d * inv;
    acc = __builtin_fmaf(d, d, acc);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

// loss += inv * sum of the partials in block order (one thread).
__global__ void k_mse_total(const float* __restrict__ part, int nb, float inv, float* __restrict__ loss) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  float s = 0.f;
  for (int b = 0; b < nb; ++b) s += part[b];
  loss[0] += s * inv;
}

// One Adam update of every parameter: m, v moments (omb = 1 - beta, formed
// in double by the caller), bias corrections bc1 = 1 - beta1^k and bc2 =
// 1 - beta2^k, p -= lr (m / bc1) / (sqrt(v / bc2) + eps).
__global__ void __launch_bounds__(256) k_adam(int64_t n, float* __restrict__ p, const float* __restrict__ g,
                                              float* __restrict__ m, float* __restrict__ v, float lr, float b1,
                                              float omb1, float b2, float omb2, float eps, float bc1, float bc2) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float gi = g[i];
  const float mi = b1 * m[i] + omb1 * gi;
  const float vi = b2 * v[i] + omb2 * gi * gi;
  m[i] = mi;
  v[i] = vi;
  p[i] -= lr * (mi / bc1) / (__builtin_sqrtf(vi / bc2) + eps);
}

}  // namespace dev

using namespace dev;

int loss_blocks() { return kLossBlocks; }

hipError_t launch_gather_noisy(int64_t n, const float* y, const float* noise, const float* sd, const int32_t* idx,
                               int64_t n_src, float* dst, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n_src <= 0) return hipErrorInvalidValue;
  const float4 s4 = {sd[0], sd[1], sd[2], sd[3]};
  hipLaunchKernelGGL(k_gather_noisy, dim3((unsigned)((n * 4 + 255) / 256)), dim3(256), 0, s, n, y, noise, s4, idx,
                     n_src, dst);
  return hipGetLastError();
}

hipError_t launch_mse(int64_t n, const float* pred, const float* target, const int32_t* idx, const uint8_t* mask,
                      int64_t n_src, float inv, float* gout, float* part, float* loss, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n_src <= 0) return hipErrorInvalidValue;
  const int nb = (int)std::min<int64_t>(kLossBlocks, (n * 4 + 255) / 256);
  hipLaunchKernelGGL(k_mse, dim3(nb), dim3(256), 0, s, n, pred, target, idx, mask, n_src, inv, gout, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_mse_total, dim3(1), dim3(64), 0, s, part, nb, inv, loss);
  return hipGetLastError();
}

hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v, float lr, float b1, float omb1, float b2,
                       float omb2, float eps, float bc1, float bc2, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_adam, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, n, p, g, m, v, lr, b1, omb1, b2, omb2,
                     eps, bc1, bc2);
  return hipGetLastError();
}

}  // namespace mgn
