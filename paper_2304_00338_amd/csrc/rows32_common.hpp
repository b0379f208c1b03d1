// The fp32 row layout shared by the fp32 edge and node kernels, at kernel
// width LD = 128 or 160 (latent 150 padded with zero columns).
//
// Lane layout.  Lane l (i = l & 15, g = l >> 4) holds row i of a 16-row
// block and the KL = LD / 4 features [KL g, KL g + KL) of it: the four lanes
// of a row hold one contiguous row, and every lane's slice is contiguous in
// memory (16-byte loads and stores).  The products run transposed on
// v_mfma_f32_16x16x4_f32, C[feature][row] = W x^T: K step s takes the
// features KL g + s from lane group g (the lane's own value s is the B
// operand), and the A operand comes from a fragment-major copy of W whose
// output rows are ordered so that the C fragment of output block ob gives
// lane group g the features KL g + 4 ob + r (r < 4), i.e. its own values
// 4 ob + r: a product's output is the next product's B operand without
// leaving registers.  The weights are read from global memory (L2) one
// 16-byte piece per lane per four K steps; in fp32 the MFMA time per row is
// about 30 times the weight traffic.
#pragma once
#include "launch.hpp"
#include "rows_common.hpp"
#include "w160_common.hpp"

namespace mgn {
namespace dev {

template <int LD>
struct R32 {
  static constexpr int KL = LD / 4;        // features per lane
  static constexpr int KC = KL / 4;        // 16-byte pieces per lane
  static constexpr int NOB = LD / 16;      // 16-feature output blocks
  static constexpr int DR = Width<LD>::DR; // real latent width
  static constexpr int SLD = LD + 4;       // LDS row stride of a staged fp32 half-tile
};

// A fragment of output block ob, K steps 4c .. 4c + 3, of a fragment-major
// fp32 matrix (lane l holds its four A values, one per K step).
template <int LD>
__device__ __forceinline__ f32x4 afrag32(const float* __restrict__ Wf, int ob, int c, int lane) {
  return *reinterpret_cast<const f32x4*>(Wf + ((size_t)(ob * R32<LD>::KC + c) * 64 + lane) * 4);
}

// acc[ob] += W x for the lane's KL values x (B operands, K step s = x[s]).
// The output blocks run in two groups of NOB / 2 interleaved accumulator
// chains; as soon as a group has used its fragments of K chunk c, the
// group's fragments of chunk c + 1 are requested into the same registers,
// so each L2 read has the other group's MFMAs (4 NOB / 2 of them) to arrive
// behind (one wave per SIMD leaves no other wave to cover it) and no
// registers beyond one chunk's fragments are used.  A scheduling barrier
// after each group's requests holds that order.  mid() runs once, halfway
// through the K chunks (for loads that the caller needs after the product).
// Every accumulator adds its K steps in ascending order.
template <int LD, class F>
__device__ __forceinline__ void gemm32(f32x4 (&acc)[R32<LD>::NOB], const float (&x)[R32<LD>::KL],
                                       const float* __restrict__ Wf, int lane, F&& mid) {
  typedef R32<LD> Z;
  constexpr int H = Z::NOB / 2;
  static_assert(Z::NOB % 2 == 0, "two groups of output blocks");
  f32x4 a[Z::NOB];
#pragma unroll
  for (int ob = 0; ob < Z::NOB; ++ob) a[ob] = afrag32<LD>(Wf, ob, 0, lane);
#pragma unroll
  for (int c = 0; c < Z::KC; ++c)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int o = h * H; o < h * H + H; ++o)
          acc[o] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[o][t], x[4 * c + t], acc[o], 0, 0, 0);
      if (c + 1 < Z::KC)
#pragma unroll
        for (int o = h * H; o < h * H + H; ++o) a[o] = afrag32<LD>(Wf, o, c + 1, lane);
      if (h == 1 && c == Z::KC / 2 - 1) mid();
      // without it the compiler interleaves the two groups by K step and
      // waits for each request a few MFMAs after issuing it
      __builtin_amdgcn_sched_barrier(0);
    }
}
template <int LD>
__device__ __forceinline__ void gemm32(f32x4 (&acc)[R32<LD>::NOB], const float (&x)[R32<LD>::KL],
                                       const float* __restrict__ Wf, int lane) {
  gemm32<LD>(acc, x, Wf, lane, [] {});
}

// The lane's KL contiguous floats of a row starting at p.
template <int LD>
__device__ __forceinline__ void load_row32(float (&x)[R32<LD>::KL], const float* __restrict__ p) {
#pragma unroll
  for (int c = 0; c < R32<LD>::KC; ++c) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p + 4 * c);
#pragma unroll
    for (int t = 0; t < 4; ++t) x[4 * c + t] = v[t];
  }
}
template <int LD>
__device__ __forceinline__ void store_row32(float* __restrict__ p, const f32x4 (&v)[R32<LD>::NOB]) {
#pragma unroll
  for (int ob = 0; ob < R32<LD>::NOB; ++ob) *reinterpret_cast<f32x4*>(p + 4 * ob) = v[ob];
}

// Four waves per block, one per SIMD: a wave has 512 registers (the fp32
// rows of a half and its prefetch need more than the 256 of two waves per
// SIMD), and its eight independent accumulator chains keep the MFMA pipe
// busy on their own.
constexpr int R32_NW = 4;
constexpr int R32_NT = 64 * R32_NW;

// Per-lane column sums over 16-row blocks of C-layout values (feature
// f0 + 4 ob + r), accumulated block after block: DPP butterflies leave lane
// i of group g with features f0 + 4 (i / 2) + 2 (i % 2) + {0, 1} of blocks
// 0..7 (v) and, at width 160, one feature of blocks 8, 9 (t, lanes of even
// i).  put() writes a wave's sums into its row of an LDS array [LD].
template <int LD>
struct ColSum32 {
  float2 v = {0.f, 0.f};
  float t = 0.f;
  __device__ __forceinline__ void add(const f32x4 (&p)[R32<LD>::NOB], int i) {
    f32x4 p8[8];
#pragma unroll
    for (int ob = 0; ob < 8; ++ob) p8[ob] = p[ob];
    const float2 c = colsum16(p8, i);
    v.x += c.x;
    v.y += c.y;
    if constexpr (R32<LD>::NOB == 10) t += w160::colsum16_tail(p, i);
  }
  __device__ __forceinline__ void put(float* row, int f0, int i) const {
    *reinterpret_cast<float2*>(row + f0 + 4 * (i >> 1) + 2 * (i & 1)) = v;
    if constexpr (R32<LD>::NOB == 10) {
      if ((i & 1) == 0) {
        const int k = (((i >> 3) & 1) << 2) | (((i >> 2) & 1) << 1) | ((i >> 1) & 1);
        row[f0 + 4 * (8 + (k >> 2)) + (k & 3)] = t;
      }
    }
  }
};

}  // namespace dev
}  // namespace mgn
