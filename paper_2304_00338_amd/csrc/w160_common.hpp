// Lane layout and LDS helpers of the bf16 row-per-wave kernels at the latent
// width 150 computed 160 wide (App. C: the 3D model; padded features are
// exactly zero).
//
// Lane l (i = l & 15, q = l >> 4) holds row i of a 16-row unit and the five
// 8-feature runs [32s + 8q, 32s + 8q + 8), s < 5.  The products run
// transposed (C[feature][row] = W x^T): the A operand is a 16-row block of a
// weight matrix whose rows are in perm_row order, so the C fragment of output
// block ob hands lane q the features fo(ob, q) + r, which are again its runs.
// Weights are staged either in LDS rows padded to 168 elements (336 bytes:
// the 16 rows of an A fragment start in distinct 4-bank groups) or unpadded
// with the 16-byte chunks of row R rotated by R / 4 (mod 20), so that both
// the row reads of A fragments and the transposing reads
// (ds_read_b64_tr_b16) for products with W^T hit distinct banks.
#pragma once
#include "rows_common.hpp"

namespace mgn {
namespace dev {
namespace w160 {
constexpr int L = 160;   // kernel width
constexpr int LR = 150;  // real latent width
constexpr int LW = 168;  // LDS row stride of the staged weights and stage (elements)
constexpr int NS = 5;    // runs per lane
constexpr int NOB = 10;  // 16-feature output blocks

constexpr int CPR = L / 8;  // 16-byte chunks per row
// LDS row stride (elements) of staged [rows][160] bf16 tiles read by
// transposing reads (ds_read_b64_tr_b16 at 8 rows x 4 columns per 16 lanes):
// 352-byte rows keep those reads free of bank conflicts.
constexpr int WG_LD = 176;

// Lane-independent part of fo(ob, q) (fo(ob, q) = 8 q + fo0(ob)): LDS
// reads at a per-lane base plus this constant fold the constant into the
// instruction's offset.
__device__ __forceinline__ constexpr int fo0(int ob) { return 32 * (ob >> 1) + 4 * (ob & 1); }
// Element offset of chunk C of row R in the rotated layout.
__device__ __forceinline__ int rot(int R, int C) {
  int p = C + (R >> 2);
  p = p >= CPR ? p - CPR : p;
  p = p >= CPR ? p - CPR : p;
  return R * L + p * 8;
}
// Copy a row-major [160][160] bf16 matrix into LDS in the rotated layout.
__device__ __forceinline__ void stage_rot(bf16* dst, const bf16* __restrict__ src, int tid) {
  for (int idx = tid; idx < L * CPR; idx += NT) {
    const int row = idx / CPR, c = idx % CPR;
    *reinterpret_cast<uint4*>(dst + rot(row, c)) = *reinterpret_cast<const uint4*>(src + row * L + c * 8);
  }
}
// Per-lane parts of the fragment addresses, so that every read is one of
// five per-lane offsets plus an immediate.
// A fragment of output block ob at K step s of W x: row 16 ob + i, chunk
// 4 s + q, rotated to (4 ((s + ob) mod 5) + q + i / 4) mod 20.
// A fragment of output block ob at K step s of W^T x from the same copy:
// A[m][k] = W[o][k'] with k' = perm_row(16 ob + m) (the lane's output runs)
// and o = 32 s + 8 q + 4 t + j' running over the B operand's run s; row o of
// W sits at packed row R = 32 s + 16 t + 4 q + j', and lane 4 j' + c
// supplies the 4 columns 32 (ob / 2) + 8 c + 4 (ob % 2) .. + 3 of it (one
// 8-byte piece of chunk 4 (ob / 2) + c), rotated by R / 4 = 8 s + 4 t + q to
// (4 ((ob / 2 + 2 s + t) mod 5) + c + q) mod 20.
struct RotOff {
  int a[5], t[5];
  __device__ __forceinline__ RotOff(int i, int q) {
    const int b = q + (i >> 2), bt = (i & 3) + q;
#pragma unroll
    for (int k = 0; k < 5; ++k) {
      const int pa = (4 * k + b) % CPR, pt = (4 * k + bt) % CPR;
      a[k] = i * L + pa * 8;
      t[k] = (4 * q + (i >> 2)) * L + pt * 8;
    }
  }
  __device__ __forceinline__ bf16x8 a_frag(const bf16* W, int ob, int s) const {
    return *reinterpret_cast<const bf16x8*>(W + ob * 16 * L + a[(s + ob) % 5]);
  }
  __device__ __forceinline__ bf16x8 t_frag(const bf16* W, int ob, int s) const {
    const int k = ((ob >> 1) + 2 * s) % 5, h = 4 * (ob & 1);
    const bf16* p0 = W + 32 * s * L + t[k] + h;
    const bf16* p1 = W + (32 * s + 16) * L + t[(k + 1) % 5] + h;
    return cat8(lds_tr(p0), lds_tr(p1));
  }
};

// Copy a row-major [160][160] bf16 matrix into LDS rows of stride LW.
__device__ __forceinline__ void stage_w(bf16* dst, const bf16* __restrict__ src, int tid) {
  constexpr int CPR = L / 8;
  for (int idx = tid; idx < L * CPR; idx += NT) {
    const int row = idx / CPR, c = idx % CPR;
    *reinterpret_cast<uint4*>(dst + row * LW + c * 8) = *reinterpret_cast<const uint4*>(src + row * L + c * 8);
  }
}

// C-layout fragment of output block ob from the lane's five bf16 runs.
__device__ __forceinline__ f32x4 run_block5(const uint4 (&runs)[NS], int ob) {
  const bf16x8 v = __builtin_bit_cast(bf16x8, runs[ob >> 1]);
  const int h = 4 * (ob & 1);
  return f32x4{(float)v[h], (float)v[h + 1], (float)v[h + 2], (float)v[h + 3]};
}

// Mask of the real features among fo(ob, q) + r, r < 4 (bit r).
__device__ __forceinline__ int live_bits(int ob, int q) {
  const int f = fo(ob, q);
  return f + 4 <= LR ? 15 : (f >= LR ? 0 : (1 << (LR - f)) - 1);
}

// Column sums over the 16 rows of a half of the 8 values v[k] = c[8 + k / 4]
// [k % 4] (output blocks 8, 9): three halving butterfly steps (partners
// 15 - i, i ^ 7, i ^ 3) and a final add with lane i ^ 1, after which lanes i
// and i ^ 1 both hold the sum of the value tail_feature names.  Every lane
// adds in a fixed order.
__device__ __forceinline__ float colsum16_tail(const f32x4 (&c)[NOB], int i) {
  float v[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = c[8 + (k >> 2)][k & 3];
  bfly_step<4, 0x140>(v, (i >> 3) & 1);  // row_mirror: lane 15 - i
  bfly_step<2, 0x141>(v, (i >> 2) & 1);  // row_half_mirror: lane i ^ 7
  bfly_step<1, 0x1B>(v, (i >> 1) & 1);   // quad_perm [3,2,1,0]: lane i ^ 3
  return v[0] + dpp_mov<0xB1>(v[0]);     // quad_perm [1,0,3,2]: lane i ^ 1
}
// Value index k (feature fo(8 + k / 4, q) + k % 4) whose column sum lane i
// holds after colsum16_tail: bit 2 of k is bit 3 of i, bit 1 is bit 2, bit 0
// is bit 1 (the halving steps keep the upper half in the lanes with the bit
// set).
__device__ __forceinline__ int tail_feature(int i, int q) {
  const int k = (((i >> 3) & 1) << 2) | (((i >> 2) & 1) << 1) | ((i >> 1) & 1);
  return fo(8 + (k >> 2), q) + (k & 3);
}
}  // namespace w160

}  // namespace dev
}  // namespace mgn
