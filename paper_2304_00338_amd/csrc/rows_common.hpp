// Register and LDS layout shared by the one-wave-per-row-block kernels (edge
// and node phases of an MP step, bf16 operands).
//
// Lane l (i = l & 15, q = l >> 4) holds row i of a 16-row block and 32
// features of it: the runs [32s + 8q, 32s + 8q + 8) for s < 4, so the four
// lanes of a row read or write 64 contiguous bytes (bf16) per instruction.
// The GEMMs run transposed (C[feature][row] = W x^T): the A operand is a
// 16-row block of the row-permuted weights (perm_row) read from LDS, the B
// operand at K step s is the lane's run s of x, and the C fragment of output
// block ob gives the lane the features fo(ob, q) + r, r < 4, which are again
// its runs.  So GEMM outputs are already the next GEMM's B operand, and every
// LayerNorm statistic is a sum over the lane's 32 values plus two cross-lane
// steps (the four lanes that share a row).
#pragma once

#include "dev_common.hpp"

namespace mgn {
namespace dev {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// First feature of the 4-feature run of output block ob held by lane group q.
__device__ __forceinline__ int fo(int ob, int q) { return 32 * (ob >> 1) + 8 * q + 4 * (ob & 1); }

// The staged bf16 weights keep rows unpadded ([rows][LD], LD a multiple of
// 128) and XOR-swizzle the 16-byte chunks of row R inside every 256-byte
// span, so that both the row reads of A fragments (8 lanes: 8 consecutive
// rows, one chunk) and the transposing reads (16 lanes: 4 consecutive rows
// x 4 chunks) hit distinct banks.
__device__ __forceinline__ int wswz(int R) { return 4 * (R & 3) + ((R >> 2) & 3); }
template <int LD = D>
__device__ __forceinline__ const bf16* wchunk(const bf16* W, int R, int C) {
  return W + R * LD + ((C ^ wswz(R)) << 3);
}
template <int LD = D>
__device__ __forceinline__ bf16* wchunk_w(bf16* W, int R, int C) {
  return W + R * LD + ((C ^ wswz(R)) << 3);
}

// Stage the row-permuted [D][LD] bf16 matrix src into LDS in the swizzled
// layout (all threads of the block take part; a barrier must follow).
template <int LD>
__device__ __forceinline__ void stage_weights(bf16* dst, const bf16* src, int tid) {
  constexpr int CPR = LD / 8;  // 16-byte chunks per row
  for (int idx = tid; idx < D * CPR; idx += NT) {
    const int row = idx / CPR, c = idx % CPR;
    *reinterpret_cast<uint4*>(wchunk_w<LD>(dst, row, c)) = *reinterpret_cast<const uint4*>(src + row * LD + c * 8);
  }
}

// The 0/1 operand that adds a B fragment (run s: features 32s + 8q + j) into
// the C fragment of output block ob = 2s + h: A[m][k] = 1 iff k = (m/4)*8 +
// 4h + m%4.
__device__ __forceinline__ bf16x8 select_frag(int h, int i, int q) {
  bf16x8 a;
#pragma unroll
  for (int j = 0; j < 8; ++j) a[j] = (bf16)(((i >> 2) == q && j == 4 * h + (i & 3)) ? 1.f : 0.f);
  return a;
}

// Rows of a receiver-aligned tile {node_begin, node_end | -1 - slot, edge_begin, edge_end}.
__device__ __forceinline__ int tile_rows(int4 d) { return d.w - d.z; }

// Descriptor t of the tile table.  The table is read-only while a kernel
// runs, and a wave reads one descriptor at a time (t uniform): read through
// the constant address space it becomes a scalar load, which the compiler
// waits for with lgkmcnt.  As a vector load it was waited for with vmcnt,
// and the kernels need its fields early as scalars, so that wait also
// waited for the next half's streams requested before it.
typedef int TileWords __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(4))) const TileWords ConstTileWords;
__device__ __forceinline__ int4 tile_desc(const int32_t* tiles, int64_t t) {
  const TileWords v = ((const ConstTileWords*)tiles)[t];
  return make_int4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ bf16x8 as_frag(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

// B operand of run s from the two C-layout fragments of blocks 2s, 2s + 1.
__device__ __forceinline__ bf16x8 pack_run(const f32x4& lo, const f32x4& hi) {
  bf16x8 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    v[r] = (bf16)lo[r];
    v[4 + r] = (bf16)hi[r];
  }
  return v;
}

// C-layout fragment of output block ob (fp32) from the lane's four bf16
// runs: run ob / 2, elements 4 (ob % 2) .. + 4.
__device__ __forceinline__ f32x4 run_block(const uint4 (&runs)[4], int ob) {
  const bf16x8 v = __builtin_bit_cast(bf16x8, runs[ob >> 1]);
  const int h = 4 * (ob & 1);
  return f32x4{(float)v[h], (float)v[h + 1], (float)v[h + 2], (float)v[h + 3]};
}

// max(x, 0) as one integer max on the bit pattern (negative floats have the
// sign bit set, so they compare below +0.0 as signed integers).
__device__ __forceinline__ float relu(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

// Sum over the four lanes that hold the same row (q = 0..3).
__device__ __forceinline__ float sum_rowlanes(float s) { return sum_q(s); }

// Transposing LDS read (gfx950 ds_read_b64_tr_b16): within each group of 16
// lanes, result lane l, element j' is element l & 3 of the 8 bytes addressed
// by lane 4j' + (l >> 2).
// A 16-byte global load with the nontemporal hint, for streams read once
// (the weight-gradient passes read their four streams with it: they are not
// re-read, so they need not displace cached lines).
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}

__device__ __forceinline__ bf16x4 lds_tr(const bf16* p) {
  typedef __attribute__((address_space(3))) bf16x4 lds_v4;
  typedef __attribute__((address_space(3))) bf16 lds_b;
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)((lds_b*)p));
}
__device__ __forceinline__ bf16x8 cat8(bf16x4 lo, bf16x4 hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// A operand of the transposed product C = W^T x from the row-permuted LDS
// copy WP ([D][LD]) of W (rows = output features o of W): A[m][k] = W[o][k']
// with output slot m of block ob being input feature k' = 128 (ob / 8) +
// perm_row(16 (ob % 8) + m) and k = 8q + 4t + j' running over o = 32s + 8q +
// 4t + j' (lane q's run s).  Row o of W sits at packed row 16(2s + t) + 4q +
// j'; lane 4j' + c supplies the 4 columns k'(16ob + 4c + 0..3) of it (one
// 8-byte piece).
template <int LD = D>
__device__ __forceinline__ bf16x8 wt_frag(const bf16* WP, int ob, int s, int lam, int q) {
  const int jp = lam >> 2, c = lam & 3;
  const int R = (2 * s) * 16 + 4 * q + jp, C = 16 * (ob >> 3) + 4 * ((ob & 7) >> 1) + c, h = 4 * (ob & 1);
  const bf16* p0 = wchunk<LD>(WP, R, C) + h;
  const bf16* p1 = wchunk<LD>(WP, R + 16, C) + h;
  return cat8(lds_tr(p0), lds_tr(p1));
}

// Per-lane parts of the A-operand addresses, so that every fragment read is
// a per-lane base plus an immediate.  Row ob*16 + i has the swizzle wswz(i)
// and chunk 4s + q of it sits at 16 (s / 4) + ((4 (s % 4) + q) ^ wswz(i)):
// four bases per matrix (s % 4).  For the transposing reads of wt_frag the
// rows are R = 32s + 16t + 4q + j' with wswz(R) = 4j' + q, and chunk
// 16 (ob / 8) + 4 ((ob / 2) % 4) + c sits at 16 (ob / 8) + 4 (((ob / 2) % 4)
// ^ j') + (c ^ q): four bases per matrix ((ob / 2) % 4).
template <int LD = D>
struct AOff {
  int row[4], tr[4];
  __device__ __forceinline__ AOff(int i, int q) {
    const int jp = i >> 2, c = i & 3;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      row[k] = i * LD + (((4 * k + q) ^ wswz(i)) << 3);
      tr[k] = (4 * q + jp) * LD + 32 * (k ^ jp) + 8 * (c ^ q);
    }
  }
  // A fragment of output block ob at K step s of W x (same as
  // *wchunk<LD>(W, ob * 16 + i, 4 * s + q))
  __device__ __forceinline__ bf16x8 a(const bf16* W, int ob, int s) const {
    return *reinterpret_cast<const bf16x8*>(W + ob * 16 * LD + 128 * (s >> 2) + row[s & 3]);
  }
  // A fragment of output block ob at K step s of W^T x (same as wt_frag<LD>)
  __device__ __forceinline__ bf16x8 t(const bf16* W, int ob, int s) const {
    const bf16* p = W + tr[(ob >> 1) & 3] + 32 * s * LD + 128 * (ob >> 3) + 4 * (ob & 1);
    return cat8(lds_tr(p), lds_tr(p + 16 * LD));
  }
};

// Overwrites z with xhat = (z - mean) * rstd over the row's 128 features
// (biased variance, two passes) and returns rstd.
__device__ __forceinline__ float ln_normalize(f32x4 (&z)[8], float eps) {
  float sm = 0.f;
#pragma unroll
  for (int ob = 0; ob < 8; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) sm += z[ob][r];
  const float mean = sum_rowlanes(sm) * (1.0f / D);
  float sq = 0.f;
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) {
    z[ob] -= mean;
#pragma unroll
    for (int r = 0; r < 4; ++r) sq += z[ob][r] * z[ob][r];
  }
  const float rstd = __builtin_amdgcn_rsqf(sum_rowlanes(sq) * (1.0f / D) + eps);
#pragma unroll
  for (int ob = 0; ob < 8; ++ob) z[ob] *= rstd;
  return rstd;
}

// Column sums over the 16 rows of a unit (the 16 lanes of one DPP row) of
// the 32 C-layout values v[ob][r], as a butterfly that halves the values
// held at every step (partners i ^ 15, i ^ 7, i ^ 3, i ^ 1): lane i ends
// with the sums of value indices 2i and 2i + 1 (= 4ob + r), i.e. features
// fo(i / 2, q) + 2 (i % 2) + {0, 1}.  Every lane adds in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
template <int N, int CTRL>
__device__ __forceinline__ void bfly_step(float* v, bool hi) {
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const float send = hi ? v[k] : v[k + N];
    const float keep = hi ? v[k + N] : v[k];
    v[k] = keep + dpp_mov<CTRL>(send);
  }
}
__device__ __forceinline__ float2 colsum16(const f32x4 (&c)[8], int i) {
  float v[32];
#pragma unroll
  for (int ob = 0; ob < 8; ++ob)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[4 * ob + r] = c[ob][r];
  bfly_step<16, 0x140>(v, (i >> 3) & 1);  // row_mirror: lane 15 - i
  bfly_step<8, 0x141>(v, (i >> 2) & 1);   // row_half_mirror: lane i ^ 7
  bfly_step<4, 0x1B>(v, (i >> 1) & 1);    // quad_perm [3,2,1,0]: lane i ^ 3
  bfly_step<2, 0xB1>(v, i & 1);           // quad_perm [1,0,3,2]: lane i ^ 1
  return float2{v[0], v[1]};
}

// A zero the compiler cannot see through.  Kernels whose unit loop writes
// no LDS index their staged weights with a fresh one per unit; otherwise
// every weight fragment read is loop-invariant and gets hoisted into (far
// too many) registers.
__device__ __forceinline__ int opaque_zero() {
  int z = 0;
  asm volatile("" : "+v"(z));
  return z;
}
template <class T>
__device__ __forceinline__ const T& fresh(const T& lds) {
  return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(&lds) + opaque_zero());
}

// Persistent unit range of wave wv: blocks are dealt to the 8 XCDs
// round-robin, so with a grid of a multiple of 8 blocks the waves of one
// XCD walk one contiguous eighth of the units.
struct UnitRange {
  int64_t t, stride, end;
};
template <int NWB = NW>  // waves per block
__device__ __forceinline__ UnitRange unit_range(int64_t n_units, int wv) {
  const int G = gridDim.x;
  UnitRange u;
  if ((G & 7) == 0) {
    const int x = blockIdx.x & 7, per = G >> 3;
    const int64_t chunk = (n_units + 7) >> 3;
    const int64_t lo = x * chunk;
    u.end = min(n_units, lo + chunk);
    u.t = lo + (int64_t)(blockIdx.x >> 3) * NWB + wv;
    u.stride = (int64_t)per * NWB;
  } else {
    u.t = (int64_t)blockIdx.x * NWB + wv;
    u.stride = (int64_t)G * NWB;
    u.end = n_units;
  }
  return u;
}

}  // namespace dev
}  // namespace mgn
