// Host-side launchers of the gfx950 kernels (internal to libmgn).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mgn {

// Weights of one two-layer MLP as the kernels see them.  W1/W2 point into
// the packed operand copy (precision of the MFMA operands), row-major
// [out][in]; W1t/W2t are the transposed copies [in][out].  Biases and
// LayerNorm parameters are the caller's float32 values.
struct MlpW {
  const void* W1p;   // row-permuted copy of W1 (edge MLPs: its edge-latent column block)
  const void* W2p;   // row-permuted copy of W2
  const void* W1sp;  // edge MLPs: row-permuted sender column block of W1
  const void* W1rp;  // edge MLPs: row-permuted receiver column block of W1
  const void* W1ap;  // node MLPs at width 160: row-permuted agg column block of W1 (W1p: the h block)
  const void* W1;
  const void* W1t;
  const void* W2;
  const void* W2t;
  const float* F1;   // fp32 row-layout kernels: fragment-major copies of the edge
  const float* F2;   // MLP's W1e (first layer, edge-latent block) and W2, and of
  const float* F1t;  // their transposes (node MLPs: F1 is W1's h block)
  const float* F2t;
  const float* F1a;   // fp32 node MLPs: fragment-major agg block of W1 and its transpose
  const float* F1at;
  const float* F1s;   // fp32 edge MLPs: fragment-major sender / receiver blocks of W1
  const float* F1r;   // (the node products P = [W1s h, W1r h]) and their transposes
  const float* F1st;
  const float* F1rt;
  const float* W1f;  // float32 first-layer weights (encoders: K = 4 / 8 on VALU)
  const float* W2f;  // float32 second-layer weights (decoder: 4 outputs on VALU)
  const float* b1;
  const float* b2;
  const float* gamma;
  const float* beta;
};

struct PackEnt {
  int64_t src;   // float offset of the [rows][cols] matrix in params
  int64_t dst;   // element offset of the copy in the pack
  int64_t dstt;  // element offset of the transposed copy (-1: none)
  int32_t rows, cols;
  int32_t ld;    // source row stride (floats)
  int32_t perm;  // 1: copy row perm_row(p) of the source into row p; 2 / 3: the
                 // fp32 fragment-major copy of the square matrix / of its transpose
};

// Output-row order of the weights used by the row-per-wave edge kernels:
// packed row p = ob*16 + m holds row 32*(ob/2) + 8*(m/4) + 4*(ob%2) + m%4 of
// W, so that the MFMA C fragment of output block ob gives lane group q the
// features 32*(ob/2) + 8q + 4*(ob%2) + r (r < 4): over the 8 blocks, the
// runs [32s + 8q, 32s + 8q + 8) that are exactly the lane's B operand of
// the next product.
__host__ __device__ inline int perm_row(int p) {
  const int ob = p >> 4, m = p & 15;
  return 32 * (ob >> 1) + 8 * (m >> 2) + 4 * (ob & 1) + (m & 3);
}
constexpr int kPackMax = 64;
struct PackList {
  PackEnt e[kPackMax];
  int32_t n;
};

struct EdgeTiles {
  const int32_t* tiles;  // [n_tiles][4]
  int64_t n_tiles;
  const int32_t* rowptr;
  const int32_t* senders;
  const int32_t* receivers;
  int64_t n_edges;
};

// Per-block partial buffers for deterministic weight-gradient reductions.
struct Partials {
  float* buf;
  int64_t stride;  // floats per block
  int32_t max_blocks;
};

// Persistent grid size: number of blocks the kernels are launched with for
// a given number of tiles (also the number of partial rows to reduce).
int grid_for(int64_t n_tiles, int max_blocks);
// Blocks of a reverse kernel whose per-block weight-gradient partials are
// summed afterwards: at most max_blocks, and on small inputs at most one
// block per 16 tiles (but at least 256, one per CU), so the reduction reads
// no more partial copies than the work needs.
int part_grid(int64_t n_tiles, int max_blocks);

hipError_t launch_pack(int prec, const float* params, void* pack, const PackList& L, hipStream_t s);

// Feature-split kernels: lat is the kernel width (128, or 160 for the
// latent 150 padded with zero columns).  bf16 at width 128 runs on the
// row-layout kernels for the edge encoder, edge phase, node phase and their
// reverse, and the bf16 edge reverse at 160 on k_edge_bwd_w160 /
// k_wgrad2_w160 (those launchers return hipErrorInvalidValue for them); the
// node encoder, decoder, sender sums and node-encoder reverse serve both
// widths.
hipError_t launch_node_enc(int prec, int lat, int64_t N, const float* node_in, const MlpW& w, const MlpW* next_edge,
                           float eps, float* h_out, void* P_out, hipStream_t s);
// fp32 edge encoder in the row layout (width 128 or 160; needs the
// fragment-major W2 and, for the reverse, its transpose): e = LN(W2 relu(W1
// f + b1) + b2), and all encoder parameter gradients from ebar as per-block
// partials in the encoder's parameter order.
// fp32 node phase in the row layout (width 128 or 160; needs the node MLP's
// fragment-major F1, F1a, F2 and, with nx, the next edge MLP's F1s, F1r):
// h_out = h + LN(W2 relu(W1 [h, agg] + b1) + b2), and with nx the next
// block's node products P_out = [W1s h_out, W1r h_out] ([N][2 lat] fp32).
hipError_t launch_node_fwd_r32(int lat, int64_t N, const float* h_in, const float* agg, const MlpW& w,
                               const MlpW* nx, float eps, float* h_out, float* P_out, hipStream_t s);
// Its reverse: hbar_part = hbar_in + W1h^T dz1, aggbar = W1a^T dz1, the
// rows of a1, dz2, dz1 into streams ([3][N][lat] fp32, for the weight
// gradients by launch_wgrad_r32), and per-block [4][lat] partials of db1,
// db2, dgamma, dbeta (needs F1t, F1at, F2t too).
hipError_t launch_node_bwd_r32(int lat, int64_t N, const float* h, const float* agg, const float* hbar_in,
                               const MlpW& w, float eps, float* hbar_part, float* aggbar, float* streams,
                               const Partials& part, int* nblocks, hipStream_t s);
// fp32 sender-side sums in the row layout (needs the edge MLP's F1st, F1rt):
// S = sum of zbar over each node's out-edges (through rev, in edge order)
// into S_out ([N][lat]), hbar_out = hbar_part + W1s^T S + W1r^T R.
hipError_t launch_node_srcsum_r32(int lat, int64_t N, const int32_t* rowptr, const int32_t* rev, const float* zbar,
                                  const float* R, const float* hbar_part, const MlpW& w, float* hbar_out,
                                  float* S_out, hipStream_t s);
// fp32 decoder in the row layout (needs the decoder's fragment-major F1 and,
// for the reverse, F1t): out = W2 relu(W1 h + b1) + b2 ([N][4]); the
// reverse writes hbar = W1^T dz1, the dz1 rows (for dW1 by launch_wgrad_r32)
// and per-block partials [lat] db1, [4][lat] dW2, [4] db2.
hipError_t launch_decoder_r32(int lat, int64_t N, const float* h, const MlpW& w, float* out, hipStream_t s);
hipError_t launch_decoder_bwd_r32(int lat, int64_t N, const float* h, const float* gout, const MlpW& w, float* hbar,
                                  float* dz1s, const Partials& part, int* nblocks, hipStream_t s);
// fp32 node encoder in the row layout (needs the encoder's fragment-major F2
// and, for the reverse, F2t; with nx the first edge MLP's F1s, F1r): h0 =
// LN(W2 relu(W1 x + b1) + b2) from the 8 node inputs, with nx also the node
// products of the first MP block.  The reverse writes gin = dL/dx (when
// given), the a1 and dz2 rows into streams ([2][N][lat], for dW2 by
// launch_wgrad_r32) and per-block partials [lat][8] dW1, [lat] db1, db2,
// dgamma, dbeta.
hipError_t launch_node_enc_r32(int lat, int64_t N, const float* x, const MlpW& w, const MlpW* nx, float eps,
                               float* h_out, float* P_out, hipStream_t s);
hipError_t launch_node_enc_bwd_r32(int lat, int64_t N, const float* x, const float* ybar, const MlpW& w, float eps,
                                   float* gin, float* streams, const Partials& part, int* nblocks, hipStream_t s);
hipError_t launch_edge_enc_r32(int lat, int64_t E, const float* f, const MlpW& w, float eps, void* e_out,
                               hipStream_t s);
hipError_t launch_edge_enc_bwd_r32(int lat, int64_t E, const float* f, const void* ebar, const MlpW& w, float eps,
                                   const Partials& part, int* nblocks, hipStream_t s);
// bf16 edge forward with one wave per tile (uses MlpW::W1p / W2p); a1_out
// (nullable) receives the first-layer activations of every edge.
hipError_t launch_edge_fwd_rows(const EdgeTiles& t, const void* e_in, void* e_out, int write_e, const void* P,
                                const MlpW& w, float eps, float* agg, float* slots, void* a1_out, hipStream_t s);
// fp32 edge forward with one wave per 16-row half of a tile at width lat
// (128 or 160; uses MlpW::F1 / F2, the fragment-major W1e and W2, and the
// fp32 vectors): e_out = e_in + m (write_e), agg / slots = receiver sums of m.
hipError_t launch_edge_fwd_r32(int lat, const EdgeTiles& t, const void* e_in, void* e_out, int write_e,
                               const void* Pn, const MlpW& w, float eps, float* agg, float* slots, hipStream_t s);
// fp32 edge backward at width 128 with its weight gradients in one pass (one
// wave per row block, four waves per block in lockstep rounds; recomputes
// the first layer from e and P; uses MlpW::F1, F2, F1t, F2t): writes zbar,
// R / slots, ebar_out (in place allowed) and per-block partials dW1e (0),
// db1 (16384), dW2 (16512), db2 (32896), dgamma (33024), dbeta (33152).
hipError_t launch_edge_bwd_r32(int lat, const EdgeTiles& t, const void* e, const float* ebar_in, int have_ebar,
                               float* ebar_out, const void* Pn, const float* aggbar, const MlpW& w, float eps,
                               void* zbar, float* R, float* slots, const Partials& part, int* nblocks,
                               hipStream_t s);
// bf16 edge backward with its weight gradients in one pass (four waves per
// block in lockstep rounds): from the saved a1, the block's input edge
// latents e and ebar_in (in place allowed), writes zbar, R / slots,
// ebar_out and per-block partials dW1e (0), db1 (16384), dW2 (16512), db2
// (32896), dgamma (33024), dbeta (33152).
hipError_t launch_edge_bwd_fused(const EdgeTiles& t, const void* a1, const void* e, const void* ebar_in,
                                 int have_ebar, void* ebar_out, const float* aggbar, const MlpW& w, float eps,
                                 void* zbar, float* R, float* slots, const Partials& part, int* nblocks,
                                 hipStream_t s);
// bf16 edge forward at width 160 (latent 150) with one wave per 16-row half of
// a tile (uses MlpW::W1p, W2p and the fp32 vectors); a1_out (nullable)
// receives the first-layer activations.
hipError_t launch_edge_fwd_w160(const EdgeTiles& t, const void* e_in, void* e_out, int write_e, const void* Pn,
                                const MlpW& w, float eps, float* agg, float* slots, void* a1_out, hipStream_t s);
// bf16 edge backward at width 160 (latent 150) with one wave per 16-row half
// of a tile, from the saved a1 (uses MlpW::W1p, W2p, b2, gamma); bf16
// edge-gradient stream (in place allowed); writes zbar, dz2, R / slots and
// per-block partials [db1 | db2 | dgamma | dbeta] (4 x 160 floats).
hipError_t launch_edge_bwd_w160(const EdgeTiles& t, const void* a1, const void* ebar_in, int have_ebar,
                                void* ebar_out, const float* aggbar, const MlpW& w, float eps, void* zbar, void* dz,
                                float* R, float* slots, const Partials& part, int* nblocks, hipStream_t s);
// Width 160 (bf16): dW1e = sum zbar^T e at 0 and dW2 = sum dz2^T a1 at
// 160 * 160 as per-block partials.
hipError_t launch_wgrad2_w160(int64_t M, const void* zbar, const void* e, const void* dz, const void* a1,
                              const Partials& part, int* nblocks, hipStream_t s);
// bf16 node phase with one wave per 16-node block (uses MlpW::W1p / W2p of
// the node MLP): h_out = h_in + LN(MLP([h_in, agg])), h_out may alias h_in.
hipError_t launch_node_fwd_rows(int64_t N, const float* h_in, const float* agg, const MlpW& w, float eps,
                                float* h_out, hipStream_t s);
// bf16 node products P = [W1s h; W1r h] of the next edge layer (W1sp / W1rp).
hipError_t launch_emit_rows(int64_t N, const float* h, const MlpW& next_edge, void* P, hipStream_t s);
// bf16 node backward: hbar_part, aggbar, the bf16 streams a1, dz2, dz1 and
// per-block partials of dgamma, dbeta (node-MLP partial layout).
hipError_t launch_node_bwd_rows(int64_t N, const float* h, const float* agg, const float* hbar_in, const MlpW& w,
                                float eps, float* hbar_part, float* aggbar, void* a1, void* dz2, void* dz1,
                                const Partials& part, int* nblocks, hipStream_t s);
// bf16 node-MLP weight gradients dW1, db1, dW2, db2 from those streams.
hipError_t launch_wgrad_node(int64_t N, const float* h, const float* agg, const void* dz1, const void* dz2,
                             const void* a1, const Partials& part, int* nblocks, hipStream_t s);
// bf16 node phase reverse at width 160 (latent 150): the node backward
// writes the a1 / dz2 / dz1 streams and the dgamma / dbeta partials, the
// weight-gradient pass (two launches on one grid) the other partials.
hipError_t launch_node_bwd_w160(int64_t N, const float* h, const float* agg, const float* hbar_in, const MlpW& w,
                                float eps, float* hbar_part, float* aggbar, void* a1, void* dz2, void* dz1,
                                const Partials& part, int* nblocks, hipStream_t s);
hipError_t launch_wgrad_node_w160(int64_t N, const float* h, const float* agg, const void* dz1, const void* dz2,
                                  const void* a1, const Partials& part, int* nblocks, hipStream_t s);
// bf16 node phase forward at width 160: h_out (may alias h_in), and the
// next edge layer's node products P (uses its MlpW::W1sp / W1rp).
hipError_t launch_node_fwd_w160(int64_t N, const float* h_in, const float* agg, const MlpW& w, float eps,
                                float* h_out, hipStream_t s);
hipError_t launch_emit_w160(int64_t N, const float* h, const MlpW& next_edge, void* P, hipStream_t s);
// bf16 per-sender sums at width 160: hbar_out = hbar_part + W1s^T S + W1r^T
// R and per-block partials of dW1s (at 0) and dW1r (at 160^2); S_buf: N x
// 160 bf16 scratch for S.
hipError_t launch_srcsum_w160(int64_t N, const int32_t* rowptr, const int32_t* rev, const void* zbar, const float* R,
                              const float* h, const float* hbar_part, const MlpW& w, float* hbar_out, void* S_buf,
                              const Partials& part, int* nblocks, hipStream_t s);
// bf16 edge encoder in the row layout (uses MlpW::W2p and the fp32 W1f).
hipError_t launch_edge_enc_rows(int64_t E, const float* efeat, const MlpW& w, float eps, void* e_out, hipStream_t s);
// bf16 edge-encoder backward from the bf16 edge-gradient stream: per-block
// partials of every encoder parameter (encoder parameter order).
hipError_t launch_edge_enc_bwd_rows(int64_t E, const float* efeat, const void* ebar, const MlpW& w, float eps,
                                    const Partials& part, int* nblocks, hipStream_t s);
// bf16 edge encoder at width 160 (latent 150) in the row layout of the
// width-160 edge kernels (uses MlpW::W2p and the fp32 W1f); the backward
// writes per-block partials of all encoder parameters.
hipError_t launch_edge_enc_w160(int64_t E, const float* efeat, const MlpW& w, float eps, void* e_out, hipStream_t s);
hipError_t launch_edge_enc_bwd_w160(int64_t E, const float* efeat, const void* ebar, const MlpW& w, float eps,
                                    const Partials& part, int* nblocks, hipStream_t s);
hipError_t launch_node_enc_bwd_w160(int64_t N, const float* node_in, const float* hbar, const MlpW& w, float eps,
                                    float* gin, const Partials& part, int* nblocks, hipStream_t s);
hipError_t launch_slot_fixup(int lat, const int32_t* long_nodes, int64_t n_long, const float* slots, float* dst,
                             hipStream_t s);
hipError_t launch_decoder(int prec, int lat, int64_t N, const float* h, const MlpW& w, float* out, hipStream_t s);

hipError_t launch_decoder_bwd(int prec, int lat, int64_t N, const float* h, const float* gout, const MlpW& w,
                              float* hbar, const Partials& part, int* nblocks, hipStream_t s);
// dW[o][i] = sum_rows G[row][o] X[row][i] for fp32 [M][lat] streams (lat
// 128 or 160), in the fp32 row layout, written as per-block [lat][lat]
// partials.
hipError_t launch_wgrad_r32(int lat, int64_t M, const float* G, const float* X, const Partials& part, int* nblocks,
                            hipStream_t s);
hipError_t launch_node_srcsum(int prec, int lat, int64_t N, const int32_t* rowptr, const int32_t* rev, const void* zbar,
                              const float* R, const float* h, const float* hbar_part, const MlpW& w,
                              float* hbar_out, const Partials& part, int* nblocks, hipStream_t s);
hipError_t launch_node_enc_bwd(int prec, int lat, int64_t N, const float* node_in, const float* hbar, const MlpW& w,
                               float eps, float* gin, const Partials& part, int* nblocks, hipStream_t s);

// grad[dst + r*dst_ld + c] += sum_b part[b*stride + src + r*cols + c]
hipError_t launch_reduce(const Partials& part, int nblocks, int64_t src, int32_t rows, int32_t cols,
                         float* grad, int64_t dst, int64_t dst_ld, hipStream_t s);
// Several reductions of per-block partials in one launch (same per-entry sum
// order as launch_reduce, so the same results): job k sums rows x cols
// entries at src of region `region` (regions lie region_floats apart from
// part.buf) over its nblocks partial rows into grad[dst + r ld + c].
struct ReduceJob {
  int64_t src, dst, ld, blk0;  // blk0: first launch block of the job (set by the launcher)
  int32_t rows, cols, nblocks, region;
};
constexpr int kMaxReduceJobs = 8;
struct ReduceBatch {
  ReduceJob j[kMaxReduceJobs];
  int32_t n;
};
hipError_t launch_reduce_batch(const Partials& part, int64_t region_floats, ReduceBatch b, float* grad,
                               hipStream_t s);

// out[v][c] = c0 * x0[v][c] + sum_j cj * xj[v][ldx_j*v + off_j + c], c < 4
struct LinComb {
  const float* x[6];
  int32_t ld[6];
  int32_t off[6];
  float c[6];
  int32_t n;
};
hipError_t launch_lincomb(int64_t N, const LinComb& lc, float* out, int32_t out_ld, int32_t out_off,
                          hipStream_t s);
// Block moves between parameter layouts: for every block,
// b[b_off + r*b_ld + c] = a[a_off + r*a_ld + c] (or += with accumulate),
// r < rows, c < cols.
struct CopyBlock {
  int64_t a_off, b_off;
  int32_t rows, cols, a_ld, b_ld;
};
constexpr int kCopyMax = 64;
struct CopyList {
  CopyBlock b[kCopyMax];
  int32_t n;
};
hipError_t launch_copy_blocks(const CopyList& L, const float* a, float* b, int accumulate, hipStream_t s);
// p[0..n) = v
hipError_t launch_fill(float* p, int64_t n, float v, hipStream_t s);
// b += a over n values of an edge-latent stream in precision prec (n a
// multiple of 8; bf16 values added in fp32 and rounded to nearest even)
hipError_t launch_add_stream(int prec, int64_t n, const void* a, void* b, hipStream_t s);
// Training step: partial rows of the loss sum; noisy gather dst[r] =
// y[idx[r]] + sd * noise[idx[r]] (noise nullable); masked squared error of
// pred against target[idx[r]] over mask rows: gradient 2 d inv, loss +=
// inv sum d^2 (fixed order); fused Adam update.
int loss_blocks();
hipError_t launch_gather_noisy(int64_t n, const float* y, const float* noise, const float* sd, const int32_t* idx,
                               int64_t n_src, float* dst, hipStream_t s);
hipError_t launch_mse(int64_t n, const float* pred, const float* target, const int32_t* idx, const uint8_t* mask,
                      int64_t n_src, float inv, float* gout, float* part, float* loss, hipStream_t s);
hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v, float lr, float b1, float omb1, float b2,
                       float omb2, float eps, float bc1, float bc2, hipStream_t s);
// dst[r][0..4) = src[idx[r]][0..4) for r < n (idx clamped into [0, n_src))
hipError_t launch_gather_rows4(int64_t n, const float* src, const int32_t* idx, int64_t n_src, float* dst,
                               hipStream_t s);
// dst[idx[r]][0..4) = src[r][0..4) for r < n with mask[r] != 0 (idx clamped)
hipError_t launch_scatter_rows4(int64_t n, const float* src, const int32_t* idx, const uint8_t* mask, int64_t n_dst,
                                float* dst, hipStream_t s);
// node_in[v] = [static[v][0..4), y-combination[v][0..4)]
hipError_t launch_stage_input(int64_t N, const float* st, const LinComb& lc, float* node_in, hipStream_t s);

}  // namespace mgn
