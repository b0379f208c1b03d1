// C-ABI entry points for device execution: context and workspace planning,
// one MGN call (Sec. 2.1), its reverse mode (with the gradient accumulation
// of Sec. 2.2, condition 3) and explicit integration steps (Sec. 2.1, 2.3,
// App. A).  All device memory is the caller's workspace; every launch goes
// to the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "internal.hpp"
#include "launch.hpp"

namespace mgn {

namespace {

constexpr int kPartBlocks = 512;  // persistent blocks of the backward kernels
// Partial regions: the backward kernels of one MP block write their
// per-block partials to distinct regions, reduced together after the block.
constexpr int kPartRegions = 5;
// Largest per-block partial at kernel width LD: the node MLP's parameters,
// W1 [LD][2 LD], b1, W2 [LD][LD], b2, gamma, beta.
inline int64_t part_stride(int LD) { return 3LL * LD * LD + 4LL * LD; }
// Offset of dgamma in the node MLP's parameters (and per-block partials):
// W1 [D][2D], b1, W2 [D][D], b2 precede it.
constexpr int64_t node_gamma_part(int D) { return (int64_t)3 * D * D + 2 * D; }
// the row-layout (bf16) kernels' fixed latent width
constexpr int kRowsD = 128;

struct Off {
  int64_t W1 = 0, b1 = 0, W2 = 0, b2 = 0, g = -1, bt = -1, size = 0;
};

struct PackOff {
  int64_t W1 = -1, W1t = -1, W2 = -1, W2t = -1, W1p = -1, W2p = -1;
  int64_t F1 = -1, F2 = -1, F1t = -1, F2t = -1;  // fp32 edge MLPs (encoder: W2): fragment-major W1e, W2, transposes
  int64_t W1sp = -1, W1rp = -1;  // edge MLPs: row-permuted sender / receiver column blocks of W1
  int64_t W1ap = -1;             // node MLPs at width 160: row-permuted agg column block of W1
  // fp32 row-layout node kernels: node MLPs' W1 agg block (F1: its h block),
  // edge MLPs' W1 sender and receiver blocks, fragment-major and transposed
  int64_t F1a = -1, F1at = -1, F1s = -1, F1r = -1, F1st = -1, F1rt = -1;
};

struct Model {
  int m = 0, lat = 0;  // MP steps, latent width
  Off enc_node, enc_edge, dec;
  std::vector<Off> edge, node;
  int64_t total = 0;
  PackOff p_enc_node, p_enc_edge, p_dec;
  std::vector<PackOff> p_edge, p_node;
  int64_t pack_elems = 0;
  std::vector<PackEnt> ents;
};

// Two-layer MLP din -> hid -> dout, parameters in the order W1 [hid][din],
// b1, W2 [dout][hid], b2, then gamma, beta when it ends in a LayerNorm.
Off mlp_off(int64_t& o, int din, int hid, int dout, bool ln) {
  Off r;
  r.W1 = o;
  o += (int64_t)hid * din;
  r.b1 = o;
  o += hid;
  r.W2 = o;
  o += (int64_t)dout * hid;
  r.b2 = o;
  o += dout;
  if (ln) {
    r.g = o;
    o += dout;
    r.bt = o;
    o += dout;
  }
  r.size = o - r.W1;
  return r;
}

void add_pack(Model& M, int64_t src, int rows, int cols, int64_t& W, int64_t& Wt) {
  auto al = [](int64_t x) { return (x + 63) & ~int64_t(63); };
  M.pack_elems = al(M.pack_elems);
  W = M.pack_elems;
  M.pack_elems = al(M.pack_elems + (int64_t)rows * cols);
  Wt = M.pack_elems;
  M.pack_elems += (int64_t)rows * cols;
  PackEnt e;
  e.src = src;
  e.dst = W;
  e.dstt = Wt;
  e.rows = rows;
  e.cols = cols;
  e.ld = cols;
  e.perm = 0;
  M.ents.push_back(e);
}

// Row-permuted copy (perm_row) of `cols` columns of a [rows][ld] matrix
// starting at float offset src.
void add_perm(Model& M, int64_t src, int ld, int64_t& W, int cols = kRowsD, int rows = kRowsD) {
  auto al = [](int64_t x) { return (x + 63) & ~int64_t(63); };
  M.pack_elems = al(M.pack_elems);
  W = M.pack_elems;
  M.pack_elems += (int64_t)rows * cols;
  PackEnt e;
  e.src = src;
  e.dst = W;
  e.dstt = -1;
  e.rows = rows;
  e.cols = cols;
  e.ld = ld;
  e.perm = 1;
  M.ents.push_back(e);
}

// Fragment-major fp32 copy (mode 2) or copy of the transpose (mode 3) of
// the square [n][n] block at float offset src (row stride ld).
void add_frag(Model& M, int64_t src, int ld, int n, int mode, int64_t& W) {
  auto al = [](int64_t x) { return (x + 63) & ~int64_t(63); };
  M.pack_elems = al(M.pack_elems);
  W = M.pack_elems;
  M.pack_elems += (int64_t)n * n;
  PackEnt e;
  e.src = src;
  e.dst = W;
  e.dstt = -1;
  e.rows = n;
  e.cols = n;
  e.ld = ld;
  e.perm = mode;
  M.ents.push_back(e);
}

// Parameter layout and packed operand copies of an MGN with m MP steps and
// latent width lat (both MLP layers of every block are lat wide); fp32
// models also carry the fragment-major edge-MLP copies of the fp32
// row-layout edge kernels.
Model make_model(int m, int lat, bool fp32 = false) {
  const int D = lat;
  Model M;
  M.m = m;
  M.lat = lat;
  int64_t o = 0;
  M.enc_node = mlp_off(o, 8, D, D, true);
  M.enc_edge = mlp_off(o, 4, D, D, true);
  for (int i = 0; i < m; ++i) {
    M.edge.push_back(mlp_off(o, 3 * D, D, D, true));
    M.node.push_back(mlp_off(o, 2 * D, D, D, true));
  }
  M.dec = mlp_off(o, D, D, 4, false);
  M.total = o;
  const bool rows = lat == kRowsD;  // row-permuted copies for the row-layout kernels
  add_pack(M, M.enc_node.W2, D, D, M.p_enc_node.W2, M.p_enc_node.W2t);
  if (!rows) add_perm(M, M.enc_node.W2, D, M.p_enc_node.W2p, D, D);  // width-160 node encoder backward
  add_pack(M, M.enc_edge.W2, D, D, M.p_enc_edge.W2, M.p_enc_edge.W2t);
  add_perm(M, M.enc_edge.W2, D, M.p_enc_edge.W2p, D, D);  // row-layout edge encoders
  if (fp32) {
    // fp32 row-layout encoders: fragment-major W2 and its transpose
    add_frag(M, M.enc_edge.W2, D, D, 2, M.p_enc_edge.F2);
    add_frag(M, M.enc_edge.W2, D, D, 3, M.p_enc_edge.F2t);
    add_frag(M, M.enc_node.W2, D, D, 2, M.p_enc_node.F2);
    add_frag(M, M.enc_node.W2, D, D, 3, M.p_enc_node.F2t);
  }
  M.p_edge.resize(m);
  M.p_node.resize(m);
  for (int i = 0; i < m; ++i) {
    add_pack(M, M.edge[i].W1, D, 3 * D, M.p_edge[i].W1, M.p_edge[i].W1t);
    add_pack(M, M.edge[i].W2, D, D, M.p_edge[i].W2, M.p_edge[i].W2t);
    if (rows) {
      add_perm(M, M.edge[i].W1, 3 * D, M.p_edge[i].W1p);
      add_perm(M, M.edge[i].W2, D, M.p_edge[i].W2p);
      add_perm(M, M.edge[i].W1 + D, 3 * D, M.p_edge[i].W1sp);
      add_perm(M, M.edge[i].W1 + 2 * D, 3 * D, M.p_edge[i].W1rp);
      add_perm(M, M.node[i].W1, 2 * D, M.p_node[i].W1p, 2 * D);
      add_perm(M, M.node[i].W2, D, M.p_node[i].W2p);
    } else {
      // width 160 (bf16 row-per-wave edge kernels): W1's edge-latent block
      // and W2, rows in perm_row order
      add_perm(M, M.edge[i].W1, 3 * D, M.p_edge[i].W1p, D, D);
      add_perm(M, M.edge[i].W2, D, M.p_edge[i].W2p, D, D);
      add_perm(M, M.edge[i].W1 + D, 3 * D, M.p_edge[i].W1sp, D, D);
      add_perm(M, M.edge[i].W1 + 2 * D, 3 * D, M.p_edge[i].W1rp, D, D);
      // node MLP: W1's h and agg column blocks and W2
      add_perm(M, M.node[i].W1, 2 * D, M.p_node[i].W1p, D, D);
      add_perm(M, M.node[i].W1 + D, 2 * D, M.p_node[i].W1ap, D, D);
      add_perm(M, M.node[i].W2, D, M.p_node[i].W2p, D, D);
    }
    add_pack(M, M.node[i].W1, D, 2 * D, M.p_node[i].W1, M.p_node[i].W1t);
    add_pack(M, M.node[i].W2, D, D, M.p_node[i].W2, M.p_node[i].W2t);
    if (fp32) {
      add_frag(M, M.edge[i].W1, 3 * D, D, 2, M.p_edge[i].F1);
      add_frag(M, M.edge[i].W2, D, D, 2, M.p_edge[i].F2);
      add_frag(M, M.edge[i].W1, 3 * D, D, 3, M.p_edge[i].F1t);
      add_frag(M, M.edge[i].W2, D, D, 3, M.p_edge[i].F2t);
      add_frag(M, M.edge[i].W1 + D, 3 * D, D, 2, M.p_edge[i].F1s);
      add_frag(M, M.edge[i].W1 + 2 * D, 3 * D, D, 2, M.p_edge[i].F1r);
      add_frag(M, M.edge[i].W1 + D, 3 * D, D, 3, M.p_edge[i].F1st);
      add_frag(M, M.edge[i].W1 + 2 * D, 3 * D, D, 3, M.p_edge[i].F1rt);
      add_frag(M, M.node[i].W1, 2 * D, D, 2, M.p_node[i].F1);
      add_frag(M, M.node[i].W1 + D, 2 * D, D, 2, M.p_node[i].F1a);
      add_frag(M, M.node[i].W2, D, D, 2, M.p_node[i].F2);
      add_frag(M, M.node[i].W1, 2 * D, D, 3, M.p_node[i].F1t);
      add_frag(M, M.node[i].W1 + D, 2 * D, D, 3, M.p_node[i].F1at);
      add_frag(M, M.node[i].W2, D, D, 3, M.p_node[i].F2t);
    }
  }
  add_pack(M, M.dec.W1, D, D, M.p_dec.W1, M.p_dec.W1t);
  if (fp32) {
    // fp32 row-layout decoder: fragment-major W1 and its transpose
    add_frag(M, M.dec.W1, D, D, 2, M.p_dec.F1);
    add_frag(M, M.dec.W1, D, D, 3, M.p_dec.F1t);
  }
  return M;
}

// Blocks that move the parameters of the real model R (latent dr) to the
// zero-padded kernel model K (width LD): per MLP, W1 by input-column block
// (node / edge input blocks of width 8 / 4 unpadded, latent blocks dr -> LD),
// then b1, W2, b2 and the LayerNorm gain and offset.  a = R, b = K.
std::vector<CopyBlock> pad_blocks(const Model& R, const Model& K) {
  std::vector<CopyBlock> v;
  const int dr = R.lat, LD = K.lat;
  auto mlp = [&](const Off& r, const Off& k, int nin, int win_r, int win_k, int dout_r, int dout_k, bool ln) {
    const int din_r = nin * win_r, din_k = nin * win_k;
    for (int j = 0; j < nin; ++j) v.push_back({r.W1 + (int64_t)j * win_r, k.W1 + (int64_t)j * win_k, dr, win_r, din_r, din_k});
    v.push_back({r.b1, k.b1, 1, dr, dr, LD});
    v.push_back({r.W2, k.W2, dout_r, dr, dr, LD});
    v.push_back({r.b2, k.b2, 1, dout_r, dout_r, dout_k});
    if (ln) {
      v.push_back({r.g, k.g, 1, dout_r, dout_r, dout_k});
      v.push_back({r.bt, k.bt, 1, dout_r, dout_r, dout_k});
    }
  };
  mlp(R.enc_node, K.enc_node, 1, 8, 8, dr, LD, true);
  mlp(R.enc_edge, K.enc_edge, 1, 4, 4, dr, LD, true);
  for (int i = 0; i < R.m; ++i) {
    mlp(R.edge[i], K.edge[i], 3, dr, LD, dr, LD, true);
    mlp(R.node[i], K.node[i], 2, dr, LD, dr, LD, true);
  }
  mlp(R.dec, K.dec, 1, dr, LD, 4, 4, false);
  return v;
}

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
  size_t pack = 0;
  size_t ppad = 0, gpad = 0;  // latent 150: padded parameter and gradient copies
  // activation sets
  size_t act = 0, act_stride = 0;
  size_t e_off = 0, h_off = 0, agg_off = 0, P_off = 0, a1_off = 0;  // within a set
  size_t e0 = 0;  // without saving, several stages: the shared edge-encoder output
  size_t node_in = 0, K = 0, slots = 0;
  // backward
  size_t pio = 0, lossp = 0, pcopy = 0;
  size_t ebar = 0, ebar_st = 0, zbar = 0, dz = 0, nstr = 0, hb_a = 0, hb_b = 0, aggbar = 0, R = 0, part = 0, kbar = 0, ystage = 0, gin = 0;
  size_t total = 0;
};

}  // namespace

enum Kern {
  K_PACK, K_NODE_ENC, K_EDGE_ENC, K_EDGE_FWD, K_FIXUP, K_NODE_FWD, K_DECODER, K_DECODER_BWD, K_NODE_BWD,
  K_EDGE_BWD, K_SRCSUM, K_EDGE_ENC_BWD, K_NODE_ENC_BWD, K_REDUCE, K_LINCOMB, K_WGRAD, K_EMIT, K_WGRAD_NODE, K_COUNT
};
const char* const kKernName[K_COUNT] = {
    "pack", "node_enc", "edge_enc", "edge_fwd", "slot_fixup", "node_fwd", "decoder", "decoder_bwd", "node_bwd",
    "edge_bwd", "node_srcsum", "edge_enc_bwd", "node_enc_bwd", "reduce", "lincomb", "wgrad", "emit_p", "wgrad_node"};

struct Prof {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<int> kind;  // per event pair
};

struct Ctx {
  mgn_config cfg;
  int64_t maxN = 0, maxE = 0;
  int32_t max_stages = 1, save = 0;
  int se = 4;  // bytes per element of the edge-latent stream
  int ne_sets = 1;
  // latent widths: DR the model's (128 or 150), LD the kernels' (128 or 160)
  int DR = 128, LD = 128;
  Model M;   // kernel-width model (parameters as the kernels see them)
  Model Mr;  // the caller's parameter layout (same as M when DR == LD)
  std::vector<CopyBlock> pad;  // Mr -> M moves when DR != LD
  Layout L;
  // saved state of the last call with save != 0
  int saved = 0;  // 0 none, 1 forward, 2 integration step
  int32_t scheme = 0, stages = 0;
  mgn_dgraph g{};
  const float* params = nullptr;
  const float* efeat = nullptr;
  const float* node_in = nullptr;
  char* ws = nullptr;
  Prof prof;
  ~Ctx() {
    for (hipEvent_t e : prof.pool) (void)hipEventDestroy(e);
  }
};

namespace {

struct Tableau {
  int s;
  float a[4][4];
  float b[4];
};

bool tableau(int32_t scheme, Tableau& t) {
  std::memset(&t, 0, sizeof(t));
  switch (scheme) {
    case MGN_EULER:
      t.s = 1;
      t.b[0] = 1.f;
      return true;
    case MGN_HEUN2:
      t.s = 2;
      t.a[1][0] = 1.f;
      t.b[0] = 0.5f;
      t.b[1] = 0.5f;
      return true;
    case MGN_MIDPOINT:
      t.s = 2;
      t.a[1][0] = 0.5f;
      t.b[1] = 1.f;
      return true;
    case MGN_HEUN3:
      t.s = 3;
      t.a[1][0] = 1.f / 3.f;
      t.a[2][1] = 2.f / 3.f;
      t.b[0] = 0.25f;
      t.b[2] = 0.75f;
      return true;
    case MGN_RALSTON2:
      t.s = 2;
      t.a[1][0] = 2.f / 3.f;
      t.b[0] = 0.25f;
      t.b[1] = 0.75f;
      return true;
    case MGN_RALSTON3:
      t.s = 3;
      t.a[1][0] = 0.5f;
      t.a[2][1] = 0.75f;
      t.b[0] = 2.f / 9.f;
      t.b[1] = 1.f / 3.f;
      t.b[2] = 4.f / 9.f;
      return true;
    case MGN_RK4:
      t.s = 4;
      t.a[1][0] = 0.5f;
      t.a[2][1] = 0.5f;
      t.a[3][2] = 1.f;
      t.b[0] = 1.f / 6.f;
      t.b[1] = 1.f / 3.f;
      t.b[2] = 1.f / 3.f;
      t.b[3] = 1.f / 6.f;
      return true;
  }
  return false;
}

void plan(Ctx& c) {
  const int64_t N = c.maxN, E = c.maxE;
  const int m = c.cfg.mp_steps;
  const int D = c.LD;
  const size_t tsz = c.cfg.precision == MGN_BF16 ? 2 : 4;
  Layout& L = c.L;
  size_t o = 0;
  L.pack = o;
  o = al256(o + (size_t)c.M.pack_elems * tsz);
  if (c.LD != c.DR) {
    L.ppad = o;  // the zero-padded copy of the parameters every call computes from
    o = al256(o + (size_t)c.M.total * 4);
  }
  const int le = c.save ? std::max(m, 1) : 1;
  const int lh = c.save ? m + 1 : 1;
  const int la = c.save ? std::max(m, 1) : 1;
  size_t so = 0;
  L.e_off = so;
  so = al256(so + (size_t)le * E * D * c.se);
  L.h_off = so;
  so = al256(so + (size_t)lh * N * D * 4);
  L.agg_off = so;
  so = al256(so + (size_t)la * N * D * 4);
  L.P_off = so;
  so = al256(so + (size_t)la * N * 2 * D * tsz);
  // bf16 with save: first-layer activations of every edge MLP, read by the
  // backward instead of recomputing the first layer
  // bf16 at width 128 runs on the row-layout kernels; every other case on
  // the feature-split ones, except the bf16 edge backward at width 160 (one
  // wave per row block, like the row layout)
  const bool bf = c.cfg.precision == MGN_BF16;
  const bool rows = bf && c.LD == kRowsD;
  const bool keep_a1 = c.save && bf;
  L.a1_off = so;
  so = al256(so + (keep_a1 ? (size_t)la * E * D * 2 : 0));
  L.act_stride = so;
  L.act = o;
  o = al256(o + so * c.ne_sets);
  if (!c.save && c.max_stages > 1) {
    // the stages of a non-saving step share one edge-encoder output; the
    // processor updates its own edge buffer in place, so this one stays
    L.e0 = o;
    o = al256(o + (size_t)E * D * c.se);
  }
  L.node_in = o;
  o = al256(o + (size_t)c.max_stages * N * 8 * 4);
  L.K = o;
  o = al256(o + (size_t)c.max_stages * N * 4 * 4);
  L.pio = o;  // patch steps: a patch's static, y, y_next and loss-gradient rows
  o = al256(o + (size_t)4 * N * 4 * 4);
  L.lossp = o;  // training step: partial sums of the loss
  o = al256(o + (size_t)loss_blocks() * 4);
  L.slots = o;
  o = al256(o + (size_t)max_slots(E) * D * 4);
  if (c.save) {
    L.pcopy = o;  // a saving call's own copy of the parameters (the padded copy serves at latent 150)
    o = al256(o + (c.LD == c.DR ? (size_t)c.M.total * 4 : 0));
    if (c.LD != c.DR) {
      L.gpad = o;  // gradients in the padded layout, moved to the caller's layout at the end
      o = al256(o + (size_t)c.M.total * 4);
    }
    L.ebar = o;  // edge-gradient stream, in the edge-latent element type
    o = al256(o + (size_t)E * D * c.se);
    // several stages: the encoder output's gradient summed over the stages
    // (the stages share one edge-encoder output; see Run::backward)
    L.ebar_st = o;
    o = al256(o + (c.max_stages > 1 ? (size_t)E * D * c.se : 0));
    L.zbar = o;
    o = al256(o + (size_t)E * D * c.se);
    L.dz = o;  // dz2 of the width-160 edge backward (the 128-wide one keeps it on chip)
    o = al256(o + (keep_a1 && !rows ? (size_t)E * D * 2 : 0));
    // node backward: the a1, dz2, dz1 streams of one node MLP (bf16 / fp32)
    L.nstr = o;
    o = al256(o + (size_t)3 * N * D * (bf ? 2 : 4));
    L.hb_a = o;
    o = al256(o + (size_t)N * D * 4);
    L.hb_b = o;
    o = al256(o + (size_t)N * D * 4);
    L.aggbar = o;
    o = al256(o + (size_t)N * D * 4);
    L.R = o;
    o = al256(o + (size_t)N * D * 4);
    L.part = o;
    o = al256(o + (size_t)kPartRegions * kPartBlocks * part_stride(D) * 4);
    L.kbar = o;
    o = al256(o + (size_t)N * 4 * 4);
    L.ystage = o;
    o = al256(o + (size_t)c.max_stages * N * 4 * 4);
    L.gin = o;
    o = al256(o + (size_t)N * 8 * 4);
  }
  L.total = o;
}

inline hipStream_t S(void* s) { return (hipStream_t)s; }

#define LAUNCH(kind, expr)         \
  do {                             \
    HIP_TRY(mark_begin(kind));     \
    HIP_TRY(expr);                 \
    HIP_TRY(mark_end());           \
  } while (0)

#define HIP_TRY(expr)                                                                 \
  do {                                                                                \
    hipError_t _e = (expr);                                                           \
    if (_e != hipSuccess) return fail(MGN_ERR_DEVICE, "%s: %s", #expr, hipGetErrorString(_e)); \
  } while (0)

struct Run {
  Ctx& c;
  const mgn_dgraph& g;
  const float* params;
  char* ws;
  hipStream_t s;
  int64_t N, E;
  int m;
  int prec;
  float eps;
  bool keep_a1 = false;  // this call saves (or the backward reads) the edge MLPs' a1
  // stages of the saved integration step: they share the first stage's
  // edge-encoder output, and the reverse runs the encoder once on the sum of
  // the stages' gradients of it
  int n_st = 1;
  int D = c.LD;          // kernel latent width
  // bf16 at width 128 runs on the row-layout kernels
  bool rows() const { return prec == MGN_BF16 && D == kRowsD; }

  // Bracket a launch with profiling events when enabled.
  hipError_t mark_begin(int kind) {
    Prof& p = c.prof;
    if (!p.on) return hipSuccess;
    while (p.pool.size() < p.used + 2) {
      hipEvent_t e;
      hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) return r;
      p.pool.push_back(e);
    }
    p.kind.push_back(kind);
    return hipEventRecord(p.pool[p.used++], s);
  }
  hipError_t mark_end() {
    Prof& p = c.prof;
    if (!p.on) return hipSuccess;
    return hipEventRecord(p.pool[p.used++], s);
  }

  char* pack() const { return ws + c.L.pack; }
  size_t tsz() const { return prec == MGN_BF16 ? 2 : 4; }
  const void* P(int64_t off) const { return pack() + (size_t)off * tsz(); }
  char* set(int k) const { return ws + c.L.act + (size_t)k * c.L.act_stride; }
  // With saving, stage k > 0 reads the first stage's encoder output: the
  // encoder's inputs (edge features, parameters) are the same in every stage.
  void* e_l(int k, int l) const {
    if (!c.save) return set(k) + c.L.e_off;
    return set(l == 0 ? 0 : k) + c.L.e_off + (size_t)l * E * D * c.se;
  }
  // The edge-encoder output of a call, read by its first processor block in
  // every stage: with saving the first stage's (no block overwrites it);
  // without saving, when several stages are planned, a buffer of its own
  // (the processor updates its edge buffer in place); else the edge buffer.
  bool shared_e0() const { return c.save || c.max_stages > 1; }
  void* e_enc() const { return !c.save && c.max_stages > 1 ? ws + c.L.e0 : e_l(0, 0); }
  float* h_l(int k, int l) const {
    return (float*)(set(k) + c.L.h_off) + (c.save ? (size_t)l * N * D : 0);
  }
  float* agg_l(int k, int l) const {
    return (float*)(set(k) + c.L.agg_off) + (c.save ? (size_t)l * N * D : 0);
  }
  void* a1_l(int k, int l) const {
    if (!(keep_a1 && c.save && prec == MGN_BF16)) return nullptr;
    return set(k) + c.L.a1_off + (size_t)l * E * D * 2;
  }
  void* P_l(int k, int l) const {
    return set(k) + c.L.P_off + (c.save ? (size_t)l * N * 2 * D * tsz() : 0);
  }
  float* slots() const { return (float*)(ws + c.L.slots); }

  MlpW W(const Off& o, const PackOff& p) const {
    MlpW w;
    w.W1p = p.W1p >= 0 ? P(p.W1p) : nullptr;
    w.W2p = p.W2p >= 0 ? P(p.W2p) : nullptr;
    w.W1sp = p.W1sp >= 0 ? P(p.W1sp) : nullptr;
    w.W1rp = p.W1rp >= 0 ? P(p.W1rp) : nullptr;
    w.W1ap = p.W1ap >= 0 ? P(p.W1ap) : nullptr;
    w.W1 = p.W1 >= 0 ? P(p.W1) : nullptr;
    w.W1t = p.W1t >= 0 ? P(p.W1t) : nullptr;
    w.W2 = p.W2 >= 0 ? P(p.W2) : nullptr;
    w.W2t = p.W2t >= 0 ? P(p.W2t) : nullptr;
    w.F1 = p.F1 >= 0 ? (const float*)P(p.F1) : nullptr;
    w.F2 = p.F2 >= 0 ? (const float*)P(p.F2) : nullptr;
    w.F1t = p.F1t >= 0 ? (const float*)P(p.F1t) : nullptr;
    w.F2t = p.F2t >= 0 ? (const float*)P(p.F2t) : nullptr;
    w.F1a = p.F1a >= 0 ? (const float*)P(p.F1a) : nullptr;
    w.F1at = p.F1at >= 0 ? (const float*)P(p.F1at) : nullptr;
    w.F1s = p.F1s >= 0 ? (const float*)P(p.F1s) : nullptr;
    w.F1r = p.F1r >= 0 ? (const float*)P(p.F1r) : nullptr;
    w.F1st = p.F1st >= 0 ? (const float*)P(p.F1st) : nullptr;
    w.F1rt = p.F1rt >= 0 ? (const float*)P(p.F1rt) : nullptr;
    w.W1f = params + o.W1;
    w.W2f = params + o.W2;
    w.b1 = params + o.b1;
    w.b2 = params + o.b2;
    w.gamma = o.g >= 0 ? params + o.g : nullptr;
    w.beta = o.bt >= 0 ? params + o.bt : nullptr;
    return w;
  }
  EdgeTiles tiles() const {
    EdgeTiles t;
    t.tiles = g.tiles;
    t.n_tiles = g.n_tiles;
    t.rowptr = g.rowptr;
    t.senders = g.senders;
    t.receivers = g.receivers;
    t.n_edges = g.n_edges;
    return t;
  }
  Partials part() const {
    Partials p;
    p.buf = (float*)(ws + c.L.part);
    p.stride = part_stride(D);
    p.max_blocks = kPartBlocks;
    return p;
  }
  Partials partr(int r) const {
    Partials p = part();
    p.buf += (size_t)r * kPartBlocks * p.stride;
    return p;
  }

  int pack_weights() {
    const Model& M = c.M;
    for (size_t b = 0; b < M.ents.size(); b += kPackMax) {
      PackList L;
      L.n = (int32_t)std::min<size_t>(kPackMax, M.ents.size() - b);
      for (int j = 0; j < L.n; ++j) L.e[j] = M.ents[b + j];
      LAUNCH(K_PACK, launch_pack(prec, params, pack(), L, s));
    }
    return MGN_OK;
  }

  // k: the activation set (the stage with saving, else 0); stage: the stage
  // of the call (later stages reuse the edge-encoder output when it is kept)
  int forward(const float* node_in, const float* efeat, float* out, int k, int stage = 0) {
    const Model& M = c.M;
    const EdgeTiles tl = tiles();
    MlpW e0;
    if (m > 0) e0 = W(M.edge[0], M.p_edge[0]);
    if (prec == MGN_FP32)
      LAUNCH(K_NODE_ENC, launch_node_enc_r32(D, N, node_in, W(M.enc_node, M.p_enc_node), m > 0 ? &e0 : nullptr, eps,
                                             h_l(k, 0), m > 0 ? (float*)P_l(k, 0) : nullptr, s));
    else
      LAUNCH(K_NODE_ENC, launch_node_enc(prec, D, N, node_in, W(M.enc_node, M.p_enc_node), m > 0 ? &e0 : nullptr, eps,
                                         h_l(k, 0), P_l(k, 0), s));
    if (m > 0 && !(stage > 0 && shared_e0())) {
      if (rows())
        LAUNCH(K_EDGE_ENC, launch_edge_enc_rows(E, efeat, W(M.enc_edge, M.p_enc_edge), eps, e_enc(), s));
      else
        LAUNCH(K_EDGE_ENC, prec == MGN_FP32
                               ? launch_edge_enc_r32(D, E, efeat, W(M.enc_edge, M.p_enc_edge), eps, e_enc(), s)
                               : launch_edge_enc_w160(E, efeat, W(M.enc_edge, M.p_enc_edge), eps, e_enc(), s));
    }
    for (int l = 0; l < m; ++l) {
      const bool last = l == m - 1;
      const void* e_in = l == 0 ? e_enc() : e_l(k, l);
      void* e_out = c.save ? (last ? nullptr : e_l(k, l + 1)) : e_l(k, 0);
      if (E > 0 && prec == MGN_FP32)
        LAUNCH(K_EDGE_FWD, launch_edge_fwd_r32(D, tl, e_in, e_out, last ? 0 : 1, P_l(k, l),
                                               W(M.edge[l], M.p_edge[l]), eps, agg_l(k, l), slots(), s));
      else if (E > 0)
        LAUNCH(K_EDGE_FWD, rows() ? launch_edge_fwd_rows(tl, e_in, e_out, last ? 0 : 1, P_l(k, l),
                                                         W(M.edge[l], M.p_edge[l]), eps, agg_l(k, l), slots(),
                                                         a1_l(k, l), s)
                                  : launch_edge_fwd_w160(tl, e_in, e_out, last ? 0 : 1, P_l(k, l),
                                                         W(M.edge[l], M.p_edge[l]), eps, agg_l(k, l), slots(),
                                                         a1_l(k, l), s));
      else
        LAUNCH(K_EDGE_FWD, launch_fill(agg_l(k, l), N * D, 0.f, s));  // no edges: every aggregate is zero
      if (g.n_long > 0) LAUNCH(K_FIXUP, launch_slot_fixup(D, g.long_nodes, g.n_long, slots(), agg_l(k, l), s));
      MlpW nx;
      if (!last) nx = W(M.edge[l + 1], M.p_edge[l + 1]);
      if (rows()) {
        LAUNCH(K_NODE_FWD, launch_node_fwd_rows(N, h_l(k, l), agg_l(k, l), W(M.node[l], M.p_node[l]), eps, h_l(k, l + 1), s));
        if (!last) LAUNCH(K_EMIT, launch_emit_rows(N, h_l(k, l + 1), nx, P_l(k, l + 1), s));
      } else if (prec == MGN_BF16) {
        LAUNCH(K_NODE_FWD, launch_node_fwd_w160(N, h_l(k, l), agg_l(k, l), W(M.node[l], M.p_node[l]), eps, h_l(k, l + 1), s));
        if (!last) LAUNCH(K_EMIT, launch_emit_w160(N, h_l(k, l + 1), nx, P_l(k, l + 1), s));
      } else {
        LAUNCH(K_NODE_FWD, launch_node_fwd_r32(D, N, h_l(k, l), agg_l(k, l), W(M.node[l], M.p_node[l]),
                                               last ? nullptr : &nx, eps, h_l(k, l + 1),
                                               last ? nullptr : (float*)P_l(k, l + 1), s));
      }
    }
    LAUNCH(K_DECODER, prec == MGN_FP32 ? launch_decoder_r32(D, N, h_l(k, m), W(M.dec, M.p_dec), out, s)
                                       : launch_decoder(prec, D, N, h_l(k, m), W(M.dec, M.p_dec), out, s));
    return MGN_OK;
  }

  int reduce(int nb, int64_t src, int rows, int cols, float* grad, int64_t dst, int64_t ld) {
    LAUNCH(K_REDUCE, launch_reduce(part(), nb, src, rows, cols, grad, dst, ld, s));
    return MGN_OK;
  }
  // Queued reductions of partial region r (launched together by flush).
  ReduceBatch rq{};
  int flush(float* grad) {
    if (rq.n > 0) LAUNCH(K_REDUCE, launch_reduce_batch(part(), (int64_t)kPartBlocks * part_stride(D), rq, grad, s));
    rq.n = 0;
    return MGN_OK;
  }
  int job(int nb, int r, int64_t src, int rows, int cols, float* grad, int64_t dst, int64_t ld) {
    if (nb <= 0 || rows <= 0 || cols <= 0) return MGN_OK;
    int rc;
    if (rq.n == kMaxReduceJobs && (rc = flush(grad)) != MGN_OK) return rc;
    ReduceJob& j = rq.j[rq.n++];
    j.src = src;
    j.dst = dst;
    j.ld = ld;
    j.blk0 = 0;
    j.rows = rows;
    j.cols = cols;
    j.nblocks = nb;
    j.region = r;
    return MGN_OK;
  }

  int backward(int k, const float* node_in, const float* efeat, const float* gout, float* grad, float* gin) {
    const Model& M = c.M;
    const EdgeTiles tl = tiles();
    const Partials pt = part();
    const Partials P0 = partr(0), P1 = partr(1), P2 = partr(2), P3 = partr(3), P4 = partr(4);
    rq.n = 0;
    float* hb_cur = (float*)(ws + c.L.hb_a);
    float* hb_part = (float*)(ws + c.L.hb_b);
    float* aggbar = (float*)(ws + c.L.aggbar);
    float* R = (float*)(ws + c.L.R);
    // the edge-latent element type; the last stage of several keeps its
    // gradient of the shared encoder output in the stage-sum buffer
    void* ebar = ws + (n_st > 1 && k == n_st - 1 ? c.L.ebar_st : c.L.ebar);
    void* zbar = ws + c.L.zbar;
    int nb = 0, rc;
    if (prec == MGN_FP32) {
      // fp32: the row-layout reverse (db1, dW2, db2 as its partials), then
      // dW1 = sum dz1^T h from its dz1 rows (the node-stream scratch); each
      // reduction runs before the next launch reuses the partial region
      float* dz1 = (float*)(ws + c.L.nstr);
      LAUNCH(K_DECODER_BWD, launch_decoder_bwd_r32(D, N, h_l(k, m), gout, W(M.dec, M.p_dec), hb_cur, dz1, pt, &nb, s));
      if ((rc = reduce(nb, 0, 1, 5 * D + 4, grad, M.dec.b1, 0)) != MGN_OK) return rc;
      LAUNCH(K_DECODER_BWD, launch_wgrad_r32(D, N, dz1, h_l(k, m), pt, &nb, s));
      if ((rc = reduce(nb, 0, D, D, grad, M.dec.W1, D)) != MGN_OK) return rc;
    } else {
      LAUNCH(K_DECODER_BWD, launch_decoder_bwd(prec, D, N, h_l(k, m), gout, W(M.dec, M.p_dec), hb_cur, pt, &nb, s));
      if ((rc = reduce(nb, 0, 1, (int)M.dec.size, grad, M.dec.W1, 0)) != MGN_OK) return rc;
    }
    for (int l = m - 1; l >= 0; --l) {
      const Off& oe = M.edge[l];
      const Off& on = M.node[l];
      if (prec == MGN_BF16) {
        // one wave per 16-node unit, then the weight gradients from its
        // a1 / dz2 / dz1 streams
        char* ns = ws + c.L.nstr;
        void *na1 = ns, *ndz2 = ns + (size_t)N * D * 2, *ndz1 = ns + (size_t)2 * N * D * 2;
        const int64_t gpart = node_gamma_part(D);
        if (rows())
          LAUNCH(K_NODE_BWD, launch_node_bwd_rows(N, h_l(k, l), agg_l(k, l), hb_cur, W(on, M.p_node[l]), eps, hb_part,
                                                  aggbar, na1, ndz2, ndz1, P0, &nb, s));
        else
          LAUNCH(K_NODE_BWD, launch_node_bwd_w160(N, h_l(k, l), agg_l(k, l), hb_cur, W(on, M.p_node[l]), eps, hb_part,
                                                  aggbar, na1, ndz2, ndz1, P0, &nb, s));
        if ((rc = job(nb, 0, gpart, 1, 2 * D, grad, on.g, 0)) != MGN_OK) return rc;
        if (rows())
          LAUNCH(K_WGRAD_NODE, launch_wgrad_node(N, h_l(k, l), agg_l(k, l), ndz1, ndz2, na1, P1, &nb, s));
        else
          LAUNCH(K_WGRAD_NODE, launch_wgrad_node_w160(N, h_l(k, l), agg_l(k, l), ndz1, ndz2, na1, P1, &nb, s));
        if ((rc = job(nb, 1, 0, 1, (int)gpart, grad, on.W1, 0)) != MGN_OK) return rc;
      } else {
        // fp32: the row-layout reverse (db1, db2, dgamma, dbeta as its
        // partials), then the weight gradients from its a1 / dz2 / dz1
        // streams: dW1 by its h and agg column blocks, and dW2
        float* ns = (float*)(ws + c.L.nstr);
        const size_t nd = (size_t)N * D;
        LAUNCH(K_NODE_BWD, launch_node_bwd_r32(D, N, h_l(k, l), agg_l(k, l), hb_cur, W(on, M.p_node[l]), eps,
                                               hb_part, aggbar, ns, P0, &nb, s));
        if ((rc = job(nb, 0, 0, 1, D, grad, on.b1, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 0, D, 1, D, grad, on.b2, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 0, 2 * D, 1, 2 * D, grad, on.g, 0)) != MGN_OK) return rc;
        Partials q = P1;
        LAUNCH(K_WGRAD_NODE, launch_wgrad_r32(D, N, ns + 2 * nd, h_l(k, l), q, &nb, s));
        if ((rc = job(nb, 1, 0, D, D, grad, on.W1, 2 * D)) != MGN_OK) return rc;
        q.buf += (size_t)D * D;
        LAUNCH(K_WGRAD_NODE, launch_wgrad_r32(D, N, ns + 2 * nd, agg_l(k, l), q, &nb, s));
        if ((rc = job(nb, 1, (int64_t)D * D, D, D, grad, on.W1 + D, 2 * D)) != MGN_OK) return rc;
        q.buf += (size_t)D * D;
        LAUNCH(K_WGRAD_NODE, launch_wgrad_r32(D, N, ns + nd, ns, q, &nb, s));
        if ((rc = job(nb, 1, 2 * (int64_t)D * D, D, D, grad, on.W2, D)) != MGN_OK) return rc;
      }
      if (E == 0) {
        // no edges: the edge MLP gets no gradient and every R is zero
        LAUNCH(K_EDGE_BWD, launch_fill(R, N * D, 0.f, s));
      } else if (rows()) {
        // one pass: the edge MLP's reverse and its weight gradients
        LAUNCH(K_EDGE_BWD, launch_edge_bwd_fused(tl, a1_l(k, l), e_l(k, l), ebar, l < m - 1 ? 1 : 0, ebar, aggbar,
                                                 W(oe, M.p_edge[l]), eps, zbar, R, slots(), P2, &nb, s));
        if ((rc = job(nb, 2, 0, D, D, grad, oe.W1, 3 * D)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 16384, 1, D, grad, oe.b1, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 16512, 1, D * D + D, grad, oe.W2, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 33024, 1, 2 * D, grad, oe.g, 0)) != MGN_OK) return rc;
      } else if (prec == MGN_BF16) {
        // width 160: one wave per row block from the saved a1; weight
        // gradients dW1e = sum zbar^T e and dW2 = sum dz2^T a1 in one pass
        // over the saved streams
        void* dz = ws + c.L.dz;
        LAUNCH(K_EDGE_BWD, launch_edge_bwd_w160(tl, a1_l(k, l), ebar, l < m - 1 ? 1 : 0, ebar, aggbar, W(oe, M.p_edge[l]),
                                    eps, zbar, dz, R, slots(), P2, &nb, s));
        if ((rc = job(nb, 2, 0, 1, D, grad, oe.b1, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, D, 1, 3 * D, grad, oe.b2, 0)) != MGN_OK) return rc;
        LAUNCH(K_WGRAD, launch_wgrad2_w160(E, zbar, e_l(k, l), dz, a1_l(k, l), P3, &nb, s));
        if ((rc = job(nb, 3, 0, D, D, grad, oe.W1, 3 * D)) != MGN_OK) return rc;
        if ((rc = job(nb, 3, (int64_t)D * D, D, D, grad, oe.W2, D)) != MGN_OK) return rc;
      } else if (D == kRowsD) {
        // fp32, width 128: one wave per row block, the reverse and the edge
        // MLP's weight gradients in one pass
        LAUNCH(K_EDGE_BWD, launch_edge_bwd_r32(D, tl, e_l(k, l), (float*)ebar, l < m - 1 ? 1 : 0, (float*)ebar,
                                               P_l(k, l), aggbar, W(oe, M.p_edge[l]), eps, zbar, R, slots(), P2, &nb,
                                               s));
        if ((rc = job(nb, 2, 0, D, D, grad, oe.W1, 3 * D)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 16384, 1, D, grad, oe.b1, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 16512, 1, D * D + D, grad, oe.W2, 0)) != MGN_OK) return rc;
        if ((rc = job(nb, 2, 33024, 1, 2 * D, grad, oe.g, 0)) != MGN_OK) return rc;
      } else {
        // fp32, width 160: one wave per row block (dW2 and the vectors in the
        // pass), then dW1e = sum zbar^T e over the two streams
        LAUNCH(K_EDGE_BWD, launch_edge_bwd_r32(D, tl, e_l(k, l), (float*)ebar, l < m - 1 ? 1 : 0, (float*)ebar,
                                               P_l(k, l), aggbar, W(oe, M.p_edge[l]), eps, zbar, R, slots(), P2, &nb,
                                               s));
        if ((rc = job(nb, 2, (int64_t)D * D, 1, (int)(oe.size - 3 * D * D), grad, oe.b1, 0)) != MGN_OK) return rc;
        LAUNCH(K_WGRAD, launch_wgrad_r32(D, E, (const float*)zbar, (const float*)e_l(k, l), P3, &nb, s));
        if ((rc = job(nb, 3, 0, D, D, grad, oe.W1, 3 * D)) != MGN_OK) return rc;
      }
      if (g.n_long > 0) LAUNCH(K_FIXUP, launch_slot_fixup(D, g.long_nodes, g.n_long, slots(), R, s));
      if (prec == MGN_BF16 && !rows())
        // width 160: one wave per 16-node unit, S through the node-stream
        // scratch (its streams are consumed by now) into the weight gradients
        LAUNCH(K_SRCSUM, launch_srcsum_w160(N, g.rowptr, g.rev, zbar, R, h_l(k, l), hb_part, W(oe, M.p_edge[l]), hb_cur,
                                            ws + c.L.nstr, P4, &nb, s));
      else if (prec == MGN_FP32) {
        // fp32: S into the node-stream scratch (its streams are consumed by
        // now), then dW1s = sum S h^T and dW1r = sum R h^T from the rows
        float* Sv = (float*)(ws + c.L.nstr);
        LAUNCH(K_SRCSUM, launch_node_srcsum_r32(D, N, g.rowptr, g.rev, (const float*)zbar, R, hb_part,
                                                W(oe, M.p_edge[l]), hb_cur, Sv, s));
        Partials q = P4;
        LAUNCH(K_SRCSUM, launch_wgrad_r32(D, N, Sv, h_l(k, l), q, &nb, s));
        if ((rc = job(nb, 4, 0, D, D, grad, oe.W1 + D, 3 * D)) != MGN_OK) return rc;
        q.buf += (size_t)D * D;
        LAUNCH(K_SRCSUM, launch_wgrad_r32(D, N, R, h_l(k, l), q, &nb, s));
        if ((rc = job(nb, 4, (int64_t)D * D, D, D, grad, oe.W1 + 2 * D, 3 * D)) != MGN_OK) return rc;
      } else {
        LAUNCH(K_SRCSUM, launch_node_srcsum(prec, D, N, g.rowptr, g.rev, zbar, R, h_l(k, l), hb_part, W(oe, M.p_edge[l]),
                                            hb_cur, P4, &nb, s));
      }
      if (prec != MGN_FP32) {
        if ((rc = job(nb, 4, 0, D, D, grad, oe.W1 + D, 3 * D)) != MGN_OK) return rc;
        if ((rc = job(nb, 4, (int64_t)D * D, D, D, grad, oe.W1 + 2 * D, 3 * D)) != MGN_OK) return rc;
      }
      // the block's partial regions are reused by the next block
      if ((rc = flush(grad)) != MGN_OK) return rc;
    }
    if (m > 0 && n_st > 1) {
      // dL/de0 summed over the stages, accumulated from the last stage to
      // the first (each stage's own gradient of the shared encoder output
      // is in ebar when its block reverses are done)
      void* est = ws + c.L.ebar_st;
      if (k > 0 && k < n_st - 1) LAUNCH(K_EDGE_ENC_BWD, launch_add_stream(prec, E * D, ebar, est, s));
      if (k == 0) LAUNCH(K_EDGE_ENC_BWD, launch_add_stream(prec, E * D, est, ebar, s));
    }
    if (m > 0 && (n_st == 1 || k == 0)) {
      if (rows())
        LAUNCH(K_EDGE_ENC_BWD, launch_edge_enc_bwd_rows(E, efeat, ebar, W(M.enc_edge, M.p_enc_edge), eps, pt, &nb, s));
      else
        LAUNCH(K_EDGE_ENC_BWD,
               prec == MGN_FP32
                   ? launch_edge_enc_bwd_r32(D, E, efeat, ebar, W(M.enc_edge, M.p_enc_edge), eps, pt, &nb, s)
                   : launch_edge_enc_bwd_w160(E, efeat, ebar, W(M.enc_edge, M.p_enc_edge), eps, pt, &nb, s));
      if ((rc = reduce(nb, 0, 1, (int)M.enc_edge.size, grad, M.enc_edge.W1, 0)) != MGN_OK) return rc;
    }
    if (prec == MGN_FP32) {
      // fp32: the row-layout reverse (W1, b1 and the vectors as its
      // partials), then dW2 = sum dz2^T a1 from its streams
      float* ns = (float*)(ws + c.L.nstr);
      const Off& o = M.enc_node;
      LAUNCH(K_NODE_ENC_BWD, launch_node_enc_bwd_r32(D, N, node_in, hb_cur, W(o, M.p_enc_node), eps, gin, ns, pt, &nb, s));
      if ((rc = reduce(nb, 0, 1, 9 * D, grad, o.W1, 0)) != MGN_OK) return rc;
      if ((rc = reduce(nb, 9 * D, 1, 3 * D, grad, o.b2, 0)) != MGN_OK) return rc;
      LAUNCH(K_NODE_ENC_BWD, launch_wgrad_r32(D, N, ns + (size_t)N * D, ns, pt, &nb, s));
      if ((rc = reduce(nb, 0, D, D, grad, o.W2, D)) != MGN_OK) return rc;
    } else {
      LAUNCH(K_NODE_ENC_BWD, launch_node_enc_bwd(prec, D, N, node_in, hb_cur, W(M.enc_node, M.p_enc_node), eps, gin, pt,
                                                 &nb, s));
      if ((rc = reduce(nb, 0, 1, (int)M.enc_node.size, grad, M.enc_node.W1, 0)) != MGN_OK) return rc;
    }
    return MGN_OK;
  }
};

int check_cfg(const mgn_config* cfg) {
  if (!cfg) return fail(MGN_ERR_ARG, "null config");
  if (cfg->node_in != 8 || cfg->edge_in != 4 || (cfg->latent != 128 && cfg->latent != 150) || cfg->out != 4 ||
      cfg->mlp_layers != 2)
    return fail(MGN_ERR_SHAPE,
                "unsupported config (node_in 8, edge_in 4, latent 128 or 150, out 4, mlp_layers 2 are supported)");
  if (cfg->mp_steps < 0 || cfg->mp_steps > 4096) return fail(MGN_ERR_ARG, "mp_steps out of range");
  if (cfg->precision != MGN_FP32 && cfg->precision != MGN_BF16) return fail(MGN_ERR_ARG, "unknown precision");
  if (!(cfg->ln_eps > 0.f)) return fail(MGN_ERR_ARG, "ln_eps must be > 0");
  return MGN_OK;
}

int check_call(Ctx* c, const mgn_dgraph* g, const float* params, void* ws, size_t ws_bytes, int32_t save) {
  if (!c || !g) return fail(MGN_ERR_ARG, "null ctx or graph");
  if (g->n_nodes < 0 || g->n_edges < 0) return fail(MGN_ERR_ARG, "negative graph size");
  if (g->n_nodes > c->maxN || g->n_edges > c->maxE)
    return fail(MGN_ERR_SHAPE, "graph (%lld nodes, %lld edges) larger than the context (%lld, %lld)",
                (long long)g->n_nodes, (long long)g->n_edges, (long long)c->maxN, (long long)c->maxE);
  if (save && !c->save) return fail(MGN_ERR_STATE, "context was created without save");
  if (ws_bytes < c->L.total)
    return fail(MGN_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, c->L.total);
  if (g->n_nodes > 0) {
    if (!params || !ws) return fail(MGN_ERR_ARG, "null params or workspace");
    if (!g->rowptr || !g->tiles || g->n_tiles <= 0 ||
        (g->n_edges > 0 && (!g->senders || !g->receivers || !g->rev)))
      return fail(MGN_ERR_ARG, "device graph arrays missing");
    if (g->n_long > 0 && !g->long_nodes) return fail(MGN_ERR_ARG, "long_nodes missing");
  }
  return MGN_OK;
}

// The parameters a call computes from: at latent 150 the zero-padded
// kernel-width copy (written here, in the workspace); otherwise the caller's
// buffer, or for a saving call the workspace copy that the backward reads.
int stage_params(Ctx& c, const float*& params, char* ws, int save, hipStream_t s) {
  if (c.LD != c.DR) {
    float* pp = (float*)(ws + c.L.ppad);
    HIP_TRY(launch_fill(pp, c.M.total, 0.f, s));
    for (size_t b = 0; b < c.pad.size(); b += kCopyMax) {
      CopyList L{};
      L.n = (int32_t)std::min<size_t>(kCopyMax, c.pad.size() - b);
      for (int j = 0; j < L.n; ++j) L.b[j] = c.pad[b + j];
      HIP_TRY(launch_copy_blocks(L, params, pp, 0, s));
    }
    params = pp;
  } else if (save) {
    float* pc = (float*)(ws + c.L.pcopy);
    HIP_TRY(hipMemcpyAsync(pc, params, (size_t)c.M.total * sizeof(float), hipMemcpyDeviceToDevice, s));
    params = pc;
  }
  return MGN_OK;
}

// One integration step on graph g (the body of mgn_integrate_step, also run
// per patch by mgn_patch_step): K_i = MGN([static, y + sum_j a_ij K_j]),
// y_next = y + sum_i b_i K_i.
int integrate_core(Ctx& c, const mgn_dgraph& g, const float* params, const Tableau& tb, const float* static_feat,
                   const float* y, const float* efeat, float* y_next, int save, char* w, hipStream_t s,
                   bool pack) {
  const int64_t N = g.n_nodes;
  if (N == 0) return MGN_OK;
  int rc;
  Run r{c, g, params, w, s, N, g.n_edges, c.cfg.mp_steps, c.cfg.precision, c.cfg.ln_eps};
  r.keep_a1 = save != 0;
  if (pack && (rc = r.pack_weights()) != MGN_OK) return rc;
  float* node_in = (float*)(w + c.L.node_in);
  float* K = (float*)(w + c.L.K);
  for (int i = 0; i < tb.s; ++i) {
    LinComb lc{};
    lc.x[0] = y;
    lc.ld[0] = 4;
    lc.c[0] = 1.f;
    lc.n = 1;
    for (int j = 0; j < i; ++j)
      if (tb.a[i][j] != 0.f) {
        lc.x[lc.n] = K + (size_t)j * N * 4;
        lc.ld[lc.n] = 4;
        lc.c[lc.n] = tb.a[i][j];
        ++lc.n;
      }
    float* ni = node_in + (size_t)i * N * 8;
    HIP_TRY(launch_stage_input(N, static_feat, lc, ni, s));
    if ((rc = r.forward(ni, efeat, K + (size_t)i * N * 4, save ? i : 0, i)) != MGN_OK) return rc;
  }
  LinComb lc{};
  lc.x[0] = y;
  lc.ld[0] = 4;
  lc.c[0] = 1.f;
  lc.n = 1;
  for (int i = 0; i < tb.s; ++i)
    if (tb.b[i] != 0.f) {
      lc.x[lc.n] = K + (size_t)i * N * 4;
      lc.ld[lc.n] = 4;
      lc.c[lc.n] = tb.b[i];
      ++lc.n;
    }
  HIP_TRY(launch_lincomb(N, lc, y_next, 4, 0, s));
  return MGN_OK;
}

// Reverse mode of the saved forward or integration step (the body of
// mgn_backward, also run per patch by mgn_train_step).
int backward_steps(Ctx& c, const float* grad_out, float* grad_params, float* grad_in, hipStream_t s);

// At latent 150 the kernels accumulate into a zero-initialised padded
// gradient, which is then added to the caller's buffer in its own layout.
int backward_core(Ctx& c, const float* grad_out, float* grad_params, float* grad_in, hipStream_t s) {
  if (c.LD == c.DR) return backward_steps(c, grad_out, grad_params, grad_in, s);
  float* gp = (float*)(c.ws + c.L.gpad);
  HIP_TRY(launch_fill(gp, c.M.total, 0.f, s));
  int rc = backward_steps(c, grad_out, gp, grad_in, s);
  if (rc != MGN_OK) return rc;
  for (size_t b = 0; b < c.pad.size(); b += kCopyMax) {
    CopyList L{};
    L.n = (int32_t)std::min<size_t>(kCopyMax, c.pad.size() - b);
    for (int j = 0; j < L.n; ++j) {
      const CopyBlock& f = c.pad[b + j];
      L.b[j] = CopyBlock{f.b_off, f.a_off, f.rows, f.cols, f.b_ld, f.a_ld};
    }
    HIP_TRY(launch_copy_blocks(L, gp, grad_params, 1, s));
  }
  return MGN_OK;
}

int backward_steps(Ctx& c, const float* grad_out, float* grad_params, float* grad_in, hipStream_t s) {
  const int64_t N = c.g.n_nodes;
  Run r{c, c.g, c.params, c.ws, s, N, c.g.n_edges, c.cfg.mp_steps, c.cfg.precision, c.cfg.ln_eps};
  r.keep_a1 = true;
  int rc;
  if (c.saved == 1) return r.backward(0, c.node_in, c.efeat, grad_out, grad_params, grad_in);
  Tableau tb;
  tableau(c.scheme, tb);
  r.n_st = tb.s;
  char* w = c.ws;
  float* node_in = (float*)(w + c.L.node_in);
  float* kbar = (float*)(w + c.L.kbar);
  float* ys = (float*)(w + c.L.ystage);
  float* gin = (float*)(w + c.L.gin);
  for (int i = tb.s - 1; i >= 0; --i) {
    LinComb lc{};
    lc.x[0] = grad_out;
    lc.ld[0] = 4;
    lc.c[0] = tb.b[i];
    lc.n = 1;
    for (int j = i + 1; j < tb.s; ++j)
      if (tb.a[j][i] != 0.f) {
        lc.x[lc.n] = ys + (size_t)j * N * 4;
        lc.ld[lc.n] = 4;
        lc.c[lc.n] = tb.a[j][i];
        ++lc.n;
      }
    HIP_TRY(launch_lincomb(N, lc, kbar, 4, 0, s));
    if ((rc = r.backward(i, node_in + (size_t)i * N * 8, c.efeat, kbar, grad_params, gin)) != MGN_OK) return rc;
    LinComb cp{};
    cp.x[0] = gin;
    cp.ld[0] = 8;
    cp.off[0] = 4;
    cp.c[0] = 1.f;
    cp.n = 1;
    HIP_TRY(launch_lincomb(N, cp, ys + (size_t)i * N * 4, 4, 0, s));
  }
  if (grad_in) {
    LinComb lc{};
    lc.x[0] = grad_out;
    lc.ld[0] = 4;
    lc.c[0] = 1.f;
    lc.n = 1;
    for (int i = 0; i < tb.s; ++i) {
      lc.x[lc.n] = ys + (size_t)i * N * 4;
      lc.ld[lc.n] = 4;
      lc.c[lc.n] = 1.f;
      ++lc.n;
    }
    HIP_TRY(launch_lincomb(N, lc, grad_in, 4, 0, s));
  }
  return MGN_OK;
}


}  // namespace
}  // namespace mgn

struct mgn_ctx {
  mgn::Ctx c;
};

using namespace mgn;

extern "C" {

const char* mgn_version(void) { return "mgn-gfx950 0.1.0"; }

int mgn_scheme_stages(int32_t scheme) {
  Tableau t;
  if (!tableau(scheme, t)) return fail(MGN_ERR_ARG, "unknown scheme %d", scheme);
  return t.s;
}

int64_t mgn_param_count(const mgn_config* cfg) {
  if (check_cfg(cfg) != MGN_OK) return -1;
  return make_model(cfg->mp_steps, cfg->latent).total;
}

int mgn_ctx_create(const mgn_config* cfg, int64_t max_nodes, int64_t max_edges, int32_t max_stages, int32_t save,
                   size_t* ws_bytes, mgn_ctx** out) {
  int rc = check_cfg(cfg);
  if (rc != MGN_OK) return rc;
  if (!ws_bytes || !out) return fail(MGN_ERR_ARG, "mgn_ctx_create: null output pointer");
  if (max_nodes < 0 || max_edges < 0 || max_stages < 1 || max_stages > 4)
    return fail(MGN_ERR_ARG, "mgn_ctx_create: bad sizes or max_stages (1..4)");
  if (max_nodes >= (int64_t)INT32_MAX || max_edges >= (int64_t)INT32_MAX)
    return fail(MGN_ERR_SHAPE, "mgn_ctx_create: sizes must be < 2^31");
  mgn_ctx* h = new (std::nothrow) mgn_ctx();
  if (!h) return fail(MGN_ERR_NOMEM, "mgn_ctx_create: out of host memory");
  Ctx& c = h->c;
  c.cfg = *cfg;
  c.maxN = max_nodes;
  c.maxE = max_edges;
  c.max_stages = max_stages;
  c.save = save ? 1 : 0;
  c.se = cfg->precision == MGN_BF16 ? 2 : 4;
  c.ne_sets = c.save ? max_stages : 1;
  c.DR = cfg->latent;
  c.LD = cfg->latent == 150 ? 160 : cfg->latent;
  try {
    c.M = make_model(cfg->mp_steps, c.LD, cfg->precision == MGN_FP32);
    c.Mr = c.LD == c.DR ? c.M : make_model(cfg->mp_steps, c.DR);
    if (c.LD != c.DR) c.pad = pad_blocks(c.Mr, c.M);
  } catch (const std::bad_alloc&) {
    delete h;
    return fail(MGN_ERR_NOMEM, "mgn_ctx_create: out of host memory");
  }
  plan(c);
  *ws_bytes = c.L.total;
  *out = h;
  return MGN_OK;
}

void mgn_ctx_destroy(mgn_ctx* ctx) { delete ctx; }

int mgn_profile_enable(mgn_ctx* ctx, int32_t enable) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_profile_enable: null ctx");
  ctx->c.prof.on = enable != 0;
  return MGN_OK;
}

int mgn_profile_collect(mgn_ctx* ctx, int32_t max_kernels, char* names, double* total_ms, int64_t* launches,
                        int32_t* n_kernels) {
  if (!ctx || !n_kernels || max_kernels < 0 || (max_kernels > 0 && (!names || !total_ms || !launches)))
    return fail(MGN_ERR_ARG, "mgn_profile_collect: bad arguments");
  Prof& p = ctx->c.prof;
  double ms[K_COUNT] = {0};
  int64_t cnt[K_COUNT] = {0};
  if (p.used > 0) HIP_TRY(hipEventSynchronize(p.pool[p.used - 1]));
  for (size_t k = 0; k < p.kind.size(); ++k) {
    float t = 0.f;
    HIP_TRY(hipEventElapsedTime(&t, p.pool[2 * k], p.pool[2 * k + 1]));
    ms[p.kind[k]] += t;
    cnt[p.kind[k]] += 1;
  }
  p.used = 0;
  p.kind.clear();
  int32_t n = 0;
  for (int k = 0; k < K_COUNT; ++k) {
    if (!cnt[k]) continue;
    if (n < max_kernels) {
      std::strncpy(names + 32 * n, kKernName[k], 31);
      names[32 * n + 31] = 0;
      total_ms[n] = ms[k];
      launches[n] = cnt[k];
    }
    ++n;
  }
  *n_kernels = n;
  return MGN_OK;
}

int mgn_forward(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, const float* node_in, const float* efeat,
                float* out, int32_t save, void* ws, size_t ws_bytes, void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_forward: null ctx");
  int rc = check_call(&ctx->c, g, params, ws, ws_bytes, save);
  if (rc != MGN_OK) return rc;
  Ctx& c = ctx->c;
  if (g->n_nodes > 0 && (!node_in || !out || (g->n_edges > 0 && !efeat)))
    return fail(MGN_ERR_ARG, "mgn_forward: null input or output");
  c.saved = 0;
  // a saving call keeps its own copies of the parameters and node_in for
  // mgn_backward, and computes the forward from them
  float* kept = (float*)((char*)ws + c.L.node_in);
  if (g->n_nodes > 0 && (rc = stage_params(c, params, (char*)ws, save, S(stream))) != MGN_OK) return rc;
  Run r{c, *g, params, (char*)ws, S(stream), g->n_nodes, g->n_edges, c.cfg.mp_steps, c.cfg.precision, c.cfg.ln_eps};
  r.keep_a1 = save != 0;
  if (g->n_nodes > 0) {
    if ((rc = r.pack_weights()) != MGN_OK) return rc;
    if (save) HIP_TRY(hipMemcpyAsync(kept, node_in, (size_t)g->n_nodes * 8 * sizeof(float), hipMemcpyDeviceToDevice,
                                     S(stream)));
    if ((rc = r.forward(node_in, efeat, out, 0)) != MGN_OK) return rc;
  }
  if (save) {
    c.saved = 1;
    c.stages = 1;
    c.g = *g;
    c.params = params;
    c.efeat = efeat;
    c.node_in = kept;
    c.ws = (char*)ws;
  }
  return MGN_OK;
}

}  // extern "C"

namespace mgn {

size_t ctx_workspace_bytes(const mgn_ctx* ctx) { return ctx->c.L.total; }

int forward_in_scratch(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, const float* node_in,
                       const float* efeat, float* out, void* scratch, size_t scratch_bytes, void* stream) {
  // no event creation inside this call: profiling is suspended for it
  Prof& p = ctx->c.prof;
  const bool on = p.on;
  p.on = false;
  const int rc = mgn_forward(ctx, g, params, node_in, efeat, out, 0, scratch, scratch_bytes, stream);
  p.on = on;
  return rc;
}

}  // namespace mgn

extern "C" {

int mgn_integrate_step(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, int32_t scheme,
                       const float* static_feat, const float* y, const float* efeat, float* y_next, int32_t save,
                       void* ws, size_t ws_bytes, void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_integrate_step: null ctx");
  Tableau tb;
  if (!tableau(scheme, tb)) return fail(MGN_ERR_ARG, "mgn_integrate_step: unknown scheme %d", scheme);
  int rc = check_call(&ctx->c, g, params, ws, ws_bytes, save);
  if (rc != MGN_OK) return rc;
  Ctx& c = ctx->c;
  if (tb.s > c.max_stages)
    return fail(MGN_ERR_ARG, "mgn_integrate_step: scheme needs %d stages, context plans %d", tb.s, c.max_stages);
  if (g->n_nodes > 0 && (!static_feat || !y || !y_next || (g->n_edges > 0 && !efeat)))
    return fail(MGN_ERR_ARG, "mgn_integrate_step: null input or output");
  c.saved = 0;
  char* w = (char*)ws;
  // a saving call computes from, and keeps, its own copy of the parameters
  if (g->n_nodes > 0 && (rc = stage_params(c, params, w, save, S(stream))) != MGN_OK) return rc;
  if ((rc = integrate_core(c, *g, params, tb, static_feat, y, efeat, y_next, save, w, S(stream), true)) != MGN_OK)
    return rc;
  if (save) {
    c.saved = 2;
    c.scheme = scheme;
    c.stages = tb.s;
    c.g = *g;
    c.params = params;
    c.efeat = efeat;
    c.node_in = nullptr;
    c.ws = w;
  }
  return MGN_OK;
}

int mgn_patch_step(mgn_ctx* ctx, int32_t n_patches, const mgn_dpatch* patches, const float* params,
                   int32_t scheme, const float* static_feat, const float* y, float* y_next, int64_t n_global,
                   void* ws, size_t ws_bytes, void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_patch_step: null ctx");
  Tableau tb;
  if (!tableau(scheme, tb)) return fail(MGN_ERR_ARG, "mgn_patch_step: unknown scheme %d", scheme);
  if (n_patches < 0 || (n_patches > 0 && !patches) || n_global < 0)
    return fail(MGN_ERR_ARG, "mgn_patch_step: bad patch list or global size");
  Ctx& c = ctx->c;
  if (tb.s > c.max_stages)
    return fail(MGN_ERR_ARG, "mgn_patch_step: scheme needs %d stages, context plans %d", tb.s, c.max_stages);
  if (n_global > 0 && (!static_feat || !y || !y_next))
    return fail(MGN_ERR_ARG, "mgn_patch_step: null global state");
  if (n_global > 0 && y_next == y) return fail(MGN_ERR_ARG, "mgn_patch_step: y_next must not alias y");
  int rc;
  bool any = false;
  for (int32_t p = 0; p < n_patches; ++p) {
    const mgn_dpatch& P = patches[p];
    if ((rc = check_call(&c, &P.g, params, ws, ws_bytes, 0)) != MGN_OK) return rc;
    if (P.g.n_nodes > 0) {
      if (!P.node_l2g || !P.interior || (P.g.n_edges > 0 && !P.efeat))
        return fail(MGN_ERR_ARG, "mgn_patch_step: patch %d: null maps or edge features", p);
      if (n_global == 0) return fail(MGN_ERR_ARG, "mgn_patch_step: patch %d has nodes but n_global is 0", p);
      any = true;
    }
  }
  c.saved = 0;
  if (!any) return MGN_OK;
  char* w = (char*)ws;
  hipStream_t s = S(stream);
  if ((rc = stage_params(c, params, w, 0, s)) != MGN_OK) return rc;
  bool packed = false;
  for (int32_t p = 0; p < n_patches; ++p) {
    const mgn_dpatch& P = patches[p];
    const int64_t Np = P.g.n_nodes;
    if (Np == 0) continue;
    float* st_p = (float*)(w + c.L.pio);
    float* y_p = st_p + (size_t)c.maxN * 4;
    float* yn_p = y_p + (size_t)c.maxN * 4;
    // ghost refresh: every patch node takes the current state of its global node
    HIP_TRY(launch_gather_rows4(Np, static_feat, P.node_l2g, n_global, st_p, s));
    HIP_TRY(launch_gather_rows4(Np, y, P.node_l2g, n_global, y_p, s));
    if ((rc = integrate_core(c, P.g, params, tb, st_p, y_p, P.efeat, yn_p, 0, w, s, !packed)) != MGN_OK) return rc;
    packed = true;
    HIP_TRY(launch_scatter_rows4(Np, yn_p, P.node_l2g, P.interior, n_global, y_next, s));
  }
  return MGN_OK;
}

double mgn_adam_lr(const mgn_adam* a, int64_t k) {
  if (!a || k < 1 || a->decay_steps <= 0 || !(a->lr_start > 0) || !(a->lr_end > 0)) return -1.0;
  return a->lr_start * std::pow(a->lr_end / a->lr_start, (double)(k - 1) / (double)a->decay_steps);
}

static int adam_checked(const mgn_adam* a, int64_t k, float* params, const float* grad, float* m, float* v, int64_t n,
                        hipStream_t s, const char* who) {
  const double lr = mgn_adam_lr(a, k);
  if (lr < 0) return fail(MGN_ERR_ARG, "%s: bad Adam settings or update index %lld", who, (long long)k);
  if (!(a->beta1 >= 0.0 && a->beta1 < 1.0 && a->beta2 >= 0.0 && a->beta2 < 1.0 && a->eps > 0.0))
    return fail(MGN_ERR_ARG, "%s: Adam betas must lie in [0, 1) and eps be > 0", who);
  if (n < 0 || (n > 0 && (!params || !grad || !m || !v))) return fail(MGN_ERR_ARG, "%s: null Adam buffer", who);
  const double bc1 = 1.0 - std::pow(a->beta1, (double)k), bc2 = 1.0 - std::pow(a->beta2, (double)k);
  HIP_TRY(launch_adam(n, params, grad, m, v, (float)lr, (float)a->beta1, (float)(1.0 - a->beta1), (float)a->beta2,
                      (float)(1.0 - a->beta2), (float)a->eps, (float)bc1, (float)bc2, s));
  return MGN_OK;
}

int mgn_adam_step(const mgn_adam* a, int64_t k, float* params, const float* grad, float* m, float* v, int64_t n,
                  void* stream) {
  return adam_checked(a, k, params, grad, m, v, n, S(stream), "mgn_adam_step");
}

int mgn_train_step(mgn_ctx* ctx, int32_t n_patches, const mgn_dpatch* patches, float* params, int32_t scheme,
                   const float* static_feat, const float* y, const float* y_target, const float* noise,
                   const float* noise_std, int64_t n_loss_nodes, float* grad, float* adam_m, float* adam_v,
                   const mgn_adam* adam, int64_t k, float* loss, int64_t n_global, void* ws, size_t ws_bytes,
                   void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_train_step: null ctx");
  Ctx& c = ctx->c;
  Tableau tb;
  if (!tableau(scheme, tb)) return fail(MGN_ERR_ARG, "mgn_train_step: unknown scheme %d", scheme);
  if (tb.s > c.max_stages)
    return fail(MGN_ERR_ARG, "mgn_train_step: scheme needs %d stages, context plans %d", tb.s, c.max_stages);
  if (!c.save) return fail(MGN_ERR_STATE, "mgn_train_step: context was created without save");
  if (n_patches < 0 || (n_patches > 0 && !patches) || n_global < 0 || n_loss_nodes <= 0)
    return fail(MGN_ERR_ARG, "mgn_train_step: bad patch list, global size or loss node count");
  if (!params || !grad || !adam_m || !adam_v || !adam || !loss)
    return fail(MGN_ERR_ARG, "mgn_train_step: null parameter, gradient, Adam or loss buffer");
  if (n_global > 0 && (!static_feat || !y || !y_target)) return fail(MGN_ERR_ARG, "mgn_train_step: null global state");
  int rc;
  for (int32_t p = 0; p < n_patches; ++p) {
    const mgn_dpatch& P = patches[p];
    if ((rc = check_call(&c, &P.g, params, ws, ws_bytes, 1)) != MGN_OK) return rc;
    if (P.g.n_nodes > 0 && (!P.node_l2g || !P.interior || (P.g.n_edges > 0 && !P.efeat) || n_global == 0))
      return fail(MGN_ERR_ARG, "mgn_train_step: patch %d: null maps or edge features", p);
  }
  static const float kPaperStd[4] = {0.02f, 0.02f, 0.03f, 0.05f};
  const float* sd = noise_std ? noise_std : kPaperStd;
  const int64_t P_n = c.Mr.total;
  char* w = (char*)ws;
  hipStream_t s = S(stream);
  HIP_TRY(launch_fill(grad, P_n, 0.f, s));
  HIP_TRY(launch_fill(loss, 1, 0.f, s));
  // the step's forward and backward compute from run_params (the caller's
  // buffer, or its padded copy at latent 150); Adam then updates params
  const float* run_params = params;
  if ((rc = stage_params(c, run_params, w, 0, s)) != MGN_OK) return rc;
  const float inv = (float)(1.0 / (4.0 * (double)n_loss_nodes));
  bool packed = false;
  for (int32_t p = 0; p < n_patches; ++p) {
    const mgn_dpatch& P = patches[p];
    const int64_t Np = P.g.n_nodes;
    if (Np == 0) continue;
    float* st_p = (float*)(w + c.L.pio);
    float* y_p = st_p + (size_t)c.maxN * 4;
    float* yn_p = y_p + (size_t)c.maxN * 4;
    float* go_p = yn_p + (size_t)c.maxN * 4;
    HIP_TRY(launch_gather_rows4(Np, static_feat, P.node_l2g, n_global, st_p, s));
    HIP_TRY(launch_gather_noisy(Np, y, noise, sd, P.node_l2g, n_global, y_p, s));
    if ((rc = integrate_core(c, P.g, run_params, tb, st_p, y_p, P.efeat, yn_p, 1, w, s, !packed)) != MGN_OK) return rc;
    packed = true;
    c.saved = 2;
    c.scheme = scheme;
    c.stages = tb.s;
    c.g = P.g;
    c.params = run_params;
    c.efeat = P.efeat;
    c.node_in = nullptr;
    c.ws = w;
    HIP_TRY(launch_mse(Np, yn_p, y_target, P.node_l2g, P.interior, n_global, inv, go_p, (float*)(w + c.L.lossp), loss,
                       s));
    if ((rc = backward_core(c, go_p, grad, nullptr, s)) != MGN_OK) return rc;
  }
  c.saved = 0;
  return adam_checked(adam, k, params, grad, adam_m, adam_v, P_n, s, "mgn_train_step");
}

int mgn_pec_step(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, const float* static_feat, const float* y,
                 float* khist, const float* efeat, float* y_next, int32_t first, void* ws, size_t ws_bytes,
                 void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_pec_step: null ctx");
  int rc = check_call(&ctx->c, g, params, ws, ws_bytes, 0);
  if (rc != MGN_OK) return rc;
  Ctx& c = ctx->c;
  const int64_t N = g->n_nodes;
  if (N > 0 && (!static_feat || !y || !khist || !y_next || (g->n_edges > 0 && !efeat)))
    return fail(MGN_ERR_ARG, "mgn_pec_step: null input or output");
  if (N > 0 && (y_next == y || y_next == khist || y_next == khist + (size_t)N * 4))
    return fail(MGN_ERR_ARG, "mgn_pec_step: y_next must not alias y or khist");
  c.saved = 0;
  if (N == 0) return MGN_OK;
  char* w = (char*)ws;
  if ((rc = stage_params(c, params, w, 0, S(stream))) != MGN_OK) return rc;
  Run r{c, *g, params, w, S(stream), N, g->n_edges, c.cfg.mp_steps, c.cfg.precision, c.cfg.ln_eps};
  if ((rc = r.pack_weights()) != MGN_OK) return rc;
  float* node_in = (float*)(w + c.L.node_in);
  float* Kp = (float*)(w + c.L.K);
  float* K0 = khist;
  float* K1 = khist + (size_t)N * 4;
  auto comb = [&](std::initializer_list<std::pair<const float*, float>> terms) {
    LinComb lc{};
    for (const auto& t : terms) {
      lc.x[lc.n] = t.first;
      lc.ld[lc.n] = 4;
      lc.c[lc.n] = t.second;
      ++lc.n;
    }
    return lc;
  };
  if (first) {
    // K_0 = K_-1 = MGN([static, y])
    HIP_TRY(launch_stage_input(N, static_feat, comb({{y, 1.f}}), node_in, S(stream)));
    if ((rc = r.forward(node_in, efeat, K0, 0)) != MGN_OK) return rc;
    HIP_TRY(launch_lincomb(N, comb({{K0, 1.f}}), K1, 4, 0, S(stream)));
  }
  // predict, evaluate, correct
  HIP_TRY(launch_stage_input(N, static_feat, comb({{y, 1.f}, {K0, 1.5f}, {K1, -0.5f}}), node_in, S(stream)));
  if ((rc = r.forward(node_in, efeat, Kp, 0, first ? 1 : 0)) != MGN_OK) return rc;
  HIP_TRY(launch_lincomb(N, comb({{y, 1.f}, {Kp, 0.5f}, {K0, 0.5f}}), y_next, 4, 0, S(stream)));
  // history <- (K_p, K_n)
  HIP_TRY(launch_lincomb(N, comb({{K0, 1.f}}), K1, 4, 0, S(stream)));
  HIP_TRY(launch_lincomb(N, comb({{Kp, 1.f}}), K0, 4, 0, S(stream)));
  return MGN_OK;
}

int mgn_backward(mgn_ctx* ctx, const float* grad_out, float* grad_params, float* grad_in, void* stream) {
  if (!ctx) return fail(MGN_ERR_ARG, "mgn_backward: null ctx");
  Ctx& c = ctx->c;
  if (!c.saved) return fail(MGN_ERR_STATE, "mgn_backward: no saved forward or integration step");
  const int64_t N = c.g.n_nodes;
  if (N == 0) return MGN_OK;
  if (!grad_out || !grad_params) return fail(MGN_ERR_ARG, "mgn_backward: null gradient buffer");
  return backward_core(c, grad_out, grad_params, grad_in, S(stream));
}

}  // extern "C"
