/*
 * mgn.h -- C ABI of the MI355X (gfx950) MeshGraphNets message-passing library.
 *
 * What the library computes (Bartoldson, Hu et al., "Scientific Computing
 * Algorithms to Learn Enhanced Scalable Surrogates for Mesh Physics",
 * arXiv 2304.00338):
 *   - the mesh graph whose edges come from the simplices of the mesh
 *     (App. B) with MGN edge features (App. C);
 *   - equal-split subdomains and k-hop ghost-zone patches (Sec. 2.2);
 *   - one MGN call: encoder, m message-passing steps (each updates every edge
 *     from its incident nodes, then every node from the sum of its incident
 *     edge messages, Sec. 2.1), decoder; and its reverse mode;
 *   - one explicit integration step y' = y + sum_i b_i K_i with
 *     K_i = MGN(stage i), i.e. the update rule of Sec. 2.1 and the Heun forms
 *     of Sec. 2.3 / App. A (equation heun) generalised to a Butcher tableau.
 *
 * Conventions
 *   - Every function returns an int status: MGN_OK (0) or a negative MGN_ERR_*.
 *     On error the out-parameters are left untouched and mgn_last_error()
 *     returns a message (thread-local, valid until the next call on the same
 *     thread).  No C++ exception crosses this boundary.
 *   - Host pointers are used for graph and patch construction.  Device
 *     pointers (HIP device memory) are used by mgn_forward, mgn_backward and
 *     mgn_integrate_step; those calls are asynchronous on the HIP stream
 *     passed as `stream` (a hipStream_t cast to void*, NULL = default
 *     stream), and every buffer must stay alive until that stream has
 *     finished the work (and, for a saved call, until mgn_backward has run).
 *   - The caller owns every buffer it passes; the library never frees caller
 *     memory and never allocates device memory: all device scratch lives in
 *     the caller's workspace, whose size mgn_ctx_create reports.
 *   - Opaque handles (mgn_graph, mgn_ctx) are created and destroyed by the
 *     library; destroying NULL is a no-op.
 *   - Index arrays are int32 (E < 2^31 and N < 2^31 are checked); features
 *     and parameters are float32, row-major.
 */
#ifndef MGN_H
#define MGN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define MGN_OK 0
#define MGN_ERR_ARG (-1)       /* null pointer, negative size, unknown enum */
#define MGN_ERR_RANGE (-2)     /* an index outside [0, N) or a bad subdomain id */
#define MGN_ERR_SHAPE (-3)     /* unsupported dimensions, or N/E too large */
#define MGN_ERR_WORKSPACE (-4) /* caller workspace smaller than required */
#define MGN_ERR_STATE (-5)     /* backward without a saved call, ctx/graph mismatch */
#define MGN_ERR_DEVICE (-6)    /* a HIP runtime error (message kept) */
#define MGN_ERR_NOMEM (-7)     /* host allocation failed */

/* ---- enums ----------------------------------------------------------- */
#define MGN_FP32 0 /* fp32 MFMA, fp32 latent streams */
#define MGN_BF16 1 /* bf16 MFMA operands, bf16 edge-latent stream, fp32
                      accumulation, LayerNorm statistics, sums and node state */

/* Integration schemes: Butcher tableaux with MGN in place of h*f.
 * EULER    y' = y + K1                                  (Sec. 2.1)
 * HEUN2    a21 = 1, b = (1/2, 1/2)                       (App. A, eq. heun)
 * MIDPOINT a21 = 1/2, b = (0, 1)
 * HEUN3    a21 = 1/3, a32 = 2/3, b = (1/4, 0, 3/4)       (Heun's 3rd order, Sec. 2.3)
 * RK4      a21 = a32 = 1/2, a43 = 1, b = (1, 2, 2, 1)/6
 * RALSTON2 a21 = 2/3, b = (1/4, 3/4)                     (Ralston's methods,
 * RALSTON3 a21 = 1/2, a32 = 3/4, b = (2/9, 1/3, 4/9)      outlook, App. D) */
#define MGN_EULER 0
#define MGN_HEUN2 1
#define MGN_MIDPOINT 2
#define MGN_HEUN3 3
#define MGN_RK4 4
#define MGN_RALSTON2 5
#define MGN_RALSTON3 6

/* ---- model configuration --------------------------------------------- */
typedef struct mgn_config {
  int32_t node_in;    /* node input features; must be 8 (4 one-hot + 4 state) */
  int32_t edge_in;    /* edge input features; must be 4 */
  int32_t latent;     /* latent width D: 128 (App. C, 2D model) or 150 (App. C,
                         3D model; MGN_FP32 only, computed 160 wide with zero
                         padding, LayerNorm over the 150 real features) */
  int32_t out;        /* decoder outputs; must be 4 */
  int32_t mp_steps;   /* m >= 0 message-passing steps (unshared weights) */
  int32_t mlp_layers; /* Linear layers per MLP; must be 2 */
  float ln_eps;       /* LayerNorm epsilon (biased variance), e.g. 1e-5 */
  int32_t precision;  /* MGN_FP32 or MGN_BF16 */
} mgn_config;

/* Flat float32 parameter buffer, in this order (weights [out][in] row-major,
 * D = latent):
 *   enc_node: W1[D][8]  b1[D] W2[D][D] b2[D] gamma[D] beta[D]
 *   enc_edge: W1[D][4]  b1 W2[D][D] b2 gamma beta
 *   for each block i < m:
 *     edge:   W1[D][3D] (input order: edge latent, sender latent,
 *             receiver latent) b1 W2[D][D] b2 gamma beta
 *     node:   W1[D][2D] (input order: node latent, aggregate) b1
 *             W2[D][D] b2 gamma beta
 *   dec:      W1[D][D] b1[D] W2[4][D] b2[4]          (no LayerNorm)
 * At D = 128: 17,920 + 17,408 + m * (66,048 + 49,664) + 17,028 floats
 * (1,788,036 at m = 15); at D = 150: 547,354 floats at m = 3.  Gradients
 * are returned in the same layout. */
int64_t mgn_param_count(const mgn_config* cfg);

/* ---- host graphs (App. B edges, Sec. 2.2 patches) --------------------- */
typedef struct mgn_graph mgn_graph;

/* Every unordered pair of distinct vertices that share a cell becomes one
 * undirected mesh edge, stored as two directed edges; duplicates are merged
 * and repeated vertices in a cell make no self-loop.  Edges are sorted by
 * (receiver, sender).  rev[e] is the edge in the opposite direction.  Edge
 * features: [x_s - x_r, |x_s - x_r|] evaluated in fp64 from the float32
 * positions and rounded once to float32 (2D: [dx, dy, |d|, 0]).
 * cells [n_cells][verts_per_cell] (2, 3 or 4), pos [n_nodes][dim] (2 or 3).
 * Errors: ARG (null, bad dim / verts_per_cell), RANGE (vertex id outside
 * [0, n_nodes)), SHAPE (n_nodes or edge count >= 2^31). */
int mgn_build_graph(const int32_t* cells, int64_t n_cells,
                    int32_t verts_per_cell, const float* pos, int64_t n_nodes,
                    int32_t dim, mgn_graph** out);

/* Node and directed-edge counts; either pointer may be NULL. */
int mgn_graph_info(const mgn_graph* g, int64_t* n_nodes, int64_t* n_edges);

/* Copy the CSR arrays out (host buffers; any pointer may be NULL):
 * rowptr[N+1], senders[E], receivers[E], rev[E], efeat[E][4]. */
int mgn_graph_copy(const mgn_graph* g, int32_t* rowptr, int32_t* senders,
                   int32_t* receivers, int32_t* rev, float* efeat);

/* Receiver-aligned edge tiles for the device kernels.  Tile t is int32[4]
 * {node_begin, node_end, edge_begin, edge_end}: the whole in-edge segments
 * of nodes [node_begin, node_end), at most mgn_tile_edges() edges and
 * mgn_tile_nodes() nodes.  A node with more in-edges than one tile holds is
 * split into chunk tiles {v, -1 - slot, edge_begin, edge_end} whose sums go to
 * partial slot `slot`, and listed in long_nodes as int32[4]
 * {v, first_slot, n_chunks, 0}.  Tiles cover every node in order, so the
 * sum over a segment never depends on where the segment sits in the array.
 * Query the counts with NULL buffers first. */
int mgn_graph_schedule(const mgn_graph* g, int32_t* tiles, int64_t* n_tiles,
                       int32_t* long_nodes, int64_t* n_long);
int32_t mgn_tile_edges(void);
int32_t mgn_tile_nodes(void);

void mgn_graph_destroy(mgn_graph* g);

/* Subdomain ids from an equal split of the bounding box along every axis
 * (Sec. 2.2; App. C uses 3 x 4 in 2D and 12 x 12 x 15 in 3D).  Per axis the
 * index is floor(splits * (x - lo) / (hi - lo)), evaluated in fp64 left to
 * right and clamped to [0, splits - 1] (0 on a degenerate axis); ids run x
 * fastest.  pos [n][dim], splits [dim], part_out [n] (host).
 * Errors: ARG. */
int mgn_partition(const float* pos, int64_t n, int32_t dim,
                  const int32_t* splits, int32_t* part_out);

/* Patch p of a partition (Sec. 2.2, Fig. 1): the nodes of subdomain p plus
 * every node within k undirected hops (the ghost zone), with the induced
 * edges.  Local node ids follow ascending global ids, so in-segment edge
 * order matches the whole graph.  An empty subdomain gives a valid 0-node
 * patch.  part [N] is a host array of subdomain ids >= 0.
 * Errors: ARG (k < 0, null), RANGE (p outside [0, max(part)], or a negative
 * id in part). */
int mgn_extract_patch(const mgn_graph* g, const int32_t* part, int32_t p,
                      int32_t k, mgn_graph** patch);

/* Disjoint union of n patches (of one graph): one patch-like graph whose
 * parts are the given patches in order, with their nodes and edges renumbered
 * consecutively (part j's local ids offset by the node / edge counts of parts
 * 0..j-1) and no edge between parts.  One MGN call on the union computes, for
 * every node, bitwise what the call on its own patch computes (rows interact
 * only through their own in-segment sums), so a batch of patches (Sec. 2.2,
 * condition 3: gradients summed over patches) runs as one launch per kernel;
 * only the summation order of the weight gradients differs.  Maps: node_l2g
 * and hop concatenated (a global node that is in several patches appears once
 * per patch), edge_l2g concatenated, n_interior summed.  The union is owned
 * by the caller (mgn_graph_destroy) and does not refer to the parts.
 * Errors: ARG (null), STATE (a part is not a patch), SHAPE (2^31 nodes or
 * edges). */
int mgn_patch_union(const mgn_graph* const* patches, int32_t n, mgn_graph** out);

/* Patch maps (host buffers; any pointer may be NULL): node_l2g[Np] global id
 * of each local node, hop[Np] ghost distance (0 = subdomain node),
 * interior[Np] 1 for subdomain nodes, edge_l2g[Ep] global edge id,
 * n_interior number of subdomain nodes.  Errors: STATE if g is not a patch. */
int mgn_patch_copy_maps(const mgn_graph* patch, int32_t* node_l2g,
                        int32_t* hop, uint8_t* interior, int64_t* edge_l2g,
                        int64_t* n_interior);

/* ---- device execution -------------------------------------------------- */

/* Device view of a graph: device copies of the arrays above. */
typedef struct mgn_dgraph {
  int64_t n_nodes;
  int64_t n_edges;
  const int32_t* rowptr;     /* [N+1] */
  const int32_t* senders;    /* [E] */
  const int32_t* receivers;  /* [E] */
  const int32_t* rev;        /* [E] */
  const int32_t* tiles;      /* [n_tiles][4] from mgn_graph_schedule */
  int64_t n_tiles;
  const int32_t* long_nodes; /* [n_long][4], may be NULL when n_long == 0 */
  int64_t n_long;
} mgn_dgraph;

/* One patch of a decomposed mesh (Sec. 2.2) as mgn_patch_step sees it; all
 * arrays on the device.  g is the patch's local graph (mgn_extract_patch,
 * mgn_graph_schedule), efeat its [E_p][4] edge features, node_l2g the global
 * id of every local node and interior 1 for the subdomain nodes
 * (mgn_patch_copy_maps). */
typedef struct mgn_dpatch {
  mgn_dgraph g;
  const float* efeat;
  const int32_t* node_l2g;  /* [N_p] */
  const uint8_t* interior;  /* [N_p] */
} mgn_dpatch;

typedef struct mgn_ctx mgn_ctx;

/* A context plans the device workspace for graphs of up to max_nodes nodes
 * and max_edges edges, integration schemes of up to max_stages stages, and
 * (save != 0) keeping activations for mgn_backward.  *ws_bytes receives the
 * workspace size, a pure function of these arguments.
 * Errors: ARG, SHAPE (unsupported config, sizes >= 2^31). */
int mgn_ctx_create(const mgn_config* cfg, int64_t max_nodes, int64_t max_edges,
                   int32_t max_stages, int32_t save, size_t* ws_bytes,
                   mgn_ctx** out);
void mgn_ctx_destroy(mgn_ctx* ctx);

/* One MGN call (Sec. 2.1): out[N][4] = decoder(processor^m(encoder(node_in,
 * efeat))).  params: flat float32 buffer (device).  node_in [N][8],
 * efeat [E][4], out [N][4] (device).  With save != 0 the activations stay in
 * the workspace for mgn_backward (the context must have been created with
 * save).  The workspace must stay untouched until backward, and the graph
 * arrays and efeat must stay alive and unchanged until then (params and
 * node_in are copied into the workspace by a saving call).  N = 0 is a
 * no-op.
 * Errors: ARG, SHAPE (graph larger than the context), WORKSPACE, DEVICE. */
int mgn_forward(mgn_ctx* ctx, const mgn_dgraph* g, const float* params,
                const float* node_in, const float* efeat, float* out,
                int32_t save, void* workspace, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory at call time (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * mgn_forward with save = 0 whose device scratch is a static device array of
 * MGN_NOALLOC_SCRATCH_BYTES bytes instead of a caller workspace.  The array
 * is held once per GPU, from the library's first use on that GPU until the
 * process ends; its address is looked up on the first call made with that
 * GPU current (the GPU that runs `stream` must be the current device).  The
 * call allocates nothing: the caller passes inputs and outputs as for
 * mgn_forward (params, node_in, efeat, out on the device; the result is
 * bitwise that of mgn_forward with save = 0).  Every scratch element is
 * written before it is read, so no clearing is needed between calls.  All
 * calls on one GPU share its array: two calls that overlap in time on one
 * GPU (different streams, or different host threads) race and give
 * undefined results; calls on one stream are ordered and safe.  The call
 * does not touch the context's saved state other than clearing it (as any
 * mgn_forward does) and records no profiling events.
 * Errors: WORKSPACE when the context plans more workspace than the array
 * holds (mgn_ctx_create's *ws_bytes > MGN_NOALLOC_SCRATCH_BYTES, checked
 * before any device work), then those of mgn_forward. */
#define MGN_NOALLOC_SCRATCH_BYTES (128ull << 20)
int mgn_forward_noalloc(mgn_ctx* ctx, const mgn_dgraph* g, const float* params,
                        const float* node_in, const float* efeat, float* out,
                        void* stream);

/* Reverse mode of the last saved mgn_forward or mgn_integrate_step on ctx.
 * grad_out: [N][4] gradient of the loss with respect to out (or to y_next).
 * grad_params: flat float32 [mgn_param_count]; the gradient is ADDED to it, so
 * gradients of several patches accumulate (Sec. 2.2, condition 3).
 * grad_in (nullable): for a forward call, [N][8] gradient with respect to
 * node_in; for an integration step, [N][4] gradient with respect to y.  The
 * accumulation order is fixed, so results are bitwise reproducible.
 * Errors: ARG, STATE (nothing saved), DEVICE. */
int mgn_backward(mgn_ctx* ctx, const float* grad_out, float* grad_params,
                 float* grad_in, void* stream);

/* One explicit integration step with MGN as the scaled derivative
 * (Sec. 2.1, Sec. 2.3, App. A): K_i = MGN([static, y + sum_j a_ij K_j]),
 * y_next = y + sum_i b_i K_i.  static [N][4] (one-hot node type),
 * y [N][4], efeat [E][4], y_next [N][4] (device).  The edge encoder's inputs
 * (efeat, parameters) are the same in every stage, so the edges are encoded
 * once per step and the stages share that output (and, with save, the
 * backward sums the stages' gradients of it before the encoder's reverse).
 * Errors: ARG (unknown scheme, or more stages than the context plans), plus
 * those of mgn_forward. */
int mgn_integrate_step(mgn_ctx* ctx, const mgn_dgraph* g, const float* params,
                       int32_t scheme, const float* static_feat,
                       const float* y, const float* efeat, float* y_next,
                       int32_t save, void* workspace, size_t ws_bytes,
                       void* stream);

/* Number of stages of a scheme (1, 2, 2, 3, 4, 2, 3), or MGN_ERR_ARG. */
int mgn_scheme_stages(int32_t scheme);

/* One integration step of the whole mesh computed patch by patch (Sec. 2.2:
 * patch-decomposed inference on one GPU).  For each patch in order: every
 * patch node takes the current global static and y rows of its global node
 * (so ghost nodes are refreshed from their owners), the patch takes one step
 * of the scheme as in mgn_integrate_step, and the next state of its interior
 * nodes is written to y_next.  static, y, y_next: [n_global][4] (device);
 * y_next must not alias y.  Rows of y_next whose node is interior to no
 * patch are left as they were.  With ghost depth k >= s m for an s-stage
 * scheme and m MP steps, and every node interior to exactly one patch, the
 * result equals mgn_integrate_step on the whole mesh bitwise (patch nodes in
 * ascending global order, Sec. 2.2 condition 1).  The context must hold the
 * largest patch; node ids outside [0, n_global) give unspecified rows (they
 * are clamped, never read or written out of bounds).
 * Errors: ARG (null pointers, bad scheme or sizes, aliasing), SHAPE (a patch
 * larger than the context), WORKSPACE, DEVICE. */
int mgn_patch_step(mgn_ctx* ctx, int32_t n_patches, const mgn_dpatch* patches,
                   const float* params, int32_t scheme,
                   const float* static_feat, const float* y, float* y_next,
                   int64_t n_global, void* workspace, size_t ws_bytes,
                   void* stream);

/* Adam with the exponentially decaying learning rate of the paper's
 * training (App. C: 1e-3 to 1e-7 over 4,000,000 steps).  The k-th update
 * (k = 1, 2, ...) uses lr = lr_start (lr_end / lr_start)^((k - 1) /
 * decay_steps) and the bias corrections 1 - beta^k. */
typedef struct mgn_adam {
  double lr_start;     /* 1e-3 */
  double lr_end;       /* 1e-7 */
  int64_t decay_steps; /* 4000000 */
  double beta1;        /* 0.9 */
  double beta2;        /* 0.999 */
  double eps;          /* 1e-8 */
} mgn_adam;

/* Learning rate of the k-th update, or -1 for bad settings (k < 1,
 * non-positive rates or decay_steps). */
double mgn_adam_lr(const mgn_adam* adam, int64_t k);

/* The k-th Adam update of n float32 parameters in place (device):
 * m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2,
 * p -= lr (m / (1 - b1^k)) / (sqrt(v / (1 - b2^k)) + eps), in float32 with
 * b, 1 - b, lr and the bias corrections formed in double and rounded once.
 * Errors: ARG (bad settings, null buffers), DEVICE. */
int mgn_adam_step(const mgn_adam* adam, int64_t k, float* params,
                  const float* grad, float* m, float* v, int64_t n,
                  void* stream);

/* One patch-training step (Sec. 2.2 conditions 2 and 3; App. C): for each
 * patch in order, the noisy input y + std * noise of its nodes (ghost rows
 * from their owners), one step of the scheme with saved activations, the
 * squared error of the stepped state against y_target on its subdomain
 * nodes, and the backward pass into grad; then grad holds the gradient of
 * loss = sum over the patches' subdomain nodes and the 4 channels of
 * (y_step - y_target)^2 / (4 n_loss_nodes), and one Adam update (k-th) is
 * applied to params with the moments adam_m, adam_v.
 * static, y, y_target, noise (standard normal draws, nullable: no noise):
 * [n_global][4]; noise_std: host [4] (nullable: the paper's 3D values 0.02,
 * 0.02, 0.03, 0.05); grad, adam_m, adam_v: [mgn_param_count] (grad is
 * overwritten); loss: one device float (overwritten).  The context must have
 * been created with save and hold the largest patch.  n_loss_nodes is
 * normally the number of subdomain nodes of the given patches.
 * Errors: ARG, STATE (context without save), SHAPE, WORKSPACE, DEVICE. */
int mgn_train_step(mgn_ctx* ctx, int32_t n_patches, const mgn_dpatch* patches,
                   float* params, int32_t scheme, const float* static_feat,
                   const float* y, const float* y_target, const float* noise,
                   const float* noise_std, int64_t n_loss_nodes, float* grad,
                   float* adam_m, float* adam_v, const mgn_adam* adam, int64_t k,
                   float* loss, int64_t n_global, void* workspace,
                   size_t ws_bytes, void* stream);

/* One predict-evaluate-correct step at inference (the paper's outlook,
 * App. D: a higher-order update for one MGN evaluation per step): two-step
 * Adams-Bashforth predictor, trapezoidal corrector, MGN in place of h*f,
 *   y_p = y + 3/2 K_n - 1/2 K_n-1,  K_p = MGN([static, y_p]),
 *   y_next = y + 1/2 (K_p + K_n),   history <- (K_p, K_n).
 * khist [2][N][4] (device, in/out): khist[0] = K_n, khist[1] = K_n-1.  With
 * first != 0 the history is initialised first as K_0 = K_-1 = MGN([static,
 * y]) (one extra MGN call), which makes this step Heun's second-order step.
 * static, y, efeat, y_next as in mgn_integrate_step; y_next must not alias y
 * or khist.  No activations are saved (inference only).
 * Errors: those of mgn_integrate_step. */
int mgn_pec_step(mgn_ctx* ctx, const mgn_dgraph* g, const float* params,
                 const float* static_feat, const float* y, float* khist,
                 const float* efeat, float* y_next, int32_t first,
                 void* workspace, size_t ws_bytes, void* stream);

/* Per-kernel timing for benchmarks.  While enabled, every kernel launch of
 * the context is bracketed by two HIP events recorded on the caller's stream.
 * mgn_profile_collect waits for the last recorded event, then fills, for up
 * to max_kernels kernel kinds, the kind's name (NUL-terminated, 32 bytes per
 * entry in `names`), its summed duration in milliseconds and its launch
 * count; *n_kernels receives the number of kinds.  Collecting resets the
 * counters.  Events are created on first use and released by
 * mgn_ctx_destroy.  Errors: ARG, DEVICE. */
int mgn_profile_enable(mgn_ctx* ctx, int32_t enable);
int mgn_profile_collect(mgn_ctx* ctx, int32_t max_kernels, char* names,
                        double* total_ms, int64_t* launches,
                        int32_t* n_kernels);

/* Library version string and the last error message of this thread. */
const char* mgn_version(void);
const char* mgn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MGN_H */
