// Internal declarations shared by the host-side sources of libmgn.
#pragma once

#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/mgn.h"

namespace mgn {

// Receiver-aligned edge tiles: at most this many edges and nodes per tile.
constexpr int kTileEdges = 32;
constexpr int kTileNodes = 32;
// Node kernels process this many consecutive nodes per tile.
constexpr int kNodeTile = 32;

void set_error(const char* fmt, ...);

// Returned by the C-ABI functions: records the message, returns the code.
int fail(int code, const char* fmt, ...);

struct Graph {
  int64_t n_nodes = 0;
  int64_t n_edges = 0;
  std::vector<int32_t> rowptr;     // [N+1]
  std::vector<int32_t> senders;    // [E]
  std::vector<int32_t> receivers;  // [E]
  std::vector<int32_t> rev;        // [E]
  std::vector<float> efeat;        // [E*4]
  std::vector<int32_t> tiles;      // [n_tiles*4]
  std::vector<int32_t> long_nodes; // [n_long*4]
  // patch maps (is_patch only)
  bool is_patch = false;
  std::vector<int32_t> node_l2g;
  std::vector<int32_t> hop;
  std::vector<int64_t> edge_l2g;
  int64_t n_interior = 0;
};

// Greedy receiver-aligned tiling (see mgn_graph_schedule in mgn.h).
void build_schedule(Graph& g);

// Workspace bytes planned by a context (mgn_ctx_create's *ws_bytes).
size_t ctx_workspace_bytes(const mgn_ctx* ctx);

// mgn_forward without saved activations into the given scratch (the body of
// mgn_forward_noalloc): per-kernel profiling events are not recorded.
int forward_in_scratch(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, const float* node_in,
                       const float* efeat, float* out, void* scratch, size_t scratch_bytes, void* stream);

// Upper bound on the number of chunk slots a graph with E edges can need.
inline int64_t max_slots(int64_t n_edges) {
  return 2 * (n_edges / kTileEdges) + 2;
}

}  // namespace mgn

struct mgn_graph {
  mgn::Graph g;
};
