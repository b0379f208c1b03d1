// Host-side mesh graph construction, equal-split partition, ghost-zone patch
// extraction and the receiver-aligned tile schedule.
//
// Mesh edges come from the simplices of the mesh (App. B); the edge features
// are the MGN ones (App. C): sender-minus-receiver displacement and its
// length.  Subdomains and patches follow Sec. 2.2 and Fig. 1.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstring>
#include <limits>
#include <new>

#include "internal.hpp"

namespace mgn {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

const char* last_error() { return g_last_error.c_str(); }

void build_schedule(Graph& g) {
  g.tiles.clear();
  g.long_nodes.clear();
  const int64_t N = g.n_nodes;
  const int32_t* rp = g.rowptr.data();
  int32_t slot = 0;
  int64_t v = 0;
  while (v < N) {
    const int64_t deg = rp[v + 1] - rp[v];
    if (deg > kTileEdges) {
      const int32_t nch = (int32_t)((deg + kTileEdges - 1) / kTileEdges);
      g.long_nodes.insert(g.long_nodes.end(), {(int32_t)v, slot, nch, 0});
      for (int32_t c = 0; c < nch; ++c) {
        const int32_t eb = rp[v] + c * kTileEdges;
        const int32_t ee = std::min<int32_t>(eb + kTileEdges, rp[v + 1]);
        g.tiles.insert(g.tiles.end(), {(int32_t)v, -1 - slot, eb, ee});
        ++slot;
      }
      ++v;
      continue;
    }
    const int64_t nb = v;
    const int32_t eb = rp[v];
    while (v < N && (v - nb) < kTileNodes && rp[v + 1] - eb <= kTileEdges) ++v;
    g.tiles.insert(g.tiles.end(), {(int32_t)nb, (int32_t)v, eb, rp[v]});
  }
}

// rev[e] for every edge, by binary search in the sender's segment.
static bool fill_rev(Graph& g) {
  g.rev.resize(g.n_edges);
  for (int64_t r = 0; r < g.n_nodes; ++r) {
    for (int32_t e = g.rowptr[r]; e < g.rowptr[r + 1]; ++e) {
      const int32_t s = g.senders[e];
      const int32_t* b = g.senders.data() + g.rowptr[s];
      const int32_t* en = g.senders.data() + g.rowptr[s + 1];
      const int32_t* it = std::lower_bound(b, en, (int32_t)r);
      if (it == en || *it != (int32_t)r) return false;
      g.rev[e] = (int32_t)(it - g.senders.data());
    }
  }
  return true;
}

static void fill_efeat(Graph& g, const float* pos, int dim) {
  g.efeat.assign((size_t)g.n_edges * 4, 0.0f);
  for (int64_t e = 0; e < g.n_edges; ++e) {
    const int64_t s = g.senders[e], r = g.receivers[e];
    double d[3] = {0.0, 0.0, 0.0};
    for (int c = 0; c < dim; ++c)
      d[c] = (double)pos[s * dim + c] - (double)pos[r * dim + c];
    double sq = d[0] * d[0];
    for (int c = 1; c < dim; ++c) sq = sq + d[c] * d[c];
    const double nrm = std::sqrt(sq);
    for (int c = 0; c < dim; ++c) g.efeat[e * 4 + c] = (float)d[c];
    g.efeat[e * 4 + dim] = (float)nrm;
  }
}

}  // namespace mgn

using namespace mgn;

extern "C" {

const char* mgn_last_error(void) { return mgn::last_error(); }

int32_t mgn_tile_edges(void) { return kTileEdges; }
int32_t mgn_tile_nodes(void) { return kTileNodes; }

int mgn_build_graph(const int32_t* cells, int64_t n_cells, int32_t vpc,
                    const float* pos, int64_t n_nodes, int32_t dim,
                    mgn_graph** out) {
  if (!out || (!cells && n_cells > 0) || (!pos && n_nodes > 0))
    return fail(MGN_ERR_ARG, "mgn_build_graph: null pointer");
  if (n_cells < 0 || n_nodes < 0)
    return fail(MGN_ERR_ARG, "mgn_build_graph: negative size");
  if (vpc < 2 || vpc > 4)
    return fail(MGN_ERR_ARG, "mgn_build_graph: verts_per_cell must be 2, 3 or 4");
  if (dim != 2 && dim != 3)
    return fail(MGN_ERR_ARG, "mgn_build_graph: dim must be 2 or 3");
  if (n_nodes >= (int64_t)std::numeric_limits<int32_t>::max())
    return fail(MGN_ERR_SHAPE, "mgn_build_graph: too many nodes");
  const int64_t n_ent = n_cells * vpc;
  for (int64_t i = 0; i < n_ent; ++i)
    if (cells[i] < 0 || cells[i] >= n_nodes)
      return fail(MGN_ERR_RANGE, "mgn_build_graph: cell %lld vertex id %d outside [0,%lld)",
                  (long long)(i / vpc), cells[i], (long long)n_nodes);
  mgn_graph* h = nullptr;
  try {
    h = new mgn_graph();
    Graph& g = h->g;
    g.n_nodes = n_nodes;
    // counting sort of candidate (receiver, sender) pairs by receiver
    std::vector<int64_t> off(n_nodes + 1, 0);
    for (int64_t c = 0; c < n_cells; ++c) {
      const int32_t* cv = cells + c * vpc;
      for (int a = 0; a < vpc; ++a)
        for (int b = 0; b < vpc; ++b)
          if (a != b && cv[a] != cv[b]) ++off[cv[b] + 1];
    }
    for (int64_t v = 0; v < n_nodes; ++v) off[v + 1] += off[v];
    std::vector<int32_t> buf(off[n_nodes]);
    {
      std::vector<int64_t> fillp(off.begin(), off.end() - 1);
      for (int64_t c = 0; c < n_cells; ++c) {
        const int32_t* cv = cells + c * vpc;
        for (int a = 0; a < vpc; ++a)
          for (int b = 0; b < vpc; ++b)
            if (a != b && cv[a] != cv[b]) buf[fillp[cv[b]]++] = cv[a];
      }
    }
    // sort and deduplicate every receiver's senders, compacting in place
    g.rowptr.assign(n_nodes + 1, 0);
    int64_t w = 0;
    for (int64_t v = 0; v < n_nodes; ++v) {
      int32_t* b = buf.data() + off[v];
      int32_t* e = buf.data() + off[v + 1];
      std::sort(b, e);
      int32_t* u = std::unique(b, e);
      const int64_t cnt = u - b;
      if (w + cnt >= (int64_t)std::numeric_limits<int32_t>::max()) {
        delete h;
        return fail(MGN_ERR_SHAPE, "mgn_build_graph: edge count exceeds 2^31-1");
      }
      std::memmove(buf.data() + w, b, cnt * sizeof(int32_t));
      w += cnt;
      g.rowptr[v + 1] = (int32_t)w;
    }
    g.n_edges = w;
    buf.resize(w);
    buf.shrink_to_fit();
    g.senders.swap(buf);
    g.receivers.resize(w);
    for (int64_t v = 0; v < n_nodes; ++v)
      for (int32_t e = g.rowptr[v]; e < g.rowptr[v + 1]; ++e) g.receivers[e] = (int32_t)v;
    if (!fill_rev(g)) {
      delete h;
      return fail(MGN_ERR_STATE, "mgn_build_graph: internal error, graph not symmetric");
    }
    fill_efeat(g, pos, dim);
    build_schedule(g);
  } catch (const std::bad_alloc&) {
    delete h;
    return fail(MGN_ERR_NOMEM, "mgn_build_graph: out of host memory");
  }
  *out = h;
  return MGN_OK;
}

int mgn_graph_info(const mgn_graph* h, int64_t* n_nodes, int64_t* n_edges) {
  if (!h) return fail(MGN_ERR_ARG, "mgn_graph_info: null graph");
  if (n_nodes) *n_nodes = h->g.n_nodes;
  if (n_edges) *n_edges = h->g.n_edges;
  return MGN_OK;
}

int mgn_graph_copy(const mgn_graph* h, int32_t* rowptr, int32_t* senders,
                   int32_t* receivers, int32_t* rev, float* efeat) {
  if (!h) return fail(MGN_ERR_ARG, "mgn_graph_copy: null graph");
  const Graph& g = h->g;
  if (rowptr) std::memcpy(rowptr, g.rowptr.data(), (g.n_nodes + 1) * sizeof(int32_t));
  if (senders && g.n_edges) std::memcpy(senders, g.senders.data(), g.n_edges * sizeof(int32_t));
  if (receivers && g.n_edges) std::memcpy(receivers, g.receivers.data(), g.n_edges * sizeof(int32_t));
  if (rev && g.n_edges) std::memcpy(rev, g.rev.data(), g.n_edges * sizeof(int32_t));
  if (efeat && g.n_edges) std::memcpy(efeat, g.efeat.data(), g.n_edges * 4 * sizeof(float));
  return MGN_OK;
}

int mgn_graph_schedule(const mgn_graph* h, int32_t* tiles, int64_t* n_tiles,
                       int32_t* long_nodes, int64_t* n_long) {
  if (!h) return fail(MGN_ERR_ARG, "mgn_graph_schedule: null graph");
  const Graph& g = h->g;
  if (n_tiles) *n_tiles = (int64_t)g.tiles.size() / 4;
  if (n_long) *n_long = (int64_t)g.long_nodes.size() / 4;
  if (tiles && !g.tiles.empty())
    std::memcpy(tiles, g.tiles.data(), g.tiles.size() * sizeof(int32_t));
  if (long_nodes && !g.long_nodes.empty())
    std::memcpy(long_nodes, g.long_nodes.data(), g.long_nodes.size() * sizeof(int32_t));
  return MGN_OK;
}

void mgn_graph_destroy(mgn_graph* g) { delete g; }

int mgn_partition(const float* pos, int64_t n, int32_t dim,
                  const int32_t* splits, int32_t* part_out) {
  if ((!pos && n > 0) || !splits || (!part_out && n > 0))
    return fail(MGN_ERR_ARG, "mgn_partition: null pointer");
  if (n < 0 || dim < 1 || dim > 3)
    return fail(MGN_ERR_ARG, "mgn_partition: bad size or dim");
  int64_t total = 1;
  for (int a = 0; a < dim; ++a) {
    if (splits[a] < 1) return fail(MGN_ERR_ARG, "mgn_partition: splits must be >= 1");
    total *= splits[a];
  }
  if (total >= (int64_t)std::numeric_limits<int32_t>::max())
    return fail(MGN_ERR_ARG, "mgn_partition: too many subdomains");
  double lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0};
  for (int a = 0; a < dim; ++a) {
    lo[a] = std::numeric_limits<double>::infinity();
    hi[a] = -std::numeric_limits<double>::infinity();
    for (int64_t i = 0; i < n; ++i) {
      const double x = (double)pos[i * dim + a];
      lo[a] = std::min(lo[a], x);
      hi[a] = std::max(hi[a], x);
    }
  }
  for (int64_t i = 0; i < n; ++i) {
    int64_t id = 0, stride = 1;
    for (int a = 0; a < dim; ++a) {
      int64_t idx = 0;
      if (hi[a] > lo[a]) {
        const double x = (double)pos[i * dim + a];
        const double t = ((double)splits[a] * (x - lo[a])) / (hi[a] - lo[a]);
        idx = (int64_t)std::floor(t);
        idx = std::min<int64_t>(std::max<int64_t>(idx, 0), splits[a] - 1);
      }
      id += idx * stride;
      stride *= splits[a];
    }
    part_out[i] = (int32_t)id;
  }
  return MGN_OK;
}

int mgn_extract_patch(const mgn_graph* h, const int32_t* part, int32_t p,
                      int32_t k, mgn_graph** patch) {
  if (!h || !patch || (!part && h->g.n_nodes > 0))
    return fail(MGN_ERR_ARG, "mgn_extract_patch: null pointer");
  if (k < 0) return fail(MGN_ERR_ARG, "mgn_extract_patch: k must be >= 0");
  const Graph& g = h->g;
  const int64_t N = g.n_nodes;
  int32_t pmax = -1;
  for (int64_t v = 0; v < N; ++v) {
    if (part[v] < 0) return fail(MGN_ERR_RANGE, "mgn_extract_patch: negative subdomain id at node %lld", (long long)v);
    pmax = std::max(pmax, part[v]);
  }
  if (p < 0 || p > pmax)
    return fail(MGN_ERR_RANGE, "mgn_extract_patch: subdomain %d outside [0,%d]", p, pmax);
  mgn_graph* out = nullptr;
  try {
    out = new mgn_graph();
    Graph& q = out->g;
    q.is_patch = true;
    // multi-source breadth-first search up to k hops
    std::vector<int32_t> hop(N, -1);
    std::vector<int32_t> frontier, next;
    for (int64_t v = 0; v < N; ++v)
      if (part[v] == p) {
        hop[v] = 0;
        frontier.push_back((int32_t)v);
      }
    for (int32_t d = 1; d <= k && !frontier.empty(); ++d) {
      next.clear();
      for (int32_t v : frontier)
        for (int32_t e = g.rowptr[v]; e < g.rowptr[v + 1]; ++e) {
          const int32_t u = g.senders[e];
          if (hop[u] < 0) {
            hop[u] = d;
            next.push_back(u);
          }
        }
      frontier.swap(next);
    }
    std::vector<int32_t> g2l(N, -1);
    for (int64_t v = 0; v < N; ++v)
      if (hop[v] >= 0) {
        g2l[v] = (int32_t)q.node_l2g.size();
        q.node_l2g.push_back((int32_t)v);
        q.hop.push_back(hop[v]);
        if (hop[v] == 0) ++q.n_interior;
      }
    q.n_nodes = (int64_t)q.node_l2g.size();
    q.rowptr.assign(q.n_nodes + 1, 0);
    // induced edges; ascending local ids keep the (receiver, sender) order
    for (int64_t lv = 0; lv < q.n_nodes; ++lv) {
      const int32_t v = q.node_l2g[lv];
      for (int32_t e = g.rowptr[v]; e < g.rowptr[v + 1]; ++e) {
        const int32_t ls = g2l[g.senders[e]];
        if (ls < 0) continue;
        q.senders.push_back(ls);
        q.receivers.push_back((int32_t)lv);
        q.edge_l2g.push_back(e);
      }
      q.rowptr[lv + 1] = (int32_t)q.senders.size();
    }
    q.n_edges = (int64_t)q.senders.size();
    if (!fill_rev(q)) {
      delete out;
      return fail(MGN_ERR_STATE, "mgn_extract_patch: internal error, patch not symmetric");
    }
    q.efeat.resize((size_t)q.n_edges * 4);
    for (int64_t le = 0; le < q.n_edges; ++le)
      std::memcpy(&q.efeat[le * 4], &g.efeat[q.edge_l2g[le] * 4], 4 * sizeof(float));
    build_schedule(q);
  } catch (const std::bad_alloc&) {
    delete out;
    return fail(MGN_ERR_NOMEM, "mgn_extract_patch: out of host memory");
  }
  *patch = out;
  return MGN_OK;
}

int mgn_patch_union(const mgn_graph* const* patches, int32_t n, mgn_graph** out) {
  if (!out || n < 0 || (n > 0 && !patches)) return fail(MGN_ERR_ARG, "mgn_patch_union: bad arguments");
  int64_t N = 0, E = 0;
  for (int32_t j = 0; j < n; ++j) {
    if (!patches[j]) return fail(MGN_ERR_ARG, "mgn_patch_union: patch %d is null", j);
    if (!patches[j]->g.is_patch) return fail(MGN_ERR_STATE, "mgn_patch_union: graph %d is not a patch", j);
    N += patches[j]->g.n_nodes;
    E += patches[j]->g.n_edges;
  }
  if (N >= (int64_t)INT32_MAX || E >= (int64_t)INT32_MAX)
    return fail(MGN_ERR_SHAPE, "mgn_patch_union: %lld nodes / %lld edges do not fit int32", (long long)N,
                (long long)E);
  mgn_graph* res = nullptr;
  try {
    res = new mgn_graph();
    Graph& q = res->g;
    q.is_patch = true;
    q.n_nodes = N;
    q.n_edges = E;
    q.rowptr.reserve(N + 1);
    q.rowptr.push_back(0);
    q.senders.reserve(E);
    q.receivers.reserve(E);
    q.rev.reserve(E);
    q.efeat.reserve((size_t)E * 4);
    q.node_l2g.reserve(N);
    q.hop.reserve(N);
    q.edge_l2g.reserve(E);
    int32_t nb = 0, eb = 0;  // node and edge offsets of the current part
    for (int32_t j = 0; j < n; ++j) {
      const Graph& g = patches[j]->g;
      for (int64_t v = 0; v < g.n_nodes; ++v) q.rowptr.push_back(eb + g.rowptr[v + 1]);
      for (int64_t e = 0; e < g.n_edges; ++e) {
        q.senders.push_back(nb + g.senders[e]);
        q.receivers.push_back(nb + g.receivers[e]);
        q.rev.push_back(eb + g.rev[e]);
      }
      q.efeat.insert(q.efeat.end(), g.efeat.begin(), g.efeat.end());
      q.node_l2g.insert(q.node_l2g.end(), g.node_l2g.begin(), g.node_l2g.end());
      q.hop.insert(q.hop.end(), g.hop.begin(), g.hop.end());
      q.edge_l2g.insert(q.edge_l2g.end(), g.edge_l2g.begin(), g.edge_l2g.end());
      q.n_interior += g.n_interior;
      nb += (int32_t)g.n_nodes;
      eb += (int32_t)g.n_edges;
    }
    build_schedule(q);
  } catch (const std::bad_alloc&) {
    delete res;
    return fail(MGN_ERR_NOMEM, "mgn_patch_union: out of host memory");
  }
  *out = res;
  return MGN_OK;
}

int mgn_patch_copy_maps(const mgn_graph* h, int32_t* node_l2g, int32_t* hop,
                        uint8_t* interior, int64_t* edge_l2g,
                        int64_t* n_interior) {
  if (!h) return fail(MGN_ERR_ARG, "mgn_patch_copy_maps: null graph");
  const Graph& g = h->g;
  if (!g.is_patch) return fail(MGN_ERR_STATE, "mgn_patch_copy_maps: not a patch");
  if (node_l2g && g.n_nodes) std::memcpy(node_l2g, g.node_l2g.data(), g.n_nodes * sizeof(int32_t));
  if (hop && g.n_nodes) std::memcpy(hop, g.hop.data(), g.n_nodes * sizeof(int32_t));
  if (interior)
    for (int64_t v = 0; v < g.n_nodes; ++v) interior[v] = g.hop[v] == 0 ? 1 : 0;
  if (edge_l2g && g.n_edges) std::memcpy(edge_l2g, g.edge_l2g.data(), g.n_edges * sizeof(int64_t));
  if (n_interior) *n_interior = g.n_interior;
  return MGN_OK;
}

}  // extern "C"
