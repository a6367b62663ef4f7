// Host-side graph compilation: reverse Cuthill-McKee ordering, bandwidth and
// block-band packing (Compilation section and Eq. 3 of arXiv 1906.11786).
// Plain C++17, no HIP: these run once per graph, before any device work.

#include <algorithm>
#include <cstring>
#include <new>
#include <tuple>
#include <utility>
#include <vector>

#include "common.h"

namespace ggnn {

static thread_local std::string g_last_error;

ggnn_status fail(ggnn_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = std::string(ggnn_status_string(st)) + ": " + buf;
  return st;
}

void clear_error() { g_last_error.clear(); }

namespace {

// Undirected simple graph in CSR form: the union of all edge types with both
// directions, self-loops and repeated pairs removed.  Each neighbour list is
// sorted by (degree, label), the order in which the search visits them.
struct SymGraph {
  std::vector<int64_t> off;
  std::vector<int32_t> adj;
  std::vector<int32_t> deg;
};

SymGraph build_sym(int32_t n, int64_t m, const int32_t* src, const int32_t* dst) {
  SymGraph g;
  std::vector<std::pair<int32_t, int32_t>> pairs;
  pairs.reserve(static_cast<size_t>(2 * m));
  for (int64_t k = 0; k < m; ++k) {
    if (src[k] == dst[k]) continue;
    pairs.emplace_back(src[k], dst[k]);
    pairs.emplace_back(dst[k], src[k]);
  }
  std::sort(pairs.begin(), pairs.end());
  pairs.erase(std::unique(pairs.begin(), pairs.end()), pairs.end());
  g.off.assign(static_cast<size_t>(n) + 1, 0);
  for (auto& p : pairs) g.off[p.first + 1]++;
  for (int32_t v = 0; v < n; ++v) g.off[v + 1] += g.off[v];
  g.adj.resize(pairs.size());
  for (size_t k = 0; k < pairs.size(); ++k) g.adj[k] = pairs[k].second;  // already grouped by first
  g.deg.resize(n);
  for (int32_t v = 0; v < n; ++v) g.deg[v] = static_cast<int32_t>(g.off[v + 1] - g.off[v]);
  for (int32_t v = 0; v < n; ++v) {
    std::sort(g.adj.begin() + g.off[v], g.adj.begin() + g.off[v + 1], [&](int32_t a, int32_t b) {
      return g.deg[a] != g.deg[b] ? g.deg[a] < g.deg[b] : a < b;
    });
  }
  return g;
}

inline bool less_deg_label(const SymGraph& g, int32_t a, int32_t b) {
  return g.deg[a] != g.deg[b] ? g.deg[a] < g.deg[b] : a < b;
}

// Breadth-first level structure rooted at `root`.  Fills `nodes` with the
// visit order and returns the number of levels; `last_begin` receives the
// index in `nodes` where the deepest level starts.  `stamp`/`cur` mark
// visited nodes without clearing between calls.
int32_t level_structure(const SymGraph& g, int32_t root, std::vector<int32_t>& stamp, int32_t cur,
                        std::vector<int32_t>& nodes, size_t& last_begin) {
  nodes.clear();
  nodes.push_back(root);
  stamp[root] = cur;
  size_t lo = 0, hi = 1;
  int32_t levels = 1;
  last_begin = 0;
  while (true) {
    for (size_t q = lo; q < hi; ++q) {
      int32_t v = nodes[q];
      for (int64_t k = g.off[v]; k < g.off[v + 1]; ++k) {
        int32_t w = g.adj[k];
        if (stamp[w] != cur) {
          stamp[w] = cur;
          nodes.push_back(w);
        }
      }
    }
    if (nodes.size() == hi) break;
    last_begin = hi;
    lo = hi;
    hi = nodes.size();
    ++levels;
  }
  return levels;
}

}  // namespace
}  // namespace ggnn

using namespace ggnn;

extern "C" {

int ggnn_abi_version(void) { return GGNN_ABI_VERSION; }

const char* ggnn_last_error(void) { return g_last_error.c_str(); }

const char* ggnn_status_string(ggnn_status s) {
  switch (s) {
    case GGNN_OK: return "GGNN_OK";
    case GGNN_ERR_INVALID_ARG: return "GGNN_ERR_INVALID_ARG";
    case GGNN_ERR_UNSUPPORTED: return "GGNN_ERR_UNSUPPORTED";
    case GGNN_ERR_OUT_OF_BAND: return "GGNN_ERR_OUT_OF_BAND";
    case GGNN_ERR_DEVICE: return "GGNN_ERR_DEVICE";
    case GGNN_ERR_HOST_ALLOC: return "GGNN_ERR_HOST_ALLOC";
    case GGNN_ERR_WORKSPACE: return "GGNN_ERR_WORKSPACE";
  }
  return "GGNN_ERR_UNKNOWN";
}

ggnn_status ggnn_bandwidth(int32_t n, int64_t m, const int32_t* src, const int32_t* dst, const int32_t* rank,
                           int32_t* bandwidth) {
  clear_error();
  GGNN_CHECK_ARG(n >= 0 && m >= 0, "n=%d m=%lld must be >= 0", n, (long long)m);
  GGNN_CHECK_ARG(bandwidth != nullptr, "bandwidth is NULL");
  GGNN_CHECK_ARG(m == 0 || (src && dst), "src/dst is NULL");
  if (rank != nullptr)
    for (int32_t v = 0; v < n; ++v)
      GGNN_CHECK_ARG(rank[v] >= 0 && rank[v] < n, "rank[%d]=%d out of range [0,%d)", v, rank[v], n);
  int32_t bw = 0;
  for (int64_t k = 0; k < m; ++k) {
    int32_t s = src[k], d = dst[k];
    GGNN_CHECK_ARG(s >= 0 && s < n && d >= 0 && d < n, "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, s,
                   d, n);
    if (rank) {
      s = rank[s];
      d = rank[d];
    }
    int32_t span = s > d ? s - d : d - s;
    bw = std::max(bw, span);
  }
  *bandwidth = bw;
  return GGNN_OK;
}

ggnn_status ggnn_rcm_order(int32_t n, int64_t m, const int32_t* src, const int32_t* dst, int32_t* order,
                           int32_t* rank, int32_t* bandwidth) {
  clear_error();
  GGNN_CHECK_ARG(n >= 0 && m >= 0, "n=%d m=%lld must be >= 0", n, (long long)m);
  GGNN_CHECK_ARG(m == 0 || (src && dst), "src/dst is NULL");
  GGNN_CHECK_ARG(n == 0 || (order && rank), "order/rank is NULL");
  for (int64_t k = 0; k < m; ++k)
    GGNN_CHECK_ARG(src[k] >= 0 && src[k] < n && dst[k] >= 0 && dst[k] < n,
                   "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, src[k], dst[k], n);
  try {
    SymGraph g = build_sym(n, m, src, dst);
    std::vector<int32_t> stamp(n, -1), nodes, seq;
    std::vector<char> visited(n, 0);
    seq.reserve(n);
    int32_t cur = 0;
    for (int32_t v0 = 0; v0 < n; ++v0) {
      if (visited[v0]) continue;
      size_t last = 0;
      level_structure(g, v0, stamp, cur++, nodes, last);
      int32_t root = nodes[0];
      for (int32_t v : nodes)
        if (less_deg_label(g, v, root)) root = v;
      // George-Liu: move to the smallest (degree, label) node of the deepest
      // level while that deepens the level structure.
      int32_t depth = level_structure(g, root, stamp, cur++, nodes, last);
      while (true) {
        int32_t cand = nodes[last];
        for (size_t q = last; q < nodes.size(); ++q)
          if (less_deg_label(g, nodes[q], cand)) cand = nodes[q];
        std::vector<int32_t> cnodes;
        size_t clast = 0;
        int32_t cdepth = level_structure(g, cand, stamp, cur++, cnodes, clast);
        if (cdepth > depth) {
          root = cand;
          depth = cdepth;
          nodes.swap(cnodes);
          last = clast;
        } else {
          break;
        }
      }
      // Cuthill-McKee search from the root.
      size_t head = seq.size();
      seq.push_back(root);
      visited[root] = 1;
      while (head < seq.size()) {
        int32_t x = seq[head++];
        for (int64_t k = g.off[x]; k < g.off[x + 1]; ++k) {
          int32_t w = g.adj[k];
          if (!visited[w]) {
            visited[w] = 1;
            seq.push_back(w);
          }
        }
      }
    }
    for (int32_t p = 0; p < n; ++p) order[p] = seq[n - 1 - p];
    for (int32_t p = 0; p < n; ++p) rank[order[p]] = p;
  } catch (const std::bad_alloc&) {
    return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed (n=%d, m=%lld)", n, (long long)m);
  }
  if (bandwidth) return ggnn_bandwidth(n, m, src, dst, rank, bandwidth);
  return GGNN_OK;
}

ggnn_status ggnn_batch_graphs(int32_t n_graphs, const int32_t* node_counts, const int64_t* edge_counts,
                              const int32_t* src, const int32_t* dst, int32_t reorder, int32_t* out_src,
                              int32_t* out_dst, int64_t* offsets, int32_t* bandwidth) {
  clear_error();
  GGNN_CHECK_ARG(n_graphs >= 0, "n_graphs=%d must be >= 0", n_graphs);
  GGNN_CHECK_ARG(reorder == 0 || reorder == 1, "reorder=%d must be 0 or 1", reorder);
  GGNN_CHECK_ARG(offsets != nullptr && bandwidth != nullptr, "offsets/bandwidth is NULL");
  GGNN_CHECK_ARG(n_graphs == 0 || (node_counts && edge_counts), "node_counts/edge_counts is NULL");
  int64_t total_n = 0, total_m = 0;
  for (int32_t i = 0; i < n_graphs; ++i) {
    GGNN_CHECK_ARG(node_counts[i] >= 0 && edge_counts[i] >= 0, "graph %d: node count %d, edge count %lld must be >= 0",
                   i, node_counts[i], (long long)edge_counts[i]);
    total_n += node_counts[i];
    total_m += edge_counts[i];
    GGNN_CHECK_ARG(total_n < ((int64_t)1 << 31), "more than 2^31 - 1 nodes in all");
  }
  GGNN_CHECK_ARG(total_m == 0 || (src && dst && out_src && out_dst), "src/dst/out_src/out_dst is NULL");
  offsets[0] = 0;
  int32_t bw = 0;
  int64_t e0 = 0;
  try {
    std::vector<int32_t> order, rank;
    for (int32_t i = 0; i < n_graphs; ++i) {
      const int32_t n = node_counts[i];
      const int64_t m = edge_counts[i];
      const int32_t* s = src + e0;
      const int32_t* d = dst + e0;
      const int32_t off = (int32_t)offsets[i];
      int32_t b = 0;
      ggnn_status st;
      if (reorder) {
        order.resize(n);
        rank.resize(n);
        st = ggnn_rcm_order(n, m, s, d, order.data(), rank.data(), &b);
      } else {
        st = ggnn_bandwidth(n, m, s, d, nullptr, &b);
      }
      if (st != GGNN_OK) {
        const std::string why = g_last_error;
        return fail(st, "graph %d: %s", i, why.c_str());
      }
      for (int64_t k = 0; k < m; ++k) {
        out_src[e0 + k] = (reorder ? rank[s[k]] : s[k]) + off;
        out_dst[e0 + k] = (reorder ? rank[d[k]] : d[k]) + off;
      }
      bw = std::max(bw, b);
      offsets[i + 1] = offsets[i] + n;
      e0 += m;
    }
  } catch (const std::bad_alloc&) {
    return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed (%d graphs)", n_graphs);
  }
  *bandwidth = bw;
  return GGNN_OK;
}

ggnn_status ggnn_batch_graphs_super(int32_t n_graphs, const int32_t* node_counts, const int64_t* edge_counts,
                                    const int32_t* src, const int32_t* dst, const int32_t* hub_counts,
                                    const int32_t* hubs, int32_t s, int32_t* out_src, int32_t* out_dst,
                                    int32_t* n_nodes, int32_t* bandwidth) {
  clear_error();
  GGNN_CHECK_ARG(n_graphs >= 0 && s >= 0, "n_graphs=%d and s=%d must be >= 0", n_graphs, s);
  GGNN_CHECK_ARG(n_nodes != nullptr && bandwidth != nullptr, "n_nodes/bandwidth is NULL");
  GGNN_CHECK_ARG(n_graphs == 0 || (node_counts && edge_counts && hub_counts), "node/edge/hub counts are NULL");
  int64_t total_n = s, total_m = 0, total_h = 0;
  for (int32_t i = 0; i < n_graphs; ++i) {
    GGNN_CHECK_ARG(node_counts[i] >= 0 && edge_counts[i] >= 0 && hub_counts[i] >= 0 && hub_counts[i] <= node_counts[i],
                   "graph %d: node count %d, edge count %lld, hub count %d out of range", i, node_counts[i],
                   (long long)edge_counts[i], hub_counts[i]);
    total_n += node_counts[i] - hub_counts[i];
    total_m += edge_counts[i];
    total_h += hub_counts[i];
    GGNN_CHECK_ARG(total_n < ((int64_t)1 << 31), "more than 2^31 - 1 nodes in all");
  }
  GGNN_CHECK_ARG(total_h <= s, "%lld hubs do not fit in s=%d supernode slots", (long long)total_h, s);
  GGNN_CHECK_ARG(total_h == 0 || hubs, "hubs is NULL");
  GGNN_CHECK_ARG(total_m == 0 || (src && dst && out_src && out_dst), "src/dst/out_src/out_dst is NULL");
  int32_t bw = 0, next_hub = 0, base = s;
  int64_t e0 = 0, h0 = 0;
  try {
    std::vector<int32_t> label, local, is, id, order, rank;
    for (int32_t i = 0; i < n_graphs; ++i) {
      const int32_t n = node_counts[i];
      const int64_t m = edge_counts[i];
      const int32_t* gs = src + e0;
      const int32_t* gd = dst + e0;
      label.assign(n, -1);
      for (int32_t j = 0; j < hub_counts[i]; ++j) {
        const int32_t v = hubs[h0 + j];
        GGNN_CHECK_ARG(v >= 0 && v < n && label[v] < 0, "graph %d: hub %d is out of range [0,%d) or repeated", i, v,
                       n);
        label[v] = next_hub++;
      }
      for (int64_t k = 0; k < m; ++k)
        GGNN_CHECK_ARG(gs[k] >= 0 && gs[k] < n && gd[k] >= 0 && gd[k] < n,
                       "graph %d: edge %lld (%d -> %d) out of range [0,%d)", i, (long long)k, gs[k], gd[k], n);
      // the other nodes, in label order, and the edges between them (the band's share)
      local.assign(n, -1);
      int32_t nr = 0;
      for (int32_t v = 0; v < n; ++v)
        if (label[v] < 0) local[v] = nr++;
      is.clear();
      id.clear();
      for (int64_t k = 0; k < m; ++k)
        if (label[gs[k]] < 0 && label[gd[k]] < 0) {
          is.push_back(local[gs[k]]);
          id.push_back(local[gd[k]]);
        }
      order.resize(nr);
      rank.resize(nr);
      int32_t b = 0;
      const ggnn_status st = ggnn_rcm_order(nr, (int64_t)is.size(), is.data(), id.data(), order.data(), rank.data(), &b);
      if (st != GGNN_OK) {
        const std::string why = g_last_error;
        return fail(st, "graph %d: %s", i, why.c_str());
      }
      for (int32_t v = 0; v < n; ++v)
        if (label[v] < 0) label[v] = base + rank[local[v]];
      for (int64_t k = 0; k < m; ++k) {
        out_src[e0 + k] = label[gs[k]];
        out_dst[e0 + k] = label[gd[k]];
      }
      bw = std::max(bw, b);
      base += nr;
      e0 += m;
      h0 += hub_counts[i];
    }
  } catch (const std::bad_alloc&) {
    return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed (%d graphs)", n_graphs);
  }
  *n_nodes = base;
  *bandwidth = bw;
  return GGNN_OK;
}

size_t ggnn_band_bytes(int32_t n_pad, int32_t E, int32_t B, ggnn_dtype dt) {
  if (n_pad <= 0 || E <= 0 || B <= 0 || n_pad % B != 0 || !supported_dtype(dt)) return 0;
  size_t nb = static_cast<size_t>(n_pad / B);
  return static_cast<size_t>(E) * nb * 3 * static_cast<size_t>(B) * static_cast<size_t>(B) * dtype_bytes(dt);
}

ggnn_status ggnn_banded_pack(int32_t n_pad, int32_t E, int32_t B, int64_t m, const int32_t* src, const int32_t* dst,
                             const int32_t* etype, const int32_t* rank, ggnn_dtype dt, int strict, void* band,
                             int64_t* n_packed, int64_t* n_dropped, int64_t* n_duplicate) {
  clear_error();
  GGNN_CHECK_ARG(supported_dtype(dt), "unknown dtype %d", (int)dt);
  GGNN_CHECK_ARG(B >= 1 && n_pad >= B && n_pad % B == 0, "n_pad=%d must be a positive multiple of B=%d", n_pad, B);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  GGNN_CHECK_ARG(m >= 0, "m=%lld must be >= 0", (long long)m);
  GGNN_CHECK_ARG(m == 0 || (src && dst && etype), "src/dst/etype is NULL");
  GGNN_CHECK_ARG(band != nullptr, "band is NULL");
  const int64_t nb = n_pad / B;
  if (rank)
    for (int32_t v = 0; v < n_pad; ++v)
      GGNN_CHECK_ARG(rank[v] >= 0 && rank[v] < n_pad, "rank[%d]=%d out of range [0,%d)", v, rank[v], n_pad);
  for (int64_t k = 0; k < m; ++k) {
    GGNN_CHECK_ARG(src[k] >= 0 && src[k] < n_pad && dst[k] >= 0 && dst[k] < n_pad,
                   "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, src[k], dst[k], n_pad);
    GGNN_CHECK_ARG(etype[k] >= 0 && etype[k] < E, "edge %lld has type %d outside [0,%d)", (long long)k, etype[k],
                   E);
  }
  const size_t elems = ggnn_band_bytes(n_pad, E, B, dt) / dtype_bytes(dt);
  std::memset(band, 0, elems * dtype_bytes(dt));
  int64_t packed = 0, dup = 0;
  std::vector<std::tuple<int32_t, int64_t, int64_t>> out_of_band;  // distinct dropped edges are counted once
  const size_t BB = static_cast<size_t>(B) * B;
  for (int64_t k = 0; k < m; ++k) {
    int64_t i = rank ? rank[dst[k]] : dst[k];
    int64_t j = rank ? rank[src[k]] : src[k];
    int64_t kr = i / B, kc = j / B;
    int64_t s = kc - kr + 1;
    if (s < 0 || s > 2) {
      try {
        out_of_band.emplace_back(etype[k], i, j);
      } catch (const std::bad_alloc&) {
        return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed");
      }
      continue;
    }
    size_t idx = ((static_cast<size_t>(etype[k]) * nb + kr) * 3 + s) * BB + static_cast<size_t>(i % B) * B + (j % B);
    if (dt == GGNN_F32) {
      float* p = static_cast<float*>(band) + idx;
      if (*p != 0.0f) { ++dup; continue; }
      *p = 1.0f;
    } else {
      uint16_t* p = static_cast<uint16_t*>(band) + idx;
      if (*p != 0) { ++dup; continue; }
      *p = 0x3F80;  // bf16 bit pattern of 1.0
    }
    ++packed;
  }
  std::sort(out_of_band.begin(), out_of_band.end());
  const int64_t n_oob = static_cast<int64_t>(out_of_band.size());
  const int64_t dropped = static_cast<int64_t>(std::unique(out_of_band.begin(), out_of_band.end()) - out_of_band.begin());
  dup += n_oob - dropped;
  if (n_packed) *n_packed = packed;
  if (n_dropped) *n_dropped = dropped;
  if (n_duplicate) *n_duplicate = dup;
  if (strict && dropped > 0)
    return fail(GGNN_ERR_OUT_OF_BAND, "%lld edge(s) fall outside the three block diagonals (B=%d)",
                (long long)dropped, B);
  return GGNN_OK;
}

size_t ggnn_band_bits_bytes(int32_t n_pad, int32_t E, int32_t B) {
  if (n_pad <= 0 || E <= 0 || B < 8 || B % 8 != 0 || n_pad % B != 0) return 0;
  return static_cast<size_t>(E) * static_cast<size_t>(n_pad / B) * 3 * static_cast<size_t>(B) * (B / 8);
}

ggnn_status ggnn_banded_pack_bits(int32_t n_pad, int32_t E, int32_t B, int64_t m, const int32_t* src,
                                  const int32_t* dst, const int32_t* etype, const int32_t* rank, int strict,
                                  void* bits, void* bits_t, int64_t* n_packed, int64_t* n_dropped,
                                  int64_t* n_duplicate) {
  clear_error();
  GGNN_CHECK_ARG(B >= 8 && B % 8 == 0 && n_pad >= B && n_pad % B == 0,
                 "n_pad=%d must be a positive multiple of B=%d, B a multiple of 8", n_pad, B);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  GGNN_CHECK_ARG(m >= 0, "m=%lld must be >= 0", (long long)m);
  GGNN_CHECK_ARG(m == 0 || (src && dst && etype), "src/dst/etype is NULL");
  GGNN_CHECK_ARG(bits != nullptr, "bits is NULL");
  const int64_t nb = n_pad / B;
  if (rank)
    for (int32_t v = 0; v < n_pad; ++v)
      GGNN_CHECK_ARG(rank[v] >= 0 && rank[v] < n_pad, "rank[%d]=%d out of range [0,%d)", v, rank[v], n_pad);
  for (int64_t k = 0; k < m; ++k) {
    GGNN_CHECK_ARG(src[k] >= 0 && src[k] < n_pad && dst[k] >= 0 && dst[k] < n_pad,
                   "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, src[k], dst[k], n_pad);
    GGNN_CHECK_ARG(etype[k] >= 0 && etype[k] < E, "edge %lld has type %d outside [0,%d)", (long long)k, etype[k],
                   E);
  }
  const size_t nbytes = ggnn_band_bits_bytes(n_pad, E, B);
  uint8_t* out = static_cast<uint8_t*>(bits);
  uint8_t* out_t = static_cast<uint8_t*>(bits_t);
  std::memset(out, 0, nbytes);
  if (out_t) std::memset(out_t, 0, nbytes);
  const size_t row_bytes = static_cast<size_t>(B / 8);
  const size_t blk = static_cast<size_t>(B) * row_bytes;
  int64_t packed = 0, dup = 0;
  std::vector<std::tuple<int32_t, int64_t, int64_t>> out_of_band;
  for (int64_t k = 0; k < m; ++k) {
    const int64_t i = rank ? rank[dst[k]] : dst[k];
    const int64_t j = rank ? rank[src[k]] : src[k];
    const int64_t ki = i / B, kj = j / B;
    const int64_t s = kj - ki + 1;
    if (s < 0 || s > 2) {
      try {
        out_of_band.emplace_back(etype[k], i, j);
      } catch (const std::bad_alloc&) {
        return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed");
      }
      continue;
    }
    const int64_t r = i % B, c = j % B;
    // row r of block (e, ki, s), bit c
    uint8_t* byte = out + ((static_cast<size_t>(etype[k]) * nb + ki) * 3 + s) * blk + r * row_bytes + c / 8;
    const uint8_t bit = static_cast<uint8_t>(1u << (c % 8));
    if (*byte & bit) {
      ++dup;
      continue;
    }
    *byte |= bit;
    ++packed;
    if (out_t) {
      // transposed block: row c of block (e, kj, 2 - s), bit r
      uint8_t* tb = out_t + ((static_cast<size_t>(etype[k]) * nb + kj) * 3 + (2 - s)) * blk + c * row_bytes + r / 8;
      *tb |= static_cast<uint8_t>(1u << (r % 8));
    }
  }
  std::sort(out_of_band.begin(), out_of_band.end());
  const int64_t n_oob = static_cast<int64_t>(out_of_band.size());
  const int64_t dropped = static_cast<int64_t>(std::unique(out_of_band.begin(), out_of_band.end()) - out_of_band.begin());
  dup += n_oob - dropped;
  if (n_packed) *n_packed = packed;
  if (n_dropped) *n_dropped = dropped;
  if (n_duplicate) *n_duplicate = dup;
  if (strict && dropped > 0)
    return fail(GGNN_ERR_OUT_OF_BAND, "%lld edge(s) fall outside the three block diagonals (B=%d)",
                (long long)dropped, B);
  return GGNN_OK;
}

// Receiver-major lists of all edges, deduplicated (A_e has entries in
// {0, 1}): the sparse form of sum_e A_e X used to evaluate on every edge.
ggnn_status ggnn_sparse_csr(int32_t n_pad, int32_t E, int64_t m, const int32_t* src, const int32_t* dst,
                            const int32_t* etype, int32_t* row_ptr, int32_t* col, int64_t* nnz,
                            int64_t* n_duplicate) {
  clear_error();
  GGNN_CHECK_ARG(n_pad > 0, "n_pad=%d must be positive", n_pad);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  GGNN_CHECK_ARG(m >= 0 && m < ((int64_t)1 << 31), "m=%lld must be in [0, 2^31)", (long long)m);
  GGNN_CHECK_ARG(m == 0 || (src && dst && etype), "src/dst/etype is NULL");
  GGNN_CHECK_ARG(row_ptr != nullptr && (m == 0 || col != nullptr), "row_ptr/col is NULL");
  GGNN_CHECK_ARG((int64_t)n_pad * E < ((int64_t)1 << 31), "n_pad*E exceeds 2^31");
  for (int64_t k = 0; k < m; ++k) {
    GGNN_CHECK_ARG(src[k] >= 0 && src[k] < n_pad && dst[k] >= 0 && dst[k] < n_pad,
                   "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, src[k], dst[k], n_pad);
    GGNN_CHECK_ARG(etype[k] >= 0 && etype[k] < E, "edge %lld has type %d outside [0,%d)", (long long)k, etype[k],
                   E);
  }
  // (receiver, type, sender) keys, sorted and made unique
  std::vector<int64_t> key;
  try {
    key.resize(static_cast<size_t>(m));
  } catch (const std::bad_alloc&) {
    return fail(GGNN_ERR_HOST_ALLOC, "temporary allocation failed");
  }
  for (int64_t k = 0; k < m; ++k)
    key[k] = ((static_cast<int64_t>(dst[k]) * E + etype[k]) << 31) | static_cast<int64_t>(src[k]);
  std::sort(key.begin(), key.end());
  const int64_t uniq = static_cast<int64_t>(std::unique(key.begin(), key.end()) - key.begin());
  const int64_t rows = static_cast<int64_t>(n_pad) * E;
  int64_t r = 0;
  row_ptr[0] = 0;
  for (int64_t k = 0; k < uniq; ++k) {
    const int64_t row = key[k] >> 31;
    while (r < row) row_ptr[++r] = static_cast<int32_t>(k);
    col[k] = static_cast<int32_t>(key[k] & 0x7FFFFFFF);
  }
  while (r < rows) row_ptr[++r] = static_cast<int32_t>(uniq);
  if (nnz) *nnz = uniq;
  if (n_duplicate) *n_duplicate = m - uniq;
  return GGNN_OK;
}

// Dense 1-bit slices of the first s rows and columns (supernodes 0 .. s-1):
// rows [E][s][n_pad/8] holds edges into a supernode, cols [E][n_pad][s/8]
// edges out of a supernode into any other node; rows_t / cols_t (optional)
// their transposes with the same two layouts swapped.  Every other edge is
// counted in *n_rest (the band's).
size_t ggnn_super_bytes(int32_t n_pad, int32_t E, int32_t s) {
  if (n_pad <= 0 || n_pad % 64 != 0 || E < 1 || E > 64 || s < 32 || s > 128 || s % 32 != 0 || s > n_pad) return 0;
  return static_cast<size_t>(E) * s * (n_pad / 8);
}

ggnn_status ggnn_super_pack(int32_t n_pad, int32_t E, int32_t s, int64_t m, const int32_t* src, const int32_t* dst,
                            const int32_t* etype, void* rows, void* cols, void* rows_t, void* cols_t,
                            int64_t* n_rows, int64_t* n_cols, int64_t* n_rest, int64_t* n_duplicate) {
  clear_error();
  const size_t nbytes = ggnn_super_bytes(n_pad, E, s);
  GGNN_CHECK_ARG(nbytes > 0, "n_pad=%d (a positive multiple of 64), E=%d (1..64), s=%d (32, 64, 96 or 128, <= n_pad)",
                 n_pad, E, s);
  GGNN_CHECK_ARG(m >= 0, "m=%lld must be >= 0", (long long)m);
  GGNN_CHECK_ARG(m == 0 || (src && dst && etype), "src/dst/etype is NULL");
  GGNN_CHECK_ARG(rows != nullptr && cols != nullptr, "rows/cols is NULL");
  for (int64_t k = 0; k < m; ++k) {
    GGNN_CHECK_ARG(src[k] >= 0 && src[k] < n_pad && dst[k] >= 0 && dst[k] < n_pad,
                   "edge %lld (%d -> %d) out of range [0,%d)", (long long)k, src[k], dst[k], n_pad);
    GGNN_CHECK_ARG(etype[k] >= 0 && etype[k] < E, "edge %lld has type %d outside [0,%d)", (long long)k, etype[k],
                   E);
  }
  uint8_t* R = static_cast<uint8_t*>(rows);
  uint8_t* Cc = static_cast<uint8_t*>(cols);
  uint8_t* Rt = static_cast<uint8_t*>(rows_t);
  uint8_t* Ct = static_cast<uint8_t*>(cols_t);
  std::memset(R, 0, nbytes);
  std::memset(Cc, 0, nbytes);
  if (Rt) std::memset(Rt, 0, nbytes);
  if (Ct) std::memset(Ct, 0, nbytes);
  const size_t wide = static_cast<size_t>(n_pad / 8), narrow = static_cast<size_t>(s / 8);
  int64_t nr = 0, nc = 0, rest = 0, dup = 0;
  for (int64_t k = 0; k < m; ++k) {
    const int64_t i = dst[k], j = src[k], e = etype[k];
    uint8_t* byte;
    uint8_t bit;
    if (i < s) {   // into a supernode: row i of the row slice, column j
      byte = R + (static_cast<size_t>(e) * s + i) * wide + j / 8;
      bit = static_cast<uint8_t>(1u << (j % 8));
    } else if (j < s) {   // out of a supernode: row i of the column slice, column j
      byte = Cc + (static_cast<size_t>(e) * n_pad + i) * narrow + j / 8;
      bit = static_cast<uint8_t>(1u << (j % 8));
    } else {
      ++rest;
      continue;
    }
    if (*byte & bit) {
      ++dup;
      continue;
    }
    *byte |= bit;
    if (i < s) {
      ++nr;
      if (Rt) Rt[(static_cast<size_t>(e) * n_pad + j) * narrow + i / 8] |= static_cast<uint8_t>(1u << (i % 8));
    } else {
      ++nc;
      if (Ct) Ct[(static_cast<size_t>(e) * s + j) * wide + i / 8] |= static_cast<uint8_t>(1u << (i % 8));
    }
  }
  if (n_rows) *n_rows = nr;
  if (n_cols) *n_cols = nc;
  if (n_rest) *n_rest = rest;
  if (n_duplicate) *n_duplicate = dup;
  return GGNN_OK;
}

int32_t ggnn_super_active(int32_t n_pad, int32_t E, int32_t s, const void* rows, const void* cols) {
  clear_error();
  if (ggnn_super_bytes(n_pad, E, s) == 0) {
    fail(GGNN_ERR_INVALID_ARG, "n_pad=%d (a positive multiple of 64), E=%d (1..64), s=%d (32, 64, 96 or 128, <= n_pad)",
         n_pad, E, s);
    return -1;
  }
  if (rows == nullptr || cols == nullptr) {
    fail(GGNN_ERR_INVALID_ARG, "rows/cols is NULL");
    return -1;
  }
  const uint8_t* R = static_cast<const uint8_t*>(rows);
  const uint8_t* Cc = static_cast<const uint8_t*>(cols);
  const size_t wide = static_cast<size_t>(n_pad / 8), narrow = static_cast<size_t>(s / 8);
  int top = -1;   // largest supernode index with an edge
  for (int e = 0; e < E; ++e)
    for (int i = s - 1; i > top; --i) {
      const uint8_t* row = R + (static_cast<size_t>(e) * s + i) * wide;
      bool any = false;
      for (size_t b = 0; b < wide && !any; ++b) any = row[b] != 0;
      if (any) top = i;
    }
  uint8_t orb[16] = {0};   // s / 8 <= 16 bytes: the union of every row of the column slice
  for (size_t r = 0; r < static_cast<size_t>(E) * n_pad; ++r)
    for (size_t b = 0; b < narrow; ++b) orb[b] |= Cc[r * narrow + b];
  for (int j = 0; j < s; ++j)
    if ((orb[j / 8] >> (j % 8)) & 1u) top = j > top ? j : top;
  return top < 0 ? 0 : (top / 16 + 1) * 16;
}

}  // extern "C"
