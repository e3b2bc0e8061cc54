// gts_host.cpp — host side of libgts.so: graph validation, device image
// construction and upload, scratch sizing, argument checks and launch of the
// simulation kernels.  Implements the C ABI declared in include/gts.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <unordered_map>
#include <new>
#include <string>
#include <vector>

#include "../../include/gts.h"
#include "gts_dev.h"

namespace gts {
hipError_t launch_sim(const Launch& L, uint32_t lds_bytes, hipStream_t stream);
hipError_t launch_window(const Launch& L, uint32_t lds_bytes, hipStream_t stream);
}

struct gts_graph {
  gts::Image img;
  uint64_t bytes;
  uint32_t max_cta_nodes, max_outdeg;
  uint64_t max_tile_lines;
  bool all_mem_txn;  // every load / store streams at least one line (transaction-level memory)
  uint32_t full_lanes;  // bit n: at n_subpart = n every compute op holds every subpartition lane
};

struct gts_hwset {
  const uint32_t* dev;  // [B][32] in the caller's device buffer
  uint32_t B, max_nsm, max_nsub, max_noc;
};

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool is_compute(uint8_t c) { return c <= gts::C_SFU; }
uint32_t cluster_of(const gts_graph_host* h, uint32_t k) { return h->kernel_cluster ? h->kernel_cluster[k] : 1u; }
bool is_memory(uint8_t c) { return c == gts::C_GLOAD || c == gts::C_GSTORE; }

// A kernel whose CTAs share one template of node records.
struct KTemplate {
  uint32_t t_n = 0;     // nodes per CTA (0: not templated)
  uint32_t t_base = 0;  // first template record
  uint32_t t_ops = 0;   // first class x slot entry
  uint32_t nslot = 0;
  uint32_t tsucc = 0;   // first template successor
  int32_t sink = -1;    // local index of the template's retiring sink, or -1
};

// Everything the image needs that is derived from a valid host graph.
struct Derived {
  std::vector<uint32_t> indeg, node_cta, roots, root_begin, root_count;
  std::vector<uint8_t> shared;  // node has an in-edge from another CTA
  uint32_t props = 0, max_cta_nodes = 0, max_outdeg = 0;
  std::vector<KTemplate> ktmpl;  // per kernel
  std::vector<uint8_t> cclass;   // per CTA: class within its templated kernel
  std::vector<uint16_t> tslot;   // per template record: slot
  std::vector<uint16_t> tops;    // class x slot -> op
  uint32_t n_tnodes = 0, n_tsucc = 0;
  uint32_t n_tiles = 0;          // distinct tiles named by loads / stores
  uint64_t max_tile_lines = 0;   // the most lines of any of them
  bool all_mem_txn = false;      // every load / store streams at least one line (transaction-level memory)
  uint32_t full_lanes = 0;       // bit n: at n_subpart = n every compute op holds every subpartition lane
  // transaction-level memory: node v's lines txn_line[txn_ptr[v] ..
  // txn_ptr[v + 1]), numbered densely in order of first use
  std::vector<uint32_t> txn_ptr, txn_line;
  uint32_t n_lines = 0;
};

// Template sharing: find the kernels whose CTAs run isomorphic tile graphs
// (same node count, same local successor lists and kinds, no cross-CTA
// edges) and group their CTAs into classes by the op ids of their nodes.
// Kernels that would take the class x slot table past kMaxTops entries, or
// that have more than 255 classes, stay expanded.  GTS_TEMPLATES=0 turns the
// detection off.
void find_templates(const gts_graph_host* h, Derived* d) {
  const uint32_t K = h->n_kernels, C = h->n_ctas;
  d->ktmpl.assign(K, KTemplate());
  d->cclass.assign(C, 0);
  d->tslot.clear();
  d->tops.clear();
  d->n_tnodes = d->n_tsucc = 0;
  if (const char* e = std::getenv("GTS_TEMPLATES"))
    if (std::strcmp(e, "0") == 0) return;
  const uint32_t* nb = h->cta_node_begin;
  for (uint32_t k = 0; k < K; ++k) {
    const uint32_t c0 = h->kernel_cta_begin[k], c1 = h->kernel_cta_begin[k + 1];
    const uint32_t n = nb[c0 + 1] - nb[c0];
    if (c1 - c0 < 2 || cluster_of(h, k) > 1) continue;
    bool ok = true;
    for (uint32_t c = c0; c < c1 && ok; ++c) ok = nb[c + 1] - nb[c] == n;
    // identical local structure, every edge inside its CTA, no shared node
    for (uint32_t c = c0; c < c1 && ok; ++c) {
      for (uint32_t i = 0; i < n && ok; ++i) {
        const uint32_t u = nb[c] + i, u0 = nb[c0] + i;
        if (d->shared[u]) ok = false;
        const uint32_t e0 = h->succ_ptr[u0], deg = h->succ_ptr[u + 1] - h->succ_ptr[u];
        if (deg != h->succ_ptr[u0 + 1] - e0) ok = false;
        for (uint32_t j = 0; j < deg && ok; ++j) {
          const uint32_t a = h->succ[h->succ_ptr[u] + j], a0 = h->succ[e0 + j];
          const uint32_t v = a & GTS_EDGE_TARGET_MASK, v0 = a0 & GTS_EDGE_TARGET_MASK;
          ok = (a >> GTS_EDGE_KIND_SHIFT) == (a0 >> GTS_EDGE_KIND_SHIFT) && v >= nb[c] && v < nb[c] + n &&
               v - nb[c] == v0 - nb[c0];
        }
      }
    }
    if (!ok) continue;
    // classes by op vector, slots by op column
    std::map<std::vector<uint16_t>, uint32_t> classes;
    std::vector<uint32_t> cls(c1 - c0);
    std::vector<std::vector<uint16_t>> class_ops;
    for (uint32_t c = c0; c < c1 && ok; ++c) {
      std::vector<uint16_t> ops(h->node_op + nb[c], h->node_op + nb[c] + n);
      auto it = classes.find(ops);
      if (it == classes.end()) {
        if (classes.size() >= 255) ok = false;
        it = classes.emplace(ops, (uint32_t)class_ops.size()).first;
        class_ops.push_back(ops);
      }
      cls[c - c0] = it->second;
    }
    if (!ok) continue;
    const uint32_t nclass = (uint32_t)class_ops.size();
    std::map<std::vector<uint16_t>, uint32_t> slots;
    std::vector<uint16_t> slot_of(n);
    std::vector<std::vector<uint16_t>> slot_cols;
    for (uint32_t i = 0; i < n; ++i) {
      std::vector<uint16_t> col(nclass);
      for (uint32_t q = 0; q < nclass; ++q) col[q] = class_ops[q][i];
      auto it = slots.find(col);
      if (it == slots.end()) {
        it = slots.emplace(col, (uint32_t)slot_cols.size()).first;
        slot_cols.push_back(col);
      }
      slot_of[i] = (uint16_t)it->second;
    }
    const uint32_t nslot = (uint32_t)slot_cols.size();
    if (d->tops.size() + (uint64_t)nclass * nslot > gts::kMaxTops) continue;
    KTemplate& t = d->ktmpl[k];
    t.t_n = n;
    t.t_base = d->n_tnodes;
    t.t_ops = (uint32_t)d->tops.size();
    t.nslot = nslot;
    t.tsucc = d->n_tsucc;
    for (uint32_t q = 0; q < nclass; ++q)
      for (uint32_t s = 0; s < nslot; ++s) d->tops.push_back(slot_cols[s][q]);
    for (uint32_t c = c0; c < c1; ++c) d->cclass[c] = (uint8_t)cls[c - c0];
    d->tslot.insert(d->tslot.end(), slot_of.begin(), slot_of.end());
    // A CTA whose only node without a successor is a load / store that every
    // other node reaches over DATA / SYNC edges retires exactly when that
    // node finishes (each such edge starts its target no earlier than the
    // source's finish, so the sink finishes last): the kernel then needs no
    // per-CTA count of finished nodes.
    {
      const uint32_t u0 = nb[c0];
      int32_t sink = -1;
      bool single = true;
      for (uint32_t i = 0; i < n; ++i)
        if (h->succ_ptr[u0 + i + 1] == h->succ_ptr[u0 + i]) {
          if (sink >= 0) single = false;
          sink = (int32_t)i;
        }
      bool memory_sink = single && sink >= 0;
      for (uint32_t q = 0; q < nclass && memory_sink; ++q) memory_sink = is_memory(h->op_cls[class_ops[q][sink]]);
      if (memory_sink) {
        // reverse reachability from the sink over DATA / SYNC edges
        std::vector<std::vector<uint32_t>> pred(n);
        for (uint32_t i = 0; i < n; ++i)
          for (uint32_t e = h->succ_ptr[u0 + i]; e < h->succ_ptr[u0 + i + 1]; ++e)
            if ((h->succ[e] >> GTS_EDGE_KIND_SHIFT) != GTS_EDGE_ORDER)
              pred[(h->succ[e] & GTS_EDGE_TARGET_MASK) - u0].push_back(i);
        std::vector<uint8_t> seen(n, 0);
        std::vector<uint32_t> stack{(uint32_t)sink};
        seen[sink] = 1;
        uint32_t reached = 1;
        while (!stack.empty()) {
          const uint32_t v = stack.back();
          stack.pop_back();
          for (uint32_t u : pred[v])
            if (!seen[u]) {
              seen[u] = 1;
              ++reached;
              stack.push_back(u);
            }
        }
        if (reached == n) t.sink = sink;
      }
    }
    d->n_tnodes += n;
    d->n_tsucc += h->succ_ptr[nb[c0] + n] - h->succ_ptr[nb[c0]];
  }
}

int check_graph(const gts_graph_host* h, Derived* d) {
  if (!h) return fail(GTS_E_ARG, "graph is NULL");
  const uint32_t N = h->n_nodes, E = h->n_edges, C = h->n_ctas, K = h->n_kernels, P = h->n_ops;
  if (N > GTS_MAX_NODES) return fail(GTS_E_ARG, "n_nodes %u exceeds %u", N, GTS_MAX_NODES);
  if (C > GTS_MAX_CTAS) return fail(GTS_E_ARG, "n_ctas %u exceeds %u", C, GTS_MAX_CTAS);
  if (K > GTS_MAX_KERNELS) return fail(GTS_E_ARG, "n_kernels %u exceeds %u", K, GTS_MAX_KERNELS);
  if (P > GTS_MAX_OPS) return fail(GTS_E_ARG, "n_ops %u exceeds %u", P, GTS_MAX_OPS);
  if (!h->succ_ptr || !h->cta_node_begin || !h->kernel_cta_begin)
    return fail(GTS_E_ARG, "succ_ptr, cta_node_begin and kernel_cta_begin are required");
  if (N == 0) {
    if (C || K || E) return fail(GTS_E_RANGE, "an empty graph has no CTAs, kernels or edges");
    if (h->succ_ptr[0] || h->cta_node_begin[0] || h->kernel_cta_begin[0])
      return fail(GTS_E_RANGE, "offset arrays of an empty graph must be {0}");
    if (d) *d = Derived();
    return GTS_OK;
  }
  if (!C || !K) return fail(GTS_E_RANGE, "a non-empty graph needs at least one CTA and one kernel");
  if (!h->node_op || !h->kernel_warps || !h->kernel_smem || (E && !h->succ))
    return fail(GTS_E_ARG, "node, kernel or edge arrays are NULL");
  if (P && (!h->op_cls || !h->op_flags || !h->op_work || !h->op_warps))
    return fail(GTS_E_ARG, "op arrays are NULL");
  // offsets
  if (h->kernel_cta_begin[0] != 0 || h->kernel_cta_begin[K] != C)
    return fail(GTS_E_RANGE, "kernel_cta_begin must run from 0 to n_ctas");
  for (uint32_t k = 0; k < K; ++k) {
    if (h->kernel_cta_begin[k + 1] <= h->kernel_cta_begin[k]) return fail(GTS_E_RANGE, "kernel %u has no CTA", k);
    if (h->kernel_warps[k] < 1 || h->kernel_warps[k] > GTS_MAX_WARPS)
      return fail(GTS_E_RANGE, "kernel %u has %u warps per CTA (1..%u)", k, h->kernel_warps[k], GTS_MAX_WARPS);
    const uint32_t cl = cluster_of(h, k);
    if (cl < 1 || cl > GTS_MAX_CLUSTER || (h->kernel_cta_begin[k + 1] - h->kernel_cta_begin[k]) % cl)
      return fail(GTS_E_RANGE, "kernel %u has clusters of %u CTAs (1..%u, dividing its CTA count)", k, cl,
                  GTS_MAX_CLUSTER);
  }
  if (h->cta_node_begin[0] != 0 || h->cta_node_begin[C] != N)
    return fail(GTS_E_RANGE, "cta_node_begin must run from 0 to n_nodes");
  for (uint32_t c = 0; c < C; ++c)
    if (h->cta_node_begin[c + 1] <= h->cta_node_begin[c]) return fail(GTS_E_RANGE, "CTA %u has no node", c);
  if (h->succ_ptr[0] != 0 || h->succ_ptr[N] != E) return fail(GTS_E_RANGE, "succ_ptr must run from 0 to n_edges");
  for (uint32_t v = 0; v < N; ++v)
    if (h->succ_ptr[v + 1] < h->succ_ptr[v]) return fail(GTS_E_RANGE, "succ_ptr decreases at node %u", v);
  // ops
  for (uint32_t p = 0; p < P; ++p) {
    if (h->op_cls[p] >= GTS_N_CLASSES) return fail(GTS_E_RANGE, "op %u has class %u", p, h->op_cls[p]);
    const uint32_t allowed = h->op_cls[p] == GTS_REMOTE ? 0xF0u : GTS_OPF_MISS;
    if (h->op_flags[p] & ~allowed) return fail(GTS_E_RANGE, "op %u has unknown flags 0x%x", p, h->op_flags[p]);
    if (is_compute(h->op_cls[p]) && h->op_warps[p] == 0)
      return fail(GTS_E_RANGE, "compute op %u has an empty warp mask", p);
  }
  // nodes
  std::vector<uint32_t> node_cta(N), cta_kernel(C);
  for (uint32_t k = 0; k < K; ++k)
    for (uint32_t c = h->kernel_cta_begin[k]; c < h->kernel_cta_begin[k + 1]; ++c) cta_kernel[c] = k;
  uint32_t max_cta_nodes = 0;
  for (uint32_t c = 0; c < C; ++c) {
    max_cta_nodes = std::max(max_cta_nodes, h->cta_node_begin[c + 1] - h->cta_node_begin[c]);
    for (uint32_t v = h->cta_node_begin[c]; v < h->cta_node_begin[c + 1]; ++v) node_cta[v] = c;
  }
  for (uint32_t v = 0; v < N; ++v) {
    const uint32_t p = h->node_op[v];
    if (p >= P) return fail(GTS_E_RANGE, "node %u uses op %u of %u", v, p, P);
    if (is_compute(h->op_cls[p])) {
      const uint32_t w = h->kernel_warps[cta_kernel[node_cta[v]]];
      if (w < 32 && (h->op_warps[p] >> w) != 0)
        return fail(GTS_E_RANGE, "node %u runs on warps 0x%x outside its %u-warp CTA", v, h->op_warps[p], w);
    }
    if (h->op_cls[p] == GTS_REMOTE && (uint32_t)(h->op_flags[p] >> GTS_OPF_RANK_SHIFT) >=
                                          cluster_of(h, cta_kernel[node_cta[v]]))
      return fail(GTS_E_RANGE, "node %u targets rank %u outside its cluster", v, h->op_flags[p] >> GTS_OPF_RANK_SHIFT);
  }
  // tiles: only loads / stores, one line count per tile
  uint32_t n_tiles = 0;
  uint64_t max_tile_lines = 0;
  if (h->node_tile) {
    std::unordered_map<uint32_t, uint64_t> lines;
    for (uint32_t v = 0; v < N; ++v) {
      const uint32_t t = h->node_tile[v];
      if (t == GTS_NO_TILE) continue;
      const uint32_t p = h->node_op[v];
      if (!is_memory(h->op_cls[p])) return fail(GTS_E_RANGE, "node %u is not a load or store but names tile %u", v, t);
      // 64-bit, as in the kernels and the oracle: work near 2^32 must not wrap
      const uint64_t n = ((uint64_t)h->op_work[p] + GTS_LINE_BYTES - 1) / GTS_LINE_BYTES;
      max_tile_lines = std::max(max_tile_lines, n);
      auto it = lines.emplace(t, n).first;
      if (it->second != n)
        return fail(GTS_E_RANGE, "tile %u is touched with %llu and with %llu lines (node %u)", t,
                    (unsigned long long)it->second, (unsigned long long)n, v);
    }
    n_tiles = (uint32_t)lines.size();
  }
  // tile addresses: only loads / stores, never beside tile ids; each
  // addressed op's shape (rows dividing its bytes, a stride of at least a
  // row, a bounded transaction count) and each tile's bytes below NO_ADDR
  uint64_t n_txn_bound = 0;
  if (h->op_rows)
    for (uint32_t p = 0; p < P; ++p)
      if (h->op_rows[p] == 0) return fail(GTS_E_RANGE, "op %u has 0 rows", p);
  if (h->node_addr) {
    for (uint32_t v = 0; v < N; ++v) {
      const uint64_t a = h->node_addr[v];
      if (a == GTS_NO_ADDR) continue;
      const uint32_t p = h->node_op[v];
      if (!is_memory(h->op_cls[p])) return fail(GTS_E_RANGE, "node %u is not a load or store but has a tile address", v);
      if (h->node_tile && h->node_tile[v] != GTS_NO_TILE)
        return fail(GTS_E_RANGE, "node %u names a tile both by id and by address", v);
      const uint64_t R = h->op_rows ? h->op_rows[p] : 1u, work = h->op_work[p];
      if (work == 0 || work % R) return fail(GTS_E_RANGE, "op %u: %llu bytes in %llu rows (node %u)", p,
                                               (unsigned long long)work, (unsigned long long)R, v);
      const uint64_t W = work / R, pitch = h->op_pitch ? h->op_pitch[p] : W;
      if (pitch < W) return fail(GTS_E_RANGE, "op %u: row stride %llu below the row's %llu bytes", p,
                                 (unsigned long long)pitch, (unsigned long long)W);
      const uint64_t bound = R * (W / GTS_LINE_BYTES + 2);
      if (bound > GTS_MAX_NODE_TXN) return fail(GTS_E_RANGE, "op %u: tile of up to %llu transactions (at most %u)",
                                                p, (unsigned long long)bound, GTS_MAX_NODE_TXN);
      const uint64_t span = (R - 1) * pitch + W;  // <= 2^32 * 2^32: no wrap in 64 bits for R, W, pitch < 2^32
      if (a > GTS_NO_ADDR - 1 - span) return fail(GTS_E_RANGE, "node %u: tile at 0x%llx wraps the address space", v,
                                                  (unsigned long long)a);
      n_txn_bound += bound;
    }
    if (n_txn_bound && h->node_tile)
      for (uint32_t v = 0; v < N; ++v)
        if (h->node_tile[v] != GTS_NO_TILE)
          return fail(GTS_E_RANGE, "node %u names a tile by id in a graph whose tiles have addresses", v);
    if (n_txn_bound >= (1ull << 31)) return fail(GTS_E_RANGE, "addressed tiles of up to %llu transactions in all",
                                                 (unsigned long long)n_txn_bound);
  }
  // first CTA of each CTA's cluster (clusters are dispatched together, so
  // edges between their CTAs may go either way)
  std::vector<uint32_t> cluster_first(C);
  for (uint32_t c = 0; c < C; ++c) {
    const uint32_t k = cta_kernel[c], kb = h->kernel_cta_begin[k], cl = cluster_of(h, k);
    cluster_first[c] = kb + (c - kb) / cl * cl;
  }
  // edges: range, self loops, CTA order, duplicates, in-degree
  std::vector<uint32_t> indeg(N, 0), stamp(N, 0xFFFFFFFFu), intra_in(N, 0);
  uint32_t max_outdeg = 0;
  bool cross_from_memory = true;
  for (uint32_t u = 0; u < N; ++u) {
    max_outdeg = std::max(max_outdeg, h->succ_ptr[u + 1] - h->succ_ptr[u]);
    for (uint32_t e = h->succ_ptr[u]; e < h->succ_ptr[u + 1]; ++e) {
      const uint32_t v = h->succ[e] & GTS_EDGE_TARGET_MASK;
      const uint32_t kind = h->succ[e] >> GTS_EDGE_KIND_SHIFT;
      if (kind > GTS_EDGE_SYNC) return fail(GTS_E_RANGE, "edge %u has kind %u", e, kind);
      if (v >= N) return fail(GTS_E_RANGE, "edge %u targets node %u of %u", e, v, N);
      if (v == u) return fail(GTS_E_CYCLE, "self loop on node %u", u);
      if (node_cta[u] > node_cta[v] && cluster_first[node_cta[u]] != cluster_first[node_cta[v]])
        return fail(GTS_E_EDGE_ORDER, "edge %u -> %u goes from CTA %u back to CTA %u", u, v, node_cta[u], node_cta[v]);
      if (stamp[v] == u) return fail(GTS_E_DUP, "duplicate edge %u -> %u", u, v);
      stamp[v] = u;
      if (++indeg[v] > GTS_MAX_INDEG) return fail(GTS_E_RANGE, "node %u has in-degree above %u", v, GTS_MAX_INDEG);
      if (node_cta[u] == node_cta[v])
        ++intra_in[v];
      else if (!is_memory(h->op_cls[h->node_op[u]]) || kind == GTS_EDGE_ORDER)
        cross_from_memory = false;
    }
  }
  // acyclicity (Kahn)
  {
    std::vector<uint32_t> deg(indeg), queue;
    queue.reserve(N);
    for (uint32_t v = 0; v < N; ++v)
      if (!deg[v]) queue.push_back(v);
    for (size_t i = 0; i < queue.size(); ++i) {
      const uint32_t u = queue[i];
      for (uint32_t e = h->succ_ptr[u]; e < h->succ_ptr[u + 1]; ++e) {
        const uint32_t v = h->succ[e] & GTS_EDGE_TARGET_MASK;
        if (--deg[v] == 0) queue.push_back(v);
      }
    }
    if (queue.size() != N) return fail(GTS_E_CYCLE, "graph has a cycle through %zu node(s)", N - queue.size());
  }
  if (!d) return GTS_OK;
  // derived: roots per CTA, graph properties
  d->root_begin.assign(C, 0);
  d->root_count.assign(C, 0);
  d->roots.clear();
  bool sinks_memory = true, compute_feeds_data = true;
  for (uint32_t c = 0; c < C; ++c) {
    d->root_begin[c] = (uint32_t)d->roots.size();
    for (uint32_t v = h->cta_node_begin[c]; v < h->cta_node_begin[c + 1]; ++v) {
      if (intra_in[v] == 0) d->roots.push_back(v);
      bool has_intra_succ = false;
      for (uint32_t e = h->succ_ptr[v]; e < h->succ_ptr[v + 1] && !has_intra_succ; ++e)
        has_intra_succ = node_cta[h->succ[e] & GTS_EDGE_TARGET_MASK] == c;
      if (!has_intra_succ && !is_memory(h->op_cls[h->node_op[v]])) sinks_memory = false;
      bool feeds = is_memory(h->op_cls[h->node_op[v]]);
      for (uint32_t e = h->succ_ptr[v]; e < h->succ_ptr[v + 1] && !feeds; ++e)
        feeds = node_cta[h->succ[e] & GTS_EDGE_TARGET_MASK] == c &&
                (h->succ[e] >> GTS_EDGE_KIND_SHIFT) != GTS_EDGE_ORDER;
      if (!feeds) compute_feeds_data = false;
    }
    d->root_count[c] = (uint32_t)d->roots.size() - d->root_begin[c];
  }
  d->shared.assign(N, 0);
  for (uint32_t u = 0; u < N; ++u)
    for (uint32_t e = h->succ_ptr[u]; e < h->succ_ptr[u + 1]; ++e) {
      const uint32_t v = h->succ[e] & GTS_EDGE_TARGET_MASK;
      if (node_cta[u] != node_cta[v]) d->shared[v] = 1;
    }
  d->indeg.swap(indeg);
  d->node_cta.swap(node_cta);
  bool any_shared = false;
  for (uint32_t v = 0; v < N && !any_shared; ++v) any_shared = d->shared[v] != 0;
  uint32_t classes = 0;
  bool clusters = false, has_smem = false;
  for (uint32_t p = 0; p < P; ++p) {
    if (is_compute(h->op_cls[p])) classes |= 1u << h->op_cls[p];
    if (h->op_cls[p] == GTS_SMEM) has_smem = true;
    if (h->op_cls[p] == GTS_REMOTE) clusters = true;
  }
  for (uint32_t k = 0; k < K; ++k) clusters |= cluster_of(h, k) > 1;
  d->n_tiles = n_tiles;
  d->max_tile_lines = max_tile_lines;
  d->txn_ptr.clear();
  d->txn_line.clear();
  d->n_lines = 0;
  if (n_txn_bound) {
    // each addressed tile's distinct lines in the order its rows reach them
    // (a line two rows share is one transaction), lines numbered densely
    std::unordered_map<uint64_t, uint32_t> dense;
    std::vector<uint64_t> mine;
    d->txn_ptr.assign((size_t)N + 1, 0);
    for (uint32_t v = 0; v < N; ++v) {
      d->txn_ptr[v] = (uint32_t)d->txn_line.size();
      const uint64_t a = h->node_addr[v];
      if (a == GTS_NO_ADDR) continue;
      const uint32_t p = h->node_op[v];
      const uint64_t R = h->op_rows ? h->op_rows[p] : 1u, W = h->op_work[p] / R;
      const uint64_t pitch = h->op_pitch ? h->op_pitch[p] : W;
      mine.clear();
      for (uint64_t r = 0; r < R; ++r) {
        const uint64_t lo = (a + r * pitch) / GTS_LINE_BYTES, hi = (a + r * pitch + W - 1) / GTS_LINE_BYTES;
        for (uint64_t line = lo; line <= hi; ++line) {
          // rows reach lines in increasing order unless the stride is below
          // a line: only the last few lines can repeat
          bool seen = false;
          for (size_t i = mine.size(); i-- > 0 && !seen && mine[i] >= lo;) seen = mine[i] == line;
          if (!seen) mine.push_back(line);
        }
      }
      for (uint64_t line : mine) d->txn_line.push_back(dense.emplace(line, (uint32_t)dense.size()).first->second);
    }
    d->txn_ptr[N] = (uint32_t)d->txn_line.size();
    d->n_lines = (uint32_t)dense.size();
  }
  d->props = (sinks_memory ? gts::kGraphSinksAreMemory : 0u) | (cross_from_memory ? gts::kGraphCrossFromMemory : 0u) |
             (max_outdeg < 0xFFFFu ? gts::kGraphSmallOutdeg : 0u) | (any_shared ? gts::kGraphHasShared : 0u) |
             (compute_feeds_data ? gts::kGraphComputeFeedsData : 0u) | classes << gts::kGraphClassShift |
             (clusters ? gts::kGraphClusters : 0u) | (n_tiles ? gts::kGraphTiles : 0u) |
             (has_smem ? gts::kGraphSmem : 0u) |
             (d->txn_line.empty() ? 0u : gts::kGraphTxn);
  d->max_cta_nodes = max_cta_nodes;
  d->max_outdeg = max_outdeg;
  d->full_lanes = 0;
  for (uint32_t ns = 1; ns <= GTS_MAX_SUBPART && ns < 32; ++ns) {
    bool full = true;
    for (uint32_t p = 0; p < P && full; ++p) {
      if (!is_compute(h->op_cls[p])) continue;
      uint32_t lanes = 0;
      for (uint32_t w = 0; w < 32; ++w)
        if ((h->op_warps[p] >> w) & 1u) lanes |= 1u << (w % ns);
      full = lanes == (1u << ns) - 1u;
    }
    if (full) d->full_lanes |= 1u << ns;
  }
  d->all_mem_txn = !d->txn_line.empty();
  for (uint32_t v = 0; v < N && d->all_mem_txn; ++v)
    if (is_memory(h->op_cls[h->node_op[v]]) && d->txn_ptr[v + 1] == d->txn_ptr[v]) d->all_mem_txn = false;
  find_templates(h, d);
  return GTS_OK;
}

struct ImageLayout {
  uint64_t ops, nodes, succ, ctas, kernels, roots, indeg, tnodes, tsucc, tindeg, cclass, tops, tile, txn_ptr, txn_line,
      total;
};

ImageLayout image_layout(const gts_graph_host* h, const Derived& d) {
  const uint64_t n_roots = d.roots.size();
  ImageLayout L;
  uint64_t off = align_up(sizeof(gts::ImageHeader), gts::kAlign);
  L.ops = off;
  off = align_up(off + (uint64_t)h->n_ops * sizeof(gts::OpDev), gts::kAlign);
  L.nodes = off;
  off = align_up(off + ((uint64_t)h->n_nodes + 1) * sizeof(gts::NodeDev), gts::kAlign);
  L.succ = off;
  off = align_up(off + (uint64_t)h->n_edges * 4, gts::kAlign);
  L.ctas = off;
  off = align_up(off + (uint64_t)h->n_ctas * sizeof(gts::CtaDev), gts::kAlign);
  L.kernels = off;
  off = align_up(off + (uint64_t)h->n_kernels * sizeof(gts::KernelDev), gts::kAlign);
  L.roots = off;
  off = align_up(off + n_roots * 4, gts::kAlign);
  L.indeg = off;
  off = align_up(off + (uint64_t)h->n_nodes * 2, gts::kAlign);
  L.tnodes = off;
  off = align_up(off + (uint64_t)d.n_tnodes * sizeof(gts::NodeDev), gts::kAlign);
  L.tsucc = off;
  off = align_up(off + (uint64_t)d.n_tsucc * 4, gts::kAlign);
  L.tindeg = off;
  off = align_up(off + (uint64_t)d.n_tnodes * 2, gts::kAlign);
  L.cclass = off;
  off = align_up(off + (uint64_t)h->n_ctas, gts::kAlign);
  L.tops = off;
  off = align_up(off + d.tops.size() * 2, gts::kAlign);
  L.tile = off;
  off = align_up(off + (d.n_tiles ? (uint64_t)h->n_nodes * 4 : 0u), gts::kAlign);
  L.txn_ptr = off;
  off = align_up(off + d.txn_ptr.size() * 4, gts::kAlign);
  L.txn_line = off;
  off = align_up(off + d.txn_line.size() * 4, gts::kAlign);
  L.total = off;
  return L;
}

// keys: tiles or lines the LRU L2 tracks (0: no LRU state); accesses: a
// bound on the LRU accesses of one simulation (the stamps of its tree)
gts::SimLayout sim_layout(uint32_t N, uint32_t C, uint32_t P, uint32_t keys, uint32_t accesses, uint32_t ring_words) {
  gts::SimLayout s;
  uint64_t off = 0;
  s.off_state = off;
  off = align_up(off + (uint64_t)N * 8, gts::kAlign);
  s.off_cta = off;
  off = align_up(off + (uint64_t)C * sizeof(gts::CtaState), gts::kAlign);
  s.pend_cap = (uint64_t)N + C + 64;
  s.off_pend = off;
  off = align_up(off + s.pend_cap * 12, gts::kAlign);
  s.off_optab = off;
  off = align_up(off + (uint64_t)P * 16, gts::kAlign);
  // The windowed kernel's per-SM queues overlay the general kernel's pending
  // list and op table (a simulation the windowed kernel hands back is
  // restarted from scratch by the general kernel); both kernels use the LRU
  // state, which follows.
  s.off_rp = s.off_pend;
  s.off_mq = align_up(s.off_rp + 8ull * gts::kPoolSpill * 64, gts::kAlign);
  s.off_ret = align_up(s.off_mq + 4ull * ring_words * gts::kRing * gts::kWinMaxSm, gts::kAlign);
  off = std::max(off, align_up(s.off_ret + 8ull * (gts::kRetireCap - gts::kRetireLds), gts::kAlign));
  s.off_lru = off;
  off = align_up(off + (uint64_t)keys * 4, gts::kAlign);
  s.off_lru_bit = off;
  off = align_up(off + (keys ? ((uint64_t)accesses + 1) * 8 : 0u), gts::kAlign);
  s.stride = off + gts::kStatsBytes;
  return s;
}

uint64_t hw_area_bytes(uint32_t B) { return align_up((uint64_t)B * sizeof(gts_hw_params), gts::kAlign); }

int check_hw(const gts_hw_params* hw, uint32_t index) {
  if (hw->n_sm < 1 || hw->n_sm > GTS_MAX_SM)
    return fail(GTS_E_HW, "hw[%u].n_sm = %u (1..%u)", index, hw->n_sm, GTS_MAX_SM);
  if (hw->n_subpart < 1 || hw->n_subpart > GTS_MAX_SUBPART)
    return fail(GTS_E_HW, "hw[%u].n_subpart = %u (1..%u)", index, hw->n_subpart, GTS_MAX_SUBPART);
  for (int i = 0; i < 7; ++i) {
    if (hw->rate_q16[i] == 0) return fail(GTS_E_HW, "hw[%u].rate_q16[%d] is zero", index, i);
    if (hw->lat[i] > (1u << 30)) return fail(GTS_E_HW, "hw[%u].lat[%d] = %u exceeds 2^30", index, i, hw->lat[i]);
  }
  if (hw->cta_launch_lat > (1u << 30) || hw->kernel_launch_lat > (1u << 30))
    return fail(GTS_E_HW, "hw[%u] launch latency exceeds 2^30", index);
  if (hw->noc_nodes > GTS_MAX_NOC) return fail(GTS_E_HW, "hw[%u].noc_nodes = %u (0..%u)", index, hw->noc_nodes, GTS_MAX_NOC);
  if (hw->noc_nodes) {
    if (hw->noc_width > hw->noc_nodes || (hw->noc_width && hw->noc_nodes % hw->noc_width))
      return fail(GTS_E_HW, "hw[%u].noc_width = %u does not divide noc_nodes = %u", index, hw->noc_width,
                  hw->noc_nodes);
    if (hw->noc_rate_q16 == 0) return fail(GTS_E_HW, "hw[%u].noc_rate_q16 is zero", index);
  } else if (hw->noc_width || hw->noc_rate_q16 || hw->noc_map) {
    return fail(GTS_E_HW, "hw[%u] sets NoC fields without noc_nodes", index);
  }
  if (hw->noc_lat > (1u << 24)) return fail(GTS_E_HW, "hw[%u].noc_lat = %u exceeds 2^24", index, hw->noc_lat);
  if (hw->noc_map > 2) return fail(GTS_E_HW, "hw[%u].noc_map = %u (0 strips, 1 blocks, 2 strided)", index, hw->noc_map);
  for (int i = 0; i < 5; ++i)
    if (hw->reserved[i]) return fail(GTS_E_HW, "hw[%u].reserved[%d] is not zero", index, i);
  return GTS_OK;
}

gts::SimLayout layout_of(const gts_graph* g) {
  const gts::Image& m = g->img;
  return m.n_txn ? sim_layout(m.n_nodes, m.n_ctas, m.n_ops, m.n_lines, m.n_txn, gts::kRingWordsTxn)
                 : sim_layout(m.n_nodes, m.n_ctas, m.n_ops, m.n_tiles, m.n_nodes, gts::kRingWords);
}

uint64_t sim_scratch_bytes(const gts_graph* g, uint32_t B) {
  return (uint64_t)B * layout_of(g).stride;
}

int check_sim_args(const gts_graph* g, uint32_t B, const uint32_t* out_cycles, const uint32_t* out_makespan,
                   const int32_t* out_status, const uint64_t* out_digest, uint32_t flags) {
  if (!g) return fail(GTS_E_ARG, "graph handle is NULL");
  if (flags & ~GTS_FLAGS_ALL) return fail(GTS_E_ARG, "unknown flags 0x%x", flags);
  if (B == 0) return GTS_OK;
  if (!out_makespan || !out_status) return fail(GTS_E_ARG, "out_makespan and out_status are required");
  if ((flags & GTS_OUT_NODES) && !out_cycles && g->img.n_nodes)
    return fail(GTS_E_ARG, "GTS_OUT_NODES without out_cycles");
  if ((flags & GTS_OUT_DIGEST) && !out_digest) return fail(GTS_E_ARG, "GTS_OUT_DIGEST without out_digest");
  return GTS_OK;
}

// Enqueue the simulation for B records at hw_dev (device, validated).  Graphs
// whose CTAs end in memory nodes and whose cross-CTA edges leave memory
// nodes go to the windowed kernel first; simulations it cannot finish within
// its queue capacities (and every other graph) run on the general kernel.
constexpr uint32_t kLdsBudget = 64 * 1024;

// LDS of the general kernel: every SM's servers, then NoC servers (four per
// domain node; at most ceil(n_sm / D) * D <= n_sm + D nodes), then the op
// table when it still fits the budget (else it stays in scratch).
struct GeneralLds {
  uint32_t server_bytes, noc_words, total;
  bool optab;
};
// Every compute op holds every subpartition lane at each n_subpart up to
// max_nsub: a class's lanes are always busy together, and both kernels keep
// one server word per class instead of one per lane.
bool one_word_per_class(const gts_graph* g, uint32_t max_nsub) {
  const uint32_t upto = max_nsub < 31u ? ((2u << max_nsub) - 2u) : 0xFFFFFFFEu;  // bits 1..max_nsub
  return (g->full_lanes & upto) == upto;
}

GeneralLds general_lds(const gts_graph* g, uint32_t max_nsm, uint32_t max_nsub, uint32_t max_noc) {
  GeneralLds r;
  const uint32_t sstride = gts::server_stride(g->img.props, one_word_per_class(g, max_nsub) ? 1u : max_nsub);
  r.noc_words = (g->img.props & gts::kGraphClusters) && max_noc ? 4u * (max_nsm + max_noc) : 0u;
  r.server_bytes = 4u * (max_nsm * sstride + max_nsm + r.noc_words);
  const uint64_t optab_bytes = (uint64_t)g->img.n_ops * 16;
  r.optab = r.server_bytes + optab_bytes <= kLdsBudget;
  r.total = r.server_bytes + (r.optab ? (uint32_t)optab_bytes : 0u);
  return r;
}

// The largest records (many SMs x many subpartitions x three compute
// classes) can need more LDS for the general kernel's servers than one
// workgroup may hold on the current device: refused before anything is
// enqueued.
int check_lds(const gts_graph* g, uint32_t max_nsm, uint32_t max_nsub, uint32_t max_noc) {
  const uint32_t need = general_lds(g, max_nsm, max_nsub, max_noc).total;
  int dev = 0, max_lds = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return fail(GTS_E_HIP, "cannot query the device's LDS limit");
  if ((uint64_t)need > (uint64_t)max_lds)
    return fail(GTS_E_HW, "servers of %u SMs x %u subpartitions need %u B of LDS per simulation; the device allows %d",
                max_nsm, max_nsub, need, max_lds);
  return GTS_OK;
}

// Compute units of the current device (0 if it cannot be queried), once per
// device.
uint32_t device_cus() {
  static std::atomic<uint32_t> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  uint32_t c = cached[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
    c = (uint32_t)n;
    cached[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

int launch(const gts_graph* g, const uint32_t* hw_dev, uint32_t B, uint32_t max_nsm, uint32_t max_nsub, uint32_t max_noc,
           uint32_t* out_cycles, uint32_t* out_makespan, int32_t* out_status, uint64_t* out_digest, uint8_t* sims,
           uint32_t flags, hipStream_t st) {
  const GeneralLds gl = general_lds(g, max_nsm, max_nsub, max_noc);
  const uint32_t noc_words = gl.noc_words, server_bytes = gl.server_bytes, lds_general = gl.total;
  const bool lds_optab = gl.optab;
  gts::Launch L;
  L.img = g->img;
  L.hw = hw_dev;
  L.sims = sims;
  L.layout = layout_of(g);
  L.out_cycles = (flags & GTS_OUT_NODES) ? out_cycles : nullptr;
  L.out_makespan = out_makespan;
  L.out_status = out_status;
  L.out_digest = (flags & GTS_OUT_DIGEST) ? out_digest : nullptr;
  L.B = B;
  L.flags = flags;
  L.lds_optab = lds_optab ? 1u : 0u;
  L.lds_words_servers = server_bytes / 4;
  L.retry_only = 0;
  L.max_nsm = max_nsm;
  L.max_nsub = max_nsub;
  L.noc_words = noc_words;
  L.qp = 0;
  const char* clocks = std::getenv("GTS_WINDOW_CLOCKS");  // diagnostics: per-phase shader clocks
  L.clocks = clocks && std::strcmp(clocks, "0") != 0 ? 1u : 0u;

  // one server word per compute class when the lanes move together (less
  // LDS per simulation: more simulations per CU, and in the windowed kernel
  // more of the ready lists in LDS)
  L.srv_one = one_word_per_class(g, max_nsub) ? 1u : 0u;
  const uint32_t wstride = gts::server_stride(g->img.props, L.srv_one ? 1u : max_nsub);
  const uint32_t need_props = gts::kGraphSinksAreMemory | gts::kGraphCrossFromMemory | gts::kGraphSmallOutdeg;
  const char* force = std::getenv("GTS_KERNEL");  // "general": skip the windowed kernel
  // tiles (LRU L2): the memory phase packs a tile's line count into 22 bits;
  // transaction-level memory: every load / store streams lines (no node on
  // the whole-cycle servers of R6.4 beside them)
  const bool lru = (g->img.props & gts::kGraphTiles) != 0;
  const bool txn = (g->img.props & gts::kGraphTxn) != 0;
  const uint32_t mode = txn ? gts::kWinTxn : lru ? gts::kWinTiles : gts::kWinPlain;
  bool windowed = (g->img.props & need_props) == need_props && !(g->img.props & gts::kGraphClusters) &&
                  (!lru || g->max_tile_lines < gts::kWinMaxTileLines) && (!txn || g->all_mem_txn) &&
                  g->img.n_nodes > 0 && max_nsm <= gts::kWinMaxSm &&
                  !(force && std::strcmp(force, "general") == 0);
  uint32_t lds_window = 0;
  if (windowed) {
    // LDS per simulation: fixed tables plus qp later-ready entries per lane;
    // take the largest qp that keeps twelve simulations per CU (the register
    // limit of the kernel), or one per CU for a batch of at most one
    // simulation per CU, whose simulations then hold more of their
    // later-ready entries in LDS rather than in scratch.  Measured: a
    // 64-simulation decoder layer (long later-ready lists) 1.22x faster at
    // one per CU than at twelve, 16 and 256 simulations unchanged; a
    // 1024-simulation launch 3 % faster at four per CU than at twelve, but
    // launches of 1364 - 2048 simulations beside another stream's launches
    // (the GEMM design sweep) 15 % slower overall at six or eight per CU,
    // whose LDS keeps the other launch's simulations off the CU.
    constexpr uint32_t kLdsPerCu = 160 * 1024, kWavesPerCu = 12, kMaxQp = 160;
    auto bytes = [&](uint32_t qp) {
      return 4u * gts::win_lds(g->img.n_ops, max_nsm, wstride, qp, g->img.n_tops, mode).total;
    };
    auto per_cu = [&](uint32_t qp) { return std::min(kWavesPerCu, kLdsPerCu / bytes(qp)); };
    const uint32_t cus = device_cus();
    uint32_t want = cus && B <= cus ? 1u : kWavesPerCu;
    if (const char* w = std::getenv("GTS_WINDOW_WAVES"))  // tuning: target simulations per CU
      want = std::min<uint32_t>(kWavesPerCu, std::max<uint32_t>(1u, (uint32_t)std::strtoul(w, nullptr, 10)));
    constexpr uint32_t kMinQp = 0;
    uint32_t qp = kMinQp;
    for (uint32_t q = kMinQp + 1; q <= kMaxQp; ++q)
      if (bytes(q) <= kLdsBudget && per_cu(q) >= std::min(want, per_cu(kMinQp))) qp = q;
    L.qp = qp;
    windowed = bytes(qp) <= kLdsBudget;
    lds_window = bytes(qp);
  }
  // GTS_KERNEL=window (diagnostics): no general-kernel pass, so simulations
  // the windowed kernel hands back keep their internal retry status.
  const bool window_only = windowed && force && std::strcmp(force, "window") == 0;
  hipError_t e = hipSuccess;
  if (windowed) {
    e = gts::launch_window(L, lds_window, st);
    L.retry_only = 1;
  }
  if (e == hipSuccess && !window_only) e = gts::launch_sim(L, lds_general, st);
  if (e != hipSuccess) return fail(GTS_E_HIP, "kernel launch: %s", hipGetErrorString(e));
  return GTS_OK;
}

}  // namespace

namespace gts {
// For gts_simulate_hwset_noalloc (gts_noalloc.hip): B simulations of g must
// fit a fixed scratch array of `limit` bytes.
int check_fixed_scratch(const gts_graph* g, uint32_t B, uint64_t limit) {
  g_last_error.clear();
  if (!g) return fail(GTS_E_ARG, "graph handle is NULL");
  const uint64_t need = sim_scratch_bytes(g, B);
  if (need > limit)
    return fail(GTS_E_SCRATCH,
                "%u simulations of this graph need %llu bytes of scratch; the no-allocation entry point holds %llu "
                "(at most %llu simulations per call)",
                B, (unsigned long long)need, (unsigned long long)limit,
                (unsigned long long)(limit / std::max<uint64_t>(1, sim_scratch_bytes(g, 1))));
  return GTS_OK;
}
int report_hip(hipError_t e, const char* what) { return fail(GTS_E_HIP, "%s: %s", what, hipGetErrorString(e)); }
}  // namespace gts

extern "C" {

const char* gts_strerror(int code) {
  switch (code) {
    case GTS_OK: return "success";
    case GTS_E_ARG: return "invalid argument";
    case GTS_E_CYCLE: return "graph has a cycle";
    case GTS_E_EDGE_ORDER: return "edge from a later CTA to an earlier CTA";
    case GTS_E_RANGE: return "index, class, warp mask or degree out of range";
    case GTS_E_HW: return "invalid hardware parameters";
    case GTS_E_SCRATCH: return "buffer too small";
    case GTS_E_HIP: return "HIP runtime error";
    case GTS_E_DUP: return "duplicate edge";
    default: return "unknown error";
  }
}

const char* gts_last_error(void) { return g_last_error.c_str(); }

int gts_graph_validate(const gts_graph_host* h) {
  g_last_error.clear();
  return check_graph(h, nullptr);
}

int gts_hw_validate(const gts_hw_params* hw) {
  g_last_error.clear();
  if (!hw) return fail(GTS_E_ARG, "hw is NULL");
  return check_hw(hw, 0);
}

int gts_graph_device_bytes(const gts_graph_host* h, uint64_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(GTS_E_ARG, "bytes is NULL");
  Derived d;
  int rc = check_graph(h, &d);
  if (rc) return rc;
  *bytes = image_layout(h, d).total;
  return GTS_OK;
}

int gts_graph_templates(const gts_graph_host* h, uint32_t* templated_kernels, uint32_t* template_nodes,
                        uint32_t* expanded_nodes, uint32_t* class_ops) {
  g_last_error.clear();
  Derived d;
  int rc = check_graph(h, &d);
  if (rc) return rc;
  uint32_t nk = 0, expanded = 0;
  for (uint32_t k = 0; k < h->n_kernels; ++k) {
    if (d.ktmpl[k].t_n)
      ++nk;
    else
      expanded += h->cta_node_begin[h->kernel_cta_begin[k + 1]] - h->cta_node_begin[h->kernel_cta_begin[k]];
  }
  if (templated_kernels) *templated_kernels = nk;
  if (template_nodes) *template_nodes = d.n_tnodes;
  if (expanded_nodes) *expanded_nodes = expanded;
  if (class_ops) *class_ops = (uint32_t)d.tops.size();
  return GTS_OK;
}

int gts_graph_upload(const gts_graph_host* h, void* dev_image, uint64_t dev_bytes, void* hip_stream,
                     gts_graph** out) {
  g_last_error.clear();
  if (!out) return fail(GTS_E_ARG, "out is NULL");
  *out = nullptr;
  Derived d;
  int rc = check_graph(h, &d);
  if (rc) return rc;
  const ImageLayout L = image_layout(h, d);
  if (!dev_image) return fail(GTS_E_ARG, "device image buffer is NULL");
  if (dev_bytes < L.total)
    return fail(GTS_E_SCRATCH, "device image needs %llu bytes, got %llu", (unsigned long long)L.total,
                (unsigned long long)dev_bytes);
  std::vector<uint8_t> img;
  try {
    img.assign(L.total, 0);
  } catch (const std::bad_alloc&) {
    return fail(GTS_E_ARG, "host staging of %llu bytes failed", (unsigned long long)L.total);
  }
  auto* hdr = reinterpret_cast<gts::ImageHeader*>(img.data());
  hdr->magic = gts::kImageMagic;
  hdr->n_nodes = h->n_nodes;
  hdr->n_edges = h->n_edges;
  hdr->n_ctas = h->n_ctas;
  hdr->n_kernels = h->n_kernels;
  hdr->n_ops = h->n_ops;
  hdr->n_roots = (uint32_t)d.roots.size();
  hdr->props = d.props;
  hdr->off_ops = L.ops;
  hdr->off_nodes = L.nodes;
  hdr->off_succ = L.succ;
  hdr->off_ctas = L.ctas;
  hdr->off_kernels = L.kernels;
  hdr->off_roots = L.roots;
  hdr->off_indeg = L.indeg;
  hdr->off_tnodes = L.tnodes;
  hdr->off_tsucc = L.tsucc;
  hdr->off_tindeg = L.tindeg;
  hdr->off_cclass = L.cclass;
  hdr->off_tops = L.tops;
  hdr->off_tile = L.tile;
  hdr->off_txn_ptr = L.txn_ptr;
  hdr->off_txn_line = L.txn_line;
  hdr->max_cta_nodes = d.max_cta_nodes;
  hdr->max_outdeg = d.max_outdeg;
  hdr->n_tnodes = d.n_tnodes;
  hdr->n_tsucc = d.n_tsucc;
  hdr->n_tops = (uint32_t)d.tops.size();
  auto* ops = reinterpret_cast<gts::OpDev*>(img.data() + L.ops);
  for (uint32_t p = 0; p < h->n_ops; ++p) {
    ops[p].cls = h->op_cls[p];
    ops[p].flags = h->op_flags[p];
    ops[p].work = h->op_work[p];
    ops[p].warps = h->op_warps[p];
  }
  auto* nodes = reinterpret_cast<gts::NodeDev*>(img.data() + L.nodes);
  auto* succ_dev = reinterpret_cast<uint32_t*>(img.data() + L.succ);
  auto* indeg16 = reinterpret_cast<uint16_t*>(img.data() + L.indeg);
  // DATA and SYNC share one pattern; mark ORDER edges and edges into
  // shared nodes; the first three successors and their in-degrees are also
  // copied into the node record.
  for (uint32_t u = 0; u < h->n_nodes; ++u) {
    for (uint32_t e = h->succ_ptr[u]; e < h->succ_ptr[u + 1]; ++e) {
      const uint32_t v = h->succ[e] & GTS_EDGE_TARGET_MASK;
      const uint32_t kind = h->succ[e] >> GTS_EDGE_KIND_SHIFT;
      const uint32_t bits = (kind == GTS_EDGE_ORDER ? gts::kDevOrder : 0u) | (d.shared[v] ? gts::kDevShared : 0u);
      succ_dev[e] = v | (bits << GTS_EDGE_KIND_SHIFT);
    }
    gts::NodeDev& n = nodes[u];
    const uint32_t deg = h->succ_ptr[u + 1] - h->succ_ptr[u];
    n.op_nsucc = (uint32_t)h->node_op[u] | (std::min<uint32_t>(deg, 0xFFFFu) << 16);
    n.cta = d.node_cta[u];
    n.succ_begin = h->succ_ptr[u];
    for (uint32_t k = 0; k < gts::kInlineSucc; ++k) {
      n.succ[k] = k < deg ? succ_dev[n.succ_begin + k] : 0u;
      n.sindeg[k] = k < deg ? (uint16_t)d.indeg[h->succ[n.succ_begin + k] & GTS_EDGE_TARGET_MASK] : (uint16_t)0;
    }
    indeg16[u] = (uint16_t)d.indeg[u];
  }
  nodes[h->n_nodes].succ_begin = h->n_edges;  // sentinel: end of the last node's successors
  auto* ctas = reinterpret_cast<gts::CtaDev*>(img.data() + L.ctas);
  for (uint32_t c = 0; c < h->n_ctas; ++c) {
    ctas[c].node_begin = h->cta_node_begin[c];
    ctas[c].node_count = h->cta_node_begin[c + 1] - h->cta_node_begin[c];
    ctas[c].root_begin = d.root_begin[c];
    bool shared = false;
    for (uint32_t v = h->cta_node_begin[c]; v < h->cta_node_begin[c + 1] && !shared; ++v) shared = d.shared[v] != 0;
    ctas[c].root_count = d.root_count[c] | (shared ? gts::kCtaShared : 0u);
    uint32_t mem = 0;
    for (uint32_t v = h->cta_node_begin[c]; v < h->cta_node_begin[c + 1]; ++v) mem += is_memory(h->op_cls[h->node_op[v]]);
    ctas[c].mem_count = mem;
    for (uint32_t r = 0; r < gts::kInlineRoots; ++r)
      ctas[c].root[r] = r < d.root_count[c] ? d.roots[d.root_begin[c] + r] : 0u;
  }
  auto* ks = reinterpret_cast<gts::KernelDev*>(img.data() + L.kernels);
  for (uint32_t k = 0; k < h->n_kernels; ++k) {
    ks[k].cta_begin = h->kernel_cta_begin[k];
    ks[k].cta_end = h->kernel_cta_begin[k + 1];
    ks[k].warps = h->kernel_warps[k];
    ks[k].smem = h->kernel_smem[k];
    ks[k].node_begin = h->cta_node_begin[h->kernel_cta_begin[k]];
    const KTemplate& t = d.ktmpl[k];
    ks[k].t_n = t.t_n;
    ks[k].t_base = t.t_base;
    ks[k].t_ops = t.t_ops | t.nslot << 16;
    ks[k].pad[0] = t.sink >= 0 ? 1u : 0u;  // retires with its sink (kKernelSinkRetire)
    bool remote = false;
    for (uint32_t v = h->cta_node_begin[ks[k].cta_begin]; v < h->cta_node_begin[ks[k].cta_end] && !remote; ++v)
      remote = h->op_cls[h->node_op[v]] == GTS_REMOTE;
    ks[k].cluster = cluster_of(h, k) | (remote ? gts::kKernelRemote : 0u);
  }
  // template records: the first CTA's nodes with local successor targets and
  // slots for ops; their successors in the same form
  auto* tn = reinterpret_cast<gts::NodeDev*>(img.data() + L.tnodes);
  auto* ts = reinterpret_cast<uint32_t*>(img.data() + L.tsucc);
  auto* ti = reinterpret_cast<uint16_t*>(img.data() + L.tindeg);
  for (uint32_t k = 0; k < h->n_kernels; ++k) {
    const KTemplate& t = d.ktmpl[k];
    if (!t.t_n) continue;
    const uint32_t base = h->cta_node_begin[h->kernel_cta_begin[k]];
    const uint32_t e_base = h->succ_ptr[base];
    for (uint32_t i = 0; i < t.t_n; ++i) {
      const uint32_t u = base + i;
      const uint32_t deg = h->succ_ptr[u + 1] - h->succ_ptr[u];
      gts::NodeDev& r = tn[t.t_base + i];
      r.op_nsucc = (uint32_t)d.tslot[t.t_base + i] | (std::min<uint32_t>(deg, 0xFFFFu) << 16);
      r.cta = i;
      r.succ_begin = t.tsucc + (h->succ_ptr[u] - e_base);
      for (uint32_t j = 0; j < deg; ++j) {
        const uint32_t a = succ_dev[h->succ_ptr[u] + j];
        ts[r.succ_begin + j] = ((a & GTS_EDGE_TARGET_MASK) - base) | (a & ~GTS_EDGE_TARGET_MASK);
      }
      for (uint32_t j = 0; j < gts::kInlineSucc; ++j) {
        r.succ[j] = j < deg ? ts[r.succ_begin + j] : 0u;
        r.sindeg[j] = j < deg ? nodes[u].sindeg[j] : (uint16_t)0;
      }
      r.pad = (uint16_t)(t.sink == (int32_t)i ? gts::kRecSink : 0u);
      ti[t.t_base + i] = (uint16_t)d.indeg[u];
    }
  }
  std::memcpy(img.data() + L.cclass, d.cclass.data(), d.cclass.size());
  if (d.n_tiles) {
    // tiles numbered densely in order of first appearance (the kernel indexes
    // its per-tile stamps by them)
    std::unordered_map<uint32_t, uint32_t> dense;
    uint32_t* out = reinterpret_cast<uint32_t*>(img.data() + L.tile);
    for (uint32_t v = 0; v < h->n_nodes; ++v) {
      const uint32_t x = h->node_tile[v];
      out[v] = x == GTS_NO_TILE ? GTS_NO_TILE : dense.emplace(x, (uint32_t)dense.size()).first->second;
    }
  }
  if (!d.txn_ptr.empty()) std::memcpy(img.data() + L.txn_ptr, d.txn_ptr.data(), d.txn_ptr.size() * 4);
  if (!d.txn_line.empty()) std::memcpy(img.data() + L.txn_line, d.txn_line.data(), d.txn_line.size() * 4);
  if (!d.tops.empty()) std::memcpy(img.data() + L.tops, d.tops.data(), d.tops.size() * 2);
  if (!d.roots.empty()) std::memcpy(img.data() + L.roots, d.roots.data(), d.roots.size() * 4);

  hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
  hipError_t e = hipMemcpyAsync(dev_image, img.data(), L.total, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(GTS_E_HIP, "image upload: %s", hipGetErrorString(e));

  gts_graph* g = new (std::nothrow) gts_graph;
  if (!g) return fail(GTS_E_ARG, "out of host memory");
  uint8_t* base = static_cast<uint8_t*>(dev_image);
  g->img.ops = reinterpret_cast<const gts::OpDev*>(base + L.ops);
  g->img.nodes = reinterpret_cast<const gts::NodeDev*>(base + L.nodes);
  g->img.succ = reinterpret_cast<const uint32_t*>(base + L.succ);
  g->img.ctas = reinterpret_cast<const gts::CtaDev*>(base + L.ctas);
  g->img.kernels = reinterpret_cast<const gts::KernelDev*>(base + L.kernels);
  g->img.roots = reinterpret_cast<const uint32_t*>(base + L.roots);
  g->img.indeg = reinterpret_cast<const uint16_t*>(base + L.indeg);
  g->img.tnodes = reinterpret_cast<const gts::NodeDev*>(base + L.tnodes);
  g->img.tsucc = reinterpret_cast<const uint32_t*>(base + L.tsucc);
  g->img.tindeg = reinterpret_cast<const uint16_t*>(base + L.tindeg);
  g->img.cclass = reinterpret_cast<const uint8_t*>(base + L.cclass);
  g->img.tops = reinterpret_cast<const uint16_t*>(base + L.tops);
  g->img.n_tops = (uint32_t)d.tops.size();
  g->img.tile = d.n_tiles ? reinterpret_cast<const uint32_t*>(base + L.tile) : nullptr;
  g->img.n_tiles = d.n_tiles;
  g->max_tile_lines = d.max_tile_lines;
  g->full_lanes = d.full_lanes;
  g->all_mem_txn = d.all_mem_txn;
  const bool txn = !d.txn_line.empty();
  g->img.txn_ptr = txn ? reinterpret_cast<const uint32_t*>(base + L.txn_ptr) : nullptr;
  g->img.txn_line = txn ? reinterpret_cast<const uint32_t*>(base + L.txn_line) : nullptr;
  g->img.n_txn = (uint32_t)d.txn_line.size();
  g->img.n_lines = d.n_lines;
  g->img.n_nodes = h->n_nodes;
  g->img.n_edges = h->n_edges;
  g->img.n_ctas = h->n_ctas;
  g->img.n_kernels = h->n_kernels;
  g->img.n_ops = h->n_ops;
  g->img.props = d.props;
  g->bytes = L.total;
  g->max_cta_nodes = d.max_cta_nodes;
  g->max_outdeg = d.max_outdeg;
  *out = g;
  return GTS_OK;
}

int gts_graph_release(gts_graph* g) {
  delete g;
  return GTS_OK;
}

int gts_graph_sizes(const gts_graph* g, uint32_t* n_nodes, uint32_t* n_edges, uint32_t* n_ctas,
                    uint32_t* n_kernels, uint32_t* n_ops) {
  g_last_error.clear();
  if (!g) return fail(GTS_E_ARG, "graph handle is NULL");
  if (n_nodes) *n_nodes = g->img.n_nodes;
  if (n_edges) *n_edges = g->img.n_edges;
  if (n_ctas) *n_ctas = g->img.n_ctas;
  if (n_kernels) *n_kernels = g->img.n_kernels;
  if (n_ops) *n_ops = g->img.n_ops;
  return GTS_OK;
}

int gts_scratch_bytes(const gts_graph* g, uint32_t B, uint32_t flags, uint64_t* bytes) {
  g_last_error.clear();
  if (!g || !bytes) return fail(GTS_E_ARG, "graph handle or bytes is NULL");
  if (flags & ~GTS_FLAGS_ALL) return fail(GTS_E_ARG, "unknown flags 0x%x", flags);
  *bytes = hw_area_bytes(B) + sim_scratch_bytes(g, B);
  return GTS_OK;
}

int gts_simulate_batch(const gts_graph* g, const gts_hw_params* hw_host, uint32_t B, uint32_t* out_cycles,
                       uint32_t* out_makespan, int32_t* out_status, uint64_t* out_digest, void* scratch,
                       uint64_t scratch_bytes, uint32_t flags, void* hip_stream) {
  g_last_error.clear();
  int rc = check_sim_args(g, B, out_cycles, out_makespan, out_status, out_digest, flags);
  if (rc || B == 0) return rc;
  if (!hw_host) return fail(GTS_E_ARG, "hw_host is NULL");
  uint32_t max_nsm = 0, max_nsub = 0, max_noc = 0;
  for (uint32_t b = 0; b < B; ++b) {
    rc = check_hw(&hw_host[b], b);
    if (rc) return rc;
    max_nsm = std::max(max_nsm, hw_host[b].n_sm);
    max_nsub = std::max(max_nsub, hw_host[b].n_subpart);
    max_noc = std::max(max_noc, hw_host[b].noc_nodes);
  }
  const uint64_t need = hw_area_bytes(B) + sim_scratch_bytes(g, B);
  if (!scratch) return fail(GTS_E_ARG, "scratch is NULL");
  if (scratch_bytes < need)
    return fail(GTS_E_SCRATCH, "scratch needs %llu bytes, got %llu", (unsigned long long)need,
                (unsigned long long)scratch_bytes);
  rc = check_lds(g, max_nsm, max_nsub, max_noc);
  if (rc) return rc;
  hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
  uint8_t* base = static_cast<uint8_t*>(scratch);
  hipError_t e = hipMemcpyAsync(base, hw_host, (size_t)B * sizeof(gts_hw_params), hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return fail(GTS_E_HIP, "hw upload: %s", hipGetErrorString(e));
  return launch(g, reinterpret_cast<const uint32_t*>(base), B, max_nsm, max_nsub, max_noc, out_cycles, out_makespan,
                out_status, out_digest, base + hw_area_bytes(B), flags, st);
}

int gts_hwset_device_bytes(uint32_t B, uint64_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(GTS_E_ARG, "bytes is NULL");
  *bytes = hw_area_bytes(B);
  return GTS_OK;
}

int gts_hwset_upload(const gts_hw_params* hw_host, uint32_t B, void* dev_buf, uint64_t dev_bytes, void* hip_stream,
                     gts_hwset** out) {
  g_last_error.clear();
  if (!out) return fail(GTS_E_ARG, "out is NULL");
  *out = nullptr;
  if (B && !hw_host) return fail(GTS_E_ARG, "hw_host is NULL");
  uint32_t max_nsm = 0, max_nsub = 0, max_noc = 0;
  for (uint32_t b = 0; b < B; ++b) {
    int rc = check_hw(&hw_host[b], b);
    if (rc) return rc;
    max_nsm = std::max(max_nsm, hw_host[b].n_sm);
    max_nsub = std::max(max_nsub, hw_host[b].n_subpart);
    max_noc = std::max(max_noc, hw_host[b].noc_nodes);
  }
  if (B && !dev_buf) return fail(GTS_E_ARG, "dev_buf is NULL");
  if (dev_bytes < (uint64_t)B * sizeof(gts_hw_params))
    return fail(GTS_E_SCRATCH, "hw set needs %llu bytes, got %llu",
                (unsigned long long)((uint64_t)B * sizeof(gts_hw_params)), (unsigned long long)dev_bytes);
  if (B) {
    hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
    hipError_t e = hipMemcpyAsync(dev_buf, hw_host, (size_t)B * sizeof(gts_hw_params), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail(GTS_E_HIP, "hw set upload: %s", hipGetErrorString(e));
  }
  gts_hwset* h = new (std::nothrow) gts_hwset;
  if (!h) return fail(GTS_E_ARG, "out of host memory");
  h->dev = static_cast<const uint32_t*>(dev_buf);
  h->B = B;
  h->max_nsm = max_nsm;
  h->max_nsub = max_nsub;
  h->max_noc = max_noc;
  *out = h;
  return GTS_OK;
}

int gts_hwset_release(gts_hwset* hw) {
  delete hw;
  return GTS_OK;
}

int gts_simulate_hwset(const gts_graph* g, const gts_hwset* hw, uint32_t first, uint32_t B, uint32_t* out_cycles,
                       uint32_t* out_makespan, int32_t* out_status, uint64_t* out_digest, void* scratch,
                       uint64_t scratch_bytes, uint32_t flags, void* hip_stream) {
  g_last_error.clear();
  int rc = check_sim_args(g, B, out_cycles, out_makespan, out_status, out_digest, flags);
  if (rc || B == 0) return rc;
  if (!hw) return fail(GTS_E_ARG, "hw set handle is NULL");
  if ((uint64_t)first + B > hw->B)
    return fail(GTS_E_ARG, "records %u..%u exceed the set of %u", first, first + B, hw->B);
  const uint64_t need = sim_scratch_bytes(g, B);
  if (!scratch) return fail(GTS_E_ARG, "scratch is NULL");
  if (scratch_bytes < need)
    return fail(GTS_E_SCRATCH, "scratch needs %llu bytes, got %llu", (unsigned long long)need,
                (unsigned long long)scratch_bytes);
  rc = check_lds(g, hw->max_nsm, hw->max_nsub, hw->max_noc);
  if (rc) return rc;
  return launch(g, hw->dev + (uint64_t)first * gts::HW_WORDS, B, hw->max_nsm, hw->max_nsub, hw->max_noc, out_cycles,
                out_makespan, out_status, out_digest, static_cast<uint8_t*>(scratch), flags,
                reinterpret_cast<hipStream_t>(hip_stream));
}

}  // extern "C"
