/*
 * gts_oracle.c — plain, serial CPU oracle of the tile-graph simulation
 * backend of GTSim (arXiv 2607.11262, Sec. 5).
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load or call this code.  It shares no
 * code, header, table or constant generator with the HIP library; the only
 * things both sides agree on are interface formats (the 32-word hardware
 * record, the edge encoding, the class numbers), each restated here.
 *
 * Method.  A serial event-driven list scheduler over one binary heap keyed
 * (cycle, phase, id), exactly the rules below, one simulation per call.
 * Where the paper fixes a behaviour the rule cites it; where it is silent the
 * reading used is stated with the rule.
 *
 *  R2  Resources (Sec. 5.2 compute: tensor cores, CUDA cores, SFUs; memory:
 *      TMA/LSU front end, L2, DRAM).  Each subpartition of an SM has one
 *      pipeline per compute class (Sec. 5.2: one pipeline per execution-unit
 *      type); a TENSOR/ALU/SFU node occupies the lanes of its own class's
 *      pipelines named by its warps (lane of warp w = w mod n_subpart;
 *      Sec. 2.2 subpartitions, Sec. 5.3 warp-group issue across
 *      subpartitions), so nodes of different classes never delay each other
 *      on a lane.  SMEM nodes occupy the SM's shared-memory
 *      pipe.  GLOAD/GSTORE nodes occupy the SM's global-memory engine, then
 *      the chip-wide L2 server (or DRAM server when the op's MISS flag is
 *      set).  SYNC nodes occupy nothing.
 *  R3  Durations, integer cycles, rates in Q16.16, cdiv(a,b) = ceil(a/b):
 *        compute on k distinct lanes:
 *            occ = max(1, cdiv(work*65536*n_subpart, k*rate)), latency lat
 *        SMEM: occ = max(1, cdiv(work*65536, rate_smem)), latency lat_smem
 *        GMEM engine: occ_e = max(1, cdiv(work*65536, rate_gmem))
 *        L2/DRAM:     occ_m = max(1, cdiv(work*65536, rate_srv)), lat_srv
 *        SYNC: finish = start + max(1, lat_sync)
 *  R4  Every server is FIFO and non-preemptive with one "available" cycle;
 *      reserving at s for occ cycles sets it to s + occ.  A multi-lane node
 *      starts at max(ready, avail of each of its lanes) and advances them all.
 *      finish = start + occ + lat for compute and SMEM nodes (Sec. 5.2: each
 *      resource = latency, width, sustained throughput; latency overlaps the
 *      next node's occupancy).
 *  R6  One step per distinct event cycle t, in this phase order:
 *        1. CTA_RETIRE events at t free their SM slot;
 *        2. dispatch (Sec. 5.1 TB scheduler): pending CTAs in index order,
 *           each to the SM with the most free slots (ties: lowest SM id);
 *           a CTA of kernel k may go only once every CTA of kernels < k has
 *           retired; launch = t + cta_launch_lat (+ kernel_launch_lat for the
 *           CTAs dispatched in the step in which their kernel first
 *           dispatches); every node of the CTA whose in-edges are all
 *           released becomes ready at max(its release cycle, launch);
 *        3. NODE_READY events at t in increasing node id: issue;
 *           a GLOAD/GSTORE reserves its engine at s = max(t, avail) (its
 *           start), releases its ORDER edges and raises MEM_ARRIVE at s;
 *        4. MEM_ARRIVE events at t in increasing node id: m = max(t, avail
 *           of its L2/DRAM server), server avail = m + occ_m,
 *           finish = max(s + occ_e, m + occ_m) + lat_srv.
 *  R8  Release (Sec. 5.1/5.3: order edges at issue, data edges at
 *      completion): ORDER at start + 1, DATA and SYNC at finish (ORDER too
 *      under ORDER_AT_FINISH).  A node is ready when every in-edge has been
 *      released, at the latest release cycle (and not before its CTA's
 *      launch); if its CTA is not yet dispatched it waits for dispatch.
 *  R9  Residency per kernel: slots = min(max_cta_per_sm,
 *      smem_per_sm / smem_per_cta, max_warps_per_sm / warps_per_cta); a zero
 *      makes the simulation INFEASIBLE.  A CTA retires at the largest finish
 *      of its nodes (Sec. 5.1 / 5.3: a TB completes when all its nodes have
 *      finished; its SM resources are then released).
 *  R10 makespan = max finish; any cycle above 0xFFFFFFFE is OVERFLOW.
 *  R11 digest = sum over v of mix64(((start<<32)|finish) ^ mix64(v+1)),
 *      mod 2^64, mix64 = the SplitMix64 finaliser (Steele, Lea, Flood 2014).
 *  R12 NO_CONTENTION: servers never delay (start = ready, m = s).
 *  R13 Clusters (Sec. 5.2: thread-block clusters communicate through
 *      distributed shared memory).  Kernel k's CTAs form clusters of
 *      cl = kernel_cluster[k] consecutive CTAs; rank = (c - first CTA of k)
 *      mod cl.  SM s is node s mod D of NoC domain s / D (D = noc_nodes).
 *      A kernel with cl > 1 dispatches whole clusters in index order, all
 *      launched in the same step: for domain d = 0, 1, ... and slot j = 0,
 *      1, ... of the placement list, the first (d, j) whose SMs
 *      d*D + node(j, r), r < cl, all exist and all have a free slot takes
 *      the cluster (rank r on node(j, r)); if none, dispatch waits.
 *      Placement lists (Sec. 7.2 mapping): strips, node(j, r) = j*cl + r for
 *      j < D / cl; blocks (noc_map 1 on a W x H mesh), bh = the largest
 *      divisor of cl with bh*bh <= cl such that bw = cl / bh divides W and
 *      bh divides H: block j in row-major block order, rank r at
 *      x = (j mod (W/bw))*bw + r mod bw, y = (j div (W/bw))*bh + r div bw;
 *      without such a shape, or on a crossbar, strips; strided (noc_map 2),
 *      node(j, r) = j + r * (D / cl) for j < D / cl (ranks spread over the
 *      domain, as a placement that ignores the topology would).
 *  R14 REMOTE nodes (Sec. 5.2 DSMEM over the SM-cluster NoC; the target is
 *      carried by the node): target CTA = first CTA of the source's cluster
 *      + rank (op flags >> 4); route from node a (source SM) to node b
 *      (target CTA's SM) of their domain.  Crossbar (noc_width 0): the
 *      injection port of a and the ejection port of b, latency noc_lat.
 *      Mesh (noc_width W, H = D / W rows, node i at (i mod W, i div W)):
 *      the directed links of the XY route (x first), hops = |dx| + |dy|,
 *      latency hops * noc_lat.  occ = max(1, cdiv(work*65536, noc_rate));
 *      start s = max(t, avail of every server on the route), each set to
 *      s + occ; finish = s + occ + latency; ORDER edges at s + 1, DATA /
 *      SYNC at finish.  Reading: the route is reserved as a whole, like a
 *      multi-lane compute node (no per-hop store-and-forward).
 *  R15 A kernel with cl > 1 or with REMOTE nodes is INFEASIBLE when
 *      noc_nodes = 0, when cl > noc_nodes, or when no placement of R13 has
 *      all its SMs in the machine.
 *  R16 L2 as a fully associative LRU cache of C = l2_lines 128-B lines
 *      (Sec. 5.2: hits and misses from tile-derived accesses mapped to cache
 *      lines).  A GLOAD / GSTORE node with a tile id accesses the
 *      n = cdiv(work, 128) lines of that tile, in order, at its L2 arrival
 *      (MEM_ARRIVE, in (cycle, id) order).  With D = the number of distinct
 *      lines of other tiles accessed since the tile's last access, each of
 *      its lines sits at stack distance D + n - 1, so the access hits (all
 *      lines) iff the tile was accessed before and D + n <= C, and misses
 *      (all lines) otherwise; either way the tile becomes most recent.  A
 *      hit is served by the L2 server, a miss by the DRAM server (R7).
 *      Nodes without a tile id, or C = 0, keep the op's MISS flag.
 *  R17 Transaction-level memory (Sec. 5.2 Memory; Sec. 5.3 memory nodes: a
 *      tile access is expanded into transactions from the tile's shape,
 *      coordinates and layout at the transaction granularity, the TMA front
 *      end streams 128-B transactions at its issue rate, each transaction is
 *      serviced on its own, and the node completes with its last one).  A
 *      GLOAD / GSTORE node with a byte address a (node_addr; the tensor's
 *      base, layout and the tile's coordinates folded into it) accesses its
 *      op's tile of R = op_rows rows of W = work / R bytes, row r starting at
 *      a + r * P (P = op_pitch, the row stride).  Its transactions are the
 *      distinct 128-B lines floor(x / 128) of those bytes, in the order the
 *      rows first reach them (row by row, lines in increasing address); n of
 *      them.  At issue (engine start s, R6.3) the engine is held for
 *      occ_e = max(1, cdiv(n*128*65536, rate_gmem)); transaction j enters at
 *      e_j = s + cdiv(j*128*65536, rate_gmem) and has left the engine at
 *      e'_j = s + cdiv((j+1)*128*65536, rate_gmem).  It arrives at the L2
 *      at e_j (MEM_ARRIVE in (cycle, node id, j) order): with an L2 capacity
 *      (l2_lines = C > 0) its line hits iff it is among the C most recently
 *      accessed lines (then becomes the most recent), else the op's MISS
 *      flag decides; a hit is served by the L2 server, a miss by DRAM.  A
 *      server holds one 128-B transaction for q = cdiv(128*2^32, rate_srv)
 *      units of 2^-16 cycle (rate_srv in Q16.16 B/cycle), so it sustains its
 *      rate even when a line takes less than a cycle: with avail in those
 *      units, m_j = max(e_j * 2^16, avail), avail = m_j + q (NO_CONTENTION:
 *      m_j = e_j * 2^16), done_j = ceil((m_j + q) / 2^16) and
 *      finish_j = max(e'_j, done_j) + lat_srv.  The node finishes at the
 *      largest finish_j, decided when its last transaction arrives; then its
 *      DATA / SYNC edges release (R8).  A whole-cycle node of R6.4 sharing the
 *      server starts at the first whole cycle at or after avail and leaves
 *      avail on a whole cycle (so graphs without addresses time as before).
 *      A lone one-transaction tile times exactly as R6.4 does for the same
 *      node without an address.
 *      Readings: one transaction per distinct line of the tile (a line two
 *      rows share is fetched once); servers account transactions in 2^-16
 *      cycles (whole-cycle occupancy would cap an L2 of thousands of bytes
 *      per cycle at 128); a transaction arrives at the L2 when the
 *      engine starts injecting it and completes no earlier than its last
 *      byte leaves the engine (cut-through, as R6.4); conventional loads and
 *      stores use the same engine at its rate (the A100 record's engine is
 *      the LSU at the SRAM bandwidth), stores allocate in the LRU as loads do.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- interface formats (restated, not shared) ---------------------------- */
enum { K_TENSOR = 0, K_ALU = 1, K_SFU = 2, K_SMEM = 3, K_GLOAD = 4, K_GSTORE = 5, K_SYNC = 6, K_REMOTE = 7 };
enum { E_DATA = 0, E_ORDER = 1, E_SYNC = 2 };
/* hardware record: 32 u32 words */
enum {
  HW_NSM = 0, HW_NSUB = 1, HW_MAXCTA = 2, HW_MAXWARPS = 3, HW_SMEM = 4,
  HW_RATE = 5,  /* +0 tensor +1 alu +2 sfu +3 smem +4 gmem +5 l2 +6 dram */
  HW_LAT = 12,  /* +0 tensor +1 alu +2 sfu +3 smem +4 l2 +5 dram +6 sync */
  HW_CTALAT = 19, HW_KLAT = 20,
  HW_NOC_NODES = 21, HW_NOC_W = 22, HW_NOC_RATE = 23, HW_NOC_LAT = 24, HW_NOC_MAP = 25, HW_L2_LINES = 26
};
#define NO_TILE 0xFFFFFFFFu
#define NO_ADDR 0xFFFFFFFFFFFFFFFFull
enum { F_NODES = 1, F_DIGEST = 2, F_NOCONT = 4, F_ORDER_FIN = 8 };
enum { ST_OK = 0, ST_INFEASIBLE = 1, ST_OVERFLOW = 2, ST_DEADLOCK = 3 };

#define MAXCYC 0xFFFFFFFEull
#define EV_RETIRE 0ull
#define EV_READY 1ull
#define EV_MEM 2ull

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

static uint64_t cdiv(uint64_t a, uint64_t b) { return (a + b - 1) / b; }
static uint64_t max64(uint64_t a, uint64_t b) { return a > b ? a : b; }

/* ---- binary min-heap of events: key (cycle << 32 | phase << 30 | id), then
 * j (the transaction index of an R17 memory arrival, else 0) ------------- */
typedef struct { uint64_t key; uint32_t j; } ev_t;
typedef struct { ev_t *a; size_t n; } heap_t;

static int ev_less(ev_t x, ev_t y) { return x.key < y.key || (x.key == y.key && x.j < y.j); }

static void heap_push_j(heap_t *h, uint64_t key, uint32_t j) {
  ev_t e = {key, j};
  size_t i = h->n++;
  while (i > 0) {
    size_t p = (i - 1) / 2;
    if (!ev_less(e, h->a[p])) break;
    h->a[i] = h->a[p];
    i = p;
  }
  h->a[i] = e;
}

static void heap_push(heap_t *h, uint64_t key) { heap_push_j(h, key, 0); }

static ev_t heap_pop(heap_t *h) {
  ev_t top = h->a[0];
  ev_t last = h->a[--h->n];
  size_t i = 0;
  for (;;) {
    size_t l = 2 * i + 1, r = l + 1, m = i;
    ev_t mv = last;
    if (l < h->n && ev_less(h->a[l], mv)) { m = l; mv = h->a[l]; }
    if (r < h->n && ev_less(h->a[r], mv)) { m = r; mv = h->a[r]; }
    if (m == i) break;
    h->a[i] = h->a[m];
    i = m;
  }
  if (h->n) h->a[i] = last;
  return top;
}

static uint64_t mkkey(uint64_t t, uint64_t phase, uint64_t id) {
  return (t << 32) | (phase << 30) | id;
}

/* ---- one simulation ------------------------------------------------------- */
typedef struct {
  /* graph */
  uint32_t N, C, K, P;
  const uint8_t *op_cls, *op_flags;
  const uint32_t *op_work, *op_warps;
  const uint16_t *node_op;
  const uint32_t *succ_ptr, *succ, *cta_node_begin, *kernel_cta_begin;
  const uint16_t *kernel_warps;
  const uint32_t *kernel_smem;
  const uint8_t *kernel_cluster;
  const uint32_t *node_tile;   /* or NULL */
  /* hw */
  uint32_t nsm, nsub, flags;
  const uint32_t *hw;
  uint32_t noc_d, noc_w;   /* SMs per NoC domain, mesh width (0: crossbar) */
  /* derived per op */
  uint64_t *occ, *occm, *lat; uint32_t *lanes; int *to_dram;
  uint64_t *occ_l2, *occ_d, *lat_l2, *lat_d;  /* memory ops served by L2 / by DRAM */
  uint64_t *slots;
  /* per node */
  uint32_t *indeg, *cnt, *node_cta, *acc, *st, *fin;
  /* per CTA */
  int64_t *cta_sm; uint32_t *cta_launch, *cta_left, *cta_maxfin, *cta_kernel;
  /* per SM */
  uint64_t *resident, *lane_av, *smem_av, *eng_av;
  uint64_t l2_av, dram_av;   /* in 2^-16 cycles (R17) */
  uint64_t *noc_av;        /* per domain node: 4 link/port servers */
  /* R16: tiles in recency order (most recent first) and their lines */
  uint32_t *lru_tile, *lru_lines; uint32_t lru_n;
  /* R17: tile addresses, shapes; per issued node its lines, transactions
   * left and largest transaction finish; lines in recency order */
  const uint64_t *node_addr;   /* or NULL */
  const uint32_t *op_rows, *op_pitch;  /* or NULL */
  uint64_t **txn_lines; uint32_t *txn_n, *txn_left; uint64_t *txn_maxf;
  uint64_t *lru_line; uint64_t lru_line_n;
  /* control */
  heap_t heap;
  uint32_t next_cta; uint64_t retired;
  int64_t *kstart;
  int overflow, oom;
  uint64_t nfinished;
} sim_t;

static void release_edge(sim_t *S, uint32_t w, uint64_t r) {
  if (r > S->acc[w]) S->acc[w] = (uint32_t)r;
  S->cnt[w]++;
  if (S->cnt[w] == S->indeg[w]) {
    uint32_t c = S->node_cta[w];
    if (S->cta_sm[c] >= 0)
      heap_push(&S->heap, mkkey(max64(S->acc[w], S->cta_launch[c]), EV_READY, w));
  }
}

/* release the out-edges of v whose release cycle is decided now:
 * which = 0: ORDER edges at start+1; which = 1: DATA/SYNC edges at finish
 * (and ORDER edges too when ORDER_AT_FINISH). */
static void release_out(sim_t *S, uint32_t v, int which, uint64_t cyc) {
  int order_at_fin = (S->flags & F_ORDER_FIN) != 0;
  for (uint32_t e = S->succ_ptr[v]; e < S->succ_ptr[v + 1]; e++) {
    uint32_t w = S->succ[e] & 0x3FFFFFFFu;
    uint32_t kind = S->succ[e] >> 30;
    int is_order_now = (kind == E_ORDER) && !order_at_fin;
    if (which == 0 && is_order_now) release_edge(S, w, cyc);
    if (which == 1 && !is_order_now) release_edge(S, w, cyc);
  }
}

/* record v's (start, finish) and do the CTA bookkeeping */
static int complete(sim_t *S, uint32_t v, uint64_t start, uint64_t finish) {
  if (finish > MAXCYC) { S->overflow = 1; return 0; }
  S->st[v] = (uint32_t)start;
  S->fin[v] = (uint32_t)finish;
  S->nfinished++;
  uint32_t c = S->node_cta[v];
  if (finish > S->cta_maxfin[c]) S->cta_maxfin[c] = (uint32_t)finish;
  if (--S->cta_left[c] == 0) heap_push(&S->heap, mkkey(S->cta_maxfin[c], EV_RETIRE, c));
  return 1;
}

/* R13: node of rank r in placement slot j of a domain, or -1 if the list has
 * no slot j */
static int64_t slot_node(const sim_t *S, uint32_t cl, uint32_t j, uint32_t r) {
  uint32_t D = S->noc_d, W = S->noc_w;
  if (S->hw[HW_NOC_MAP] == 1 && W > 0) {
    uint32_t H = D / W, bh = 0;
    for (uint32_t h = 1; h * h <= cl; h++)
      if (cl % h == 0 && W % (cl / h) == 0 && H % h == 0) bh = h;
    if (bh) {
      uint32_t bw = cl / bh, nbx = W / bw, nby = H / bh;
      if (j >= nbx * nby) return -1;
      uint32_t x = (j % nbx) * bw + r % bw, y = (j / nbx) * bh + r / bw;
      return (int64_t)y * W + x;
    }
  }
  if (j >= D / cl) return -1;
  if (S->hw[HW_NOC_MAP] == 2) return (int64_t)j + (int64_t)r * (D / cl);
  return (int64_t)j * cl + r;
}

/* R13: first placement (domain-major, then slot) whose SMs exist and, if
 * `need_free`, all have a free slot for kernel k; writes the SM of each rank */
static int place_cluster(const sim_t *S, uint32_t k, uint32_t cl, int need_free, uint64_t *sm_of_rank) {
  uint32_t ndom = (S->nsm + S->noc_d - 1) / S->noc_d;
  for (uint32_t d = 0; d < ndom; d++)
    for (uint32_t j = 0; slot_node(S, cl, j, 0) >= 0; j++) {
      int ok = 1;
      for (uint32_t r = 0; r < cl && ok; r++) {
        uint64_t s = (uint64_t)d * S->noc_d + (uint64_t)slot_node(S, cl, j, r);
        if (s >= S->nsm) ok = 0;
        else if (need_free && S->resident[s] >= S->slots[k]) ok = 0;
        else sm_of_rank[r] = s;
      }
      if (ok) return 1;
    }
  return 0;
}

static void push_roots(sim_t *S, uint32_t c, uint64_t launch) {
  for (uint32_t v = S->cta_node_begin[c]; v < S->cta_node_begin[c + 1]; v++)
    if (S->cnt[v] == S->indeg[v])
      heap_push(&S->heap, mkkey(max64(S->acc[v], launch), EV_READY, v));
}

static void dispatch(sim_t *S, uint64_t t) {
  while (S->next_cta < S->C) {
    uint32_t c = S->next_cta;
    uint32_t k = S->cta_kernel[c];
    if (S->retired < S->kernel_cta_begin[k]) break;   /* previous kernel still running */
    uint32_t cl = S->kernel_cluster[k];
    if (cl > 1) {                                        /* R13: a whole cluster */
      uint64_t sm_of_rank[16];
      if (!place_cluster(S, k, cl, 1, sm_of_rank)) break;
      if (S->kstart[k] < 0) S->kstart[k] = (int64_t)t;
      uint64_t launch = t + S->hw[HW_CTALAT];
      if ((uint64_t)S->kstart[k] == t) launch += S->hw[HW_KLAT];
      if (launch > MAXCYC) { S->overflow = 1; return; }
      for (uint32_t r = 0; r < cl; r++) {
        S->cta_sm[c + r] = (int64_t)sm_of_rank[r];
        S->cta_launch[c + r] = (uint32_t)launch;
        S->resident[sm_of_rank[r]]++;
      }
      for (uint32_t r = 0; r < cl; r++) push_roots(S, c + r, launch);
      S->next_cta += cl;
      continue;
    }
    int64_t best = -1; uint64_t bestfree = 0;
    for (uint32_t m = 0; m < S->nsm; m++) {
      uint64_t fr = S->slots[k] - S->resident[m];
      if (fr > bestfree) { bestfree = fr; best = m; }
    }
    if (best < 0) break;                                 /* every SM full */
    if (S->kstart[k] < 0) S->kstart[k] = (int64_t)t;
    uint64_t launch = t + S->hw[HW_CTALAT];
    if ((uint64_t)S->kstart[k] == t) launch += S->hw[HW_KLAT];
    if (launch > MAXCYC) { S->overflow = 1; return; }
    S->cta_sm[c] = best;
    S->cta_launch[c] = (uint32_t)launch;
    S->resident[best]++;
    push_roots(S, c, launch);
    S->next_cta++;
  }
}

/* R17: the distinct 128-B lines of node v's tile, in the order the rows
 * first reach them; stored for the node, returns their number (0 when host
 * memory runs out) */
static uint32_t tile_lines(sim_t *S, uint32_t v) {
  uint32_t p = S->node_op[v];
  uint64_t R = S->op_rows ? S->op_rows[p] : 1;
  uint64_t W = S->op_work[p] / R;
  uint64_t P = S->op_pitch ? S->op_pitch[p] : W;
  uint64_t cap = R * (W / 128 + 2);
  uint64_t *lines = malloc(cap * sizeof *lines);
  if (!lines) return 0;
  uint32_t n = 0;
  for (uint64_t r = 0; r < R; r++) {
    uint64_t first = (S->node_addr[v] + r * P) / 128, last = (S->node_addr[v] + r * P + W - 1) / 128;
    for (uint64_t L = first; L <= last; L++) {
      uint32_t i = 0;
      while (i < n && lines[i] != L) i++;
      if (i == n) lines[n++] = L;
    }
  }
  free(S->txn_lines[v]);
  S->txn_lines[v] = lines;
  S->txn_n[v] = n;
  return n;
}

static void issue(sim_t *S, uint32_t v, uint64_t t) {
  uint32_t p = S->node_op[v];
  uint32_t c = S->node_cta[v];
  uint64_t sm = (uint64_t)S->cta_sm[c];
  int nocont = (S->flags & F_NOCONT) != 0;
  uint32_t cls = S->op_cls[p];
  if (cls == K_TENSOR || cls == K_ALU || cls == K_SFU) {
    uint64_t s = t;
    uint64_t *lanes = S->lane_av + (sm * 3 + cls) * S->nsub;  /* class cls's lanes */
    if (!nocont)
      for (uint32_t l = 0; l < S->nsub; l++)
        if (S->lanes[p] >> l & 1) s = max64(s, lanes[l]);
    for (uint32_t l = 0; l < S->nsub; l++)
      if (S->lanes[p] >> l & 1) lanes[l] = s + S->occ[p];
    if (!complete(S, v, s, s + S->occ[p] + S->lat[p])) return;
    release_out(S, v, 0, s + 1);
    release_out(S, v, 1, S->fin[v]);
  } else if (cls == K_SMEM) {
    uint64_t s = nocont ? t : max64(t, S->smem_av[sm]);
    S->smem_av[sm] = s + S->occ[p];
    if (!complete(S, v, s, s + S->occ[p] + S->lat[p])) return;
    release_out(S, v, 0, s + 1);
    release_out(S, v, 1, S->fin[v]);
  } else if (cls == K_SYNC) {
    if (!complete(S, v, t, t + S->lat[p])) return;
    release_out(S, v, 0, t + 1);
    release_out(S, v, 1, S->fin[v]);
  } else if (cls == K_REMOTE) { /* R14 */
    uint32_t k = S->cta_kernel[c], cl = S->kernel_cluster[k], kb = S->kernel_cta_begin[k];
    uint32_t tgt = kb + (c - kb) / cl * cl + (S->op_flags[p] >> 4);
    uint64_t D = S->noc_d, dom = sm / D;
    uint64_t a = sm % D, b = (uint64_t)S->cta_sm[tgt] % D;
    uint64_t *route[2 * 64];
    uint32_t nr = 0, lat_mult = 1;
    uint64_t *dav = S->noc_av + dom * D * 4;
    if (S->noc_w == 0) {           /* crossbar: injection port of a, ejection port of b */
      route[nr++] = &dav[a * 4 + 0];
      route[nr++] = &dav[b * 4 + 1];
    } else {                        /* mesh, XY routing: link (node, dir), dir 0 +x 1 -x 2 +y 3 -y */
      uint64_t W = S->noc_w, x = a % W, y = a / W, xb = b % W, yb = b / W;
      while (x != xb) { uint32_t dir = xb > x ? 0 : 1; route[nr++] = &dav[(y * W + x) * 4 + dir]; x = dir == 0 ? x + 1 : x - 1; }
      while (y != yb) { uint32_t dir = yb > y ? 2 : 3; route[nr++] = &dav[(y * W + x) * 4 + dir]; y = dir == 2 ? y + 1 : y - 1; }
      lat_mult = nr;
    }
    uint64_t s = t;
    if (!nocont)
      for (uint32_t i = 0; i < nr; i++) s = max64(s, *route[i]);
    for (uint32_t i = 0; i < nr; i++) *route[i] = s + S->occ[p];
    if (!complete(S, v, s, s + S->occ[p] + S->lat[p] * lat_mult)) return;
    release_out(S, v, 0, s + 1);
    release_out(S, v, 1, S->fin[v]);
  } else if (S->node_addr && S->node_addr[v] != NO_ADDR) { /* R17: transactions */
    uint32_t n = tile_lines(S, v);
    if (n == 0) { S->oom = S->overflow = 1; return; }   /* out of host memory: stop */
    uint64_t rate = S->hw[HW_RATE + 4];
    uint64_t occ_e = max64(1, cdiv((uint64_t)n * 128 * 65536, rate));
    uint64_t s = nocont ? t : max64(t, S->eng_av[sm]);
    if (s + occ_e > MAXCYC) { S->overflow = 1; return; }
    S->eng_av[sm] = s + occ_e;
    S->st[v] = (uint32_t)s;
    S->txn_left[v] = n;
    S->txn_maxf[v] = 0;
    release_out(S, v, 0, s + 1);
    for (uint32_t j = 0; j < n; j++)
      heap_push_j(&S->heap, mkkey(s + cdiv((uint64_t)j * 128 * 65536, rate), EV_MEM, v), j);
  } else { /* GLOAD / GSTORE: engine now, global server at MEM_ARRIVE */
    uint64_t s = nocont ? t : max64(t, S->eng_av[sm]);
    if (s + S->occ[p] > MAXCYC) { S->overflow = 1; return; }
    S->eng_av[sm] = s + S->occ[p];
    S->st[v] = (uint32_t)s;
    release_out(S, v, 0, s + 1);
    heap_push(&S->heap, mkkey(s, EV_MEM, v));
  }
}

/* R16: one tile access; returns 1 on a hit */
static int lru_access(sim_t *S, uint32_t tile, uint32_t n) {
  uint64_t D = 0;
  uint32_t i = 0;
  while (i < S->lru_n && S->lru_tile[i] != tile) D += S->lru_lines[i++];
  int found = i < S->lru_n;
  int hit = found && D + n <= S->hw[HW_L2_LINES];
  if (!found) S->lru_n++;
  memmove(S->lru_tile + 1, S->lru_tile, (size_t)i * sizeof *S->lru_tile);
  memmove(S->lru_lines + 1, S->lru_lines, (size_t)i * sizeof *S->lru_lines);
  S->lru_tile[0] = tile;
  S->lru_lines[0] = n;
  return hit;
}

static void mem_arrive(sim_t *S, uint32_t v, uint64_t t) {
  uint32_t p = S->node_op[v];
  int dram = S->to_dram[p];
  if (S->node_tile && S->node_tile[v] != NO_TILE && S->hw[HW_L2_LINES])
    dram = !lru_access(S, S->node_tile[v], (uint32_t)cdiv(S->op_work[p], 128));
  uint64_t *av = dram ? &S->dram_av : &S->l2_av;
  uint64_t occm = dram ? S->occ_d[p] : S->occ_l2[p];
  uint64_t m = (S->flags & F_NOCONT) ? t : max64(t, (*av + 65535) >> 16);
  *av = (m + occm) << 16;
  uint64_t s = S->st[v];
  uint64_t f = max64(s + S->occ[p], m + occm) + (dram ? S->lat_d[p] : S->lat_l2[p]);
  if (!complete(S, v, s, f)) return;
  release_out(S, v, 1, f);
}

/* R17: line access to the LRU of lines; returns 1 on a hit */
static int lru_line_access(sim_t *S, uint64_t line) {
  uint64_t i = 0;
  while (i < S->lru_line_n && S->lru_line[i] != line) i++;
  int hit = i < S->lru_line_n && i < S->hw[HW_L2_LINES];
  if (i == S->lru_line_n) S->lru_line_n++;
  memmove(S->lru_line + 1, S->lru_line, (size_t)i * sizeof *S->lru_line);
  S->lru_line[0] = line;
  return hit;
}

/* R17: transaction j of node v arrives at the L2 at cycle t */
static void mem_txn(sim_t *S, uint32_t v, uint32_t j, uint64_t t) {
  uint32_t p = S->node_op[v];
  int dram = S->to_dram[p];
  if (S->hw[HW_L2_LINES]) dram = !lru_line_access(S, S->txn_lines[v][j]);
  uint64_t rate_srv = S->hw[HW_RATE + (dram ? 6 : 5)];
  uint64_t q = cdiv(128ull << 32, rate_srv);   /* 2^-16 cycles per transaction */
  uint64_t lat = S->hw[HW_LAT + (dram ? 5 : 4)];
  uint64_t *av = dram ? &S->dram_av : &S->l2_av;
  uint64_t m = (S->flags & F_NOCONT) ? t << 16 : max64(t << 16, *av);
  *av = m + q;
  uint64_t done = (m + q + 65535) >> 16;
  uint64_t left_engine = (uint64_t)S->st[v] + cdiv((uint64_t)(j + 1) * 128 * 65536, S->hw[HW_RATE + 4]);
  uint64_t f = max64(left_engine, done) + lat;
  if (f > S->txn_maxf[v]) S->txn_maxf[v] = f;
  if (--S->txn_left[v]) return;
  if (!complete(S, v, S->st[v], S->txn_maxf[v])) return;
  release_out(S, v, 1, S->fin[v]);
}

#define ALLOC(ptr, n) do { size_t cnt_ = (size_t)(n); (ptr) = calloc(cnt_ ? cnt_ : 1, sizeof(*(ptr))); if (!(ptr)) goto oom; } while (0)

int gtso_simulate(uint32_t n_nodes, uint32_t n_edges, uint32_t n_ctas, uint32_t n_kernels,
                  uint32_t n_ops, const uint8_t *op_cls, const uint8_t *op_flags,
                  const uint32_t *op_work, const uint32_t *op_warps, const uint16_t *node_op,
                  const uint32_t *succ_ptr, const uint32_t *succ, const uint32_t *cta_node_begin,
                  const uint32_t *kernel_cta_begin, const uint16_t *kernel_warps,
                  const uint32_t *kernel_smem, const uint8_t *kernel_cluster, const uint32_t *node_tile,
                  const uint64_t *node_addr, const uint32_t *op_rows, const uint32_t *op_pitch,
                  const uint32_t *hw, uint32_t flags,
                  uint32_t *out_cycles, uint32_t *out_makespan, int32_t *out_status,
                  uint64_t *out_digest, uint32_t *out_cta) {
  (void)n_edges;
  if (!hw || !out_makespan || !out_status) return -1;
  sim_t S;
  memset(&S, 0, sizeof S);
  S.N = n_nodes; S.C = n_ctas; S.K = n_kernels; S.P = n_ops;
  S.op_cls = op_cls; S.op_flags = op_flags; S.op_work = op_work; S.op_warps = op_warps;
  S.node_op = node_op; S.succ_ptr = succ_ptr; S.succ = succ;
  S.cta_node_begin = cta_node_begin; S.kernel_cta_begin = kernel_cta_begin;
  S.kernel_warps = kernel_warps; S.kernel_smem = kernel_smem; S.kernel_cluster = kernel_cluster;
  S.node_tile = node_tile;
  S.node_addr = node_addr; S.op_rows = op_rows; S.op_pitch = op_pitch;
  S.hw = hw; S.nsm = hw[HW_NSM]; S.nsub = hw[HW_NSUB]; S.flags = flags;
  S.noc_d = hw[HW_NOC_NODES]; S.noc_w = hw[HW_NOC_W];
  int rc = 0;

  /* R9 residency per kernel */
  ALLOC(S.slots, S.K);
  int infeasible = 0;
  for (uint32_t k = 0; k < S.K; k++) {
    uint64_t s = hw[HW_MAXCTA];
    if (kernel_smem[k]) s = s < hw[HW_SMEM] / kernel_smem[k] ? s : hw[HW_SMEM] / kernel_smem[k];
    uint64_t wl = hw[HW_MAXWARPS] / kernel_warps[k];
    s = s < wl ? s : wl;
    S.slots[k] = s;
    if (s == 0) infeasible = 1;
  }
  /* R15: clusters and REMOTE nodes need a NoC that can place them */
  for (uint32_t k = 0; k < S.K && !infeasible; k++) {
    uint32_t cl = kernel_cluster[k];
    int remote = 0;
    for (uint32_t v = cta_node_begin[kernel_cta_begin[k]]; v < cta_node_begin[kernel_cta_begin[k + 1]]; v++)
      if (op_cls[node_op[v]] == K_REMOTE) remote = 1;
    if (cl == 1 && !remote) continue;
    uint64_t sm_of_rank[16];
    if (S.noc_d == 0 || cl > S.noc_d || !place_cluster(&S, k, cl, 0, sm_of_rank)) infeasible = 1;
  }
  if (infeasible) {
    *out_status = ST_INFEASIBLE; *out_makespan = 0xFFFFFFFFu;
    if (out_digest) *out_digest = 0;
    free(S.slots);
    return 0;
  }

  /* R3 durations per op */
  ALLOC(S.occ, S.P); ALLOC(S.occm, S.P); ALLOC(S.lat, S.P); ALLOC(S.lanes, S.P); ALLOC(S.to_dram, S.P);
  ALLOC(S.occ_l2, S.P); ALLOC(S.occ_d, S.P); ALLOC(S.lat_l2, S.P); ALLOC(S.lat_d, S.P);
  for (uint32_t p = 0; p < S.P; p++) {
    uint64_t w = op_work[p];
    uint32_t cls = op_cls[p];
    if (cls == K_TENSOR || cls == K_ALU || cls == K_SFU) {
      uint32_t lanes = 0;
      for (uint32_t wp = 0; wp < 32; wp++)
        if (op_warps[p] >> wp & 1) lanes |= 1u << (wp % S.nsub);
      uint64_t k = (uint64_t)__builtin_popcount(lanes);
      S.lanes[p] = lanes;
      S.occ[p] = max64(1, cdiv(w * 65536ull * S.nsub, k * hw[HW_RATE + cls]));
      S.lat[p] = hw[HW_LAT + cls];
    } else if (cls == K_SMEM) {
      S.occ[p] = max64(1, cdiv(w * 65536ull, hw[HW_RATE + 3]));
      S.lat[p] = hw[HW_LAT + 3];
    } else if (cls == K_SYNC) {
      S.lat[p] = max64(1, hw[HW_LAT + 6]);
    } else if (cls == K_REMOTE) {
      S.occ[p] = hw[HW_NOC_RATE] ? max64(1, cdiv(w * 65536ull, hw[HW_NOC_RATE])) : 1;
      S.lat[p] = hw[HW_NOC_LAT];
    } else {
      int dram = (op_flags[p] & 1) != 0;
      S.to_dram[p] = dram;
      S.occ[p] = max64(1, cdiv(w * 65536ull, hw[HW_RATE + 4]));
      S.occm[p] = max64(1, cdiv(w * 65536ull, hw[HW_RATE + (dram ? 6 : 5)]));
      S.lat[p] = hw[HW_LAT + (dram ? 5 : 4)];
      S.occ_l2[p] = max64(1, cdiv(w * 65536ull, hw[HW_RATE + 5]));
      S.occ_d[p] = max64(1, cdiv(w * 65536ull, hw[HW_RATE + 6]));
      S.lat_l2[p] = hw[HW_LAT + 4];
      S.lat_d[p] = hw[HW_LAT + 5];
    }
  }

  /* per node / per CTA / per SM state */
  ALLOC(S.indeg, S.N); ALLOC(S.cnt, S.N); ALLOC(S.node_cta, S.N); ALLOC(S.acc, S.N);
  ALLOC(S.st, S.N); ALLOC(S.fin, S.N);
  for (uint32_t e = 0; e < succ_ptr[S.N]; e++) S.indeg[succ[e] & 0x3FFFFFFFu]++;
  ALLOC(S.cta_sm, S.C); ALLOC(S.cta_launch, S.C); ALLOC(S.cta_left, S.C);
  ALLOC(S.cta_maxfin, S.C); ALLOC(S.cta_kernel, S.C);
  for (uint32_t k = 0; k < S.K; k++)
    for (uint32_t c = kernel_cta_begin[k]; c < kernel_cta_begin[k + 1]; c++) S.cta_kernel[c] = k;
  for (uint32_t c = 0; c < S.C; c++) {
    S.cta_sm[c] = -1;
    S.cta_left[c] = cta_node_begin[c + 1] - cta_node_begin[c];
    for (uint32_t v = cta_node_begin[c]; v < cta_node_begin[c + 1]; v++) S.node_cta[v] = c;
  }
  ALLOC(S.resident, S.nsm); ALLOC(S.lane_av, (uint64_t)S.nsm * 3 * S.nsub);
  ALLOC(S.smem_av, S.nsm); ALLOC(S.eng_av, S.nsm);
  ALLOC(S.noc_av, S.noc_d ? ((uint64_t)S.nsm + S.noc_d) / S.noc_d * S.noc_d * 4 : 1);
  ALLOC(S.lru_tile, S.N); ALLOC(S.lru_lines, S.N);
  ALLOC(S.kstart, S.K);
  for (uint32_t k = 0; k < S.K; k++) S.kstart[k] = -1;
  uint64_t txn_bound = 0;  /* R17: transactions a node's tile can have */
  if (node_addr)
    for (uint32_t v = 0; v < S.N; v++)
      if (node_addr[v] != NO_ADDR) {
        uint32_t p = node_op[v];
        uint64_t R = op_rows ? op_rows[p] : 1;
        txn_bound += R * (op_work[p] / R / 128 + 2);
      }
  ALLOC(S.heap.a, (uint64_t)S.N + S.C + txn_bound);
  ALLOC(S.txn_lines, S.N); ALLOC(S.txn_n, S.N); ALLOC(S.txn_left, S.N); ALLOC(S.txn_maxf, S.N);
  ALLOC(S.lru_line, txn_bound);

  /* R6 event loop */
  dispatch(&S, 0);
  while (S.heap.n && !S.overflow) {
    uint64_t t = S.heap.a[0].key >> 32;
    int any_retire = 0;
    while (S.heap.n && (S.heap.a[0].key >> 32) == t && ((S.heap.a[0].key >> 30) & 3) == EV_RETIRE) {
      uint32_t c = (uint32_t)(heap_pop(&S.heap).key & 0x3FFFFFFFu);
      S.resident[S.cta_sm[c]]--;
      S.retired++;
      any_retire = 1;
    }
    if (any_retire) dispatch(&S, t);
    while (!S.overflow && S.heap.n && (S.heap.a[0].key >> 32) == t && ((S.heap.a[0].key >> 30) & 3) == EV_READY)
      issue(&S, (uint32_t)(heap_pop(&S.heap).key & 0x3FFFFFFFu), t);
    while (!S.overflow && S.heap.n && (S.heap.a[0].key >> 32) == t && ((S.heap.a[0].key >> 30) & 3) == EV_MEM) {
      ev_t e = heap_pop(&S.heap);
      uint32_t v = (uint32_t)(e.key & 0x3FFFFFFFu);
      if (S.node_addr && S.node_addr[v] != NO_ADDR)
        mem_txn(&S, v, e.j, t);
      else
        mem_arrive(&S, v, t);
    }
  }

  if (S.oom) goto oom;
  if (S.overflow) {
    *out_status = ST_OVERFLOW; *out_makespan = 0xFFFFFFFFu;
    if (out_digest) *out_digest = 0;
  } else if (S.nfinished != S.N) {
    *out_status = ST_DEADLOCK; *out_makespan = 0xFFFFFFFFu;
    if (out_digest) *out_digest = 0;
  } else {
    uint64_t mk = 0, dg = 0;
    for (uint32_t v = 0; v < S.N; v++) {
      if (S.fin[v] > mk) mk = S.fin[v];
      dg += mix64((((uint64_t)S.st[v] << 32) | S.fin[v]) ^ mix64((uint64_t)v + 1));
    }
    *out_status = ST_OK; *out_makespan = (uint32_t)mk;
    if (out_digest) *out_digest = dg;
  }
  if (out_cycles)
    for (uint32_t v = 0; v < S.N; v++) { out_cycles[2 * (uint64_t)v] = S.st[v]; out_cycles[2 * (uint64_t)v + 1] = S.fin[v]; }
  if (out_cta)
    for (uint32_t c = 0; c < S.C; c++) {
      out_cta[2 * (uint64_t)c] = (uint32_t)S.cta_sm[c];
      out_cta[2 * (uint64_t)c + 1] = S.cta_launch[c];
    }
  goto done;
oom:
  rc = -2;
done:
  free(S.slots); free(S.occ); free(S.occm); free(S.lat); free(S.lanes); free(S.to_dram);
  free(S.indeg); free(S.cnt); free(S.node_cta); free(S.acc); free(S.st); free(S.fin);
  free(S.cta_sm); free(S.cta_launch); free(S.cta_left); free(S.cta_maxfin); free(S.cta_kernel);
  free(S.resident); free(S.lane_av); free(S.smem_av); free(S.eng_av); free(S.kstart); free(S.heap.a);
  free(S.noc_av); free(S.lru_tile); free(S.lru_lines);
  free(S.occ_l2); free(S.occ_d); free(S.lat_l2); free(S.lat_d);
  if (S.txn_lines)
    for (uint32_t v = 0; v < S.N; v++) free(S.txn_lines[v]);
  free(S.txn_lines); free(S.txn_n); free(S.txn_left); free(S.txn_maxf); free(S.lru_line);
  return rc;
}

/* The batched call of the library's interface, restated: a graph given as
 * one struct with the field order of the library's host graph (counts, then
 * the array pointers), B hardware records of 32 words each, outputs per
 * record b at out_cycles + b * 2 * n_nodes (optional), out_makespan[b],
 * out_status[b], out_digest[b] (optional).  Each record is one independent
 * simulation run by gtso_simulate, in record order.  Returns 0, -1 for a
 * missing argument, -2 when host memory runs out. */
typedef struct gtso_graph_host {
  uint32_t n_nodes, n_edges, n_ctas, n_kernels, n_ops;
  const uint8_t *op_cls, *op_flags;
  const uint32_t *op_work, *op_warps;
  const uint16_t *node_op;
  const uint32_t *succ_ptr, *succ, *cta_node_begin, *kernel_cta_begin;
  const uint16_t *kernel_warps;
  const uint32_t *kernel_smem;
  const uint8_t *kernel_cluster; /* NULL: one CTA per cluster everywhere */
  const uint32_t *node_tile;     /* NULL: no node names a tile */
  const uint64_t *node_addr;     /* NULL: no node has a tile address */
  const uint32_t *op_rows, *op_pitch;  /* NULL: one row; pitch = row bytes */
} gtso_graph_host;

int gts_oracle_simulate(const gtso_graph_host *h, const uint32_t *hw, uint32_t B, uint32_t *out_cycles,
                        uint32_t *out_makespan, int32_t *out_status, uint64_t *out_digest, uint32_t flags) {
  if (!h || (B && (!hw || !out_makespan || !out_status))) return -1;
  uint8_t *ones = NULL;
  const uint8_t *cluster = h->kernel_cluster;
  if (!cluster) {
    ones = malloc(h->n_kernels ? h->n_kernels : 1);
    if (!ones) return -2;
    memset(ones, 1, h->n_kernels ? h->n_kernels : 1);
    cluster = ones;
  }
  int rc = 0;
  for (uint32_t b = 0; b < B && rc == 0; b++)
    rc = gtso_simulate(h->n_nodes, h->n_edges, h->n_ctas, h->n_kernels, h->n_ops, h->op_cls, h->op_flags,
                       h->op_work, h->op_warps, h->node_op, h->succ_ptr, h->succ, h->cta_node_begin,
                       h->kernel_cta_begin, h->kernel_warps, h->kernel_smem, cluster, h->node_tile,
                       h->node_addr, h->op_rows, h->op_pitch, hw + 32 * (uint64_t)b, flags,
                       out_cycles ? out_cycles + 2 * (uint64_t)h->n_nodes * b : NULL, out_makespan + b,
                       out_status + b, out_digest ? out_digest + b : NULL, NULL);
  free(ones);
  return rc;
}
