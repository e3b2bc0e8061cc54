/*
 * gts.h — C ABI of the batched tile-graph simulation library (libgts.so).
 *
 * The library simulates warp-level tile graphs (GTSim, arXiv 2607.11262)
 * under a throughput-oriented hardware model and returns, for every node of
 * the graph and every hardware configuration of a batch, the integer cycle at
 * which the node starts and finishes.  One MI355X wavefront simulates one
 * (graph, hardware) pair; the batch is data-parallel.
 *
 * Paper passages the calls follow:
 *   - graph model, node and edge semantics ........ Sec. 4.1 (Tile Graph Abstraction)
 *   - user-built graphs consumed by the backend .... Sec. 4.3 (second path)
 *   - backend execution flow, order edges released
 *     at issue, data edges at completion, TB
 *     retire / re-dispatch ......................... Sec. 5.1, Sec. 5.3
 *   - resources as (latency, width, throughput) ... Sec. 5.2
 *   - DSMEM / SM-cluster NoC, thread-block
 *     clusters ..................................... Sec. 5.2, Sec. 7.2
 *   - L2 as a fully associative LRU of lines ...... Sec. 5.2
 *   - template sharing of isomorphic CTA graphs ... Sec. 6.4
 *   - hardware parameters ......................... Sec. 6.1, Table 3
 * Every point the paper leaves open (integer cycles, tie-breaking, phase order
 * within a cycle, servers, residency, NoC arithmetic) is fixed by one set of
 * timing rules, restated at the top of each kernel source (gts_sim.hip,
 * gts_window.hip) and next to the code that implements each rule.
 *
 * Conventions
 *   - Every entry point returns an int status: GTS_OK (0) or a negative
 *     GTS_E_* code.  No C++ exception crosses this boundary.  gts_strerror()
 *     names a code; gts_last_error() returns a thread-local message with the
 *     offending index or value of the last failing call on this thread.
 *   - The caller owns every buffer.  Device buffers are plain device pointers
 *     (hipMalloc'd, or a torch CUDA tensor's data_ptr()); host buffers are
 *     plain host pointers.  The library owns only the small opaque gts_graph
 *     handle, which refers to (does not own) the caller's device image buffer;
 *     that buffer must outlive the handle and every simulation using it.
 *   - Streams are passed as void* (a hipStream_t; NULL = the null stream).
 */
#ifndef GTS_H
#define GTS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------ */
#define GTS_OK            0
#define GTS_E_ARG        -1  /* null pointer, zero/oversized count, bad flag   */
#define GTS_E_CYCLE      -2  /* graph has a directed cycle (incl. self-loop)   */
#define GTS_E_EDGE_ORDER -3  /* edge from a higher to a lower CTA, not within
                                one cluster                                  */
#define GTS_E_RANGE      -4  /* index / class / warp mask / degree out of range*/
#define GTS_E_HW         -5  /* invalid hardware parameter record             */
#define GTS_E_SCRATCH    -6  /* scratch or device image buffer too small       */
#define GTS_E_HIP        -7  /* a HIP runtime call failed                      */
#define GTS_E_DUP        -8  /* the same (u, v) pair appears twice in succ     */

/* ---- per-simulation status (written to out_status[b]) ------------------ */
#define GTS_SIM_OK         0
#define GTS_SIM_INFEASIBLE 1  /* some kernel fits zero CTAs on an SM          */
#define GTS_SIM_OVERFLOW   2  /* some finish cycle would exceed 0xFFFFFFFE    */
#define GTS_SIM_DEADLOCK   3  /* events ran out with nodes unscheduled        */
/* For a non-OK simulation out_makespan[b] = 0xFFFFFFFF, out_digest[b] = 0 and
 * its rows of out_cycles are unspecified. */

/* ---- operation classes (Sec. 4.1 operation descriptor; Sec. 5.2 units) - */
#define GTS_TENSOR 0  /* tensor-core MMA;  work = FLOPs (2 per FMA)           */
#define GTS_ALU    1  /* CUDA-core / elementwise; work = operations           */
#define GTS_SFU    2  /* special-function unit;  work = operations            */
#define GTS_SMEM   3  /* shared-memory LD/ST pipe; work = bytes               */
#define GTS_GLOAD  4  /* global->shared tile load (TMA / cp.async); bytes     */
#define GTS_GSTORE 5  /* shared->global tile store; bytes                     */
#define GTS_SYNC   6  /* barrier / signal-wait node; no resource, work unused */
#define GTS_REMOTE 7  /* DSMEM access to another CTA of the cluster over the
                         SM-cluster NoC (Sec. 5.2); work = bytes            */
#define GTS_N_CLASSES 8

#define GTS_OPF_MISS 1u  /* GLOAD/GSTORE: served by DRAM instead of L2       */
/* REMOTE: the target CTA's rank within the source CTA's cluster is
 * (flags >> GTS_OPF_RANK_SHIFT); no other flag bit is set. */
#define GTS_OPF_RANK_SHIFT 4
#define GTS_NO_TILE 0xFFFFFFFFu  /* node_tile entry of an untracked node    */
#define GTS_LINE_BYTES 128u      /* L2 line of the LRU model, and the memory
                                    transaction of transaction-level tiles  */
#define GTS_NO_ADDR 0xFFFFFFFFFFFFFFFFull  /* node_addr entry of a node
                                              without a tile address      */
#define GTS_MAX_NODE_TXN (1u << 21)  /* bound on one addressed tile's
                                        transactions: rows * (row bytes / 128
                                        + 2) may not exceed it             */

/* ---- edge kinds (Sec. 4.1 edge semantics) ------------------------------ */
/* succ[] entries are  target | (kind << GTS_EDGE_KIND_SHIFT).              */
#define GTS_EDGE_DATA  0u  /* released when the source finishes            */
#define GTS_EDGE_ORDER 1u  /* program order: released at source start + 1  */
#define GTS_EDGE_SYNC  2u  /* signal/wait, barrier, buffer reuse: at finish */
#define GTS_EDGE_KIND_SHIFT 30
#define GTS_EDGE_TARGET_MASK 0x3FFFFFFFu

/* ---- simulate flags ---------------------------------------------------- */
#define GTS_OUT_NODES       1u  /* write out_cycles                            */
#define GTS_OUT_DIGEST      2u  /* write out_digest                            */
#define GTS_NO_CONTENTION   4u  /* servers never delay a node (test mode)      */
#define GTS_ORDER_AT_FINISH 8u  /* ORDER edges release at finish (test mode)   */
#define GTS_FLAGS_ALL      15u

/* ---- limits -------------------------------------------------------------- */
#define GTS_MAX_NODES   0x3FFFFFFFu  /* node ids fit the 30-bit edge target  */
#define GTS_MAX_CTAS    (1u << 24)
#define GTS_MAX_KERNELS 65535u
#define GTS_MAX_OPS     65535u
#define GTS_MAX_INDEG   65535u
#define GTS_MAX_WARPS   32u           /* warps per CTA (op warp masks are u32) */
#define GTS_MAX_SM      1024u
#define GTS_MAX_SUBPART 8u
#define GTS_MAX_CLUSTER 16u           /* CTAs per thread-block cluster        */
#define GTS_MAX_NOC     64u           /* SMs per NoC domain                   */

/* ---- hardware parameters (Table 3; integer cycles, Q16.16 rates) -------- */
/* Rates are work units per core cycle in Q16.16 (value * 65536), per SM for
 * TENSOR/ALU/SFU/SMEM/GMEM and chip-wide for L2/DRAM.  Latencies are core
 * cycles.  A record is exactly 32 little-endian u32 words. */
#define GTS_RATE_TENSOR 0
#define GTS_RATE_ALU    1
#define GTS_RATE_SFU    2
#define GTS_RATE_SMEM   3
#define GTS_RATE_GMEM   4   /* per-SM global-memory engine (TMA / LSU)      */
#define GTS_RATE_L2     5
#define GTS_RATE_DRAM   6
#define GTS_LAT_TENSOR  0
#define GTS_LAT_ALU     1
#define GTS_LAT_SFU     2
#define GTS_LAT_SMEM    3
#define GTS_LAT_L2      4
#define GTS_LAT_DRAM    5
#define GTS_LAT_SYNC    6

typedef struct gts_hw_params {
  uint32_t n_sm;             /* 1 .. GTS_MAX_SM                              */
  uint32_t n_subpart;        /* 1 .. GTS_MAX_SUBPART; lane of warp w = w % n */
  uint32_t max_cta_per_sm;   /* 0 makes every simulation INFEASIBLE          */
  uint32_t max_warps_per_sm;
  uint32_t smem_per_sm;      /* bytes                                        */
  uint32_t rate_q16[7];      /* GTS_RATE_*, each >= 1                        */
  uint32_t lat[7];           /* GTS_LAT_*, each <= 2^30                      */
  uint32_t cta_launch_lat;   /* added to every CTA's launch, <= 2^30         */
  uint32_t kernel_launch_lat;/* added to a kernel's first-wave CTAs, <= 2^30 */
  /* SM-cluster NoC (Sec. 5.2 DSMEM; Sec. 7.2 crossbar vs mesh, mapping).  SM
   * s belongs to NoC domain s / noc_nodes as its node s % noc_nodes; a
   * cluster's CTAs are placed on distinct SMs of one domain.  noc_nodes = 0:
   * no NoC (a kernel with clusters of more than one CTA is then INFEASIBLE). */
  uint32_t noc_nodes;        /* SMs per domain, 0 .. GTS_MAX_NOC             */
  uint32_t noc_width;        /* 0: crossbar; else a mesh noc_width wide with
                                noc_nodes / noc_width rows (XY routing)      */
  uint32_t noc_rate_q16;     /* bytes per cycle of one crossbar port / mesh
                                link, Q16.16, >= 1 when noc_nodes > 0        */
  uint32_t noc_lat;          /* crossbar traversal / mesh per-hop cycles,
                                <= 2^24                                      */
  uint32_t noc_map;          /* cluster placement: 0 strips of consecutive
                                nodes, 1 compact blocks (mesh), 2 strided
                                (ranks noc_nodes / cluster nodes apart)      */
  /* L2 as a fully associative LRU cache of l2_lines 128-B lines (Sec. 5.2):
   * a load / store that names its tile (node_tile) touches the tile's
   * cdiv(bytes, 128) lines at its L2 arrival and hits (L2 server) iff the
   * tile was touched before and its lines plus the distinct lines of other
   * tiles touched since fit in l2_lines, else misses (DRAM server).  0: the
   * op's GTS_OPF_MISS flag decides, as for nodes without a tile. */
  uint32_t l2_lines;
  uint32_t reserved[5];      /* must be zero                                 */
} gts_hw_params;

/* ---- host-side graph (Sec. 4.1; dictionary-encoded descriptors) --------- */
/* Nodes are numbered CTA-major: CTA c owns nodes [cta_node_begin[c],
 * cta_node_begin[c+1]); CTAs are numbered kernel-major: kernel k owns CTAs
 * [kernel_cta_begin[k], kernel_cta_begin[k+1]).  Every CTA and every kernel
 * is non-empty.  An op is one distinct (class, flags, work, warp mask) tuple;
 * node v executes op node_op[v].  The successors of v are
 * succ[succ_ptr[v] .. succ_ptr[v+1]).  Validity: acyclic; no duplicate (u,v);
 * cta(u) <= cta(v) for every edge, except between two CTAs of one cluster
 * (whose CTAs are dispatched together); in-degree <= GTS_MAX_INDEG; compute
 * ops (TENSOR/ALU/SFU) have a non-empty warp mask inside [0, warps of the
 * kernel of every CTA that uses them); the CTAs of kernel k form clusters of
 * kernel_cluster[k] consecutive CTAs (1 .. GTS_MAX_CLUSTER, dividing the
 * kernel's CTA count; kernel_cluster = NULL means 1 for every kernel), and a
 * REMOTE op's target rank is below the cluster size of every kernel that
 * uses it; only GLOAD / GSTORE nodes carry a tile, and every node of one
 * tile has the same cdiv(work, 128) lines; only GLOAD / GSTORE nodes carry
 * an address, never in a graph whose nodes name tiles by id, and an
 * addressed node's op has work > 0 divisible by its rows, a row stride of at
 * least the row bytes, at most GTS_MAX_NODE_TXN transactions, and its bytes
 * below GTS_NO_ADDR.  An empty graph has all counts zero. */
typedef struct gts_graph_host {
  uint32_t n_nodes, n_edges, n_ctas, n_kernels, n_ops;
  const uint8_t  *op_cls;           /* [n_ops]  GTS_TENSOR .. GTS_REMOTE     */
  const uint8_t  *op_flags;         /* [n_ops]  GTS_OPF_*                    */
  const uint32_t *op_work;          /* [n_ops]                               */
  const uint32_t *op_warps;         /* [n_ops]  warp mask within the CTA     */
  const uint16_t *node_op;          /* [n_nodes]                             */
  const uint32_t *succ_ptr;         /* [n_nodes + 1], succ_ptr[0] = 0        */
  const uint32_t *succ;             /* [n_edges]                             */
  const uint32_t *cta_node_begin;   /* [n_ctas + 1]                          */
  const uint32_t *kernel_cta_begin; /* [n_kernels + 1]                       */
  const uint16_t *kernel_warps;     /* [n_kernels], 1 .. GTS_MAX_WARPS       */
  const uint32_t *kernel_smem;      /* [n_kernels], shared memory per CTA    */
  const uint8_t  *kernel_cluster;   /* [n_kernels] CTAs per cluster, or NULL */
  const uint32_t *node_tile;        /* [n_nodes] tile of a GLOAD / GSTORE, or
                                       GTS_NO_TILE; NULL: no node has one    */
  /* Transaction-level memory (Sec. 5.2 Memory, Sec. 5.3 memory nodes): a
   * GLOAD / GSTORE node with an address accesses its op's tile of op_rows
   * rows of op_work / op_rows bytes, row r at node_addr + r * op_pitch; the
   * tile's distinct 128-B lines (in the order the rows first reach them)
   * are its transactions, streamed by the SM's engine at its rate and
   * served one by one by the L2 / DRAM servers (an LRU of lines decides
   * which when l2_lines > 0, else the op's MISS flag); the node completes
   * with its last transaction. */
  const uint64_t *node_addr;        /* [n_nodes] tile address or GTS_NO_ADDR;
                                       NULL: no node has one                 */
  const uint32_t *op_rows;          /* [n_ops] rows of the tile, >= 1;
                                       NULL: one row                         */
  const uint32_t *op_pitch;         /* [n_ops] bytes between rows, >= row
                                       bytes for ops of addressed nodes;
                                       NULL: row bytes (rows packed)         */
} gts_graph_host;

typedef struct gts_graph gts_graph;  /* opaque handle to an uploaded graph */

/* ---- entry points --------------------------------------------------------- */

/* Checks every validity rule above on the host.  Needs no GPU.  Returns
 * GTS_OK or the first violated rule's code (message: gts_last_error()).
 * Follows Sec. 4.1 (nodes, data / order edges, the CTA and warp each node is
 * bound to); the CTA-order and acyclicity rules are what keep the Sec. 5.1
 * dispatch order deadlock-free. */
int gts_graph_validate(const gts_graph_host *h);

/* Validates h and returns in *bytes the size of its device image (the layout
 * the simulation kernels read).  Needs no GPU.  Sizing only (no passage of
 * the paper: the image layout is this library's). */
int gts_graph_device_bytes(const gts_graph_host *h, uint64_t *bytes);

/* Template sharing (GTSim Sec. 6.4: CTAs that execute isomorphic tile graphs
 * share one graph structure; each logical CTA keeps only light metadata).
 * Validates h and reports how its device image shares structure: a kernel
 * whose CTAs all have the same node count and the same local successor lists
 * and edge kinds, with no edge leaving or entering a CTA, keeps one template
 * of node records; its CTAs then differ only in op ids, grouped into classes
 * (at most 255 per kernel) by a class x slot op table of at most 128 entries
 * per graph.  Outputs (any may be NULL): *templated_kernels, *template_nodes
 * (records of all templates), *expanded_nodes (nodes of the kernels without
 * a template), *class_ops (table entries).  The device image always also
 * holds every node's expanded record.  Setting the environment variable
 * GTS_TEMPLATES=0 before an upload turns sharing off (this call then reports
 * no templated kernel).  Needs no GPU.  Returns GTS_OK or a validation
 * error. */
int gts_graph_templates(const gts_graph_host *h, uint32_t *templated_kernels, uint32_t *template_nodes,
                        uint32_t *expanded_nodes, uint32_t *class_ops);

/* Validates h, builds its device image on the host and copies it into the
 * caller's device buffer dev_image (dev_bytes >= gts_graph_device_bytes) on
 * hip_stream, waiting for the copy to finish before returning.  On success
 * *out receives a new handle; h's arrays are not referenced afterwards.
 * Follows Sec. 4.3 (a graph built directly by the user is handed to the
 * simulation backend) over the Sec. 4.1 graph model; isomorphic CTAs share
 * one template (Sec. 6.4).  Errors: the validation codes above, GTS_E_SCRATCH
 * when dev_bytes is too small, GTS_E_HIP when the copy fails. */
int gts_graph_upload(const gts_graph_host *h, void *dev_image, uint64_t dev_bytes,
                     void *hip_stream, gts_graph **out);

/* Frees the handle (not the caller's device image).  NULL is accepted. */
int gts_graph_release(gts_graph *g);

/* Graph sizes of an uploaded graph (any pointer may be NULL). */
int gts_graph_sizes(const gts_graph *g, uint32_t *n_nodes, uint32_t *n_edges,
                    uint32_t *n_ctas, uint32_t *n_kernels, uint32_t *n_ops);

/* Bytes of device scratch gts_simulate_batch needs for B simulations of g
 * with these flags.  The scratch holds the batch's hardware records and every
 * simulation's private state; its contents need not be initialised.  Sizing
 * only (no passage of the paper). */
int gts_scratch_bytes(const gts_graph *g, uint32_t B, uint32_t flags, uint64_t *bytes);

/* Simulates g under hw_host[0..B) (host array, read before return): the
 * backend of Sec. 5 -- execution flow and release of order edges at issue,
 * data edges at completion, thread-block retire and re-dispatch (Sec. 5.1,
 * Sec. 5.3), resources as latency / width / throughput servers, the memory
 * path and the NoC (Sec. 5.2) -- under the hardware parameters of Table 3
 * (Sec. 6.1).  Outputs
 * (device pointers, written asynchronously on hip_stream):
 *   out_cycles   [B][n_nodes][2] u32 {start, finish}; required iff
 *                flags & GTS_OUT_NODES, else ignored (may be NULL)
 *   out_makespan [B]  max finish over all nodes (0 for an empty graph)
 *   out_status   [B]  GTS_SIM_*
 *   out_digest   [B]  order-independent 64-bit digest of all (start, finish)
 *                pairs; required iff flags & GTS_OUT_DIGEST
 * Errors in arguments or in any hw record (GTS_E_HW, with the record index in
 * gts_last_error()) are reported before anything is enqueued; so is
 * GTS_E_HW for a batch whose largest n_sm and n_subpart need more LDS for
 * the per-SM servers than one workgroup may hold on the current device
 * (about 108 KiB at 1024 SMs x 8 subpartitions).  Per-simulation
 * outcomes go to out_status.  Results are valid once hip_stream completes;
 * calls on different streams with disjoint scratch and outputs are
 * independent.  B = 0 is a no-op. */
int gts_simulate_batch(const gts_graph *g, const gts_hw_params *hw_host, uint32_t B,
                       uint32_t *out_cycles, uint32_t *out_makespan, int32_t *out_status,
                       uint64_t *out_digest, void *scratch, uint64_t scratch_bytes,
                       uint32_t flags, void *hip_stream);

/* ---- device-resident hardware sets ---------------------------------------- */
typedef struct gts_hwset gts_hwset;  /* opaque handle to uploaded hw records */

/* Bytes of device memory gts_hwset_upload needs for B records. */
int gts_hwset_device_bytes(uint32_t B, uint64_t *bytes);

/* Hardware records of Table 3 (Sec. 6.1) resident in device memory.
 * Validates hw_host[0..B) (GTS_E_HW names the first bad record), copies the
 * records into the caller's device buffer dev_buf (>= gts_hwset_device_bytes)
 * on hip_stream and waits for the copy.  *out receives a handle that refers
 * to (does not own) dev_buf and remembers the largest n_sm / n_subpart /
 * noc_nodes of the set. */
int gts_hwset_upload(const gts_hw_params *hw_host, uint32_t B, void *dev_buf, uint64_t dev_bytes,
                     void *hip_stream, gts_hwset **out);

/* Frees the handle (not the caller's buffer).  NULL is accepted. */
int gts_hwset_release(gts_hwset *hw);

/* As gts_simulate_batch (Sec. 5.1-5.3 under Table 3 parameters), for the B
 * records hw[first .. first + B) of an uploaded set (already in device
 * memory: no host copy is made).  Output row b belongs to record first + b.
 * Scratch: gts_scratch_bytes(g, B, ...).  Errors as gts_simulate_batch, plus
 * GTS_E_ARG when first + B exceeds the set. */
int gts_simulate_hwset(const gts_graph *g, const gts_hwset *hw, uint32_t first, uint32_t B,
                       uint32_t *out_cycles, uint32_t *out_makespan, int32_t *out_status,
                       uint64_t *out_digest, void *scratch, uint64_t scratch_bytes,
                       uint32_t flags, void *hip_stream);

/* ---- no-allocation entry point ------------------------------------------- */
/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, results and errors as gts_simulate_hwset without the scratch
 * pair: the simulations' scratch is a static device array of
 * GTS_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held from the
 * library's first use on that GPU until the process ends.  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine);
 * on its first call on a device it looks up the array's device address once.
 * B must satisfy gts_scratch_bytes(g, B, flags) - 128 * B (rounded up to 256)
 * <= GTS_NOALLOC_SCRATCH_BYTES, i.e. the scratch gts_simulate_hwset would
 * need; a larger B returns GTS_E_SCRATCH (the message names the largest B
 * that fits) before anything is enqueued.  The array needs no
 * initialisation and keeps the last call's contents.  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (other streams,
 * other threads) race and give undefined results -- serialise them, e.g. on
 * one stream. */
#define GTS_NOALLOC_SCRATCH_BYTES (128ull << 20)
int gts_simulate_hwset_noalloc(const gts_graph *g, const gts_hwset *hw, uint32_t first, uint32_t B,
                               uint32_t *out_cycles, uint32_t *out_makespan, int32_t *out_status,
                               uint64_t *out_digest, uint32_t flags, void *hip_stream);

/* Checks one hardware record (Table 3 parameters) on the host (GTS_OK or
 * GTS_E_HW). */
int gts_hw_validate(const gts_hw_params *hw);

const char *gts_strerror(int code);
const char *gts_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GTS_H */
