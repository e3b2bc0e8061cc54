// gts_dev.h — device image and scratch layouts shared by the host library
// (gts_host.cpp) and the simulation kernels (gts_sim.hip).  Internal to
// libgts.so; the public ABI is include/gts.h.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gts {

constexpr uint32_t kImageMagic = 0x47545331u;  // "GTS1"
constexpr uint32_t kMaxCycle = 0xFFFFFFFEu;     // largest representable finish
constexpr uint32_t kAlign = 256;

// Graph property bits (computed at upload).
constexpr uint32_t kGraphSinksAreMemory = 1u;   // every node without an intra-CTA
                                                // successor is a GLOAD/GSTORE
constexpr uint32_t kGraphCrossFromMemory = 2u;  // every cross-CTA edge has a
                                                // GLOAD/GSTORE source, DATA/SYNC kind
constexpr uint32_t kGraphSmallOutdeg = 4u;      // every out-degree is below 0xFFFF
constexpr uint32_t kGraphHasShared = 8u;        // some CTA receives cross-CTA edges
constexpr uint32_t kGraphComputeFeedsData = 16u;  // every non-memory node has a DATA or
                                                  // SYNC out-edge inside its CTA
constexpr uint32_t kGraphClassShift = 5u;         // bits 5-7: the op table has TENSOR /
                                                  // ALU / SFU ops (one bit per class)
constexpr uint32_t kGraphClusters = 256u;         // some kernel has clusters of more than
                                                  // one CTA or REMOTE nodes
constexpr uint32_t kGraphTiles = 512u;            // some load / store names its tile
constexpr uint32_t kGraphTxn = 1024u;             // some load / store has a tile address
                                                  // (transaction-level memory)
constexpr uint32_t kGraphSmem = 2048u;            // the op table has shared-memory ops

// Compute pipelines: every subpartition of an SM has one lane per compute
// class.  Server state holds lanes only for the classes a graph uses, class
// slot-major: slot(c) = number of used classes below c.
__host__ __device__ inline uint32_t compute_slots(uint32_t props) {
  return (uint32_t)__builtin_popcount((props >> kGraphClassShift) & 7u);
}
__host__ __device__ inline uint32_t compute_slot(uint32_t props, uint32_t cls) {
  return (uint32_t)__builtin_popcount((props >> kGraphClassShift) & ((1u << cls) - 1u));
}

struct ImageHeader {            // at offset 0 of the device image
  uint32_t magic, n_nodes, n_edges, n_ctas, n_kernels, n_ops, n_roots, props;
  uint64_t off_ops, off_nodes, off_succ, off_ctas, off_kernels, off_roots, off_indeg;
  uint64_t off_tnodes, off_tsucc, off_tindeg, off_cclass, off_tops, off_tile, off_txn_ptr, off_txn_line;
  uint32_t max_cta_nodes, max_outdeg, n_tnodes, n_tsucc, n_tops, pad;
};

struct OpDev {                  // one distinct operation descriptor
  uint8_t cls, flags;
  uint16_t pad;
  uint32_t work, warps, pad2;
};

constexpr uint32_t kInlineSucc = 3;
struct NodeDev {                // 32 B, one per node and a sentinel after the last
  uint32_t op_nsucc;            // op id (low 16) | out-degree (high 16, 0xFFFF if larger)
  uint32_t cta;
  uint32_t succ_begin;          // successors: succ[succ_begin, next record's succ_begin)
  uint32_t succ[kInlineSucc];   // copies of the first three successors
  uint16_t sindeg[kInlineSucc]; // and their in-degrees
  uint16_t pad;                 // template records: kRecSink on the retiring sink
};
// Template record flag: the CTA's retiring sink (its kernel has pad[0] = 1:
// every node reaches this load / store over DATA / SYNC edges, so the CTA
// retires at its finish).
constexpr uint16_t kRecSink = 1;

constexpr uint32_t kInlineRoots = 3;
struct CtaDev {                 // 32 B, one per CTA
  uint32_t node_begin, node_count;
  uint32_t root_begin, root_count;  // nodes without intra-CTA in-edges; bit 31 of
                                    // root_count: the CTA receives cross-CTA edges
  uint32_t mem_count;               // GLOAD / GSTORE nodes
  uint32_t root[kInlineRoots];      // copies of the first three roots
};
constexpr uint32_t kCtaShared = 0x80000000u;

// Template sharing (Sec. 6.4: CTAs that run isomorphic tile graphs share one
// graph structure).  A kernel whose CTAs all have the same node count and the
// same local successor lists (no cross-CTA edges) keeps one "template" of
// node records: successor targets are local indices, and the op field is a
// slot.  The CTAs differ only in op ids (e.g. an L2-miss variant of a load
// for a first-touch tile): each CTA has a class, and the op of slot s in
// class q is tops[t_ops + q * t_nslot + s].  The expanded records stay in the
// image for the general kernel.
struct KernelDev {              // 48 B, one per kernel
  uint32_t cta_begin, cta_end, warps, smem;
  uint32_t node_begin;          // first node of the kernel
  uint32_t t_n;                 // nodes per CTA if templated, else 0
  uint32_t t_base;              // first template record (and in-degree) of the kernel
  uint32_t t_ops;               // tops offset (low 16) | slots per class (high 16)
  uint32_t cluster;             // CTAs per cluster | kKernelRemote
  uint32_t pad[3];              // pad[0]: 1 if the template's CTAs retire with their sink
};
constexpr uint32_t kKernelRemote = 0x10000u;  // the kernel has REMOTE nodes
constexpr uint32_t kMaxTops = 128;   // class x slot op entries per graph (held in LDS)

// Device-side view passed to kernels by value.
struct Image {
  const OpDev* ops;
  const NodeDev* nodes;
  const uint32_t* succ;
  const CtaDev* ctas;
  const KernelDev* kernels;
  const uint32_t* roots;
  const uint16_t* indeg;        // in-degree per node
  const NodeDev* tnodes;        // template records (succ: local index | bits)
  const uint32_t* tsucc;        // template successors beyond the records' inline ones
  const uint16_t* tindeg;       // in-degree per template record
  const uint8_t* cclass;        // class of each CTA of a templated kernel
  const uint16_t* tops;         // [n_tops] class x slot -> op id
  const uint32_t* tile;         // [N] tile of each load / store, numbered 0..n_tiles-1 (kGraphTiles), else null
  // transaction-level memory (kGraphTxn, else null): node v's transactions
  // are the lines txn_line[txn_ptr[v] .. txn_ptr[v + 1]) (none: the node has
  // no address), lines numbered densely 0..n_lines-1 in order of first use
  const uint32_t* txn_ptr;      // [N + 1]
  const uint32_t* txn_line;     // [n_txn]
  uint32_t n_nodes, n_edges, n_ctas, n_kernels, n_ops, props, n_tops;
  uint32_t n_tiles;             // distinct tiles
  uint32_t n_txn, n_lines;      // transactions of all addressed nodes, distinct lines
};

// Hardware record word indices (gts_hw_params field order).
enum : uint32_t {
  HW_NSM = 0, HW_NSUB = 1, HW_MAXCTA = 2, HW_MAXWARPS = 3, HW_SMEM = 4,
  HW_RATE = 5, HW_LAT = 12, HW_CTALAT = 19, HW_KLAT = 20, HW_WORDS = 32
};
enum : uint32_t { R_TENSOR = 0, R_ALU, R_SFU, R_SMEM, R_GMEM, R_L2, R_DRAM };
enum : uint32_t { L_TENSOR = 0, L_ALU, L_SFU, L_SMEM, L_L2, L_DRAM, L_SYNC };
enum : uint32_t { C_TENSOR = 0, C_ALU, C_SFU, C_SMEM, C_GLOAD, C_GSTORE, C_SYNC, C_REMOTE };
enum : uint32_t { HW_NOC_NODES = 21, HW_NOC_W = 22, HW_NOC_RATE = 23, HW_NOC_LAT = 24, HW_NOC_MAP = 25,
                  HW_L2_LINES = 26 };
// Device-image edge encoding: target | bits << 30.  DATA and SYNC edges time
// identically (released at the source's finish) and share bit pattern 0;
// bit 30 marks an ORDER edge (released at the source's start + 1), bit 31 an
// edge into a "shared" node (one with an in-edge from another CTA), whose
// state is updated with atomics by the windowed kernel.
constexpr uint32_t kDevOrder = 1u, kDevShared = 2u;

// Per-SM server words: compute lanes (slots x n_subpart), then the shared-
// memory pipe (only for graphs with shared-memory ops, or without compute
// ops) and the global-memory engine; the pipe's index is stride - 2, the
// engine's stride - 1.
__host__ __device__ inline uint32_t server_stride(uint32_t props, uint32_t nsub) {
  const uint32_t slots = compute_slots(props);
  return slots * nsub + ((props & kGraphSmem) || slots == 0u ? 2u : 1u);
}

// Per-simulation scratch regions (byte offsets within one simulation's slice).
struct SimLayout {
  uint64_t off_state;   // u64 per node: acc (low 32) | released in-edges (high 32)
  uint64_t off_cta;     // CtaState per CTA
  uint64_t off_pend;    // pending events: u64 key + u32 aux per entry
  uint64_t off_optab;   // per-op duration table when it does not fit LDS
  uint64_t off_rp;      // windowed kernel: later ready entries beyond LDS, [kPoolSpill][64] u64
  uint64_t off_mq;      // windowed kernel: memory-arrival rings, [kWinMaxSm][kRing] x 3 u32
  uint64_t off_ret;     // windowed kernel: pending retirements beyond LDS (u64 each)
  uint64_t off_lru;     // LRU L2: latest access stamp per tile or line ([keys] u32)
  uint64_t off_lru_bit; // LRU L2: Fenwick tree of lines over stamps ([accesses + 1] u64)
  uint64_t pend_cap;
  uint64_t stride;      // bytes per simulation (multiple of kAlign)
};

struct CtaState {
  uint32_t sm, launch, left, maxfin;
};

// Windowed kernel limits.
constexpr uint32_t kWinMaxSm = 256;    // largest n_sm it simulates (four SMs per lane)
constexpr uint32_t kNear = 4;          // ready entries per lane due in the current window (LDS)
constexpr uint32_t kPoolSpill = 240;   // later ready entries per lane beyond the LDS part
constexpr uint32_t kRing = 64;         // memory-arrival FIFO entries per SM
constexpr uint32_t kRingWords = 3;     // words per entry: key low, key high, op
constexpr uint32_t kRingWordsTxn = 8;  // transaction-level memory: node, entry cycle, remainder, line index, lines left
constexpr uint32_t kRetireLds = 0;     // pending CTA retirements held in LDS (none: the room went to kWinCap) ...
constexpr uint32_t kRetireCap = 8192;  // ... and in all (the rest spilled to scratch)
constexpr uint32_t kWinCap = 256;      // memory arrivals (or retirements) per window
constexpr uint32_t kWindowMax = 1024;  // longest window, in cycles
constexpr uint64_t kWinMaxTileLines = 1ull << 22;  // LRU L2: lines of a tile the windowed kernel takes (below)
constexpr int32_t kStatusRetry = 0x52455452;  // rerun this simulation on the general kernel
constexpr uint64_t kStatsBytes = 128;          // windowed-kernel counters at the end of a slice

struct Launch {
  Image img;
  const uint32_t* hw;          // [B][32]
  uint8_t* sims;               // B slices of layout.stride bytes
  SimLayout layout;
  uint32_t* out_cycles;        // [B][N][2] or null
  uint32_t* out_makespan;
  int32_t* out_status;
  uint64_t* out_digest;        // or null
  uint32_t B, flags;
  uint32_t lds_optab;          // op table held in LDS (else in scratch)
  uint32_t lds_words_servers;  // words of per-SM server state reserved in LDS
  uint32_t retry_only;         // general kernel: run only simulations marked kStatusRetry
  uint32_t max_nsm;            // largest n_sm of the batch
  uint32_t max_nsub;           // largest n_subpart of the batch
  uint32_t qp;                 // windowed kernel: later ready entries per lane held in LDS
  uint32_t noc_words;          // general kernel: NoC server words after the per-SM servers
  uint32_t clocks;             // windowed kernel: time its phases with the shader clock
  uint32_t srv_one;            // one server word per compute class (every compute op holds every subpartition
                               // lane of every record, so their lanes' times stay equal)
};

// LDS carve-up of the windowed kernel (32-bit words; 64-bit arrays start on
// even words).  The parts of fixed size come first, at constant offsets the
// kernel addresses without registers; then the parts sized by the batch.
// NS: largest n_sm of the batch; SS: server words per SM (server_stride at
// the largest n_subpart); QP: later ready entries per lane held in LDS; NT:
// template class x slot op entries (u16); mode: kWinPlain, kWinTiles (loads /
// stores name tiles: one word per memory-batch position for the LRU
// decisions) or kWinTxn (transaction-level memory: that word, and per
// batch slot a line index, the next line's entry cycle, a node's largest
// finish so far and its start).
constexpr uint32_t kWinNrCnt = 0, kWinFrCnt = 64, kWinFrMin = 128, kWinFrHot = 192;
constexpr uint32_t kWinRetCnt = 256, kWinRetMin = 257;
constexpr uint32_t kWinNr = 258;
// the memory phase's split (per SM) and packed slots share the near lists,
// which are empty from the end of a local phase to the next window start
constexpr uint32_t kWinDsc = kWinNr, kWinStage = kWinNr + kWinMaxSm;
constexpr uint32_t kWinRetL = kWinNr + 2u * 64u * kNear;
constexpr uint32_t kWinWKey = kWinRetL + 2u * kRetireLds;
constexpr uint32_t kWinWAux = kWinWKey + 2u * kWinCap;
constexpr uint32_t kWinWFin = kWinWAux + kWinCap;
// per-simulation counters: phase clocks (u64, words 0-9), windows, local
// steps, memory arrivals, retirements, largest memory batch (u32, 10-14)
constexpr uint32_t kWinStats = kWinWFin + kWinCap;
// dispatch state: next CTA, retired CTAs, current kernel, its first and end
// CTA, the kernel whose start cycle is known, that cycle, whether known
// (u32, words 0-7), CTA slots per SM of the current kernel (u64, words 8-9)
constexpr uint32_t kWinCtl = kWinStats + 16u;
// pointers the event loop needs rarely (u64 each): kept here rather than in
// scalar registers
constexpr uint32_t kWinPtrs = kWinCtl + 10u, kWinNumPtrs = 10u;
constexpr uint32_t kWinFixed = (kWinPtrs + 2u * kWinNumPtrs + 3u) & ~3u;  // the op table needs 16-B alignment
static_assert(kWinNr % 2 == 0 && kWinRetL % 2 == 0 && kWinWKey % 2 == 0 && kWinStats % 2 == 0 && kWinCtl % 2 == 0 &&
                  kWinPtrs % 2 == 0,
              "64-bit arrays on even words");
static_assert(2 * 64 * kNear >= kWinMaxSm + kWinCap, "near lists hold the memory phase's split");
constexpr uint32_t kWinPlain = 0, kWinTiles = 1, kWinTxn = 2;
struct WinLds {
  uint32_t optab, tops, srv, mq_head, mq_pos, fr, lru, t_idx, t_next, t_max, t_start;
  uint32_t total;
};
__host__ __device__ inline WinLds win_lds(uint32_t P, uint32_t NS, uint32_t SS, uint32_t QP, uint32_t NT,
                                          uint32_t mode) {
  WinLds L;
  uint32_t o = kWinFixed;
  auto take = [&o](uint32_t words, bool wide) {
    if (wide) o = (o + 1u) & ~1u;
    const uint32_t r = o;
    o += words;
    return r;
  };
  L.optab = take(4u * P, false);
  L.tops = take((NT + 1u) / 2u, false);
  L.srv = take(NS * SS, false);
  L.mq_head = take(NS, false);
  L.mq_pos = take(NS, false);
  L.fr = take(2u * 64u * QP, true);
  L.lru = take(mode != kWinPlain ? kWinCap : 0u, false);
  const bool txn = mode == kWinTxn;
  L.t_idx = take(txn ? kWinCap : 0u, false);
  L.t_next = take(txn ? kWinCap : 0u, false);
  L.t_max = take(txn ? kWinCap : 0u, false);
  L.t_start = take(txn ? kWinCap : 0u, false);
  L.total = o;
  return L;
}

}  // namespace gts
