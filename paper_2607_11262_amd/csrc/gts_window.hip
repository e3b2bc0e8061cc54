// gts_window.hip — windowed simulation kernel for gfx950 (MI355X).
//
// One wavefront simulates one (graph, hardware record) pair, with one lane
// per simulated SM (SM s on lane s mod 64, at most four SMs per lane).
// Instead of taking one event at a time, it advances the machine through
// time windows [T, H):
//
//   T = a lower bound of the earliest pending event;  H = T + min(Lm, 1024),
//       where Lm is the smallest possible delay from a memory arrival to its
//       completion (min over the graph's memory ops of L2/DRAM occupancy +
//       latency, over both servers for graphs whose tiles go through the LRU
//       L2; one cycle plus the smaller latency for transaction-level
//       memory);
//   retirement phase: every CTA retirement with cycle < H, in cycle order,
//       each distinct cycle followed by dispatch (wave-cooperative);
//   local phase: every lane issues its SMs' ready nodes with cycle < H in
//       (cycle, node id) order -- per-SM servers, finish, release of
//       out-edges (all inside the same CTA); memory nodes reserve the SM's
//       engine and queue an arrival at their engine start;
//   memory phase: the arrivals with cycle < H from all SMs are sorted by
//       (cycle, node id) (a bitonic network across the wave; a few keys by
//       counting ranks), sent to the L2 or DRAM by their op's flag or, for a
//       tile access on a machine with an LRU L2, by LRU decisions taken for
//       the whole batch in that order (tile kernels), served by the chip-wide
//       L2 and DRAM FIFO servers through a max-plus prefix scan, and
//       completed by the lane that owns their SM (CTA bookkeeping, release of
//       out-edges).
//
// The transaction-level kernels queue one ring entry per load / store that
// streams its 128-B lines through the engine; the memory phase takes the
// lines due in the window from those entries (each line an arrival, the
// servers keeping time in 2^-16 cycles, an LRU of lines), and a node
// completes with its last line.
//
// Why this equals the one-event-at-a-time order of the general kernel and of
// the CPU oracle: an arrival at s >= T completes no earlier than s + Lm >= H,
// so nothing the memory phase releases lands inside the window, and the
// window's arrivals are served in global (cycle, id) order; inside the window
// an SM's issue decisions depend only on its own servers and on releases
// from its own CTAs; a CTA completes only with a memory arrival (every node
// without a successor in its CTA is a global load or store -- checked on
// upload), so every retirement below H is already known when the window
// opens, and dispatch depends only on retirements and earlier dispatches.
// Edges between CTAs must leave a memory node and be released at its
// completion.  H may be lowered below T + Lm (more arrivals or retirements
// than the window buffers hold, arrivals not yet loaded); the rest waits for
// the next window, which starts at or before them.  The host sends other
// graphs, and simulations that overflow a queue, to the general kernel.
//
// Memory: ready nodes wait in a per-lane pool in LDS (spilling to scratch);
// memory arrivals in per-SM rings in scratch, with each ring's position and a
// lower bound of its head's cycle in LDS; pending retirements in LDS (spilling
// to scratch).  Uniform state used rarely (dispatch state, counters, the
// pointers of cold paths) lives in LDS too, not in scalar registers, which
// the hot paths need.  Per-node state (released in-edges, latest release) lives in
// scratch and counts up from zero: a CTA's nodes are zeroed when it is
// dispatched (nodes that receive cross-CTA edges once at start), and node
// records carry the first three successors with their in-degrees, so issuing
// a node costs one record load and one batch of successor-state loads; a
// lane handles one node of each of its SMs per round trip.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "../../include/gts.h"
#include "gts_common.h"
#include "gts_dev.h"

namespace gts {

namespace {

constexpr uint64_t kNoKey = ~0ull;
// far-list word: a due entry was pushed since the window start
constexpr uint32_t kFrPushedDue = 0x80000000u;
constexpr uint32_t kBadOverflow = 1u, kBadReady = 2u, kBadMemQ = 4u, kBadRetire = 8u;
// ring entries loaded per SM and window: as many as the registers allow
// at three waves per SIMD (fewer cut windows short)
template <uint32_t NB>
constexpr uint32_t kGq = NB >= 4 ? 4u : 5u;
constexpr uint32_t kMaxSubpart = GTS_MAX_SUBPART;
constexpr uint32_t kSmallBatch = 16;  // batches this small are ordered by counting ranks

// Node state: latest release cycle (low word) | released in-edges (high word).
__device__ __forceinline__ uint32_t* st_acc(uint64_t* st) { return reinterpret_cast<uint32_t*>(st); }
__device__ __forceinline__ uint32_t* st_cnt(uint64_t* st) { return reinterpret_cast<uint32_t*>(st) + 1; }

// A pointer into global memory (address space 1).
template <typename T>
using gmem = __attribute__((address_space(1))) T;

// Four consecutive words of global memory (one 16-B load).
__device__ __forceinline__ uint4 ld4(const gmem<const uint32_t>* p) { return make_uint4(p[0], p[1], p[2], p[3]); }

// Loads of words that global atomics may change bypass the L1.
template <typename T>
__device__ __forceinline__ T gld(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void mem_wait() { __builtin_amdgcn_s_waitcnt(0); }
__device__ __forceinline__ void wsync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Cross-lane steps by DPP (VALU lane shifts inside rows of 16 and row
// broadcasts) rather than LDS-crossbar shuffles: row_shr:n gives lane l the
// value of lane l - n of its row (lanes without one keep `old`); row_bcast:15
// / :31 give rows 1, 3 / rows 2, 3 lane 15 / lane 31 (other rows keep `old`).
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowBcast15 = 0x142, kRowBcast31 = 0x143;
template <int ctrl, int row_mask = 0xF>
__device__ __forceinline__ uint32_t dpp(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, ctrl, row_mask, 0xF, false);
}
__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

__device__ __forceinline__ uint32_t wave_incl_sum_u32(uint32_t x) {
  x += dpp<kRowShr1>(0u, x);
  x += dpp<kRowShr2>(0u, x);
  x += dpp<kRowShr4>(0u, x);
  x += dpp<kRowShr8>(0u, x);
  x += dpp<kRowBcast15, 0xA>(0u, x);
  x += dpp<kRowBcast31, 0xC>(0u, x);
  return x;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) { return lane_u32(wave_incl_sum_u32(x), 63); }
__device__ __forceinline__ uint32_t wave_excl_scan_u32(uint32_t x) { return wave_incl_sum_u32(x) - x; }

// Wave-wide min / max of a u64 (uniform result): row reductions by DPP, then
// the four row results.
template <bool kMax>
__device__ __forceinline__ uint64_t wave_ext_u64(uint64_t x) {
  uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
  const uint32_t id = kMax ? 0u : ~0u;
#define GTS_EXT_STEP(C)                                              \
  {                                                                  \
    const uint32_t plo = dpp<C>(id, lo), phi = dpp<C>(id, hi);       \
    const bool less = phi < hi || (phi == hi && plo < lo);           \
    if (kMax ? (!less && (phi != hi || plo != lo)) : less) {         \
      lo = plo;                                                      \
      hi = phi;                                                      \
    }                                                                \
  }
  GTS_EXT_STEP(kRowShr1)
  GTS_EXT_STEP(kRowShr2)
  GTS_EXT_STEP(kRowShr4)
  GTS_EXT_STEP(kRowShr8)
#undef GTS_EXT_STEP
  uint64_t r = kMax ? 0ull : ~0ull;
#pragma unroll
  for (int l = 15; l < 64; l += 16) {
    const uint64_t v = ((uint64_t)lane_u32(hi, l) << 32) | lane_u32(lo, l);
    r = kMax ? (v > r ? v : r) : (v < r ? v : r);
  }
  return r;
}
__device__ __forceinline__ uint64_t wmin64(uint64_t x) { return wave_ext_u64<false>(x); }
__device__ __forceinline__ uint64_t wmax64(uint64_t x) { return wave_ext_u64<true>(x); }

struct Compose {  // f(x) = max(x, a) + o on int64
  int64_t a, o;
};
constexpr int64_t kNegCycle = -(int64_t(1) << 62);  // below every cycle: max(x, kNegCycle) = x
__device__ __forceinline__ Compose compose(Compose f, Compose g) {  // g after f
  const int64_t ga = g.a - f.o;
  return Compose{f.a > ga ? f.a : ga, f.o + g.o};
}
template <int ctrl, int row_mask = 0xF>
__device__ __forceinline__ Compose dpp_c(Compose c) {  // lanes without a source get the identity
  const uint64_t a = (uint64_t)c.a, o = (uint64_t)c.o, na = (uint64_t)kNegCycle;
  const uint32_t alo = dpp<ctrl, row_mask>((uint32_t)na, (uint32_t)a);
  const uint32_t ahi = dpp<ctrl, row_mask>((uint32_t)(na >> 32), (uint32_t)(a >> 32));
  const uint32_t olo = dpp<ctrl, row_mask>(0u, (uint32_t)o);
  const uint32_t ohi = dpp<ctrl, row_mask>(0u, (uint32_t)(o >> 32));
  return Compose{(int64_t)(((uint64_t)ahi << 32) | alo), (int64_t)(((uint64_t)ohi << 32) | olo)};
}
// Inclusive scan of compositions across the wave (lane 0 first).
__device__ __forceinline__ Compose wave_incl_compose(Compose c) {
  c = compose(dpp_c<kRowShr1>(c), c);
  c = compose(dpp_c<kRowShr2>(c), c);
  c = compose(dpp_c<kRowShr4>(c), c);
  c = compose(dpp_c<kRowShr8>(c), c);
  c = compose(dpp_c<kRowBcast15, 0xA>(c), c);
  c = compose(dpp_c<kRowBcast31, 0xC>(c), c);
  return c;
}
__device__ __forceinline__ Compose lane_c(Compose c, int l) {
  const uint64_t a = (uint64_t)c.a, o = (uint64_t)c.o;
  return Compose{(int64_t)(((uint64_t)lane_u32((uint32_t)(a >> 32), l) << 32) | lane_u32((uint32_t)a, l)),
                 (int64_t)(((uint64_t)lane_u32((uint32_t)(o >> 32), l) << 32) | lane_u32((uint32_t)o, l))};
}

// A node record held in registers: a = {op | out-degree << 16, cta,
// succ_begin, succ0}, b = {succ1, succ2, indeg0 | indeg1 << 16, indeg2}.
struct Rec {
  uint4 a, b;
  __device__ __forceinline__ uint32_t op() const { return a.x & 0xFFFFu; }
  __device__ __forceinline__ uint32_t nsucc() const { return a.x >> 16; }
  __device__ __forceinline__ uint32_t cta() const { return a.y; }
  __device__ __forceinline__ uint32_t sb() const { return a.z; }
  __device__ __forceinline__ uint32_t succ(uint32_t k) const { return k == 0 ? a.w : k == 1 ? b.x : b.y; }
  __device__ __forceinline__ uint32_t sindeg(uint32_t k) const {
    return k == 0 ? (b.z & 0xFFFFu) : k == 1 ? (b.z >> 16) : (b.w & 0xFFFFu);
  }
};
__device__ __forceinline__ Rec load_rec(const NodeDev* nodes, uint32_t v) {
  const uint4* p = reinterpret_cast<const uint4*>(nodes + v);
  return Rec{p[0], p[1]};
}

// Does a node need the one-edge-at-a-time path (more than three successors,
// or an inline successor that is a shared node)?
__device__ __forceinline__ bool needs_slow(const Rec r) {
  const uint32_t n = r.nsucc();
  if (n > kInlineSucc) return true;
  bool sh = false;
#pragma unroll
  for (uint32_t k = 0; k < kInlineSucc; ++k) sh |= k < n && ((r.succ(k) >> GTS_EDGE_KIND_SHIFT) & kDevShared);
  return sh;
}

// Loaded ring entries whose key (cycle << 32 | kind << 30 | node) is below K.
template <uint32_t NB>
__device__ __forceinline__ uint32_t due_count(const uint32_t (&ehi)[NB][kGq<NB>], const uint32_t (&elo)[NB][kGq<NB>],
                                              uint64_t K) {
  uint32_t c = 0;
#pragma unroll
  for (uint32_t j = 0; j < NB; ++j)
#pragma unroll
    for (uint32_t q = 0; q < kGq<NB>; ++q) c += (((uint64_t)ehi[j][q] << 32) | elo[j][q]) < K;
  return c;
}

// One simulation on one wavefront; NB = SMs per lane (ceil(n_sm / 64) of the
// largest hardware record of the batch).
// The simulation's LDS (dynamic, so it starts at LDS address 0).
extern __shared__ uint32_t win_lds_words[];
__device__ __forceinline__ uint32_t* lds_base() { return win_lds_words; }

template <uint32_t NB, uint32_t MODE>
struct WSim {
  // LRU decisions in the memory phase (tiles, or the lines of transaction-
  // level memory); transaction-level memory
  static constexpr bool LRU = MODE != kWinPlain, TXN = MODE == kWinTxn;
  Image G;
  const uint32_t* hw;
  uint32_t b, lane, flags, nsm, nsub, sstride, smem_w, nslot, QF;
  bool nocont, ofin;
  bool mem_only;  // CTA bookkeeping on memory nodes only (compute nodes always feed a later memory node)
  bool sink_ret;  // the running kernel's CTAs retire with their sink: no CTA bookkeeping at all
  // LDS
  uint4* optab;
  uint16_t* tops;  // template class x slot -> op
  // mq_pos[s]: SM s's ring head (bits 0-7) and entry count (bits 8-15), and
  // its resident CTAs (bits 16-31)
  uint32_t *srv, *mq_head, *mq_pos, *dsc, *nr_cnt, *fr_cnt, *fr_min, *fr_hot;
  uint64_t *nr, *fr;
  uint32_t *ret_cnt, *ret_min;
  uint64_t* ret_l;
  uint64_t* w_key;
  uint32_t *w_aux, *w_fin, *stage;
  // scratch
  uint64_t* state;
  CtaState* cst;
  uint32_t* mq_g;
  uint32_t* out_cycles;
  // uniform control
  // dispatch state lives in LDS (kWinCtl): it is needed once per dispatch,
  // not in scalar registers across the event loop
  // the kernel whose CTAs are live (kernels run one after another) and its
  // template: nodes per CTA (0: expanded records), first node, first CTA, CTAs,
  // first template record, class x slot table offset and slots per class
  uint32_t run_k, t_n, t_node0, t_kc0, t_nc, t_base, t_ops, t_nslot;
  uint64_t l2_av, dram_av, Lm, Hnear;
  // LRU L2 (LRU only): each tile's latest access stamp (a count of tile
  // accesses, 0 = never; scratch), a Fenwick tree over stamps holding at each
  // tile's latest stamp its line count (scratch, entry 0 unused), one LDS
  // word per memory-batch position; the stamps handed out so far, the lines
  // of every tile touched so far, the L2's lines, the bound on stamps
  gmem<uint32_t>* lru_last;
  gmem<uint64_t>* lru_bit;
  uint32_t* lw;
  uint32_t lru_now, l2_lines, lru_acc;
  uint64_t lru_total;
  // transaction-level memory (TXN only): per batch slot the index of its
  // line in txn_line, the next transaction's entry cycle, and for the first
  // slot of a node the node's largest finish so far and its start (LDS); the
  // engine rate, the L2 / DRAM line occupancy in 2^-16 cycles, latencies
  uint32_t *t_idx, *t_next, *t_max, *t_start;
  uint32_t r_gmem, lat_l2, lat_dr;
  uint64_t q_l2, q_dr;
  // per lane
  uint64_t digest;
  uint32_t makespan, nfin, bad;
  uint32_t st_local, st_maxrq, st_maxmq, st_maxret;
  // uniform counters live in LDS (kWinStats), not in scalar registers: lane
  // 0 adds to them with fire-and-forget LDS atomics
  __device__ __forceinline__ void count(uint32_t word, uint32_t n) {
    if (lane == 0) atomicAdd(reinterpret_cast<uint32_t*>(lds_base()) + kWinStats + word, n);
  }
  __device__ __forceinline__ void count_max(uint32_t word, uint32_t n) {
    if (lane == 0) atomicMax(reinterpret_cast<uint32_t*>(lds_base()) + kWinStats + word, n);
  }
  __device__ __forceinline__ void count_retired(uint32_t n) {
    if (lane == 0) atomicAdd(lds_base() + kWinCtl + 1, n);
  }
  __device__ __forceinline__ void count_clk(uint32_t phase, uint64_t ticks) {
    if (lane == 0) atomicAdd(reinterpret_cast<unsigned long long*>(reinterpret_cast<uint32_t*>(lds_base()) + kWinStats) + phase,
                             (unsigned long long)ticks);
  }

  // ---- ready nodes of lane l's SMs, entries (cycle << 32 | SM slot << 30 |
  // node) with SM slot = SM / 64, in two lists: "near" holds only entries
  // below the current window end (kNear per lane, LDS), "far" the rest ([0,
  // QF) in LDS, [QF, QF + kPoolSpill) in scratch) with a lower bound of its
  // cycles in fr_min.  At each window start the far entries below the window
  // end move to near; those that do not fit (near is full) are put first, so
  // a far list is [due | later | pushed since the window start].  fr_hot
  // holds the end of the due part (bits 0-15), the start of the pushed part
  // (bits 16-30) and whether a due entry was pushed (bit 31); the local
  // phase scans the due part, and the pushed part once that bit is set.
  // rarely used pointers, from LDS (kWinPtrs)
  enum : uint32_t { kPSucc, kPIndeg, kPRoots, kPCtas, kPKernels, kPTsucc, kPTindeg, kPFrG, kPRetG, kPHw };
  // The pointers are global-memory ones: typed so, their accesses compile to
  // global instructions rather than flat ones (a flat access also counts
  // against the LDS wait counter, so every later LDS wait would wait for it).
  template <typename T>
  __device__ __forceinline__ gmem<T>* cold(uint32_t i) const {
    return (gmem<T>*)(uni64(reinterpret_cast<const uint64_t*>(lds_base() + kWinPtrs)[i]));
  }

  __device__ __forceinline__ uint64_t fr_get(uint32_t l, uint32_t i) const {
    return i < QF ? fr[i * 64u + l] : cold<uint64_t>(kPFrG)[(i - QF) * 64u + l];
  }
  __device__ __forceinline__ void fr_set(uint32_t l, uint32_t i, uint64_t k) {
    if (i < QF)
      fr[i * 64u + l] = k;
    else
      cold<uint64_t>(kPFrG)[(i - QF) * 64u + l] = k;
  }
  __device__ __forceinline__ uint32_t fr_n(uint32_t l) const {
    const uint32_t n = fr_cnt[l];
    return n < QF + kPoolSpill ? n : QF + kPoolSpill;
  }
  __device__ __forceinline__ void far_push(uint32_t l, uint64_t key) {
    const uint32_t slot = atomicAdd(&fr_cnt[l], 1u);
    st_maxrq = slot + 1 > st_maxrq ? slot + 1 : st_maxrq;
    if (slot < QF + kPoolSpill) {
      fr_set(l, slot, key);
      atomicMin(&fr_min[l], (uint32_t)(key >> 32));
    } else {
      bad |= kBadReady;
    }
  }
  // m (<= 8) entries of one cycle onto SM s's far list, their slots
  // reserved at once (as m single pushes would take them)
  __device__ __forceinline__ void far_push_n(uint32_t s, uint32_t cyc, const uint32_t (&v)[8], uint32_t m) {
    const uint32_t l = s & 63u;
    const uint32_t slot = atomicAdd(&fr_cnt[l], m);
    st_maxrq = slot + m > st_maxrq ? slot + m : st_maxrq;
#pragma unroll
    for (uint32_t u = 0; u < 8; ++u) {
      if (u >= m) continue;
      if (slot + u < QF + kPoolSpill)
        fr_set(l, slot + u, ((uint64_t)cyc << 32) | ((uint64_t)(s >> 6) << 30) | v[u]);
      else
        bad |= kBadReady;
    }
    atomicMin(&fr_min[l], cyc);
  }
  __device__ __forceinline__ void rq_push(uint32_t s, uint32_t cyc, uint32_t v) {
    const uint32_t l = s & 63u;
    const uint64_t key = ((uint64_t)cyc << 32) | ((uint64_t)(s >> 6) << 30) | v;
    if (cyc < Hnear) {
      const uint32_t slot = atomicAdd(&nr_cnt[l], 1u);
      if (slot < kNear) {
        nr[slot * 64u + l] = key;
        return;
      }
      atomicSub(&nr_cnt[l], 1u);
      atomicOr(&fr_hot[l], kFrPushedDue);
    }
    far_push(l, key);
  }

  // Up to kInlineSucc entries of one lane onto SM s's lists (want[k]): the
  // near slots are reserved with all atomics in flight, then filled; as for
  // one push at a time, the first free slots go to near entries and the rest
  // to far (hot).  The order within a list does not matter.
  __device__ __forceinline__ void rq_push_n(uint32_t s, const bool (&want)[kInlineSucc],
                                            const uint32_t (&cyc)[kInlineSucc], const uint32_t (&v)[kInlineSucc]) {
    const uint32_t l = s & 63u;
    uint32_t slot[kInlineSucc];
#pragma unroll
    for (uint32_t k = 0; k < kInlineSucc; ++k) slot[k] = want[k] && cyc[k] < Hnear ? atomicAdd(&nr_cnt[l], 1u) : kNear;
#pragma unroll
    for (uint32_t k = 0; k < kInlineSucc; ++k) {
      if (!want[k]) continue;
      const uint64_t key = ((uint64_t)cyc[k] << 32) | ((uint64_t)(s >> 6) << 30) | v[k];
      if (slot[k] < kNear) {
        nr[slot[k] * 64u + l] = key;
      } else {
        if (cyc[k] < Hnear) {
          atomicSub(&nr_cnt[l], 1u);
          atomicOr(&fr_hot[l], kFrPushedDue);
        }
        far_push(l, key);
      }
    }
  }

  // Smallest entry of each SM slot with its index (far indices carry bit 31).
  // Selects rather than branches: a branch per slot costs more exec-mask
  // bookkeeping than the compare it guards.
  __device__ __forceinline__ static void consider(uint64_t k, uint32_t i, uint64_t (&best)[NB], uint32_t (&bi)[NB]) {
    const uint32_t j = (uint32_t)(k >> 30) & 3u;
#pragma unroll
    for (uint32_t jj = 0; jj < NB; ++jj) {
      const bool t = (j == jj) & (k < best[jj]);
      best[jj] = t ? k : best[jj];
      bi[jj] = t ? i : bi[jj];
    }
  }
  // Far entries [b, e): the LDS part and the scratch part are read in loops
  // of their own, eight reads in flight, past the end clamped to the last
  // entry (a choice between the two per entry made every LDS read wait for
  // all outstanding global accesses).
  __device__ __forceinline__ void scan_far(uint32_t b, uint32_t e, uint64_t (&best)[NB], uint32_t (&bi)[NB]) const {
    const uint32_t el = e < QF ? e : QF;
    for (uint32_t i0 = b; i0 < el; i0 += 8) {
      uint64_t kk[8];
#pragma unroll
      for (uint32_t q = 0; q < 8; ++q) kk[q] = fr[(i0 + q < el ? i0 + q : el - 1u) * 64u + lane];
#pragma unroll
      for (uint32_t q = 0; q < 8; ++q)
        if (i0 + q < el) consider(kk[q], (i0 + q) | 0x80000000u, best, bi);
    }
    if (e > QF) {
      const gmem<uint64_t>* g = cold<uint64_t>(kPFrG);
      for (uint32_t i0 = b > QF ? b : QF; i0 < e; i0 += 8) {
        uint64_t kk[8];
#pragma unroll
        for (uint32_t q = 0; q < 8; ++q) kk[q] = g[((i0 + q < e ? i0 + q : e - 1u) - QF) * 64u + lane];
#pragma unroll
        for (uint32_t q = 0; q < 8; ++q)
          if (i0 + q < e) consider(kk[q], (i0 + q) | 0x80000000u, best, bi);
      }
    }
  }

  // Window start: move this lane's far entries below H to near, and put
  // those that do not fit first.
  __device__ __forceinline__ void pool_rebuild(uint64_t H) {
    if (fr_min[lane] < H) {
      const uint32_t n = fr_n(lane);
      uint32_t nn = nr_cnt[lane], kp = 0, h = 0, mn = 0xFFFFFFFFu;
      // in place, writes at or below the entry at hand (the kept entries
      // [0, h) due, [h, kp) later); the LDS part, then the scratch part, as
      // in scan_far (inside the LDS part every position written is in LDS)
      auto take = [&](auto in_lds, const uint64_t(&kk)[8], uint32_t i0, uint32_t m) {
        constexpr bool kLds = decltype(in_lds)::value;
        auto get = [&](uint32_t p) -> uint64_t {
          if constexpr (kLds) return fr[p * 64u + lane]; else return fr_get(lane, p);
        };
        auto set = [&](uint32_t p, uint64_t k) {
          if constexpr (kLds) fr[p * 64u + lane] = k; else fr_set(lane, p, k);
        };
#pragma unroll
        for (uint32_t q = 0; q < 8; ++q) {
          if (i0 + q < m) {
            const uint32_t i = i0 + q, cyc = (uint32_t)(kk[q] >> 32);
            if (cyc < H && nn < kNear) {
              nr[nn * 64u + lane] = kk[q];
              ++nn;
              continue;
            }
            if (cyc < H) {  // due: the first later entry moves to the end
              if (h != kp) set(kp, get(h));
              if (h != i) set(h, kk[q]);
              ++h;
            } else if (kp != i) {
              // an entry that keeps its place is not written back: most
              // windows move nothing, and rewriting unchanged entries
              // dirtied the far list's lines in the L2 on every window
              set(kp, kk[q]);
            }
            ++kp;
            mn = cyc < mn ? cyc : mn;
          }
        }
      };
      const uint32_t nl = n < QF ? n : QF;
      for (uint32_t i0 = 0; i0 < nl; i0 += 8) {
        uint64_t kk[8];
#pragma unroll
        for (uint32_t q = 0; q < 8; ++q) kk[q] = fr[(i0 + q < nl ? i0 + q : nl - 1u) * 64u + lane];
        take(std::true_type{}, kk, i0, nl);
      }
      if (n > QF) {
        const gmem<uint64_t>* g = cold<uint64_t>(kPFrG);
        for (uint32_t i0 = QF; i0 < n; i0 += 8) {
          uint64_t kk[8];
#pragma unroll
          for (uint32_t q = 0; q < 8; ++q) kk[q] = g[((i0 + q < n ? i0 + q : n - 1u) - QF) * 64u + lane];
          take(std::false_type{}, kk, i0, n);
        }
      }
      fr_cnt[lane] = kp;
      fr_min[lane] = mn;
      nr_cnt[lane] = nn;
      fr_hot[lane] = h | (kp << 16);
    } else {
      fr_hot[lane] = fr_n(lane) << 16;  // nothing due; pushes go after the present entries
    }
  }

  // ---- per-SM memory-arrival FIFO (strictly increasing cycles): a ring of
  // kRing entries {key lo, key hi, op} in scratch; LDS holds the position
  // (head | count << 8) and a lower bound of the head entry's cycle.  Owner
  // lane only.
  __device__ __forceinline__ void mq_push(uint32_t s, uint64_t key, uint32_t op) {
    const uint32_t pos = mq_pos[s];
    const uint32_t h = pos & 0xFFu, c = (pos >> 8) & 0xFFu;
    if (c >= kRing) {
      bad |= kBadMemQ;
      return;
    }
    uint32_t* e = mq_g + ((uint64_t)s * kRing + (h + c) % kRing) * 3u;
    e[0] = (uint32_t)key;
    e[1] = (uint32_t)(key >> 32);
    e[2] = op;
    if (c == 0) mq_head[s] = (uint32_t)(key >> 32);
    mq_pos[s] = (pos & 0xFFFF0000u) | h | ((c + 1) << 8);
    st_maxmq = c + 1 > st_maxmq ? c + 1 : st_maxmq;
  }

  // ---- transaction-level memory: a load / store streams its lines through
  // the SM's engine, line k entering at e_k = s + ceil(k L / r) (L = 128 B in
  // 2^-16 cycles, r the engine rate).  Its ring entry (kRingWordsTxn words):
  // {node | MISS << 31, entry cycle e of its next line, remainder rem, index
  // of that line in txn_line, lines left, largest finish so far, start s}
  // with e = s + c and rem = c r - k L for the next line k; from there line
  // k + i enters at e + ceil((i L - rem) / r), so the lines entering below a
  // cycle X number min(left, floor(((X - e - 1) r + rem) / L) + 1) for X > e.
  static constexpr uint32_t kLineShift = 23;  // L = 2^23
  static constexpr uint32_t kTxnMiss = 1u, kTxnLast = 2u, kTxnHead = 4u;  // slot flags (w_aux bits 0-7)
  __device__ __forceinline__ void mq_push_txn(uint32_t s, uint32_t v, uint32_t st, uint32_t idx, uint32_t n,
                                              uint32_t miss) {
    const uint32_t pos = mq_pos[s];
    const uint32_t h = pos & 0xFFu, c = (pos >> 8) & 0xFFu;
    if (c >= kRing) {
      bad |= kBadMemQ;
      return;
    }
    uint32_t* e = mq_g + ((uint64_t)s * kRing + (h + c) % kRing) * kRingWordsTxn;
    *reinterpret_cast<uint4*>(e) = make_uint4(v | (miss << 31), st, 0u, idx);
    *reinterpret_cast<uint4*>(e + 4) = make_uint4(n, 0u, st, 0u);
    if (c == 0) mq_head[s] = st;
    mq_pos[s] = (pos & 0xFFFF0000u) | h | ((c + 1) << 8);
    st_maxmq = c + 1 > st_maxmq ? c + 1 : st_maxmq;
  }
  // lines of an entry whose key (e << 32 | kEvMem << 30 | node) is below K
  __device__ __forceinline__ uint32_t txn_due(uint32_t w0, uint32_t e, uint32_t rem, uint32_t left,
                                              uint64_t K) const {
    const uint32_t low = (kEvMem << 30) | (w0 & GTS_EDGE_TARGET_MASK);
    const uint64_t X = (K >> 32) + (low < (uint32_t)K ? 1u : 0u);
    if (left == 0u || X <= e) return 0u;
    const uint64_t k = ((((X - e - 1u) * (uint64_t)r_gmem) + rem) >> kLineShift) + 1u;
    return k < left ? (uint32_t)k : left;
  }
  // the engine's end for the entry: the entry cycle after its last line
  __device__ __forceinline__ uint64_t txn_end(uint32_t e, uint32_t rem, uint32_t left) const {
    const uint64_t a = (uint64_t)left << kLineShift;
    return a > rem ? e + cdiv64(a - rem, r_gmem) : e;
  }
  // the next line's entry cycle and remainder
  __device__ __forceinline__ void txn_step(uint32_t& e, uint32_t& rem) const {
    constexpr uint32_t Lb = 1u << kLineShift;
    if (rem >= Lb) {
      rem -= Lb;
      return;
    }
    const uint64_t d = cdiv64(Lb - rem, r_gmem);
    e += (uint32_t)d;
    rem = (uint32_t)((uint64_t)rem + d * r_gmem - Lb);
  }

  // ---- pending CTA retirements, (cycle << 32 | SM) each, unordered: entries
  // [0, kRetireLds) in LDS, the rest in scratch; ret_min holds a lower bound
  // of their cycles (exact after each retirement phase).
  __device__ __forceinline__ uint64_t ret_get(uint32_t i) const {
    return i < kRetireLds ? ret_l[i] : cold<uint64_t>(kPRetG)[i - kRetireLds];
  }
  __device__ __forceinline__ void ret_set(uint32_t i, uint64_t k) {
    if (i < kRetireLds)
      ret_l[i] = k;
    else
      cold<uint64_t>(kPRetG)[i - kRetireLds] = k;
  }
  __device__ __forceinline__ void ret_push(uint32_t cyc, uint32_t sm) {
    const uint32_t slot = atomicAdd(ret_cnt, 1u);
    st_maxret = slot + 1 > st_maxret ? slot + 1 : st_maxret;
    if (slot < kRetireCap) {
      ret_set(slot, ((uint64_t)cyc << 32) | sm);
      atomicMin(ret_min, cyc);
    } else {
      bad |= kBadRetire;
    }
  }
  // pending retirements with cycle < X (this lane's share of [0, n))
  __device__ __forceinline__ uint32_t count_ret(uint64_t X, uint32_t n) const {
    uint32_t c = 0;
    for (uint32_t i = lane; i < n; i += 64) c += (ret_get(i) >> 32) < X;
    return c;
  }

  __device__ __forceinline__ void record(uint32_t v, uint64_t s, uint64_t f) {
    if (out_cycles) {
      uint64_t* o = reinterpret_cast<uint64_t*>(out_cycles) + ((uint64_t)b * G.n_nodes + v);
      *o = (f << 32) | s;
    }
    digest += mix64(((s << 32) | f) ^ mix64((uint64_t)v + 1));
    makespan = (uint32_t)f > makespan ? (uint32_t)f : makespan;
    ++nfin;
  }

  // Release along one edge into a shared node (atomics; the target may be in
  // another CTA on another SM).
  __device__ __forceinline__ void release_shared(uint32_t w, uint64_t r, uint32_t src_cta, uint32_t src_sm) {
    atomicMax(st_acc(&state[w]), (uint32_t)r);
    mem_wait();
    const uint32_t old = atomicAdd(st_cnt(&state[w]), 1u);
    if (old + 1u != (uint32_t)cold<const uint16_t>(kPIndeg)[w]) return;
    const uint32_t acc = gld(st_acc(&state[w]));
    const uint32_t cw = G.nodes[w].cta;
    if (cw == src_cta) {
      rq_push(src_sm, acc, w);
    } else if (cw < uni(lds_base()[kWinCtl])) {  // dispatched: ready at max(release, launch)
      const uint32_t launch = gld(&cst[cw].launch);
      rq_push(gld(&cst[cw].sm), acc > launch ? acc : launch, w);
    }
  }

  // Successors beyond the inline three, and inline ones into shared nodes,
  // one edge at a time.  which: 0 = edges released at issue, 1 = edges
  // released at completion, 2 = both.
  __device__ __forceinline__ void release_slow(const Rec rec, uint32_t which, uint64_t r_issue, uint64_t r_fin,
                                               uint32_t s) {
    const uint32_t n = rec.nsucc();
    for (uint32_t k = 0; k < n; ++k) {
      const uint32_t ent = k < kInlineSucc ? rec.succ(k) : succ_of(rec, k);
      const uint32_t bits = ent >> GTS_EDGE_KIND_SHIFT;
      if (k < kInlineSucc && !(bits & kDevShared)) continue;  // done by the batched path
      const bool at_issue = (bits & kDevOrder) && !ofin;
      if (which == 0 && !at_issue) continue;
      if (which == 1 && at_issue) continue;
      const uint32_t w = ent & GTS_EDGE_TARGET_MASK;
      const uint64_t r = at_issue ? r_issue : r_fin;
      if (bits & kDevShared) {
        release_shared(w, r, rec.cta(), s);
      } else {
        const uint32_t ind = indeg_of(rec, w);
        const uint64_t sv = ind != 1 ? state[w] : 0ull;
        const uint32_t cnt = (uint32_t)(sv >> 32) + 1u;
        uint32_t acc = (uint32_t)sv;
        acc = r > acc ? (uint32_t)r : acc;
        if (ind != 1 && cnt != ind) state[w] = ((uint64_t)cnt << 32) | acc;  // a readied node's state is not read again
        if (cnt == ind) rq_push(s, acc, w);
      }
    }
  }

  // ---- node records: expanded, or the running kernel's template with the
  // CTA derived from the node id, the op looked up by the CTA's class and
  // the successors moved from local to global ids
  __device__ __forceinline__ Rec rec_of(uint32_t v) const {
    if (t_n == 0) return load_rec(G.nodes, v);
    const uint32_t rel = v >= t_node0 ? v - t_node0 : 0u;  // idle lanes pass node 0
    uint32_t ci = rel / t_n;
    ci = ci < t_nc ? ci : t_nc - 1u;
    const uint32_t loc = rel - ci * t_n < t_n ? rel - ci * t_n : 0u;
    const uint32_t c = t_kc0 + ci;
    Rec r = load_rec(G.tnodes, t_base + loc);
    const uint32_t q = G.cclass[c];
    const uint32_t base = t_node0 + ci * t_n;
    r.a.x = (r.a.x & 0xFFFF0000u) | tops[t_ops + q * t_nslot + (r.a.x & 0xFFFFu)];
    r.a.y = c;
    r.a.w += base;
    r.b.x += base;
    r.b.y += base;
    return r;
  }
  // successor k of a record beyond the inline ones, and an unshared node's in-degree
  __device__ __forceinline__ uint32_t succ_of(const Rec& r, uint32_t k) const {
    if (t_n == 0) return cold<const uint32_t>(kPSucc)[r.sb() + k];
    return cold<const uint32_t>(kPTsucc)[r.sb() + k] + t_node0 + (r.cta() - t_kc0) * t_n;
  }
  __device__ __forceinline__ uint32_t indeg_of(const Rec& r, uint32_t w) const {
    if (t_n == 0) return cold<const uint16_t>(kPIndeg)[w];
    return cold<const uint16_t>(kPTindeg)[t_base + (w - t_node0 - (r.cta() - t_kc0) * t_n)];
  }
  __device__ __forceinline__ void load_template(uint32_t k) {
    const KernelDev kd = kernel_rec(k);
    run_k = k;
    t_n = uni(kd.t_n);
    t_node0 = uni(kd.node_begin);
    t_kc0 = uni(kd.cta_begin);
    t_nc = uni(kd.cta_end) - t_kc0;
    t_base = uni(kd.t_base);
    t_ops = uni(kd.t_ops & 0xFFFFu);
    t_nslot = uni(kd.t_ops >> 16);
    sink_ret = uni(kd.pad[0]) != 0;
  }

  // kernel k's record, read as words from global memory
  __device__ __forceinline__ KernelDev kernel_rec(uint32_t k) const {
    static_assert(sizeof(KernelDev) == 48, "three 16-B words");
    const gmem<const uint32_t>* p = (const gmem<const uint32_t>*)(cold<const KernelDev>(kPKernels) + k);
    KernelDev kd;
    uint4* d = reinterpret_cast<uint4*>(&kd);
    d[0] = ld4(p);
    d[1] = ld4(p + 4);
    d[2] = ld4(p + 8);
    return kd;
  }
  // first and end CTA and CTA slots per SM of kernel k
  __device__ __forceinline__ void load_kernel(uint32_t k, uint32_t& k_begin, uint32_t& k_end, uint64_t& slots) const {
    const KernelDev kd = kernel_rec(k);
    k_begin = uni(kd.cta_begin);
    k_end = uni(kd.cta_end);
    slots = uni64(kernel_slots(kd, (const uint32_t*)cold<const uint32_t>(kPHw)));
  }

  // ---- wave-cooperative dispatch at cycle t (after the retirements at t):
  // up to 64 CTAs at a time are placed on SMs (most free slots, lowest id),
  // then set up by one lane each.
  __device__ __forceinline__ void dispatch(uint32_t t) {
    uint32_t* const ctl = lds_base() + kWinCtl;
    uint32_t next_cta = uni(ctl[0]), cur_k = uni(ctl[2]), k_begin = uni(ctl[3]), k_end = uni(ctl[4]);
    uint32_t kstart_k = uni(ctl[5]), kstart_t = uni(ctl[6]), kstart_valid = uni(ctl[7]);
    uint64_t slots = uni64(*reinterpret_cast<const uint64_t*>(ctl + 8));
    const uint32_t retired = uni(ctl[1]);
    dispatch_loop(t, next_cta, retired, cur_k, k_begin, k_end, kstart_k, kstart_t, kstart_valid, slots);
    wsync();
    if (lane == 0) {
      ctl[0] = next_cta;
      ctl[2] = cur_k;
      ctl[3] = k_begin;
      ctl[4] = k_end;
      ctl[5] = kstart_k;
      ctl[6] = kstart_t;
      ctl[7] = kstart_valid;
      *reinterpret_cast<uint64_t*>(ctl + 8) = slots;
    }
    wsync();
  }
  __device__ __forceinline__ void dispatch_loop(uint32_t t, uint32_t& next_cta, uint32_t retired, uint32_t& cur_k,
                                                uint32_t& k_begin, uint32_t& k_end, uint32_t& kstart_k,
                                                uint32_t& kstart_t, uint32_t& kstart_valid, uint64_t& slots) {
    while (next_cta < G.n_ctas) {
      while (next_cta >= k_end) {
        ++cur_k;
        load_kernel(cur_k, k_begin, k_end, slots);
      }
      if (retired < k_begin) return;  // the previous kernel is still running
      // every CTA before next_cta is dispatched and `retired` of them have
      // retired, all of the running kernel: its free slots are known, and
      // the placement takes exactly that many (no search that finds none)
      const uint64_t cap = (uint64_t)nsm * slots, busy = next_cta - retired;
      const uint64_t room = cap > busy ? cap - busy : 0u;
      uint32_t lim = k_end - next_cta < 64u ? k_end - next_cta : 64u;
      lim = room < lim ? (uint32_t)room : lim;
      // the hardware record's launch latencies and the records of the CTAs
      // that may be placed (k <= lim of them), in flight during the placement
      const gmem<const uint32_t>* const hwc = cold<const uint32_t>(kPHw);
      const uint32_t cta_lat = hwc[HW_CTALAT], k_lat = hwc[HW_KLAT];
      const uint32_t c = next_cta + lane;
      uint4 c0 = make_uint4(0, 0, 0, 0), c1 = make_uint4(0, 0, 0, 0);
      if (lane < lim) {
        const gmem<const uint32_t>* p = (const gmem<const uint32_t>*)(cold<const CtaDev>(kPCtas) + c);
        c0 = ld4(p);      // node_begin, node_count, root_begin, root_count
        c1 = ld4(p + 4);  // memory nodes, first three roots
      }
      uint32_t k = 0, mysm = 0;
      while (k < lim) {
        uint64_t best = 0;
        for (uint32_t m = lane; m < nsm; m += 64) {
          const uint64_t fr = slots - (mq_pos[m] >> 16);
          const uint64_t key = (fr << 32) | (0xFFFFFFFFu - m);
          best = key > best ? key : best;
        }
        best = wmax64(best);
        if ((best >> 32) == 0) break;  // every SM is full
        const uint32_t sm = 0xFFFFFFFFu - (uint32_t)best;
        if (lane == k) mysm = sm;
        if (lane == (sm & 63u)) mq_pos[sm] += 1u << 16;
        wsync();
        ++k;
      }
      if (k == 0) return;
      if (run_k != cur_k) load_template(cur_k);  // the first CTAs of a kernel: it is now the running one
      if (!kstart_valid || kstart_k != cur_k) {
        kstart_valid = 1;
        kstart_k = cur_k;
        kstart_t = t;
      }
      const uint64_t launch = (uint64_t)t + cta_lat + (kstart_t == t ? k_lat : 0u);
      if (launch > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      if (lane < k && !sink_ret)  // a CTA that retires with its sink keeps no state
        *reinterpret_cast<uint4*>(&cst[c]) = make_uint4(mysm, (uint32_t)launch, mem_only ? c1.x : c0.y, 0u);
      // zero the node state of unshared CTAs (shared ones were zeroed at start)
      for (uint32_t j = 0; j < k; ++j) {
        const uint32_t nb = __shfl(c0.x, j, 64), nc = __shfl(c0.y, j, 64), rc = __shfl(c0.w, j, 64);
        if (!(rc & kCtaShared))
          for (uint32_t i = lane; i < nc; i += 64) state[nb + i] = 0ull;
      }
      if (lane < k && !(c0.w & kCtaShared) && launch >= Hnear) {
        // no in-edges at all: every root is ready at launch; up to eight
        // root ids read together, their far-list slots reserved at once
        const uint32_t nroots = c0.w;
        for (uint32_t r0 = 0; r0 < nroots; r0 += 8) {
          const uint32_t m = nroots - r0 < 8u ? nroots - r0 : 8u;
          uint32_t v[8];
#pragma unroll
          for (uint32_t u = 0; u < 8; ++u) {
            const uint32_t r = r0 + u;
            v[u] = r == 0 ? c1.y : r == 1 ? c1.z : r == 2 ? c1.w : u < m ? cold<const uint32_t>(kPRoots)[c0.z + r] : 0u;
          }
          far_push_n(mysm, (uint32_t)launch, v, m);
        }
      } else if (lane < k) {
        const bool shared = (c0.w & kCtaShared) != 0;
        const uint32_t nroots = c0.w & ~kCtaShared;
        for (uint32_t r = 0; r < nroots; ++r) {
          const uint32_t v = r == 0 ? c1.y : r == 1 ? c1.z : r == 2 ? c1.w : cold<const uint32_t>(kPRoots)[c0.z + r];
          if (!shared) {  // no in-edges at all
            rq_push(mysm, (uint32_t)launch, v);
          } else {
            const uint64_t sv = gld(&state[v]);
            if ((uint32_t)(sv >> 32) == (uint32_t)cold<const uint16_t>(kPIndeg)[v]) {
              const uint32_t acc = (uint32_t)sv;
              rq_push(mysm, acc > launch ? acc : (uint32_t)launch, v);
            }
          }
        }
      }
      next_cta += k;
      wsync();
    }
  }

  // ---- local phase step: each lane takes the smallest ready entry below H of
  // each of its SMs (at most one node per SM per step, so the nodes of one
  // step touch disjoint servers, CTAs and node states); the taken nodes are
  // packed into w_key / w_aux and issued W per lane.
  __device__ __forceinline__ bool local_step(uint64_t H) {
    uint32_t nn = nr_cnt[lane];
    nn = nn < kNear ? nn : kNear;
    const uint32_t fw = fr_hot[lane];
    uint32_t fh = fw & 0xFFFFu, fa = (fw >> 16) & 0x7FFFu;
    const bool pushed_due = (fw & kFrPushedDue) != 0, hot = fh != 0 || pushed_due;
    uint32_t fn = hot ? fr_n(lane) : 0u;
    uint64_t best[NB];
    uint32_t bi[NB];
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      best[j] = kNoKey;
      bi[j] = 0;
    }
    if (!bad) {
      for (uint32_t i0 = 0; i0 < nn; i0 += 4) {  // four LDS reads in flight
        uint64_t kk[4];
#pragma unroll
        for (uint32_t q = 0; q < 4; ++q) kk[q] = nr[(i0 + q < kNear ? i0 + q : kNear - 1) * 64u + lane];
#pragma unroll
        for (uint32_t q = 0; q < 4; ++q)
          if (i0 + q < nn) consider(kk[q], i0 + q, best, bi);
      }
      if (hot) {
        scan_far(0, fh, best, bi);
        if (pushed_due) scan_far(fa, fn, best, bi);
      }
    }
    uint32_t taken = 0, cnt = 0;
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const bool ok = best[j] != kNoKey && (best[j] >> 32) < H;
      taken |= ok ? 1u << j : 0u;
      cnt += ok;
    }
    const uint32_t incl = wave_incl_sum_u32(cnt);
    const uint32_t total = lane_u32(incl, 63);
    if (total == 0) return false;
    // at most kWinCap nodes per step (SMs do not interact inside a window, so
    // the others simply wait for the next step)
    const uint32_t E = total < kWinCap ? total : kWinCap;
    uint32_t p = incl - cnt;
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j)
      if ((taken >> j) & 1u) {
        if (p < kWinCap) {
          w_key[p] = best[j];
          w_aux[p] = lane + 64u * j;
          ++p;
        } else {
          taken &= ~(1u << j);
        }
      }
    // remove the taken entries, highest index first (far ones first)
#pragma unroll
    for (uint32_t rep = 0; rep < NB; ++rep) {
      uint32_t sel = NB, mx = 0;
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j) {
        const bool t = ((taken >> j) & 1u) & ((sel == NB) | (bi[j] > mx));
        sel = t ? j : sel;
        mx = t ? bi[j] : mx;
      }
      if (sel != NB) {
        taken &= ~(1u << sel);
        if (mx & 0x80000000u) {
          const uint32_t i = mx & 0x7FFFFFFFu;
          if (i >= fa) {  // pushed since the window start: the last entry fills its place
            if (i != fn - 1) fr_set(lane, i, fr_get(lane, fn - 1));
          } else {  // in the due part: the last due, later and pushed entries each move down one place
            const uint64_t v1 = fr_get(lane, fh - 1), v2 = fr_get(lane, fa - 1), v3 = fr_get(lane, fn - 1);
            if (i != fh - 1) fr_set(lane, i, v1);
            if (fh != fa) fr_set(lane, fh - 1, v2);
            if (fa != fn) fr_set(lane, fa - 1, v3);
            --fh;
            --fa;
          }
          --fn;
        } else {
          if (mx != nn - 1) nr[mx * 64u + lane] = nr[(nn - 1) * 64u + lane];
          --nn;
        }
      }
    }
    nr_cnt[lane] = nn;
    if (hot) {
      fr_cnt[lane] = fn;
      fr_hot[lane] = fh | (fa << 16) | (pushed_due ? kFrPushedDue : 0u);
    }
    wsync();
    if (E <= 64) {
      issue_events<1>(0, E);
    } else {
      issue_events<2>(0, E < 128u ? E : 128u);
      if (E > 128) issue_events<2>(128, E);
    }
    return true;
  }

  // Issue the packed nodes [i0, E) of w_key (cycle << 32 | slot << 30 |
  // node) / w_aux (SM), node i on lane (i - i0) mod 64: one record load and
  // one batch of state loads for all of them.
  template <uint32_t W>
  __device__ __forceinline__ void issue_events(uint32_t i0, uint32_t E) {
    uint32_t ev_t[W], ev_v[W], ev_s[W];
    bool ok[W];
    Rec rec[W];
    uint32_t tb[W], tn[W];  // TXN: the node's first line index and line count
#pragma unroll
    for (uint32_t w = 0; w < W; ++w) {
      const uint32_t i = i0 + w * 64u + lane;
      ok[w] = i < E;
      const uint64_t key = ok[w] ? w_key[i] : 0ull;
      ev_t[w] = (uint32_t)(key >> 32);
      ev_v[w] = (uint32_t)key & GTS_EDGE_TARGET_MASK;
      ev_s[w] = ok[w] ? w_aux[i] : 0u;
      rec[w] = rec_of(ev_v[w]);
      tb[w] = tn[w] = 0u;
      if constexpr (TXN) {
        if (ok[w]) {
          const gmem<const uint32_t>* tp = (const gmem<const uint32_t>*)G.txn_ptr;
          tb[w] = tp[ev_v[w]];
          tn[w] = tp[ev_v[w] + 1u] - tb[w];
        }
      }
    }
    // timing on the SM's servers: the node holds its class's subpartition
    // lanes (compute), the shared-memory pipe, or the global-memory engine
    // (memory nodes; L2 / DRAM follow in the memory phase), SYNC nothing;
    // every held server becomes free at start + occupancy.  One code path
    // for all classes, the server reads issued together.
    uint64_t rel_i[W], rel_f[W];
    bool is_mem[W];
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      is_mem[j] = false;
      rel_i[j] = rel_f[j] = 0;
      if (ok[j]) {
        const uint4 od = optab[rec[j].op()];
        const uint32_t cls = od.w & 7u;
        const bool comp = cls <= C_SFU;
        is_mem[j] = cls == C_GLOAD || cls == C_GSTORE;
        const uint32_t held = comp ? (od.w >> 8) & 0xFFu : (cls == C_SYNC ? 0u : 1u);
        uint32_t* Sv = srv + ev_s[j] * sstride + (comp ? (od.w >> 16) : smem_w + (is_mem[j] ? 1u : 0u));
        uint64_t st = ev_t[j];
        if (!nocont) {
          uint32_t busy = 0;
#pragma unroll
          for (uint32_t l = 0; l < kMaxSubpart; ++l)
            if (l < nsub) {
              const uint32_t a = Sv[comp ? l : 0u];
              busy = ((held >> l) & 1u) && a > busy ? a : busy;
            }
          st = busy > st ? busy : st;
        }
        // a load / store of transaction-level memory holds the engine while
        // its lines stream through
        const uint64_t occ = TXN && is_mem[j] ? (uint64_t)clamp_occ(cdiv64((uint64_t)tn[j] << kLineShift, r_gmem))
                                              : (uint64_t)od.x;
        const uint64_t f = st + occ + (is_mem[j] ? 0u : od.z);
        if (f > kMaxCycle) {
          bad |= kBadOverflow;
          ok[j] = false;
        } else {
          const uint32_t free_at = (uint32_t)(st + occ);
#pragma unroll
          for (uint32_t l = 0; l < kMaxSubpart; ++l)
            if (l < nsub && ((held >> l) & 1u)) Sv[comp ? l : 0u] = free_at;
          if (is_mem[j]) {
            if constexpr (TXN)
              mq_push_txn(ev_s[j], ev_v[j], (uint32_t)st, tb[j], tn[j], (od.w >> 3) & 1u);
            else
              mq_push(ev_s[j], mkkey(st, kEvMem, ev_v[j]), rec[j].op());
          }
          rel_i[j] = st + 1;
          rel_f[j] = f;
          if (!is_mem[j]) record(ev_v[j], st, f);
        }
      }
    }
    // successor states (inline, unshared) and CTA state, loads in flight together
    uint64_t sv[W][kInlineSucc];
    uint4 cs[W];
    bool sel[W][kInlineSucc];
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      const uint32_t nout = ok[j] ? rec[j].nsucc() : 0u;
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        sel[j][k] = false;
        sv[j][k] = 0;
        if (k < nout) {
          const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
          const bool at_issue = (bits & kDevOrder) && !ofin;
          sel[j][k] = !(bits & kDevShared) && (at_issue || !is_mem[j]);
          // a node with one in-edge needs no state: this release readies it
          if (sel[j][k] && rec[j].sindeg(k) != 1) sv[j][k] = state[rec[j].succ(k) & GTS_EDGE_TARGET_MASK];
        }
      }
      cs[j] = make_uint4(0, 0, 0, 0);
      if (ok[j] && !is_mem[j] && !mem_only && !sink_ret) cs[j] = *reinterpret_cast<const uint4*>(&cst[rec[j].cta()]);
    }
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      bool rdy[kInlineSucc];
      uint32_t racc[kInlineSucc], rw[kInlineSucc];
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
        const uint32_t w = rec[j].succ(k) & GTS_EDGE_TARGET_MASK;
        const uint64_t r = ((bits & kDevOrder) && !ofin) ? rel_i[j] : rel_f[j];
        const uint32_t cnt = (uint32_t)(sv[j][k] >> 32) + 1u;
        uint32_t acc = (uint32_t)sv[j][k];
        acc = r > acc ? (uint32_t)r : acc;
        // the release that readies a node is its last: its state is not read again
        if (sel[j][k] && rec[j].sindeg(k) != 1 && cnt != rec[j].sindeg(k)) state[w] = ((uint64_t)cnt << 32) | acc;
        rdy[k] = sel[j][k] && cnt == rec[j].sindeg(k);
        racc[k] = acc;
        rw[k] = w;
      }
      rq_push_n(ev_s[j], rdy, racc, rw);
      if (ok[j]) {
        if (!is_mem[j] && !mem_only && !sink_ret) {  // a compute node never completes its CTA
          const uint32_t mf = (uint32_t)rel_f[j] > cs[j].w ? (uint32_t)rel_f[j] : cs[j].w;
          *reinterpret_cast<uint2*>(&cst[rec[j].cta()].left) = make_uint2(cs[j].z - 1u, mf);
        }
        if (needs_slow(rec[j])) release_slow(rec[j], is_mem[j] ? 0u : 2u, rel_i[j], rel_f[j], ev_s[j]);
        ++st_local;
      }
    }
  }

  // ---- sort of w_key[0, M) (M <= 64 E) by (key, slot): position lane * E
  // + r gets the key and slot of the (lane * E + r)-th smallest (equal keys
  // in slot order; rank_sort also writes stage[i] = that slot).  A bitonic network
  // over 64 E positions, position lane * E + r in register r of the lane
  // (slots past M sort last); partners in other lanes come by cross-lane
  // shuffles, the rest are the lane's own registers.
  template <uint32_t E>
  __device__ __forceinline__ void sort_batch(uint32_t M, uint64_t (&k)[E], uint32_t (&sl)[E]) {
    static_assert(E == 1 || E == 2 || E == 4, "64, 128 or 256 positions");
    if (M <= kSmallBatch) {
      // few keys (one SM's arrivals, say): count each key's rank across the
      // lanes and pick, for each position, the key of that rank
      const uint64_t mine = lane < M ? w_key[lane] : kNoKey;
      uint32_t rank = 0;
      for (uint32_t j = 0; j < M; ++j) {
        const uint64_t kj = ((uint64_t)lane_u32((uint32_t)(mine >> 32), (int)j) << 32) | lane_u32((uint32_t)mine, (int)j);
        rank += (kj < mine || (kj == mine && j < lane)) ? 1u : 0u;
      }
#pragma unroll
      for (uint32_t r = 0; r < E; ++r) {
        k[r] = kNoKey;
        sl[r] = r * 64u + lane;
      }
      for (uint32_t j = 0; j < M; ++j) {
        const uint32_t rj = lane_u32(rank, (int)j);
        const uint64_t kj = ((uint64_t)lane_u32((uint32_t)(mine >> 32), (int)j) << 32) | lane_u32((uint32_t)mine, (int)j);
#pragma unroll
        for (uint32_t r = 0; r < E; ++r) {
          const bool t = rj == lane * E + r;
          k[r] = t ? kj : k[r];
          sl[r] = t ? j : sl[r];
        }
      }
      return;
    }
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      const uint32_t s = r * 64u + lane;
      k[r] = s < M ? w_key[s] : kNoKey;
      sl[r] = s;  // distinct, so every comparison is strict
    }
    bitonic<E>(k, sl);
  }
  // Bitonic network over the wave's 64 * E (key, tag) pairs, ordered by key,
  // then tag (distinct tags make every comparison strict): position
  // lane * E + r ends with the pair of that rank.
  template <uint32_t E, bool kTags = true>
  __device__ __forceinline__ void bitonic(uint64_t (&k)[E], uint32_t (&sl)[E]) const {
    constexpr uint32_t n = 64u * E;
#pragma unroll
    for (uint32_t kk = 2; kk <= n; kk <<= 1) {
#pragma unroll
      for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
        if (j >= E) {
#pragma unroll
          for (uint32_t r = 0; r < E; ++r) {
            const int lj = (int)(j / E);
            const uint64_t pk = ((uint64_t)(uint32_t)__shfl_xor((int)(uint32_t)(k[r] >> 32), lj, 64) << 32) |
                                (uint32_t)__shfl_xor((int)(uint32_t)k[r], lj, 64);
            const uint32_t ps = kTags ? (uint32_t)__shfl_xor((int)sl[r], lj, 64) : 0u;
            const uint32_t i = lane * E + r;
            const bool keep_min = ((i & j) == 0) == ((i & kk) == 0);
            const bool pless = pk < k[r] || (kTags && pk == k[r] && ps < sl[r]);
            const bool take = keep_min == pless;
            k[r] = take ? pk : k[r];
            if (kTags) sl[r] = take ? ps : sl[r];
          }
        } else {
#pragma unroll
          for (uint32_t r = 0; r < E; ++r) {
            if ((r & j) != 0) continue;  // r is the lower position of its pair
            const uint32_t q = r | j, i = lane * E + r;
            const bool up = (i & kk) == 0;
            const bool qless = k[q] < k[r] || (kTags && k[q] == k[r] && sl[q] < sl[r]);
            const bool sw = up == qless;
            const uint64_t tk = k[r];
            const uint32_t ts = sl[r];
            k[r] = sw ? k[q] : k[r];
            k[q] = sw ? tk : k[q];
            if (kTags) {
              sl[r] = sw ? sl[q] : sl[r];
              sl[q] = sw ? ts : sl[q];
            }
          }
        }
      }
    }
  }
  template <uint32_t E>
  __device__ __forceinline__ void rank_sort(uint32_t M) {
    uint64_t k[E];
    uint32_t sl[E];
    sort_batch<E>(M, k, sl);
    wsync();
#pragma unroll
    for (uint32_t r = 0; r < E; ++r)
      if (lane * E + r < M) stage[lane * E + r] = sl[r];
    wsync();
  }

  // ---- LRU L2 (tiles): a load / store that names a tile hits iff the tile
  // was touched before and its lines plus those of the distinct tiles touched
  // since fit the L2 (then the L2 server takes it, else DRAM); the tile
  // becomes the most recent.  Decided here for the whole memory batch, in its
  // (cycle, id) order, from the state before the batch and the batch itself.
  // For the arrival at sorted position i, of tile x with stamp q before the
  // batch, the distinct tiles touched since x's last access are
  //  * x also at earlier positions, the latest j: the tiles at positions
  //    (j, i), each counted at its first position after j;
  //  * else (q = 0: never touched, a miss): the tiles whose stamp before the
  //    batch follows q -- the tree's total minus its prefix sum to q -- and
  //    the tiles at positions before i (counted at their first position in
  //    the batch) whose stamp before it was at most q (the others are in the
  //    tree's part already).
  // The batch's tiles then move to stamps following every earlier one, in
  // position order: each tile's entry moves from its old stamp to the stamp
  // of its last position.  The positions' tiles sort by (tile, position) to
  // find each one's previous and next position of the same tile.  LDS per
  // position i: w_fin[i] = stamp before the batch, lw[i] = lines | (previous
  // position + 1) << 22 | (a later position follows) << 31.
  __device__ __forceinline__ uint64_t fen_prefix(uint32_t q) const {
    uint64_t s = 0;
    while (q) {  // up to eight tree nodes per round trip; entry 0 holds 0
      uint64_t v[8];
#pragma unroll
      for (uint32_t u = 0; u < 8; ++u) {
        v[u] = __hip_atomic_load(lru_bit + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        q &= q - 1u;
      }
#pragma unroll
      for (uint32_t u = 0; u < 8; ++u) s += v[u];
    }
    return s;
  }
  __device__ __forceinline__ void fen_add(uint32_t u, uint64_t d) const {
    for (; u != 0u && u <= lru_acc; u += u & (0u - u))
      __hip_atomic_fetch_add(lru_bit + u, d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // Tile accesses: tile and lines of each arrival, the decisions, and the
  // chosen server's occupancy and latency.
  template <uint32_t E>
  __device__ __forceinline__ void lru_batch(const uint64_t (&k)[E], const uint32_t (&p)[E], uint4 (&od)[E]) {
    const gmem<const uint32_t>* tile = (const gmem<const uint32_t>*)G.tile;
    const gmem<const OpDev>* ops = (const gmem<const OpDev>*)G.ops;
    uint32_t x[E], n[E], wk[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      x[r] = GTS_NO_TILE;
      wk[r] = 0;
      if (k[r] != kNoKey) {
        x[r] = tile[(uint32_t)k[r] & GTS_EDGE_TARGET_MASK];
        wk[r] = ops[w_aux[p[r]] & 0xFFFFu].work;
      }
    }
#pragma unroll
    for (uint32_t r = 0; r < E; ++r)
      n[r] = x[r] != GTS_NO_TILE ? (uint32_t)(((uint64_t)wk[r] + GTS_LINE_BYTES - 1) / GTS_LINE_BYTES) : 0u;
    bool hit[E];
    lru_core<E>(x, n, hit);
    const gmem<const uint32_t>* hw_w = cold<const uint32_t>(kPHw);
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      if (x[r] == GTS_NO_TILE) continue;
      const bool dram = !hit[r];
      od[r].y = clamp_occ(cdiv64((uint64_t)wk[r] * 65536ull, hw_w[HW_RATE + (dram ? R_DRAM : R_L2)]));
      od[r].z = hw_w[HW_LAT + (dram ? L_DRAM : L_L2)];
      od[r].w = (od[r].w & ~8u) | (dram ? 8u : 0u);
    }
  }
  // The decisions for keys x (GTS_NO_TILE: none) of n lines at batch
  // positions lane * E + r.
  template <uint32_t E>
  __device__ __forceinline__ void lru_core(const uint32_t (&x)[E], const uint32_t (&n)[E], bool (&hit)[E]) {
    constexpr uint32_t kLines = (1u << 22) - 1u, kLater = 1u << 31;
    uint32_t q[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) q[r] = x[r] != GTS_NO_TILE ? lru_last[x[r]] : 0u;
    uint64_t tk[E];
    uint32_t unused[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      const uint32_t i = lane * E + r;
      w_fin[i] = q[r];
      lw[i] = n[r];
      tk[r] = ((uint64_t)x[r] << 32) | i;  // distinct keys: no tags
    }
    bitonic<E, false>(tk, unused);
    wsync();
    // previous / next position of the same tile: the neighbours in (tile,
    // position) order (untracked positions sort last and are skipped)
    {
      const uint64_t before = __shfl_up(tk[E - 1], 1, 64), after = __shfl_down(tk[0], 1, 64);
#pragma unroll
      for (uint32_t r = 0; r < E; ++r) {
        const uint32_t xt = (uint32_t)(tk[r] >> 32);
        const uint64_t pk = r > 0 ? tk[r - 1] : before, nk = r + 1 < E ? tk[r + 1] : after;
        const bool has_prev = (lane > 0 || r > 0) && (uint32_t)(pk >> 32) == xt;
        const bool has_next = (lane < 63 || r + 1 < E) && (uint32_t)(nk >> 32) == xt;
        if (xt != GTS_NO_TILE)
          atomicOr(&lw[(uint32_t)tk[r]], (has_prev ? ((uint32_t)pk + 1u) << 22 : 0u) | (has_next ? kLater : 0u));
      }
    }
    wsync();
    uint64_t above[E];
    bool seen[E];
    uint32_t word[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      const uint32_t i = lane * E + r;
      word[r] = lw[i];
      const uint32_t j1 = (word[r] >> 22) & 511u;  // previous position + 1
      uint64_t a = 0;
      seen[r] = x[r] != GTS_NO_TILE && (j1 != 0u || q[r] != 0u);
      if (x[r] != GTS_NO_TILE && j1 != 0u) {
#pragma unroll 8
        for (uint32_t t = j1; t < i; ++t) {
          const uint32_t wt = lw[t];
          a += ((wt >> 22) & 511u) <= j1 ? (wt & kLines) : 0u;
        }
      } else if (x[r] != GTS_NO_TILE && q[r] != 0u) {
#pragma unroll 8
        for (uint32_t t = 0; t < i; ++t) {
          const uint32_t wt = lw[t];
          a += ((wt >> 22) & 511u) == 0u && w_fin[t] <= q[r] ? (wt & kLines) : 0u;
        }
      }
      above[r] = a;
    }
    mem_wait();  // the previous batch's tree updates are done
#pragma unroll
    for (uint32_t r = 0; r < E; ++r)
      if (x[r] != GTS_NO_TILE && ((word[r] >> 22) & 511u) == 0u && q[r] != 0u)
        above[r] += lru_total - fen_prefix(q[r]);
    // stamps in position order; a tile's last position moves its tree entry
    uint32_t c = 0;
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) c += x[r] != GTS_NO_TILE ? 1u : 0u;
    const uint32_t incl = wave_incl_sum_u32(c);
    uint32_t st = lru_now + incl - c;
    uint32_t fresh = 0;
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      hit[r] = false;
      if (x[r] == GTS_NO_TILE) continue;
      ++st;
      if (!(word[r] & kLater)) {
        if (q[r] != 0u)
          fen_add(q[r], (uint64_t)0 - n[r]);
        else
          fresh += n[r];
        fen_add(st, n[r]);
        lru_last[x[r]] = st;
      }
      hit[r] = seen[r] && above[r] + n[r] <= (uint64_t)l2_lines;
    }
    lru_now += lane_u32(incl, 63);
    lru_total += wave_sum_u32(fresh);
    wsync();
  }

  // ---- transaction-level memory: the window's due lines.  Up to two ring
  // entries of each SM whose head may be below H0 are loaded; the entries
  // after them start no earlier than the last loaded one's engine end, so K
  // stays at or below the smallest key any of them can have.  At most `cap`
  // lines are due (the largest cycle boundary that keeps them, or a key
  // boundary inside cycle T: one node's lines of one cycle share a key, and
  // the host keeps them within the cap).  The due lines fill slots SM by SM,
  // each SM's in ring order, an entry's lines consecutive: w_key = entry
  // cycle << 32 | kEvMem << 30 | node, w_aux = SM << 16 | ring position << 8
  // | flags, t_idx = line index, t_next = the next line's entry cycle (after
  // the last line, the engine's end); an entry's first slot also carries its
  // largest finish so far and its start.  Entries keep their progress in the
  // ring, and the head moves past the front entries with no line left.  (An
  // entry's lines can be due while an earlier one still has lines: the last
  // line of a node and the first of the next can enter in one cycle, and the
  // order between them is by node.)
  __device__ __forceinline__ uint32_t txn_select(uint64_t T, uint64_t H0, uint32_t cap) {
    constexpr uint32_t GQ = 2;
    uint32_t ew[NB][GQ], ee[NB][GQ], er[NB][GQ], ei[NB][GQ], el[NB][GQ], em[NB][GQ], es[NB][GQ];
    uint32_t cnt[NB], hd[NB];
    bool ld[NB];
    uint64_t Kl = H0 << 32;
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const uint32_t s = lane + 64u * j;
      const bool valid = j < nslot && s < nsm;
      const uint32_t pos = valid ? mq_pos[s] : 0u;
      hd[j] = pos & 0xFFu;
      cnt[j] = (pos >> 8) & 0xFFu;
      ld[j] = valid && cnt[j] > 0 && mq_head[s] < H0;
#pragma unroll
      for (uint32_t q = 0; q < GQ; ++q) {
        ew[j][q] = ee[j][q] = er[j][q] = ei[j][q] = el[j][q] = em[j][q] = es[j][q] = 0u;
        if (ld[j] && q < cnt[j]) {
          const gmem<const uint32_t>* e =
              (const gmem<const uint32_t>*)(mq_g + ((uint64_t)s * kRing + (hd[j] + q) % kRing) * kRingWordsTxn);
          const uint4 a = ld4(e), c = ld4(e + 4);
          ew[j][q] = a.x;
          ee[j][q] = a.y;
          er[j][q] = a.z;
          ei[j][q] = a.w;
          el[j][q] = c.x;
          em[j][q] = c.y;
          es[j][q] = c.z;
        }
      }
      if (ld[j] && cnt[j] > GQ) {
        const uint64_t x = (txn_end(ee[j][GQ - 1], er[j][GQ - 1], el[j][GQ - 1]) << 32) | ((uint64_t)kEvMem << 30);
        Kl = x < Kl ? x : Kl;
      }
    }
    auto due = [&](uint64_t K) -> uint32_t {
      uint32_t c = 0;
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j)
#pragma unroll
        for (uint32_t q = 0; q < GQ; ++q)
          if (ld[j] && q < cnt[j]) c += txn_due(ew[j][q], ee[j][q], er[j][q], el[j][q], K);
      return c;
    };
    uint64_t K = wmin64(Kl);
    uint32_t M = wave_sum_u32(due(K));
    if (M > cap) {
      const uint64_t Kmax = K;  // due(Kmax) > cap
      uint64_t lo = T, hi = Kmax >> 32;  // cycles; due(T << 32) = 0
      if (wave_sum_u32(due(hi << 32)) <= cap) {
        lo = hi;
      } else {
        while (hi - lo > 1) {
          const uint64_t mid = lo + (hi - lo) / 2;
          if (wave_sum_u32(due(mid << 32)) <= cap)
            lo = mid;
          else
            hi = mid;
        }
      }
      K = lo << 32;
      if (lo == T) {
        uint64_t klo = T << 32, khi = (T + 1) << 32;
        khi = Kmax < khi ? Kmax : khi;
        while (khi - klo > 1) {
          const uint64_t mid = klo + (khi - klo) / 2;
          if (wave_sum_u32(due(mid)) <= cap)
            klo = mid;
          else
            khi = mid;
        }
        K = klo;
      }
      M = wave_sum_u32(due(K));
    }
    uint32_t p = wave_excl_scan_u32(due(K));
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const uint32_t s = lane + 64u * j;
      if (!(j < nslot && s < nsm)) continue;
      uint32_t d = 0, gone = 0;
      bool front = true;
      uint64_t nh = kNoKey;  // lower bound of the next line's entry cycle among the entries that stay
#pragma unroll
      for (uint32_t q = 0; q < GQ; ++q) {
        if (!(ld[j] && q < cnt[j])) continue;
        const uint32_t c = txn_due(ew[j][q], ee[j][q], er[j][q], el[j][q], K);
        const uint32_t rp = (hd[j] + q) % kRing;
        const uint32_t v = ew[j][q] & GTS_EDGE_TARGET_MASK;
        const uint32_t fl = (ew[j][q] >> 31) ? kTxnMiss : 0u;
        uint32_t e = ee[j][q], rem = er[j][q];
        for (uint32_t k = 0; k < c; ++k) {
          const uint32_t slot = p + d + k;
          w_key[slot] = ((uint64_t)e << 32) | ((uint64_t)kEvMem << 30) | v;
          txn_step(e, rem);
          t_next[slot] = e;
          t_idx[slot] = ei[j][q] + k;
          w_aux[slot] = (s << 16) | (rp << 8) | fl | (k + 1u == el[j][q] ? kTxnLast : 0u) | (k == 0u ? kTxnHead : 0u);
          if (k == 0u) {
            t_max[slot] = em[j][q];
            t_start[slot] = es[j][q];
          }
        }
        d += c;
        const uint32_t left = el[j][q] - c;
        if (c) {  // progress stays in the ring (the largest finish is written after the batch)
          gmem<uint32_t>* g = (gmem<uint32_t>*)(mq_g + ((uint64_t)s * kRing + rp) * kRingWordsTxn);
          g[1] = e;
          g[2] = rem;
          g[3] = ei[j][q] + c;
          g[4] = left;
        }
        if (front && left == 0u)
          ++gone;
        else
          front = false;
        if (left) nh = e < nh ? e : nh;
      }
      dsc[s] = p | (d << 16);
      p += d;
      if (ld[j]) {
        const uint32_t rest = cnt[j] - gone;
        mq_pos[s] = (mq_pos[s] & 0xFFFF0000u) | ((hd[j] + gone) % kRing) | (rest << 8);
        if (rest) {
          if (cnt[j] > GQ) {
            const uint64_t x = txn_end(ee[j][GQ - 1], er[j][GQ - 1], el[j][GQ - 1]);
            nh = x < nh ? x : nh;
          }
          mq_head[s] = (uint32_t)nh;
        }
      }
    }
    return M;
  }

  // Memory phase of transaction-level memory: each due line, in (cycle,
  // node, line) order, hits iff it is among the L2's most recent lines (an
  // LRU of lines; without a capacity the op's MISS flag decides) and is
  // served FIFO by the L2 or DRAM server, which keeps time in 2^-16 cycles
  // and holds a line for q of them: m = max(e << 16, avail), avail = m + q,
  // finish = max(next entry cycle, ceil((m + q) / 2^16)) + latency.
  template <uint32_t E>
  __device__ __forceinline__ void memory_phase_txn(uint32_t M) {
    uint64_t k[E];
    uint32_t p[E];
    sort_batch<E>(M, k, p);
    const gmem<const uint32_t>* tl = (const gmem<const uint32_t>*)G.txn_line;
    uint32_t x[E], one[E], nxt[E];
    bool dram[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      x[r] = GTS_NO_TILE;
      one[r] = nxt[r] = 0u;
      dram[r] = false;
      if (k[r] != kNoKey) {
        dram[r] = (w_aux[p[r]] & kTxnMiss) != 0u;
        nxt[r] = t_next[p[r]];
        if (l2_lines) {
          x[r] = tl[t_idx[p[r]]];
          one[r] = 1u;
        }
      }
    }
    if (l2_lines) {
      bool hit[E];
      lru_core<E>(x, one, hit);
#pragma unroll
      for (uint32_t r = 0; r < E; ++r)
        if (x[r] != GTS_NO_TILE) dram[r] = !hit[r];
    }
    Compose fl2{kNegCycle, 0}, fdr{kNegCycle, 0};
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      if (k[r] != kNoKey) {
        const Compose g{(int64_t)((k[r] >> 32) << 16), (int64_t)(dram[r] ? q_dr : q_l2)};
        if (dram[r])
          fdr = compose(fdr, g);
        else
          fl2 = compose(fl2, g);
      }
    }
    const Compose il2 = wave_incl_compose(fl2), idr = wave_incl_compose(fdr);
    Compose el2 = Compose{__shfl_up(il2.a, 1, 64), __shfl_up(il2.o, 1, 64)};
    Compose edr = Compose{__shfl_up(idr.a, 1, 64), __shfl_up(idr.o, 1, 64)};
    if (lane == 0) el2 = edr = Compose{kNegCycle, 0};
    const Compose tl2 = lane_c(il2, 63), tdr = lane_c(idr, 63);
    int64_t xl2 = ((int64_t)l2_av > el2.a ? (int64_t)l2_av : el2.a) + el2.o;
    int64_t xdr = ((int64_t)dram_av > edr.a ? (int64_t)dram_av : edr.a) + edr.o;
    if (!nocont) {
      l2_av = (uint64_t)(((int64_t)l2_av > tl2.a ? (int64_t)l2_av : tl2.a) + tl2.o);
      dram_av = (uint64_t)(((int64_t)dram_av > tdr.a ? (int64_t)dram_av : tdr.a) + tdr.o);
    }
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      if (k[r] != kNoKey) {
        const int64_t st = (int64_t)((k[r] >> 32) << 16);
        const int64_t q = (int64_t)(dram[r] ? q_dr : q_l2);
        const int64_t xs = dram[r] ? xdr : xl2;
        const int64_t m = nocont ? st : (xs > st ? xs : st);
        if (dram[r])
          xdr = m + q;
        else
          xl2 = m + q;
        const uint64_t done = ((uint64_t)(m + q) + 65535u) >> 16;
        const uint64_t f = (nxt[r] > done ? (uint64_t)nxt[r] : done) + (dram[r] ? lat_dr : lat_l2);
        if (f > kMaxCycle) bad |= kBadOverflow;
        w_fin[p[r]] = f > kMaxCycle ? 0xFFFFFFFFu : (uint32_t)f;
      }
    }
    wsync();
    if (__ballot(bad != 0)) return;
    txn_fold();
    complete_arrivals();
  }

  // Each SM's lines of the batch, in ring order (an entry's lines are
  // consecutive slots, led by its first): the node's largest finish folds
  // over them; a node whose last line is here completes (the slot then
  // holds the node's finish and, in t_next, its start); an entry with lines
  // left keeps its largest finish in the ring.  The completing slots are
  // listed from each SM's first slot on (lw), for the completion rounds.
  __device__ __forceinline__ void txn_fold() {
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const uint32_t s = lane + 64u * j;
      if (!(j < nslot && s < nsm)) continue;
      const uint32_t sp = dsc[s], first = sp & 0xFFFFu, d = sp >> 16;
      uint32_t m = 0, st = 0, c = 0;
      for (uint32_t i = first; i < first + d; ++i) {
        const uint32_t a = w_aux[i];
        if (a & kTxnHead) {
          m = t_max[i];
          st = t_start[i];
        }
        const uint32_t f = w_fin[i];
        m = f > m ? f : m;
        if (a & kTxnLast) {
          w_fin[i] = m;
          t_next[i] = st;
          lw[first + c] = i;
          ++c;
        } else if (i + 1u == first + d || (w_aux[i + 1u] & kTxnHead)) {
          gmem<uint32_t>* g = (gmem<uint32_t>*)(mq_g + ((uint64_t)s * kRing + ((a >> 8) & 0xFFu)) * kRingWordsTxn);
          g[5] = m;
        }
      }
      dsc[s] = first | (c << 16);
    }
    wsync();
  }

  // ---- memory phase, E arrivals per lane: sort w_key[0, M) by (cycle, id),
  // serve them in that order, then complete them on their SMs' lanes.
  template <uint32_t E>
  __device__ __forceinline__ void memory_phase(uint32_t M) {
    // arrival lane * E + r in (cycle, id) order: key k[r], slot p[r]
    // (positions past M hold kNoKey)
    uint64_t k[E];
    uint32_t p[E];
    sort_batch<E>(M, k, p);
    uint4 od[E];
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) od[r] = k[r] != kNoKey ? optab[w_aux[p[r]] & 0xFFFFu] : make_uint4(0, 0, 0, 0);
    if constexpr (LRU) {
      if (l2_lines) lru_batch<E>(k, p, od);
    }
    Compose fl2{kNegCycle, 0}, fdr{kNegCycle, 0};
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      if (k[r] != kNoKey) {
        const Compose g{(int64_t)(k[r] >> 32), (int64_t)od[r].y};
        if ((od[r].w >> 3) & 1u)
          fdr = compose(fdr, g);
        else
          fl2 = compose(fl2, g);
      }
    }
    const Compose il2 = wave_incl_compose(fl2), idr = wave_incl_compose(fdr);
    Compose el2 = Compose{__shfl_up(il2.a, 1, 64), __shfl_up(il2.o, 1, 64)};
    Compose edr = Compose{__shfl_up(idr.a, 1, 64), __shfl_up(idr.o, 1, 64)};
    if (lane == 0) el2 = edr = Compose{kNegCycle, 0};
    const Compose tl2 = lane_c(il2, 63), tdr = lane_c(idr, 63);
    int64_t xl2 = ((int64_t)l2_av > el2.a ? (int64_t)l2_av : el2.a) + el2.o;
    int64_t xdr = ((int64_t)dram_av > edr.a ? (int64_t)dram_av : edr.a) + edr.o;
    if (!nocont) {
      l2_av = (uint64_t)(((int64_t)l2_av > tl2.a ? (int64_t)l2_av : tl2.a) + tl2.o);
      dram_av = (uint64_t)(((int64_t)dram_av > tdr.a ? (int64_t)dram_av : tdr.a) + tdr.o);
    }
#pragma unroll
    for (uint32_t r = 0; r < E; ++r) {
      if (k[r] != kNoKey) {
        const int64_t st = (int64_t)(k[r] >> 32);
        const bool dram = (od[r].w >> 3) & 1u;
        const int64_t x = dram ? xdr : xl2;
        const int64_t m = nocont ? st : (x > st ? x : st);
        if (dram)
          xdr = m + (int64_t)od[r].y;
        else
          xl2 = m + (int64_t)od[r].y;
        const int64_t e = st + (int64_t)od[r].x;
        const int64_t mend = m + (int64_t)od[r].y;
        const uint64_t f = (uint64_t)(e > mend ? e : mend) + od[r].z;
        if (f > kMaxCycle) bad |= kBadOverflow;
        w_fin[p[r]] = f > kMaxCycle ? 0xFFFFFFFFu : (uint32_t)f;
      }
    }
    wsync();
    if (__ballot(bad != 0)) return;
    complete_arrivals();
  }

  // Completion of the window's arrivals in rounds: round r takes the r-th
  // arrival of every SM (arrivals of different SMs touch different CTAs and
  // nodes; shared nodes use atomics), packs their slots into stage[] and
  // completes them W per lane.
  __device__ __forceinline__ void complete_arrivals() {
    // each SM's split (first slot | count << 16), read once: completions
    // push only to far lists, so the near lists it shares stay untouched
    uint32_t sp[NB];
    uint32_t rounds = 0;
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const uint32_t s = lane + 64u * j;
      sp[j] = j < nslot && s < nsm ? dsc[s] : 0u;
      rounds = (sp[j] >> 16) > rounds ? (sp[j] >> 16) : rounds;
    }
    rounds = (uint32_t)wmax64(rounds);
    for (uint32_t r = 0; r < rounds; ++r) {
      uint32_t cnt = 0;
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j) cnt += r < (sp[j] >> 16);
      const uint32_t incl = wave_incl_sum_u32(cnt);
      const uint32_t E = lane_u32(incl, 63);
      uint32_t p = incl - cnt;
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j)
        if (r < (sp[j] >> 16)) stage[p++] = TXN ? lw[(sp[j] & 0xFFFFu) + r] : (sp[j] & 0xFFFFu) + r;
      wsync();
      if (E <= 64) {
        complete_events<1>(0, E);
      } else {
        complete_events<2>(0, E < 128u ? E : 128u);
        if (E > 128) complete_events<2>(128, E);
      }
      wsync();
    }
  }

  // Complete the packed arrivals stage[i0, E) (slots of w_key / w_aux /
  // w_fin), arrival i on lane (i - i0) mod 64.
  template <uint32_t W>
  __device__ __forceinline__ void complete_events(uint32_t i0, uint32_t E) {
    Rec rec[W];
    uint32_t vv[W], ss[W], ff[W], tt[W];
    bool ok[W];
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      const uint32_t i = i0 + j * 64u + lane;
      ok[j] = i < E;
      const uint32_t slot = ok[j] ? stage[i] : 0u;
      const uint64_t key = ok[j] ? w_key[slot] : 0ull;
      vv[j] = (uint32_t)key & GTS_EDGE_TARGET_MASK;
      tt[j] = TXN ? (ok[j] ? t_next[slot] : 0u) : (uint32_t)(key >> 32);  // the node's start
      ff[j] = ok[j] ? w_fin[slot] : 0u;
      ss[j] = ok[j] ? w_aux[slot] >> 16 : 0u;
      rec[j] = rec_of(vv[j]);
    }
    uint64_t sv[W][kInlineSucc];
    bool sel[W][kInlineSucc];
    uint4 cs[W];
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      const uint32_t nout = ok[j] ? rec[j].nsucc() : 0u;
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        sel[j][k] = false;
        sv[j][k] = 0;
        if (k < nout) {
          const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
          const bool at_issue = (bits & kDevOrder) && !ofin;
          sel[j][k] = !(bits & kDevShared) && !at_issue;
          if (sel[j][k] && rec[j].sindeg(k) != 1) sv[j][k] = state[rec[j].succ(k) & GTS_EDGE_TARGET_MASK];
        }
      }
      cs[j] = make_uint4(0, 0, 0, 0);
      if (ok[j] && !sink_ret) cs[j] = *reinterpret_cast<const uint4*>(&cst[rec[j].cta()]);
    }
#pragma unroll
    for (uint32_t j = 0; j < W; ++j) {
      const uint32_t f = ff[j];
      bool rdy[kInlineSucc];
      uint32_t racc[kInlineSucc], rw[kInlineSucc];
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        const uint32_t w = rec[j].succ(k) & GTS_EDGE_TARGET_MASK;
        const uint32_t cnt = (uint32_t)(sv[j][k] >> 32) + 1u;
        uint32_t acc = (uint32_t)sv[j][k];
        acc = f > acc ? f : acc;
        // the release that readies a node is its last: its state is not read again
        if (sel[j][k] && rec[j].sindeg(k) != 1 && cnt != rec[j].sindeg(k)) state[w] = ((uint64_t)cnt << 32) | acc;
        rdy[k] = sel[j][k] && cnt == rec[j].sindeg(k);
        racc[k] = acc;
        rw[k] = w;
      }
      rq_push_n(ss[j], rdy, racc, rw);
      if (ok[j]) {
        record(vv[j], tt[j], f);
        if (sink_ret) {
          if ((rec[j].b.w >> 16) & kRecSink) ret_push(f, ss[j]);  // the sink finishes last
        } else {
          const uint32_t left = cs[j].z - 1u;
          const uint32_t mf = f > cs[j].w ? f : cs[j].w;
          *reinterpret_cast<uint2*>(&cst[rec[j].cta()].left) = make_uint2(left, mf);
          if (left == 0) ret_push(mf, ss[j]);  // the CTA retires at its largest finish
        }
        if (needs_slow(rec[j])) release_slow(rec[j], 1u, 0, f, ss[j]);
      }
    }
  }

};


template <uint32_t NB, uint32_t MODE>
__device__ __forceinline__ void window_body(const Launch& L) {
  constexpr bool LRU = MODE != kWinPlain, TXN = MODE == kWinTxn;
  const uint32_t b = blockIdx.x;
  if (b >= L.B) return;
  uint32_t* const lds = lds_base();
  WSim<NB, MODE> S;
  S.G = L.img;
  S.hw = L.hw + (uint64_t)b * HW_WORDS;
  S.b = b;
  S.lane = threadIdx.x;
  S.flags = L.flags;
  S.nocont = (L.flags & GTS_NO_CONTENTION) != 0;
  S.ofin = (L.flags & GTS_ORDER_AT_FINISH) != 0;
  S.mem_only = (L.img.props & kGraphComputeFeedsData) != 0;
  S.nsm = S.hw[HW_NSM];
  S.nsub = L.srv_one ? 1u : S.hw[HW_NSUB];  // server words per compute class (one when the lanes move together)
  S.sstride = server_stride(S.G.props, S.nsub);
  S.smem_w = S.sstride - 2;
  S.nslot = (S.nsm + 63) / 64;
  S.QF = L.qp;
  const uint32_t lane = S.lane;
  uint8_t* sim = L.sims + (uint64_t)b * L.layout.stride;
  S.state = reinterpret_cast<uint64_t*>(sim + L.layout.off_state);
  S.cst = reinterpret_cast<CtaState*>(sim + L.layout.off_cta);
  S.mq_g = reinterpret_cast<uint32_t*>(sim + L.layout.off_mq);
  const WinLds W =
      win_lds(S.G.n_ops, L.max_nsm, server_stride(S.G.props, L.srv_one ? 1u : L.max_nsub), L.qp, S.G.n_tops, MODE);
  S.optab = reinterpret_cast<uint4*>(lds + W.optab);
  S.tops = reinterpret_cast<uint16_t*>(lds + W.tops);
  S.srv = lds + W.srv;
  S.mq_head = lds + W.mq_head;
  S.mq_pos = lds + W.mq_pos;
  S.fr = reinterpret_cast<uint64_t*>(lds + W.fr);
  S.dsc = lds + kWinDsc;
  S.nr_cnt = lds + kWinNrCnt;
  S.fr_cnt = lds + kWinFrCnt;
  S.fr_min = lds + kWinFrMin;
  S.fr_hot = lds + kWinFrHot;
  S.nr = reinterpret_cast<uint64_t*>(lds + kWinNr);
  S.ret_cnt = lds + kWinRetCnt;
  S.ret_min = lds + kWinRetMin;
  S.ret_l = reinterpret_cast<uint64_t*>(lds + kWinRetL);
  S.w_key = reinterpret_cast<uint64_t*>(lds + kWinWKey);
  S.w_aux = lds + kWinWAux;
  S.w_fin = lds + kWinWFin;
  S.stage = lds + kWinStage;
  if (lane == 0) {
    uint64_t* const ptrs = reinterpret_cast<uint64_t*>(lds + kWinPtrs);
    ptrs[S.kPSucc] = reinterpret_cast<uint64_t>(S.G.succ);
    ptrs[S.kPIndeg] = reinterpret_cast<uint64_t>(S.G.indeg);
    ptrs[S.kPRoots] = reinterpret_cast<uint64_t>(S.G.roots);
    ptrs[S.kPCtas] = reinterpret_cast<uint64_t>(S.G.ctas);
    ptrs[S.kPKernels] = reinterpret_cast<uint64_t>(S.G.kernels);
    ptrs[S.kPTsucc] = reinterpret_cast<uint64_t>(S.G.tsucc);
    ptrs[S.kPTindeg] = reinterpret_cast<uint64_t>(S.G.tindeg);
    ptrs[S.kPFrG] = reinterpret_cast<uint64_t>(sim + L.layout.off_rp);
    ptrs[S.kPRetG] = reinterpret_cast<uint64_t>(sim + L.layout.off_ret);
    ptrs[S.kPHw] = reinterpret_cast<uint64_t>(S.hw);
  }
  S.out_cycles = (L.flags & GTS_OUT_NODES) ? L.out_cycles : nullptr;

  bool infeasible = false;
  for (uint32_t k = lane; k < S.G.n_kernels; k += 64) infeasible |= kernel_slots(S.G.kernels[k], S.hw) == 0;
  if (__ballot(infeasible)) {
    if (lane == 0) {
      L.out_makespan[b] = 0xFFFFFFFFu;
      L.out_status[b] = GTS_SIM_INFEASIBLE;
      if (L.out_digest) L.out_digest[b] = 0;
    }
    return;
  }

  // Setup: duration table and Lm, idle servers, empty queues; node state of
  // CTAs that receive cross-CTA edges (the others are zeroed at dispatch).
  uint64_t lm = ~0ull;
  for (uint32_t q = lane; q < S.G.n_ops; q += 64) {
    uint4 e = op_entry(S.G.ops[q], S.hw, S.G.props);
    const uint32_t cls = e.w & 7u;
    if (L.srv_one && cls <= C_SFU)  // the class's single word: lane 0 of its slot
      e.w = (e.w & 0xFFu) | (1u << 8) | (compute_slot(S.G.props, cls) << 16);
    S.optab[q] = e;
    if (cls == C_GLOAD || cls == C_GSTORE) {
      const uint64_t d = (uint64_t)e.y + e.z;
      lm = d < lm ? d : lm;
      if constexpr (LRU) {  // a tile access may take either server
        const bool other_dram = ((e.w >> 3) & 1u) == 0u;
        const uint64_t d2 = (uint64_t)clamp_occ(cdiv64((uint64_t)S.G.ops[q].work * 65536ull,
                                                        S.hw[HW_RATE + (other_dram ? R_DRAM : R_L2)])) +
                            S.hw[HW_LAT + (other_dram ? L_DRAM : L_L2)];
        lm = d2 < lm ? d2 : lm;
      }
    }
  }
  lm = wmin64(lm);
  if constexpr (TXN) {
    // a node completes with its last line, no earlier than a cycle after the
    // line enters plus the faster server's latency
    S.t_idx = lds + W.t_idx;
    S.t_next = lds + W.t_next;
    S.t_max = lds + W.t_max;
    S.t_start = lds + W.t_start;
    S.r_gmem = S.hw[HW_RATE + R_GMEM];
    S.q_l2 = cdiv64((uint64_t)GTS_LINE_BYTES << 32, S.hw[HW_RATE + R_L2]);
    S.q_dr = cdiv64((uint64_t)GTS_LINE_BYTES << 32, S.hw[HW_RATE + R_DRAM]);
    S.lat_l2 = S.hw[HW_LAT + L_L2];
    S.lat_dr = S.hw[HW_LAT + L_DRAM];
    lm = 1ull + (S.lat_l2 < S.lat_dr ? S.lat_l2 : S.lat_dr);
    // one node's lines of one cycle share a key and must fit one batch: at
    // most ceil(rate / 128 B) of them; faster engines go to the general
    // kernel.  So does NO_CONTENTION: without the engine's order the lines
    // of the nodes queued on an SM interleave, and looking ahead a bounded
    // number of ring entries no longer finds every due line.
    if (S.r_gmem > (kWinCap / 2) << S.kLineShift || S.nocont) {
      if (lane == 0) L.out_status[b] = kStatusRetry;
      return;
    }
  }
  S.Lm = lm < kWindowMax ? lm : kWindowMax;
  for (uint32_t i = lane; i < S.G.n_tops; i += 64) S.tops[i] = S.G.tops[i];
  for (uint32_t i = lane; i < S.nsm * S.sstride; i += 64) S.srv[i] = 0;
  for (uint32_t i = lane; i < S.nsm; i += 64) {
    S.mq_head[i] = 0xFFFFFFFFu;
    S.mq_pos[i] = 0;
  }
  S.nr_cnt[lane] = 0;
  S.fr_cnt[lane] = 0;
  S.fr_min[lane] = 0xFFFFFFFFu;
  S.fr_hot[lane] = 0;
  S.Hnear = 0;
  if (lane == 0) {
    *S.ret_cnt = 0;
    *S.ret_min = 0xFFFFFFFFu;
  }
  if constexpr (LRU) {
    S.l2_lines = S.hw[HW_L2_LINES];
    S.lru_last = (gmem<uint32_t>*)(sim + L.layout.off_lru);
    S.lru_bit = (gmem<uint64_t>*)(sim + L.layout.off_lru_bit);
    S.lw = lds + W.lru;
    S.lru_acc = TXN ? S.G.n_txn : S.G.n_nodes;  // at most one access per node, or per line of a node
    S.lru_now = 0;
    S.lru_total = 0;
    if (S.l2_lines) {
      const uint32_t keys = TXN ? S.G.n_lines : S.G.n_tiles;
      for (uint32_t x = lane; x < keys; x += 64) S.lru_last[x] = 0u;
      for (uint32_t i = lane; i <= S.lru_acc; i += 64) S.lru_bit[i] = 0ull;
    }
  }
  if (S.G.props & kGraphHasShared) {
    for (uint32_t c = lane; c < S.G.n_ctas; c += 64) {
      const CtaDev cd = S.G.ctas[c];
      if (cd.root_count & kCtaShared)
        for (uint32_t i = 0; i < cd.node_count; ++i) S.state[cd.node_begin + i] = 0ull;
    }
  }
  mem_wait();
  __syncthreads();

  {
    uint32_t kb, ke;
    uint64_t sl;
    S.load_kernel(0, kb, ke, sl);
    if (lane == 0) {
      uint32_t* const ctl = lds + kWinCtl;
      ctl[0] = 0;  // next CTA
      ctl[1] = 0;  // retired
      ctl[2] = 0;  // current kernel
      ctl[3] = kb;
      ctl[4] = ke;
      ctl[5] = ctl[6] = ctl[7] = 0;
      *reinterpret_cast<uint64_t*>(ctl + 8) = sl;
    }
  }
  S.run_k = 0xFFFFFFFFu;  // no CTA dispatched yet
  S.t_n = 0;
  S.sink_ret = false;
  S.l2_av = 0;
  S.dram_av = 0;
  S.digest = 0;
  S.makespan = 0;
  S.nfin = 0;
  S.bad = 0;
  S.st_local = S.st_maxrq = S.st_maxmq = S.st_maxret = 0;
  if (lane < 16) lds[kWinStats + lane] = 0;

  // phase clocks only on request: reading the clock waits for every
  // outstanding scalar and LDS access
  const bool clk = L.clocks != 0;
  // memory arrivals per window: the LRU decisions keep registers for half
  // the batch positions
  constexpr uint32_t kMemCap = LRU ? kWinCap / 2 : kWinCap;
  S.dispatch(0);
  wsync();
  uint64_t last_T = kNoKey;  // TXN: windows in a row that start at one cycle (a bound, never reached)
  uint32_t same_T = 0;
  while (!__ballot(S.bad != 0)) {
    const uint64_t c0 = clk ? __builtin_amdgcn_s_memtime() : 0ull;
    // T: lower bound of the earliest pending event
    uint64_t tmin = kNoKey;
    {
      const uint32_t fm = S.fr_min[lane];  // near is empty between windows
      tmin = fm == 0xFFFFFFFFu ? kNoKey : fm;  // 0xFFFFFFFF: empty (cycles stop at kMaxCycle)
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j) {
        const uint32_t s = lane + 64u * j;
        if (j < S.nslot && s < S.nsm && ((S.mq_pos[s] >> 8) & 0xFFu)) {
          const uint64_t k = S.mq_head[s];
          tmin = k < tmin ? k : tmin;
        }
      }
    }
    const uint32_t rmin = uni(*S.ret_min);
    if (uni(*S.ret_cnt)) tmin = rmin < tmin ? rmin : tmin;
    const uint64_t T = wmin64(tmin);
    if (T == kNoKey) break;
    if constexpr (TXN) {
      // every window processes an event or raises a lower bound; should one
      // cycle ever open 2^20 windows in a row, the simulation goes back to
      // the general kernel rather than spinning
      same_T = T == last_T ? same_T + 1u : 0u;
      last_T = T;
      if (same_T > (1u << 20)) {
        S.bad |= kBadMemQ;
        break;
      }
    }
    uint64_t H0 = T + S.Lm;
    H0 = H0 < 0xFFFFFFFFull ? H0 : 0xFFFFFFFFull;  // cycles never exceed kMaxCycle
    const uint64_t c1 = clk ? __builtin_amdgcn_s_memtime() : 0ull;

    // Retirement phase: retirements below H0, in cycle order, each distinct
    // cycle followed by dispatch.  More than kWinCap of them lower H0.
    if (rmin < H0 && uni(*S.ret_cnt)) {
      const uint32_t n = min(uni(*S.ret_cnt), kRetireCap);
      uint32_t D = wave_sum_u32(S.count_ret(H0, n));
      if (D > kWinCap) {
        uint64_t lo = T + 1, hi = H0;
        while (hi - lo > 1) {
          const uint64_t mid = (lo + hi) / 2;
          if (wave_sum_u32(S.count_ret(mid, n)) <= kWinCap)
            lo = mid;
          else
            hi = mid;
        }
        H0 = lo;
        D = wave_sum_u32(S.count_ret(H0, n));
      }
      // more than kWinCap at cycle T alone: released together without a sort
      const bool single = D > kWinCap;
      // compact in place, 64 entries at a time: due ones to w_key, the rest
      // to the front of the list
      uint32_t dp = 0, kp = 0, kmin = 0xFFFFFFFFu;
      for (uint32_t base = 0; base < n; base += 64) {
        const uint32_t i = base + lane;
        const uint64_t k = i < n ? S.ret_get(i) : kNoKey;
        const bool due = i < n && (k >> 32) < H0;
        const bool keep = i < n && !due;
        const uint64_t bd = __ballot(due), bk = __ballot(keep);
        if (due) {
          if (single)
            atomicSub(&S.mq_pos[(uint32_t)k], 1u << 16);
          else
            S.w_key[dp + lanes_below(bd, lane)] = k;
        }
        if (keep) {
          const uint32_t dst = kp + lanes_below(bk, lane);
          if (dst != i) S.ret_set(dst, k);  // an entry that keeps its place is not rewritten
          kmin = (uint32_t)(k >> 32) < kmin ? (uint32_t)(k >> 32) : kmin;
        }
        dp += (uint32_t)__popcll(bd);
        kp += (uint32_t)__popcll(bk);
      }
      kmin = (uint32_t)wmin64(kmin);
      wsync();
      if (lane == 0) {
        *S.ret_cnt = kp;
        *S.ret_min = kmin;
      }
      wsync();
      const uint32_t R = single ? 0u : dp;
      if (single) {
        wsync();
        S.count_retired(dp);
        S.count(13, dp);
        S.dispatch((uint32_t)T);
        wsync();
        if (__ballot(S.bad != 0)) break;
      }
      if (R) {
        if (R <= 64)
          S.template rank_sort<1>(R);
        else if (R <= 128)
          S.template rank_sort<2>(R);
        else
          S.template rank_sort<4>(R);
        bool stop = false;
        for (uint32_t i = 0; i < R && !stop;) {  // retirement i in cycle order is w_key[stage[i]]
          const uint64_t r = uni64(S.w_key[S.stage[i]] >> 32);
          uint32_t j = i;
          while (j < R && uni64(S.w_key[S.stage[j]] >> 32) == r) ++j;
          for (uint32_t x = i + lane; x < j; x += 64) atomicSub(&S.mq_pos[(uint32_t)S.w_key[S.stage[x]]], 1u << 16);
          wsync();
          S.count_retired(j - i);
          S.count(13, j - i);
          S.dispatch((uint32_t)r);
          i = j;
          stop = __ballot(S.bad != 0) != 0;
        }
        wsync();
        if (__ballot(S.bad != 0)) break;
      }
    }
    const uint64_t c2 = clk ? __builtin_amdgcn_s_memtime() : 0ull;

    // Local phase.
    S.pool_rebuild(H0);
    wsync();
    S.Hnear = H0;
    uint32_t steps = 1;
    while (S.local_step(H0)) ++steps;
    S.count(11, steps);
    S.Hnear = 0;
    wsync();
    const uint64_t c3 = clk ? __builtin_amdgcn_s_memtime() : 0ull;
    if (__ballot(S.bad != 0)) break;

    // Memory phase: the arrivals whose key (cycle, id) is below K <= H0 << 32.
    uint32_t M = 0;
    if constexpr (TXN) {
      M = S.txn_select(T, H0, kMemCap);
    } else {
      constexpr uint32_t GQ = kGq<NB>;
      // Up to GQ head entries of each SM whose head may be below H0 are loaded;
      // K is lowered so that every due arrival is among them, and so that at
      // most kMemCap are due -- the rest, possibly of the same cycle, wait for
      // the next window (they complete after it starts, and no arrival of a
      // cycle below H0 can still appear).
      {
        uint32_t elo[NB][GQ], ehi[NB][GQ], eop[NB][GQ], cnt[NB], hd[NB];
        bool ld[NB];
        uint64_t Kl = H0 << 32;
  #pragma unroll
        for (uint32_t j = 0; j < NB; ++j) {
          const uint32_t s = lane + 64u * j;
          const bool valid = j < S.nslot && s < S.nsm;
          const uint32_t pos = valid ? S.mq_pos[s] : 0u;
          hd[j] = pos & 0xFFu;
          cnt[j] = (pos >> 8) & 0xFFu;
          ld[j] = valid && cnt[j] > 0 && S.mq_head[s] < H0;
  #pragma unroll
          for (uint32_t q = 0; q < GQ; ++q) {
            eop[j][q] = 0;
            elo[j][q] = ehi[j][q] = 0xFFFFFFFFu;
            if (ld[j] && q < cnt[j]) {
              const uint32_t* e = S.mq_g + ((uint64_t)s * kRing + (hd[j] + q) % kRing) * 3u;
              elo[j][q] = e[0];
              ehi[j][q] = e[1];
              eop[j][q] = e[2];
            }
          }
          if (ld[j] && cnt[j] > GQ) {
            const uint64_t x = (((uint64_t)ehi[j][GQ - 1] << 32) | elo[j][GQ - 1]) + 1;
            Kl = x < Kl ? x : Kl;
          }
        }
        uint64_t K = wmin64(Kl);
        M = wave_sum_u32(due_count(ehi, elo, K));
        if (M > kMemCap) {
          // keep at most kMemCap: the largest cycle boundary that does (a
          // window spans at most 1024 cycles: a few halvings), or, when cycle T
          // alone holds more, a boundary between the keys of cycle T
          const uint64_t Kmax = K;  // count(< Kmax) > kMemCap
          uint64_t lo = T, hi = Kmax >> 32;  // cycles; count(< T << 32) = 0
          if (wave_sum_u32(due_count(ehi, elo, hi << 32)) <= kMemCap) {
            lo = hi;
          } else {
            while (hi - lo > 1) {
              const uint64_t mid = lo + (hi - lo) / 2;
              if (wave_sum_u32(due_count(ehi, elo, mid << 32)) <= kMemCap)
                lo = mid;
              else
                hi = mid;
            }
          }
          K = lo << 32;
          if (lo == T) {
            uint64_t klo = T << 32, khi = (T + 1) << 32;  // count(< khi) > kMemCap
            khi = Kmax < khi ? Kmax : khi;
            while (khi - klo > 1) {
              const uint64_t mid = klo + (khi - klo) / 2;
              if (wave_sum_u32(due_count(ehi, elo, mid)) <= kMemCap)
                klo = mid;
              else
                khi = mid;
            }
            K = klo;
          }
          M = wave_sum_u32(due_count(ehi, elo, K));
        }
        {
          uint32_t p = wave_excl_scan_u32(due_count(ehi, elo, K));
  #pragma unroll
          for (uint32_t j = 0; j < NB; ++j) {
            const uint32_t s = lane + 64u * j;
            if (j < S.nslot && s < S.nsm) {
              uint32_t d = 0;
  #pragma unroll
              for (uint32_t q = 0; q < GQ; ++q) {
                if ((((uint64_t)ehi[j][q] << 32) | elo[j][q]) < K) {
                  S.w_key[p + d] = ((uint64_t)ehi[j][q] << 32) | elo[j][q];
                  S.w_aux[p + d] = eop[j][q] | (s << 16);
                  ++d;
                }
              }
              S.dsc[s] = p | (d << 16);
              p += d;
              if (ld[j]) {
                const uint32_t left = cnt[j] - d;
                S.mq_pos[s] = (S.mq_pos[s] & 0xFFFF0000u) | ((hd[j] + d) % kRing) | (left << 8);
                if (left) {
                  uint32_t nh = ehi[j][GQ - 1] + 1;  // lower bound when the next entry was not loaded
  #pragma unroll
                  for (uint32_t q = 0; q < GQ; ++q)
                    if (q == d) nh = ehi[j][q];
                  S.mq_head[s] = nh;
                }
              }
            }
          }
        }
      }
    }
    wsync();
    if (__ballot(S.bad != 0)) break;
    const uint64_t c4 = clk ? __builtin_amdgcn_s_memtime() : 0ull;
    if constexpr (TXN) {
      if (M && M <= 64)
        S.template memory_phase_txn<1>(M);
      else if (M)
        S.template memory_phase_txn<2>(M);
    } else {
      if (M && M <= 64)
        S.template memory_phase<1>(M);
      else if (M && (LRU || M <= 128))
        S.template memory_phase<2>(M);
      else if (M)
        S.template memory_phase<4>(M);
    }
    wsync();
    const uint64_t c5 = clk ? __builtin_amdgcn_s_memtime() : 0ull;
    S.count(10, 1);
    S.count(12, M);
    S.count_max(14, M);
    if (clk) {
      S.count_clk(0, c1 - c0);
      S.count_clk(1, c2 - c1);
      S.count_clk(2, c3 - c2);
      S.count_clk(3, c4 - c3);
      S.count_clk(4, c5 - c4);
    }
  }

  const uint64_t bad_any = __ballot(S.bad != 0);
  const uint64_t ovf_any = __ballot((S.bad & kBadOverflow) != 0);
  uint64_t dg = S.digest, mk = S.makespan, nf = S.nfin, nl = S.st_local;
  uint32_t why = S.bad, mrq = S.st_maxrq, mmq = S.st_maxmq, mret = S.st_maxret;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    why |= __shfl_xor(why, o, 64);
    mrq = max(mrq, (uint32_t)__shfl_xor(mrq, o, 64));
    mmq = max(mmq, (uint32_t)__shfl_xor(mmq, o, 64));
    mret = max(mret, (uint32_t)__shfl_xor(mret, o, 64));
    dg += __shfl_xor(dg, o, 64);
    const uint64_t om = __shfl_xor(mk, o, 64);
    mk = om > mk ? om : mk;
    nf += __shfl_xor(nf, o, 64);
    nl += __shfl_xor(nl, o, 64);
  }
  if (lane == 0) {
    uint64_t* stats = reinterpret_cast<uint64_t*>(sim + L.layout.stride - kStatsBytes);
    const uint32_t* cw = lds + kWinStats;
    const uint64_t* ck = reinterpret_cast<const uint64_t*>(cw);
    stats[0] = cw[10];
    stats[1] = cw[11];
    stats[2] = nl;
    stats[3] = cw[12];
    stats[4] = cw[13];
    stats[5] = cw[14];
    stats[6] = ck[0];
    stats[7] = ck[1];
    stats[8] = ck[2];
    stats[9] = ck[3];
    stats[10] = ck[4];
    stats[11] = 0;
    stats[12] = why;
    stats[13] = mrq;
    stats[14] = mmq;
    stats[15] = mret;
    int32_t st = GTS_SIM_OK;
    if (ovf_any)
      st = GTS_SIM_OVERFLOW;
    else if (bad_any)
      st = kStatusRetry;
    else if (nf != S.G.n_nodes)
      st = GTS_SIM_DEADLOCK;
    L.out_status[b] = st;
    L.out_makespan[b] = st == GTS_SIM_OK ? (uint32_t)mk : 0xFFFFFFFFu;
    if (L.out_digest) L.out_digest[b] = st == GTS_SIM_OK ? dg : 0ull;
  }
}

}  // namespace

// The kernels of each mode are compiled in a part of their own (the same
// source built with GTS_WINDOW_PART = 0, 1, 2, in parallel); the launch
// lives in part 0 and names the others by declaration.
#ifndef GTS_WINDOW_PART
#define GTS_WINDOW_PART 0
#endif
#if GTS_WINDOW_PART == 0
extern "C" __global__ __launch_bounds__(64) void gts_sim_window1(Launch L) { window_body<1, kWinPlain>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window2(Launch L) { window_body<2, kWinPlain>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window3(Launch L) { window_body<3, kWinPlain>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window4(Launch L) { window_body<4, kWinPlain>(L); }
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window1_lru(Launch L);
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window2_lru(Launch L);
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window3_lru(Launch L);
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window4_lru(Launch L);
extern "C" __global__ __launch_bounds__(64) void gts_sim_window1_txn(Launch L);
extern "C" __global__ __launch_bounds__(64) void gts_sim_window2_txn(Launch L);
extern "C" __global__ __launch_bounds__(64) void gts_sim_window3_txn(Launch L);
extern "C" __global__ __launch_bounds__(64) void gts_sim_window4_txn(Launch L);
#elif GTS_WINDOW_PART == 1
// graphs whose loads / stores name tiles (LRU L2): held to three waves per
// SIMD, as the others (a few registers spill at three and four SMs per
// lane; measured faster than two waves per SIMD without spills)
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window1_lru(Launch L) { window_body<1, kWinTiles>(L); }
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window2_lru(Launch L) { window_body<2, kWinTiles>(L); }
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window3_lru(Launch L) { window_body<3, kWinTiles>(L); }
extern "C" __global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void gts_sim_window4_lru(Launch L) { window_body<4, kWinTiles>(L); }
#else
// graphs whose loads / stores stream 128-B lines (transaction-level memory):
// the register allocator's own occupancy (measured 15 % faster than three
// waves per SIMD with spills)
extern "C" __global__ __launch_bounds__(64) void gts_sim_window1_txn(Launch L) { window_body<1, kWinTxn>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window2_txn(Launch L) { window_body<2, kWinTxn>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window3_txn(Launch L) { window_body<3, kWinTxn>(L); }
extern "C" __global__ __launch_bounds__(64) void gts_sim_window4_txn(Launch L) { window_body<4, kWinTxn>(L); }
#endif

#if GTS_WINDOW_PART == 0
hipError_t launch_window(const Launch& L, uint32_t lds_bytes, hipStream_t stream) {
  if (L.B == 0) return hipSuccess;
  const uint32_t nb = (L.max_nsm + 63) / 64;
  void (*const plain[4])(Launch) = {gts_sim_window1, gts_sim_window2, gts_sim_window3, gts_sim_window4};
  void (*const tiled[4])(Launch) = {gts_sim_window1_lru, gts_sim_window2_lru, gts_sim_window3_lru,
                                    gts_sim_window4_lru};
  void (*const txn[4])(Launch) = {gts_sim_window1_txn, gts_sim_window2_txn, gts_sim_window3_txn,
                                  gts_sim_window4_txn};
  const uint32_t i = nb <= 1 ? 0u : nb >= 4 ? 3u : nb - 1u;
  void (*const k)(Launch) = (L.img.props & kGraphTxn) ? txn[i] : (L.img.props & kGraphTiles) ? tiled[i] : plain[i];
  hipLaunchKernelGGL(k, dim3(L.B), dim3(64), lds_bytes, stream, L);
  return hipGetLastError();
}
#endif

}  // namespace gts
