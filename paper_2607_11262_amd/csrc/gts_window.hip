// gts_window.hip — windowed simulation kernel for gfx950 (MI355X).
//
// One wavefront simulates one (graph, hardware record) pair, with one lane
// per simulated SM (SM s on lane s mod 64).  Instead of taking one event at a
// time, it advances the machine through time windows [T, H):
//
//   T = the earliest pending event;  H = T + min(Lm, 1024), where Lm is the
//       smallest possible delay from a memory arrival to its completion
//       (min over the graph's memory ops of L2/DRAM occupancy + latency).
//   retirement phase: every CTA retirement with cycle < H, in cycle order,
//       each distinct cycle followed by dispatch (wave-cooperative);
//   local phase: every lane issues its SMs' ready nodes with cycle < H in
//       (cycle, node id) order -- per-SM servers, finish, release of
//       out-edges (all inside the same CTA), memory nodes reserve the SM's
//       engine and queue an arrival at their engine start;
//   memory phase: the arrivals with cycle < H from all SMs are counting-
//       sorted in LDS by (cycle, node id), served by the chip-wide L2 and
//       DRAM FIFO servers through a max-plus prefix scan across the wave, and
//       handed back to the lane that owns their SM, which completes them
//       (CTA bookkeeping, release of out-edges).
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
// completion.  If a window's arrivals do not fit in LDS, the memory phase
// takes the prefix (in cycle order) that fits and leaves the rest for the
// next window, whose start is then at or before them.  The host sends other
// graphs, and simulations whose queues overflow, to the general kernel.
//
// Memory: per-SM ready queues and memory-arrival FIFOs live in LDS (with a
// spill area in the simulation's scratch), as do the window's arrivals,
// counting buckets and pending retirements; per-node state (remaining
// in-edges, latest release) lives in scratch and is initialised when its CTA
// is dispatched.  Node records carry their first four successors, so issuing
// a node costs one record load and one batch of successor-state loads, and a
// lane batches one node of each of up to four of its SMs per round trip.
#include <hip/hip_runtime.h>

#include "../../include/gts.h"
#include "gts_common.h"
#include "gts_dev.h"

namespace gts {

namespace {

constexpr uint64_t kNoKey = ~0ull;
constexpr uint32_t kBadOverflow = 1u, kBadReady = 2u, kBadMemQ = 4u, kBadRetire = 8u, kBadWindow = 16u;
constexpr uint32_t NB = 4;  // SMs per lane handled per batch

// Node state: remaining in-edges (low word) | latest release cycle (high word).
__device__ __forceinline__ uint32_t* st_rem(uint64_t* st) { return reinterpret_cast<uint32_t*>(st); }
__device__ __forceinline__ uint32_t* st_acc(uint64_t* st) { return reinterpret_cast<uint32_t*>(st) + 1; }

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

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return uni(x);
}

__device__ __forceinline__ uint32_t wave_excl_scan_u32(uint32_t x, uint32_t lane) {
  uint32_t inc = x;
#pragma unroll
  for (uint32_t d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d, 64);
    if (lane >= d) inc += y;
  }
  return inc - x;
}

struct Compose {  // f(x) = max(x, a) + o on int64
  int64_t a, o;
};
__device__ __forceinline__ Compose compose(Compose f, Compose g) {  // g after f
  const int64_t ga = g.a - f.o;
  return Compose{f.a > ga ? f.a : ga, f.o + g.o};
}
__device__ __forceinline__ Compose shfl_up_c(Compose c, uint32_t d) {
  return Compose{__shfl_up(c.a, d, 64), __shfl_up(c.o, d, 64)};
}

// A node record held in registers: a = {op | indeg << 16, cta, succ_begin,
// succ_end}, b = the first four successors.
struct Rec {
  uint4 a, b;
  __device__ __forceinline__ uint32_t op() const { return a.x & 0xFFFFu; }
  __device__ __forceinline__ uint32_t cta() const { return a.y; }
  __device__ __forceinline__ uint32_t sb() const { return a.z; }
  __device__ __forceinline__ uint32_t se() const { return a.w; }
  __device__ __forceinline__ uint32_t nsucc() const { return a.w - a.z; }
  __device__ __forceinline__ uint32_t succ(uint32_t k) const {  // selects, no dynamic register index
    return k == 0 ? b.x : k == 1 ? b.y : k == 2 ? b.z : b.w;
  }
};
__device__ __forceinline__ Rec load_rec(const NodeDev* nodes, uint32_t v) {
  const uint4* p = reinterpret_cast<const uint4*>(nodes + v);
  return Rec{p[0], p[1]};
}

// Does a node need the one-edge-at-a-time path (more than four successors,
// or an inline successor that is a shared node)?
__device__ __forceinline__ bool needs_slow(const Rec r) {
  const uint32_t n = r.nsucc();
  if (n > kInlineSucc) return true;
  bool sh = false;
#pragma unroll
  for (uint32_t k = 0; k < kInlineSucc; ++k)
    sh |= k < n && ((r.succ(k) >> GTS_EDGE_KIND_SHIFT) & kDevShared);
  return sh;
}

struct WSim {
  Image G;
  const uint32_t* hw;
  uint32_t b, lane, flags, nsm, nsub, sstride, nslot, NS, ql, qml, memcap;
  bool nocont, ofin;
  // LDS
  uint4* optab;
  uint32_t *srv, *resident, *rq_cnt;
  uint64_t* rq_l;
  uint32_t *mq_lh, *mq_nl, *mq_gh, *mq_ng;
  uint64_t* mq_lk;
  uint32_t* mq_la;
  uint32_t *ret_cnt, *ret_min;
  uint64_t* ret_l;
  uint32_t *dstart, *dcnt, *bucket;
  uint64_t* w_key0;
  uint32_t* w_aux0;
  uint64_t* s_key;
  uint32_t *s_slot, *w_fin;
  // scratch
  uint64_t* state;
  CtaState* cst;
  uint64_t* rq_g;
  uint64_t* mq_gk;
  uint32_t* mq_ga;
  uint64_t* ret_g;
  uint32_t* out_cycles;
  // uniform control
  uint32_t next_cta, retired, cur_k, kstart_k, kstart_t, kstart_valid;
  uint64_t l2_av, dram_av, Lm;
  // per lane
  uint64_t digest;
  uint32_t makespan, nfin, bad;
  uint64_t st_windows, st_iters, st_local, st_mem, st_retires, st_maxm;
  uint32_t st_maxrq, st_maxmq, st_maxret;
  uint64_t tm0, tm1, tm2, tm3, tm4, tm5;

  // ---- per-SM ready queue: entries [0, ql) in LDS, [ql, ql + kQueueReady) spilled
  __device__ __forceinline__ uint32_t rq_n(uint32_t s) const {
    const uint32_t n = rq_cnt[s];
    return n < ql + kQueueReady ? n : ql + kQueueReady;
  }
  __device__ __forceinline__ uint64_t rq_get(uint32_t s, uint32_t i) const {
    return i < ql ? rq_l[i * NS + s] : rq_g[(uint64_t)(i - ql) * nsm + s];
  }
  __device__ __forceinline__ void rq_set(uint32_t s, uint32_t i, uint64_t k) {
    if (i < ql)
      rq_l[i * NS + s] = k;
    else
      rq_g[(uint64_t)(i - ql) * nsm + s] = k;
  }
  __device__ __forceinline__ void rq_push(uint32_t s, uint64_t key) {
    const uint32_t slot = atomicAdd(&rq_cnt[s], 1u);
    st_maxrq = slot + 1 > st_maxrq ? slot + 1 : st_maxrq;
    if (slot < ql + kQueueReady)
      rq_set(s, slot, key);
    else
      bad |= kBadReady;
  }

  // ---- per-SM memory-arrival FIFO (strictly increasing cycles): the oldest
  // entries in an LDS ring, the rest in a spill ring; owner lane only.
  // Invariant: the spill ring is non-empty only while the LDS ring is full.
  __device__ __forceinline__ uint32_t mq_size(uint32_t s) const { return mq_nl[s] + mq_ng[s]; }
  __device__ __forceinline__ uint64_t mq_peek(uint32_t s, uint32_t i) const {
    const uint32_t nl = mq_nl[s];
    if (i < nl) return mq_lk[((mq_lh[s] + i) % qml) * NS + s];
    return mq_gk[(uint64_t)((mq_gh[s] + i - nl) % kQueueMem) * nsm + s];
  }
  __device__ __forceinline__ void mq_push(uint32_t s, uint64_t key, uint32_t op) {
    const uint32_t nl = mq_nl[s], ng = mq_ng[s];
    if (ng == 0 && nl < qml) {
      const uint32_t i = ((mq_lh[s] + nl) % qml) * NS + s;
      mq_lk[i] = key;
      mq_la[i] = op;
      mq_nl[s] = nl + 1;
    } else if (ng < kQueueMem) {
      const uint64_t i = (uint64_t)((mq_gh[s] + ng) % kQueueMem) * nsm + s;
      mq_gk[i] = key;
      mq_ga[i] = op;
      mq_ng[s] = ng + 1;
    } else {
      bad |= kBadMemQ;
    }
    st_maxmq = nl + ng + 1 > st_maxmq ? nl + ng + 1 : st_maxmq;
  }
  __device__ __forceinline__ void mq_pop(uint32_t s, uint64_t& key, uint32_t& op) {
    uint32_t lh = mq_lh[s], nl = mq_nl[s];
    const uint32_t i = lh * NS + s;
    key = mq_lk[i];
    op = mq_la[i];
    lh = (lh + 1) % qml;
    --nl;
    const uint32_t ng = mq_ng[s];
    if (ng) {  // refill the LDS ring from the spill ring
      const uint32_t gh = mq_gh[s];
      const uint64_t gi = (uint64_t)gh * nsm + s;
      const uint32_t li = ((lh + nl) % qml) * NS + s;
      mq_lk[li] = mq_gk[gi];
      mq_la[li] = mq_ga[gi];
      ++nl;
      mq_gh[s] = (gh + 1) % kQueueMem;
      mq_ng[s] = ng - 1;
    }
    mq_lh[s] = lh;
    mq_nl[s] = nl;
  }

  // arrivals of this lane's SMs with cycle < X
  __device__ __forceinline__ uint32_t count_due(uint64_t X) const {
    uint32_t cnt = 0;
    for (uint32_t j = 0; j < nslot; ++j) {
      const uint32_t s = lane + 64u * j;
      if (s < nsm) {
        const uint32_t n = mq_size(s);
        uint32_t i = 0;
        while (i < n && (mq_peek(s, i) >> 32) < X) ++i;
        cnt += i;
      }
    }
    return cnt;
  }

  // ---- pending CTA retirements, (cycle << 32 | SM) each, unordered: entries
  // [0, kRetireLds) in LDS, the rest in scratch; ret_min holds a lower bound
  // of their cycles (exact after each retirement phase).
  __device__ __forceinline__ uint64_t ret_get(uint32_t i) const {
    return i < kRetireLds ? ret_l[i] : ret_g[i - kRetireLds];
  }
  __device__ __forceinline__ void ret_set(uint32_t i, uint64_t k) {
    if (i < kRetireLds)
      ret_l[i] = k;
    else
      ret_g[i - kRetireLds] = k;
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
    const uint32_t old = atomicSub(st_rem(&state[w]), 1u);
    if (old != 1u) return;
    const uint32_t acc = gld(st_acc(&state[w]));
    const uint32_t cw = G.nodes[w].cta;
    if (cw == src_cta) {
      rq_push(src_sm, mkkey(acc, kEvReady, w));
    } else if (cw < next_cta) {  // dispatched: ready at max(release, launch)
      const uint32_t launch = gld(&cst[cw].launch);
      rq_push(gld(&cst[cw].sm), mkkey(acc > launch ? acc : launch, kEvReady, w));
    }
  }

  // Successors beyond the inline four, and inline ones into shared nodes,
  // one edge at a time.  which: 0 = edges released at issue, 1 = edges
  // released at completion, 2 = both.
  __device__ __forceinline__ void release_slow(const Rec rec, uint32_t which, uint64_t r_issue, uint64_t r_fin, uint32_t s) {
    for (uint32_t e = rec.sb(); e < rec.se(); ++e) {
      const uint32_t k = e - rec.sb();
      const uint32_t ent = k < kInlineSucc ? rec.succ(k) : G.succ[e];
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
        const uint64_t sv = state[w];
        const uint32_t rem = (uint32_t)sv - 1u;
        uint32_t acc = (uint32_t)(sv >> 32);
        acc = r > acc ? (uint32_t)r : acc;
        state[w] = ((uint64_t)acc << 32) | rem;
        if (rem == 0) rq_push(s, mkkey(acc, kEvReady, w));
      }
    }
  }

  // ---- wave-cooperative dispatch at cycle t (after the retirements at t)
  __device__ __forceinline__ void dispatch(uint32_t t) {
    while (next_cta < G.n_ctas) {
      while (next_cta >= G.kernels[cur_k].cta_end) ++cur_k;
      const KernelDev kd = G.kernels[cur_k];
      if (retired < kd.cta_begin) return;
      const uint64_t slots = kernel_slots(kd, hw);
      uint64_t best = 0;
      for (uint32_t m = lane; m < nsm; m += 64) {
        const uint64_t fr = slots - resident[m];
        const uint64_t k = (fr << 32) | (0xFFFFFFFFu - m);
        best = k > best ? k : best;
      }
      best = uni64(wave_max_u64(best));
      if ((best >> 32) == 0) return;
      const uint32_t sm = 0xFFFFFFFFu - (uint32_t)best;
      if (!kstart_valid || kstart_k != cur_k) {
        kstart_valid = 1;
        kstart_k = cur_k;
        kstart_t = t;
      }
      const uint64_t launch = (uint64_t)t + hw[HW_CTALAT] + (kstart_t == t ? hw[HW_KLAT] : 0u);
      if (launch > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      const uint32_t c = next_cta;
      const CtaDev cd = G.ctas[c];
      const bool shared = (cd.root_count & kCtaShared) != 0;
      const uint32_t nroots = cd.root_count & ~kCtaShared;
      if (lane == 0) {
        cst[c].sm = sm;
        cst[c].launch = (uint32_t)launch;
        cst[c].left = cd.node_count;
        cst[c].maxfin = 0u;
        resident[sm] += 1;
      }
      if (!shared)  // node state of an unshared CTA is initialised at dispatch
        for (uint32_t i = lane; i < cd.node_count; i += 64)
          state[cd.node_begin + i] = (uint64_t)G.indeg[cd.node_begin + i];
      mem_wait();
      wsync();
      ++next_cta;
      for (uint32_t r0 = 0; r0 < nroots; r0 += 64) {
        const uint32_t ri = r0 + lane;
        if (ri < nroots) {
          const uint32_t v = G.roots[cd.root_begin + ri];
          const uint64_t sv = shared ? gld(&state[v]) : state[v];
          if ((uint32_t)sv == 0) {
            const uint32_t acc = (uint32_t)(sv >> 32);
            rq_push(sm, mkkey(acc > launch ? acc : launch, kEvReady, v));
          }
        }
      }
      wsync();
    }
  }

  // ---- counting sort of w_key0[0, M) by cycle (bucket = cycle - T < Wb)
  // into s_key / s_slot; ties broken by node id when fix_ties.
  __device__ __forceinline__ void csort(uint32_t M, uint64_t T, uint32_t Wb, bool fix_ties) {
    for (uint32_t i = lane; i < Wb; i += 64) bucket[i] = 0;
    wsync();
    for (uint32_t i = lane; i < M; i += 64) atomicAdd(&bucket[(uint32_t)((w_key0[i] >> 32) - T)], 1u);
    wsync();
    const uint32_t per = (Wb + 63) / 64;
    const uint32_t b0 = lane * per < Wb ? lane * per : Wb;
    const uint32_t b1 = b0 + per < Wb ? b0 + per : Wb;
    uint32_t sum = 0;
    for (uint32_t i = b0; i < b1; ++i) sum += bucket[i];
    uint32_t run = wave_excl_scan_u32(sum, lane);
    for (uint32_t i = b0; i < b1; ++i) {
      const uint32_t c = bucket[i];
      bucket[i] = run;
      run += c;
    }
    wsync();
    for (uint32_t i = lane; i < M; i += 64) {
      const uint64_t k = w_key0[i];
      const uint32_t p = atomicAdd(&bucket[(uint32_t)((k >> 32) - T)], 1u);
      s_key[p] = k;
      s_slot[p] = i;
    }
    wsync();
    if (fix_ties) {  // bucket[i] is now the end of bucket i
      for (uint32_t i = lane; i < Wb; i += 64) {
        const uint32_t end = bucket[i];
        const uint32_t beg = i ? bucket[i - 1] : 0u;
        for (uint32_t x = beg + 1; x < end; ++x) {  // insertion sort by key
          const uint64_t k = s_key[x];
          const uint32_t sl = s_slot[x];
          uint32_t y = x;
          while (y > beg && s_key[y - 1] > k) {
            s_key[y] = s_key[y - 1];
            s_slot[y] = s_slot[y - 1];
            --y;
          }
          s_key[y] = k;
          s_slot[y] = sl;
        }
      }
      wsync();
    }
  }

  // ---- local phase: one ready node below H from each of NB of this lane's
  // SMs, with one record load and one state load per node in flight together.
  __device__ __forceinline__ bool local_batch(uint32_t g0, uint64_t H) {
    uint32_t ev_v[NB], ev_t[NB], ev_s[NB];
    bool ok[NB];
    bool any = false;
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      ok[j] = false;
      ev_v[j] = ev_t[j] = 0;
      const uint32_t s = lane + 64u * (g0 + j);
      ev_s[j] = s;
      if (g0 + j < nslot && s < nsm && !bad) {
        const uint32_t n = rq_n(s);
        uint64_t best = kNoKey;
        uint32_t bi = 0;
        for (uint32_t i = 0; i < n; ++i) {
          const uint64_t k = rq_get(s, i);
          if (k < best) {
            best = k;
            bi = i;
          }
        }
        if (best != kNoKey && (best >> 32) < H) {
          rq_set(s, bi, rq_get(s, n - 1));
          rq_cnt[s] = n - 1;
          ok[j] = true;
          any = true;
          ev_t[j] = (uint32_t)(best >> 32);
          ev_v[j] = (uint32_t)best & GTS_EDGE_TARGET_MASK;
        }
      }
    }
    if (!__ballot(any)) return false;
    Rec rec[NB];
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      rec[j] = Rec{make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
      if (ok[j]) rec[j] = load_rec(G.nodes, ev_v[j]);
    }
    // timing on the SM's servers
    uint64_t rel_i[NB], rel_f[NB];
    bool is_mem[NB];
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      is_mem[j] = false;
      rel_i[j] = rel_f[j] = 0;
      if (ok[j]) {
      const uint4 od = optab[rec[j].op()];
      const uint32_t cls = od.w & 7u;
      uint32_t* S = srv + ev_s[j] * sstride;
      uint64_t st = ev_t[j], f = 0;
      if (cls <= C_SFU) {
        const uint32_t lanes = (od.w >> 8) & 0xFFu;
        if (!nocont)
          for (uint32_t l = 0; l < nsub; ++l)
            if ((lanes >> l) & 1u) st = S[l] > st ? S[l] : st;
        f = st + od.x + od.z;
        if (f <= kMaxCycle)
          for (uint32_t l = 0; l < nsub; ++l)
            if ((lanes >> l) & 1u) S[l] = (uint32_t)(st + od.x);
      } else if (cls == C_SMEM) {
        if (!nocont) st = S[nsub] > st ? S[nsub] : st;
        f = st + od.x + od.z;
        if (f <= kMaxCycle) S[nsub] = (uint32_t)(st + od.x);
      } else if (cls == C_SYNC) {
        f = st + od.z;
      } else {  // memory node: engine now, L2/DRAM in the memory phase
        if (!nocont) st = S[nsub + 1] > st ? S[nsub + 1] : st;
        is_mem[j] = true;
        f = st + od.x;  // end of engine occupancy
        if (f <= kMaxCycle) {
          S[nsub + 1] = (uint32_t)f;
          mq_push(ev_s[j], mkkey(st, kEvMem, ev_v[j]), rec[j].op());
        }
      }
      if (f > kMaxCycle) {
        bad |= kBadOverflow;
        ok[j] = false;
      } else {
        rel_i[j] = st + 1;
        rel_f[j] = f;
        if (!is_mem[j]) record(ev_v[j], st, f);
      }
      }
    }
    // successor states (inline, unshared) and CTA state, loads in flight together
    uint64_t sv[NB][kInlineSucc];
    uint4 cs[NB];
    bool sel[NB][kInlineSucc];
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
      const uint32_t nout = ok[j] ? rec[j].nsucc() : 0u;
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        sel[j][k] = false;
        sv[j][k] = 0;
        if (k < nout) {
          const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
          const bool at_issue = (bits & kDevOrder) && !ofin;
          sel[j][k] = !(bits & kDevShared) && (at_issue || !is_mem[j]);
          if (sel[j][k]) sv[j][k] = state[rec[j].succ(k) & GTS_EDGE_TARGET_MASK];
        }
      }
      cs[j] = make_uint4(0, 0, 0, 0);
      if (ok[j] && !is_mem[j]) cs[j] = *reinterpret_cast<const uint4*>(&cst[rec[j].cta()]);
    }
#pragma unroll
    for (uint32_t j = 0; j < NB; ++j) {
#pragma unroll
      for (uint32_t k = 0; k < kInlineSucc; ++k) {
        if (sel[j][k]) {
          const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
          const uint32_t w = rec[j].succ(k) & GTS_EDGE_TARGET_MASK;
          const uint64_t r = ((bits & kDevOrder) && !ofin) ? rel_i[j] : rel_f[j];
          const uint32_t rem = (uint32_t)sv[j][k] - 1u;
          uint32_t acc = (uint32_t)(sv[j][k] >> 32);
          acc = r > acc ? (uint32_t)r : acc;
          state[w] = ((uint64_t)acc << 32) | rem;
          if (rem == 0) rq_push(ev_s[j], mkkey(acc, kEvReady, w));
        }
      }
      if (!ok[j]) continue;
      if (!is_mem[j]) {  // a compute node never completes its CTA
        const uint32_t mf = (uint32_t)rel_f[j] > cs[j].w ? (uint32_t)rel_f[j] : cs[j].w;
        *reinterpret_cast<uint2*>(&cst[rec[j].cta()].left) = make_uint2(cs[j].z - 1u, mf);
      }
      if (needs_slow(rec[j])) release_slow(rec[j], is_mem[j] ? 0u : 2u, rel_i[j], rel_f[j], ev_s[j]);
      ++st_local;
    }
    return true;
  }

  // ---- memory phase: serve the M sorted arrivals, then complete them.
  __device__ __forceinline__ void memory_phase(uint32_t M) {
    constexpr int64_t kNeg = -(int64_t(1) << 62);
    const uint32_t per = (M + 63) / 64;
    const uint32_t i0 = lane * per < M ? lane * per : M;
    const uint32_t i1 = i0 + per < M ? i0 + per : M;
    Compose fl2{kNeg, 0}, fdr{kNeg, 0};
    for (uint32_t i = i0; i < i1; ++i) {
      const uint4 od = optab[w_aux0[s_slot[i]] & 0xFFFFu];
      const Compose g{(int64_t)(s_key[i] >> 32), (int64_t)od.y};
      if ((od.w >> 3) & 1u)
        fdr = compose(fdr, g);
      else
        fl2 = compose(fl2, g);
    }
    Compose il2 = fl2, idr = fdr;
#pragma unroll
    for (uint32_t d = 1; d < 64; d <<= 1) {
      const Compose pl2 = shfl_up_c(il2, d), pdr = shfl_up_c(idr, d);
      if (lane >= d) {
        il2 = compose(pl2, il2);
        idr = compose(pdr, idr);
      }
    }
    Compose el2 = shfl_up_c(il2, 1), edr = shfl_up_c(idr, 1);
    if (lane == 0) el2 = edr = Compose{kNeg, 0};
    const Compose tl2{__shfl(il2.a, 63, 64), __shfl(il2.o, 63, 64)};
    const Compose tdr{__shfl(idr.a, 63, 64), __shfl(idr.o, 63, 64)};
    int64_t xl2 = ((int64_t)l2_av > el2.a ? (int64_t)l2_av : el2.a) + el2.o;
    int64_t xdr = ((int64_t)dram_av > edr.a ? (int64_t)dram_av : edr.a) + edr.o;
    if (!nocont) {
      l2_av = (uint64_t)(((int64_t)l2_av > tl2.a ? (int64_t)l2_av : tl2.a) + tl2.o);
      dram_av = (uint64_t)(((int64_t)dram_av > tdr.a ? (int64_t)dram_av : tdr.a) + tdr.o);
    }
    for (uint32_t i = i0; i < i1; ++i) {
      const uint32_t slot = s_slot[i];
      const uint4 od = optab[w_aux0[slot] & 0xFFFFu];
      const int64_t st = (int64_t)(s_key[i] >> 32);
      const bool dram = (od.w >> 3) & 1u;
      const int64_t x = dram ? xdr : xl2;
      const int64_t m = nocont ? st : (x > st ? x : st);
      if (dram)
        xdr = m + (int64_t)od.y;
      else
        xl2 = m + (int64_t)od.y;
      const int64_t e = st + (int64_t)od.x;
      const int64_t mend = m + (int64_t)od.y;
      const uint64_t f = (uint64_t)(e > mend ? e : mend) + od.z;
      if (f > kMaxCycle) bad |= kBadOverflow;
      w_fin[slot] = f > kMaxCycle ? 0xFFFFFFFFu : (uint32_t)f;
    }
    wsync();
    if (__ballot(bad != 0)) return;
    // Completion by the owner lane, one arrival per SM per round (arrivals of
    // different SMs touch different CTAs and nodes; shared nodes use atomics).
    for (uint32_t g0 = 0; g0 < nslot; g0 += NB) {
      uint32_t rounds = 0;
#pragma unroll
      for (uint32_t j = 0; j < NB; ++j) {
        const uint32_t s = lane + 64u * (g0 + j);
        if (g0 + j < nslot && s < nsm) rounds = dcnt[s] > rounds ? dcnt[s] : rounds;
      }
      for (uint32_t r = 0; r < rounds; ++r) {
        Rec rec[NB];
        uint32_t vv[NB], ss[NB], ff[NB], tt[NB];
        bool ok[NB];
#pragma unroll
        for (uint32_t j = 0; j < NB; ++j) {
          const uint32_t s = lane + 64u * (g0 + j);
          ok[j] = g0 + j < nslot && s < nsm && r < dcnt[s];
          vv[j] = ff[j] = tt[j] = 0;
          ss[j] = s;
          rec[j] = Rec{make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
          if (ok[j]) {
            const uint32_t slot = dstart[s] + r;
            const uint64_t key = w_key0[slot];
            vv[j] = (uint32_t)key & GTS_EDGE_TARGET_MASK;
            tt[j] = (uint32_t)(key >> 32);
            ff[j] = w_fin[slot];
            rec[j] = load_rec(G.nodes, vv[j]);
          }
        }
        uint64_t sv[NB][kInlineSucc];
        bool sel[NB][kInlineSucc];
        uint4 cs[NB];
#pragma unroll
        for (uint32_t j = 0; j < NB; ++j) {
          const uint32_t nout = ok[j] ? rec[j].nsucc() : 0u;
#pragma unroll
          for (uint32_t k = 0; k < kInlineSucc; ++k) {
            sel[j][k] = false;
            sv[j][k] = 0;
            if (k < nout) {
              const uint32_t bits = rec[j].succ(k) >> GTS_EDGE_KIND_SHIFT;
              const bool at_issue = (bits & kDevOrder) && !ofin;
              sel[j][k] = !(bits & kDevShared) && !at_issue;
              if (sel[j][k]) sv[j][k] = state[rec[j].succ(k) & GTS_EDGE_TARGET_MASK];
            }
          }
          cs[j] = make_uint4(0, 0, 0, 0);
          if (ok[j]) cs[j] = *reinterpret_cast<const uint4*>(&cst[rec[j].cta()]);
        }
#pragma unroll
        for (uint32_t j = 0; j < NB; ++j) {
          const uint32_t f = ff[j];
#pragma unroll
          for (uint32_t k = 0; k < kInlineSucc; ++k) {
            if (sel[j][k]) {
              const uint32_t w = rec[j].succ(k) & GTS_EDGE_TARGET_MASK;
              const uint32_t rem = (uint32_t)sv[j][k] - 1u;
              uint32_t acc = (uint32_t)(sv[j][k] >> 32);
              acc = f > acc ? f : acc;
              state[w] = ((uint64_t)acc << 32) | rem;
              if (rem == 0) rq_push(ss[j], mkkey(acc, kEvReady, w));
            }
          }
          if (!ok[j]) continue;
          record(vv[j], tt[j], f);
          const uint32_t left = cs[j].z - 1u;
          const uint32_t mf = f > cs[j].w ? f : cs[j].w;
          *reinterpret_cast<uint2*>(&cst[rec[j].cta()].left) = make_uint2(left, mf);
          if (left == 0) ret_push(mf, ss[j]);  // the CTA retires at its largest finish
          if (needs_slow(rec[j])) release_slow(rec[j], 1u, 0, f, ss[j]);
        }
      }
    }
  }
};

}  // namespace

extern "C" __global__ __launch_bounds__(64) void gts_sim_window(Launch L) {
  const uint32_t b = blockIdx.x;
  if (b >= L.B) return;
  extern __shared__ uint32_t lds[];
  WSim S;
  S.G = L.img;
  S.hw = L.hw + (uint64_t)b * HW_WORDS;
  S.b = b;
  S.lane = threadIdx.x;
  S.flags = L.flags;
  S.nocont = (L.flags & GTS_NO_CONTENTION) != 0;
  S.ofin = (L.flags & GTS_ORDER_AT_FINISH) != 0;
  S.nsm = S.hw[HW_NSM];
  S.nsub = S.hw[HW_NSUB];
  S.sstride = S.nsub + 2;
  S.nslot = (S.nsm + 63) / 64;
  S.NS = L.max_nsm;
  S.ql = L.ql;
  S.qml = L.qml;
  S.memcap = L.memcap;
  const uint32_t lane = S.lane;
  uint8_t* sim = L.sims + (uint64_t)b * L.layout.stride;
  S.state = reinterpret_cast<uint64_t*>(sim + L.layout.off_state);
  S.cst = reinterpret_cast<CtaState*>(sim + L.layout.off_cta);
  S.rq_g = reinterpret_cast<uint64_t*>(sim + L.layout.off_rq);
  S.mq_gk = reinterpret_cast<uint64_t*>(sim + L.layout.off_mq);
  S.mq_ga = reinterpret_cast<uint32_t*>(S.mq_gk + (uint64_t)kQueueMem * S.nsm);
  const WinLds W = win_lds(S.G.n_ops, L.max_nsm, L.max_nsub, L.ql, L.qml, L.memcap);
  S.optab = reinterpret_cast<uint4*>(lds + W.optab);
  S.srv = lds + W.srv;
  S.resident = lds + W.resident;
  S.rq_cnt = lds + W.rq_cnt;
  S.rq_l = reinterpret_cast<uint64_t*>(lds + W.rq_l);
  S.mq_lh = lds + W.mq_lh;
  S.mq_nl = lds + W.mq_nl;
  S.mq_gh = lds + W.mq_gh;
  S.mq_ng = lds + W.mq_ng;
  S.mq_lk = reinterpret_cast<uint64_t*>(lds + W.mq_lk);
  S.mq_la = lds + W.mq_la;
  S.ret_cnt = lds + W.ret_cnt;
  S.ret_min = lds + W.ret_min;
  S.ret_l = reinterpret_cast<uint64_t*>(lds + W.ret_l);
  S.ret_g = reinterpret_cast<uint64_t*>(sim + L.layout.off_ret);
  S.dstart = lds + W.dstart;
  S.dcnt = lds + W.dcnt;
  S.bucket = lds + W.bucket;
  S.w_key0 = reinterpret_cast<uint64_t*>(lds + W.w_key0);
  S.w_aux0 = lds + W.w_aux0;
  S.s_key = reinterpret_cast<uint64_t*>(lds + W.s_key);
  S.s_slot = lds + W.s_slot;
  S.w_fin = lds + W.w_fin;
  S.out_cycles = (L.flags & GTS_OUT_NODES) ? L.out_cycles : nullptr;

  bool infeasible = false;
  for (uint32_t k = lane; k < S.G.n_kernels; k += 64)
    infeasible |= kernel_slots(S.G.kernels[k], S.hw) == 0;
  if (__ballot(infeasible)) {
    if (lane == 0) {
      L.out_makespan[b] = 0xFFFFFFFFu;
      L.out_status[b] = GTS_SIM_INFEASIBLE;
      if (L.out_digest) L.out_digest[b] = 0;
    }
    return;
  }

  // Setup: duration table and Lm, idle servers, empty queues; node state of
  // CTAs that receive cross-CTA edges (the others are set at dispatch).
  uint64_t lm = ~0ull;
  for (uint32_t q = lane; q < S.G.n_ops; q += 64) {
    const uint4 e = op_entry(S.G.ops[q], S.hw);
    S.optab[q] = e;
    const uint32_t cls = e.w & 7u;
    if (cls == C_GLOAD || cls == C_GSTORE) {
      const uint64_t d = (uint64_t)e.y + e.z;
      lm = d < lm ? d : lm;
    }
  }
  lm = uni64(wave_min_u64(lm));
  S.Lm = lm < kWindowMax ? lm : kWindowMax;
  for (uint32_t i = lane; i < S.nsm * S.sstride; i += 64) S.srv[i] = 0;
  for (uint32_t i = lane; i < S.nsm; i += 64) {
    S.resident[i] = 0;
    S.rq_cnt[i] = 0;
    S.mq_lh[i] = 0;
    S.mq_nl[i] = 0;
    S.mq_gh[i] = 0;
    S.mq_ng[i] = 0;
    S.dstart[i] = 0;
    S.dcnt[i] = 0;
  }
  if (lane == 0) {
    *S.ret_cnt = 0;
    *S.ret_min = 0xFFFFFFFFu;
  }
  for (uint32_t c = lane; c < S.G.n_ctas; c += 64) {
    const CtaDev cd = S.G.ctas[c];
    if (cd.root_count & kCtaShared)
      for (uint32_t i = 0; i < cd.node_count; ++i)
        S.state[cd.node_begin + i] = (uint64_t)S.G.indeg[cd.node_begin + i];
  }
  mem_wait();
  __syncthreads();

  S.next_cta = 0;
  S.retired = 0;
  S.cur_k = 0;
  S.kstart_k = 0;
  S.kstart_t = 0;
  S.kstart_valid = 0;
  S.l2_av = 0;
  S.dram_av = 0;
  S.digest = 0;
  S.makespan = 0;
  S.nfin = 0;
  S.bad = 0;
  S.st_windows = S.st_iters = S.st_local = S.st_mem = S.st_retires = S.st_maxm = 0;
  S.st_maxrq = S.st_maxmq = S.st_maxret = 0;
  S.tm0 = S.tm1 = S.tm2 = S.tm3 = S.tm4 = S.tm5 = 0;

  S.dispatch(0);
  mem_wait();
  wsync();
  while (!__ballot(S.bad != 0)) {
    const uint64_t c0 = __builtin_amdgcn_s_memtime();
    // T: earliest pending event
    uint64_t tmin = kNoKey;
    for (uint32_t j = 0; j < S.nslot; ++j) {
      const uint32_t s = lane + 64u * j;
      if (s < S.nsm) {
        const uint32_t n = S.rq_n(s);
        for (uint32_t i = 0; i < n; ++i) {
          const uint64_t k = S.rq_get(s, i) >> 32;
          tmin = k < tmin ? k : tmin;
        }
        if (S.mq_nl[s]) {
          const uint64_t k = S.mq_lk[S.mq_lh[s] * S.NS + s] >> 32;
          tmin = k < tmin ? k : tmin;
        }
      }
    }
    const uint32_t rmin = uni(*S.ret_min);
    if (*S.ret_cnt) tmin = rmin < tmin ? rmin : tmin;
    const uint64_t T = uni64(wave_min_u64(tmin));
    if (T == kNoKey) break;
    uint64_t H0 = T + S.Lm;
    const uint32_t Wb = (uint32_t)(H0 - T);  // bucket range (H0 may be lowered below)
    const uint64_t c1 = __builtin_amdgcn_s_memtime();

    // Retirement phase: retirements below H0, in cycle order, each distinct
    // cycle followed by dispatch.  More than memcap of them lower H0.
    if (rmin < H0 && uni(*S.ret_cnt)) {
      const uint32_t n = min(uni(*S.ret_cnt), kRetireCap);
      uint32_t D = wave_sum_u32(S.count_ret(H0, n));
      if (D > S.memcap) {
        uint64_t lo = T + 1, hi = H0;
        while (hi - lo > 1) {
          const uint64_t mid = (lo + hi) / 2;
          if (wave_sum_u32(S.count_ret(mid, n)) <= S.memcap)
            lo = mid;
          else
            hi = mid;
        }
        H0 = lo;
        D = wave_sum_u32(S.count_ret(H0, n));
        if (D > S.memcap) S.bad |= kBadWindow;
      }
      if (__ballot(S.bad != 0)) break;
      // compact in place, 64 entries at a time: due ones to w_key0, the rest
      // to the front of the list
      uint32_t dp = 0, kp = 0, kmin = 0xFFFFFFFFu;
      for (uint32_t base = 0; base < n; base += 64) {
        const uint32_t i = base + lane;
        const uint64_t k = i < n ? S.ret_get(i) : kNoKey;
        const bool due = i < n && (k >> 32) < H0;
        const bool keep = i < n && !due;
        const uint64_t bd = __ballot(due), bk = __ballot(keep);
        if (due) S.w_key0[dp + lanes_below(bd, lane)] = k;
        if (keep) {
          S.ret_set(kp + lanes_below(bk, lane), k);
          kmin = (uint32_t)(k >> 32) < kmin ? (uint32_t)(k >> 32) : kmin;
        }
        dp += (uint32_t)__popcll(bd);
        kp += (uint32_t)__popcll(bk);
      }
      kmin = (uint32_t)uni64(wave_min_u64(kmin));
      wsync();
      if (lane == 0) {
        *S.ret_cnt = kp;
        *S.ret_min = kmin;
      }
      wsync();
      const uint32_t R = dp;
      if (R) {
        S.csort(R, T, Wb, false);
        bool stop = false;
        for (uint32_t i = 0; i < R && !stop;) {
          const uint64_t r = uni64(S.s_key[i] >> 32);
          uint32_t j = i;
          while (j < R && uni64(S.s_key[j] >> 32) == r) ++j;
          for (uint32_t x = i + lane; x < j; x += 64) atomicSub(&S.resident[(uint32_t)S.s_key[x]], 1u);
          wsync();
          S.retired += j - i;
          S.st_retires += j - i;
          S.dispatch((uint32_t)r);
          i = j;
          stop = __ballot(S.bad != 0) != 0;
        }
        mem_wait();
        wsync();
        if (__ballot(S.bad != 0)) break;
      }
    }
    const uint64_t c2 = __builtin_amdgcn_s_memtime();

    // Local phase.
    for (;;) {
      ++S.st_iters;
      bool worked = false;
      for (uint32_t g0 = 0; g0 < S.nslot; g0 += NB) worked |= S.local_batch(g0, H0);
      if (!worked) break;
    }
    mem_wait();
    wsync();
    const uint64_t c3 = __builtin_amdgcn_s_memtime();
    if (__ballot(S.bad != 0)) break;

    // Memory phase: the arrivals below H (H <= H0, lowered if they do not fit).
    uint64_t H = H0;
    uint32_t mine = S.count_due(H);
    uint32_t M = wave_sum_u32(mine);
    if (M > S.memcap) {  // keep the prefix, in cycle order, that fits
      uint64_t lo = T + 1, hi = H;
      while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) / 2;
        if (wave_sum_u32(S.count_due(mid)) <= S.memcap)
          lo = mid;
        else
          hi = mid;
      }
      H = lo;
      mine = S.count_due(H);
      M = wave_sum_u32(mine);
      if (M > S.memcap) S.bad |= kBadWindow;
    }
    if (__ballot(S.bad != 0)) break;
    {
      uint32_t p = wave_excl_scan_u32(mine, lane);
      for (uint32_t j = 0; j < S.nslot; ++j) {
        const uint32_t s = lane + 64u * j;
        if (s < S.nsm) {
          S.dstart[s] = p;
          const uint32_t p0 = p;
          while (S.mq_nl[s] && (S.mq_lk[S.mq_lh[s] * S.NS + s] >> 32) < H) {
            uint64_t key;
            uint32_t op;
            S.mq_pop(s, key, op);
            S.w_key0[p] = key;
            S.w_aux0[p] = op | (s << 16);
            ++p;
          }
          S.dcnt[s] = p - p0;
        }
      }
    }
    wsync();
    const uint64_t c4 = __builtin_amdgcn_s_memtime();
    uint64_t c5 = c4;
    if (M) {
      S.csort(M, T, Wb, true);
      c5 = __builtin_amdgcn_s_memtime();
      S.memory_phase(M);
    }
    mem_wait();
    wsync();
    const uint64_t c6 = __builtin_amdgcn_s_memtime();
    ++S.st_windows;
    S.st_mem += M;
    S.st_maxm = M > S.st_maxm ? M : S.st_maxm;
    S.tm0 += c1 - c0;
    S.tm1 += c2 - c1;
    S.tm2 += c3 - c2;
    S.tm3 += c4 - c3;
    S.tm4 += c5 - c4;
    S.tm5 += c6 - c5;
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
    stats[0] = S.st_windows;
    stats[1] = S.st_iters;
    stats[2] = nl;
    stats[3] = S.st_mem;
    stats[4] = S.st_retires;
    stats[5] = S.st_maxm;
    stats[6] = S.tm0;
    stats[7] = S.tm1;
    stats[8] = S.tm2;
    stats[9] = S.tm3;
    stats[10] = S.tm4;
    stats[11] = S.tm5;
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

hipError_t launch_window(const Launch& L, uint32_t lds_bytes, hipStream_t stream) {
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(gts_sim_window, dim3(L.B), dim3(64), lds_bytes, stream, L);
  return hipGetLastError();
}

}  // namespace gts
