// gts_window.hip — windowed simulation kernel for gfx950 (MI355X).
//
// One wavefront simulates one (graph, hardware record) pair, like the
// general kernel, but instead of taking one event at a time it advances the
// whole machine through time windows [T, H) in which the SMs cannot affect
// one another, with one lane per simulated SM (SM s on lane s mod 64):
//
//   T = the earliest pending event.  CTA retirements at T, then dispatch.
//   H = min(T + Lm, next retirement), Lm = the smallest possible delay from
//       a memory arrival to its completion (min over memory ops of L2/DRAM
//       occupancy + latency).
//   local phase:  every lane issues its SMs' ready nodes with cycle < H in
//       (cycle, node id) order: per-SM servers, node finish, release of
//       out-edges into the same CTA, memory nodes reserve their SM's engine
//       and queue an arrival at their engine start.
//   memory phase: the arrivals with cycle < H from all SMs are sorted by
//       (cycle, node id) in LDS and served by the chip-wide L2 and DRAM FIFO
//       servers through a max-plus prefix scan across the wave; completions
//       release their out-edges (global atomics: several arrivals of one
//       window may feed the same node) and retire CTAs.
//
// Why this equals the one-event-at-a-time order (the general kernel and the
// CPU oracle): within [T, H) an SM's issue decisions depend only on its own
// servers and on releases from its own CTAs; a memory arrival at s >= T
// completes no earlier than s + Lm >= H, so none of this window's arrivals
// can release anything inside the window; and a CTA can only retire when its
// last node completes, which for the graphs this kernel accepts is always a
// memory node (every node without a successor in its CTA is a global load or
// store) and therefore at or after H.  Edges between CTAs must leave a memory
// node and be released at its completion, for the same reason.  The host
// sends other graphs, and any simulation whose queues overflow, to the
// general kernel.
#include <hip/hip_runtime.h>

#include "../../include/gts.h"
#include "gts_common.h"
#include "gts_dev.h"

namespace gts {

namespace {

constexpr uint64_t kNoKey = ~0ull;
constexpr uint32_t kBadOverflow = 1u, kBadCapacity = 2u;

// Node state of the windowed kernel: remaining in-edges (low word, counts
// down from the in-degree) | latest release cycle (high word).
__device__ __forceinline__ uint32_t* st_rem(uint64_t* st) { return reinterpret_cast<uint32_t*>(st); }
__device__ __forceinline__ uint32_t* st_acc(uint64_t* st) { return reinterpret_cast<uint32_t*>(st) + 1; }

// Loads of words that global atomics may have changed bypass the L1.
template <typename T>
__device__ __forceinline__ T gld(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void mem_wait() { __builtin_amdgcn_s_waitcnt(0); }

struct Compose {  // f(x) = max(x, a) + o on int64
  int64_t a, o;
};
__device__ __forceinline__ Compose compose(Compose f, Compose g) {  // g after f
  const int64_t ga = g.a - f.o;
  return Compose{f.a > ga ? f.a : ga, f.o + g.o};
}
__device__ __forceinline__ Compose shfl_up_c(Compose c, uint32_t d) {
  Compose r;
  r.a = __shfl_up(c.a, d, 64);
  r.o = __shfl_up(c.o, d, 64);
  return r;
}

struct WSim {
  Image G;
  const uint32_t* hw;
  uint32_t b, lane, flags, nsm, nsub, sstride, nslot, memcap;
  // LDS
  uint4* optab;
  uint32_t* srv;        // [nsm][nsub + 2]
  uint32_t* resident;   // [nsm]
  uint32_t* rq_cnt;     // [nsm]
  uint32_t* mq_head;    // [nsm]
  uint32_t* mq_tail;    // [nsm]
  uint32_t* wcount;     // [1]
  uint64_t* wkey;       // [memcap rounded to a power of two]
  uint32_t* wsm;        // [same]
  // per-simulation scratch
  uint64_t* state;      // [N]
  CtaState* cst;        // [C]
  uint64_t* rq;         // [kQueueReady][nsm]
  uint64_t* mq;         // [kQueueMem][nsm]
  uint32_t* out_cycles;
  // uniform control
  uint32_t next_cta, retired, cur_k, kstart_k, kstart_t, kstart_valid;
  uint64_t l2_av, dram_av;
  uint64_t Lm;
  // per lane
  uint64_t digest;
  uint32_t makespan, nfin, bad;
  // statistics (written to the end of the simulation's scratch slice)
  uint64_t st_windows, st_iters, st_local, st_mem, st_retires, st_maxm;
  uint64_t tm[6];

  __device__ void push_rq(uint32_t s, uint64_t key) {
    const uint32_t slot = atomicAdd(&rq_cnt[s], 1u);
    if (slot < kQueueReady)
      rq[(uint64_t)slot * nsm + s] = key;
    else
      bad |= kBadCapacity;
  }

  __device__ void push_mq(uint32_t s, uint64_t key) {
    const uint32_t tail = mq_tail[s];
    if (tail - mq_head[s] >= kQueueMem) {
      bad |= kBadCapacity;
      return;
    }
    mq[(uint64_t)(tail % kQueueMem) * nsm + s] = key;
    mq_tail[s] = tail + 1;
  }

  __device__ void record(uint32_t v, uint64_t s, uint64_t f) {
    if (out_cycles) {
      uint64_t* o = reinterpret_cast<uint64_t*>(out_cycles) + ((uint64_t)b * G.n_nodes + v);
      *o = (f << 32) | s;
    }
    digest += mix64(((s << 32) | f) ^ mix64((uint64_t)v + 1));
    makespan = (uint32_t)f > makespan ? (uint32_t)f : makespan;
    ++nfin;
  }

  // Local phase: one lane, its own SM s.  Releases go to nodes of the same
  // CTA, which only this lane touches during the phase.
  __device__ void release_local(const NodeDev& rec, bool at_issue, uint64_t r, uint32_t s) {
    const bool ofin = (flags & GTS_ORDER_AT_FINISH) != 0;
    for (uint32_t e = rec.succ_begin; e < rec.succ_end; ++e) {
      const uint32_t ent = G.succ[e];
      const uint32_t bits = ent >> GTS_EDGE_KIND_SHIFT;
      if ((((bits & kDevOrder) != 0) && !ofin) != at_issue) continue;
      const uint32_t w = ent & GTS_EDGE_TARGET_MASK;
      const uint64_t sv = gld(&state[w]);
      const uint32_t rem = (uint32_t)sv - 1u;
      uint32_t acc = (uint32_t)(sv >> 32);
      acc = r > acc ? (uint32_t)r : acc;
      state[w] = ((uint64_t)acc << 32) | rem;
      if (rem == 0) push_rq(s, mkkey(acc, kEvReady, w));
    }
  }

  __device__ void cta_local(uint32_t c, uint64_t f) {
    const uint32_t left = gld(&cst[c].left);
    const uint32_t mf = gld(&cst[c].maxfin);
    cst[c].left = left - 1u;
    cst[c].maxfin = (uint32_t)f > mf ? (uint32_t)f : mf;
  }

  __device__ void issue_local(uint32_t s, uint32_t t, uint32_t v) {
    const NodeDev rec = G.nodes[v];
    const uint4 od = optab[rec.op_indeg & 0xFFFFu];
    const uint32_t cls = od.w & 7u;
    const bool nocont = (flags & GTS_NO_CONTENTION) != 0;
    uint32_t* S = srv + s * sstride;
    if (cls <= C_SFU) {
      const uint32_t lanes = (od.w >> 8) & 0xFFu;
      uint64_t st = t;
      if (!nocont)
        for (uint32_t l = 0; l < nsub; ++l)
          if ((lanes >> l) & 1u) st = S[l] > st ? S[l] : st;
      const uint64_t f = st + od.x + od.z;
      if (f > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      for (uint32_t l = 0; l < nsub; ++l)
        if ((lanes >> l) & 1u) S[l] = (uint32_t)(st + od.x);
      record(v, st, f);
      cta_local(rec.cta, f);
      release_local(rec, true, st + 1, s);
      release_local(rec, false, f, s);
    } else if (cls == C_SMEM) {
      const uint32_t a = S[nsub];
      const uint64_t st = nocont ? (uint64_t)t : (a > t ? a : t);
      const uint64_t f = st + od.x + od.z;
      if (f > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      S[nsub] = (uint32_t)(st + od.x);
      record(v, st, f);
      cta_local(rec.cta, f);
      release_local(rec, true, st + 1, s);
      release_local(rec, false, f, s);
    } else if (cls == C_SYNC) {
      const uint64_t f = (uint64_t)t + od.z;
      if (f > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      record(v, t, f);
      cta_local(rec.cta, f);
      release_local(rec, true, (uint64_t)t + 1, s);
      release_local(rec, false, f, s);
    } else {
      const uint32_t a = S[nsub + 1];
      const uint64_t st = nocont ? (uint64_t)t : (a > t ? a : t);
      if (st + od.x > kMaxCycle) {
        bad |= kBadOverflow;
        return;
      }
      S[nsub + 1] = (uint32_t)(st + od.x);
      release_local(rec, true, st + 1, s);
      push_mq(s, mkkey(st, kEvMem, v));
    }
  }

  // Wave-cooperative dispatch at cycle t (phase 2 of a step).
  __device__ void dispatch(uint32_t t) {
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
      if (lane == 0) {
        cst[c].sm = sm;
        cst[c].launch = (uint32_t)launch;
        cst[c].left = cd.node_count;
        cst[c].maxfin = 0u;
        resident[sm] += 1;
      }
      ++next_cta;
      for (uint32_t r0 = 0; r0 < cd.root_count; r0 += 64) {
        const uint32_t ri = r0 + lane;
        if (ri < cd.root_count) {
          const uint32_t v = G.roots[cd.root_begin + ri];
          const uint64_t sv = gld(&state[v]);
          if ((uint32_t)sv == 0) {
            const uint32_t acc = (uint32_t)(sv >> 32);
            push_rq(sm, mkkey(acc > launch ? acc : launch, kEvReady, v));
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

  // Bitonic sort of the window's arrivals (keys with their SM ids) in LDS.
  __device__ void sort_window(uint32_t M) {
    uint32_t n = 1;
    while (n < M) n <<= 1;
    for (uint32_t i = M + lane; i < n; i += 64) wkey[i] = kNoKey;
    __builtin_amdgcn_wave_barrier();
    for (uint32_t k = 2; k <= n; k <<= 1) {
      for (uint32_t j = k >> 1; j > 0; j >>= 1) {
        for (uint32_t i = lane; i < n; i += 64) {
          const uint32_t p = i ^ j;
          if (p > i) {
            const uint64_t a = wkey[i], c = wkey[p];
            const bool up = (i & k) == 0;
            if ((a > c) == up) {
              wkey[i] = c;
              wkey[p] = a;
              const uint32_t sa = wsm[i];
              wsm[i] = wsm[p];
              wsm[p] = sa;
            }
          }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      }
    }
  }

  // Memory phase for the M sorted arrivals: L2 / DRAM FIFO service in
  // (cycle, id) order as a max-plus scan, then completion and release.
  __device__ void memory_phase(uint32_t M) {
    const bool nocont = (flags & GTS_NO_CONTENTION) != 0;
    const bool ofin = (flags & GTS_ORDER_AT_FINISH) != 0;
    const uint32_t per = (M + 63) / 64;
    const uint32_t i0 = lane * per;
    const uint32_t i1 = i0 + per < M ? i0 + per : M;
    constexpr int64_t kNeg = -(int64_t(1) << 62);
    Compose fl2{kNeg, 0}, fdr{kNeg, 0};
    for (uint32_t i = i0; i < i1; ++i) {
      const uint32_t v = (uint32_t)wkey[i] & GTS_EDGE_TARGET_MASK;
      const uint4 od = optab[G.nodes[v].op_indeg & 0xFFFFu];
      const Compose g{(int64_t)(wkey[i] >> 32), (int64_t)od.y};
      if ((od.w >> 3) & 1u)
        fdr = compose(fdr, g);
      else
        fl2 = compose(fl2, g);
    }
    // inclusive scan of the per-lane compositions in lane order
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
    if (lane == 0) {
      el2 = Compose{kNeg, 0};
      edr = Compose{kNeg, 0};
    }
    const Compose tl2{__shfl(il2.a, 63, 64), __shfl(il2.o, 63, 64)};
    const Compose tdr{__shfl(idr.a, 63, 64), __shfl(idr.o, 63, 64)};
    int64_t xl2 = (int64_t)l2_av > el2.a ? (int64_t)l2_av : el2.a;
    xl2 += el2.o;
    int64_t xdr = (int64_t)dram_av > edr.a ? (int64_t)dram_av : edr.a;
    xdr += edr.o;
    if (!nocont) {
      int64_t nl2 = (int64_t)l2_av > tl2.a ? (int64_t)l2_av : tl2.a;
      int64_t ndr = (int64_t)dram_av > tdr.a ? (int64_t)dram_av : tdr.a;
      l2_av = (uint64_t)(nl2 + tl2.o);
      dram_av = (uint64_t)(ndr + tdr.o);
    }
    // completion, in lock step over each lane's run of arrivals
    for (uint32_t r = 0; r < per; ++r) {
      const uint32_t i = i0 + r;
      const bool act = i < i1;
      uint32_t v = 0, s = 0, c = 0;
      uint64_t f = 0;
      NodeDev rec{};
      if (act) {
        const uint64_t key = wkey[i];
        v = (uint32_t)key & GTS_EDGE_TARGET_MASK;
        s = wsm[i];
        rec = G.nodes[v];
        c = rec.cta;
        const uint4 od = optab[rec.op_indeg & 0xFFFFu];
        const uint64_t st = key >> 32;
        const bool dram = (od.w >> 3) & 1u;
        int64_t& x = dram ? xdr : xl2;
        const int64_t m = nocont ? (int64_t)st : (x > (int64_t)st ? x : (int64_t)st);
        x = m + (int64_t)od.y;
        const uint64_t e = st + od.x;
        const uint64_t mend = (uint64_t)m + od.y;
        f = (e > mend ? e : mend) + od.z;
        if (f > kMaxCycle) {
          bad |= kBadOverflow;
        } else {
          record(v, st, f);
          atomicMax(&cst[c].maxfin, (uint32_t)f);
        }
      }
      mem_wait();
      if (act && f <= kMaxCycle) {
        const uint32_t old = atomicSub(&cst[c].left, 1u);
        if (old == 1u) push_rq(s, mkkey(gld(&cst[c].maxfin), kEvRetire, c));
      }
      // release the arrival's completion edges
      const uint32_t nout = act && f <= kMaxCycle ? rec.succ_end - rec.succ_begin : 0u;
      const uint32_t maxout = uni((uint32_t)wave_max_u64(nout));
      for (uint32_t k = 0; k < maxout; ++k) {
        bool sel = false;
        uint32_t w = 0, bits = 0;
        if (k < nout) {
          const uint32_t ent = G.succ[rec.succ_begin + k];
          bits = ent >> GTS_EDGE_KIND_SHIFT;
          w = ent & GTS_EDGE_TARGET_MASK;
          sel = !((bits & kDevOrder) && !ofin);
          if (sel) atomicMax(st_acc(&state[w]), (uint32_t)f);
        }
        mem_wait();
        if (sel) {
          const uint32_t old = atomicSub(st_rem(&state[w]), 1u);
          if (old == 1u) {
            const uint32_t acc = gld(st_acc(&state[w]));
            if (bits & kDevCross) {
              const uint32_t cw = G.nodes[w].cta;
              if (cw < next_cta) {
                const uint32_t launch = gld(&cst[cw].launch);
                push_rq(gld(&cst[cw].sm), mkkey(acc > launch ? acc : launch, kEvReady, w));
              }
            } else {
              push_rq(s, mkkey(acc, kEvReady, w));
            }
          }
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
  S.nsm = S.hw[HW_NSM];
  S.nsub = S.hw[HW_NSUB];
  S.sstride = S.nsub + 2;
  S.nslot = (S.nsm + 63) / 64;
  S.memcap = L.memcap;
  const uint32_t lane = S.lane;
  uint8_t* sim = L.sims + (uint64_t)b * L.layout.stride;
  S.state = reinterpret_cast<uint64_t*>(sim + L.layout.off_state);
  S.cst = reinterpret_cast<CtaState*>(sim + L.layout.off_cta);
  S.rq = reinterpret_cast<uint64_t*>(sim + L.layout.off_rq);
  S.mq = reinterpret_cast<uint64_t*>(sim + L.layout.off_mq);
  // LDS carve-up (sizes from the batch maxima; the host sized the block)
  uint32_t* p = lds;
  S.optab = reinterpret_cast<uint4*>(p);
  p += 4u * S.G.n_ops;
  S.srv = p;
  p += L.max_nsm * (L.max_nsub + 2);
  S.resident = p;
  p += L.max_nsm;
  S.rq_cnt = p;
  p += L.max_nsm;
  S.mq_head = p;
  p += L.max_nsm;
  S.mq_tail = p;
  p += L.max_nsm;
  S.wcount = p;
  p += 1;
  p += (uintptr_t)p & 4u ? 1 : 0;  // 8-byte alignment for the keys
  S.wkey = reinterpret_cast<uint64_t*>(p);
  p += 2u * L.memcap;
  S.wsm = p;
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

  // Setup: duration table and Lm, idle servers, empty queues, node state.
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
  S.Lm = lm < (1ull << 33) ? lm : (1ull << 33);
  for (uint32_t i = lane; i < S.nsm * S.sstride; i += 64) S.srv[i] = 0;
  for (uint32_t i = lane; i < S.nsm; i += 64) {
    S.resident[i] = 0;
    S.rq_cnt[i] = 0;
    S.mq_head[i] = 0;
    S.mq_tail[i] = 0;
  }
  for (uint32_t v = lane; v < S.G.n_nodes; v += 64) S.state[v] = (uint64_t)(S.G.nodes[v].op_indeg >> 16);
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
  for (int i = 0; i < 6; ++i) S.tm[i] = 0;

  S.dispatch(0);
  mem_wait();
  __builtin_amdgcn_wave_barrier();
  while (!__ballot(S.bad != 0)) {
    const uint64_t c0 = __builtin_amdgcn_s_memtime();
    // T: earliest pending event of the machine
    uint64_t tmin = kNoKey;
    for (uint32_t j = 0; j < S.nslot; ++j) {
      const uint32_t s = lane + 64u * j;
      if (s < S.nsm) {
        const uint32_t n = min(S.rq_cnt[s], kQueueReady);
        for (uint32_t i = 0; i < n; ++i) {
          const uint64_t k = S.rq[(uint64_t)i * S.nsm + s] >> 32;
          tmin = k < tmin ? k : tmin;
        }
        if (S.mq_head[s] != S.mq_tail[s]) {
          const uint64_t k = S.mq[(uint64_t)(S.mq_head[s] % kQueueMem) * S.nsm + s] >> 32;
          tmin = k < tmin ? k : tmin;
        }
      }
    }
    const uint64_t T64 = uni64(wave_min_u64(tmin));
    if (T64 == kNoKey) break;
    const uint32_t T = (uint32_t)T64;
    const uint64_t H = T64 + S.Lm;
    const uint64_t c1 = __builtin_amdgcn_s_memtime();
    // Retirement phase: every CTA retirement with cycle < H, in cycle order,
    // each distinct cycle followed by dispatch.  Retirements and dispatch
    // depend only on earlier retirements and dispatches, and every
    // retirement that can fall before H is already known (a CTA completes
    // with a memory arrival, whose completion is at least Lm later).
    if (lane == 0) *S.wcount = 0;
    __builtin_amdgcn_wave_barrier();
    for (uint32_t j = 0; j < S.nslot; ++j) {
      const uint32_t s = lane + 64u * j;
      if (s < S.nsm) {
        uint32_t n = min(S.rq_cnt[s], kQueueReady);
        for (uint32_t i = 0; i < n;) {
          const uint64_t k = S.rq[(uint64_t)i * S.nsm + s];
          if (((k >> 30) & 3u) == kEvRetire && (k >> 32) < H) {
            S.rq[(uint64_t)i * S.nsm + s] = S.rq[(uint64_t)(n - 1) * S.nsm + s];
            --n;
            const uint32_t slot = atomicAdd(S.wcount, 1u);
            if (slot < S.memcap) {
              S.wkey[slot] = k;
              S.wsm[slot] = s;
            } else {
              S.bad |= kBadCapacity;
            }
            continue;
          }
          ++i;
        }
        S.rq_cnt[s] = n;
      }
    }
    __builtin_amdgcn_wave_barrier();
    if (__ballot(S.bad != 0)) break;
    const uint32_t R = uni(*S.wcount);
    if (R) {
      S.sort_window(R);
      for (uint32_t i = 0; i < R;) {
        const uint64_t r = uni64(S.wkey[i] >> 32);
        uint32_t j = i;
        while (j < R && uni64(S.wkey[j] >> 32) == r) {
          if (lane == 0) S.resident[S.wsm[j]] -= 1;
          ++j;
        }
        __builtin_amdgcn_wave_barrier();
        S.retired += j - i;
        S.st_retires += j - i;
        S.dispatch((uint32_t)r);
        i = j;
        if (__ballot(S.bad != 0)) break;
      }
      mem_wait();
      __builtin_amdgcn_wave_barrier();
      if (__ballot(S.bad != 0)) break;
    }
    const uint64_t c2 = __builtin_amdgcn_s_memtime();
    // local phase: each lane issues its SMs' ready nodes with cycle < H
    for (;;) {
      ++S.st_iters;
      bool worked = false;
      for (uint32_t j = 0; j < S.nslot; ++j) {
        const uint32_t s = lane + 64u * j;
        if (s < S.nsm && !S.bad) {
          const uint32_t n = min(S.rq_cnt[s], kQueueReady);
          uint64_t best = kNoKey;
          uint32_t bi = 0;
          for (uint32_t i = 0; i < n; ++i) {
            const uint64_t k = S.rq[(uint64_t)i * S.nsm + s];
            if (((k >> 30) & 3u) == kEvReady && k < best) {
              best = k;
              bi = i;
            }
          }
          if (best != kNoKey && (best >> 32) < H) {
            S.rq[(uint64_t)bi * S.nsm + s] = S.rq[(uint64_t)(n - 1) * S.nsm + s];
            S.rq_cnt[s] = n - 1;
            S.issue_local(s, (uint32_t)(best >> 32), (uint32_t)best & GTS_EDGE_TARGET_MASK);
            ++S.st_local;
            worked = true;
          }
        }
      }
      if (!__ballot(worked)) break;
    }
    mem_wait();
    const uint64_t c3 = __builtin_amdgcn_s_memtime();
    if (__ballot(S.bad != 0)) break;
    // memory phase: gather the arrivals with cycle < H
    if (lane == 0) *S.wcount = 0;
    __builtin_amdgcn_wave_barrier();
    for (uint32_t j = 0; j < S.nslot; ++j) {
      const uint32_t s = lane + 64u * j;
      if (s < S.nsm) {
        uint32_t h = S.mq_head[s];
        const uint32_t tl = S.mq_tail[s];
        while (h != tl) {
          const uint64_t k = S.mq[(uint64_t)(h % kQueueMem) * S.nsm + s];
          if ((k >> 32) >= H) break;
          const uint32_t slot = atomicAdd(S.wcount, 1u);
          if (slot >= S.memcap) {
            S.bad |= kBadCapacity;
            break;
          }
          S.wkey[slot] = k;
          S.wsm[slot] = s;
          ++h;
        }
        S.mq_head[s] = h;
      }
    }
    __builtin_amdgcn_wave_barrier();
    if (__ballot(S.bad != 0)) break;
    const uint32_t M = uni(*S.wcount);
    const uint64_t c4 = __builtin_amdgcn_s_memtime();
    uint64_t c5 = c4;
    if (M) {
      S.sort_window(M);
      c5 = __builtin_amdgcn_s_memtime();
      S.memory_phase(M);
    }
    mem_wait();
    const uint64_t c6 = __builtin_amdgcn_s_memtime();
    ++S.st_windows;
    S.st_mem += M;
    S.st_maxm = M > S.st_maxm ? M : S.st_maxm;
    S.tm[0] += c1 - c0;
    S.tm[1] += c2 - c1;
    S.tm[2] += c3 - c2;
    S.tm[3] += c4 - c3;
    S.tm[4] += c5 - c4;
    S.tm[5] += c6 - c5;
  }

  // reductions and status
  const uint64_t bad_any = __ballot(S.bad != 0);
  const uint64_t ovf_any = __ballot((S.bad & kBadOverflow) != 0);
  uint64_t dg = S.digest;
  uint64_t mk = S.makespan;
  uint64_t nf = S.nfin;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    dg += __shfl_xor(dg, o, 64);
    const uint64_t om = __shfl_xor(mk, o, 64);
    mk = om > mk ? om : mk;
    nf += __shfl_xor(nf, o, 64);
  }
  uint64_t nl = S.st_local;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) nl += __shfl_xor(nl, o, 64);
  if (lane == 0) {
    uint64_t* stats = reinterpret_cast<uint64_t*>(sim + L.layout.stride - kStatsBytes);
    const uint64_t vals[12] = {S.st_windows, S.st_iters, nl, S.st_mem, S.st_retires, S.st_maxm,
                               S.tm[0], S.tm[1], S.tm[2], S.tm[3], S.tm[4], S.tm[5]};
    for (int i = 0; i < 12; ++i) stats[i] = vals[i];
  }
  if (lane == 0) {
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
