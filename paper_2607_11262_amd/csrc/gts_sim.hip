// gts_sim.hip — batched tile-graph simulation kernels for gfx950 (MI355X).
//
// One wavefront (one 64-thread block) simulates one (graph, hardware record)
// pair.  The wave walks the simulation's events in (cycle, phase, node id)
// order; the 64 lanes share the work inside each step: the minimum search
// over pending events, the release of a node's out-edges (one lane per
// edge), the search for the SM with the most free slots, the scan of a
// dispatched CTA's root nodes, and appending newly ready nodes (ballot +
// prefix count).  Per-SM server state and the per-op duration table live in
// LDS; per-node and per-CTA state live in the simulation's scratch slice.
//
// Timing rules (GTSim Sec. 5.1-5.3, readings fixed where the paper is
// silent; the CPU oracle states the same rules independently):
//  * servers: per subpartition of each SM one lane for each compute class
//    (tensor / CUDA-core / SFU pipelines; lane of warp w = w mod n_subpart),
//    one shared-memory pipe and one
//    global-memory engine per SM, one chip-wide L2 and one DRAM server; all
//    FIFO, non-preemptive, "available at cycle a";
//  * durations: occ = max(1, ceil(work * 2^16 * n_subpart / (k * rate_q16)))
//    on k lanes; SMEM / engine / L2 / DRAM occ = max(1, ceil(work * 2^16 /
//    rate_q16)); finish = start + occ + latency; a SYNC node lasts
//    max(1, latency);
//  * one step per distinct event cycle t: CTA retirements, then dispatch
//    (pending CTAs in index order to the SM with most free slots, lowest id
//    on ties; a kernel starts after the previous one has fully retired),
//    then node issue in id order (a memory node reserves its engine and
//    arrives at the L2/DRAM queue at its engine start), then memory
//    arrivals in id order: m = max(t, avail), finish = max(start + occ_e,
//    m + occ_m) + latency;
//  * release: ORDER edges at start + 1 (issue time), DATA / SYNC edges at
//    finish (completion); a node becomes ready at the latest release of its
//    in-edges, not before its CTA's launch;
//  * clusters (Sec. 5.2 DSMEM): a kernel's clusters of consecutive CTAs are
//    dispatched whole onto the first NoC domain and placement slot (strips
//    of nodes, or compact blocks on a mesh) whose SMs all have a free slot;
//    a REMOTE node reserves every server of its route (crossbar injection
//    and ejection ports, or the mesh links of the XY route) at once:
//    start = max(t, their availability), finish = start + occ + latency
//    (once per hop on a mesh);
//  * LRU L2 (tiles): a load / store that names its tile, on a machine with
//    an L2 capacity, hits iff the tile was touched before and its lines plus
//    the distinct lines of other tiles touched since fit, else goes to DRAM;
//    the tile then becomes the most recent;
//  * transaction-level memory (Sec. 5.2, 5.3): a load / store with a tile
//    address holds its engine for its n distinct 128-B lines; transaction j
//    enters at e_j = s + ceil(j * 128 * 2^16 / rate_gmem), arrives at the L2
//    then (memory events in (cycle, node id, j) order), is a hit iff its line
//    is among the l2_lines most recent (an LRU of lines; without a capacity
//    the op's MISS flag decides) and is served FIFO for ceil(128 * 2^32 /
//    rate) units of 2^-16 cycle (server time is kept in those units; a
//    whole-cycle node starts at the first whole cycle after): finish_j =
//    max(e_(j+1), ceil((m_j + q) / 2^16)) + latency; the node completes at
//    its largest finish_j, when its last transaction arrives.
#include <hip/hip_runtime.h>

#include "../../include/gts.h"
#include "gts_dev.h"
#include "gts_common.h"

namespace gts {

namespace {

struct Sim {
  // graph and launch
  Image G;
  const uint32_t* hw;
  uint32_t b, lane, flags, nsm, nsub, sstride;
  // storage
  uint4* optab;
  uint32_t smem_w;      // server word of the shared-memory pipe (the engine follows)
  uint32_t* srv;        // [nsm][sstride]: compute lanes, smem pipe, memory engine
  uint32_t* resident;   // [nsm]
  uint32_t* noc;        // [domains][noc_d][4]: crossbar ports / mesh links
  uint32_t noc_d, noc_w, noc_map;
  // LRU L2 state (scratch): each tile's latest access stamp (1-based count
  // of tile accesses, 0 = never) and a Fenwick tree over stamps holding, at
  // each tile's latest stamp, that tile's line count
  uint32_t* lru_last;   // [keys]: tiles, or the lines of addressed tiles, numbered densely at upload
  uint64_t* lru_bit;    // [accesses + 1], entry 0 unused
  uint32_t lru_now, l2_lines, lru_acc;  // lru_acc: bound on this simulation's accesses
  uint64_t lru_total;   // lines of all distinct tiles touched so far
  uint64_t* state;      // [N]
  CtaState* cst;        // [C]
  uint64_t* pkey;       // [cap]
  uint32_t* paux;       // [cap]
  uint32_t* out_cycles;
  // uniform control state
  uint32_t npend, next_cta, retired, cur_k, kstart_k, kstart_t, kstart_valid;
  uint32_t run_kb, run_cl;  // first CTA and cluster size of the kernel whose CTAs are live
  uint64_t l2_av, dram_av;  // chip-wide servers' availability, in 2^-16 cycles
  uint64_t digest;
  uint32_t makespan, nfin, overflow;

  __device__ void push_one(uint64_t key, uint32_t aux) {
    if (lane == 0) {
      pst(&pkey[npend], key);
      pst(&paux[npend], aux);
    }
    ++npend;
  }

  __device__ void push_lanes(bool flag, uint64_t key, uint32_t aux) {
    const uint64_t m = __ballot(flag);
    if (flag) {
      const uint32_t pos = npend + lanes_below(m, lane);
      pst(&pkey[pos], key);
      pst(&paux[pos], aux);
    }
    npend += (uint32_t)__popcll(m);
  }

  // Release the out-edges of a node selected by `which`: 0 = ORDER edges
  // released at issue, 1 = every other edge, released at completion.
  static_assert(kInlineSucc == 3, "release reads the record's three inline successor copies");
  __device__ void release(uint32_t v, const NodeDev& rec, uint32_t which, uint64_t r, uint32_t src_cta,
                          uint32_t src_sm) {
    const bool ofin = (flags & GTS_ORDER_AT_FINISH) != 0;
    const uint32_t deg = rec.op_nsucc >> 16;
    const uint32_t n = deg < 0xFFFFu ? deg : G.nodes[v + 1].succ_begin - rec.succ_begin;
    for (uint32_t e0 = 0; e0 < n; e0 += 64) {
      const uint32_t e = e0 + lane;
      const bool active = e < n;
      // the first successors and their in-degrees are copied into the record
      uint32_t ent = 0;
      if (active)
        ent = e == 0 ? rec.succ[0] : e == 1 ? rec.succ[1] : e == 2 ? rec.succ[2] : G.succ[rec.succ_begin + e];
      const uint32_t kind = ent >> GTS_EDGE_KIND_SHIFT;
      const uint32_t w = ent & GTS_EDGE_TARGET_MASK;
      const bool at_issue = (kind & kDevOrder) && !ofin;
      const bool sel = active && (at_issue == (which == 0));
      bool ready = false;
      uint64_t key = 0;
      uint32_t aux = 0;
      if (sel) {
        const uint64_t s = pld(&state[w]);
        const uint32_t nr_indeg = e == 0   ? (uint32_t)rec.sindeg[0]
                                  : e == 1 ? (uint32_t)rec.sindeg[1]
                                  : e == 2 ? (uint32_t)rec.sindeg[2]
                                           : (uint32_t)G.indeg[w];
        // an edge into a node without cross-CTA in-edges stays in the source's CTA
        const uint32_t nr_cta = (kind & kDevShared) ? G.nodes[w].cta : src_cta;
        uint32_t acc = (uint32_t)s;
        const uint32_t cnt = (uint32_t)(s >> 32) + 1;
        acc = r > acc ? (uint32_t)r : acc;
        pst(&state[w], ((uint64_t)cnt << 32) | acc);
        if (cnt == nr_indeg && nr_cta < next_cta) {
          uint32_t launch = 0, sm = src_sm;
          if (nr_cta != src_cta) {
            launch = pld(&cst[nr_cta].launch);
            sm = pld(&cst[nr_cta].sm);
          }
          ready = true;
          key = mkkey(acc > launch ? acc : launch, kEvReady, w);
          aux = sm;
        }
      }
      push_lanes(ready, key, aux);
    }
  }

  // Record (start, finish) of node v; CTA bookkeeping; false on overflow.
  __device__ bool complete(uint32_t v, const NodeDev& rec, uint64_t s, uint64_t f, uint32_t sm) {
    if (f > kMaxCycle) {
      overflow = 1;
      return false;
    }
    if (out_cycles && lane == 0) {
      uint64_t* o = reinterpret_cast<uint64_t*>(out_cycles) + ((uint64_t)b * G.n_nodes + v);
      *o = ((uint64_t)(uint32_t)f << 32) | (uint32_t)s;
    }
    digest += mix64(((s << 32) | f) ^ mix64((uint64_t)v + 1));
    makespan = (uint32_t)f > makespan ? (uint32_t)f : makespan;
    ++nfin;
    const uint32_t c = rec.cta;
    uint32_t left = pld(&cst[c].left) - 1;
    uint32_t mf = pld(&cst[c].maxfin);
    mf = (uint32_t)f > mf ? (uint32_t)f : mf;
    left = uni(left);
    mf = uni(mf);
    if (lane == 0) {
      pst(&cst[c].left, left);
      pst(&cst[c].maxfin, mf);
    }
    if (left == 0) push_one(mkkey(mf, kEvRetire, c), sm);
    return true;
  }

  // Node of rank r in placement slot j of a NoC domain, or -1 when the
  // placement list has no slot j: strips of consecutive nodes, on a mesh
  // with the compact mapping the most square blocks that tile it, or with
  // the strided mapping ranks noc_d / cl nodes apart.
  __device__ int32_t slot_node(uint32_t cl, uint32_t j, uint32_t r) const {
    if (noc_map == 1 && noc_w > 0) {
      const uint32_t rows = noc_d / noc_w;
      uint32_t bh = 0;
      for (uint32_t h = 1; h * h <= cl; ++h)
        if (cl % h == 0 && noc_w % (cl / h) == 0 && rows % h == 0) bh = h;
      if (bh) {
        const uint32_t bw = cl / bh, nbx = noc_w / bw;
        if (j >= nbx * (rows / bh)) return -1;
        return (int32_t)(((j / nbx) * bh + r / bw) * noc_w + (j % nbx) * bw + r % bw);
      }
    }
    if (j >= noc_d / cl) return -1;
    return noc_map == 2 ? (int32_t)(j + r * (noc_d / cl)) : (int32_t)(j * cl + r);
  }

  // First placement, domain by domain and slot by slot, whose SMs all exist
  // (and, with `slots`, all have a free slot); lane r < cl gets rank r's SM.
  __device__ bool place(uint32_t cl, uint64_t slots, bool need_free, uint32_t& mysm) const {
    const uint32_t ndom = (nsm + noc_d - 1) / noc_d;
    const uint64_t want = cl >= 64 ? ~0ull : ((1ull << cl) - 1ull);
    for (uint32_t d = 0; d < ndom; ++d)
      for (uint32_t j = 0; slot_node(cl, j, 0) >= 0; ++j) {
        bool ok = false;
        uint32_t s = 0;
        if (lane < cl) {
          s = d * noc_d + (uint32_t)slot_node(cl, j, lane);
          ok = s < nsm && (!need_free || resident[s] < slots);
        }
        if ((__ballot(ok) & want) == want) {
          mysm = s;
          return true;
        }
      }
    return false;
  }

  __device__ void push_roots(uint32_t c, const CtaDev& cd, uint64_t launch, uint32_t sm) {
    const uint32_t nroots = cd.root_count & ~kCtaShared;
    for (uint32_t r0 = 0; r0 < nroots; r0 += 64) {
      const uint32_t ri = r0 + lane;
      bool ready = false;
      uint64_t key = 0;
      if (ri < nroots) {
        const uint32_t v = G.roots[cd.root_begin + ri];
        const uint64_t s = pld(&state[v]);
        const uint32_t indeg = G.indeg[v];
        if ((uint32_t)(s >> 32) == indeg) {
          const uint32_t acc = (uint32_t)s;
          ready = true;
          key = mkkey(acc > launch ? acc : launch, kEvReady, v);
        }
      }
      push_lanes(ready, key, sm);
    }
  }

  __device__ void dispatch(uint32_t t) {
    while (next_cta < G.n_ctas && !overflow) {
      while (next_cta >= G.kernels[cur_k].cta_end) ++cur_k;
      const KernelDev kd = G.kernels[cur_k];
      if (retired < kd.cta_begin) return;  // the previous kernel is still running
      const uint64_t slots = kernel_slots(kd, hw);
      const uint32_t cl = kd.cluster & 0xFFFFu;
      run_kb = kd.cta_begin;
      run_cl = cl;
      if (cl > 1) {  // a whole cluster onto the first placement with room
        uint32_t mysm = 0;
        if (!place(cl, slots, true, mysm)) return;
        if (!kstart_valid || kstart_k != cur_k) {
          kstart_valid = 1;
          kstart_k = cur_k;
          kstart_t = t;
        }
        const uint64_t launch = (uint64_t)t + hw[HW_CTALAT] + (kstart_t == t ? hw[HW_KLAT] : 0u);
        if (launch > kMaxCycle) {
          overflow = 1;
          return;
        }
        const uint32_t c0 = next_cta;
        if (lane < cl) {
          pst(&cst[c0 + lane].sm, mysm);
          pst(&cst[c0 + lane].launch, (uint32_t)launch);
          pst(&cst[c0 + lane].left, G.ctas[c0 + lane].node_count);
          pst(&cst[c0 + lane].maxfin, 0u);
          resident[mysm] += 1;  // distinct SMs
        }
        next_cta += cl;
        for (uint32_t r = 0; r < cl; ++r) {
          const CtaDev cd = G.ctas[c0 + r];
          push_roots(c0 + r, cd, launch, (uint32_t)__shfl((int)mysm, (int)r, 64));
        }
        __builtin_amdgcn_wave_barrier();
        continue;
      }
      uint64_t best = 0;
      for (uint32_t m = lane; m < nsm; m += 64) {
        const uint64_t fr = slots - resident[m];
        const uint64_t k = (fr << 32) | (0xFFFFFFFFu - m);
        best = k > best ? k : best;
      }
      best = uni64(wave_max_u64(best));
      if ((best >> 32) == 0) return;  // every SM is full
      const uint32_t sm = 0xFFFFFFFFu - (uint32_t)best;
      if (!kstart_valid || kstart_k != cur_k) {
        kstart_valid = 1;
        kstart_k = cur_k;
        kstart_t = t;
      }
      uint64_t launch = (uint64_t)t + hw[HW_CTALAT] + (kstart_t == t ? hw[HW_KLAT] : 0u);
      if (launch > kMaxCycle) {
        overflow = 1;
        return;
      }
      const uint32_t c = next_cta;
      const CtaDev cd = G.ctas[c];
      if (lane == 0) {
        pst(&cst[c].sm, sm);
        pst(&cst[c].launch, (uint32_t)launch);
        pst(&cst[c].left, cd.node_count);
        pst(&cst[c].maxfin, 0u);
        resident[sm] += 1;
      }
      ++next_cta;
      push_roots(c, cd, launch, sm);
      __builtin_amdgcn_wave_barrier();
    }
  }

  __device__ void issue(uint32_t v, uint32_t t, uint32_t sm) {
    const NodeDev rec = G.nodes[v];
    const uint4 od = optab[rec.op_nsucc & 0xFFFFu];
    const uint32_t cls = od.w & 7u;
    const bool nocont = (flags & GTS_NO_CONTENTION) != 0;
    uint32_t* S = srv + sm * sstride;
    if (cls <= C_SFU) {
      const uint32_t lanes = (od.w >> 8) & 0xFFu;
      S += od.w >> 16;  // this class's lanes
      uint32_t a = 0;
      if (!nocont && lane < nsub && ((lanes >> lane) & 1u)) a = S[lane];
      uint64_t s = (uint64_t)t;
      if (!nocont) {
        uint64_t m = wave_max_u64(a);
        m = uni64(m);
        s = m > s ? m : s;
      }
      const uint64_t f = s + od.x + od.z;
      if (!complete(v, rec, s, f, sm)) return;
      if (lane < nsub && ((lanes >> lane) & 1u)) S[lane] = (uint32_t)(s + od.x);
      release(v, rec, 0, s + 1, rec.cta, sm);
      release(v, rec, 1, f, rec.cta, sm);
    } else if (cls == C_SMEM) {
      const uint32_t a = S[smem_w];
      const uint64_t s = nocont ? (uint64_t)t : (a > t ? a : t);
      const uint64_t f = s + od.x + od.z;
      if (!complete(v, rec, s, f, sm)) return;
      if (lane == 0) S[smem_w] = (uint32_t)(s + od.x);
      release(v, rec, 0, s + 1, rec.cta, sm);
      release(v, rec, 1, f, rec.cta, sm);
    } else if (cls == C_SYNC) {
      const uint64_t f = (uint64_t)t + od.z;
      if (!complete(v, rec, t, f, sm)) return;
      release(v, rec, 0, (uint64_t)t + 1, rec.cta, sm);
      release(v, rec, 1, f, rec.cta, sm);
    } else if (cls == C_REMOTE) {
      // the target CTA (same cluster) and the route between the two SMs'
      // nodes of their NoC domain; lane i holds route server i
      const uint32_t c = rec.cta;
      const uint32_t tgt = run_kb + (c - run_kb) / run_cl * run_cl + ((od.w >> 16) & 0xFu);
      const uint32_t tsm = uni(pld(&cst[tgt].sm));
      const uint32_t dom = sm / noc_d, a = sm % noc_d, bn = tsm % noc_d;
      uint32_t* dav = noc + dom * noc_d * 4u;
      uint32_t nr, idx = 0;
      uint64_t lat = od.z;
      if (noc_w == 0) {  // crossbar: injection port of a, ejection port of b
        nr = 2;
        idx = lane == 0 ? a * 4u : bn * 4u + 1u;
      } else {           // mesh: x links first, then y links
        const int32_t xa = (int32_t)(a % noc_w), ya = (int32_t)(a / noc_w);
        const int32_t xb = (int32_t)(bn % noc_w), yb = (int32_t)(bn / noc_w);
        const uint32_t dx = (uint32_t)(xb > xa ? xb - xa : xa - xb), dy = (uint32_t)(yb > ya ? yb - ya : ya - yb);
        nr = dx + dy;
        lat *= nr;
        if (lane < dx) {
          const int32_t x = xb > xa ? xa + (int32_t)lane : xa - (int32_t)lane;
          idx = ((uint32_t)ya * noc_w + (uint32_t)x) * 4u + (xb > xa ? 0u : 1u);
        } else if (lane < nr) {
          const uint32_t i = lane - dx;
          const int32_t y = yb > ya ? ya + (int32_t)i : ya - (int32_t)i;
          idx = ((uint32_t)y * noc_w + (uint32_t)xb) * 4u + (yb > ya ? 2u : 3u);
        }
      }
      uint64_t s = (uint64_t)t;
      if (!nocont) {
        const uint32_t av = lane < nr ? dav[idx] : 0u;
        uint64_t m = uni64(wave_max_u64(av));
        s = m > s ? m : s;
      }
      const uint64_t f = s + od.x + lat;
      if (!complete(v, rec, s, f, sm)) return;
      if (lane < nr) dav[idx] = (uint32_t)(s + od.x);
      release(v, rec, 0, s + 1, rec.cta, sm);
      release(v, rec, 1, f, rec.cta, sm);
    } else {
      const uint32_t a = S[smem_w + 1];
      const uint64_t s = nocont ? (uint64_t)t : (a > t ? a : t);
      // a tile with an address streams its n lines through the engine
      const uint32_t n = G.txn_ptr ? G.txn_ptr[v + 1] - G.txn_ptr[v] : 0u;
      const uint64_t occ_e =
          n ? clamp_occ(cdiv64((uint64_t)n * GTS_LINE_BYTES * 65536ull, hw[HW_RATE + R_GMEM])) : (uint64_t)od.x;
      if (s + occ_e > kMaxCycle) {
        overflow = 1;
        return;
      }
      if (lane == 0) S[smem_w + 1] = (uint32_t)(s + occ_e);
      // the node's state word is free once it issues: an addressed node keeps
      // its start (high) and the largest finish of its transactions so far
      if (n && lane == 0) pst(&state[v], s << 32);
      release(v, rec, 0, s + 1, rec.cta, sm);
      push_one(mkkey(s, kEvMem, v), sm);  // transaction 0 (aux: SM | transaction << 10)
    }
  }

  // Transaction j of addressed node v arrives at the L2 at cycle t.
  __device__ void mem_txn(uint32_t v, const NodeDev& rec, uint32_t t, uint32_t sm, uint32_t j) {
    const uint32_t first = G.txn_ptr[v], n = G.txn_ptr[v + 1] - first;
    const uint4 od = optab[rec.op_nsucc & 0xFFFFu];
    bool dram = (od.w >> 3) & 1u;
    if (l2_lines) dram = !lru_access(G.txn_line[first + j], 1u, l2_lines);
    // the servers' time is kept in 2^-16 cycles: a line may take less than a
    // cycle on an L2 or DRAM of more than 128 B per cycle
    const uint64_t q = cdiv64((uint64_t)GTS_LINE_BYTES << 32, hw[HW_RATE + (dram ? R_DRAM : R_L2)]);
    const uint64_t lat = hw[HW_LAT + (dram ? L_DRAM : L_L2)];
    const bool nocont = (flags & GTS_NO_CONTENTION) != 0;
    const uint64_t av = dram ? dram_av : l2_av;
    const uint64_t tq = (uint64_t)t << 16;
    const uint64_t m = nocont ? tq : (av > tq ? av : tq);
    if (dram)
      dram_av = m + q;
    else
      l2_av = m + q;
    const uint64_t done = (m + q + 65535u) >> 16;
    const uint64_t sw = uni64(pld(&state[v]));
    const uint64_t s = sw >> 32;
    const uint64_t rg = hw[HW_RATE + R_GMEM];
    const uint64_t left = s + cdiv64((uint64_t)(j + 1) * GTS_LINE_BYTES * 65536ull, rg);
    uint64_t f = (left > done ? left : done) + lat;
    if (f > kMaxCycle) {
      overflow = 1;
      return;
    }
    f = f > (uint32_t)sw ? f : (uint32_t)sw;
    if (j + 1 < n) {
      if (lane == 0) pst(&state[v], (s << 32) | f);
      push_one(mkkey(s + cdiv64((uint64_t)(j + 1) * GTS_LINE_BYTES * 65536ull, rg), kEvMem, v), sm | (j + 1) << 10);
      return;
    }
    if (!complete(v, rec, s, f, sm)) return;
    release(v, rec, 1, f, rec.cta, sm);
  }

  // Inclusive prefix sum across the wave.
  // One access of tile x (n lines) to the LRU L2 of `cap` lines; true on a
  // hit: x was touched before and its lines plus those of the distinct tiles
  // touched since fit in cap.  Those tiles are the ones whose latest stamp
  // follows x's, so their lines are the tree's total minus its prefix sum up
  // to x's stamp.  Lanes 0-31 read the prefix's nodes (x's stamp with its k
  // lowest set bits cleared) and move x's lines off the nodes covering its
  // old stamp; lanes 32-63 add them on the nodes covering the new one; a node
  // covering both keeps its value.  Three dependent round trips per access.
  __device__ bool lru_access(uint32_t x, uint32_t n, uint32_t cap) {
    const uint32_t N = lru_acc;  // at most this many accesses, so stamps stay <= N < 2^31
    const uint32_t t = uni(pld(&lru_last[x]));
    const uint32_t now = ++lru_now;
    const uint32_t k = lane & 31u;
    const bool low = lane < 32u;
    uint32_t d = t;
    const uint32_t pc = (uint32_t)__popc(t);
    for (uint32_t s = 0; s < pc; ++s)
      if (s < k) d &= d - 1u;
    const bool pre = low && d != 0u;
    // k-th node covering the lane's stamp: stamp, then + lowest set bit
    uint32_t u = low ? t : now;
    const uint32_t steps = 32u - (uint32_t)__clz(N);
    for (uint32_t s = 0; s < steps; ++s)
      if (s < k && u != 0u && u <= N) u += u & (0u - u);
    const uint32_t other = low ? now : t;
    const bool both = other != 0u && u - (u & (0u - u)) < other && other <= u;
    const bool upd = u != 0u && u <= N && !both;
    const uint64_t pv = pre ? pld(&lru_bit[d]) : 0ull;
    const uint64_t uv = upd ? pld(&lru_bit[u]) : 0ull;
    uint64_t prefix = pv;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) prefix += __shfl_xor(prefix, o, 64);
    prefix = uni64(prefix);
    const bool hit = t != 0u && lru_total - prefix + n <= (uint64_t)cap;
    if (upd) pst(&lru_bit[u], low ? uv - n : uv + n);
    if (lane == 0) pst(&lru_last[x], now);
    if (t == 0u) lru_total += n;
    __builtin_amdgcn_s_waitcnt(0);
    return hit;
  }

  __device__ void mem_arrive(uint32_t v, uint32_t t, uint32_t aux) {
    const NodeDev rec = G.nodes[v];
    const uint32_t sm = aux & 1023u;
    if (G.txn_ptr && G.txn_ptr[v + 1] != G.txn_ptr[v]) {
      mem_txn(v, rec, t, sm, aux >> 10);
      return;
    }
    const uint4 od = optab[rec.op_nsucc & 0xFFFFu];
    bool dram = (od.w >> 3) & 1u;
    uint64_t occm = od.y, lat = od.z;
    if (G.tile && l2_lines) {
      const uint32_t x = G.tile[v];
      if (x != GTS_NO_TILE) {
        const uint64_t work = G.ops[rec.op_nsucc & 0xFFFFu].work;
        dram = !lru_access(x, (uint32_t)((work + GTS_LINE_BYTES - 1) / GTS_LINE_BYTES), l2_lines);
        occm = clamp_occ(cdiv64(work * 65536ull, hw[HW_RATE + (dram ? R_DRAM : R_L2)]));
        lat = hw[HW_LAT + (dram ? L_DRAM : L_L2)];
      }
    }
    const bool nocont = (flags & GTS_NO_CONTENTION) != 0;
    // whole-cycle service: from the first whole cycle the server is free
    const uint64_t av = ((dram ? dram_av : l2_av) + 65535u) >> 16;
    const uint64_t m = nocont ? (uint64_t)t : (av > t ? av : (uint64_t)t);
    const uint64_t mend = m + occm;
    if (dram)
      dram_av = mend << 16;
    else
      l2_av = mend << 16;
    const uint64_t e = (uint64_t)t + od.x;
    const uint64_t f = (e > mend ? e : mend) + lat;
    if (!complete(v, rec, t, f, sm)) return;
    release(v, rec, 1, f, rec.cta, sm);
  }
};

}  // namespace

extern "C" __global__ __launch_bounds__(64) void gts_sim_wave(Launch L) {
  const uint32_t b = blockIdx.x;
  if (b >= L.B) return;
  if (L.retry_only && L.out_status[b] != kStatusRetry) return;
  extern __shared__ uint32_t lds[];
  Sim S;
  S.G = L.img;
  S.hw = L.hw + (uint64_t)b * HW_WORDS;
  S.b = b;
  S.lane = threadIdx.x;
  S.flags = L.flags;
  S.nsm = S.hw[HW_NSM];
  S.nsub = L.srv_one ? 1u : S.hw[HW_NSUB];  // server words per compute class (one when the lanes move together)
  S.sstride = server_stride(S.G.props, S.nsub);
  S.smem_w = S.sstride - 2;
  uint8_t* sim = L.sims + (uint64_t)b * L.layout.stride;
  S.state = reinterpret_cast<uint64_t*>(sim + L.layout.off_state);
  S.cst = reinterpret_cast<CtaState*>(sim + L.layout.off_cta);
  S.pkey = reinterpret_cast<uint64_t*>(sim + L.layout.off_pend);
  S.paux = reinterpret_cast<uint32_t*>(S.pkey + L.layout.pend_cap);
  S.optab = L.lds_optab ? reinterpret_cast<uint4*>(lds) : reinterpret_cast<uint4*>(sim + L.layout.off_optab);
  S.srv = lds + (L.lds_optab ? 4u * S.G.n_ops : 0u);
  S.resident = S.srv + S.nsm * S.sstride;
  S.noc = S.resident + S.nsm;
  S.noc_d = S.hw[HW_NOC_NODES];
  S.noc_w = S.hw[HW_NOC_W];
  S.noc_map = S.hw[HW_NOC_MAP];
  S.lru_last = reinterpret_cast<uint32_t*>(sim + L.layout.off_lru);
  S.lru_bit = reinterpret_cast<uint64_t*>(sim + L.layout.off_lru_bit);
  S.lru_now = 0;
  S.lru_total = 0;
  S.l2_lines = S.hw[HW_L2_LINES];
  S.lru_acc = S.G.n_txn ? S.G.n_txn : S.G.n_nodes;
  S.out_cycles = (L.flags & GTS_OUT_NODES) ? L.out_cycles : nullptr;
  const uint32_t lane = S.lane;

  // R9: a kernel whose CTA fits nowhere makes the simulation infeasible.
  bool infeasible = false;
  for (uint32_t k = lane; k < S.G.n_kernels; k += 64)
    infeasible |= kernel_slots(S.G.kernels[k], S.hw) == 0;
  // clusters and REMOTE nodes need a NoC domain that can hold a cluster
  for (uint32_t k = 0; k < S.G.n_kernels && (S.G.props & kGraphClusters); ++k) {
    const uint32_t cw = S.G.kernels[k].cluster, cl = cw & 0xFFFFu;
    if (cl == 1 && !(cw & kKernelRemote)) continue;
    uint32_t unused = 0;
    if (S.noc_d == 0 || cl > S.noc_d || !S.place(cl, 0, false, unused)) infeasible = true;
  }
  if (__ballot(infeasible)) {
    if (lane == 0) {
      L.out_makespan[b] = 0xFFFFFFFFu;
      L.out_status[b] = GTS_SIM_INFEASIBLE;
      if (L.out_digest) L.out_digest[b] = 0;
    }
    return;
  }

  // Setup: duration table, idle servers, zeroed node / CTA state.
  for (uint32_t p = lane; p < S.G.n_ops; p += 64) {
    uint4 e = op_entry(S.G.ops[p], S.hw, S.G.props);
    const uint32_t cls = e.w & 7u;
    if (L.srv_one && cls <= C_SFU)  // the class's single word: lane 0 of its slot
      e.w = (e.w & 0xFFu) | (1u << 8) | (compute_slot(S.G.props, cls) << 16);
    S.optab[p] = e;
  }
  const uint32_t nsrv = S.nsm * S.sstride + S.nsm + L.noc_words;
  for (uint32_t i = lane; i < nsrv; i += 64) S.srv[i] = 0;
  for (uint32_t v = lane; v < S.G.n_nodes; v += 64) pst(&S.state[v], (uint64_t)0);
  if ((S.G.tile || S.G.txn_ptr) && S.l2_lines) {
    const uint32_t keys = S.G.txn_ptr ? S.G.n_lines : S.G.n_tiles;
    for (uint32_t x = lane; x < keys; x += 64) pst(&S.lru_last[x], 0u);
    for (uint32_t i = lane; i <= S.lru_acc; i += 64) pst(&S.lru_bit[i], (uint64_t)0);
  }
  for (uint32_t c = lane; c < S.G.n_ctas; c += 64) {
    pst(&S.cst[c].sm, 0u);
    pst(&S.cst[c].launch, 0u);
    pst(&S.cst[c].left, 0u);
    pst(&S.cst[c].maxfin, 0u);
  }
  __syncthreads();

  S.npend = 0;
  S.next_cta = 0;
  S.retired = 0;
  S.cur_k = 0;
  S.run_kb = 0;
  S.run_cl = 1;
  S.kstart_k = 0;
  S.kstart_t = 0;
  S.kstart_valid = 0;
  S.l2_av = 0;
  S.dram_av = 0;
  S.digest = 0;
  S.makespan = 0;
  S.nfin = 0;
  S.overflow = 0;

  S.dispatch(0);
  bool dispatch_due = false;
  uint32_t due_t = 0;
  while (!S.overflow) {
    if (S.npend == 0) {
      if (!dispatch_due) break;
      S.dispatch(due_t);
      dispatch_due = false;
      continue;
    }
    // minimum pending key (unique: cycle, phase, id) with its aux word; four
    // independent loads per lane per pass, and the last entry (which fills
    // the taken one's place) loaded alongside
    const uint32_t last = S.npend - 1;
    const uint64_t lk = pld(&S.pkey[last]);
    const uint32_t la = pld(&S.paux[last]);
    uint64_t best = ~0ull;
    uint32_t bi = 0, ba = 0;
    for (uint32_t i0 = 0; i0 < S.npend; i0 += 256) {
      uint64_t k[4];
      uint32_t a[4];
#pragma unroll
      for (uint32_t j = 0; j < 4; ++j) {
        const uint32_t i = i0 + j * 64u + lane;
        k[j] = i < S.npend ? pld(&S.pkey[i]) : ~0ull;
        a[j] = i < S.npend ? pld(&S.paux[i]) : 0u;
      }
#pragma unroll
      for (uint32_t j = 0; j < 4; ++j)
        if (k[j] < best) {
          best = k[j];
          bi = i0 + j * 64u + lane;
          ba = a[j];
        }
    }
    const uint64_t mn = uni64(wave_min_u64(best));
    const uint64_t who = __ballot(best == mn);
    const uint32_t src = (uint32_t)__ffsll((unsigned long long)who) - 1u;
    const uint32_t idx = (uint32_t)__shfl(bi, src, 64);
    const uint32_t t = (uint32_t)(mn >> 32);
    const uint32_t kind = (uint32_t)(mn >> 30) & 3u;
    const uint32_t id = (uint32_t)mn & GTS_EDGE_TARGET_MASK;
    if (dispatch_due && !(kind == kEvRetire && t == due_t)) {
      S.dispatch(due_t);
      dispatch_due = false;
      continue;
    }
    const uint32_t aux = uni((uint32_t)__shfl(ba, src, 64));
    if (idx != last && lane == 0) {
      pst(&S.pkey[idx], lk);
      pst(&S.paux[idx], la);
    }
    S.npend = last;
    if (kind == kEvRetire) {
      if (lane == 0) S.resident[aux] -= 1;
      ++S.retired;
      dispatch_due = true;
      due_t = t;
    } else if (kind == kEvReady) {
      S.issue(id, t, aux);
    } else {
      S.mem_arrive(id, t, aux);
    }
    __builtin_amdgcn_wave_barrier();
  }

  if (lane == 0) {
    int32_t st = GTS_SIM_OK;
    if (S.overflow)
      st = GTS_SIM_OVERFLOW;
    else if (S.nfin != S.G.n_nodes)
      st = GTS_SIM_DEADLOCK;
    L.out_status[b] = st;
    L.out_makespan[b] = st == GTS_SIM_OK ? S.makespan : 0xFFFFFFFFu;
    if (L.out_digest) L.out_digest[b] = st == GTS_SIM_OK ? S.digest : 0ull;
  }
}

hipError_t launch_sim(const Launch& L, uint32_t lds_bytes, hipStream_t stream) {
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(gts_sim_wave, dim3(L.B), dim3(64), lds_bytes, stream, L);
  return hipGetLastError();
}

}  // namespace gts
