// gts_common.h — device helpers shared by the simulation kernels of
// libgts.so (wave reductions, private-scratch accessors, duration table).
#pragma once
#include <hip/hip_runtime.h>

#include "../../include/gts.h"
#include "gts_dev.h"

namespace gts {
namespace {

constexpr uint32_t kEvRetire = 0, kEvReady = 1, kEvMem = 2;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint64_t uni64(uint64_t x) {
  return ((uint64_t)uni((uint32_t)(x >> 32)) << 32) | uni((uint32_t)x);
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    uint64_t y = __shfl_xor(x, o, 64);
    x = y < x ? y : x;
  }
  return x;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    uint64_t y = __shfl_xor(x, o, 64);
    x = y > x ? y : x;
  }
  return x;
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask, uint32_t lane) {
  return (uint32_t)__popcll(mask & ((1ull << lane) - 1ull));
}

// Simulation-private scratch is read and written by this wave only.  Relaxed
// wavefront-scope atomics keep these accesses on the vector memory path (a
// uniform address must not become a scalar-cache load of memory this wave
// has just written); a wavefront's vector accesses complete in order.
template <typename T>
__device__ __forceinline__ T pld(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
template <typename T>
__device__ __forceinline__ void pst(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

__device__ __forceinline__ uint64_t mkkey(uint64_t t, uint32_t kind, uint32_t id) {
  return (t << 32) | ((uint64_t)kind << 30) | id;
}

__device__ __forceinline__ uint64_t cdiv64(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

__device__ __forceinline__ uint32_t clamp_occ(uint64_t x) {
  x = x < 1 ? 1 : x;
  return x > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)x;
}

// Per-op duration entry: x = occupancy (engine occupancy for memory ops),
// y = L2/DRAM occupancy, z = latency, w = class | dram << 3 | lane mask << 8
// | first server word of the class's lanes << 16 (compute ops).
__device__ uint4 op_entry(const OpDev& o, const uint32_t* hw, uint32_t props) {
  const uint32_t nsub = hw[HW_NSUB];
  const uint64_t work = o.work;
  uint4 e = make_uint4(0, 0, 0, o.cls);
  if (o.cls <= C_SFU) {
    uint32_t lanes = 0;
    for (uint32_t w = 0; w < 32; ++w)
      if ((o.warps >> w) & 1u) lanes |= 1u << (w % nsub);
    const uint64_t k = (uint64_t)__popc(lanes);
    e.x = clamp_occ(cdiv64(work * 65536ull * nsub, k * hw[HW_RATE + o.cls]));
    e.z = hw[HW_LAT + o.cls];
    e.w |= lanes << 8 | (compute_slot(props, o.cls) * nsub) << 16;
  } else if (o.cls == C_SMEM) {
    e.x = clamp_occ(cdiv64(work * 65536ull, hw[HW_RATE + R_SMEM]));
    e.z = hw[HW_LAT + L_SMEM];
  } else if (o.cls == C_SYNC) {
    const uint32_t l = hw[HW_LAT + L_SYNC];
    e.z = l < 1 ? 1 : l;
  } else if (o.cls == C_REMOTE) {  // x = NoC occupancy, z = latency per traversal / hop, w: rank << 16
    const uint32_t rate = hw[HW_NOC_RATE];
    e.x = rate ? clamp_occ(cdiv64(work * 65536ull, rate)) : 1u;
    e.z = hw[HW_NOC_LAT];
    e.w |= (uint32_t)(o.flags >> GTS_OPF_RANK_SHIFT) << 16;
  } else {
    const uint32_t dram = o.flags & GTS_OPF_MISS;
    e.x = clamp_occ(cdiv64(work * 65536ull, hw[HW_RATE + R_GMEM]));
    e.y = clamp_occ(cdiv64(work * 65536ull, hw[HW_RATE + (dram ? R_DRAM : R_L2)]));
    e.z = hw[HW_LAT + (dram ? L_DRAM : L_L2)];
    e.w |= dram << 3;
  }
  return e;
}

__device__ __forceinline__ uint64_t kernel_slots(const KernelDev& kd, const uint32_t* hw) {
  uint64_t s = hw[HW_MAXCTA];
  if (kd.smem) {
    const uint64_t m = hw[HW_SMEM] / kd.smem;
    s = s < m ? s : m;
  }
  const uint64_t w = hw[HW_MAXWARPS] / kd.warps;
  return s < w ? s : w;
}

}  // namespace
}  // namespace gts
