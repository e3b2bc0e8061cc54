"""Hardware parameter records: presets from the paper's Table 3 and seeded
samplers for design-space sweeps.

A record is 32 little-endian u32 words (include/gts.h, gts_hw_params).  Rates
are Q16.16 work units per core cycle: per SM for tensor / CUDA-core / SFU /
shared-memory / global-memory-engine, chip-wide for L2 and DRAM.  Latencies
are core cycles.

Table 3 (Sec. 6.1) gives, per GPU: SMs, core MHz, CUDA cores and SFUs per SM,
tensor-core FMAs per clock per SM, SRAM bandwidth/latency, L2 bandwidth
(B/cycle) / latency, DRAM bandwidth (GB/s) / latency, TMA issue rate
(B/cycle; Sec. 5.2 measures roughly 100 B per cycle).  Conversions (readings
where the paper is silent):
  - tensor FLOP/cycle = 2 x FMAs/clk (work is counted in FLOPs);
  - DRAM B/cycle = MB/s / core MHz, floored once into Q16.16;
  - the TMA rate is per SM; A100 has no TMA and its engine (cp.async through
    the LSU) runs at the SRAM bandwidth;
  - values the paper does not give are the defaults below (subpartitions 4,
    32 CTAs / 64 warps per SM, latencies of tensor 16, ALU 4, SFU 16,
    SYNC 20, launch latencies 0; shared memory 164 KiB A100, 228 KiB H100/B200).
"""
from __future__ import annotations

import numpy as np

from .rng import SplitMix64

Q16 = 1 << 16

FIELDS = {
    "n_sm": 0, "n_subpart": 1, "max_cta_per_sm": 2, "max_warps_per_sm": 3, "smem_per_sm": 4,
    "rate_tensor": 5, "rate_alu": 6, "rate_sfu": 7, "rate_smem": 8, "rate_gmem": 9, "rate_l2": 10,
    "rate_dram": 11,
    "lat_tensor": 12, "lat_alu": 13, "lat_sfu": 14, "lat_smem": 15, "lat_l2": 16, "lat_dram": 17,
    "lat_sync": 18, "cta_launch_lat": 19, "kernel_launch_lat": 20,
    "noc_nodes": 21, "noc_width": 22, "noc_rate": 23, "noc_lat": 24, "noc_map": 25, "l2_lines": 26,
}
L2_MIB = {"A100": 40, "H100": 50, "B200": 126}  # L2 capacity (LRU model: l2_lines = MiB * 8192)


def l2_lines(mib: float) -> int:
    """128-B lines of an L2 of `mib` MiB."""
    return int(mib * (1 << 20)) // 128
NWORDS = 32


def dram_q16(mb_per_s: int, core_mhz: int) -> int:
    """DRAM bytes per core cycle in Q16.16: floor(MB/s * 65536 / MHz)."""
    return (int(mb_per_s) * Q16) // int(core_mhz)


# Table 3 rows (Sec. 6.1).  mhz is the core clock.
TABLE3 = {
    "A100": dict(n_sm=108, mhz=1410, cuda=64, sfu=16, tc_fma=1024, sram_bw=128, sram_lat=33,
                 l2_bw=2300, l2_lat=300, dram_gbs=1407, dram_lat=250, tma=None, smem_kib=164),
    "H100": dict(n_sm=132, mhz=1980, cuda=128, sfu=16, tc_fma=2048, sram_bw=128, sram_lat=33,
                 l2_bw=4300, l2_lat=380, dram_gbs=3100, dram_lat=270, tma=100, smem_kib=228),
    "B200": dict(n_sm=148, mhz=1965, cuda=128, sfu=16, tc_fma=4096, sram_bw=128, sram_lat=33,
                 l2_bw=6000, l2_lat=380, dram_gbs=8000, dram_lat=270, tma=100, smem_kib=228),
}
DEFAULTS = dict(n_subpart=4, max_cta_per_sm=32, max_warps_per_sm=64, lat_tensor=16, lat_alu=4, lat_sfu=16,
                lat_sync=20, cta_launch_lat=0, kernel_launch_lat=0)


def record(**kw) -> np.ndarray:
    """A 32-word record from named fields (rates already in Q16.16)."""
    r = np.zeros(NWORDS, dtype=np.uint32)
    for k, v in kw.items():
        if k not in FIELDS:
            raise KeyError(k)
        v = int(v)
        if not 0 <= v < (1 << 32):
            raise ValueError(f"{k}={v} does not fit u32")
        r[FIELDS[k]] = v
    return r


def preset(name: str, *, tensor_permille: int = 1000, dram_mb_s: int | None = None, n_sm: int | None = None,
           smem_kib: int | None = None, **overrides) -> np.ndarray:
    """Record for a Table 3 GPU, optionally with sweep scalings applied."""
    t = TABLE3[name]
    mb = dram_mb_s if dram_mb_s is not None else t["dram_gbs"] * 1000
    fields = dict(DEFAULTS)
    fields.update(
        n_sm=n_sm if n_sm is not None else t["n_sm"],
        smem_per_sm=(smem_kib if smem_kib is not None else t["smem_kib"]) * 1024,
        rate_tensor=(2 * t["tc_fma"] * Q16 * int(tensor_permille)) // 1000,
        rate_alu=t["cuda"] * Q16,
        rate_sfu=t["sfu"] * Q16,
        rate_smem=t["sram_bw"] * Q16,
        rate_gmem=(t["tma"] if t["tma"] is not None else t["sram_bw"]) * Q16,
        rate_l2=t["l2_bw"] * Q16,
        rate_dram=dram_q16(mb, t["mhz"]),
        lat_smem=t["sram_lat"],
        lat_l2=t["l2_lat"],
        lat_dram=t["dram_lat"],
    )
    fields.update(overrides)
    return record(**fields)


def toy(**overrides) -> np.ndarray:
    """The one-SM toy machine of the hand-computed schedules in tests/golden."""
    fields = dict(n_sm=1, n_subpart=4, max_cta_per_sm=1, max_warps_per_sm=64, smem_per_sm=64 * 1024,
                  rate_tensor=256 * Q16, rate_alu=64 * Q16, rate_sfu=16 * Q16, rate_smem=128 * Q16,
                  rate_gmem=64 * Q16, rate_l2=128 * Q16, rate_dram=32 * Q16,
                  lat_tensor=10, lat_alu=4, lat_sfu=16, lat_smem=33, lat_l2=40, lat_dram=100, lat_sync=20,
                  cta_launch_lat=0, kernel_launch_lat=0)
    fields.update(overrides)
    return record(**fields)


def sample_a100_sweep(seed: int, B: int) -> np.ndarray:
    """A100 base; DRAM 1.5-3 TB/s and tensor rate 0.5-2x, uniform."""
    rng = SplitMix64(seed)
    out = np.zeros((B, NWORDS), dtype=np.uint32)
    for b in range(B):
        mb = rng.randint(1_500_000, 3_000_000)
        tp = rng.randint(500, 2000)
        out[b] = preset("A100", tensor_permille=tp, dram_mb_s=mb)
    return out


def sample_h100_sweep(seed: int, B: int, stream: int = 0) -> np.ndarray:
    """H100 base; SMs 64-192, DRAM 1.5-8 TB/s, shared memory 96-256 KiB,
    tensor rate 0.5-4x, each uniform."""
    rng = SplitMix64(seed, stream)
    out = np.zeros((B, NWORDS), dtype=np.uint32)
    for b in range(B):
        n_sm = rng.randint(64, 192)
        mb = rng.randint(1_500_000, 8_000_000)
        smem = rng.randint(96, 256)
        tp = rng.randint(500, 4000)
        out[b] = preset("H100", tensor_permille=tp, dram_mb_s=mb, n_sm=n_sm, smem_kib=smem)
    return out


def sample_random(rng: SplitMix64, n_sm_max: int = 4) -> np.ndarray:
    """Small random machines for brute-force and cross-check tests: every
    rate and latency drawn independently, including awkward values."""
    return record(
        n_sm=rng.randint(1, n_sm_max), n_subpart=rng.choice([1, 2, 4]),
        max_cta_per_sm=rng.randint(1, 3), max_warps_per_sm=rng.randint(8, 64),
        smem_per_sm=rng.randint(16, 96) * 1024,
        rate_tensor=rng.randint(Q16 // 3, 512 * Q16), rate_alu=rng.randint(Q16 // 2, 128 * Q16),
        rate_sfu=rng.randint(Q16 // 2, 32 * Q16), rate_smem=rng.randint(Q16, 256 * Q16),
        rate_gmem=rng.randint(Q16, 256 * Q16), rate_l2=rng.randint(4 * Q16, 2048 * Q16),
        rate_dram=rng.randint(Q16, 1024 * Q16),
        lat_tensor=rng.randint(0, 40), lat_alu=rng.randint(0, 10), lat_sfu=rng.randint(0, 30),
        lat_smem=rng.randint(0, 40), lat_l2=rng.randint(0, 300), lat_dram=rng.randint(0, 400),
        lat_sync=rng.randint(0, 30), cta_launch_lat=rng.randint(0, 3) * rng.randint(0, 50),
        kernel_launch_lat=rng.randint(0, 2) * rng.randint(0, 100))


def get(rec: np.ndarray, name: str) -> int:
    return int(rec[FIELDS[name]])
