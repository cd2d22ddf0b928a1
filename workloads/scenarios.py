"""Seeded what-if scenarios: network parameters, jitter and slowdown tables.

A scenario is one set of cluster/hardware knobs that the simulator is asked
about ("what if the inter-node bandwidth doubled?", the usage in the paper's
introduction and its DDP network study, Table 10).  Scenarios are returned as
a dict of numpy arrays, one entry per field (structure of arrays):

    alpha_ns       int64  [n]        connection set-up time of a collective (ns)
    bw_intra_MBps  int64  [n]        intra-server link bandwidth (MB/s, 10^6 B/s)
    bw_inter_MBps  int64  [n]        inter-server bandwidth per GPU (MB/s)
    reduce_MBps    int64  [n]        reduction throughput of the collective kernel (MB/s)
    jitter_seed    uint64 [n]        seed of the per-op duration jitter stream
    jitter_stream  uint32 [n]        which SplitMix64 sub-stream the scenario draws from
                                     (its index in the batch it was drawn in)
    jitter_amp_q16 int32  [n]        jitter amplitude A in Q16 (0 = no jitter)
    ar_algo        uint8  [n]        all-reduce algorithm: 0 ring, 1 tree
    cc_model       uint8  [n]        collective cost model: 0 Echo (chunked), 1 alpha-beta baseline
    cc_table       int32  [n]        0: parameters from the bandwidths; k: CC parameter table k-1
    slowdown_q16   uint32 [n, 8, 4]  slowdown factor per (kernel class, collective type), Q16

CC parameter tables (int64 [6, 7]: per row max_bytes, chunk, alpha_ns,
beta_ns, gamma_ns, reduce_MBps) are inputs too.

Only input values live here; no formula of the method is evaluated.
"""
from __future__ import annotations

import numpy as np

RING, TREE = 0, 1

# Default slowdown factors per kernel class (same for every collective type), Q16.
# GEMM, Transform, Sum, Grad: per-kernel slowdowns when overlapped with a 25 MB
# all-reduce (Table 2: 1.269, 1.142, 1.508, 1.613).  LayerNorm: A800, CUDA 12.1
# (Table 3: 1.207).  Attention, optimizer and other kernels: the average increase
# of 37.76 % reported next to Table 2.  Each value is round(factor * 65536).
PAPER_SLOWDOWN_Q16 = np.array(
    [83165,    # GEMM       1.269
     74842,    # Transform  1.142
     98828,    # Sum        1.508
     105710,   # Grad       1.613
     79102,    # LayerNorm  1.207
     90282,    # Attention  1.3776
     90282,    # Optimizer  1.3776
     90282],   # Other      1.3776
    dtype=np.uint32)

DEFAULTS = dict(
    alpha_ns=10_000,            # connection set-up
    bw_intra_MBps=400_000,      # NVLink 400 GB/s per GPU (H800 cluster)
    bw_inter_MBps=50_000,       # 400 Gb/s NDR InfiniBand per GPU
    reduce_MBps=160_000,        # 256 MiB reduced in about 1.66 ms (Table 6)
)

FIELDS = ("alpha_ns", "bw_intra_MBps", "bw_inter_MBps", "reduce_MBps",
          "jitter_seed", "jitter_stream", "jitter_amp_q16", "ar_algo", "cc_model", "cc_table", "slowdown_q16")

# Table 6 of the paper: tensor-size bands (MB read as MiB) and NCCL's chunk size for each.
TABLE6_MAX_BYTES = np.array([4, 8, 16, 32, 64, 128, 256], np.int64) << 20
TABLE6_CHUNK = np.array([18000, 36000, 72000, 72000, 72000, 144000, 288000], np.int64)


def default_scenarios(n: int) -> dict:
    """n copies of the default scenario: ring AR, no jitter, the paper's slowdowns."""
    return {
        "alpha_ns": np.full(n, DEFAULTS["alpha_ns"], np.int64),
        "bw_intra_MBps": np.full(n, DEFAULTS["bw_intra_MBps"], np.int64),
        "bw_inter_MBps": np.full(n, DEFAULTS["bw_inter_MBps"], np.int64),
        "reduce_MBps": np.full(n, DEFAULTS["reduce_MBps"], np.int64),
        "jitter_seed": np.zeros(n, np.uint64),
        "jitter_stream": np.arange(n, dtype=np.uint32),
        "jitter_amp_q16": np.zeros(n, np.int32),
        "ar_algo": np.full(n, RING, np.uint8),
        "cc_model": np.zeros(n, np.uint8),
        "cc_table": np.zeros(n, np.int32),
        "slowdown_q16": np.broadcast_to(PAPER_SLOWDOWN_Q16[None, :, None], (n, 8, 4)).copy(),
    }


def _u(rng, lo, hi, n):
    return rng.integers(lo, hi + 1, size=n, dtype=np.int64)


def draw(n: int, rng: np.random.Generator, *, bw_inter=None, bw_intra=None,
         alpha=None, ar_algo_random=False, slowdown=None, jitter=None) -> dict:
    """Draw n scenarios; every knob left as None keeps its default value.

    bw_inter / bw_intra / alpha / slowdown: inclusive integer ranges (lo, hi),
    drawn uniformly and independently per scenario (and per table entry).
    jitter: (amplitude_q16, seed) applied to every scenario.
    """
    sc = default_scenarios(n)
    if bw_inter is not None:
        sc["bw_inter_MBps"] = _u(rng, *bw_inter, n)
    if bw_intra is not None:
        sc["bw_intra_MBps"] = _u(rng, *bw_intra, n)
    if alpha is not None:
        sc["alpha_ns"] = _u(rng, *alpha, n)
    if ar_algo_random:
        sc["ar_algo"] = rng.integers(0, 2, size=n).astype(np.uint8)
    if slowdown is not None:
        sc["slowdown_q16"] = rng.integers(slowdown[0], slowdown[1] + 1,
                                          size=(n, 8, 4)).astype(np.uint32)
    if jitter is not None:
        sc["jitter_amp_q16"] = np.full(n, jitter[0], np.int32)
        sc["jitter_seed"] = np.full(n, jitter[1], np.uint64)
    return sc


def take(sc: dict, idx) -> dict:
    """Sub-batch of scenarios (idx: slice, int array or list)."""
    return {k: np.ascontiguousarray(v[idx]) for k, v in sc.items()}


def count(sc: dict) -> int:
    return int(sc["alpha_ns"].shape[0])


def cc_table(*, chunk, alpha, beta, gamma, reduce, max_bytes=TABLE6_MAX_BYTES) -> np.ndarray:
    """One CC parameter table, int64 [6, 7]; each argument a scalar or 7 values."""
    rows = [np.broadcast_to(np.asarray(x, np.int64), (7,)) for x in (max_bytes, chunk, alpha, beta, gamma, reduce)]
    return np.stack(rows).astype(np.int64)


def draw_cc_tables(n: int, rng: np.random.Generator) -> np.ndarray:
    """n seeded what-if tables, int64 [n, 6, 7]: Table 6 bands and chunks scaled by
    1/2..2, alpha 2-20 us, per-chunk beta 20-400 ns and gamma 100-2000 ns (rising
    with the chunk), reduce 100-400 GB/s."""
    out = []
    for _ in range(n):
        scale = rng.integers(1, 5, 7) / 2.0
        chunk = np.maximum(1, (TABLE6_CHUNK * scale).astype(np.int64))
        out.append(cc_table(chunk=chunk, alpha=rng.integers(2_000, 20_001, 7),
                            beta=np.sort(rng.integers(20, 401, 7)), gamma=np.sort(rng.integers(100, 2001, 7)),
                            reduce=rng.integers(100_000, 400_001, 7)))
    return np.stack(out) if out else np.zeros((0, 6, 7), np.int64)
