"""The five benchmark workloads: graph recipe + scenario recipe, all seeded.

    1 tiny      GPT 2 layers, h 1024, s 512, TP2 x PP2 x DP2 (8 ranks), 4 microbatches,
                1 default scenario
    2 175b-96   GPT-175B (96 layers, h 12288, s 2048), TP8 x PP4 x DP3 (96 ranks),
                8 microbatches, 64 scenarios varying inter-node bandwidth and alpha
    3 175b-1024 GPT-175B, TP8 x PP16 x DP8 (1024 ranks), 32 microbatches, 256 scenarios
                with +-10 % duration jitter and slowdown entries in [1.0, 1.4]
    4 enum-4096 the config-1 graph, 4096 scenarios varying ring/tree, both bandwidths,
                alpha and the slowdown table
    5 extrap    16 GPT-70B/175B graphs (TP {4, 8} x PP {8, 16, 32} x DP up to 64,
                at most 8192 ranks), 32 scenarios each

Model shapes follow the paper's GPT table (Table 9).  Scenario arrays are drawn
with numpy's default_rng(1000 + config number).
"""
from __future__ import annotations

import numpy as np

from . import gpt1f1b, scenarios

GPT70B = dict(n_layers=80, hidden=8192, seq=2048)
GPT175B = dict(n_layers=96, hidden=12288, seq=2048)
TINY = dict(n_layers=2, hidden=1024, seq=512)

BW_RANGE = (50_000, 400_000)        # MB/s
ALPHA_RANGE = (2_000, 20_000)       # ns
SLOWDOWN_RANGE = (65536, 91750)     # Q16, factors 1.0 .. 1.4
JITTER_AMP_Q16 = 6554               # +-10 %

# Config 5: (model, TP, PP, DP, microbatches, distributed optimizer?)
EXTRAP_GRAPHS = [
    ("70b", 4, 8, 8, 8, False),
    ("70b", 4, 16, 16, 16, True),
    ("70b", 4, 8, 64, 8, False),
    ("70b", 8, 8, 8, 16, True),
    ("70b", 8, 16, 16, 16, False),
    ("70b", 8, 16, 32, 8, True),
    ("70b", 8, 16, 64, 8, False),
    ("70b", 4, 16, 32, 16, True),
    ("175b", 4, 8, 16, 8, False),
    ("175b", 4, 16, 32, 16, True),
    ("175b", 4, 32, 16, 32, False),
    ("175b", 8, 8, 8, 8, True),
    ("175b", 8, 16, 8, 32, False),
    ("175b", 8, 32, 8, 32, True),
    ("175b", 8, 32, 32, 8, False),
    ("175b", 8, 16, 64, 8, True),
]
N_SCEN = {1: 1, 2: 64, 3: 256, 4: 4096, 5: 32}
NAMES = {1: "tiny-gpt2l-tp2pp2dp2", 2: "gpt175b-tp8pp4dp3", 3: "gpt175b-tp8pp16dp8",
         4: "tiny-enum4096", 5: "extrap-16graphs"}


def graph_params(config: int, index: int = 0) -> dict:
    """Keyword arguments of gpt1f1b.gpt_graph for a config (index: config-5 graph)."""
    if config in (1, 4):
        return dict(TINY, tp=2, pp=2, dp=2, microbatches=4, seed=0)
    if config == 2:
        return dict(GPT175B, tp=8, pp=4, dp=3, microbatches=8, seed=2)
    if config == 3:
        return dict(GPT175B, tp=8, pp=16, dp=8, microbatches=32, seed=3)
    if config == 5:
        model, t, p, d, m, distopt = EXTRAP_GRAPHS[index]
        shape = GPT70B if model == "70b" else GPT175B
        return dict(shape, tp=t, pp=p, dp=d, microbatches=m, seed=50 + index, distopt=distopt)
    raise ValueError(f"unknown config {config}")


def graph(config: int, index: int = 0) -> dict:
    return gpt1f1b.gpt_graph(**graph_params(config, index))


def scenario_batch(config: int, index: int = 0, n: int | None = None) -> dict:
    """The seeded scenario batch of a config (index: config-5 graph; n: another
    batch size drawn with the same recipe)."""
    rng = np.random.default_rng(1000 + config)
    n = N_SCEN[config] if n is None else int(n)
    if config == 1:
        return scenarios.default_scenarios(n)
    if config == 2:
        return scenarios.draw(n, rng, bw_inter=BW_RANGE, alpha=ALPHA_RANGE)
    if config == 3:
        return scenarios.draw(n, rng, slowdown=SLOWDOWN_RANGE, jitter=(JITTER_AMP_Q16, 3))
    if config == 4:
        return scenarios.draw(n, rng, bw_inter=BW_RANGE, bw_intra=BW_RANGE,
                              alpha=ALPHA_RANGE, ar_algo_random=True, slowdown=SLOWDOWN_RANGE)
    if config == 5:
        sc = None
        for g in range(index + 1):        # graph g takes the g-th block of draws
            sc = scenarios.draw(n, rng, bw_inter=BW_RANGE, alpha=ALPHA_RANGE,
                                slowdown=SLOWDOWN_RANGE)
        return sc
    raise ValueError(f"unknown config {config}")
