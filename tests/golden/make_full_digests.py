"""Writes the oracle's step time and digest of EVERY scenario of the two
largest workloads, for the full-size parity tests:

  full_digests_config3.txt  GPT-175B TP8xPP16xDP8 (1024 ranks) x 256 scenarios, R = 1
  full_digests_config5.txt  the 16 extrapolation graphs x 32 scenarios each, R = 1

Every value comes from the CPU oracle (oracle.run) on the seeded synthetic
inputs of workloads.configs; nothing else is called.  Each block header holds a
hash of the inputs it was made from, so a test can tell a stale file from a
wrong result.  Takes about a quarter of an hour on 8 host threads:

  python tests/golden/make_full_digests.py [3] [5]
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

GRAPH_KEYS = ("op_rank", "op_stream", "op_kind", "op_class", "op_dur", "op_coll", "pred_off", "pred_idx",
              "coll_type", "coll_bytes", "n_ranks", "gpus_per_node")


def input_hash(g: dict, sc: dict) -> str:
    """sha256[:16] over the graph arrays and the scenario fields, in a fixed order."""
    h = hashlib.sha256()
    for k in GRAPH_KEYS:
        h.update(k.encode())
        h.update(np.ascontiguousarray(np.asarray(g[k])).tobytes())
    for k in sorted(sc):
        h.update(k.encode())
        h.update(np.ascontiguousarray(np.asarray(sc[k])).tobytes())
    return h.hexdigest()[:16]


def path(config: int) -> str:
    return os.path.join(HERE, f"full_digests_config{config}.txt")


def load(config: int) -> dict:
    """{index: (input hash, step int64 [n], digest uint64 [n])} from the stored file."""
    blocks, cur = {}, None
    for line in open(path(config)):
        if line.startswith("# graph"):
            _, _, cfg, idx, _, h = line.split()
            assert int(cfg) == config, line
            cur = int(idx)
            blocks[cur] = (h, [], [])
        elif line.strip() and not line.startswith("#"):
            _, step, dig = line.split()
            blocks[cur][1].append(int(step))
            blocks[cur][2].append(int(dig))
    return {i: (h, np.array(s, np.int64), np.array(d, np.uint64)) for i, (h, s, d) in blocks.items()}


def main(which):
    import oracle
    from workloads import configs
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    for config in which:
        indices = range(16) if config == 5 else [0]
        lines = [f"# Oracle step time and digest of every scenario, config {config} ({configs.NAMES[config]}),",
                 "# one refinement, written by tests/golden/make_full_digests.py (oracle.run only).",
                 "# Per graph: '# graph <config> <index> input <sha256[:16] of graph arrays and scenarios>',",
                 "# then one line per scenario: <scenario> <step ns> <digest as unsigned 64-bit>."]
        for i in indices:
            t = time.perf_counter()
            g, sc = configs.graph(config, i), configs.scenario_batch(config, i)
            ref = oracle.run(g, sc, 1, threads=threads, timelines=False)
            lines.append(f"# graph {config} {i} input {input_hash(g, sc)}")
            lines += [f"{s} {int(ref['step'][s])} {int(ref['digest'][s])}" for s in range(len(ref["step"]))]
            print(f"config {config} graph {i}: {len(g['op_rank'])} ops x {len(ref['step'])} scenarios "
                  f"({time.perf_counter() - t:.0f} s)", flush=True)
            del g, ref
        open(path(config), "w").write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or [3, 5])
