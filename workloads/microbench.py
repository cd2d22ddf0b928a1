"""Small synthetic graphs that isolate the composer walk's latencies.

The walk's time on a large graph is set by its longest chain of dependent walk
items (echo_walk_chain): items in a walker's list order, and every resolve
item after the launches of all members of its collective.  These graphs put a
known chain in front of the walk so that one item's latency, and one barrier's
latency in LDS or in device memory, can be measured on the device:

    chain(n, ranks)       each rank n chained compute ops: n items, no barrier
    allreduce_rounds(...) every rank runs k chained ops, then joins an all-reduce
                          of all ranks whose result its next op waits for
                          (8 ranks: one workgroup, the barrier lives in LDS)
    p2p_pingpong(...)     rank r and rank r + 8 (two workgroups) hand a token
                          back and forth by send/recv after k ops each: every
                          barrier on the chain is met in device memory

Inputs only; nothing here composes anything.
"""
from __future__ import annotations

import numpy as np

from .gpt1f1b import COLL_AR, COLL_P2P, KIND_COMM, KIND_COMPUTE, S_COMPUTE, S_RECV, S_SEND, S_TP


class _Graph:
    def __init__(self, n_ranks, gpus_per_node=8):
        self.n_ranks, self.gpn = n_ranks, gpus_per_node
        self.rank, self.stream, self.kind, self.cls, self.dur, self.coll, self.preds = ([] for _ in range(7))
        self.ctype, self.cbytes = [], []

    def collective(self, ctype, nbytes):
        self.ctype.append(ctype)
        self.cbytes.append(nbytes)
        return len(self.ctype) - 1

    def op(self, rank, stream, kind, dur=0, coll=-1, preds=()):
        self.rank.append(rank)
        self.stream.append(stream)
        self.kind.append(kind)
        self.cls.append(0 if kind == KIND_COMPUTE else 7)
        self.dur.append(dur)
        self.coll.append(coll)
        self.preds.append(list(preds))
        return len(self.rank) - 1

    def arrays(self):
        off = np.zeros(len(self.preds) + 1, np.int64)
        np.cumsum([len(p) for p in self.preds], out=off[1:])
        return {"op_rank": np.array(self.rank, np.int32), "op_stream": np.array(self.stream, np.uint8),
                "op_kind": np.array(self.kind, np.uint8), "op_class": np.array(self.cls, np.uint8),
                "op_dur": np.array(self.dur, np.int64), "op_coll": np.array(self.coll, np.int64),
                "pred_off": off, "pred_idx": np.array([u for p in self.preds for u in p], np.int32),
                "coll_type": np.array(self.ctype, np.uint8), "coll_bytes": np.array(self.cbytes, np.int64),
                "n_ranks": self.n_ranks, "gpus_per_node": self.gpn}


def _durations(rng, n):
    return np.maximum(1, np.rint(rng.lognormal(np.log(50_000.0), 0.5, n))).astype(np.int64)


def chain(n_ops, seed=0, ranks=1):
    """`ranks` ranks, each one chain of n_ops compute ops (independent of each other)."""
    g = _Graph(ranks)
    rng = np.random.default_rng(seed)
    for r in range(ranks):
        for d in _durations(rng, n_ops):
            g.op(r, S_COMPUTE, KIND_COMPUTE, int(d))
    return g.arrays()


def allreduce_rounds(n_ranks, rounds, k, seed=0, nbytes=1 << 20):
    rng = np.random.default_rng(seed)
    g = _Graph(n_ranks)
    colls = [g.collective(COLL_AR, nbytes) for _ in range(rounds)]
    for r in range(n_ranks):
        d = _durations(rng, rounds * k)
        comm = None
        for i, c in enumerate(colls):
            for j in range(k):
                g.op(r, S_COMPUTE, KIND_COMPUTE, int(d[i * k + j]), preds=[comm] if (j == 0 and comm is not None) else ())
            comm = g.op(r, S_TP, KIND_COMM, coll=c, preds=[len(g.rank) - 1])
        g.op(r, S_COMPUTE, KIND_COMPUTE, 1, preds=[comm])
    return g.arrays()


def p2p_pingpong(rounds, k, pairs=8, offset=None, seed=0, nbytes=1 << 20):
    """Ranks r and r + offset (r < pairs; offset defaults to pairs) pass a token: r
    runs k ops and sends; its partner receives, runs k ops and sends back; `rounds`
    round trips.  Ranks between the two groups have no ops."""
    rng = np.random.default_rng(seed)
    off = pairs if offset is None else offset
    n = off + pairs
    g = _Graph(n)
    fwd = [[g.collective(COLL_P2P, nbytes) for _ in range(rounds)] for _ in range(pairs)]
    bwd = [[g.collective(COLL_P2P, nbytes) for _ in range(rounds)] for _ in range(pairs)]
    for r in range(n):
        if pairs <= r < off:
            continue
        p, first = r % off, r < pairs
        d = _durations(rng, rounds * k)
        recv = None
        for i in range(rounds):
            if not first:        # the partner waits for the token before its k ops
                recv = g.op(r, S_RECV, KIND_COMM, coll=fwd[p][i])
            for j in range(k):
                g.op(r, S_COMPUTE, KIND_COMPUTE, int(d[i * k + j]), preds=[recv] if (j == 0 and recv is not None) else ())
            g.op(r, S_SEND, KIND_COMM, coll=(fwd if first else bwd)[p][i], preds=[len(g.rank) - 1])
            if first:            # the token comes back before the next round
                recv = g.op(r, S_RECV, KIND_COMM, coll=bwd[p][i])
        if recv is not None:
            g.op(r, S_COMPUTE, KIND_COMPUTE, 1, preds=[recv])
    return g.arrays()
