"""Hand-built execution graphs for the tests (same array layout as workloads.gpt1f1b)."""
from __future__ import annotations

import numpy as np

COMPUTE, COMM, MEMCPY = 0, 1, 2
AR, AG, RS, P2P = 0, 1, 2, 3


class Builder:
    """Append ops in rank-major program order; collectives are declared first."""

    def __init__(self, n_ranks, gpus_per_node=8):
        self.n_ranks, self.gpn = n_ranks, gpus_per_node
        self.rank, self.stream, self.kind, self.cls, self.dur, self.coll, self.preds = ([] for _ in range(7))
        self.ctype, self.cbytes = [], []

    def collective(self, ctype, nbytes):
        self.ctype.append(ctype)
        self.cbytes.append(nbytes)
        return len(self.ctype) - 1

    def op(self, rank, *, stream=0, kind=COMPUTE, cls=0, dur=0, coll=-1, preds=()):
        self.rank.append(rank)
        self.stream.append(stream)
        self.kind.append(kind)
        self.cls.append(cls)
        self.dur.append(dur)
        self.coll.append(coll)
        self.preds.append(list(preds))
        return len(self.rank) - 1

    def compute(self, rank, dur, *, stream=0, cls=0, preds=()):
        return self.op(rank, stream=stream, kind=COMPUTE, cls=cls, dur=dur, preds=preds)

    def comm(self, rank, coll, *, stream=1, preds=()):
        return self.op(rank, stream=stream, kind=COMM, cls=7, coll=coll, preds=preds)

    def graph(self):
        pc = [len(p) for p in self.preds]
        off = np.zeros(len(pc) + 1, np.int64)
        np.cumsum(pc, out=off[1:])
        return {
            "op_rank": np.array(self.rank, np.int32),
            "op_stream": np.array(self.stream, np.uint8),
            "op_kind": np.array(self.kind, np.uint8),
            "op_class": np.array(self.cls, np.uint8),
            "op_dur": np.array(self.dur, np.int64),
            "op_coll": np.array(self.coll, np.int64),
            "pred_off": off,
            "pred_idx": np.array([u for p in self.preds for u in p], np.int32),
            "coll_type": np.array(self.ctype, np.uint8),
            "coll_bytes": np.array(self.cbytes, np.int64),
            "n_ranks": self.n_ranks,
            "gpus_per_node": self.gpn,
        }


def pipeline_1f1b(P, m, tf, tb, gpus_per_node=8):
    """Pure 1F1B pipeline: one forward and one backward kernel per (stage,
    microbatch), activations/gradients exchanged by P2P pairs (zero bytes)."""
    b = Builder(P, gpus_per_node)
    ids = {}

    def pid(kind, boundary, mb):
        key = (kind, boundary, mb)
        if key not in ids:
            ids[key] = b.collective(P2P, 0)
        return ids[key]

    for p in range(P):           # declare collectives in a fixed order first
        for k in range(m):
            if p < P - 1:
                pid("f", p, k)
                pid("b", p, k)
    for p in range(P):
        last = [None]
        wait = []

        def compute(d):
            nonlocal wait
            v = b.compute(p, d, preds=wait)
            wait = []
            last[0] = v

        def comm(c, stream, blocking):
            v = b.comm(p, c, stream=stream, preds=[last[0]] if last[0] is not None else [])
            if blocking:
                wait.append(v)

        W = min(P - p - 1, m)
        R = m - W
        k = j = 0
        for _ in range(W):
            if p > 0:
                comm(pid("f", p - 1, k), 4, True)
            compute(tf)
            if p < P - 1:
                comm(pid("f", p, k), 3, False)
            k += 1
        if R > 0 and p > 0:
            comm(pid("f", p - 1, k), 4, True)
        for i in range(R):
            compute(tf)
            if p < P - 1:
                comm(pid("f", p, k), 3, False)
                comm(pid("b", p, j), 4, True)
            k += 1
            compute(tb)
            if p > 0:
                comm(pid("b", p - 1, j), 3, False)
                if i < R - 1:
                    comm(pid("f", p - 1, k), 4, True)
            j += 1
        for _ in range(W):
            comm(pid("b", p, j), 4, True)
            compute(tb)
            if p > 0:
                comm(pid("b", p - 1, j), 3, False)
            j += 1
    return b.graph()
