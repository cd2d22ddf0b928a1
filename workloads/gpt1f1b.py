"""Synthetic per-rank execution graphs of Megatron-style GPT training (TP x PP x DP, 1F1B).

The paper's workload tracer (Sec. 4.1) replays every rank of a real training job
on one device and records each rank's execution graph: operators, their
dependencies, the measured durations of computation operators, and placeholders
for communication operators (group and message size).  Those traces need the
real frameworks and models, so this module synthesises graphs of the same shape
instead: GPT models from the paper's model table (Table 9), Megatron tensor
parallel all-reduces, 1F1B pipeline send/recv pairs and DDP gradient buckets.

It produces inputs only.  Nothing here costs a collective, composes a timeline
or applies a slowdown.

Graph arrays (a dict of numpy arrays; ops are rank-major and, within a rank,
in program (issue) order):

    op_rank   int32 [n_ops]    rank that issues the op
    op_stream uint8 [n_ops]    stream id on that rank (0..7)
    op_kind   uint8 [n_ops]    KIND_COMPUTE / KIND_COMM / KIND_MEMCPY
    op_class  uint8 [n_ops]    kernel class 0..7 (row of the slowdown table)
    op_dur    int64 [n_ops]    base duration in ns (0 for comm ops)
    op_coll   int64 [n_ops]    collective id of a comm op, -1 otherwise
    pred_off  int64 [n_ops+1]  CSR offsets of explicit same-rank dependencies
    pred_idx  int32 [n_edges]  dependency op ids (always an earlier op of the same rank)
    coll_type uint8 [n_colls]  COLL_AR / COLL_AG / COLL_RS / COLL_P2P
    coll_bytes int64 [n_colls] message size S in bytes
    n_ranks, gpus_per_node     ints

Stream-order edges (each op waits for the previous op on its stream) are not
listed: they follow from ``op_stream`` and program order.

Stream use: 0 compute, 1 tensor-parallel comm, 2 data-parallel comm,
3 pipeline send, 4 pipeline recv, 5 host-to-device memcpy.
Rank numbering: rank = tp + TP * (dp + DP * pp).
"""
from __future__ import annotations

import numpy as np

KIND_COMPUTE, KIND_COMM, KIND_MEMCPY = 0, 1, 2
COLL_AR, COLL_AG, COLL_RS, COLL_P2P = 0, 1, 2, 3
(CLS_GEMM, CLS_TRANSFORM, CLS_SUM, CLS_GRAD,
 CLS_LAYERNORM, CLS_ATTN, CLS_OPTIMIZER, CLS_OTHER) = range(8)
S_COMPUTE, S_TP, S_DP, S_SEND, S_RECV, S_MEMCPY = range(6)

BUCKET_BYTES = 25 * 1024 * 1024          # DDP default gradient bucket (25 MiB)
VOCAB = 51200                            # padded GPT vocabulary
BYTES_PER_ELEM = 2                       # bf16 activations and gradients
COMPUTE_MEDIAN_NS = 50_000.0             # lognormal median of a compute kernel
MEMCPY_MEDIAN_NS = 5_000.0               # lognormal median of a host-to-device copy
LOG_SIGMA = 0.5

# Collective group kinds used while building a stage template.
_G_TP, _G_DP, _G_P2P = 0, 1, 2
_DUR_COMPUTE, _DUR_MEMCPY, _DUR_NONE = 0, 1, 2

# One transformer layer, forward: (class, all-reduce after this op?)
_FWD_LAYER = [
    (CLS_LAYERNORM, 0), (CLS_GEMM, 0), (CLS_SUM, 0), (CLS_TRANSFORM, 0),
    (CLS_TRANSFORM, 0), (CLS_ATTN, 0), (CLS_OTHER, 0), (CLS_ATTN, 0),
    (CLS_OTHER, 0), (CLS_ATTN, 0), (CLS_TRANSFORM, 0), (CLS_GEMM, 1),   # out-proj -> TP AR
    (CLS_SUM, 0), (CLS_OTHER, 0), (CLS_SUM, 0), (CLS_LAYERNORM, 0),
    (CLS_GEMM, 0), (CLS_SUM, 0), (CLS_OTHER, 0), (CLS_GEMM, 1),         # fc2 -> TP AR
    (CLS_SUM, 0), (CLS_OTHER, 0), (CLS_SUM, 0), (CLS_TRANSFORM, 0),
    (CLS_TRANSFORM, 0),
]
# One transformer layer, backward (50 kernels, two input-gradient all-reduces).
_BWD_LAYER = [
    (CLS_SUM, 0), (CLS_GRAD, 0), (CLS_GRAD, 0), (CLS_GEMM, 0), (CLS_GEMM, 0),
    (CLS_GRAD, 0), (CLS_GRAD, 0), (CLS_GEMM, 1),                        # fc1 dgrad -> TP AR
    (CLS_GEMM, 0), (CLS_LAYERNORM, 0), (CLS_GRAD, 0), (CLS_SUM, 0),
    (CLS_GRAD, 0), (CLS_GRAD, 0), (CLS_GEMM, 0), (CLS_GEMM, 0),
    (CLS_TRANSFORM, 0), (CLS_ATTN, 0), (CLS_ATTN, 0), (CLS_GRAD, 0),
    (CLS_ATTN, 0), (CLS_GRAD, 0), (CLS_ATTN, 0), (CLS_ATTN, 0),
    (CLS_TRANSFORM, 0), (CLS_TRANSFORM, 0), (CLS_GRAD, 0), (CLS_GEMM, 1),  # qkv dgrad -> TP AR
    (CLS_GEMM, 0), (CLS_LAYERNORM, 0), (CLS_GRAD, 0), (CLS_SUM, 0),
] + [(CLS_SUM, 0)] * 12 + [
    (CLS_TRANSFORM, 0), (CLS_OTHER, 0), (CLS_TRANSFORM, 0), (CLS_OTHER, 0),
    (CLS_GRAD, 0), (CLS_OTHER, 0),
]
assert len(_FWD_LAYER) == 25 and len(_BWD_LAYER) == 50


class _Stage:
    """Program (issue order) of one pipeline stage, shared by its TP x DP ranks."""

    def __init__(self):
        self.kind, self.stream, self.cls, self.durk = [], [], [], []
        self.preds, self.gkind, self.gj = [], [], []
        self.last_compute = -1
        self.wait_for = []            # ops the next compute op must depend on
        self.tp_specs, self.dp_specs = [], []   # (coll_type, bytes) per group collective

    def _add(self, kind, stream, cls, durk, preds, gkind=-1, gj=-1):
        self.kind.append(kind)
        self.stream.append(stream)
        self.cls.append(cls)
        self.durk.append(durk)
        self.preds.append(preds)
        self.gkind.append(gkind)
        self.gj.append(gj)
        return len(self.kind) - 1

    def compute(self, cls, extra=()):
        preds = self.wait_for + list(extra)
        self.wait_for = []
        i = self._add(KIND_COMPUTE, S_COMPUTE, cls, _DUR_COMPUTE, preds)
        self.last_compute = i
        return i

    def _after_compute(self):
        return [self.last_compute] if self.last_compute >= 0 else []

    def memcpy(self, blocking):
        i = self._add(KIND_MEMCPY, S_MEMCPY, CLS_OTHER, _DUR_MEMCPY, self._after_compute())
        if blocking:
            self.wait_for.append(i)
        return i

    def tp(self, ctype, nbytes, blocking=True):
        j = len(self.tp_specs)
        self.tp_specs.append((ctype, nbytes))
        i = self._add(KIND_COMM, S_TP, CLS_OTHER, _DUR_NONE, self._after_compute(), _G_TP, j)
        if blocking:
            self.wait_for.append(i)
        return i

    def dp(self, ctype, nbytes):
        j = len(self.dp_specs)
        self.dp_specs.append((ctype, nbytes))
        return self._add(KIND_COMM, S_DP, CLS_OTHER, _DUR_NONE, self._after_compute(), _G_DP, j)

    def p2p(self, stream, code, blocking):
        i = self._add(KIND_COMM, stream, CLS_OTHER, _DUR_NONE, self._after_compute(), _G_P2P, code)
        if blocking:
            self.wait_for.append(i)
        return i


def _layer_param_bytes(h, tp):
    return BYTES_PER_ELEM * ((12 * h * h + 13 * h) // tp)


def _build_stage(p, P, tp, dp, m, n_layers, h, seq, distopt):
    """Issue order of stage p under Megatron's non-interleaved 1F1B schedule."""
    st = _Stage()
    first, last = p == 0, p == P - 1
    ls = n_layers // P
    act = seq * h * BYTES_PER_ELEM            # microbatch 1: b*s*h bf16 activation
    small = seq * 4                            # fp32 per-token reductions of the loss
    use_tp = tp > 1

    # Gradient buckets of the stage, in the order their gradients become ready.
    ready = []                                  # (when, bytes); when = layer index or a tag
    if last:
        ready.append(("head", BYTES_PER_ELEM * 2 * h))
    for layer in reversed(range(ls)):
        ready.append((layer, _layer_param_bytes(h, tp)))
    if first:
        ready.append(("embed", BYTES_PER_ELEM * (VOCAB * h // tp + seq * h)))
    bucket = {"cum": 0, "issued": 0, "ops": [], "sizes": []}

    def grads_ready(tag):
        for when, nbytes in ready:
            if when == tag:
                bucket["cum"] += nbytes
        while (bucket["issued"] + 1) * BUCKET_BYTES <= bucket["cum"]:
            issue_bucket(BUCKET_BYTES)

    def issue_bucket(nbytes):
        bucket["issued"] += 1
        bucket["sizes"].append(nbytes)
        if dp > 1:
            bucket["ops"].append(st.dp(COLL_RS if distopt else COLL_AR, nbytes))
        else:
            bucket["ops"].append(-1)

    def p2p_code(boundary, direction, mb):
        return (boundary * 2 + direction) * m + mb

    def recv_forward(mb):
        if not first:
            st.p2p(S_RECV, p2p_code(p - 1, 0, mb), blocking=True)

    def send_forward(mb):
        if not last:
            st.p2p(S_SEND, p2p_code(p, 0, mb), blocking=False)

    def recv_backward(mb):
        if not last:
            st.p2p(S_RECV, p2p_code(p, 1, mb), blocking=True)

    def send_backward(mb):
        if not first:
            st.p2p(S_SEND, p2p_code(p - 1, 1, mb), blocking=False)

    def forward_step(mb):
        labels = -1
        if first:
            st.memcpy(blocking=True)                      # token ids to the device
            st.compute(CLS_OTHER)                         # embedding lookup
            if use_tp:
                st.tp(COLL_AR, act)                       # vocab-parallel embedding reduce
            st.compute(CLS_OTHER)                         # embedding dropout
        if last:
            labels = st.memcpy(blocking=False)            # labels to the device
        for _ in range(ls):
            for cls, ar in _FWD_LAYER:
                st.compute(cls)
                if ar and use_tp:
                    st.tp(COLL_AR, act)
        if last:
            st.compute(CLS_LAYERNORM)                     # final layernorm
            st.compute(CLS_GEMM)                          # vocab-parallel logits
            if use_tp:
                st.tp(COLL_AR, small)                     # logit max
            st.compute(CLS_OTHER)                         # exp / partial sums
            if use_tp:
                st.tp(COLL_AR, small)                     # sum of exp
            st.compute(CLS_SUM, extra=[labels])           # loss

    def backward_step(mb):
        last_mb = mb == m - 1
        if last:
            st.compute(CLS_GRAD)
            st.compute(CLS_GRAD)
            st.compute(CLS_GEMM)                          # logits dgrad
            if use_tp:
                st.tp(COLL_AR, act)
            st.compute(CLS_GEMM)                          # logits wgrad
            st.compute(CLS_LAYERNORM)                     # final layernorm backward
            if last_mb:
                grads_ready("head")
        for layer in reversed(range(ls)):
            for cls, ar in _BWD_LAYER:
                st.compute(cls)
                if ar and use_tp:
                    st.tp(COLL_AR, act)
            if last_mb:
                grads_ready(layer)
        if first:
            st.compute(CLS_GRAD)                          # embedding gradient
            if last_mb:
                grads_ready("embed")
        if last_mb and bucket["cum"] > bucket["issued"] * BUCKET_BYTES:
            issue_bucket(bucket["cum"] - bucket["issued"] * BUCKET_BYTES)

    warmup = min(P - p - 1, m)
    steady = m - warmup
    fwd_mb = bwd_mb = 0
    for _ in range(warmup):
        recv_forward(fwd_mb)
        forward_step(fwd_mb)
        send_forward(fwd_mb)
        fwd_mb += 1
    if steady > 0:
        recv_forward(fwd_mb)
    for i in range(steady):
        forward_step(fwd_mb)
        send_forward(fwd_mb)                 # batched with the recv below
        recv_backward(bwd_mb)
        fwd_mb += 1
        backward_step(bwd_mb)
        if i == steady - 1:
            send_backward(bwd_mb)
        else:
            send_backward(bwd_mb)            # batched with the recv below
            recv_forward(fwd_mb)
        bwd_mb += 1
    for _ in range(warmup):
        recv_backward(bwd_mb)
        backward_step(bwd_mb)
        send_backward(bwd_mb)
        bwd_mb += 1
    assert fwd_mb == m and bwd_mb == m

    # Optimizer: one kernel per gradient bucket once its reduction is done,
    # then (distributed optimizer) an all-gather of the updated parameter shard.
    for op, nbytes in zip(bucket["ops"], bucket["sizes"]):
        st.compute(CLS_OPTIMIZER, extra=[op] if op >= 0 else [])
        if distopt and dp > 1:
            st.dp(COLL_AG, nbytes)
    return st


def gpt_graph(*, n_layers, hidden, seq, tp, pp, dp, microbatches, seed,
              distopt=False, gpus_per_node=8, replica_invariant=False):
    """Build the execution graphs of all TP*PP*DP ranks of one training step.

    replica_invariant: every data-parallel replica gets the same durations (one
    draw per pipeline stage, tensor-parallel rank and op), as when a single
    replica is traced and copied."""
    if n_layers % pp:
        raise ValueError("n_layers must be divisible by pp")
    P, T, D, m = pp, tp, dp, microbatches
    stages = [_build_stage(p, P, T, D, m, n_layers, hidden, seq, distopt) for p in range(P)]

    # Collective id layout: TP groups, then DP groups, then pipeline pairs.
    n_tp = [len(s.tp_specs) for s in stages]
    n_dp = [len(s.dp_specs) for s in stages]
    tp_off = np.concatenate([[0], np.cumsum([D * n for n in n_tp])]).astype(np.int64)
    dp_off = np.concatenate([[0], np.cumsum([T * n for n in n_dp])]).astype(np.int64)
    dp_base = int(tp_off[-1])
    p2p_base = dp_base + int(dp_off[-1])
    n_p2p = max(P - 1, 0) * 2 * m * D * T
    n_colls = p2p_base + n_p2p
    coll_type = np.empty(n_colls, np.uint8)
    coll_bytes = np.empty(n_colls, np.int64)
    for p, s in enumerate(stages):
        if n_tp[p]:
            ct = np.array([c for c, _ in s.tp_specs], np.uint8)
            cb = np.array([b for _, b in s.tp_specs], np.int64)
            sl = slice(int(tp_off[p]), int(tp_off[p + 1]))
            coll_type[sl] = np.tile(ct, D)
            coll_bytes[sl] = np.tile(cb, D)
        if n_dp[p]:
            ct = np.array([c for c, _ in s.dp_specs], np.uint8)
            cb = np.array([b for _, b in s.dp_specs], np.int64)
            sl = slice(dp_base + int(dp_off[p]), dp_base + int(dp_off[p + 1]))
            coll_type[sl] = np.tile(ct, T)
            coll_bytes[sl] = np.tile(cb, T)
    coll_type[p2p_base:] = COLL_P2P
    coll_bytes[p2p_base:] = seq * hidden * BYTES_PER_ELEM

    # Instantiate every stage template for its T*D ranks (rank-major op ids).
    parts = {k: [] for k in ("rank", "stream", "kind", "cls", "durk", "coll", "pcount", "pidx")}
    base = 0
    q = np.arange(T * D, dtype=np.int64)
    tpi, dpi = q % T, q // T
    for p, s in enumerate(stages):
        n = len(s.kind)
        ranks = q + T * D * p
        bases = base + q * n
        parts["rank"].append(np.repeat(ranks.astype(np.int32), n))
        for key, src in (("stream", s.stream), ("kind", s.kind), ("cls", s.cls), ("durk", s.durk)):
            parts[key].append(np.tile(np.asarray(src, np.uint8), T * D))
        gk = np.asarray(s.gkind, np.int64)
        gj = np.asarray(s.gj, np.int64)
        coll = np.full((T * D, n), -1, np.int64)
        is_tp, is_dp, is_pp = gk == _G_TP, gk == _G_DP, gk == _G_P2P
        coll[:, is_tp] = tp_off[p] + dpi[:, None] * n_tp[p] + gj[None, is_tp]
        coll[:, is_dp] = dp_base + dp_off[p] + tpi[:, None] * n_dp[p] + gj[None, is_dp]
        coll[:, is_pp] = p2p_base + (gj[None, is_pp] * D + dpi[:, None]) * T + tpi[:, None]
        parts["coll"].append(coll.reshape(-1))
        pc = np.array([len(x) for x in s.preds], np.int64)
        pl = np.array([u for x in s.preds for u in x], np.int64)
        parts["pcount"].append(np.tile(pc, T * D))
        parts["pidx"].append((np.tile(pl, T * D) + np.repeat(bases, len(pl))).astype(np.int32))
        base += T * D * n

    n_ops = base
    durk = np.concatenate(parts["durk"])
    rng = np.random.default_rng(seed)
    if replica_invariant:
        z = np.concatenate([np.tile(rng.standard_normal((T, len(s.kind))), (D, 1)).reshape(-1) for s in stages]) \
            if n_ops else np.zeros(0)
    else:
        z = rng.standard_normal(n_ops)
    med = np.where(durk == _DUR_MEMCPY, MEMCPY_MEDIAN_NS, COMPUTE_MEDIAN_NS)
    dur = np.maximum(np.rint(med * np.exp(LOG_SIGMA * z)), 1.0).astype(np.int64)
    dur[durk == _DUR_NONE] = 0
    pcount = np.concatenate(parts["pcount"])
    pred_off = np.zeros(n_ops + 1, np.int64)
    np.cumsum(pcount, out=pred_off[1:])
    return {
        "op_rank": np.concatenate(parts["rank"]),
        "op_stream": np.concatenate(parts["stream"]),
        "op_kind": np.concatenate(parts["kind"]),
        "op_class": np.concatenate(parts["cls"]),
        "op_dur": dur,
        "op_coll": np.concatenate(parts["coll"]),
        "pred_off": pred_off,
        "pred_idx": np.concatenate(parts["pidx"]) if n_ops else np.zeros(0, np.int32),
        "coll_type": coll_type,
        "coll_bytes": coll_bytes,
        "n_ranks": P * T * D,
        "gpus_per_node": gpus_per_node,
    }


def dp_replica(graph: dict, tp: int, dp: int, replica: int = 0):
    """The graph of one data-parallel replica, as Echo's DDP mode simulates it
    (Sec. 8.5: one copy of the workload per DP group).

    Keeps the ranks with data-parallel index `replica` (rank = tp + TP*(dp + DP*pp)),
    renumbered tp + TP*pp, and every collective with a member among them.  Each
    kept collective carries the membership of its whole group -- coll_N members,
    coll_M distinct servers, coll_K most members on one server, from the full
    placement -- so its cost is unchanged while its barrier only involves the
    members kept.  Returns (replica graph, op_map) with op_map[new op] = old op.
    """
    rank = graph["op_rank"].astype(np.int64)
    keep = (rank // tp) % dp == replica
    op_map = np.flatnonzero(keep)
    new_id = np.full(rank.shape[0], -1, np.int64)
    new_id[op_map] = np.arange(op_map.shape[0])
    comm = graph["op_kind"] == KIND_COMM
    coll = graph["op_coll"]
    n_colls = graph["coll_type"].shape[0]
    # whole-group membership of every collective
    node = rank // int(graph["gpus_per_node"])
    cm = coll[comm]
    N = np.bincount(cm, minlength=n_colls)
    pairs, cnt = np.unique(np.stack([cm, node[comm]], 1), axis=0, return_counts=True) if cm.size else \
        (np.zeros((0, 2), np.int64), np.zeros(0, np.int64))
    M = np.bincount(pairs[:, 0], minlength=n_colls)
    K = np.zeros(n_colls, np.int64)
    np.maximum.at(K, pairs[:, 0], cnt)
    kept_colls = np.unique(coll[keep & comm])
    cmap = np.full(n_colls, -1, np.int64)
    cmap[kept_colls] = np.arange(kept_colls.shape[0])
    # dependencies: same-rank, so every predecessor of a kept op is kept
    pcount = np.diff(graph["pred_off"])[op_map]
    src = np.repeat(np.arange(rank.shape[0]), np.diff(graph["pred_off"]))
    pidx = graph["pred_idx"][keep[src]]
    pred_off = np.zeros(op_map.shape[0] + 1, np.int64)
    np.cumsum(pcount, out=pred_off[1:])
    r = rank[op_map]
    out = {
        "op_rank": ((r % tp) + tp * (r // (tp * dp))).astype(np.int32),
        "op_stream": graph["op_stream"][op_map],
        "op_kind": graph["op_kind"][op_map],
        "op_class": graph["op_class"][op_map],
        "op_dur": graph["op_dur"][op_map],
        "op_coll": np.where(coll[op_map] >= 0, cmap[np.maximum(coll[op_map], 0)], -1).astype(np.int64),
        "pred_off": pred_off,
        "pred_idx": new_id[pidx].astype(np.int32),
        "coll_type": graph["coll_type"][kept_colls],
        "coll_bytes": graph["coll_bytes"][kept_colls],
        "coll_N": N[kept_colls].astype(np.int32),
        "coll_M": M[kept_colls].astype(np.int32),
        "coll_K": K[kept_colls].astype(np.int32),
        "n_ranks": int(graph["n_ranks"]) // dp,
        "gpus_per_node": int(graph["gpus_per_node"]),
    }
    return out, op_map
