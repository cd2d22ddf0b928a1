"""Brute-force composer for tiny graphs: longest paths by enumerating every path.

Independent of the oracle's event queue: it lists every path of the merged
dependency graph (each collective is one node that all its member ops feed,
weighted by its running time; every other op is a node weighted by its
duration) and takes maxima over the lists.  Exponential; for <= ~25 nodes.
"""
from __future__ import annotations

import numpy as np

COMPUTE, COMM = 0, 1


class Cycle(Exception):
    pass


def _preds(g):
    n = len(g["op_rank"])
    last = {}
    preds = []
    for v in range(n):
        key = (int(g["op_rank"][v]), int(g["op_stream"][v]))
        p = set(int(u) for u in g["pred_idx"][g["pred_off"][v]:g["pred_off"][v + 1]])
        if key in last:
            p.add(last[key])
        last[key] = v
        preds.append(sorted(p))
    return preds


def all_paths_to(node, node_preds, stack=()):
    """Every path (tuple of nodes) that ends at `node`."""
    if node in stack:
        raise Cycle(node)
    yield (node,)
    for p in node_preds[node]:
        for path in all_paths_to(p, node_preds, stack + (node,)):
            yield path + (node,)


def compose(g, dur, cost):
    """Per-op start/finish by path enumeration. dur: per-op durations, cost: per-collective times."""
    n = len(g["op_rank"])
    kind, coll = g["op_kind"], g["op_coll"]
    preds = _preds(g)

    def node(v):
        return ("c", int(coll[v])) if kind[v] == COMM else ("o", v)

    node_preds, weight = {}, {}
    for v in range(n):
        x = node(v)
        node_preds.setdefault(x, set()).update(node(u) for u in preds[v])
        weight[x] = int(cost[x[1]]) if x[0] == "c" else int(dur[v])
    node_preds = {x: sorted(ps) for x, ps in node_preds.items()}
    longest = {x: max(sum(weight[y] for y in path) for path in all_paths_to(x, node_preds))
               for x in node_preds}
    s = np.zeros(n, np.int64)
    f = np.zeros(n, np.int64)
    for v in range(n):
        s[v] = max([longest[node(u)] for u in preds[v]], default=0)
        f[v] = longest[node(v)]
    return s, f


def factors(g, s, f, slowdown):
    """Slowdown factor of every op by checking every (compute, comm) pair of a rank."""
    n = len(g["op_rank"])
    F = np.full(n, 65536, np.int64)
    for v in range(n):
        if g["op_kind"][v] != COMPUTE:
            continue
        for c in range(n):
            if g["op_kind"][c] == COMM and g["op_rank"][c] == g["op_rank"][v]:
                if max(s[v], s[c]) < min(f[v], f[c]):
                    F[v] = max(F[v], int(slowdown[g["op_class"][v]][g["coll_type"][g["op_coll"][c]]]))
    return F


def compose_validated(g, base, cost, slowdown, n_refine):
    """Pass 1 with base durations, then n_refine rounds of overlap -> inflate -> recompose."""
    s, f = compose(g, base, cost)
    for _ in range(n_refine):
        F = factors(g, s, f, slowdown)
        d = np.array([(int(base[v]) * int(F[v]) + 32768) >> 16 if g["op_kind"][v] == COMPUTE
                      else int(base[v]) for v in range(len(base))], np.int64)
        s, f = compose(g, d, cost)
    return s, f


def covered(g, s, f, v):
    """Nanoseconds of [s_v, f_v) during which some comm op of v's rank runs: the
    endpoints of all these intervals cut the time axis into pieces on which coverage is
    constant; each piece inside [s_v, f_v) that lies inside some comm interval counts
    whole."""
    comm = [c for c in range(len(g["op_rank"]))
            if g["op_kind"][c] == COMM and g["op_rank"][c] == g["op_rank"][v]]
    cuts = sorted({int(s[v]), int(f[v])} | {int(s[c]) for c in comm} | {int(f[c]) for c in comm})
    total = 0
    for a, b in zip(cuts, cuts[1:]):
        if s[v] <= a and b <= f[v] and any(s[c] <= a and b <= f[c] for c in comm):
            total += b - a
    return total


def forest_predict(forest, x):
    """Walk every tree from its root (left when x[feature] < threshold), add the leaves
    to the base score, keep the sum inside [65536, 2^20)."""
    nodes = forest["nodes"]
    total = int(forest["base"])
    for root in forest["roots"]:
        i = int(root)
        while nodes[i]["feature"] >= 0:
            i = int(nodes[i]["left"] if x[nodes[i]["feature"]] < nodes[i]["threshold"] else nodes[i]["right"])
        total += int(nodes[i]["value"])
    return min(max(total, 65536), (1 << 20) - 1)


def factors_forest(g, s, f, forest, knobs):
    """Ensemble factors by checking every (compute, comm) pair of a rank: per collective
    type overlapping v, the largest message and member count, then the largest prediction.
    knobs: (ar_algo, bw_intra, bw_inter)."""
    n = len(g["op_rank"])
    coll, ctype = g["op_coll"], g["coll_type"]
    members = np.bincount(coll[g["op_kind"] == COMM], minlength=len(ctype)) if len(ctype) else np.zeros(0, np.int64)
    if g.get("coll_N") is not None:
        members = np.asarray(g["coll_N"])
    F = np.full(n, 65536, np.int64)
    for v in range(n):
        if g["op_kind"][v] != COMPUTE:
            continue
        smax, nmax = {}, {}
        for c in range(n):
            if g["op_kind"][c] == COMM and g["op_rank"][c] == g["op_rank"][v] and max(s[v], s[c]) < min(f[v], f[c]):
                t = int(ctype[coll[c]])
                smax[t] = max(smax.get(t, -1), int(g["coll_bytes"][coll[c]]))
                nmax[t] = max(nmax.get(t, 0), int(members[coll[c]]))
        cls = int(g["op_class"][v])
        for t in smax:
            x = [cls, int(g["op_dur"][v]), t, smax[t], nmax[t], *knobs] + [int(m) for m in forest["class_metrics"][cls]]
            F[v] = max(F[v], forest_predict(forest, x))
    return F


def compose_variants(g, base, cost, slowdown, n_refine, *, until_stable=False, prorate=False, forest=None,
                     knobs=(0, 400000, 50000)):
    """Validator variants: refine at most n_refine times, stopping early (until_stable) when
    a refinement would change no duration; prorate inflates only the covered part of a
    compute op (the covered time of the previous timeline, capped at the base duration).
    Returns (s, f, refinements composed)."""
    q16 = lambda d, F: (int(d) * int(F) + 32768) >> 16
    n = len(base)
    d = np.array(base, np.int64)
    s, f = compose(g, d, cost)
    done = 0
    for _ in range(n_refine):
        F = factors(g, s, f, slowdown) if forest is None else factors_forest(g, s, f, forest, knobs)
        new = d.copy()
        for v in range(n):
            if g["op_kind"][v] != COMPUTE:
                continue
            if prorate:
                o = min(covered(g, s, f, v), int(base[v]))
                new[v] = int(base[v]) - o + q16(o, F[v])
            else:
                new[v] = q16(base[v], F[v])
        if until_stable and (new == d).all():
            break
        d = new
        s, f = compose(g, d, cost)
        done += 1
    return s, f, done
