"""CPU oracle of Echo's timeline composer (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never does, and the two share no code: the oracle is the
plain C event-driven replay in ``echo_oracle.c``, built with gcc.

``run(graph, scen, n_refine)`` returns scenario-major arrays; see ``oracle_run``
in echo_oracle.c for the rules it follows and the paper passages they come from.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "echo_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

ERRORS = {0: "OK", -1: "ARG", -2: "RANGE", -3: "MATCH", -4: "CYCLE", -5: "NOMEM"}


class OracleError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"oracle error {code} ({ERRORS.get(code, '?')}): {msg}")
        self.code = code


def build() -> str:
    """Compile the oracle with gcc (always rebuilds)."""
    tmp = _LIB + ".tmp"
    subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-pthread",
                    "-o", tmp, _SRC], check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i64, i32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
    lib.oracle_run.restype = ctypes.c_int
    lib.oracle_run.argtypes = [i64, i32, i32] + [P] * 8 + [i64, P, P, P, P, P, i32] + [P] * 8 \
        + [P, P, i32, P] + [P] + [P, i64, P, i32, i32, P] + [i32, i32, i32, i32] + [P] * 7 \
        + [ctypes.c_char_p, i64]
    lib.oracle_chunk_bytes.restype = i64
    lib.oracle_chunk_bytes.argtypes = [i64]
    lib.oracle_cc_time.restype = i64
    lib.oracle_cc_time.argtypes = [i32, i64, i64, i64, i64, i64, i64, i64, i64, i32, i32, P]
    lib.oracle_splitmix64_at.restype = u64
    lib.oracle_splitmix64_at.argtypes = [u64, u64]
    lib.oracle_q16.restype = i64
    lib.oracle_q16.argtypes = [i64, u64]
    lib.oracle_mix64.restype = u64
    lib.oracle_mix64.argtypes = [u64]
    _lib = lib
    return lib


# One node of a tree ensemble (the oracle's tree_node_t): feature index (-1: leaf),
# children, leaf value (Q16), threshold (left when x[feature] < threshold).
TREE_NODE_DTYPE = np.dtype([("feature", "<i4"), ("left", "<i4"), ("right", "<i4"), ("value", "<i4"),
                            ("threshold", "<i8")])


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def run(graph: dict, scen: dict, n_refine: int = 1, *, threads: int = 1, timelines: bool = True,
        costs: bool = False, factors: bool = False, jitter_stream=None, until_stable: bool = False,
        prorate: bool = False, cc_tables=None, forest=None) -> dict:
    """Compose every scenario of `scen` on `graph`.

    Returns a dict with 'step' [n_scen] int64 and 'digest' [n_scen] uint64, plus
    'start'/'finish' [n_scen, n_ops] int64 (timelines=True), 'cost'
    [n_scen, n_colls] int64 (costs=True) and 'factor' [n_scen, n_ops] uint32
    (factors=True), and 'refinements' [n_scen] int32: the refined passes composed.
    until_stable: refine until a refinement would change no duration (at most
    n_refine times); prorate: inflate only the overlapped part of a compute op.
    cc_tables: int64 [n_tables, 6, 7] CC parameter tables that scenarios name with
    cc_table = index + 1 (scenario fields cc_model / cc_table default to 0).
    forest: a tree ensemble {'nodes': TREE_NODE_DTYPE array, 'roots': int32 [n_trees],
    'base': Q16 base score, 'class_metrics': int64 [8, 4]} whose predictions replace
    the scenario's slowdown table.
    jitter_stream defaults to the scenario's index in `scen`.
    Raises OracleError on invalid input or a deadlocked graph.
    """
    lib = _load()
    g = {k: graph[k] for k in ("op_rank", "op_stream", "op_kind", "op_class", "op_dur",
                                "op_coll", "pred_off", "pred_idx", "coll_type", "coll_bytes")}
    op_rank = _c(g["op_rank"], np.int32)
    op_stream = _c(g["op_stream"], np.uint8)
    op_kind = _c(g["op_kind"], np.uint8)
    op_class = _c(g["op_class"], np.uint8)
    op_dur = _c(g["op_dur"], np.int64)
    op_coll = _c(g["op_coll"], np.int64)
    pred_off = _c(g["pred_off"], np.int64)
    pred_idx = _c(g["pred_idx"], np.int32)
    coll_type = _c(g["coll_type"], np.uint8)
    coll_bytes = _c(g["coll_bytes"], np.int64)
    n_ops, n_colls = op_rank.shape[0], coll_type.shape[0]
    # optional membership the costs use (one DP replica simulated alone)
    given = [None if graph.get(k) is None else _c(graph[k], np.int32) for k in ("coll_N", "coll_M", "coll_K")]
    if any(x is not None and x.shape[0] != n_colls for x in given):
        raise OracleError(-1, "coll_N, coll_M and coll_K must have n_colls entries")
    if pred_off.shape[0] != n_ops + 1:
        raise OracleError(-1, "pred_off must have n_ops + 1 entries")
    n = int(np.asarray(scen["alpha_ns"]).shape[0])
    alpha = _c(scen["alpha_ns"], np.int64)
    bwa = _c(scen["bw_intra_MBps"], np.int64)
    bwe = _c(scen["bw_inter_MBps"], np.int64)
    red = _c(scen["reduce_MBps"], np.int64)
    jseed = _c(scen["jitter_seed"], np.uint64)
    if jitter_stream is None:
        jitter_stream = scen.get("jitter_stream", np.arange(n))
    jstream = _c(jitter_stream, np.uint32)
    jamp = _c(scen["jitter_amp_q16"], np.int32)
    algo = _c(scen["ar_algo"], np.uint8)
    ccm = _c(scen["cc_model"], np.uint8) if "cc_model" in scen else np.zeros(n, np.uint8)
    cct = _c(scen["cc_table"], np.int32) if "cc_table" in scen else np.zeros(n, np.int32)
    tables = np.zeros((0, 6, 7), np.int64) if cc_tables is None else _c(cc_tables, np.int64).reshape(-1, 6, 7)
    if forest is not None:
        f_nodes = np.ascontiguousarray(forest["nodes"], TREE_NODE_DTYPE)
        f_roots = _c(forest["roots"], np.int32)
        f_metrics = _c(forest["class_metrics"], np.int64).reshape(8, 4)
        f_args = (_p(f_nodes), int(f_nodes.shape[0]), _p(f_roots), int(f_roots.shape[0]), int(forest["base"]),
                  _p(f_metrics))
    else:
        f_args = (None, 0, None, 0, 0, None)
    slow = _c(scen["slowdown_q16"], np.uint32).reshape(n, 8, 4)
    out = {"step": np.zeros(n, np.int64), "digest": np.zeros(n, np.uint64),
           "refinements": np.zeros(n, np.int32)}
    if timelines:
        out["start"] = np.zeros((n, n_ops), np.int64)
        out["finish"] = np.zeros((n, n_ops), np.int64)
    if costs:
        out["cost"] = np.zeros((n, n_colls), np.int64)
    if factors:
        out["factor"] = np.zeros((n, n_ops), np.uint32)
    err = ctypes.create_string_buffer(512)
    rc = lib.oracle_run(
        n_ops, int(graph["n_ranks"]), int(graph["gpus_per_node"]),
        _p(op_rank), _p(op_stream), _p(op_kind), _p(op_class), _p(op_dur), _p(op_coll),
        _p(pred_off), _p(pred_idx), n_colls, _p(coll_type), _p(coll_bytes), *[_p(x) for x in given],
        n, _p(alpha), _p(bwa), _p(bwe), _p(red), _p(jseed), _p(jstream), _p(jamp), _p(algo), _p(ccm), _p(cct),
        int(tables.shape[0]), _p(tables) if tables.shape[0] else None, _p(slow), *f_args,
        int(n_refine), int(bool(until_stable)), int(bool(prorate)), int(max(1, threads)),
        _p(out.get("start")), _p(out.get("finish")), _p(out["step"]), _p(out["digest"]),
        _p(out.get("cost")), _p(out.get("factor")), _p(out["refinements"]), err, 512)
    if rc != 0:
        raise OracleError(rc, err.value.decode(errors="replace"))
    return out


def chunk_bytes(S: int) -> int:
    return int(_load().oracle_chunk_bytes(S))


def cc_time(ctype, S, N, M, K, *, alpha, bw_intra, bw_inter, reduce, algo=0, cc_model=0, table=None) -> int:
    """Cost of one collective; table: an int64 [6, 7] CC parameter table or None."""
    t = None if table is None else _c(table, np.int64).reshape(6, 7)
    return int(_load().oracle_cc_time(ctype, S, N, M, K, alpha, bw_intra, bw_inter, reduce, algo, cc_model,
                                      _p(t)))


def splitmix64_at(seed: int, k: int) -> int:
    return int(_load().oracle_splitmix64_at(seed, k))


def q16(d: int, f: int) -> int:
    return int(_load().oracle_q16(d, f))


def mix64(z: int) -> int:
    return int(_load().oracle_mix64(z))
