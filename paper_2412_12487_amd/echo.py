"""ctypes binding of libecho.so (argument marshalling only).

Every step of the composer runs inside the library's HIP kernels; this module
converts numpy graph arrays into an ``echo_graph_desc``, packs scenarios into
``echo_scenario`` records, allocates output tensors with torch and passes
their device pointers and the current HIP stream through the C ABI.
There is no fallback: if libecho.so is missing, importing the library fails.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import sys
import weakref

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libecho.so")

ECHO_OK, ECHO_ERR_ARG, ECHO_ERR_RANGE, ECHO_ERR_MATCH = 0, -1, -2, -3
ECHO_ERR_CYCLE, ECHO_ERR_NOMEM, ECHO_ERR_HIP, ECHO_ERR_DEVICE = -4, -5, -6, -7
ERROR_NAMES = {0: "OK", -1: "ARG", -2: "RANGE", -3: "MATCH", -4: "CYCLE", -5: "NOMEM", -6: "HIP",
               -7: "DEVICE"}
EXPORTS = ("echo_load_graph", "echo_load_graph_ex", "echo_graph_info", "echo_free_graph", "echo_cc_cost",
           "echo_compose_batch", "echo_compose_validated", "echo_set_cc_tables", "echo_set_forest",
           "echo_sync_status", "echo_set_timing", "echo_kernel_times", "echo_set_spin_limit",
           "echo_set_launch_tiles", "echo_walk_chain", "echo_compose_batch_static", "echo_last_error")
KERNEL_KINDS = {0: "init", 1: "cc_cost", 2: "walk", 3: "overlap", 4: "clear"}

# echo_scenario (include/echo.h): 192 bytes.
SCENARIO_DTYPE = np.dtype({
    "names": ["alpha_ns", "bw_intra_MBps", "bw_inter_MBps", "reduce_MBps", "jitter_seed",
              "jitter_stream", "jitter_amp_q16", "ar_algo", "cc_model", "cc_table", "slowdown_q16"],
    "formats": ["<i8", "<i8", "<i8", "<i8", "<u8", "<u4", "<i4", "u1", "u1", "<i4", ("<u4", (8, 4))],
    "offsets": [0, 8, 16, 24, 32, 40, 44, 48, 49, 52, 64],
    "itemsize": 192,
})
CC_ROWS = 7           # rows of a CC parameter table; as int64 [6, CC_ROWS]: max_bytes, chunk,
                      # alpha_ns, beta_ns, gamma_ns, reduce_MBps (the echo_cc_table layout)


class EchoError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libecho error {code} ({ERROR_NAMES.get(code, '?')}): {msg}")
        self.code = code


class _Desc(ctypes.Structure):
    _fields_ = [
        ("n_ops", ctypes.c_int64), ("n_ranks", ctypes.c_int32), ("gpus_per_node", ctypes.c_int32),
        ("op_rank", ctypes.c_void_p), ("op_stream", ctypes.c_void_p), ("op_kind", ctypes.c_void_p),
        ("op_class", ctypes.c_void_p), ("op_dur_ns", ctypes.c_void_p), ("op_coll", ctypes.c_void_p),
        ("pred_off", ctypes.c_void_p), ("pred_idx", ctypes.c_void_p), ("n_colls", ctypes.c_int64),
        ("coll_type", ctypes.c_void_p), ("coll_bytes", ctypes.c_void_p),
        ("coll_N", ctypes.c_void_p), ("coll_M", ctypes.c_void_p), ("coll_K", ctypes.c_void_p),
    ]


class _Validator(ctypes.Structure):
    _fields_ = [("max_refine", ctypes.c_int32), ("until_stable", ctypes.c_int32), ("prorate", ctypes.c_int32),
                ("forest", ctypes.c_int32)]


# echo_tree_node: feature (-1 leaf), left, right, value (Q16), threshold (left when x < threshold)
TREE_NODE_DTYPE = np.dtype([("feature", "<i4"), ("left", "<i4"), ("right", "<i4"), ("value", "<i4"),
                            ("threshold", "<i8")])


_lib = None


def lib():
    """The loaded libecho.so.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    # torch first: libecho.so then binds to the HIP runtime torch has loaded, so the process
    # has one.  Loaded the other way round, the library would bring in the system's runtime
    # first and torch could no longer open the GPU ("No HIP GPUs are available").
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.echo_load_graph.argtypes = [ctypes.POINTER(_Desc), ctypes.c_int, ctypes.POINTER(P)]
    L.echo_load_graph.restype = ctypes.c_int
    L.echo_load_graph_ex.argtypes = [ctypes.POINTER(_Desc), ctypes.c_int, ctypes.c_int32, ctypes.POINTER(P)]
    L.echo_load_graph_ex.restype = ctypes.c_int
    L.echo_graph_info.argtypes = [P, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)]
    L.echo_graph_info.restype = ctypes.c_int
    L.echo_free_graph.argtypes = [P]
    L.echo_free_graph.restype = None
    L.echo_cc_cost.argtypes = [P, P, i32, P, P]
    L.echo_cc_cost.restype = ctypes.c_int
    L.echo_compose_batch.argtypes = [P, P, i32, i32, P, P, P, P, P]
    L.echo_compose_batch.restype = ctypes.c_int
    L.echo_compose_validated.argtypes = [P, P, i32, ctypes.POINTER(_Validator), P, P, P, P, P, P]
    L.echo_compose_validated.restype = ctypes.c_int
    L.echo_set_cc_tables.argtypes = [P, P, i32]
    L.echo_set_cc_tables.restype = ctypes.c_int
    L.echo_set_forest.argtypes = [P, P, i64, P, i32, i32, P]
    L.echo_set_forest.restype = ctypes.c_int
    L.echo_sync_status.argtypes = [P, P]
    L.echo_sync_status.restype = ctypes.c_int
    L.echo_set_timing.argtypes = [P, ctypes.c_int]
    L.echo_set_timing.restype = ctypes.c_int
    L.echo_kernel_times.argtypes = [P, i32, P, P, ctypes.POINTER(i32)]
    L.echo_kernel_times.restype = ctypes.c_int
    L.echo_set_spin_limit.argtypes = [P, i64]
    L.echo_set_spin_limit.restype = ctypes.c_int
    L.echo_set_launch_tiles.argtypes = [P, i32]
    L.echo_set_launch_tiles.restype = ctypes.c_int
    L.echo_walk_chain.argtypes = [P, P, P]
    L.echo_walk_chain.restype = ctypes.c_int
    L.echo_compose_batch_static.argtypes = [P, P, i32, i32, P, P, P, P, P]
    L.echo_compose_batch_static.restype = ctypes.c_int
    L.echo_last_error.argtypes = []
    L.echo_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(rc):
    if rc != ECHO_OK:
        raise EchoError(rc, lib().echo_last_error().decode(errors="replace"))


def pack_scenarios(sc: dict) -> np.ndarray:
    """Scenario dict (workloads.scenarios layout) -> array of echo_scenario records."""
    n = int(np.asarray(sc["alpha_ns"]).shape[0])
    rec = np.zeros(n, SCENARIO_DTYPE)
    for k in ("alpha_ns", "bw_intra_MBps", "bw_inter_MBps", "reduce_MBps", "jitter_seed",
              "jitter_amp_q16", "ar_algo"):
        rec[k] = sc[k]
    rec["jitter_stream"] = sc["jitter_stream"] if "jitter_stream" in sc else np.arange(n)
    for k in ("cc_model", "cc_table"):
        if k in sc:
            rec[k] = sc[k]
    rec["slowdown_q16"] = np.asarray(sc["slowdown_q16"]).reshape(n, 8, 4)
    return rec


def scenarios_to_device(sc, device="cuda"):
    """Upload scenarios (dict or packed records) as a uint8 tensor; returns (tensor, n)."""
    import torch
    rec = sc if isinstance(sc, np.ndarray) else pack_scenarios(sc)
    t = torch.from_numpy(rec.view(np.uint8).copy()).to(device)
    return t, int(rec.shape[0])


def _device_buffer(t, name, device, nbytes, dtype=None):
    """Check that tensor t can take nbytes at its data pointer on `device`: a
    contiguous tensor of that device (and dtype), large enough."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise EchoError(ECHO_ERR_ARG, f"{name} must be a torch tensor")
    if t.device != device:
        raise EchoError(ECHO_ERR_ARG, f"{name} is on {t.device}, the graph on {device}")
    if not t.is_contiguous():
        raise EchoError(ECHO_ERR_ARG, f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise EchoError(ECHO_ERR_ARG, f"{name} must be {dtype} (got {t.dtype})")
    if t.numel() * t.element_size() < nbytes:
        raise EchoError(ECHO_ERR_ARG, f"{name} holds {t.numel() * t.element_size()} bytes, needs {nbytes}")
    return ctypes.c_void_p(t.data_ptr())


def _stream_ptr(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


# Graphs still open are freed at interpreter exit, before modules are torn down and
# while the HIP runtime (and any profiler attached to it) is still up; a graph
# collected later than that is left to the process's exit.
_open_graphs = weakref.WeakSet()


@atexit.register
def _close_open_graphs():
    for g in list(_open_graphs):
        g.close()


class Graph:
    """A loaded graph: validated, matched, levelled and resident on one GPU."""

    def __init__(self, arrays: dict, device: int = 0, ranks_per_walker: int = 0):
        L = lib()
        self._keep = {
            "op_rank": np.ascontiguousarray(arrays["op_rank"], np.int32),
            "op_stream": np.ascontiguousarray(arrays["op_stream"], np.uint8),
            "op_kind": np.ascontiguousarray(arrays["op_kind"], np.uint8),
            "op_class": np.ascontiguousarray(arrays["op_class"], np.uint8),
            "op_dur": np.ascontiguousarray(arrays["op_dur"], np.int64),
            "op_coll": np.ascontiguousarray(arrays["op_coll"], np.int64),
            "pred_off": np.ascontiguousarray(arrays["pred_off"], np.int64),
            "pred_idx": np.ascontiguousarray(arrays["pred_idx"], np.int32),
            "coll_type": np.ascontiguousarray(arrays["coll_type"], np.uint8),
            "coll_bytes": np.ascontiguousarray(arrays["coll_bytes"], np.int64),
        }
        nc = self._keep["coll_type"].shape[0]
        for key in ("coll_N", "coll_M", "coll_K"):       # optional: membership of partial collectives
            if arrays.get(key) is not None:
                self._keep[key] = np.ascontiguousarray(arrays[key], np.int32)
                if self._keep[key].shape[0] != nc:
                    raise EchoError(ECHO_ERR_ARG, f"{key} must have n_colls entries")
        k = self._keep
        n = k["op_rank"].shape[0]
        if k["pred_off"].shape[0] != n + 1:
            raise EchoError(ECHO_ERR_ARG, "pred_off must have n_ops + 1 entries")
        ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
        opt = lambda key: ptr(k[key]) if key in k else None
        d = _Desc(n, int(arrays["n_ranks"]), int(arrays["gpus_per_node"]),
                  ptr(k["op_rank"]), ptr(k["op_stream"]), ptr(k["op_kind"]), ptr(k["op_class"]),
                  ptr(k["op_dur"]), ptr(k["op_coll"]), ptr(k["pred_off"]), ptr(k["pred_idx"]),
                  nc, ptr(k["coll_type"]), ptr(k["coll_bytes"]),
                  opt("coll_N"), opt("coll_M"), opt("coll_K"))
        h = ctypes.c_void_p()
        _check(L.echo_load_graph_ex(ctypes.byref(d), int(device), int(ranks_per_walker), ctypes.byref(h)))
        self._keep = None
        self.handle = h
        self.device = int(device)
        a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(L.echo_graph_info(h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
        self.n_ops, self.n_colls, self.n_levels = a.value, b.value, c.value
        _open_graphs.add(self)

    def close(self):
        """Free the graph's host and device memory (waits for the device to be idle)."""
        if getattr(self, "handle", None):
            lib().echo_free_graph(self.handle)
            self.handle = None
        _open_graphs.discard(self)

    def __del__(self):
        # no HIP calls while the interpreter shuts down: the runtime may be gone
        if sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # ---------------------------------------------------------------- calls
    def cc_cost(self, d_scen, n_scen, *, check=True):
        """Collective costs [n_colls, n_scen] int64 (torch, on the graph's device)."""
        import torch
        dev = torch.device("cuda", self.device)
        if int(n_scen) < 1:
            raise EchoError(ECHO_ERR_ARG, "n_scen must be >= 1")
        scen = _device_buffer(d_scen, "scenarios", dev, int(n_scen) * SCENARIO_DTYPE.itemsize)
        out = torch.empty((self.n_colls, n_scen), dtype=torch.int64, device=dev)
        L = lib()
        _check(L.echo_cc_cost(self.handle, scen, int(n_scen),
                              ctypes.c_void_p(out.data_ptr()), _stream_ptr(dev)))
        if check:
            self.sync_status()
        return out

    def compose(self, d_scen, n_scen, n_refine=1, *, timelines=True, digest=False, out=None, check=True,
                until_stable=False, prorate=False, forest=False, refinements=False):
        """Compose all scenarios.  Returns dict of torch tensors: 'step' [n_scen],
        optional 'start'/'finish' [n_ops, n_scen], 'digest' [n_scen] (uint64 bits
        in an int64 tensor) and 'refinements' [n_scen] int32.  `out` may supply
        preallocated tensors of those names.  until_stable / prorate select the
        validator variants of echo_compose_validated (n_refine is then the most
        refinements)."""
        import torch
        dev = torch.device("cuda", self.device)
        res = dict(out or {})
        if "step" not in res:
            res["step"] = torch.empty(n_scen, dtype=torch.int64, device=dev)
        if timelines:
            for k in ("start", "finish"):
                if k not in res:
                    res[k] = torch.empty((self.n_ops, n_scen), dtype=torch.int64, device=dev)
        if digest and "digest" not in res:
            res["digest"] = torch.empty(n_scen, dtype=torch.int64, device=dev)
        if refinements and "refinements" not in res:
            res["refinements"] = torch.empty(n_scen, dtype=torch.int32, device=dev)
        if int(n_scen) < 1:
            raise EchoError(ECHO_ERR_ARG, "n_scen must be >= 1")
        scen = _device_buffer(d_scen, "scenarios", dev, int(n_scen) * SCENARIO_DTYPE.itemsize)
        rows = {"start": self.n_ops, "finish": self.n_ops, "step": 1, "digest": 1, "refinements": 1}
        types = {"start": torch.int64, "finish": torch.int64, "step": torch.int64, "digest": torch.int64,
                 "refinements": torch.int32}
        ptrs = {k: _device_buffer(res[k], k, dev, rows[k] * int(n_scen) * (4 if k == "refinements" else 8),
                                  types[k]) for k in res if k in rows}
        p = lambda k: ptrs.get(k, ctypes.c_void_p(None))
        none = ctypes.c_void_p(None)
        start, finish = (p("start"), p("finish")) if timelines else (none, none)
        dig = p("digest") if digest else none
        if until_stable or prorate or forest or refinements:
            opts = _Validator(int(n_refine), int(bool(until_stable)), int(bool(prorate)), int(bool(forest)))
            _check(lib().echo_compose_validated(self.handle, scen, int(n_scen),
                                                ctypes.byref(opts), start, finish, p("step"), dig,
                                                p("refinements") if refinements else none, _stream_ptr(dev)))
        else:
            _check(lib().echo_compose_batch(self.handle, scen, int(n_scen),
                                            int(n_refine), start, finish, p("step"), dig, _stream_ptr(dev)))
        if check:
            self.sync_status()
        return res

    def compose_static(self, d_scen, n_scen, n_refine, out, *, digest=False, check=True):
        """echo_compose_batch_static: compose without any device allocation, the workspace
        taken from the library's fixed per-GPU array.  `out` supplies 'start' and
        'finish' [n_ops, n_scen] and 'step' [n_scen] int64 tensors (and 'digest' [n_scen]
        when digest=True); returns `out`."""
        import torch
        dev = torch.device("cuda", self.device)
        if int(n_scen) < 1:
            raise EchoError(ECHO_ERR_ARG, "n_scen must be >= 1")
        scen = _device_buffer(d_scen, "scenarios", dev, int(n_scen) * SCENARIO_DTYPE.itemsize)
        ptr = {k: _device_buffer(out[k], k, dev, (self.n_ops if k in ("start", "finish") else 1) * int(n_scen) * 8,
                                 torch.int64) for k in ("start", "finish", "step") + (("digest",) if digest else ())}
        _check(lib().echo_compose_batch_static(self.handle, scen, int(n_scen), int(n_refine), ptr["start"],
                                               ptr["finish"], ptr["step"], ptr.get("digest", ctypes.c_void_p(None)),
                                               _stream_ptr(dev)))
        if check:
            self.sync_status()
        return out

    def set_cc_tables(self, tables):
        """CC parameter tables: int64 array [n_tables, 6, 7] (max_bytes, chunk, alpha_ns,
        beta_ns, gamma_ns, reduce_MBps per row); scenarios pick one with cc_table = index + 1."""
        t = np.ascontiguousarray(tables, np.int64).reshape(-1, 6, CC_ROWS) if tables is not None and len(tables) \
            else np.zeros((0, 6, CC_ROWS), np.int64)
        _check(lib().echo_set_cc_tables(self.handle, t.ctypes.data_as(ctypes.c_void_p) if len(t) else None,
                                        int(t.shape[0])))

    def set_forest(self, forest):
        """Slowdown ensemble: {'nodes': TREE_NODE_DTYPE array, 'roots': int32 [n_trees],
        'base': Q16 base score, 'class_metrics': int64 [8, 4]}, or None to remove it."""
        L = lib()
        if forest is None:
            _check(L.echo_set_forest(self.handle, None, 0, None, 0, 65536, None))
            return
        nodes = np.ascontiguousarray(forest["nodes"], TREE_NODE_DTYPE)
        roots = np.ascontiguousarray(forest["roots"], np.int32)
        met = np.ascontiguousarray(forest["class_metrics"], np.int64).reshape(8, 4)
        ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
        _check(L.echo_set_forest(self.handle, ptr(nodes), int(nodes.shape[0]), ptr(roots), int(roots.shape[0]),
                                 int(forest["base"]), ptr(met)))

    def set_timing(self, enable=True):
        _check(lib().echo_set_timing(self.handle, int(bool(enable))))

    def kernel_times(self):
        """[(kernel name, ms)] of the last compose call (timing must be on, stream finished)."""
        n = ctypes.c_int32()
        _check(lib().echo_kernel_times(self.handle, 0, None, None, ctypes.byref(n)))
        kinds = np.zeros(max(n.value, 1), np.int32)
        ms = np.zeros(max(n.value, 1), np.float32)
        _check(lib().echo_kernel_times(self.handle, n.value, kinds.ctypes.data_as(ctypes.c_void_p),
                                       ms.ctypes.data_as(ctypes.c_void_p), ctypes.byref(n)))
        return [(KERNEL_KINDS[int(k)], float(t)) for k, t in zip(kinds[:n.value], ms[:n.value])]

    def set_spin_limit(self, limit_ns):
        """Give up a wait for a collective's members after limit_ns of wall clock."""
        _check(lib().echo_set_spin_limit(self.handle, int(limit_ns)))

    def set_launch_tiles(self, max_tiles):
        """At most max_tiles scenario tiles per walk launch (0: as many as fit)."""
        _check(lib().echo_set_launch_tiles(self.handle, int(max_tiles)))

    def walk_chain(self, item_ps, lds_barrier_ps, global_barrier_ps):
        """Longest chain of the walk with these per-item weights (picoseconds):
        {'ps': length, 'items': n, 'lds_barriers': n, 'global_barriers': n}."""
        w = np.array([item_ps, lds_barrier_ps, global_barrier_ps], np.int64)
        out = np.zeros(4, np.int64)
        _check(lib().echo_walk_chain(self.handle, w.ctypes.data_as(ctypes.c_void_p),
                                     out.ctypes.data_as(ctypes.c_void_p)))
        return {"ps": int(out[0]), "items": int(out[1]), "lds_barriers": int(out[2]),
                "global_barriers": int(out[3])}

    def sync_status(self):
        import torch
        _check(lib().echo_sync_status(self.handle, _stream_ptr(torch.device("cuda", self.device))))
