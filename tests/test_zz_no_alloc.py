"""The allocation-free compose (echo_compose_batch_static) against echo_compose_batch.

The entry point takes its workspace from the library's fixed per-GPU array and
allocates nothing; its results must equal the allocating compose's bit for bit.
Two calls in a row share the array (the second with a smaller input, so stale
contents of the first would show), and a call that would need more than the
array holds is refused before anything is enqueued.
"""
from __future__ import annotations

import numpy as np
import pytest

from workloads import configs, gpt1f1b, scenarios

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20


@pytest.fixture(scope="module")
def E():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2412_12487_amd as E
    E.lib()
    return E


def _outputs(G, n, digest=True):
    import torch
    dev = torch.device("cuda", G.device)
    out = {"start": torch.full((G.n_ops, n), -1, dtype=torch.int64, device=dev),
           "finish": torch.full((G.n_ops, n), -1, dtype=torch.int64, device=dev),
           "step": torch.full((n,), -1, dtype=torch.int64, device=dev)}
    if digest:
        out["digest"] = torch.zeros(n, dtype=torch.int64, device=dev)
    return out


def _same(a, b, keys):
    for k in keys:
        assert torch_equal(a[k], b[k]), k


def torch_equal(x, y):
    import torch
    return bool(torch.equal(x, y))


def _case(E, G, sc, R, digest=True):
    """The static compose and the allocating compose of the same inputs, bit for bit."""
    import torch
    d, n = E.scenarios_to_device(sc)
    want = G.compose(d, n, R, timelines=True, digest=digest)
    got = G.compose_static(d, n, R, _outputs(G, n, digest), digest=digest)
    torch.cuda.synchronize()
    _same(got, want, ["start", "finish", "step"] + (["digest"] if digest else []))
    return got


def test_static_compose_equals_the_allocating_compose_twice_in_a_row(E):
    """Config 1 (8 ranks): 200 jittered scenarios with two refinements, then 70
    scenarios with one on a smaller graph (the next call starts on the first one's
    leftovers in the shared array), then the first input again."""
    big = configs.graph(1)
    small = gpt1f1b.gpt_graph(n_layers=2, hidden=1024, seq=512, tp=2, pp=2, dp=1, microbatches=2, seed=4)
    assert len(small["op_rank"]) < len(big["op_rank"])
    sc_big = scenarios.draw(200, np.random.default_rng(31), bw_inter=(50_000, 400_000), bw_intra=(50_000, 400_000),
                            alpha=(2_000, 20_000), slowdown=(65536, 91750), jitter=(6554, 5), ar_algo_random=True)
    sc_small = scenarios.draw(70, np.random.default_rng(32), bw_inter=(50_000, 400_000), alpha=(2_000, 20_000),
                              slowdown=(65536, 120000))
    Gb, Gs = E.Graph(big, 0), E.Graph(small, 0)
    try:
        _case(E, Gb, sc_big, 2)
        _case(E, Gs, sc_small, 1, digest=False)
        _case(E, Gb, scenarios.take(sc_big, slice(0, 65)), 0)
        _case(E, Gb, sc_big, 1)
    finally:
        Gb.close()
        Gs.close()


def test_static_compose_allocates_nothing(E):
    """Device free memory is the same before and after a static compose on a graph
    that has never composed (its allocating compose would grow a workspace)."""
    import torch
    g = configs.graph(1)
    sc = configs.scenario_batch(4, n=256)
    d, n = E.scenarios_to_device(sc)
    G0 = E.Graph(g, 0)
    G0.compose_static(d, n, 1, _outputs(G0, n))       # first use of the array on this device
    G0.close()
    G = E.Graph(g, 0)
    try:
        out = _outputs(G, n)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info(0)[0]
        G.compose_static(d, n, 1, out)
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info(0)[0] == free0
    finally:
        G.close()


def test_static_compose_refuses_what_does_not_fit(E):
    """The config-1 graph with 32768 scenarios needs more workspace than the fixed
    64 MiB array (its overlap masks alone, one byte per walk item and scenario, take at
    least 2912 x 32768 bytes, 95 MB): ECHO_ERR_RANGE before any launch; the graph then
    composes the whole enumeration batch (4096 scenarios); missing outputs are argument
    errors."""
    import torch
    g = configs.graph(1)
    G = E.Graph(g, 0)
    try:
        sc = configs.scenario_batch(4, n=32768)
        d, n = E.scenarios_to_device(sc)
        with pytest.raises(E.EchoError) as x:
            G.compose_static(d, n, 1, _outputs(G, n, digest=False))
        assert x.value.code == E.ECHO_ERR_RANGE
        L = E.lib()
        import ctypes
        none = ctypes.c_void_p(None)
        out = _outputs(G, 64, digest=False)
        rc = L.echo_compose_batch_static(G.handle, ctypes.c_void_p(d.data_ptr()), 64, 1, none,
                                         ctypes.c_void_p(out["finish"].data_ptr()),
                                         ctypes.c_void_p(out["step"].data_ptr()), none, none)
        assert rc == E.ECHO_ERR_ARG
        _case(E, G, configs.scenario_batch(4), 1)
        torch.cuda.synchronize()
    finally:
        G.close()
