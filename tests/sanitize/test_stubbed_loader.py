"""Loader checks that need the host-memory stand-in of the HIP runtime
(tests/sanitize/hip_host_stub.cpp): forced allocation failures, leak-free
error paths, and the walk-chain analysis on hand-built graphs.  They run only
inside the sanitizer run of tests/test_sanitized_host.py, where the binding
loads the AddressSanitizer/UBSan build of the loader linked with the stub."""
from __future__ import annotations

import ctypes
import os

import numpy as np
import pytest

from tests.tinygraph import AR, P2P, Builder
from workloads import configs

pytestmark = pytest.mark.skipif(not os.environ.get("ECHO_HOST_STUB"),
                                reason="needs the sanitizer build linked with the HIP host stub")


@pytest.fixture(scope="module")
def E():
    import paper_2412_12487_amd as E
    L = E.lib()
    L.echo_stub_fail_after.argtypes = [ctypes.c_int64]
    L.echo_stub_live_allocations.restype = ctypes.c_int64
    return E


def _live(E):
    return int(E.lib().echo_stub_live_allocations())


def test_every_allocation_failure_is_nomem_and_leaks_nothing(E):
    """Fail each device allocation of a load in turn: the load returns
    ECHO_ERR_NOMEM and frees whatever it had allocated."""
    g = configs.graph(1)
    base = _live(E)
    G = E.Graph(g)
    n_alloc = _live(E) - base
    G.close()
    assert _live(E) == base and n_alloc > 20
    L = E.lib()
    for k in range(n_alloc):
        L.echo_stub_fail_after(k)
        with pytest.raises(E.EchoError) as x:
            E.Graph(g)
        assert x.value.code == E.ECHO_ERR_NOMEM, (k, str(x.value))
        assert _live(E) == base, k
    L.echo_stub_fail_after(-1)
    E.Graph(g).close()
    assert _live(E) == base


def test_failed_ensemble_and_table_uploads_keep_the_graph_usable(E):
    from workloads import scenarios, slowdown_forest
    G = E.Graph(configs.graph(1))
    base = _live(E)
    L = E.lib()
    L.echo_stub_fail_after(0)
    with pytest.raises(E.EchoError) as x:
        G.set_cc_tables(scenarios.draw_cc_tables(2, np.random.default_rng(1)))
    assert x.value.code == E.ECHO_ERR_NOMEM
    L.echo_stub_fail_after(-1)
    G.set_cc_tables(scenarios.draw_cc_tables(2, np.random.default_rng(1)))
    G.set_forest(slowdown_forest.synthetic_forest(0))
    G.set_forest(None)
    G.set_cc_tables(None)
    assert _live(E) == base
    G.close()


def _chain(G, w=(1000, 0, 0)):
    return G.walk_chain(*w)




def test_walk_chain_hand_cases(E):
    # one rank, a chain of n compute ops: n items, no barrier
    b = Builder(1)
    prev = []
    for _ in range(7):
        prev = [b.compute(0, 5, preds=prev)]
    with E.Graph(b.graph()) as G:
        assert _chain(G, (1000, 50, 70)) == {"ps": 7000, "items": 7, "lds_barriers": 0, "global_barriers": 0}
    # P2P: rank 0 runs a then sends; rank 1 receives, then runs b.  Walk lists:
    # rank 0 [a, send launch, send resolve], rank 1 [recv launch, recv resolve, b];
    # the recv resolve waits for the send launch (item 2 of rank 0): chain a, send,
    # recv resolve, b = 4 items through one LDS barrier (both ranks in one workgroup)
    b = Builder(2)
    c = b.collective(P2P, 1000)
    a = b.compute(0, 5)
    b.comm(0, c, stream=3, preds=[a])
    r = b.comm(1, c, stream=4)
    b.compute(1, 5, preds=[r])
    with E.Graph(b.graph()) as G:
        assert _chain(G, (1000, 300, 700)) == {"ps": 4300, "items": 4, "lds_barriers": 1, "global_barriers": 0}
    # an all-reduce of 16 ranks spans two workgroups of eight walkers: its barrier
    # is met in device memory.  Rank 15 runs three ops first; every rank's resolve
    # waits for it: chain = 3 ops + launch + resolve + the op after it
    b = Builder(16)
    c = b.collective(AR, 1 << 20)
    for r in range(16):
        prev = []
        for _ in range(3 if r == 15 else 1):
            prev = [b.compute(r, 5, preds=prev)]
        x = b.comm(r, c, preds=prev)
        b.compute(r, 5, preds=[x])
    with E.Graph(b.graph()) as G:
        got = _chain(G, (1000, 300, 700))
        assert got == {"ps": 6700, "items": 6, "lds_barriers": 0, "global_barriers": 1}, got
    # the same all-reduce as collective 1 behind a P2P between ranks 0 and 1 (collective 0,
    # met in LDS): the all-reduce is the first collective met by counting, index 0 among
    # those, and the analysis must still see its 16 members.  Every rank: one op (rank 15:
    # three), the all-reduce, one op; then rank 0 sends and rank 1 receives and runs one
    # more op.  Rank 1's chain: 3 ops and the launch of rank 15 (4000), all-reduce resolve
    # (+1000 +700), op (6700), recv launch (7700; rank 0's send launch is also at 7700),
    # recv resolve (+1000 +300), op: 10000 ps over 9 items.
    b = Builder(16)
    p2p = b.collective(P2P, 1000)
    c = b.collective(AR, 1 << 20)
    for r in range(16):
        prev = []
        for _ in range(3 if r == 15 else 1):
            prev = [b.compute(r, 5, preds=prev)]
        x = b.comm(r, c, preds=prev)
        y = b.compute(r, 5, preds=[x])
        if r == 0:
            b.comm(0, p2p, stream=3, preds=[y])
        elif r == 1:
            z = b.comm(1, p2p, stream=4, preds=[y])
            b.compute(1, 5, preds=[z])
    with E.Graph(b.graph()) as G:
        got = _chain(G, (1000, 300, 700))
        assert got == {"ps": 10000, "items": 9, "lds_barriers": 1, "global_barriers": 1}, got


def test_walk_chain_covers_the_longest_walk_list(E):
    g = configs.graph(1)
    with E.Graph(g) as G:
        ch = _chain(G, (1, 0, 0))
        per_rank = np.bincount(g["op_rank"], minlength=g["n_ranks"])
        comm_per_rank = np.bincount(g["op_rank"][g["op_kind"] == 1], minlength=g["n_ranks"])
        # every rank's list: its ops plus one resolve item per comm op
        assert ch["items"] >= int((per_rank + comm_per_rank).max())
        assert ch["ps"] == ch["items"]
        # barrier weights only add where resolve items lie on the chain
        ch2 = _chain(G, (1, 10**6, 10**6))
        assert ch2["ps"] == ch2["items"] + 10**6 * (ch2["lds_barriers"] + ch2["global_barriers"])
        assert ch2["ps"] >= ch["ps"] and ch2["lds_barriers"] + ch2["global_barriers"] > 0
