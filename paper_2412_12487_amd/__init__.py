"""MI355X timeline composer of Echo (arXiv 2412.12487): HIP kernels behind a C ABI.

    from paper_2412_12487_amd import Graph, scenarios_to_device
    g = Graph(graph_arrays, device=0)          # echo_load_graph
    d_scen, n = scenarios_to_device(scen)      # echo_scenario records on the GPU
    out = g.compose(d_scen, n, n_refine=1)     # echo_compose_batch
"""
from .echo import (ECHO_ERR_ARG, ECHO_ERR_CYCLE, ECHO_ERR_DEVICE, ECHO_ERR_HIP, ECHO_ERR_MATCH,
                   ECHO_ERR_NOMEM, ECHO_ERR_RANGE, ECHO_OK, EXPORTS, LIB_PATH, SCENARIO_DTYPE, EchoError,
                   Graph, lib, pack_scenarios, scenarios_to_device)

__all__ = ["Graph", "EchoError", "lib", "pack_scenarios", "scenarios_to_device", "SCENARIO_DTYPE",
           "LIB_PATH", "EXPORTS", "ECHO_OK", "ECHO_ERR_ARG", "ECHO_ERR_RANGE", "ECHO_ERR_MATCH",
           "ECHO_ERR_CYCLE", "ECHO_ERR_NOMEM", "ECHO_ERR_HIP", "ECHO_ERR_DEVICE"]
