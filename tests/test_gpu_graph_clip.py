"""lt_clip_coef is the one entry point documented as safe to capture in a HIP graph
(it stages nothing on the host).  Capture it once, then replay it many times with a
different sum of squares written by eager work before each replay; every replay
must give bitwise the oracle's norm and coefficient for that sum, as the same call
made eagerly does."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11919_amd as lt
from gpu_helpers import DEV, to_host

pytestmark = pytest.mark.gpu

SUMS = [0.0, 5e-324, 1e-12, 0.25, 0.9999999999, 1.0, 1.0000000002, 4.0, 261.17, 1e6,
        3.1e14, 1.7e308, math.inf]


@pytest.mark.parametrize("max_norm", [1.0, 0.5, math.inf])
def test_captured_clip_coef_replays_match_the_oracle(max_norm):
    S = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    norm = torch.zeros(1, dtype=torch.float32, device=DEV)
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # a first eager call on a side stream before capture
        lt.lt_clip_coef(S, max_norm, coef, total_norm=norm)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        lt.lt_clip_coef(S, max_norm, coef, total_norm=norm)
    eager_coef = torch.zeros_like(coef)
    eager_norm = torch.zeros_like(norm)
    for rnd in range(2):
        for s in (SUMS if rnd == 0 else SUMS[::-1]):
            S.fill_(s)
            coef.fill_(-1.0)
            norm.fill_(-1.0)
            graph.replay()
            lt.lt_clip_coef(S, max_norm, eager_coef, total_norm=eager_norm)
            torch.cuda.synchronize()
            n_o, c_o = oracle.clip_coef(s, max_norm)
            got = (to_host(norm)[0], to_host(coef)[0])
            assert got[0].tobytes() == n_o.tobytes() and got[1].tobytes() == c_o.tobytes(), \
                f"replay, S = {s!r}, max_norm {max_norm}: {got} against {(n_o, c_o)}"
            assert to_host(eager_coef)[0].tobytes() == c_o.tobytes()
            assert to_host(eager_norm)[0].tobytes() == n_o.tobytes()
    del graph
