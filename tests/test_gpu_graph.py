"""The hot path under HIP graph capture.

The library launches kernels only (no allocation, copy, memset or
synchronisation), so a step can be captured into a graph. A verify step of a
mixed decode + verify batch and a decode step are captured with torch's
graph API and replayed several times, with eager fill kernels (the poison of
every output and workspace byte) and synchronisations between replays; every
replay is checked against the oracle like an eager run, accept lengths
bit-exactly.
"""
import pytest
import torch

from paper_2607_03333_amd import runner, synth
from gpu_cases import compare_accept, compare_attention, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("index,shrink", [
    (4, dict(sessions=3, prefix=1000, suffix=("loguniform", 1, 400), vocab=3000)),
    (2, dict(sessions=2, prefix=1024, suffix=("uniform", 1, 200))),
])
def test_captured_step_replays_match_the_oracle(index, shrink):
    wl = synth.make(index, **shrink)
    dw = runner.DeviceWorkload(wl)
    try:
        step = dw.prepare_all()[-1]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step.run()                       # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step.run()
        torch.cuda.synchronize()
        for r in range(4):
            step.poison()                    # eager work between replays
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            say(f"[graph {wl.name}] replay {r}")
            compare_attention(wl, step, tag=f"graph {wl.name} replay {r}")
            if step.verify:
                compare_accept(wl, step, tag=f"graph {wl.name} replay {r}")
    finally:
        dw.close()
