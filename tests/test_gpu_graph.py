"""GPU: the stage calls captured once in a HIP graph and replayed give the
same weights and smoothed gradients, bit for bit, as the same steps issued
one by one (bench.py --graph). Each replay is checked, with other eager work
and synchronisations between the replays."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _loops(name, stream):
    import bench
    from paper_1809_02839_amd import native
    wl = synth.ALL_WORKLOADS[name]
    if len(wl.stages) > 1:
        return (bench.PipeLoop(wl.stages, torch, native, stream), bench.PipeLoop(wl.stages, torch, native, stream))
    spec = wl.stages[0]
    return bench.StageLoop(spec, torch, native, stream), bench.StageLoop(spec, torch, native, stream)


def _states(loop):
    stages = loop.st if isinstance(loop.st, list) else [loop.st]
    return [s.get_state() for s in stages]


@pytest.mark.parametrize("name", ["vgg_conv_small", "transformer_enc_small", "reslstm_small", "mlp3_small"])
def test_graph_replay_matches_eager(name):
    print(f"[graph] {name}", flush=True)
    stream = torch.cuda.Stream()
    eager, graphed = _loops(name, stream)
    period = graphed.graph_period()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        graphed.steps(period)   # captured, not run
    for r in range(3):
        eager.steps(period)
        with torch.cuda.stream(stream):
            graph.replay()
            other = (torch.arange(4096, device="cuda", dtype=torch.float32) * 0.5).sum()
        torch.cuda.synchronize()
        assert other.item() == pytest.approx(0.5 * 4095 * 4096 / 2)
        for k, ((We, ve), (Wg, vg)) in enumerate(zip(_states(eager), _states(graphed))):
            assert np.array_equal(We, Wg), (name, "W", r, k)
            assert np.array_equal(ve, vg), (name, "v", r, k)
    print(f"[graph] {name}: 3 replays of {period} steps bitwise equal to eager", flush=True)
    for loop in (eager, graphed):
        if hasattr(loop, "destroy"):
            loop.destroy()
        else:
            loop.st.destroy()
