"""The whole compression step captured into a HIP graph and replayed.

The library allocates nothing after create and, once a step's layer table
has been uploaded, issues only kernel launches and an event record per
call, so a step can be captured on a stream and replayed.  Every replay
(with other device work and synchronisations in between) must give what
the eager step gives, bit for bit.
"""
import numpy as np
import pytest
import torch

from paper_2606_07577_amd import synth
from paper_2606_07577_amd.step import DeviceStep

pytestmark = pytest.mark.gpu


def _outputs(st):
    """What a step writes: a and s of every row, the budgets, and the kept
    rows' indices and compacted K and V."""
    budgets = st.budgets.cpu().numpy()
    out = [st.a.clone(), st.s.clone(), st.budgets.clone()]
    for l in range(st.n_layers):
        m = int(budgets[l].sum())
        out += [st.idx[l, :, :m].clone(), st.k_out[l][:, :m].clone(), st.v_out[l][:, :m].clone()]
    return out


@pytest.mark.parametrize("name,budget", [("tiny-f32-640", 256), ("qwen7b-layer-6144", 4096)])
def test_step_graph_replays_match_eager(name, budget):
    layers = synth.make_workload(name)
    st = DeviceStep(layers, budget)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.run(side)              # eager step: uploads the layer table, warms everything
    torch.cuda.synchronize()
    ref = _outputs(st)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        st.run(side)
    torch.cuda.synchronize()
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        for t in [st.a, st.s, st.idx] + st.k_out + st.v_out:
            t.fill_(-7)           # outputs must be rewritten by the replay
        junk.mul_(1.0001)         # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _outputs(st)
        for i, (x, y) in enumerate(zip(got, ref)):
            assert torch.equal(x, y), f"replay {rep}: output {i} differs from the eager step"
    del graph
    st.close()
