"""HIP graph capture of a whole decoder-layer step (forward + backward through
the C ABI): every replay must equal the eager step bit for bit.

The library's calls only launch kernels on the given stream, so a step can be
captured and replayed.  Following the replay discipline for graphs, the graph is
replayed several times with unrelated eager work and synchronisations between the
replays, the outputs are poisoned with NaN before each replay, and every replay
is compared with the eager result.  The Qwen2.5-32B shape also takes the
split-K last-wave GEMM path (partials, then their reduction) inside the graph.
"""

import pytest

from paper_2606_10415_amd.synth import WORKLOADS, layer_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "qwen2.5-32b"])
def test_layer_step_graph_replays_match_eager(name):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_10415_amd.layer import DecoderLayer
    print(f"graph capture {name}", flush=True)
    w = WORKLOADS[name]
    L = DecoderLayer(w, layer_inputs(w))
    outs = (L.Y, L.dX, L.dWqkv, L.dWo, L.dWgu, L.dWd, L.dQKV)
    L.step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):            # warm the capture stream
        L.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        L.step()
    torch.cuda.synchronize()
    for r in range(3):
        junk = torch.randn(1 << 16, device="cuda").square().sum().item()   # eager work between
        assert junk > 0
        for t in outs:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs, ref)):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (r, i)
