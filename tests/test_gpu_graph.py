"""The whole step -- routing (with the masked placement), permutation, the
persistent FFN kernel and the combine -- captured once in a HIP graph and
replayed (the paper's Adaptive Persistent Kernel stays compatible with graph
replay: every launch is an ordinary kernel on the caller's stream, the
scheduler state is reset by a kernel rather than a memset, and nothing in the
launch path allocates or synchronizes).  Every replay, with eager work and
synchronizations between replays, must give the eager step's outputs bit for
bit and a clean status."""
import numpy as np
import pytest

from _helpers import layer_specs
from workload import custom_config

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_18002_amd import load_library
    load_library()
    return torch.device("cuda:0")


@pytest.mark.parametrize("masked,fused_combine", [(True, False), (False, False), (True, True)])
def test_step_replayed_from_a_graph(dev, masked, fused_combine):
    from paper_2607_18002_amd.pipeline import MoEPipeline
    cfg = custom_config(2, cfg_id=901, H=512, I=512, prefill_tokens=600, decode_tokens=70, E_global=64,
                        E_local=12, top_k=4, n_layers=2, zipf_s=(1.1, 0.7))
    specs = []
    for layer in range(2):
        s, _, _ = layer_specs(cfg, layer, dev, decode=dict(release_after_ns=5_000))
        specs += s
    kw = dict(fused_gather=True, masked_decode=masked, fused_combine=fused_combine, trace_capacity=1 << 14)
    pipe = MoEPipeline(specs, **kw)
    pipe.run()
    torch.cuda.synchronize()
    assert pipe.statuses() == (0, 0)
    eager = [b.y.clone() for b in pipe.bufs]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                      # warm the capture stream, as torch asks
        pipe.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pipe.run()
    torch.cuda.synchronize()

    other = MoEPipeline(specs[:2], fused_gather=True)  # unrelated eager work between replays
    for rep in range(4):
        for b in pipe.bufs:
            b.y.fill_(3.0)
        pipe.status.fill_(7)
        pipe.stats.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert pipe.statuses() == (0, 0), rep
        for i, (b, e) in enumerate(zip(pipe.bufs, eager)):
            assert torch.equal(b.y, e), (rep, i)
        stats = pipe.op_stats()
        assert np.all(stats["t_done"] > 0), rep
        other.run()
        torch.cuda.synchronize()
        assert other.statuses() == (0, 0)
