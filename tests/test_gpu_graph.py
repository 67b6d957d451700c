"""The layer step captured in a HIP graph (through torch's graph capture) and replayed:
the library issues no memsets, host synchronisations or allocations on this path, so
every replay must give the eager step's bits. Replays are interleaved with eager work
and synchronisations."""
import numpy as np
import pytest
import torch

from paper_2508_06024_amd import workload as W
from paper_2508_06024_amd.layer import Ec2moeLayer
from tests.gpu_common import say, up, up_f32

pytestmark = pytest.mark.gpu


def _layer(cfg, overlap=False):
    inp = W.gen_layer(cfg)
    dt = cfg.dtype
    lay = Ec2moeLayer(up(inp.x, dt), inp.mask, up(inp.w_global, dt), up_f32(inp.b_global), up(inp.w_local, dt),
                      up_f32(inp.b_local), up(inp.w_gate_up, dt), up(inp.w_down, dt), up(inp.u, dt), up(inp.v, dt),
                      n_groups=cfg.n_groups, top_k=cfg.top_k, activation=cfg.activation,
                      codec_slices=cfg.codec_slices, overlap=overlap)
    return inp, lay


@pytest.mark.parametrize("name,overlap", [("small", False), ("switch16", False), ("small", True)])
def test_graph_replays_match_eager(name, overlap):
    """overlap=True captures the routing stream's fork and join as graph dependencies."""
    cfg = W.CONFIGS[name]
    say(f"graph capture {name} overlap={overlap}")
    inp, lay = _layer(cfg, overlap)
    x2 = up(W.gen_call(cfg.scaled(seed=cfg.seed + 1))[0], cfg.dtype)
    x1 = lay.x
    # eager reference for both inputs
    refs = []
    for x in (x1, x2):
        lay.set_input(x)
        refs.append(tuple(t.clone() for t in (lay.step(), lay.topk_idx, lay.z)))
    torch.cuda.synchronize()
    # one graph per input buffer (the layer reads X through its pointer)
    graphs = []
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for x in (x1, x2):
            lay.set_input(x)
            lay.step()  # warm the side stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for x in (x1, x2):
        lay.set_input(x)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            lay.step()
        graphs.append(g)
    torch.cuda.synchronize()
    for rep in range(6):
        which = rep % 2
        graphs[which].replay()
        torch.cuda.synchronize()
        y, idx, z = (t.clone() for t in (lay.y, lay.topk_idx, lay.z))
        assert torch.equal(y, refs[which][0]), f"replay {rep}: y differs from eager"
        assert torch.equal(idx, refs[which][1]) and torch.equal(z, refs[which][2])
        # eager work in between: the other input, then back
        lay.set_input((x2, x1)[which])
        lay.step()
        torch.cuda.synchronize()
        assert torch.equal(lay.y, refs[1 - which][0])
