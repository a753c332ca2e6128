"""A layer call captured into a HIP graph (torch.cuda.CUDAGraph): the forward
path makes no allocation, copy, memset or host synchronisation, so it
captures; every replay, with eager work and synchronisations between the
replays, gives the eager result bit for bit (decode, INT4 decode, one-token
decode in both formats, prefill)."""
import numpy as np
import pytest
import torch

import paper_2609_38090_amd as mira
from gpu_layer import Layer
from mira_inputs import MoEConfig

pytestmark = pytest.mark.gpu

DEC = MoEConfig("graph_dec", 141, T=16, C=256, E=8, k=2, R=512, zipf_s=1.2)
PRE = MoEConfig("graph_pre", 142, T=40, C=128, E=64, k=6, R=128, S=2, zipf_s=1.0)


@pytest.mark.parametrize("cfg,T,fmt", [(DEC, 3, "int8"), (DEC, 2, "int4"), (DEC, 1, "int8"), (DEC, 1, "int4"),
                                       (PRE, 40, "int8")])
def test_graph_replays_match_eager(mira, cfg, T, fmt):
    lay = Layer(cfg, T=T, fmt=fmt)
    ref = lay.run()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):               # warm-up on the capture stream's side
        lay.run(sync=False)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = lay.run(sync=False)              # queued on the capture stream
    torch.cuda.synchronize()
    for rep in range(4):
        for key, t in outs.items():             # eager work between replays
            if key != "_ws" and t.dtype.is_floating_point:
                t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for key in ref:
            assert np.array_equal(ref[key], outs[key].cpu().numpy()), (rep, key)
