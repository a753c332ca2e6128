"""Calls on different streams at once: each call owns its workspace and
outputs, so concurrent decode and prefill layers (and the same layer on two
streams) give bit-identical results to the same calls one after another."""
import numpy as np
import pytest
import torch

from gpu_layer import Layer
from mira_inputs import MoEConfig

pytestmark = pytest.mark.gpu

DEC = MoEConfig("streams_dec", 131, T=16, C=256, E=8, k=2, R=512, zipf_s=1.2)
PRE = MoEConfig("streams_pre", 132, T=40, C=128, E=64, k=6, R=128, S=2, zipf_s=1.0)


def test_concurrent_streams_match_sequential(mira):
    dec = Layer(DEC, T=3)
    pre = Layer(PRE, T=40)
    i4 = Layer(DEC, T=2, fmt="int4")
    ref = [dec.run(), pre.run(), i4.run(), dec.run(two_phase=True)]
    streams = [torch.cuda.Stream() for _ in range(4)]   # default priority
    for _ in range(3):
        outs = [dec.run(stream=streams[0], sync=False),
                pre.run(stream=streams[1], sync=False),
                i4.run(stream=streams[2], sync=False),
                dec.run(two_phase=True, stream=streams[3], sync=False)]
        torch.cuda.synchronize()
        for r, o in zip(ref, outs):
            for key in r:
                assert np.array_equal(r[key], o[key].cpu().numpy()), key
