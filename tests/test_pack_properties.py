"""Property tests of the host packers (INT8 and INT4) against the oracle:
random shapes, magnitudes from 1e-7 to 1e4, all-zero rows, values planted on
the rounding boundaries of their row's (or group's) scale, fp32 and bf16
inputs, several epsilon floors.  Every packed byte must equal the oracle's.
CPU only: the host packer runs on host threads."""
import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2609_38090_amd as mira

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@st.composite
def expert_set(draw, multiple):
    C = multiple * draw(st.integers(1, 3))
    R = multiple * draw(st.integers(1, 3))
    n = draw(st.integers(1, 2))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    scale = draw(st.sampled_from([1e-7, 1e-3, 0.05, 1.0, 1e4]))
    rng = np.random.default_rng(seed)
    w = [(rng.standard_normal((n, *s)) * scale).astype(np.float32) for s in ((R, C), (R, C), (C, R))]
    # all-zero rows and rows whose entries sit on rounding boundaries
    m, e, r = draw(st.integers(0, 2)), draw(st.integers(0, n - 1)), draw(st.integers(0, min(R, C) - 1))
    w[m][e, r, :] = 0.0
    m2, r2 = draw(st.integers(0, 2)), draw(st.integers(0, min(R, C) - 1))
    row = w[m2][e, r2]
    k = row.size
    row[:] = (np.arange(k) % 16 - 7.5).astype(np.float32) * scale   # halves of the scale step
    row[0] = 127.0 * scale
    bf16 = draw(st.booleans())
    eps = draw(st.sampled_from([1e-8, 1e-6, 1e-3]))
    return C, R, w, bf16, eps


def _pack(C, R, w, bf16, eps, int4):
    n = w[0].shape[0]
    if bf16:
        tb = [torch.from_numpy(t).to(torch.bfloat16) for t in w]
        src = [t.view(torch.int16).numpy().view(np.uint16).copy() for t in tb]
        ref_w = [t.float().numpy() for t in tb]
    else:
        src, ref_w = w, w
    flags = mira.MIRA_FLAG_INT4 if int4 else 0
    stride = (oracle.packed_expert_bytes_int4 if int4 else oracle.packed_expert_bytes)(C, R)
    out = np.full((n, stride), 0xAB, dtype=np.uint8)
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1, flags=flags), n, mira.MIRA_BF16 if bf16 else mira.MIRA_F32,
                           src[0].ctypes.data, src[1].ctypes.data, src[2].ctypes.data, eps, out.ctypes.data,
                           stride, 0)
    pack = oracle.pack_expert_int4 if int4 else oracle.pack_expert
    return out, [pack(ref_w[0][e], ref_w[1][e], ref_w[2][e], eps=eps) for e in range(n)]


@SETTINGS
@given(expert_set(64))
def test_host_pack_int8_equals_oracle(case):
    C, R, w, bf16, eps = case
    got, refs = _pack(C, R, w, bf16, eps, int4=False)
    for e, ref in enumerate(refs):
        assert np.array_equal(got[e], ref), (C, R, e, bf16, eps)


@SETTINGS
@given(expert_set(128))
def test_host_pack_int4_equals_oracle(case):
    C, R, w, bf16, eps = case
    got, refs = _pack(C, R, w, bf16, eps, int4=True)
    for e, ref in enumerate(refs):
        assert np.array_equal(got[e], ref), (C, R, e, bf16, eps)
