"""Pins for the oracle's packing (paper section IV-B, Eqs. (2)-(4)).

Every check compares against something other than the oracle's own formula:
closed forms built from known integers and scales, hand-written expected
values, torch's bf16 conversion, and invariants the definition implies.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16_values(rng, n, lo=-12, hi=-4):
    """n random positive bf16-representable fp32 values in [2^lo, 2^hi)."""
    mant = rng.integers(128, 256, size=n).astype(np.float32)      # 8-bit significand
    exp = rng.integers(lo, hi, size=n)
    return (mant * np.exp2(exp - 7).astype(np.float32)).astype(np.float32)


def _grid_expert(rng, C, R, where_max):
    """Weights w = q * sigma with known q, sigma; row r's |q| max (=127) sits in slice where_max[r]."""
    sigma = _bf16_values(rng, R)
    qg = rng.integers(-126, 127, size=(R, C)).astype(np.int8)
    qu = rng.integers(-126, 127, size=(R, C)).astype(np.int8)
    qd = rng.integers(-126, 127, size=(C, R)).astype(np.int8)
    for r in range(R):
        sgn = 1 if rng.random() < 0.5 else -1
        c = rng.integers(0, C)
        if where_max[r] == 0:
            qg[r, c] = 127 * sgn
        elif where_max[r] == 1:
            qu[r, c] = 127 * sgn
        else:
            qd[c, r] = 127 * sgn
    wg = qg.astype(np.float32) * sigma[:, None]
    wu = qu.astype(np.float32) * sigma[:, None]
    wd = qd.astype(np.float32) * sigma[None, :]
    return (wg, wu, wd), (qg, qu, qd, sigma)


def _tiled_bytes(q):
    """The documented tile layout, element by element: element (r, k) of a
    [rows][K] matrix goes to tile (r // 16, k // 64), run (k % 64 // 16) * 16 + r % 16,
    byte k % 16 of the run; tiles are 1024 bytes, row-of-tiles major."""
    rows, K = q.shape
    r, k = np.meshgrid(np.arange(rows), np.arange(K), indexing="ij")
    tile = (r // 16) * (K // 64) + k // 64
    run = ((k % 64) // 16) * 16 + r % 16
    off = tile * 1024 + run * 16 + k % 16
    out = np.empty(rows * K, dtype=np.int8)
    out[off.reshape(-1)] = q.reshape(-1)
    return out.view(np.uint8)


def _expected_blob(qg, qu, qd, sigma_bits, C, R):
    raw = np.concatenate([_tiled_bytes(qg), _tiled_bytes(qu), _tiled_bytes(qd),
                          np.asarray(sigma_bits, dtype="<u2").view(np.uint8)])
    pad = (-raw.size) % 256
    return np.concatenate([raw, np.zeros(pad, dtype=np.uint8)])


def _torch_bf16_bits(v):
    t = torch.from_numpy(np.asarray(v, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    v = rng.standard_normal(100000).astype(np.float32) * np.float32(1e-3)
    # exact ties: patterns whose dropped half-word is 0x8000, both parities of the kept bit
    ties = (np.arange(1000, dtype=np.uint32) << 16 | 0x8000) + (0x3C00 << 16)
    v = np.concatenate([v, ties.view(np.float32), np.float32([0.0, -0.0, 1.0, 3.3895314e38])])
    assert np.array_equal(oracle.bf16_bits_from_f32(v), _torch_bf16_bits(v))


@pytest.mark.parametrize("C,R", [(64, 64), (256, 128), (128, 192)])
def test_pack_grid_round_trip_bit_exact(C, R):
    rng = np.random.default_rng(C * 1000 + R)
    where = rng.integers(0, 3, size=R)
    (wg, wu, wd), (qg, qu, qd, sigma) = _grid_expert(rng, C, R, where)
    blob = oracle.pack_expert(wg, wu, wd, eps=1e-8)
    sigma_bits = (sigma.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(blob, _expected_blob(qg, qu, qd, sigma_bits, C, R))


def test_shared_scale_driven_by_down_column():
    """Rows whose largest magnitude is only in W_down[:, r]: the scale must follow that column."""
    rng = np.random.default_rng(7)
    C, R = 128, 64
    (wg, wu, wd), (qg, qu, qd, sigma) = _grid_expert(rng, C, R, np.full(R, 2))
    # shrink gate/up so the down column alone carries the maximum
    qg = (qg // 8).astype(np.int8)
    qu = (qu // 8).astype(np.int8)
    wg = qg.astype(np.float32) * sigma[:, None]
    wu = qu.astype(np.float32) * sigma[:, None]
    blob = oracle.pack_expert(wg, wu, wd)
    g, u, d, sb = oracle.unpack_expert(blob, C, R)
    assert np.array_equal(g, qg) and np.array_equal(u, qu) and np.array_equal(d, qd)
    assert np.all(np.abs(d).max(axis=0) == 127)
    assert np.all(np.abs(g).max(axis=1) <= 16)
    assert np.array_equal(oracle.f32_from_bf16_bits(sb), sigma)


def test_pack_ties_golden():
    with open(os.path.join(GOLDEN, "pack_ties.json")) as f:
        g = json.load(f)
    wg, wu, wd, n = _embed_row0(g, "scale_exp2")
    s = np.float32(2.0 ** g["scale_exp2"])
    blob = oracle.pack_expert(wg, wu, wd)
    qg, qu, qd, sb = oracle.unpack_expert(blob, 64, 64)
    assert qg[0, :n].tolist() == g["gate_expected"]
    assert qu[0, :n].tolist() == g["up_expected"]
    assert qd[:n, 0].tolist() == g["down_expected"]
    assert oracle.f32_from_bf16_bits(sb)[0] == s


def test_all_zero_row_uses_eps():
    C, R = 64, 64
    rng = np.random.default_rng(3)
    wg = rng.standard_normal((R, C)).astype(np.float32) * 0.02
    wu = rng.standard_normal((R, C)).astype(np.float32) * 0.02
    wd = rng.standard_normal((C, R)).astype(np.float32) * 0.02
    wg[2] = 0.0
    wu[2] = 0.0
    wd[:, 2] = 0.0
    eps = 1e-8
    blob = oracle.pack_expert(wg, wu, wd, eps=eps)
    qg, qu, qd, sb = oracle.unpack_expert(blob, C, R)
    assert not qg[2].any() and not qu[2].any() and not qd[:, 2].any()
    expect = _torch_bf16_bits(torch.tensor([eps], dtype=torch.float32).div(127.0).numpy())
    assert sb[2] == expect[0]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_pack_invariants_random(seed):
    rng = np.random.default_rng(seed)
    C, R = 192, 128
    wg = rng.standard_normal((R, C)).astype(np.float32) * 0.02
    wu = rng.standard_normal((R, C)).astype(np.float32) * 0.02
    wd = (rng.standard_normal((C, R)) * 0.02).astype(np.float32)
    wd[5, 3] = 0.5  # an outlier in one down column
    blob = oracle.pack_expert(wg, wu, wd)
    assert blob.size == oracle.packed_expert_bytes(C, R) == ((3 * R * C + 2 * R + 255) // 256) * 256
    assert not blob[3 * R * C + 2 * R:].any()
    qg, qu, qd, sb = oracle.unpack_expert(blob, C, R)
    sigma = oracle.f32_from_bf16_bits(sb).astype(np.float64)
    for q in (qg, qu, qd):
        assert q.min() >= -127 and q.max() <= 127
    # the row maximum maps to +-127
    m = np.maximum(np.maximum(np.abs(qg).max(1), np.abs(qu).max(1)), np.abs(qd).max(0))
    assert np.all(m == 127)
    # sigma is within bf16 rounding (relative 2^-8) of alpha / 127
    alpha = np.maximum(np.maximum(np.abs(wg).max(1), np.abs(wu).max(1)), np.abs(wd).max(0))
    assert np.all(np.abs(sigma - alpha / 127.0) <= alpha / 127.0 * 2.0 ** -8)
    # rounding error bound: |sigma q - w| <= sigma / 2 (plus the fp32 quotient's rounding)
    tol = 0.5 * (1 + 2.0 ** -20)
    assert np.all(np.abs(qg * sigma[:, None] - wg) <= tol * sigma[:, None])
    assert np.all(np.abs(qu * sigma[:, None] - wu) <= tol * sigma[:, None])
    assert np.all(np.abs(qd * sigma[None, :] - wd) <= tol * sigma[None, :])
    # the column outlier drives its row's scale (shared across the three matrices)
    assert qd[5, 3] == 127 and np.abs(qg[3]).max() < 20


def test_dequantize_is_scale_times_integer():
    rng = np.random.default_rng(11)
    C, R = 64, 64
    (wg, wu, wd), _ = _grid_expert(rng, C, R, rng.integers(0, 3, size=R))
    blob = oracle.pack_expert(wg, wu, wd)
    dg, du, dd = oracle.dequantize_expert(blob, C, R)
    assert np.array_equal(dg, wg.astype(np.float64))
    assert np.array_equal(du, wu.astype(np.float64))
    assert np.array_equal(dd, wd.astype(np.float64))


def test_pack_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.pack_expert(np.zeros((4, 8)), np.zeros((4, 8)), np.zeros((4, 8)))


def test_integers_use_the_stored_bf16_scale_golden():
    with open(os.path.join(GOLDEN, "pack_scale_rounding.json")) as f:
        g = json.load(f)
    wg, wu, wd, n = _embed_row0(g, "unit_exp2")
    qg, qu, qd, sb = oracle.unpack_expert(oracle.pack_expert(wg, wu, wd), 64, 64)
    assert oracle.f32_from_bf16_bits(sb)[0] == np.float32(2.0 ** g["sigma_expected_exp2"])
    assert qg[0, :n].tolist() == g["gate_expected"]
    assert qu[0, :n].tolist() == g["up_expected"]
    assert qd[:n, 0].tolist() == g["down_expected"]


def _embed_row0(g, exp_key):
    """Place a golden case's values in row 0 of a 64x64 expert (gate/up row 0,
    down column 0); every other weight is zero."""
    u = np.float32(2.0 ** g[exp_key])
    n = len(g["gate_units"])
    wg = np.zeros((64, 64), np.float32)
    wu = np.zeros((64, 64), np.float32)
    wd = np.zeros((64, 64), np.float32)
    wg[0, :n] = np.float32(g["gate_units"]) * u
    wu[0, :n] = np.float32(g["up_units"]) * u
    wd[:n, 0] = np.float32(g["down_units"]) * u
    return wg, wu, wd, n


def test_tile_layout_golden_offsets():
    """Hand-computed byte offsets of marked elements in a C=128, R=64 blob."""
    with open(os.path.join(GOLDEN, "pack_layout.json")) as f:
        g = json.load(f)
    C, R = g["C"], g["R"]
    s = np.float32(2.0 ** -7)
    mats = {"gate": np.zeros((R, C), np.float32), "up": np.zeros((R, C), np.float32),
            "down": np.zeros((C, R), np.float32)}
    for r in range(R):                      # every row needs |q| = 127 somewhere: put it in up
        mats["up"][r, C - 1] = 127 * s
    for m in g["marks"]:
        mats[m["matrix"]][m["row"], m["col"]] = m["q"] * s
    blob = oracle.pack_expert(mats["gate"], mats["up"], mats["down"])
    for m in g["marks"]:
        assert blob.view(np.int8)[m["offset"]] == m["q"], m
    assert blob[g["sigma_offset"]:g["sigma_offset"] + 2].view("<u2")[0] == 0x3C00  # 2^-7
