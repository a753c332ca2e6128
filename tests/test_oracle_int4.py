"""Pins for the oracle's INT4 variant (group-64 fp16 scales, Table I's INT4
point; the format choices are listed in the oracle's notes).

Each pin fixes a value by hand or by an exact construction: grid weights
round-trip exactly, one element lands at the byte and nibble the layout
formula names, the fp16 scale rounding ties to even and the integers are made
against the stored scale, and the degenerate groups (all zero, overflowing)
take the stated scales.
"""
import numpy as np
import pytest

import oracle


def _grid_int4(rng, rows, K):
    """w = q * s with q in [-7, 7], every group holding a +-7, s a power of two
    per (row, group): exactly representable, so packing must return q and s."""
    q = rng.integers(-7, 8, size=(rows, K))
    g = q.reshape(rows, K // 64, 64)
    g[:, :, 5] = np.where(rng.random((rows, K // 64)) < 0.5, 7, -7)
    s = 2.0 ** rng.integers(-12, -3, size=(rows, K // 64))
    w = (q.reshape(rows, K // 64, 64) * s[:, :, None]).reshape(rows, K)
    return q.astype(np.int8), s.astype(np.float16), w.astype(np.float32)


def test_packed_bytes_closed_form():
    # per matrix rows*K/2 nibble bytes + rows*K/64 fp16 scales = rows*K*17/32
    assert oracle.packed_expert_bytes_int4(4096, 14336) == 3 * 4096 * 14336 * 17 // 32
    assert oracle.packed_expert_bytes_int4(128, 128) == 26112                   # 3*8704, a multiple of 256
    assert oracle.packed_expert_bytes_int4(128, 384) == 78336                   # multiples of 128 never need padding
    assert oracle.packed_expert_bytes_int4(256, 512) % 256 == 0


def test_grid_weights_round_trip_exactly():
    rng = np.random.default_rng(0)
    C, R = 256, 128
    (qg, sg, wg), (qu, su, wu) = _grid_int4(rng, R, C), _grid_int4(rng, R, C)
    qd, sd, wd = _grid_int4(rng, C, R)
    blob = oracle.pack_expert_int4(wg, wu, wd)
    assert blob.size == oracle.packed_expert_bytes_int4(C, R)
    got = oracle.unpack_expert_int4(blob, C, R)
    for (q, s), (q0, s0) in zip(got, ((qg, sg), (qu, su), (qd, sd))):
        assert np.array_equal(q, q0)
        assert np.array_equal(s, s0)
    dq = oracle.dequantize_expert_int4(blob, C, R)
    for a, b in zip(dq, (wg, wu, wd)):
        assert np.array_equal(a, b.astype(np.float64))


def test_layout_places_one_element_by_the_formula():
    # q[5, 128 + 64 + 16*2 + 8 + 4 + 1] = 3: nibble tile (tile-row 0, column
    # pair 1), second group of the pair (bytes 8..15 of the run), run g*16 + i
    # with g = 2, i = 5, byte b = 4*1 + 1 = 5, low nibble (the +4 half):
    # offset 1024 + (2*16 + 5)*16 + 8 + 5.
    rows, K = 16, 256
    q = np.zeros((rows, K), dtype=np.int8)
    q[5, 128 + 64 + 32 + 8 + 4 + 1] = 3
    q[0, 0] = -1        # tile 0, run 0, byte 0, high nibble
    s = np.full((rows, K // 64), 1.0, dtype=np.float16)
    s[9, 3] = 0.5       # scale region at rows*K/2 = 2048: group 3, row 9 -> 2048 + 3*32 + 2*9
    flat = oracle.int4_tile_order(q, s)
    assert flat.size == 2048 + 16 * 4 * 2
    expect = np.zeros(flat.size, dtype=np.uint8)
    expect[0] = 0xF0
    expect[1024 + (2 * 16 + 5) * 16 + 8 + 5] = 0x03
    one, half = np.float16(1.0).view(np.uint16), np.float16(0.5).view(np.uint16)
    for grp in range(4):
        for i in range(16):
            v = half if (grp, i) == (3, 9) else one
            expect[2048 + grp * 32 + 2 * i] = v & 0xFF
            expect[2048 + grp * 32 + 2 * i + 1] = v >> 8
    assert np.array_equal(flat, expect)
    q2, s2 = oracle.int4_untile_order(flat, rows, K)
    assert np.array_equal(q2, q) and np.array_equal(s2, s)


def _one_group(vals):
    w = np.zeros((128, 128), dtype=np.float32)
    w[0, :len(vals)] = vals
    return w


def test_scale_ties_to_even_and_integers_use_the_stored_scale():
    # alpha = 7 * (1 + 2^-11): alpha / 7 = 1 + 2^-11 exactly, halfway between the
    # fp16 neighbours 1 and 1 + 2^-10 -> ties to even -> 1.0.
    alpha = np.float32(7.0 * (1.0 + 2.0 ** -11))
    w = _one_group([alpha, 3.5, 0.5, 1.5, 2.5, -3.5])
    q, s = _pack_matrix(w)
    assert s[0, 0] == np.float16(1.0)
    # against the stored 1.0: 3.5 -> 4 (ties to even), 0.5 -> 0, 1.5 -> 2, 2.5 -> 2, -3.5 -> -4;
    # against the unrounded 1 + 2^-11, 3.5 would give 3.
    assert list(q[0, :6]) == [7, 4, 0, 2, 2, -4]


def _pack_matrix(w):
    """Quantize one matrix the way pack_expert_int4 does (through the public
    packer: the matrix is the gate of an expert with C = R = 128)."""
    C, R = w.shape[1], w.shape[0]
    blob = oracle.pack_expert_int4(w, np.zeros_like(w), np.zeros((C, R), dtype=np.float32))
    (q, s), _, _ = oracle.unpack_expert_int4(blob, C, R)
    return q, s


def test_degenerate_groups():
    C, R = 128, 128
    w = np.zeros((R, C), dtype=np.float32)
    w[1, 3] = 1e6          # alpha / 7 overflows fp16 -> 65504; 1e6 / 65504 -> 15 -> clamp 7
    w[2, 0] = -1e-9        # alpha below eps: eps / 7 = 1.4e-9 rounds to fp16 zero -> 2^-24
    q, s = _pack_matrix(w)
    assert s[0, 0] == np.float16(2.0 ** -24)       # all-zero row
    assert s[1, 0] == np.float16(65504.0) and q[1, 3] == 7
    assert s[2, 0] == np.float16(2.0 ** -24) and q[2, 0] == 0   # -1e-9 / 2^-24 = -0.017 -> 0
    assert not q[0].any()


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.pack_expert_int4(np.zeros((64, 128)), np.zeros((64, 128)), np.zeros((128, 64)))
    with pytest.raises(ValueError):
        oracle.int4_tile_order(np.zeros((16, 64), dtype=np.int8), np.zeros((16, 1)))


def test_int4_ffn_uses_the_dequantized_weights():
    # With grid weights the INT4 blob dequantizes to the exact weights, so the
    # expert output equals the SwiGLU of those weights computed directly.
    rng = np.random.default_rng(3)
    C, R = 128, 128
    _, _, wg = _grid_int4(rng, R, C)
    _, _, wu = _grid_int4(rng, R, C)
    _, _, wd = _grid_int4(rng, C, R)
    blob = oracle.pack_expert_int4(wg, wu, wd)
    x = rng.standard_normal((3, C))
    g = x @ wg.T.astype(np.float64)
    u = x @ wu.T.astype(np.float64)
    y = (g / (1.0 + np.exp(-g)) * u) @ wd.T.astype(np.float64)
    assert np.allclose(oracle.expert_ffn(blob, x, C, R, "int4"), y, rtol=1e-12, atol=1e-15)
    with pytest.raises(ValueError):
        oracle.expert_ffn(blob, x, C, R, "int3")


def test_layout_matches_header_formulas_everywhere():
    """Every nibble and scale of an INT4 blob, read back through the header's
    offset formulas, gives the integers and scales the weights were made
    from; the marks differ pairwise in every part of the address, so a
    swapped or misplaced axis of the layout fails."""
    import int4_layout as hl
    C, R = 256, 128
    w, q, sc = hl.marked_weights(C, R)
    blob = oracle.pack_expert_int4(*w)
    assert blob.size == oracle.packed_expert_bytes_int4(C, R)
    assert not blob[3 * hl.matrix_bytes(R, C):].any()
    for (gq, gs), name in zip(hl.decode_blob(blob, C, R), ("gate", "up", "down")):
        assert np.array_equal(gq, q[name]), name
        assert np.array_equal(gs.astype(np.float64), sc[name]), name
