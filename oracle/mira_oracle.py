"""CPU oracle for the Mira per-layer MoE expert step (test infrastructure).

This module is the plain, slow, fp64 statement of what the GPU library
computes.  It is test infrastructure only: the tests, the smoke check and the
CPU-baseline leg of the benchmark import it; the product path never does, and
it shares no code, constants or helpers with the HIP library.

Paper: "Memory-Efficient MoE Inference Using Adaptive Caching and Predictive
Expert Staging" (Mira).  Each function names the passage it follows.

Readings of passages the paper leaves open (each is also listed in the design
notes of the repository):

* Packing (section IV-B, the alpha_r / s_r displays and Eqs. (2)-(4)): the
  scale is computed in fp32 as fl32(max(alpha_r, eps) / 127), rounded to the
  stored BF16 value sigma_r (round to nearest, ties to even), and the integers
  are computed against that stored sigma_r, so the stored scale is exactly the
  one the integers were made with.  round() is round-half-to-even applied to
  the correctly rounded fp32 quotient w / sigma_r; the clamp to [-127, 127]
  follows the rounding.
* Packed byte layout (section IV-B and the memory-layout figure only say the
  three INT8 matrices and the shared scale travel together): one blob per
  expert, little-endian: int8 gate [R][C], int8 up [R][C], int8 down [C][R],
  each stored as 16-row x 64-column tiles (see tile_order), then bf16 sigma
  [R], zero padding up to a multiple of 256 bytes.
* Matrix roles: the paper calls W1 the up projection and W3 the gate
  modulation without writing the FFN formula.  The library names matrices by
  role: "gate" goes through SiLU, "up" is the linear branch (Mixtral's w1 and
  w3 respectively); the shared scale treats both alike.
* Router and combine (section II-A): logits = x . Wg^T + b, top-k by value
  descending with the lower expert index winning ties; combine weights are a
  softmax over the k selected logits (renormalised top-k); shared experts, if
  any, are added with weight 1.
* INT4 variant (the workload's 4-bit, group-64, fp16-scale format; the paper
  reports INT4 only as a quality point, Table I): per row and group of 64
  consecutive columns, alpha = max |w| over the group (exact), the fp32 value
  fl32(max(alpha, eps) / 7) is rounded to fp16 (nearest, ties to even; a
  result of zero becomes the smallest positive fp16 2^-24, an overflow the
  largest finite 65504), and q = clamp(round_half_even(fl32(w / s)), -7, 7)
  against that stored s.  gate, up and down each carry their own scales.
* INT4 byte layout (rows and K multiples of 16 and 128): each matrix
  [rows][K] is a nibble region followed by a scale region.  Nibbles: tiles of
  16 rows x 128 columns (two groups), 1024 bytes each, tile-rows in order and
  column pairs in order; inside a tile the 16-byte run g*16 + i holds row i,
  columns 16g .. 16g+15 of the first group in its bytes 0..7 and of the
  second group in bytes 8..15; in each 8-byte half, byte b carries column
  16g + 8*(b//4) + (b%4) in its high nibble and that column + 4 in its low
  nibble, each nibble the two's complement of q.  Scales: fp16 (little
  endian), ordered by tile-row, then group, then the 16 rows of the tile
  (32 bytes per tile-row and group).
* Permutation: (token, slot) pairs p = t*k + j are grouped by expert with a
  stable counting sort; shared-expert pairs follow the routed ones, in token
  order.
* Predictor (section IV-E, with the MLP shape of the workload): mean-pool a
  group of token rows, z = ReLU(W1 f + b1), scores = sigmoid(W2 z + b2).
* MixtureHead (section IV-E; the paper names its parts, not their sizes):
  per group of token rows the features are the mean hidden row h, the mean
  router logits l, the selection histogram q (tokens routed to each expert of
  the source layer over the group's (token, slot) pairs, divided by
  group * k) and the top-m indicator u (1 for the m experts with the most
  routed tokens, ranked by count descending then index ascending, and only
  if the count is positive).  ActHead: a = Wa2 ReLU(Wah h + Wal l + ba1) + ba2;
  HistHead: b = Wh2 ReLU(Whq q + Whu u + bh1) + bh2; contextual gate: one
  unit over every feature, alpha = sigmoid(gh.h + gl.l + gq.q + gu.u + bg);
  the two logit vectors are mixed, y = alpha a + (1 - alpha) b, and the
  output distribution is softmax(y) (the heads are trained with
  cross-entropy).
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "BLOB_ALIGN",
    "bf16_bits_from_f32",
    "f32_from_bf16_bits",
    "packed_expert_bytes",
    "tile_order",
    "untile_order",
    "pack_expert",
    "unpack_expert",
    "dequantize_expert",
    "int4_matrix_bytes",
    "packed_expert_bytes_int4",
    "int4_tile_order",
    "int4_untile_order",
    "pack_expert_int4",
    "unpack_expert_int4",
    "dequantize_expert_int4",
    "router_logits",
    "topk_select",
    "near_tie_tokens",
    "combine_weights",
    "permute_pairs",
    "expert_ffn",
    "moe_forward",
    "predictor_scores",
    "mixture_features",
    "mixture_head",
    "coverage_at_k",
]

BLOB_ALIGN = 256  # packed blobs are zero-padded to a multiple of this many bytes


# ----------------------------------------------------------------------------
# bf16 helpers (the storage type of the shared scale, section IV-B)
# ----------------------------------------------------------------------------

def bf16_bits_from_f32(v):
    """Round fp32 values to the nearest bf16 value, ties to even.

    Written from the definition: bf16 keeps the top 16 bits of the fp32
    pattern.  Of the two bf16 neighbours of v (truncate, and truncate plus one
    unit in the last place) take the nearer; on an exact tie take the one
    whose last kept bit is zero.  Inputs must be finite.
    """
    a = np.ascontiguousarray(np.asarray(v, dtype=np.float32))
    if not np.all(np.isfinite(a)):
        raise ValueError("bf16 rounding of a non-finite value is out of contract")
    bits = a.view(np.uint32).astype(np.uint64)
    lo = bits >> 16                       # truncated pattern (toward zero)
    rem = bits & 0xFFFF                   # dropped half-word
    up = (rem > 0x8000) | ((rem == 0x8000) & ((lo & 1) == 1))
    out = lo + up.astype(np.uint64)
    return out.astype(np.uint16)


def f32_from_bf16_bits(b):
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


# ----------------------------------------------------------------------------
# a0: packing (section IV-B, alpha_r and s_r displays, Eqs. (2)-(4))
# ----------------------------------------------------------------------------

def packed_expert_bytes(C: int, R: int) -> int:
    """Bytes of one packed expert: 3*R*C int8 plus R bf16 scales, padded to 256."""
    raw = 3 * R * C + 2 * R
    return (raw + BLOB_ALIGN - 1) // BLOB_ALIGN * BLOB_ALIGN


def tile_order(q):
    """Byte order of one int8 matrix [rows][K] inside a blob.

    The matrix is cut into tiles of 16 rows x 64 columns, stored tile-row by
    tile-row and, inside a tile-row, by increasing column block.  Inside a
    tile the 1024 bytes are 64 runs of 16 consecutive columns of one row; run
    number g*16 + i holds row i of the tile, columns 16g .. 16g+15 of the
    block.  rows must be a multiple of 16 and K of 64.
    """
    q = np.asarray(q)
    rows, K = q.shape
    if rows % 16 or K % 64:
        raise ValueError("tiled layout needs rows % 16 == 0 and K % 64 == 0")
    t = q.reshape(rows // 16, 16, K // 64, 4, 16)      # [tile-row][i][block][g][c]
    return t.transpose(0, 2, 3, 1, 4).reshape(-1)        # [tile-row][block][g][i][c]


def untile_order(flat, rows, K):
    """Inverse of tile_order."""
    t = np.asarray(flat).reshape(rows // 16, K // 64, 4, 16, 16)   # [tile-row][block][g][i][c]
    return t.transpose(0, 3, 1, 2, 4).reshape(rows, K)


def _shared_row_scale(w_gate, w_up, w_down, eps):
    """alpha_r, then s_r = max(alpha_r, eps) / 127 in fp32, then bf16 storage."""
    alpha = np.maximum(
        np.maximum(np.abs(w_gate).max(axis=1), np.abs(w_up).max(axis=1)),
        np.abs(w_down).max(axis=0),
    ).astype(np.float32)
    s32 = (np.maximum(alpha, np.float32(eps)) / np.float32(127.0)).astype(np.float32)
    sigma_bits = bf16_bits_from_f32(s32)
    return alpha, s32, sigma_bits


def _quantize(w, sigma):
    """q = clamp(round(w / sigma), -127, 127), with fp32 division and ties to even."""
    quot = (w / sigma).astype(np.float32)           # correctly rounded fp32 quotient
    q = np.rint(quot)                               # round half to even
    q = np.clip(q, -127.0, 127.0)
    return q.astype(np.int8)


def pack_expert(w_gate, w_up, w_down, eps=1e-8):
    """Pack one expert into the canonical blob (uint8 array).

    w_gate, w_up: [R][C]; w_down: [C][R]; fp32 (bf16 inputs upcast exactly).
    Returns the blob of packed_expert_bytes(C, R) bytes.
    """
    w_gate = np.asarray(w_gate, dtype=np.float32)
    w_up = np.asarray(w_up, dtype=np.float32)
    w_down = np.asarray(w_down, dtype=np.float32)
    R, C = w_gate.shape
    if w_up.shape != (R, C) or w_down.shape != (C, R):
        raise ValueError("expected gate/up [R][C] and down [C][R]")
    if R % 64 or C % 64:
        raise ValueError("C and R must be multiples of 64")
    if not (np.all(np.isfinite(w_gate)) and np.all(np.isfinite(w_up)) and np.all(np.isfinite(w_down))):
        raise ValueError("non-finite weights are out of contract")
    _, _, sigma_bits = _shared_row_scale(w_gate, w_up, w_down, eps)
    sigma = f32_from_bf16_bits(sigma_bits)
    q_gate = _quantize(w_gate, sigma[:, None])
    q_up = _quantize(w_up, sigma[:, None])
    q_down = _quantize(w_down, sigma[None, :])

    blob = np.zeros(packed_expert_bytes(C, R), dtype=np.uint8)
    o = 0
    for part in (q_gate, q_up, q_down):
        n = part.size
        blob[o:o + n] = tile_order(part).view(np.uint8)
        o += n
    blob[o:o + 2 * R] = sigma_bits.astype("<u2").view(np.uint8)
    return blob


def unpack_expert(blob, C: int, R: int):
    """Inverse of the byte layout: (q_gate [R][C], q_up [R][C], q_down [C][R], sigma_bits [R])."""
    blob = np.asarray(blob, dtype=np.uint8)
    if blob.size < 3 * R * C + 2 * R:
        raise ValueError("blob too small for the given shape")
    rc = R * C
    q_gate = untile_order(blob[0:rc].view(np.int8), R, C)
    q_up = untile_order(blob[rc:2 * rc].view(np.int8), R, C)
    q_down = untile_order(blob[2 * rc:3 * rc].view(np.int8), C, R)
    sigma_bits = blob[3 * rc:3 * rc + 2 * R].view("<u2").astype(np.uint16)
    return q_gate, q_up, q_down, sigma_bits


def dequantize_expert(blob, C: int, R: int):
    """c2: W_hat = sigma_r * q (fp64, exact) for the three matrices."""
    q_gate, q_up, q_down, sigma_bits = unpack_expert(blob, C, R)
    sigma = f32_from_bf16_bits(sigma_bits).astype(np.float64)
    wg = q_gate.astype(np.float64) * sigma[:, None]
    wu = q_up.astype(np.float64) * sigma[:, None]
    wd = q_down.astype(np.float64) * sigma[None, :]
    return wg, wu, wd


# ----------------------------------------------------------------------------
# INT4 variant: group-64 scales in fp16 (Table I's INT4 point)
# ----------------------------------------------------------------------------

INT4_QMAX = 7


def int4_matrix_bytes(rows: int, K: int) -> int:
    """Nibbles (rows*K/2) plus fp16 scales (rows*K/64 of them) of one INT4 matrix."""
    return rows * K // 2 + rows * (K // 64) * 2


def packed_expert_bytes_int4(C: int, R: int) -> int:
    """Bytes of one INT4 expert: gate, up and down matrices, padded to 256."""
    n = 2 * int4_matrix_bytes(R, C) + int4_matrix_bytes(C, R)
    return (n + BLOB_ALIGN - 1) // BLOB_ALIGN * BLOB_ALIGN


def _int4_group_scales(w, eps):
    """fp16 scale per row and 64-column group (see the module notes)."""
    rows, K = w.shape
    alpha = np.abs(w).reshape(rows, K // 64, 64).max(axis=2).astype(np.float32)
    s32 = (np.maximum(alpha, np.float32(eps)) / np.float32(INT4_QMAX)).astype(np.float32)
    with np.errstate(over="ignore"):
        s16 = s32.astype(np.float16)             # round to nearest, ties to even
    s16 = np.where(np.isinf(s16), np.float16(65504.0), s16)
    s16 = np.where(s16 == 0, np.float16(2.0 ** -24), s16)
    return s16.astype(np.float16)


def _quantize_int4(w, s16):
    """q = clamp(round_half_even(fl32(w / s)), -7, 7) per group of 64 columns."""
    rows, K = w.shape
    s = s16.astype(np.float32)[:, :, None]
    quot = (w.reshape(rows, K // 64, 64) / s).astype(np.float32)
    q = np.clip(np.rint(quot), -INT4_QMAX, INT4_QMAX)
    return q.reshape(rows, K).astype(np.int8)


def int4_tile_order(q, s16):
    """Bytes of one INT4 matrix q [rows][K] with its scales s16 [rows][K/64]."""
    q = np.asarray(q)
    rows, K = q.shape
    if rows % 16 or K % 128:
        raise ValueError("the INT4 layout needs rows % 16 == 0 and K % 128 == 0")
    nib = (q.astype(np.int16) & 0xF).astype(np.uint8)
    # column inside a 128-column tile = 64e + 16g + 8h + 4p + j: e the group of
    # the pair, p = 0 high nibble, 1 low nibble
    t = nib.reshape(rows // 16, 16, K // 128, 2, 4, 2, 2, 4)          # [tr][i][pair][e][g][h][p][j]
    byte = (t[..., 0, :] << 4) | t[..., 1, :]                          # [tr][i][pair][e][g][h][j]
    byte = byte.transpose(0, 2, 4, 1, 3, 5, 6).reshape(-1)             # [tr][pair][g][i][e][h][j]
    sc = np.asarray(s16, dtype="<f2").reshape(rows // 16, 16, K // 64).transpose(0, 2, 1)
    sc = np.ascontiguousarray(sc).view(np.uint8).reshape(-1)           # [tr][group][i]
    return np.concatenate([byte.astype(np.uint8), sc])


def int4_untile_order(flat, rows, K):
    """Inverse of int4_tile_order: (q [rows][K] int8, s16 [rows][K/64])."""
    flat = np.asarray(flat, dtype=np.uint8)
    nb = rows * K // 2
    b = flat[:nb].reshape(rows // 16, K // 128, 4, 16, 2, 2, 4)      # [tr][pair][g][i][e][h][j]
    hi = (b >> 4).astype(np.int16)
    lo = (b & 0xF).astype(np.int16)
    hi = np.where(hi >= 8, hi - 16, hi)
    lo = np.where(lo >= 8, lo - 16, lo)
    q = np.stack([hi, lo], axis=6)                                     # [tr][pair][g][i][e][h][p][j]
    q = q.transpose(0, 3, 1, 4, 2, 5, 6, 7).reshape(rows, K).astype(np.int8)
    sc = np.ascontiguousarray(flat[nb:nb + rows * (K // 64) * 2]).view("<f2")
    s16 = sc.reshape(rows // 16, K // 64, 16).transpose(0, 2, 1).reshape(rows, K // 64).astype(np.float16)
    return q, s16


def pack_expert_int4(w_gate, w_up, w_down, eps=1e-8):
    """Pack one expert in the INT4 variant (uint8 array of packed_expert_bytes_int4(C, R))."""
    w_gate = np.asarray(w_gate, dtype=np.float32)
    w_up = np.asarray(w_up, dtype=np.float32)
    w_down = np.asarray(w_down, dtype=np.float32)
    R, C = w_gate.shape
    if w_up.shape != (R, C) or w_down.shape != (C, R):
        raise ValueError("expected gate/up [R][C] and down [C][R]")
    if R % 128 or C % 128:
        raise ValueError("C and R must be multiples of 128 in the INT4 layout")
    if not (np.all(np.isfinite(w_gate)) and np.all(np.isfinite(w_up)) and np.all(np.isfinite(w_down))):
        raise ValueError("non-finite weights are out of contract")
    blob = np.zeros(packed_expert_bytes_int4(C, R), dtype=np.uint8)
    o = 0
    for w in (w_gate, w_up, w_down):
        s16 = _int4_group_scales(w, eps)
        part = int4_tile_order(_quantize_int4(w, s16), s16)
        blob[o:o + part.size] = part
        o += part.size
    return blob


def unpack_expert_int4(blob, C: int, R: int):
    """((q_gate, s_gate), (q_up, s_up), (q_down, s_down)) of an INT4 blob."""
    blob = np.asarray(blob, dtype=np.uint8)
    n = int4_matrix_bytes(R, C)
    if blob.size < 3 * n:
        raise ValueError("blob too small for the given shape")
    return (int4_untile_order(blob[0:n], R, C), int4_untile_order(blob[n:2 * n], R, C),
            int4_untile_order(blob[2 * n:3 * n], C, R))


def dequantize_expert_int4(blob, C: int, R: int):
    """W_hat = s[row, group] * q (fp64, exact) for the three matrices."""
    out = []
    for q, s16 in unpack_expert_int4(blob, C, R):
        rows, K = q.shape
        s = np.repeat(s16.astype(np.float64), 64, axis=1)
        out.append(q.astype(np.float64) * s)
    return tuple(out)


# ----------------------------------------------------------------------------
# a1-a3: router, top-k, combine weights, permutation (section II-A)
# ----------------------------------------------------------------------------

def router_logits(x, w_router, bias=None):
    """Router scores over experts: l[t, e] = sum_c x[t, c] * Wg[e, c] + b[e], fp64."""
    x = np.asarray(x, dtype=np.float64)
    wg = np.asarray(w_router, dtype=np.float64)
    logits = x @ wg.T
    if bias is not None:
        logits = logits + np.asarray(bias, dtype=np.float64)[None, :]
    return logits


def topk_select(logits, k: int):
    """Top-k experts per token: value descending, lower index first on ties."""
    logits = np.asarray(logits, dtype=np.float64)
    if not np.all(np.isfinite(logits)):
        raise ValueError("non-finite router logits are out of contract")
    T, E = logits.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    idx = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        # lexsort sorts by the last key first: primary -logit, secondary index
        order = np.lexsort((np.arange(E), -logits[t]))
        idx[t] = order[:k]
    return idx


def near_tie_tokens(logits, k: int, delta: float = 1e-4):
    """Tokens whose top-(k+1) sorted logits have an adjacent gap below delta.

    On such tokens a different but equally valid rounding of the logits can
    change the selected set or its order, so callers treat them as ambiguous.
    """
    logits = np.asarray(logits, dtype=np.float64)
    T, E = logits.shape
    m = min(k + 1, E)
    out = []
    for t in range(T):
        s = np.sort(logits[t])[::-1][:m]
        if m > 1 and np.min(s[:-1] - s[1:]) < delta:
            out.append(t)
    return np.asarray(out, dtype=np.int64)


def combine_weights(logits, idx, norm_topk: bool = True):
    """Weights of the selected experts.

    norm_topk: softmax over the k selected logits (renormalised top-k).
    Otherwise: softmax over all E logits, then the selected probabilities.
    """
    logits = np.asarray(logits, dtype=np.float64)
    idx = np.asarray(idx)
    T, k = idx.shape
    w = np.empty((T, k), dtype=np.float64)
    for t in range(T):
        sel = logits[t, idx[t]]
        if norm_topk:
            e = np.exp(sel - sel.max())
            w[t] = e / e.sum()
        else:
            full = np.exp(logits[t] - logits[t].max())
            w[t] = full[idx[t]] / full.sum()
    return w


def permute_pairs(idx, n_experts: int, n_shared: int = 0):
    """Stable grouping of the (token, slot) pairs by expert.

    Routed pair p = t*k + j belongs to expert idx[t, j]; shared expert s owns
    the pairs T*k + s*T + t, one per token.  Groups are ordered routed experts
    0..E-1, then shared experts 0..S-1; inside a group pairs keep increasing
    pair index.  Returns counts [E+S], offsets [E+S+1], perm, inv where perm[pos]
    is the pair at position pos and inv[pair] its position.
    """
    idx = np.asarray(idx, dtype=np.int64)
    T, k = idx.shape
    G = n_experts + n_shared
    P = T * k + n_shared * T
    group = np.empty(P, dtype=np.int64)
    group[:T * k] = idx.reshape(-1)
    for s in range(n_shared):
        group[T * k + s * T:T * k + (s + 1) * T] = n_experts + s
    if T * k and (group[:T * k].min() < 0 or group[:T * k].max() >= n_experts):
        raise ValueError("expert index out of range")
    counts = np.zeros(G, dtype=np.int64)
    for g in group:
        counts[g] += 1
    offsets = np.zeros(G + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    fill = offsets[:-1].copy()
    perm = np.empty(P, dtype=np.int64)
    for p in range(P):                          # visiting pairs in order keeps it stable
        g = group[p]
        perm[fill[g]] = p
        fill[g] += 1
    inv = np.empty(P, dtype=np.int64)
    inv[perm] = np.arange(P)
    return counts, offsets, perm, inv


# ----------------------------------------------------------------------------
# a5-a7: expert FFN and combine (sections IV-A, IV-F; fused dequant + FFN)
# ----------------------------------------------------------------------------

def _silu(g):
    return g / (1.0 + np.exp(-g))


def expert_ffn(blob, x_rows, C: int, R: int, fmt: str = "int8"):
    """SwiGLU expert on dequantized weights: y = Wd (silu(Wg x) * (Wu x)), fp64.
    fmt: "int8" (the paper's shared-scale format) or "int4" (group-64 variant)."""
    if fmt == "int8":
        wg, wu, wd = dequantize_expert(blob, C, R)
    elif fmt == "int4":
        wg, wu, wd = dequantize_expert_int4(blob, C, R)
    else:
        raise ValueError(f"unknown format {fmt!r}")
    x = np.asarray(x_rows, dtype=np.float64).reshape(-1, C)
    g = x @ wg.T
    u = x @ wu.T
    h = _silu(g) * u
    return h @ wd.T


def moe_forward(x, w_router, bias, blobs, k: int, C: int, R: int,
                shared_blobs=(), norm_topk: bool = True, idx=None, tokens=None, fmt: str = "int8"):
    """One MoE layer (section II-A) over experts in the packed format.

    blobs[e] is routed expert e's blob, shared_blobs[s] shared expert s's.
    idx, if given, replaces the oracle's own top-k (used to evaluate an
    alternative, equally valid selection on near-tie tokens).  tokens, if
    given, restricts the computation to those token rows (outputs in that
    order).  fmt names the blobs' format ("int8" or "int4").  Returns out
    [T'][C] fp64 plus the routing intermediates.
    """
    x = np.asarray(x, dtype=np.float64)
    logits = router_logits(x, w_router, bias)
    if idx is None:
        idx = topk_select(logits, k)
    idx = np.asarray(idx, dtype=np.int32)
    w = combine_weights(logits, idx, norm_topk)
    rows = np.arange(x.shape[0]) if tokens is None else np.asarray(tokens)
    out = np.zeros((len(rows), C), dtype=np.float64)
    E = len(blobs)
    for e in range(E):                           # one expert at a time
        sel_t, sel_j = [], []
        for i, t in enumerate(rows):
            for j in range(k):
                if idx[t, j] == e:
                    sel_t.append(i)
                    sel_j.append(j)
        if not sel_t:
            continue
        xs = x[rows[sel_t]]
        y = expert_ffn(blobs[e], xs, C, R, fmt)
        for n, (i, j) in enumerate(zip(sel_t, sel_j)):
            out[i] += w[rows[i], j] * y[n]
    for sb in shared_blobs:
        out += expert_ffn(sb, x[rows], C, R, fmt)
    return {"out": out, "logits": logits, "idx": idx, "w": w}


# ----------------------------------------------------------------------------
# a8: predictor head (section IV-E; MLP shape of the workload)
# ----------------------------------------------------------------------------

def predictor_scores(x, group: int, w1, b1, w2, b2):
    """Scores over the experts of layer l+2 for each group of token rows.

    f = mean of the group's rows of x; z = ReLU(W1 f + b1);
    scores = 1 / (1 + exp(-(W2 z + b2))).  fp64.
    """
    x = np.asarray(x, dtype=np.float64)
    T, C = x.shape
    if group <= 0 or T % group:
        raise ValueError("T must be a positive multiple of group")
    n = T // group
    w1 = np.asarray(w1, dtype=np.float64)
    w2 = np.asarray(w2, dtype=np.float64)
    b1 = np.zeros(w1.shape[0]) if b1 is None else np.asarray(b1, dtype=np.float64)
    b2 = np.zeros(w2.shape[0]) if b2 is None else np.asarray(b2, dtype=np.float64)
    scores = np.empty((n, w2.shape[0]), dtype=np.float64)
    for i in range(n):
        f = x[i * group:(i + 1) * group].mean(axis=0)
        z = np.maximum(w1 @ f + b1, 0.0)
        scores[i] = 1.0 / (1.0 + np.exp(-(w2 @ z + b2)))
    return scores


def mixture_features(x, logits, topk_idx, group: int, n_src: int, m: int):
    """Features of the MixtureHead for each group of token rows (section IV-E).

    Returns (h, l, q, u): h [n][C] mean hidden row; l [n][E] mean router
    logits; q [n][E] selection histogram over the group's (token, slot) pairs,
    as fractions of group * k; u [n][E] indicator of the m experts with the
    most routed tokens (count descending, index ascending), only for experts
    with a positive count.  fp64; counts are exact integers.
    """
    x = np.asarray(x, dtype=np.float64)
    logits = np.asarray(logits, dtype=np.float64)
    topk_idx = np.asarray(topk_idx, dtype=np.int64)
    T = x.shape[0]
    if group <= 0 or T % group:
        raise ValueError("T must be a positive multiple of group")
    if logits.shape != (T, n_src) or topk_idx.shape[0] != T:
        raise ValueError("logits must be [T][n_src] and topk_idx [T][k]")
    if not 1 <= m <= n_src:
        raise ValueError("m must lie in 1..n_src")
    if topk_idx.size and (topk_idx.min() < 0 or topk_idx.max() >= n_src):
        raise ValueError("topk_idx entries must lie in 0..n_src-1")
    n, k = T // group, topk_idx.shape[1]
    h = np.empty((n, x.shape[1]))
    l = np.empty((n, n_src))
    q = np.zeros((n, n_src))
    u = np.zeros((n, n_src))
    for i in range(n):
        rows = slice(i * group, (i + 1) * group)
        h[i] = x[rows].mean(axis=0)
        l[i] = logits[rows].mean(axis=0)
        counts = np.zeros(n_src, dtype=np.int64)
        for e in topk_idx[rows].ravel():
            counts[e] += 1
        q[i] = counts / float(group * k)
        ranked = sorted(range(n_src), key=lambda e: (-counts[e], e))
        for e in ranked[:m]:
            if counts[e] > 0:
                u[i, e] = 1.0
    return h, l, q, u


def mixture_head(x, logits, topk_idx, group: int, m: int, weights: dict):
    """MixtureHead distribution over the experts of layer l+2 (section IV-E).

    weights (fp64 arrays; any bias may be None for zero):
      wah [Pa][C], wal [Pa][E], ba1 [Pa], wa2 [N][Pa], ba2 [N]   (ActHead)
      whq [Ph][E], whu [Ph][E], bh1 [Ph], wh2 [N][Ph], bh2 [N]   (HistHead)
      gh [C], gl [E], gq [E], gu [E], bg (scalar)                (gate)
    Per group: a and b are the two heads' logits, alpha the gate,
    y = alpha a + (1 - alpha) b, probs = softmax(y).  Returns a dict with
    probs [n][N], alpha [n], y [n][N], a [n][N] and b [n][N].  fp64.
    """
    W = {k: (None if v is None else np.asarray(v, dtype=np.float64)) for k, v in weights.items()}
    n_src = W["wal"].shape[1]
    h, l, q, u = mixture_features(x, logits, topk_idx, group, n_src, m)

    def bias(name, size):
        return np.zeros(size) if W.get(name) is None else W[name]

    Pa, Ph, N = W["wah"].shape[0], W["whq"].shape[0], W["wa2"].shape[0]
    n = h.shape[0]
    out = {k: np.empty((n, N)) for k in ("probs", "y", "a", "b")}
    out["alpha"] = np.empty(n)
    for i in range(n):
        za = np.maximum(W["wah"] @ h[i] + W["wal"] @ l[i] + bias("ba1", Pa), 0.0)
        a = W["wa2"] @ za + bias("ba2", N)
        zh = np.maximum(W["whq"] @ q[i] + W["whu"] @ u[i] + bias("bh1", Ph), 0.0)
        b = W["wh2"] @ zh + bias("bh2", N)
        g = W["gh"] @ h[i] + W["gl"] @ l[i] + W["gq"] @ q[i] + W["gu"] @ u[i] + float(W.get("bg") or 0.0)
        alpha = 1.0 / (1.0 + np.exp(-g))
        y = alpha * a + (1.0 - alpha) * b
        e = np.exp(y - y.max())
        out["probs"][i] = e / e.sum()
        out["y"][i], out["a"][i], out["b"][i], out["alpha"][i] = y, a, b, alpha
    return out


def coverage_at_k(pred_scores, routed_counts, k: int):
    """Mass-weighted Coverage@k (section VI-B): routed token mass on the top-k predicted experts."""
    pred_scores = np.asarray(pred_scores, dtype=np.float64)
    routed_counts = np.asarray(routed_counts, dtype=np.float64)
    order = np.lexsort((np.arange(pred_scores.size), -pred_scores))[:k]
    total = routed_counts.sum()
    return 0.0 if total == 0 else routed_counts[order].sum() / total
