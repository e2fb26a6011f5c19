"""Dual-cache refresh: the attention of the full-row forward that rebuilds a
request's cache when its block starts, with rotary position embedding applied
at explicit position ids.

Passages followed: the dual cache (cached prefix KV and cached masked-suffix KV,
Fast-dLLM's block-wise approximate KV cache that the paper integrates,
Sections "Experimental setup" and "Diffusion LLM Inference Optimization") is
computed by a forward over the request's whole logical row at the start of
each block and reused by the block's later steps; paragraph "Logical
positional alignment": the dense tensor is left-padded and position ids are a
cumulative count over the attention mask, so the first real token is position
0 and rotary embeddings see each request's own relative distances; new
requests admitted at a block boundary are prefilled by the same forward.
dLLM attention is bidirectional: every position of the row attends to every
position of the same row.

Readings where the paper is silent (RoPE is cited, not restated):
* RoPE as defined by RoFormer: feature pair (f, f + D/2) for f < D/2 (the
  rotate-half layout of the LLaMA-family code LLaDA and Dream build on) is
  rotated by the angle pos * base^(-2 f / D); base <= 0 disables the rotation.
* Queries and keys are rotated, values are not; the cache stores the rotated
  keys, so later block steps use them as they are.
* Softmax scale 1/sqrt(D); query head h reads KV head h // (Hq / Hkv).

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import math

import numpy as np

from .attention import attention_rows
from .geometry import position_ids, widen


def rope(x, pos, base: float) -> np.ndarray:
    """Rotary embedding of x [..., D] at positions ``pos`` (broadcast against
    x.shape[:-1]), fp64. Pair (f, f + D/2) turns by pos * base^(-2f/D)."""
    x = np.asarray(x, np.float64)
    if base is None or base <= 0:
        return x.copy()
    D = x.shape[-1]
    assert D % 2 == 0
    half = D // 2
    f = np.arange(half, dtype=np.float64)
    inv_freq = float(base) ** (-2.0 * f / D)
    ang = np.asarray(pos, np.float64)[..., None] * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def row_positions(req, W: int) -> np.ndarray:
    """Position ids of the request's logical cells [off, off + p + g) of its
    dense row: the cumulative count over the row's attention mask."""
    off, ln = int(req["off"]), int(req["p"]) + int(req["g"])
    mask = np.zeros(W, np.int64)
    mask[off:off + ln] = 1
    return position_ids(mask)[off:off + ln]


def refresh_row(req, q_row, k_row, v_row, *, dtype: str = "bf16", rope_base: float = 10000.0,
                scale: float | None = None, heads=None):
    """The refresh of one request from its dense row of projections: q_row
    [W][Hq][D], k_row/v_row [W][Hkv][D] (fp32 values or bf16 bit patterns).

    Returns (out [len][Hq][D] fp64, NaN for heads not computed; K [len][Hkv][D]
    the rotated keys; V [len][Hkv][D] the values), len = p + g, position t of
    each array being the request's logical position t (row cell off + t)."""
    W, Hq, D = q_row.shape
    Hkv = k_row.shape[1]
    assert Hq % Hkv == 0
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(D)
    off, ln = int(req["off"]), int(req["p"]) + int(req["g"])
    pos = row_positions(req, W)
    kr = rope(widen(k_row[off:off + ln], dtype), pos[:, None], rope_base)   # [len][Hkv][D]
    vv = widen(v_row[off:off + ln], dtype)
    qr = rope(widen(q_row[off:off + ln], dtype), pos[:, None], rope_base)   # [len][Hq][D]
    out = np.full((ln, Hq, D), np.nan)
    for h in (range(Hq) if heads is None else heads):
        c = h // G
        out[:, h] = attention_rows(qr[:, h], kr[:, c], vv[:, c], scale)
    return out, kr, vv


def dual_cache_refresh(reqs, q, k, v, k_cache, v_cache, *, dtype: str = "bf16",
                       rope_base: float = 10000.0, scale: float | None = None,
                       only=None, heads=None):
    """Full-row attention of the refresh forward for every listed request.

    Shapes: q [R][W][Hq][D], k/v [R][W][Hkv][D] (the projections of the whole
    dense box, token-major), caches [R][Hkv][W][D]; fp32 values or bf16 bit
    patterns per ``dtype``.

    For request i (row r, offset off, logical length len = p + g) and position
    t < len, with position id pos_t from the row's attention mask:
      K_t = rope(k[r, off + t], pos_t),  Q_t = rope(q[r, off + t], pos_t)
      out[r, off + t, h] = softmax(scale * Q_t,h . K_c^T) V_c   (keys t' < len)
      cache[r, c, off + t] = K_t,c (keys) and v[r, off + t, c] (values).

    Returns (out [R][W][Hq][D] fp64, NaN outside the computed cells; the
    refreshed caches as fp64, equal to the inputs outside the requests'
    logical cells). ``only``: request indices to compute (default all);
    ``heads``: query heads to compute (default all). Caches are refreshed for
    the listed requests only.
    """
    R, W, Hq, D = q.shape
    Hkv = k.shape[2]
    out = np.full((R, W, Hq, D), np.nan)
    kc = widen(k_cache, dtype).copy()
    vc = widen(v_cache, dtype).copy()
    todo = range(len(reqs)) if only is None else only
    for i in todo:
        r = reqs[i]
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"]) + int(r["g"])
        o, kr, vv = refresh_row(r, q[row], k[row], v[row], dtype=dtype, rope_base=rope_base, scale=scale,
                                heads=heads)
        out[row, off:off + ln] = o
        for c in range(Hkv):
            kc[row, c, off:off + ln] = kr[:, c]
            vc[row, c, off:off + ln] = vv[:, c]
    return out, kc, vc
