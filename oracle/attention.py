"""Dual-cache block attention for one layer of a mixed-state batch.

Passages followed: paragraph "Vectorized mixed-schedule execution" (the active
block of each request is processed against its cache, and the fresh block KV
is written in place only at the physical offsets of that request's current
block, leaving the frozen prefix intact); the dual cache (cached prefix KV and
cached masked-suffix KV reused across the steps of a block) is the Fast-dLLM
mechanism the paper integrates unchanged (Sections "Experimental setup" and
"Diffusion LLM Inference Optimization"); dLLM attention is bidirectional.

Readings where the paper is silent: softmax scale 1/sqrt(D); query head h uses
KV head h // (Hq / Hkv) (consecutive query heads share a KV head); no causal
mask; a request never attends to another request's keys or to padding.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import math

import numpy as np

from .geometry import geometry, widen


def attention_rows(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * q keys^T) vals for q [m][D], keys/vals [t][D], fp64."""
    z = scale * (q @ keys.T)
    z = z - z.max(axis=1, keepdims=True)
    w = np.exp(z)
    w = w / w.sum(axis=1, keepdims=True)
    return w @ vals


def dual_cache_block_attention(reqs, L: int, q, k_new, v_new, k_cache, v_cache, *,
                               dtype: str = "f32", scale: float | None = None,
                               write_back: bool = True, only=None):
    """Block attention of every active block against its request's dual cache.

    Shapes: q [n][L][Hq][D], k_new/v_new [n][L][Hkv][D], caches [R][Hkv][W][D]
    (fp32 values or bf16 bit patterns per ``dtype``).

    For request i with block [s, e) and logical length len = p + g, query head
    h and block row j < B, the keys are the concatenation of the cached prefix
    (logical positions [0, s)), the fresh block keys k_new[i, :B], and the
    cached suffix ([e, len)); values likewise. Output rows j >= B are zero.

    Returns (out [n][L][Hq][D] fp64, k_cache', v_cache') where the returned
    caches equal the inputs except that, with ``write_back``, the active-block
    cells [off + s, off + e) of row_i hold k_new/v_new (the in-place KV update).
    ``only``: optional iterable of request indices to compute (others stay 0).
    """
    n, Lq, Hq, D = q.shape
    assert Lq == L
    Hkv = k_new.shape[2]
    assert Hq % Hkv == 0
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(D)
    out = np.zeros((n, L, Hq, D), np.float64)
    kc_out = k_cache.copy()
    vc_out = v_cache.copy()
    todo = range(n) if only is None else only
    for i in todo:
        r = reqs[i]
        t = geometry(r, L)
        for c in range(Hkv):
            kpre = widen(k_cache[t.row, c, t.off:t.off + t.s], dtype)
            vpre = widen(v_cache[t.row, c, t.off:t.off + t.s], dtype)
            kblk = widen(k_new[i, :t.B, c], dtype)
            vblk = widen(v_new[i, :t.B, c], dtype)
            ksuf = widen(k_cache[t.row, c, t.off + t.e:t.off + t.len], dtype)
            vsuf = widen(v_cache[t.row, c, t.off + t.e:t.off + t.len], dtype)
            keys = np.concatenate([kpre, kblk, ksuf], axis=0)
            vals = np.concatenate([vpre, vblk, vsuf], axis=0)
            assert keys.shape[0] == t.len
            for h in range(c * G, (c + 1) * G):
                out[i, :t.B, h] = attention_rows(widen(q[i, :t.B, h], dtype), keys, vals, scale)
    if write_back:
        for i, r in enumerate(reqs):
            t = geometry(r, L)
            for c in range(Hkv):
                kc_out[t.row, c, t.off + t.s:t.off + t.e] = k_new[i, :t.B, c]
                vc_out[t.row, c, t.off + t.s:t.off + t.e] = v_new[i, :t.B, c]
    return out, kc_out, vc_out
