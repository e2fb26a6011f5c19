"""Pins for the oracle's dual-cache block attention.

The anchor is the textbook case: with the same (p, g, k) for every request, no
padding and one query head per KV head, the step is plain bidirectional
scaled-dot-product attention of the block queries over the whole
[prompt | generation] row, with the block's cached keys replaced by the fresh
ones. That is checked against torch's SDPA in fp64 and against scipy's softmax.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import synth


def _full_rows(w, q, kn, vn, kc, vc):
    """Per request: queries [B][Hq][D] and the full logical key/value rows
    [len][Hkv][D] with the fresh block written over the stale slot."""
    res = []
    for i, r in enumerate(w.reqs):
        s, B, ln = synth._span(int(r["p"]), int(r["g"]), int(r["k"]), w.L)
        row, off = int(r["row"]), int(r["off"])
        K = oracle.widen(kc[row, :, off:off + ln], w.dtype).transpose(1, 0, 2).copy()
        Vv = oracle.widen(vc[row, :, off:off + ln], w.dtype).transpose(1, 0, 2).copy()
        K[s:s + B] = oracle.widen(kn[i, :B], w.dtype)
        Vv[s:s + B] = oracle.widen(vn[i, :B], w.dtype)
        res.append((oracle.widen(q[i, :B], w.dtype), K, Vv, B))
    return res


def _inputs(w, layer=0):
    q = synth.gen_q(w, layer)
    kn, vn = synth.gen_kv_new(w, layer)
    kc, vc = synth.gen_cache(w, layer)
    return q, kn, vn, kc, vc


def _uniform_workload(dtype="f32", G=1, D=32, q_sigma=1.0):
    # identical geometry for every request, W = len (no padding)
    return synth.custom(8, 2 * G, 2, D, 10, dtype, [6, 6, 6], [24, 24, 24], [1, 1, 1],
                        q_sigma=q_sigma)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_matches_torch_sdpa_fp64(dtype):
    w = _uniform_workload(dtype)
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc, dtype=dtype)
    for i, (Q, K, Vv, B) in enumerate(_full_rows(w, q, kn, vn, kc, vc)):
        tq = torch.from_numpy(Q.transpose(1, 0, 2).copy())       # [H][B][D]
        tk = torch.from_numpy(K.transpose(1, 0, 2).copy())
        tv = torch.from_numpy(Vv.transpose(1, 0, 2).copy())
        ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=False)
        np.testing.assert_allclose(out[i, :B].transpose(1, 0, 2), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_matches_scipy_softmax_with_gqa_and_padding():
    # general case: GQA (G = 3), ragged lengths, padding, a non-empty suffix,
    # a partial block, rows out of order
    w = synth.custom(8, 6, 2, 16, 10, "f32", [5, 0, 9, 3], [16, 5, 24, 20], [1, 0, 1, 2],
                     W=40, rows=[2, 0, 3, 1])
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc)
    for i, (Q, K, Vv, B) in enumerate(_full_rows(w, q, kn, vn, kc, vc)):
        for h in range(w.Hq):
            c = h // w.G
            z = (Q[:, h] @ K[:, c].T) / math.sqrt(w.D)
            ref = scipy.special.softmax(z, axis=1) @ Vv[:, c]
            np.testing.assert_allclose(out[i, :B, h], ref, rtol=1e-12, atol=1e-13)
        assert (out[i, B:] == 0).all()


def test_gqa_equals_mha_with_repeated_kv_heads():
    w = synth.custom(8, 4, 2, 16, 10, "f32", [5, 11], [16, 24], [1, 2])
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc)
    rep = lambda x: np.repeat(x, w.G, axis=-2)
    out2, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, rep(kn), rep(vn),
                                                   np.repeat(kc, w.G, axis=1),
                                                   np.repeat(vc, w.G, axis=1))
    np.testing.assert_array_equal(out, out2)


def test_single_key_returns_its_value():
    # p = 0, g = 1, L = 1: the only key is the fresh block key itself
    w = synth.custom(1, 2, 2, 8, 10, "f32", [0, 0], [1, 1], [0, 0])
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, 1, q, kn, vn, kc, vc)
    np.testing.assert_allclose(out[:, 0], vn[:, 0].astype(np.float64), rtol=0, atol=1e-15)


def test_zero_query_gives_mean_value():
    w = synth.custom(8, 2, 2, 16, 10, "f32", [5, 11], [16, 24], [1, 2], W=40)
    q, kn, vn, kc, vc = _inputs(w)
    q[:] = 0
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc)
    for i, (Q, K, Vv, B) in enumerate(_full_rows(w, q, kn, vn, kc, vc)):
        for h in range(2):
            np.testing.assert_allclose(out[i, :B, h], np.broadcast_to(Vv[:, h].mean(0), (B, w.D)),
                                       atol=1e-14)


def test_dominant_key_exact_construction():
    # orthogonal keys: key t = M * e_t; query = e_target -> weights one-hot
    D = 16
    w = synth.custom(4, 1, 1, D, 10, "f32", [6], [8], [1], W=14)
    q = np.zeros((1, 4, 1, D), np.float32)
    kc = np.zeros((1, 1, 14, D), np.float32)
    vc = np.random.default_rng(0).standard_normal((1, 1, 14, D)).astype(np.float32)
    kn = np.zeros((1, 4, 1, D), np.float32)
    vn = np.random.default_rng(1).standard_normal((1, 4, 1, D)).astype(np.float32)
    for t in range(14):
        (kc[0, 0, t] if not (10 <= t < 14) else kn[0, t - 10, 0])[t] = 400.0
    for j, target in enumerate([3, 11, 0, 13]):
        q[0, j, 0, target] = 1.0
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, 4, q, kn, vn, kc, vc)
    for j, target in enumerate([3, 11, 0, 13]):
        exp = vc[0, 0, target] if target < 10 else vn[0, target - 10, 0]
        np.testing.assert_allclose(out[0, j, 0], exp, atol=1e-12)


def test_request_alone_equals_in_batch_and_permutation():
    w = synth.custom(8, 4, 2, 16, 10, "f32", [5, 0, 9, 3], [16, 5, 24, 20], [1, 0, 1, 2], W=40)
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc)
    for i in range(w.n):
        alone, _, _ = oracle.dual_cache_block_attention(w.reqs[i:i + 1], w.L, q[i:i + 1], kn[i:i + 1],
                                                        vn[i:i + 1], kc, vc)
        np.testing.assert_array_equal(alone[0], out[i])
    perm = np.array([2, 0, 3, 1])
    outp, _, _ = oracle.dual_cache_block_attention(w.reqs[perm], w.L, q[perm], kn[perm], vn[perm], kc, vc)
    np.testing.assert_array_equal(outp, out[perm])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_poisoned_padding_and_stale_slot_do_not_change_output(dtype):
    w = synth.custom(8, 2, 2, 16, 10, dtype, [5, 0, 9, 3], [16, 5, 24, 20], [1, 0, 1, 2], W=40)
    q, kn, vn, kc, vc = _inputs(w)
    out, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc, dtype=dtype)
    kc2, vc2 = synth.poison_cache(w, kc.copy(), vc.copy())
    out2, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc2, vc2, dtype=dtype)
    assert np.isfinite(out2).all()
    np.testing.assert_array_equal(out, out2)


def test_write_back_touches_only_block_cells():
    w = synth.custom(8, 2, 2, 16, 10, "f32", [5, 0, 9, 3], [16, 5, 24, 20], [1, 0, 1, 2], W=40)
    q, kn, vn, kc, vc = _inputs(w)
    _, kc2, vc2 = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc, write_back=True)
    diff = (kc2 != kc).any(axis=(1, 3))
    expect = np.zeros((w.R, w.W), bool)
    for i, r in enumerate(w.reqs):
        s, B, _ = synth._span(int(r["p"]), int(r["g"]), int(r["k"]), 8)
        off = int(r["off"]); row = int(r["row"])
        expect[row, off + s:off + s + B] = True
        np.testing.assert_array_equal(kc2[row, :, off + s:off + s + B], kn[i, :B].transpose(1, 0, 2))
        np.testing.assert_array_equal(vc2[row, :, off + s:off + s + B], vn[i, :B].transpose(1, 0, 2))
    np.testing.assert_array_equal(diff, expect)
    _, kc3, _ = oracle.dual_cache_block_attention(w.reqs, w.L, q, kn, vn, kc, vc, write_back=False)
    np.testing.assert_array_equal(kc3, kc)


def test_default_scale_is_inverse_sqrt_head_dim():
    w = synth.custom(8, 2, 2, 16, 10, "f32", [5], [16], [1])
    q, kn, vn, kc, vc = _inputs(w)
    a, _, _ = oracle.dual_cache_block_attention(w.reqs, 8, q, kn, vn, kc, vc, scale=0.0)
    b, _, _ = oracle.dual_cache_block_attention(w.reqs, 8, q, kn, vn, kc, vc, scale=0.25)
    np.testing.assert_array_equal(a, b)
