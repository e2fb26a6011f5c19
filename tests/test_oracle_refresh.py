"""Pins for the oracle's dual-cache refresh (full-row attention with rotary
position embedding at explicit position ids).

Anchors outside the oracle: rotations written out by hand for D = 2 and D = 4
(the pairing and the frequency ladder), RoPE's complex-number form, its
relative-position property, torch's SDPA in fp64 for the unrotated case, the
already-pinned block attention on the refreshed cache, and invariants
(uniform values, a one-token row, placement in the box, batch order).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth

COS1, SIN1 = 0.5403023058681398, 0.8414709848078965
COS2, SIN2 = -0.4161468365471424, 0.9092974268256817
COS001, SIN001 = 0.9999500004166653, 0.009999833334166664


def test_rope_two_features_is_a_plane_rotation():
    # D = 2: the single pair turns by pos radians (base^0 = 1) for any base
    np.testing.assert_allclose(oracle.rope([1.0, 0.0], 1, 10000.0), [COS1, SIN1], rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.rope([0.0, 1.0], 2, 500000.0), [-SIN2, COS2], rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.rope([3.0, -2.0], 1, 7.0), [3 * COS1 + 2 * SIN1, -2 * COS1 + 3 * SIN1],
                               rtol=0, atol=1e-14)


def test_rope_pairs_feature_f_with_f_plus_half():
    # D = 4, base 10^4: pair (0, 2) turns by pos, pair (1, 3) by pos * 10^-2
    np.testing.assert_allclose(oracle.rope([1.0, 0, 0, 0], 1, 10000.0), [COS1, 0, SIN1, 0], rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.rope([0, 1.0, 0, 0], 1, 10000.0), [0, COS001, 0, SIN001], rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.rope([0, 0, 0, 1.0], 1, 10000.0), [0, -SIN001, 0, COS001], rtol=0, atol=1e-15)


def test_rope_equals_complex_multiplication():
    # RoFormer's complex form: z_f = x_f + i x_{f + D/2} times exp(i pos theta_f)
    g = np.random.default_rng(3)
    D, base = 64, 500000.0
    x = g.standard_normal((5, D))
    pos = np.array([0, 1, 17, 300, 4095])
    z = x[:, :D // 2] + 1j * x[:, D // 2:]
    theta = np.exp(-np.log(base) * np.arange(0, D, 2) / D)
    zr = z * np.exp(1j * pos[:, None] * theta[None, :])
    np.testing.assert_allclose(oracle.rope(x, pos, base), np.concatenate([zr.real, zr.imag], axis=1),
                               rtol=1e-12, atol=1e-12)


def test_rope_identity_at_zero_norm_and_disabled():
    g = np.random.default_rng(4)
    x = g.standard_normal((6, 128))
    np.testing.assert_array_equal(oracle.rope(x, np.zeros(6), 1e6), x)
    y = oracle.rope(x, np.arange(6) * 97, 1e6)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    np.testing.assert_array_equal(oracle.rope(x, np.arange(6), 0.0), x)


def test_rope_scores_depend_on_distance_only():
    g = np.random.default_rng(5)
    q, k = g.standard_normal(128), g.standard_normal(128)
    for m, n in [(5, 3), (700, 12), (3, 900), (1536, 1536)]:
        lhs = oracle.rope(q, m, 1e6) @ oracle.rope(k, n, 1e6)
        rhs = oracle.rope(q, m - n, 1e6) @ k
        assert abs(lhs - rhs) < 1e-10 * (1 + abs(lhs))


def test_row_positions_count_from_first_real_token():
    r = np.zeros(1, synth.REQ_DTYPE)[0]
    r["p"], r["g"], r["off"] = 3, 4, 5
    np.testing.assert_array_equal(oracle.row_positions(r, 12), np.arange(7))


def _wl(dtype="f32", Hq=4, Hkv=2, D=16, p=(5, 12, 7), g=(8, 16, 8), W=None, rows=None):
    return synth.custom(8, Hq, Hkv, D, 10, dtype, list(p), list(g), [0] * len(p), W=W, rows=rows,
                        kv_sigma=0.5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unrotated_refresh_matches_torch_sdpa(dtype):
    w = _wl(dtype)
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    out, _, _ = oracle.dual_cache_refresh(w.reqs, q, k, v, kc, vc, dtype=dtype, rope_base=0.0)
    G = w.Hq // w.Hkv
    for r in w.reqs:
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        Q = oracle.widen(q[row, off:off + ln], dtype).transpose(1, 0, 2).copy()        # [Hq][len][D]
        K = oracle.widen(k[row, off:off + ln], dtype).transpose(1, 0, 2).repeat(G, 0).copy()
        V = oracle.widen(v[row, off:off + ln], dtype).transpose(1, 0, 2).repeat(G, 0).copy()
        ref = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(Q), torch.from_numpy(K),
                                                               torch.from_numpy(V))
        np.testing.assert_allclose(out[row, off:off + ln].transpose(1, 0, 2), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_uniform_values_and_one_token_row():
    w = _wl(p=(0, 6), g=(1, 9))
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    r1 = w.reqs[1]
    row, off, ln = int(r1["row"]), int(r1["off"]), int(r1["p"] + r1["g"])
    v[row, off:off + ln] = v[row, off]                       # one value vector per head
    out, _, _ = oracle.dual_cache_refresh(w.reqs, q, k, v, kc, vc, dtype="f32", rope_base=10000.0)
    G = w.Hq // w.Hkv
    for h in range(w.Hq):
        np.testing.assert_allclose(out[row, off:off + ln, h], np.repeat(v[row, off, h // G][None], ln, 0),
                                   rtol=1e-12, atol=1e-14)
    r0 = w.reqs[0]                                           # len 1: the output is its own value
    row0, off0 = int(r0["row"]), int(r0["off"])
    for h in range(w.Hq):
        np.testing.assert_allclose(out[row0, off0, h], v[row0, off0, h // G], rtol=1e-12, atol=1e-15)


def test_writes_only_logical_cells():
    w = _wl("bf16")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.poison_cache(w, *synth.gen_cache(w))
    out, kc2, vc2 = oracle.dual_cache_refresh(w.reqs, q, k, v, kc, vc, dtype="bf16", rope_base=1e6)
    used = np.zeros((w.R, w.W), bool)
    for r in w.reqs:
        used[int(r["row"]), int(r["off"]):int(r["off"] + r["p"] + r["g"])] = True
    assert np.isfinite(out[used]).all() and np.isnan(out[~used]).all()
    for c in range(w.Hkv):
        assert np.isfinite(kc2[:, c][used]).all() and np.isfinite(vc2[:, c][used]).all()
        np.testing.assert_array_equal(kc2[:, c][~used], oracle.widen(kc[:, c][~used], "bf16"))
        np.testing.assert_array_equal(vc2[:, c][~used], oracle.widen(vc[:, c][~used], "bf16"))


def test_placement_in_the_box_does_not_matter():
    # the same logical rows at other offsets and rows give the same outputs and
    # cached keys at equal logical positions (position ids, not columns)
    a = _wl(W=40)
    b = _wl(W=29, rows=[2, 0, 1])
    qa, ka, va = synth.gen_refresh(a)
    kca, vca = synth.gen_cache(a)
    qb, kb, vb = synth.gen_refresh(b, poison=False)
    kcb, vcb = synth.gen_cache(b)
    for ra, rb in zip(a.reqs, b.reqs):
        ln = int(ra["p"] + ra["g"])
        sa = (int(ra["row"]), slice(int(ra["off"]), int(ra["off"]) + ln))
        sb = (int(rb["row"]), slice(int(rb["off"]), int(rb["off"]) + ln))
        qb[sb], kb[sb], vb[sb] = qa[sa], ka[sa], va[sa]
    oa, kca2, vca2 = oracle.dual_cache_refresh(a.reqs, qa, ka, va, kca, vca, dtype="f32", rope_base=10000.0)
    ob, kcb2, vcb2 = oracle.dual_cache_refresh(b.reqs, qb, kb, vb, kcb, vcb, dtype="f32", rope_base=10000.0)
    for ra, rb in zip(a.reqs, b.reqs):
        ln = int(ra["p"] + ra["g"])
        ca, cb = slice(int(ra["off"]), int(ra["off"]) + ln), slice(int(rb["off"]), int(rb["off"]) + ln)
        np.testing.assert_allclose(ob[int(rb["row"]), cb], oa[int(ra["row"]), ca], rtol=1e-13, atol=1e-14)
        np.testing.assert_array_equal(kcb2[int(rb["row"]), :, cb], kca2[int(ra["row"]), :, ca])
        np.testing.assert_array_equal(vcb2[int(rb["row"]), :, cb], vca2[int(ra["row"]), :, ca])


def test_block_rows_match_block_attention_on_the_refreshed_cache():
    # the refresh's outputs at the block rows are what the (pinned) block
    # attention computes from the refreshed cache with the rotated block q/k/v
    w = synth.custom(8, 4, 2, 16, 10, "f32", [5, 12, 7], [16, 24, 8], [1, 2, 0], kv_sigma=0.5)
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    base = 10000.0
    out, kc2, vc2 = oracle.dual_cache_refresh(w.reqs, q, k, v, kc, vc, dtype="f32", rope_base=base)
    qb = np.zeros((w.n, w.L, w.Hq, w.D)); knb = np.zeros((w.n, w.L, w.Hkv, w.D)); vnb = np.zeros_like(knb)
    for i, (r, (s, B, ln)) in enumerate(zip(w.reqs, w.spans())):
        row, off = int(r["row"]), int(r["off"])
        pos = np.arange(s, s + B)[:, None]
        qb[i, :B] = oracle.rope(q[row, off + s:off + s + B], pos, base)
        knb[i, :B] = oracle.rope(k[row, off + s:off + s + B], pos, base)
        vnb[i, :B] = v[row, off + s:off + s + B]
    blk, _, _ = oracle.dual_cache_block_attention(w.reqs, w.L, qb, knb, vnb, kc2, vc2, dtype="f64")
    for i, (r, (s, B, ln)) in enumerate(zip(w.reqs, w.spans())):
        row, off = int(r["row"]), int(r["off"])
        np.testing.assert_allclose(out[row, off + s:off + s + B], blk[i, :B], rtol=1e-12, atol=1e-14)


def test_request_alone_equals_request_in_batch():
    w = _wl("bf16")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    full, kf, vf = oracle.dual_cache_refresh(w.reqs, q, k, v, kc, vc, dtype="bf16", rope_base=5e5)
    for i, r in enumerate(w.reqs):
        one, k1, v1 = oracle.dual_cache_refresh(w.reqs[i:i + 1], q, k, v, kc, vc, dtype="bf16", rope_base=5e5)
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        np.testing.assert_array_equal(one[row, off:off + ln], full[row, off:off + ln])
        np.testing.assert_array_equal(k1[row, :, off:off + ln], kf[row, :, off:off + ln])
