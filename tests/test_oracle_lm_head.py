"""Pins for the oracle's output-head decoding step (logits = h W^T, then the
decoding rule): brute-force products, an identity head, unread rows, ties."""
import numpy as np
import pytest

import oracle
import synth


def _bits(x):
    return synth.f32_to_bf16_bits(np.asarray(x, np.float32))


def _case(seed, n=3, L=4, d=6, V=11):
    rng = np.random.default_rng(seed)
    reqs, _, _ = synth.make_reqs([3] * n, [L] * n, [0] * n)
    hidden = _bits(rng.standard_normal((n, L, d)) * 2)
    wv = _bits(rng.standard_normal((V, d)))
    masked = (rng.random((n, L)) < 0.6).astype(np.uint8)
    masked[:, 0] = 1
    tokens = np.where(masked, 0, 5).astype(np.int32)
    return reqs, hidden, wv, tokens, masked


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("chunk", [3, 4096])
def test_matches_brute_force_products(seed, chunk):
    # logits written out as sums of products in plain Python, then the
    # decoding rule: a dropped term, a transposed head or a wrong row (and a
    # vocabulary chunk boundary) changes the prediction or the confidence
    n, L, d, V = 3, 4, 6, 11
    reqs, hidden, wv, tokens, masked = _case(seed, n, L, d, V)
    hf = synth.bf16_bits_to_f32(hidden).astype(float)
    wf = synth.bf16_bits_to_f32(wv).astype(float)
    logits = np.zeros((n, L, V))
    for i in range(n):
        for j in range(L):
            for v in range(V):
                logits[i, j, v] = sum(float(hf[i, j, k]) * float(wf[v, k]) for k in range(d))
    ref = oracle.parallel_decode(reqs, L, logits, tokens, masked, tau=0.3, q_min=1, dtype="f64")
    rows = np.stack([hidden[i][j] for i in range(n) for j in range(L)])
    assert np.allclose(oracle.lm_head_logits(rows, wv, "bf16", chunk=chunk),
                       logits.reshape(n * L, V), rtol=0, atol=1e-12)
    got = oracle.lm_head_decode(reqs, L, hidden, wv, tokens, masked, tau=0.3, q_min=1, dtype="bf16")
    for key in ("tokens", "masked", "n_unmasked", "done", "pred"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    np.testing.assert_allclose(got["conf"], ref["conf"], rtol=1e-12, atol=0)


def test_identity_head_gives_softmax_of_the_hidden_state():
    # W = I: the logits are the hidden state itself, so the prediction is its
    # argmax and the confidence exp(max) / sum exp(h)
    d, L = 8, 2
    reqs, _, _ = synth.make_reqs([0], [L], [0])
    h = np.array([[[0.5, 2.0, -1.0, 2.0, 0.0, 1.0, -3.0, 0.25], [0.0] * 8]], np.float32)
    wv = _bits(np.eye(d))
    r = oracle.lm_head_decode(reqs, L, _bits(h), wv, np.zeros((1, L), np.int32), np.ones((1, L), np.uint8),
                              tau=2.0, q_min=2, dtype="bf16")
    assert r["pred"][0, 0] == 1                      # 2.0 at ids 1 and 3: the smaller id
    assert r["conf"][0, 0] == pytest.approx(np.exp(2.0) / np.exp(h[0, 0].astype(float)).sum(), rel=1e-14)
    assert r["pred"][0, 1] == 0 and r["conf"][0, 1] == pytest.approx(1 / 8, rel=1e-14)
    assert r["n_unmasked"][0] == 2


def test_unmasked_and_out_of_block_rows_are_never_read():
    n, L, d, V = 2, 4, 6, 9
    reqs, _, _ = synth.make_reqs([2, 2], [4, 3], [0, 0])          # request 1: B = 3
    rng = np.random.default_rng(4)
    hidden = _bits(rng.standard_normal((n, L, d)))
    wv = _bits(rng.standard_normal((V, d)))
    masked = np.array([[1, 0, 1, 0], [0, 1, 1, 1]], np.uint8)     # (1, 3) lies past B
    tokens = np.where(masked, 0, 3).astype(np.int32)
    a = oracle.lm_head_decode(reqs, L, hidden, wv, tokens, masked, tau=0.5, dtype="bf16")
    poisoned = hidden.copy()
    poisoned[0, 1] = poisoned[0, 3] = poisoned[1, 0] = poisoned[1, 3] = synth.BF16_NAN
    b = oracle.lm_head_decode(reqs, L, poisoned, wv, tokens, masked, tau=0.5, dtype="bf16")
    for key in ("tokens", "masked", "conf", "pred"):
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    assert np.isfinite(b["conf"]).all()


def test_duplicate_head_rows_tie_to_the_smaller_id():
    d, V = 4, 6
    reqs, _, _ = synth.make_reqs([0], [1], [0])
    wv = np.zeros((V, d), np.float32)
    wv[2] = wv[4] = [1, 2, 0, 1]
    r = oracle.lm_head_decode(reqs, 1, _bits([[[1, 1, 1, 1]]]), _bits(wv), np.zeros((1, 1), np.int32),
                              np.ones((1, 1), np.uint8), tau=0.9, dtype="bf16")
    assert r["pred"][0, 0] == 2
    assert r["conf"][0, 0] == pytest.approx(np.exp(4) / (2 * np.exp(4) + 4), rel=1e-14)


def test_synthetic_head_spreads_confidences_around_the_threshold():
    # the generator's target logit sits about m above the others' LSE, m ~ U[-2, 6)
    w = synth.custom(8, 2, 2, 16, 3000, "bf16", [4, 9], [16, 8], [1, 0])
    wv = synth.gen_lm_weight(w, 64)
    h = synth.gen_lm_hidden(w, wv)
    tok, msk, blk = synth.gen_state(w)
    tok_c, _ = oracle.gather_active_blocks(w.reqs, w.L, tok)
    msk_c, _ = oracle.gather_active_blocks(w.reqs, w.L, msk)
    r = oracle.lm_head_decode(w.reqs, w.L, h, wv, tok_c, msk_c, tau=0.9, dtype="bf16")
    c = r["conf"][r["conf"] >= 0]
    assert len(c) >= 4 and c.min() < 0.9 < c.max()
