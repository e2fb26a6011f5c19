"""Pins for the oracle's confidence-aware parallel decode."""
import itertools
import math

import numpy as np
import pytest

import oracle
import synth


def _one(L, V, logits, masked, tau=0.9, q_min=1, eos_id=-1, tokens=None):
    reqs, _, _ = synth.make_reqs([0], [L], [0])
    logits = np.asarray(logits, np.float32).reshape(1, L, V)
    masked = np.asarray(masked, np.uint8).reshape(1, L)
    if tokens is None:
        tokens = np.where(masked, 0, 7).astype(np.int32)
    return oracle.parallel_decode(reqs, L, logits, np.asarray(tokens, np.int32).reshape(1, L), masked,
                                  tau=tau, q_min=q_min, eos_id=eos_id)


def test_ln9_margin_gives_confidence_point_nine():
    # the logit is stored in fp32, so c = sigmoid(fp32(ln 9)), within 4e-9 of
    # 0.9: a case that sits inside any threshold exemption band
    r = _one(1, 2, [[math.log(9), 0.0]], [1])
    a = float(np.float32(math.log(9)))
    assert r["conf"][0, 0] == pytest.approx(1.0 / (1.0 + math.exp(-a)), rel=1e-14)
    assert abs(r["conf"][0, 0] - 0.9) < 4e-9
    assert r["pred"][0, 0] == 0


def test_single_spike_closed_form():
    for a, V in [(0.5, 5), (3.0, 1000), (-1.0, 7), (12.0, 50)]:
        row = np.zeros(V, np.float32); row[V // 2] = a
        if a < 0:
            continue
        r = _one(1, V, [row], [1])
        assert r["conf"][0, 0] == pytest.approx(math.exp(a) / (math.exp(a) + V - 1), rel=1e-12)
        assert r["pred"][0, 0] == V // 2


def test_uniform_logits_unmask_one_at_smallest_masked_position():
    L, V = 6, 4
    masked = [0, 1, 0, 1, 1, 0]
    r = _one(L, V, np.zeros((L, V)), masked)
    conf = r["conf"][0]
    assert all(conf[j] == 0.25 for j in (1, 3, 4))
    assert all(conf[j] == -1 for j in (0, 2, 5))
    assert r["n_unmasked"][0] == 1
    assert list(r["masked"][0]) == [0, 0, 0, 1, 1, 0]
    assert r["tokens"][0, 1] == 0          # argmax of a flat row is id 0
    assert r["done"][0] == 0


def test_argmax_tie_goes_to_smallest_id():
    V = 9
    row = np.zeros(V, np.float32); row[[2, 5, 8]] = 4.0
    r = _one(1, V, [row], [1])
    scan = min(v for v in range(V) if row[v] == row.max())
    assert r["pred"][0, 0] == scan == 2


def test_at_threshold_is_inclusive():
    # V = 2 with equal logits: c = 0.5 exactly; tau = 0.5 qualifies every one
    r = _one(4, 2, np.zeros((4, 2)), [1, 1, 0, 1], tau=0.5)
    assert r["n_unmasked"][0] == 3 and r["done"][0] == 1


def _literal_rule(conf, M, tau, q):
    """The selection stated as a set property, not a sort: U is the unique
    subset of M with |U| = min(|M|, max(q, #{c >= tau})) such that every
    chosen position beats every unchosen one (higher c, or equal c and a
    smaller position)."""
    n = min(len(M), max(q, sum(1 for j in M if conf[j] >= tau)))
    beats = lambda a, b: conf[a] > conf[b] or (conf[a] == conf[b] and a < b)
    sols = [set(U) for U in itertools.combinations(M, n)
            if all(beats(a, b) for a in U for b in set(M) - set(U))]
    assert len(sols) == 1
    return sols[0]


@pytest.mark.parametrize("L,V", [(1, 2), (2, 3), (3, 5), (4, 5), (4, 2)])
def test_brute_force_all_mask_patterns(L, V):
    rng = np.random.default_rng(L * 10 + V)
    for trial in range(12):
        # quantised logits make ties in both argmax and confidence frequent
        logits = rng.integers(-2, 3, size=(L, V)).astype(np.float32) * (0.5 + trial % 3)
        for q_min, tau in [(1, 0.9), (1, 0.5), (2, 0.6), (3, 1.5), (1, 0.0)]:
            for bits in itertools.product([0, 1], repeat=L):
                r = _one(L, V, logits, bits, tau=tau, q_min=q_min)
                M = [j for j in range(L) if bits[j]]
                conf = {}
                for j in M:
                    x = logits[j].astype(np.float64)
                    conf[j] = 1.0 / sum(math.exp(v - x.max()) for v in x)
                    assert r["pred"][0, j] == min(v for v in range(V) if x[v] == x.max())
                    assert r["conf"][0, j] == pytest.approx(conf[j], rel=1e-13)
                U = _literal_rule(conf, M, tau, q_min) if M else set()
                got = {j for j in M if r["masked"][0, j] == 0}
                assert got == U
                assert r["n_unmasked"][0] == len(U)
                assert r["done"][0] == (1 if len(U) == len(M) else 0)
                for j in range(L):
                    if j in U:
                        assert r["tokens"][0, j] == r["pred"][0, j]
                    else:
                        assert r["tokens"][0, j] == (0 if bits[j] else 7)
                        assert r["masked"][0, j] == bits[j]


def test_spiked_generator_confidence_is_sigmoid_of_margin():
    w = synth.workload(2, V=4096)
    for i, j in [(0, 0), (3, 7), (11, 31)]:
        row = synth.gen_logits_row(w, i, j)
        sid, m = synth.spike_margin(w, i, j)
        a, c = oracle.row_stats(row, "bf16")
        x = oracle.widen(row, "bf16")
        others = np.delete(x, sid)
        lse = others.max() + math.log(np.exp(others - others.max()).sum())
        exact = 1.0 / (1.0 + math.exp(-(x[sid] - lse)))
        assert c == pytest.approx(exact, rel=1e-12)
        assert abs(c - 1.0 / (1.0 + math.exp(-m))) < 8e-3      # spike rounded to bf16
        if m > 0.1:
            assert a == sid


def test_progress_invariants_over_repeated_steps():
    rng = np.random.default_rng(5)
    L, V = 8, 30
    for trial in range(30):
        masked = (rng.random(L) < 0.7).astype(np.uint8)
        if not masked.any():
            masked[0] = 1
        tokens = np.where(masked, 0, 7).astype(np.int32)
        B = int(masked.sum())
        steps = 0
        while masked.any():
            logits = rng.standard_normal((L, V)).astype(np.float32) * 2
            r = _one(L, V, logits, masked, tokens=tokens)
            assert r["n_unmasked"][0] >= 1                        # at least one per step
            assert not (r["masked"][0] > masked).any()            # no re-masking
            unchanged = masked == r["masked"][0]
            assert (r["tokens"][0][unchanged] == tokens[unchanged]).all()
            masked, tokens = r["masked"][0].copy(), r["tokens"][0].copy()
            steps += 1
        assert steps <= B <= L                                    # at most B steps per block
        r = _one(L, V, np.zeros((L, V)), masked, tokens=tokens)
        assert r["n_unmasked"][0] == 0 and r["done"][0] == 1      # empty mask: no-op


def test_fixed_quota_variant():
    rng = np.random.default_rng(9)
    L, V = 8, 16
    for q in (1, 2, 3):
        masked = np.ones(L, np.uint8)
        r = _one(L, V, rng.standard_normal((L, V)) * 5, masked, tau=1.5, q_min=q)
        assert r["n_unmasked"][0] == q
    r = _one(L, V, rng.standard_normal((L, V)), [1, 0, 0, 0, 0, 0, 0, 0], tau=1.5, q_min=3)
    assert r["n_unmasked"][0] == 1 and r["done"][0] == 1


def test_eos_seen_only_on_unmasked_cells():
    V = 6
    logits = np.zeros((3, V), np.float32); logits[0, 4] = 9.0; logits[1, 2] = 9.0
    r = _one(3, V, logits, [1, 1, 1], eos_id=4)
    assert r["eos_seen"][0] == 1
    r = _one(3, V, logits, [1, 1, 1], eos_id=5)
    assert r["eos_seen"][0] == 0
    # a still-masked cell holding the eos id does not count
    r = _one(3, V, logits, [0, 0, 1], eos_id=0, tokens=[3, 3, 0])
    assert r["eos_seen"][0] == (1 if r["tokens"][0, 2] == 0 and r["masked"][0, 2] == 0 else 0)


def test_unmasked_rows_are_never_read():
    L, V = 4, 10
    rng = np.random.default_rng(2)
    logits = rng.standard_normal((L, V)).astype(np.float32)
    masked = [1, 0, 1, 0]
    a = _one(L, V, logits, masked)
    logits2 = logits.copy(); logits2[[1, 3]] = np.nan
    b = _one(L, V, logits2, masked)
    for key in ("tokens", "masked", "n_unmasked", "done"):
        np.testing.assert_array_equal(a[key], b[key])


def test_partial_block_ignores_rows_beyond_block():
    reqs, _, _ = synth.make_reqs([2], [12], [1])       # L = 8: second block has 4 rows
    L, V = 8, 5
    logits = np.full((1, L, V), np.nan, np.float32)
    logits[0, :4] = np.arange(V, dtype=np.float32)
    masked = np.ones((1, L), np.uint8)
    r = oracle.parallel_decode(reqs, L, logits, np.zeros((1, L), np.int32), masked, tau=0.99)
    assert r["n_unmasked"][0] == 1 and r["masked"][0, 0] == 0
    assert (r["masked"][0, 4:] == 1).all() and (r["conf"][0, 4:] == -1).all()
