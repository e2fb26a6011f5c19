"""Pins for the oracle's KV compaction and the composed step."""
import numpy as np
import pytest

import oracle
import synth


def _box(rng, layers, R, H, W, D):
    return rng.standard_normal((layers, R, H, W, D)).astype(np.float32)


def _segs(rows):
    return np.array(rows, dtype=synth.SEG_DTYPE).reshape(-1)


def test_identity_plan_changes_nothing():
    rng = np.random.default_rng(0)
    src_k, src_v = _box(rng, 2, 3, 2, 10, 4), _box(rng, 2, 3, 2, 10, 4)
    segs = _segs([(0, r, 0, r, 0, 10) for r in range(3)])
    k, v = oracle.kv_scatter_compact(segs, src_k, src_v, None, None, src_k.copy() * 0, src_v.copy() * 0)
    np.testing.assert_array_equal(k, src_k)
    np.testing.assert_array_equal(v, src_v)


def test_round_trip_compaction_is_identity_on_valid_cells():
    rng = np.random.default_rng(1)
    L, H, W, D = 3, 2, 12, 4
    old_k, old_v = _box(rng, L, 5, H, W, D), _box(rng, L, 5, H, W, D)
    # requests live right-aligned in rows 0, 2, 4 with lengths 7, 12, 5
    live = [(0, 7), (2, 12), (4, 5)]
    fwd = _segs([(0, r, W - ln, t, W - ln, ln) for t, (r, ln) in enumerate(live)])
    new_k = np.full((L, 3, H, W, D), np.nan, np.float32); new_v = new_k.copy()
    k2, v2 = oracle.kv_scatter_compact(fwd, old_k, old_v, None, None, new_k, new_v)
    back = _segs([(0, t, W - ln, r, W - ln, ln) for t, (r, ln) in enumerate(live)])
    k3, v3 = oracle.kv_scatter_compact(back, k2, v2, None, None, np.zeros_like(old_k), np.zeros_like(old_v))
    for r, ln in live:
        np.testing.assert_array_equal(k3[:, r, :, W - ln:], old_k[:, r, :, W - ln:])
        np.testing.assert_array_equal(v3[:, r, :, W - ln:], old_v[:, r, :, W - ln:])
        assert (k3[:, r, :, :W - ln] == 0).all()
    assert (k3[:, [1, 3]] == 0).all()


def test_stable_slot_plan_leaves_survivors_untouched():
    rng = np.random.default_rng(2)
    Lr, H, W, D = 2, 2, 16, 4
    cache_k, cache_v = _box(rng, Lr, 4, H, W, D), _box(rng, Lr, 4, H, W, D)
    stg_k, stg_v = _box(rng, Lr, 2, H, W, D), _box(rng, Lr, 2, H, W, D)
    # rows 1 and 3 were evicted: admitted requests of length 9 and 16 fill them
    segs = _segs([(1, 0, 0, 1, W - 9, 9), (1, 1, 0, 3, 0, 16)])
    k, v = oracle.kv_scatter_compact(segs, cache_k, cache_v, stg_k, stg_v, cache_k, cache_v)
    np.testing.assert_array_equal(k[:, [0, 2]], cache_k[:, [0, 2]])
    np.testing.assert_array_equal(k[:, 1, :, W - 9:], stg_k[:, 0, :, :9])
    np.testing.assert_array_equal(k[:, 1, :, :W - 9], cache_k[:, 1, :, :W - 9])
    np.testing.assert_array_equal(v[:, 3], stg_v[:, 1])


def test_rejects_overlapping_destinations_and_aliasing():
    rng = np.random.default_rng(3)
    a, b = _box(rng, 1, 2, 1, 8, 2), _box(rng, 1, 2, 1, 8, 2)
    with pytest.raises(ValueError):
        oracle.kv_scatter_compact(_segs([(0, 0, 0, 1, 0, 5), (0, 0, 0, 1, 4, 3)]), a, b, None, None,
                                  a.copy(), b.copy())
    with pytest.raises(ValueError):
        oracle.kv_scatter_compact(_segs([(0, 0, 2, 0, 0, 4)]), a, b, None, None, a, b)


# ------------------------------------------------------------------ the step
def _step_inputs(w):
    tok, msk, blk = synth.gen_state(w)
    layers = []
    for l in range(w.layers):
        q = synth.gen_q(w, l); kn, vn = synth.gen_kv_new(w, l); kc, vc = synth.gen_cache(w, l)
        layers.append(dict(q=q, k_new=kn, v_new=vn, k_cache=kc, v_cache=vc))
    return tok, msk, blk, layers, synth.gen_logits(w, blk)


def _small():
    return synth.custom(8, 4, 2, 16, 40, "f32", [5, 0, 9, 3, 14], [16, 5, 24, 20, 8], [1, 0, 2, 2, 0],
                        W=40, layers=2, logits="normal", logit_sigma=3.0)


def test_step_request_alone_equals_in_batch():
    w = _small()
    tok, msk, blk, layers, logits = _step_inputs(w)
    full = oracle.mixed_state_step(w.reqs, w.L, tok, msk, layers, logits, tau=0.9)
    for i in range(w.n):
        sub = [dict(q=l["q"][i:i + 1], k_new=l["k_new"][i:i + 1], v_new=l["v_new"][i:i + 1],
                    k_cache=l["k_cache"], v_cache=l["v_cache"]) for l in layers]
        one = oracle.mixed_state_step(w.reqs[i:i + 1], w.L, tok, msk, sub, logits[i:i + 1], tau=0.9)
        row = int(w.reqs["row"][i])
        np.testing.assert_array_equal(one["tokens"][row], full["tokens"][row])
        np.testing.assert_array_equal(one["mask"][row], full["mask"][row])
        for a, b in zip(one["layers"], full["layers"]):
            np.testing.assert_array_equal(a["out"][0], b["out"][i])
            np.testing.assert_array_equal(a["k_cache"][row], b["k_cache"][row])
        for key in ("n_unmasked", "done", "eos_seen"):
            assert one["decode"][key][0] == full["decode"][key][i]


def test_step_permutation_equivariance():
    w = _small()
    tok, msk, blk, layers, logits = _step_inputs(w)
    full = oracle.mixed_state_step(w.reqs, w.L, tok, msk, layers, logits, tau=0.9)
    perm = np.array([3, 1, 4, 0, 2])
    lp = [dict(q=l["q"][perm], k_new=l["k_new"][perm], v_new=l["v_new"][perm],
               k_cache=l["k_cache"], v_cache=l["v_cache"]) for l in layers]
    pf = oracle.mixed_state_step(w.reqs[perm], w.L, tok, msk, lp, logits[perm], tau=0.9)
    np.testing.assert_array_equal(pf["tokens"], full["tokens"])
    np.testing.assert_array_equal(pf["mask"], full["mask"])
    for a, b in zip(pf["layers"], full["layers"]):
        np.testing.assert_array_equal(a["out"], b["out"][perm])
    for key in ("n_unmasked", "done"):
        np.testing.assert_array_equal(pf["decode"][key], full["decode"][key][perm])


def test_step_scatter_only_touches_active_block_cells_and_progresses():
    w = _small()
    tok, msk, blk, layers, logits = _step_inputs(w)
    r = oracle.mixed_state_step(w.reqs, w.L, tok, msk, layers, logits, tau=0.9)
    block = np.zeros((w.R, w.W), bool)
    for s_, rr in zip(w.spans(), w.reqs):
        s, B, _ = s_
        block[int(rr["row"]), int(rr["off"]) + s:int(rr["off"]) + s + B] = True
    assert ((r["tokens"] != tok) <= block).all()
    assert ((r["mask"] != msk) <= block).all()
    assert (r["decode"]["n_unmasked"] >= 1).all()
    assert int((msk.astype(int) - r["mask"].astype(int)).sum()) == int(r["decode"]["n_unmasked"].sum())
