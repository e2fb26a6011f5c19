"""Pins for the oracle's geometry, layout, gather/scatter and host closed forms."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.geometry import DescriptorError
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden", "tiny_step_geometry.json")


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def test_tiny_geometry_matches_hand_enumeration():
    gd = _gold()
    w = synth.workload(1)
    assert w.W == gd["W"] and w.L == gd["L"]
    for i, r in enumerate(w.reqs):
        t = oracle.geometry(r, w.L)
        assert (t.p, t.g, t.k) == (gd["p"][i], gd["g"][i], gd["k"][i])
        assert t.K == gd["K"][i]
        assert t.s == gd["s"][i]
        assert t.B == gd["B"][i]
        assert t.len == gd["len"][i]
        assert t.len - t.e == gd["suffix"][i]
        assert t.off == gd["off"][i]
        assert t.off + t.s == gd["block_col"][i]
    assert oracle.bbox_cost(w.reqs, w.L) == gd["eq1_cost"]
    assert sum(oracle.geometry(r, w.L).len for r in w.reqs) == gd["sum_len"]


def test_eq1_widths_and_shrink_on_eviction():
    gd = _gold()
    w = synth.workload(1)
    widths = [int(r["p"]) + (int(r["k"]) + 1) * w.L for r in w.reqs]
    assert widths == gd["eq1_width"]
    # evicting the widest request shrinks the box (Eq. 1 discussion)
    keep = w.reqs[[0, 1, 2]]
    assert oracle.bbox_cost(keep, w.L) == 3 * 21
    assert oracle.bbox_cost(w.reqs[:0], w.L) == 0


def test_partial_last_block():
    # g not a multiple of L: K = ceil(g / L) and the last block is shorter
    r = np.array([(3, 20, 2, 0, 0)], dtype=synth.REQ_DTYPE)[0]
    t = oracle.geometry(r, 8)
    assert (t.K, t.s, t.B, t.e, t.len) == (3, 19, 4, 23, 23)


def test_position_ids_cumsum_first_real_token_is_zero():
    gd = _gold()
    for i in range(4):
        W, off, ln = gd["W"], gd["off"][i], gd["len"][i]
        attn = np.zeros(W, np.int64)
        attn[off:off + ln] = 1
        pos = oracle.position_ids(attn)
        assert pos[off] == 0
        assert (pos[:off] == -1).all()
        assert list(pos[off:]) == list(range(ln))


def test_gather_positions_agree_with_cumsum_position_ids():
    w = synth.workload(1)
    tok, _, _ = synth.gen_state(w)
    _, pos = oracle.gather_active_blocks(w.reqs, w.L, tok)
    gd = _gold()
    for i, r in enumerate(w.reqs):
        attn = np.zeros(w.W, np.int64)
        attn[int(r["off"]):int(r["off"]) + gd["len"][i]] = 1
        ids = oracle.position_ids(attn)
        col = gd["block_col"][i]
        assert list(pos[i, :gd["B"][i]]) == list(ids[col:col + gd["B"][i]])


def test_transfer_schedule_uniform():
    for n, S in [(32, 32), (7, 32), (32, 8), (33, 32), (0, 4), (100, 7)]:
        sch = oracle.transfer_schedule(n, S)
        assert len(sch) == S and sum(sch) == n
        assert max(sch) - min(sch) <= 1
        assert sch == sorted(sch, reverse=True)
    # L = S = 32 (the paper's default) gives one token per step
    assert oracle.transfer_schedule(32, 32) == [1] * 32


def test_effective_compute_ratio_closed_form():
    assert oracle.effective_compute_ratio([4, 4, 2], 4) == pytest.approx(10 / 12)
    # a static batch that drains: 16 active, then stragglers only
    assert oracle.effective_compute_ratio([16] + [1] * 9, 16) == pytest.approx(25 / 160)


@pytest.mark.parametrize("bad,err", [
    ((5, 16, 2, 0, 0), "block index"),     # k = K
    ((5, 16, -1, 0, 0), "block index"),
    ((5, 0, 0, 0, 0), "g < 1"),
    ((-1, 16, 0, 0, 0), "p < 0"),
    ((5, 16, 0, 9, 0), "row outside"),
    ((5, 16, 0, 0, 40), "fit"),           # off + len > W
    ((5, 16, 0, 0, -1), "fit"),
])
def test_validate_rejects(bad, err):
    reqs = np.array([bad], dtype=synth.REQ_DTYPE)
    with pytest.raises(DescriptorError, match=err):
        oracle.validate_reqs(reqs, 8, 4, 52)


def test_validate_rejects_duplicate_row():
    reqs = np.array([(5, 16, 0, 1, 0), (5, 16, 0, 1, 0)], dtype=synth.REQ_DTYPE)
    with pytest.raises(DescriptorError, match="duplicate"):
        oracle.validate_reqs(reqs, 8, 4, 52)
    oracle.validate_reqs(synth.workload(1).reqs, 8, 4, 52)


def _encoded_box(R, W):
    return (np.arange(R)[:, None] * 100000 + np.arange(W)[None, :]).astype(np.int64)


def test_gather_reads_hand_enumerated_cells():
    gd = _gold()
    w = synth.workload(1)
    box = _encoded_box(w.R, w.W)
    c, pos = oracle.gather_active_blocks(w.reqs, w.L, box)
    for i in range(4):
        row = int(w.reqs["row"][i])
        assert list(c[i]) == [row * 100000 + gd["block_col"][i] + j for j in range(8)]
        assert list(pos[i]) == [gd["s"][i] + j for j in range(8)]


def test_gather_zero_fills_partial_block_and_marks_pos():
    reqs, R, W = synth.make_reqs([3, 0], [20, 5], [2, 0])
    box = _encoded_box(R, W) + 1
    c, pos = oracle.gather_active_blocks(reqs, 8, box)
    assert (c[0, 4:] == 0).all() and (pos[0, 4:] == -1).all()
    assert (c[1, 5:] == 0).all() and list(pos[1, :5]) == [0, 1, 2, 3, 4]
    assert (c[0, :4] != 0).all()


def test_gather_scatter_identities():
    w = synth.custom(8, 2, 2, 16, 50, "f32", [5, 0, 9, 3], [16, 5, 24, 20], [1, 0, 2, 2],
                     W=40, rows=[2, 0, 3, 1])
    rng = np.random.default_rng(1)
    box = rng.integers(-1000, 1000, size=(w.R, w.W, 3)).astype(np.int32)
    c, _ = oracle.gather_active_blocks(w.reqs, w.L, box)
    # scatter(gather(X)) = X
    assert np.array_equal(oracle.scatter_active_blocks(w.reqs, w.L, c, box), box)
    # gather(scatter(Y)) = Y on the valid cells, and scatter touches B cells only
    y = rng.integers(-1000, 1000, size=c.shape).astype(np.int32)
    box2 = oracle.scatter_active_blocks(w.reqs, w.L, y, box)
    c2, _ = oracle.gather_active_blocks(w.reqs, w.L, box2)
    for i, r in enumerate(w.reqs):
        B = oracle.geometry(r, w.L).B
        assert np.array_equal(c2[i, :B], y[i, :B])
    changed = (box2 != box).any(axis=2).sum()
    assert changed <= sum(oracle.geometry(r, w.L).B for r in w.reqs)


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
@pytest.mark.parametrize("L", [16, 64])
def test_reblocked_workloads_are_valid_and_keep_block_starts(cfg, L):
    # the block-length sweep re-blocks the same requests: every descriptor
    # stays valid and the active block starts at the same position (L = 16)
    # or at the block boundary at most 32 positions below it (L = 64)
    w32 = synth.workload(cfg)
    w = synth.workload(cfg, block_length=L)
    assert w.L == L and f"-L{L}" in w.name
    oracle.validate_reqs(w.reqs, w.L, w.R, w.W)
    s32 = w32.reqs["p"] + 32 * w32.reqs["k"]
    s = w.reqs["p"] + L * w.reqs["k"]
    assert ((s32 - s) >= 0).all() and ((s32 - s) < max(L, 32)).all()
    if L == 16:
        assert (s == s32).all()
    for r in w.reqs:
        t = oracle.geometry(r, L)
        assert 1 <= t.B <= L and t.s + t.B <= t.len


def test_reblocking_rejects_unoffered_lengths():
    with pytest.raises(ValueError):
        synth.workload(2, block_length=48)
    with pytest.raises(ValueError):
        synth.workload(1, block_length=16)
