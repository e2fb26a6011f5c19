"""Host-only checks of the attention work list and its split-KV plan (no GPU):
every row's 64-key tiles are covered exactly once, cut rows take consecutive
partial slots, the launch order is longest piece first, and the workspace
queries size exactly the plan's partial slots."""
import numpy as np

import synth
import paper_2607_08930_amd as bs


def _rows(w):
    G, RB = w.Hq // w.Hkv, (w.L + 31) // 32
    split_rb = RB if G * RB > 8 else 1
    waves = G * (1 if G * RB > 8 else RB)
    rows = {}
    for i, r in enumerate(w.reqs):
        nt = -(-(int(r["p"]) + int(r["g"])) // 64)
        for h in range(w.Hkv):
            for rb in range(split_rb):
                rows[(i, h, rb)] = nt
    return rows, waves


def _check_plan(w, items, n_parts):
    rows, _ = _rows(w)
    by_row = {}
    for req, kvh, rb, t0, t1, part in items.tolist():
        by_row.setdefault((req, kvh, rb), []).append((t0, t1, part))
    assert set(by_row) == set(rows), "every (request, KV head, row block) appears"
    slots = []
    for key, pieces in by_row.items():
        pieces.sort()
        nt = rows[key]
        if len(pieces) == 1:
            assert pieces[0] == (0, nt, -1), f"whole row {key}: {pieces[0]}"
            continue
        assert pieces[0][0] == 0 and pieces[-1][1] == nt, f"row {key} not covered: {pieces}"
        for (a0, a1, pa), (b0, b1, pb) in zip(pieces, pieces[1:]):
            assert a1 == b0 and a0 < a1, f"row {key}: gap or overlap {pieces}"
            assert pb == pa + 1, f"row {key}: partial slots not consecutive {pieces}"
        assert pieces[-1][0] < pieces[-1][1]
        slots += [p for _, _, p in pieces]
    assert sorted(slots) == list(range(n_parts)), "partial slots are 0 .. n_parts - 1, each once"
    tiles = items[:, 4] - items[:, 3]
    if w.Hq == w.Hkv and w.L <= 32 and len(tiles) % 4 == 0:
        # single-wave kernel: workgroup b holds items b, b + N/4, b + N/2, b + 3N/4
        tiles = tiles.reshape(-1, 4).T.reshape(-1)
    assert (np.diff(tiles) <= 0).all(), "launch order: longest piece first"


def _ws_bytes(w, n_parts):
    _, waves = _rows(w)
    return n_parts * waves * (w.D // 8 * 64 * 4 + 128) * 4


def _straggler_batch(n=24, long_p=8000, seed=2):
    rng = np.random.default_rng(seed)
    p = rng.integers(128, 1024, n)
    p[n // 3] = long_p
    return synth.custom(32, 28, 4, 128, 10, "bf16", p.tolist(), [512] * n, rng.integers(0, 16, n).tolist())


def test_plan_cuts_a_straggler_row():
    # one 8000-key row among 23 Dream-7B rows of 640-1536 keys: its four KV
    # heads are cut into pieces no longer than the other rows, the rest stay
    # whole, and the workspace queries size exactly the partial slots
    w = _straggler_batch()
    items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    whole, none = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 0)
    assert n_parts > 0 and none == 0
    _check_plan(w, items, n_parts)
    _check_plan(w, whole, 0)
    cut_reqs = set(items[items[:, 5] >= 0, 0].tolist())
    assert 8 in cut_reqs
    assert (items[:, 4] - items[:, 3]).max() <= 24 < (whole[:, 4] - whole[:, 3]).max()
    assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) == _ws_bytes(w, n_parts)
    dec = bs.bs_decode_workspace_bytes(w.n, w.L, w.V, bs.BS_BF16)
    assert bs.bs_step_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, w.V, bs.BS_BF16) == \
        (dec + 255) // 256 * 256 + _ws_bytes(w, n_parts)


def test_plan_leaves_full_batches_whole():
    # batches that fill the GPU (the Dream-7B layer: 256 rows of 640-1536 keys,
    # one per CU; the skewed batch: 756 rows) gain nothing from cuts: a tile
    # is slower when every CU runs the loop, so the total work bounds them
    for cfg in (3, 4):
        w = synth.workload(cfg)
        assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) == 0
        items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
        assert n_parts == 0 and (items[:, 5] == -1).all()
        dec = bs.bs_decode_workspace_bytes(w.n, w.L, w.V, bs.BS_BF16)
        assert bs.bs_step_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, w.V, bs.BS_BF16) == \
            (dec + 255) // 256 * 256


def test_plan_leaves_balanced_batches_whole():
    # the LLaDA-8B layer (1024 MHA rows of 326-745 keys) and 512 equal GQA rows
    w = synth.workload(2)
    assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) == 0
    items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    assert n_parts == 0 and (items[:, 5] == -1).all()
    n = 128
    w = synth.custom(32, 28, 4, 128, 10, "bf16", [500] * n, [256] * n, [3] * n)
    assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) == 0
    assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_F32) == 0


def test_plan_cuts_stragglers_into_several_pieces():
    rng = np.random.default_rng(1)
    for L, Hq, Hkv, D in [(32, 28, 4, 128), (64, 8, 2, 64), (64, 28, 4, 128), (32, 32, 32, 128), (32, 8, 8, 64)]:
        n = 40
        p = rng.integers(16, 300, n)
        p[3] = 6000
        g = np.full(n, 2 * L)
        w = synth.custom(L, Hq, Hkv, D, 10, "bf16", p.tolist(), g.tolist(), [1] * n)
        items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
        _check_plan(w, items, n_parts)
        long_pieces = items[items[:, 0] == 3]
        assert (long_pieces[:, 5] >= 0).all()
        per_row = len(long_pieces) // (w.Hkv * len(set(long_pieces[:, 2].tolist())))
        assert per_row >= 3, f"L={L} G={Hq // Hkv}: the 6000-key row is cut into {per_row} pieces"
        assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16) == _ws_bytes(w, n_parts)


def test_plan_is_a_function_of_the_descriptors():
    w = _straggler_batch()
    a = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    b = bs.bs_attention_work_list(w.reqs.copy(), w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    assert np.array_equal(a[0], b[0]) and a[1] == b[1]


def test_plan_edge_cases():
    # one request: a short row stays whole; a 20000-key row alone is cut into
    # pieces that spread it over the CUs, every piece within the cap
    for Hq, Hkv in [(28, 4), (32, 32)]:
        w = synth.custom(32, Hq, Hkv, 128, 10, "bf16", [10], [20], [0])
        items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
        assert n_parts == 0 and len(items) == Hkv
        w = synth.custom(32, Hq, Hkv, 128, 10, "bf16", [20000], [64], [1])
        items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
        _check_plan(w, items, n_parts)
        assert n_parts == len(items) and len(items) >= 4 * Hkv
        for h in range(Hkv):
            row = sorted((int(a), int(b)) for r, kv, rb, a, b, part in items.tolist() if kv == h)
            sizes = [b - a for a, b in row]
            # pieces of the cap, then the rest
            assert len(set(sizes[:-1])) == 1 and 0 < sizes[-1] <= sizes[0], sizes
    # rows shorter than one tile, and a batch with an empty work list (f32)
    w = synth.custom(32, 8, 2, 64, 10, "bf16", [0, 3, 5000], [1, 30, 32], [0, 0, 0])
    items, n_parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    _check_plan(w, items, n_parts)
    assert bs.bs_attention_workspace_bytes(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_F32) == 0


def test_work_list_rejects_unsupported_shapes():
    import pytest
    w = synth.custom(32, 8, 2, 128, 10, "bf16", [10], [20], [0])
    with pytest.raises(bs.BlockServeError):
        bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_F32, 1)
    with pytest.raises(bs.BlockServeError):
        bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, 96, bs.BS_BF16, 1)
