"""GPU parity of the output-head decoding step (bs_lm_head_decode) against the
oracle: logits produced from hidden states by the fused MFMA kernel and
reduced on the fly, then the selection. Small ragged shapes in full, the
LLaDA-8B (d 4096, V 126464) and Dream-7B (d 3584, V 152064) shapes on seeded
samples of requests, no-op and poisoned-row cases, argument checks.

The logits are fp32 sums of exact bf16 products on the GPU and exact fp64
sums in the oracle, so they differ by accumulation rounding (about 1e-5 on
logits of magnitude 20): confidences agree within LM_CONF_TOL, and a
position whose two largest oracle logits lie within ARG_GAP may pick either
id (that position accepts either id; counted). Selection decisions are
compared per position, with the 1e-3 band around tau and around ties exempt
and counted."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_decode, lazy, say

pytestmark = pytest.mark.gpu

LM_CONF_TOL = 2e-4
ARG_GAP = 1e-3


@pytest.fixture(scope="module")
def ctx():
    torch, bs, _ = lazy()
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    c = bs.Context(0)
    yield c
    c.close()


def run_lm(ctx, w, hidden, wv, tok_c, msk_c, tau=None, q_min=None, ldw=None, dev_hidden=None):
    torch, bs, bstep = lazy()
    n, d = w.n, wv.shape[1]
    ldw = d if ldw is None else ldw
    wpad = np.zeros((wv.shape[0], ldw), np.uint16)
    wpad[:, :d] = wv
    dw = bstep.to_device(wpad, "bf16")
    pb = bs.bs_lm_head_pack_bytes(w.V, d)
    dp = torch.full((pb // 2,), 7, dtype=torch.int16, device="cuda")     # every byte is written by the pack
    bs.bs_lm_head_pack(ctx, dw, ldw, w.V, d, bs.BS_BF16, dp, pb)
    dh = bstep.to_device(hidden, "bf16") if dev_hidden is None else dev_hidden
    dt = bstep.to_device(tok_c)
    dm = bstep.to_device(msk_c)
    nun = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    done = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    eos = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    conf = torch.full((n, w.L), float("nan"), dtype=torch.float32, device="cuda")
    wsb = bs.bs_lm_head_workspace_bytes(n, w.L, w.V)
    ws = torch.full((max(wsb, 16),), 0xAB, dtype=torch.uint8, device="cuda")
    bs.bs_lm_head_decode(ctx, w.reqs, w.L, d, w.V, bs.BS_BF16, dh, dp, dt, dm,
                         w.tau if tau is None else tau, w.q_min if q_min is None else q_min, w.eos_id,
                         nun, done, eos, conf, ws, wsb)
    torch.cuda.synchronize()
    return dict(tokens=dt.cpu().numpy(), masked=dm.cpu().numpy(), n_unmasked=nun.cpu().numpy(),
                done=done.cpu().numpy(), eos_seen=eos.cpu().numpy(), conf=conf.cpu().numpy())


def near_ties(w, hidden, wv, msk_c, reqs_idx):
    """{(a, j): ids} for masked positions whose largest oracle logits lie
    within ARG_GAP of each other (their predicted id is not fixed at fp32
    accumulation): every id within ARG_GAP of the largest logit is accepted
    there. a indexes reqs_idx."""
    keys = [(a, i, j) for a, i in enumerate(reqs_idx) for j in range(oracle.geometry(w.reqs[i], w.L).B)
            if msk_c[i, j]]
    if not keys:
        return {}
    lg = oracle.lm_head_logits(np.stack([hidden[i, j] for _, i, j in keys]), wv, "bf16")
    out = {}
    for r, (a, i, j) in enumerate(keys):
        ids = np.nonzero(lg[r] >= lg[r].max() - ARG_GAP)[0]
        if len(ids) > 1:
            out[(a, j)] = set(int(v) for v in ids)
    return out


def lm_case(ctx, w, d, label, sample=None, tau=None, q_min=None, ldw=None):
    wv = synth.gen_lm_weight(w, d)
    hidden = synth.gen_lm_hidden(w, wv)
    tok, msk, blk = synth.gen_state(w)
    tok_c, _ = oracle.gather_active_blocks(w.reqs, w.L, tok)
    msk_c, _ = oracle.gather_active_blocks(w.reqs, w.L, msk)
    say(f"[lm head {label}] n={w.n} L={w.L} d={d} V={w.V} masked={int(blk.sum())}")
    got = run_lm(ctx, w, hidden, wv, tok_c, msk_c, tau=tau, q_min=q_min, ldw=ldw)
    idx = list(range(w.n)) if sample is None else sample
    ref = oracle.lm_head_decode(w.reqs, w.L, hidden, wv, tok_c, msk_c, tau=w.tau if tau is None else tau,
                                q_min=w.q_min if q_min is None else q_min, eos_id=w.eos_id, dtype="bf16",
                                only=idx)
    ties = near_ties(w, hidden, wv, msk_c, idx)
    sub = {k: v[idx] for k, v in ref.items() if isinstance(v, np.ndarray) and len(v) == w.n}
    gsub = {k: v[idx] for k, v in got.items()}
    stats = check_decode(w, gsub, sub, reqs=w.reqs[idx], tau=tau, label=label, q_min=q_min,
                         conf_tol=LM_CONF_TOL, alt_ids=ties, tok_in=tok_c[idx], msk_in=msk_c[idx])
    say(f"  {stats}")
    return got, ref, stats, (hidden, wv, tok_c, msk_c)


def band_ok(stats):
    return stats.band + stats.near_tie <= max(2, stats.positions // 50)


def test_lm_head_small_ragged(ctx):
    # V = 1000 (last 256-tile ragged), d = 64 (two K slices), partial blocks, empty prompt
    w = synth.custom(8, 2, 2, 16, 1000, "bf16", [5, 0, 9, 3, 14], [16, 5, 24, 20, 8], [1, 0, 1, 2, 0], W=40)
    _, _, stats, _ = lm_case(ctx, w, 64, "small")
    assert band_ok(stats), stats


@pytest.mark.parametrize("V,d", [(257, 32), (32017, 4096)])
def test_lm_head_medium(ctx, V, d):
    w = synth.custom(32, 2, 2, 16, V, "bf16", list(range(3, 131, 16)), [64] * 8, [0, 1, 0, 1, 1, 0, 1, 0])
    _, _, stats, _ = lm_case(ctx, w, d, f"V={V} d={d}")
    assert band_ok(stats), stats


@pytest.mark.parametrize("n", [22, 60, 90])
def test_lm_head_row_tile_orders(ctx, n):
    # 2, 4 and 6 row tiles of 256 masked rows: the one-row-tile-per-XCD order
    # and the order that keeps all row tiles of a vocabulary tile together
    w = synth.custom(32, 2, 2, 16, 777, "bf16", [5 + 3 * i for i in range(n)], [64] * n, [i % 2 for i in range(n)])
    _, _, stats, _ = lm_case(ctx, w, 64, f"n={n} rows")
    assert band_ok(stats), stats


def test_lm_head_largest_row_count(ctx):
    # n * L = 65536, the most the call accepts: 1024 requests with 64-position
    # blocks (about 32k masked rows, 128 row tiles); a seeded sample of 64
    # requests is checked against the oracle
    n = 1024
    w = synth.custom(64, 2, 2, 16, 300, "bf16", [3 + i % 17 for i in range(n)], [64] * n, [0] * n)
    sample = sorted(np.random.default_rng(9).choice(n, size=64, replace=False).tolist())
    _, _, stats, _ = lm_case(ctx, w, 32, "n*L=65536", sample=sample)
    assert band_ok(stats), stats


@pytest.mark.parametrize("cfg", [2, 3])
def test_lm_head_full_size_sampled(ctx, cfg):
    w = synth.workload(cfg)
    d = synth.LM_HEAD_DIM[cfg]
    sample = sorted(np.random.default_rng(70 + cfg).choice(w.n, size=6, replace=False).tolist())
    _, _, stats, _ = lm_case(ctx, w, d, f"cfg{cfg}", sample=sample)
    assert band_ok(stats), stats


def test_lm_head_strided_head_and_quota(ctx):
    # w rows padded to a longer stride; fixed-quota schedule (threshold disabled)
    w = synth.custom(16, 2, 2, 16, 3001, "bf16", [7, 40, 0], [32, 48, 17], [1, 0, 1])
    got, ref, _, inp = lm_case(ctx, w, 96, "ldw=136 quota 3", tau=1.5, q_min=3, ldw=136)
    msk_c = inp[3]
    for i, r in enumerate(w.reqs):
        nm = int(msk_c[i, :oracle.geometry(r, w.L).B].sum())
        assert got["n_unmasked"][i] == min(nm, 3)


def test_lm_head_unread_rows_may_hold_nan(ctx):
    torch, bs, bstep = lazy()
    w = synth.custom(8, 2, 2, 16, 700, "bf16", [4, 9], [16, 6], [1, 0])
    wv = synth.gen_lm_weight(w, 64)
    hidden = synth.gen_lm_hidden(w, wv)
    tok, msk, blk = synth.gen_state(w)
    tok_c, _ = oracle.gather_active_blocks(w.reqs, w.L, tok)
    msk_c, _ = oracle.gather_active_blocks(w.reqs, w.L, msk)
    a = run_lm(ctx, w, hidden, wv, tok_c, msk_c)
    poisoned = hidden.copy()
    for i, r in enumerate(w.reqs):
        B = oracle.geometry(r, w.L).B
        for j in range(w.L):
            if j >= B or not msk_c[i, j]:
                poisoned[i, j] = synth.BF16_NAN
    b = run_lm(ctx, w, poisoned, wv, tok_c, msk_c)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)


def test_lm_head_nothing_masked_is_a_noop(ctx):
    w = synth.custom(8, 2, 2, 16, 300, "bf16", [4, 9], [16, 6], [1, 0])
    wv = synth.gen_lm_weight(w, 32)
    hidden = synth.gen_lm_hidden(w, wv)
    tok_c = np.full((w.n, w.L), 5, np.int32)
    msk_c = np.zeros((w.n, w.L), np.uint8)
    got = run_lm(ctx, w, hidden, wv, tok_c, msk_c)
    assert (got["tokens"] == 5).all() and (got["masked"] == 0).all()
    assert (got["n_unmasked"] == 0).all() and (got["done"] == 1).all() and (got["conf"] == -1).all()


def test_lm_head_phase_ring(ctx):
    # the profiling ring records the call's three phases (row list, GEMM,
    # merge + selection) and stops at its capacity
    torch, bs, bstep = lazy()
    w = synth.custom(8, 2, 2, 16, 1000, "bf16", [4, 9], [16, 6], [1, 0])
    wv = synth.gen_lm_weight(w, 64)
    hidden = synth.gen_lm_hidden(w, wv)
    tok, msk, _ = synth.gen_state(w)
    tok_c, _ = oracle.gather_active_blocks(w.reqs, w.L, tok)
    msk_c, _ = oracle.gather_active_blocks(w.reqs, w.L, msk)
    bs.bs_profile_begin(ctx, 2)
    for _ in range(3):
        run_lm(ctx, w, hidden, wv, tok_c, msk_c)
    ph = bs.bs_profile_end(ctx, 2)
    assert ph.shape == (2, len(bs.LM_PROFILE_PHASES)) and (ph > 0).all()


def test_lm_head_pack_layout(ctx):
    # the documented slab layout, checked cell by cell on the host: slab
    # (t, s) at element (t * (d / 32) + s) * 8192, row r, slot c ^ ((r >> 2) & 3)
    torch, bs, bstep = lazy()
    V, d, ldw = 300, 64, 72
    rng = np.random.default_rng(9)
    wv = rng.integers(0, 65536, size=(V, ldw), dtype=np.uint16)
    pb = bs.bs_lm_head_pack_bytes(V, d)
    assert pb == 2 * 256 * d * 2
    dp = torch.full((pb // 2,), 7, dtype=torch.int16, device="cuda")
    bs.bs_lm_head_pack(ctx, bstep.to_device(wv.view(np.int16)), ldw, V, d, bs.BS_BF16, dp, pb)
    torch.cuda.synchronize()
    got = dp.cpu().numpy().view(np.uint16)
    want = np.zeros(pb // 2, np.uint16)
    for t in range(2):
        for s in range(d // 32):
            for r in range(256):
                v = 256 * t + r
                for c in range(4):
                    dst = (t * (d // 32) + s) * 8192 + r * 32 + (c ^ ((r >> 2) & 3)) * 8
                    if v < V:
                        want[dst:dst + 8] = wv[v, 32 * s + 8 * c:32 * s + 8 * c + 8]
    np.testing.assert_array_equal(got, want)


def test_lm_head_rejects(ctx):
    torch, bs, bstep = lazy()
    w = synth.custom(8, 2, 2, 16, 300, "bf16", [4], [16], [1])
    h = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    wd = torch.zeros((300, 64), dtype=torch.bfloat16, device="cuda")
    t = torch.zeros((1, 8), dtype=torch.int32, device="cuda")
    m = torch.ones((1, 8), dtype=torch.uint8, device="cuda")
    o = [torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.uint8, device="cuda"),
         torch.zeros(1, dtype=torch.uint8, device="cuda")]
    wsb = bs.bs_lm_head_workspace_bytes(1, 8, 300)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    pb = bs.bs_lm_head_pack_bytes(300, 64)
    wp = torch.zeros(pb // 2, dtype=torch.bfloat16, device="cuda")
    for kw, match in [(dict(dt=bs.BS_F32), "UNSUPPORTED"), (dict(d=48), "UNSUPPORTED"),
                      (dict(ws_bytes=wsb - 16), "WORKSPACE")]:
        args = dict(dt=bs.BS_BF16, d=64, ws_bytes=wsb)
        args.update(kw)
        with pytest.raises(bs.BlockServeError, match=match):
            bs.bs_lm_head_decode(ctx, w.reqs, 8, args["d"], 300, args["dt"], h, wp, t, m, 0.9, 1, -1,
                                 o[0], o[1], o[2], None, ws, args["ws_bytes"])
    for kw, match in [(dict(ldw=60), "INVALID_ARG"), (dict(d=48), "UNSUPPORTED"), (dict(dt=bs.BS_F32), "UNSUPPORTED"),
                      (dict(pb=pb - 16), "WORKSPACE")]:
        args = dict(ldw=64, d=64, dt=bs.BS_BF16, pb=pb)
        args.update(kw)
        with pytest.raises(bs.BlockServeError, match=match):
            bs.bs_lm_head_pack(ctx, wd, args["ldw"], 300, args["d"], args["dt"], wp, args["pb"])
