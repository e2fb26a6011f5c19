"""GPU parity of the dual-cache refresh (bs_dual_cache_refresh) against the
oracle: rotated keys and values scattered into the cache, full-row attention
with rotated queries. Ragged small shapes (rows of 1 to 600 tokens, several
128-query chunks and 32-key tiles with ragged tails; MHA, GQA with groups of
2 and 7) in full, the LLaDA-8B and Dream-7B layer shapes on sampled requests
and heads plus whole-box properties, the unrotated case, argument checks.

Tolerances. Attention: the bf16 bound of the block attention (max abs error
1e-2 and max|d| / max|O| <= 1e-2). Cached keys: the kernel rounds the rotated
fp32 value to bf16 (half an ulp: at most 2^-8 of the value, 8 significant
bits) after computing the angle in fp32 (position times an fp32 inverse
frequency, in turns, through the hardware sine and cosine: a few 2^-23 of
the angle, bounded here by 2.5e-7 * pos rad, plus 2e-6 for the hardware sine
itself), so |K_gpu - K_ref| <= 2^-8 |K_ref| + (2.5e-7 * pos + 2e-6) * |pair|
+ 1e-7, |pair| being the norm of the feature pair the element belongs to and
pos its position. Values are copied
and must match bit for bit; with the rotation disabled, so must the keys."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import ATT_REL, ATT_TOL, lazy, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    torch, bs, _ = lazy()
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    c = bs.Context(0)
    yield c
    c.close()


def run_refresh(ctx, w, q, k, v, kc, vc, base):
    torch, bs, bstep = lazy()
    dq, dk, dv = (bstep.to_device(x, "bf16") for x in (q, k, v))
    dkc, dvc = bstep.to_device(kc, "bf16"), bstep.to_device(vc, "bf16")
    out = torch.full(dq.shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 0.0, base, dq, dk, dv, w.R, w.W,
                             dkc, dvc, out)
    torch.cuda.synchronize()
    return out, dkc, dvc


def used_cells(w):
    used = np.zeros((w.R, w.W), bool)
    for r in w.reqs:
        used[int(r["row"]), int(r["off"]):int(r["off"] + r["p"] + r["g"])] = True
    return used


def check_keys(got_bits, ref, k_bits, label):
    """got_bits [len][Hkv][D] bf16 cache cells, ref fp64 rotated keys, k_bits the unrotated inputs."""
    g = oracle.widen(got_bits, "bf16")
    x = oracle.widen(k_bits, "bf16")
    half = x.shape[-1] // 2
    pair = np.sqrt(x[..., :half] ** 2 + x[..., half:] ** 2)
    pair = np.concatenate([pair, pair], axis=-1)
    pos = np.arange(x.shape[0], dtype=np.float64).reshape((-1,) + (1,) * (x.ndim - 1))
    bound = 2.0 ** -8 * np.abs(ref) + (2.5e-7 * pos + 2e-6) * pair + 1e-7
    bad = np.abs(g - ref) > bound
    assert not bad.any(), f"{label}: {int(bad.sum())} cached keys outside the bound, worst " \
                          f"{float(np.max(np.abs(g - ref) - bound)):.3e}"


def check_request(w, i, out_h, kc_h, vc_h, q, k, v, base, heads=None, label=""):
    r = w.reqs[i]
    row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
    o, kr, vv = oracle.refresh_row(r, q[row], k[row], v[row], dtype="bf16", rope_base=base, heads=heads)
    hs = range(w.Hq) if heads is None else heads
    got = oracle.widen(out_h, "bf16")
    err, mx = 0.0, 0.0
    for h in hs:
        assert np.isfinite(got[:, h]).all(), f"{label}: request {i} head {h}: non-finite output"
        err = max(err, float(np.abs(got[:, h] - o[:, h]).max()))
        mx = max(mx, float(np.abs(o[:, h]).max()))
    assert err <= ATT_TOL["bf16"] and err / mx <= ATT_REL, \
        f"{label}: request {i}: max abs error {err:.3e} (relative {err / mx:.3e})"
    # cache cells of the row, [len][Hkv][D]
    check_keys(kc_h.transpose(1, 0, 2), kr, k[row, off:off + ln], f"{label}: request {i}")
    np.testing.assert_array_equal(vc_h.transpose(1, 0, 2), v[row, off:off + ln])
    return err, mx


def small_workload(Hq, Hkv, variant=0):
    p = [5, 300, 0, 77, 1, 190, 64]
    g = [32, 200, 1, 64, 511, 66, 128]
    k = [0] * len(p)
    return synth.custom(32, Hq, Hkv, 128, 10, "bf16", p, g, k, W=600, variant=variant,
                        kv_sigma=1 / np.sqrt(128))


@pytest.mark.parametrize("Hq,Hkv,base", [(4, 4, 10000.0), (4, 2, 500000.0), (14, 2, 1e6)])
def test_small_ragged_rows_in_full(ctx, Hq, Hkv, base):
    torch, bs, bstep = lazy()
    w = small_workload(Hq, Hkv)
    say(f"refresh small Hq={Hq} Hkv={Hkv} base={base}: lens {[int(r['p'] + r['g']) for r in w.reqs]}")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.poison_cache(w, *synth.gen_cache(w))
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, base)
    out_h, kc_h, vc_h = bstep.to_host(out), bstep.to_host(dkc), bstep.to_host(dvc)
    used = used_cells(w)
    worst = 0.0
    for i, r in enumerate(w.reqs):
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        e, _ = check_request(w, i, out_h[row, off:off + ln], kc_h[row, :, off:off + ln],
                             vc_h[row, :, off:off + ln], q, k, v, base, label="small")
        worst = max(worst, e)
    # nothing outside the logical cells is written
    assert (out_h[~used] == synth.BF16_NAN).all()
    for c in range(w.Hkv):
        np.testing.assert_array_equal(kc_h[:, c][~used], kc[:, c][~used])
        np.testing.assert_array_equal(vc_h[:, c][~used], vc[:, c][~used])
    say(f"  max abs error {worst:.2e}")


@pytest.mark.parametrize("seed", range(6))
def test_random_geometries(ctx, seed):
    # seeded random batches: head grouping, lengths 1..700 (ragged 32-key
    # tiles and 128-query chunks), row order with unused rows, padding slack,
    # rotary base; every request against the oracle, nothing else written
    torch, bs, bstep = lazy()
    g_ = np.random.default_rng(7000 + seed)
    Hq, Hkv = [(4, 4), (8, 2), (14, 2), (8, 1), (6, 3), (7, 7)][seed]
    base = [1e4, 5e5, 1e6, 0.0, 1e4, 5e5][seed]
    n = int(g_.integers(1, 9))
    p = g_.integers(0, 400, n)
    gen = g_.integers(1, 300, n)
    if seed % 2 == 0:                                  # a row shorter than one key tile
        p[0], gen[0] = 0, int(g_.integers(1, 40))
    rows = g_.permutation(n + int(g_.integers(0, 3)))[:n]
    W = int((p + gen).max()) + int(g_.integers(0, 40))
    w = synth.custom(32, Hq, Hkv, 128, 10, "bf16", list(p), list(gen), [0] * n, W=W, rows=list(rows),
                     variant=seed, kv_sigma=1 / np.sqrt(128))
    say(f"[refresh random {seed}] n={n} Hq={Hq} Hkv={Hkv} base={base} W={W} R={w.R} "
        f"lens={[int(r['p'] + r['g']) for r in w.reqs]}")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.poison_cache(w, *synth.gen_cache(w))
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, base)
    out_h, kc_h, vc_h = bstep.to_host(out), bstep.to_host(dkc), bstep.to_host(dvc)
    for i, r in enumerate(w.reqs):
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        check_request(w, i, out_h[row, off:off + ln], kc_h[row, :, off:off + ln], vc_h[row, :, off:off + ln],
                      q, k, v, base, label=f"random {seed}")
    used = used_cells(w)
    assert (out_h[~used] == synth.BF16_NAN).all()
    for c in range(w.Hkv):
        np.testing.assert_array_equal(kc_h[:, c][~used], kc[:, c][~used])
        np.testing.assert_array_equal(vc_h[:, c][~used], vc[:, c][~used])


def test_rotation_disabled_copies_keys(ctx):
    torch, bs, bstep = lazy()
    w = small_workload(4, 2, variant=1)
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, 0.0)
    out_h, kc_h = bstep.to_host(out), bstep.to_host(dkc)
    for i, r in enumerate(w.reqs):
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        np.testing.assert_array_equal(kc_h[row, :, off:off + ln].transpose(1, 0, 2), k[row, off:off + ln])
        o, _, _ = oracle.refresh_row(r, q[row], k[row], v[row], dtype="bf16", rope_base=0.0)
        d = np.abs(oracle.widen(out_h[row, off:off + ln], "bf16") - o)
        assert d.max() <= ATT_TOL["bf16"] and d.max() / np.abs(o).max() <= ATT_REL


def test_repeated_call_reuses_the_work_list(ctx):
    # the second call finds its descriptors in the upload ring; results equal
    torch, bs, bstep = lazy()
    w = small_workload(4, 2, variant=2)
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    a = run_refresh(ctx, w, q, k, v, kc, vc, 1e4)
    b = run_refresh(ctx, w, q, k, v, kc, vc, 1e4)
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


@pytest.mark.parametrize("cfg", [2, 3])
def test_full_size_sampled(ctx, cfg):
    torch, bs, bstep = lazy()
    w = synth.workload(cfg)
    base = synth.ROPE_BASE[cfg]
    say(f"refresh full size {w.name}: n={w.n} R={w.R} W={w.W} Hq={w.Hq} Hkv={w.Hkv}")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.poison_cache(w, *synth.gen_cache(w))
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, base)
    # whole box: logical cells finite, every other cell untouched
    used = torch.from_numpy(used_cells(w)).cuda()
    o = out.float()
    assert bool(torch.isfinite(o[used]).all()), "non-finite output in a logical cell"
    assert bool(torch.isnan(o[~used]).all()), "output written outside the logical cells"
    dkc_h, dvc_h = bstep.to_host(dkc), bstep.to_host(dvc)
    ucpu = used_cells(w)
    for c in range(w.Hkv):
        np.testing.assert_array_equal(dkc_h[:, c][~ucpu], kc[:, c][~ucpu])
        np.testing.assert_array_equal(dvc_h[:, c][~ucpu], vc[:, c][~ucpu])
    # sampled requests (the longest, the shortest, one at random) and heads
    lens = w.reqs["p"] + w.reqs["g"]
    gsel = np.random.default_rng(cfg)
    picks = sorted({int(np.argmax(lens)), int(np.argmin(lens)), int(gsel.integers(w.n))})
    out_h = bstep.to_host(out)
    for i in picks:
        heads = sorted({0, w.Hq - 1, int(gsel.integers(w.Hq))})
        r = w.reqs[i]
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        e, mx = check_request(w, i, out_h[row, off:off + ln], dkc_h[row, :, off:off + ln],
                              dvc_h[row, :, off:off + ln], q, k, v, base, heads=heads, label=w.name)
        say(f"  request {i} (len {ln}) heads {heads}: max abs error {e:.2e} of max |O| {mx:.2e}")


def test_empty_batch_is_a_no_op(ctx):
    torch, bs, bstep = lazy()
    t = torch.full((64,), 3.0, dtype=torch.bfloat16, device="cuda")
    empty = np.zeros(0, synth.REQ_DTYPE)
    bs.bs_dual_cache_refresh(ctx, empty, 32, 4, 2, 128, bs.BS_BF16, 0.0, 1e4, t, t, t, 1, 1, t, t, t)
    torch.cuda.synchronize()
    assert bool((t == 3.0).all())


def test_long_row(ctx):
    # one row of 4096 positions next to a short one: 16 query chunks, 64 key
    # tiles, rotation angles up to 4095 rad on the first feature pair
    torch, bs, bstep = lazy()
    w = synth.custom(32, 4, 2, 128, 10, "bf16", [3000, 10], [1096, 22], [0, 0], kv_sigma=1 / np.sqrt(128))
    say(f"refresh long row: lens {[int(r['p'] + r['g']) for r in w.reqs]} W={w.W}")
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.poison_cache(w, *synth.gen_cache(w))
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, 1e6)
    out_h, kc_h, vc_h = bstep.to_host(out), bstep.to_host(dkc), bstep.to_host(dvc)
    for i, heads in ((0, [0, 3]), (1, None)):
        r = w.reqs[i]
        row, off, ln = int(r["row"]), int(r["off"]), int(r["p"] + r["g"])
        e, mx = check_request(w, i, out_h[row, off:off + ln], kc_h[row, :, off:off + ln],
                              vc_h[row, :, off:off + ln], q, k, v, 1e6, heads=heads, label="long row")
        say(f"  request {i} (len {ln}): max abs error {e:.2e} of max |O| {mx:.2e}")


def test_refresh_then_block_step(ctx):
    # the block attention of the next denoising step, run on the refreshed
    # cache with the block's rotated queries and keys (rotated on the host
    # and rounded to bf16), reproduces the refresh's outputs at the block rows
    torch, bs, bstep = lazy()
    w = synth.custom(32, 4, 2, 128, 10, "bf16", [5, 300, 77], [64, 200, 96], [1, 3, 2], kv_sigma=1 / np.sqrt(128))
    base = 5e5
    q, k, v = synth.gen_refresh(w)
    kc, vc = synth.gen_cache(w)
    out, dkc, dvc = run_refresh(ctx, w, q, k, v, kc, vc, base)
    out_h = oracle.widen(bstep.to_host(out), "bf16")
    qb = np.zeros((w.n, w.L, w.Hq, w.D), np.float32)
    kn = np.zeros((w.n, w.L, w.Hkv, w.D), np.float32)
    vn = np.zeros_like(kn)
    for i, (r, (s0, B, ln)) in enumerate(zip(w.reqs, w.spans())):
        row, off = int(r["row"]), int(r["off"])
        pos = np.arange(s0, s0 + B)[:, None]
        qb[i, :B] = oracle.rope(oracle.widen(q[row, off + s0:off + s0 + B], "bf16"), pos, base)
        kn[i, :B] = oracle.rope(oracle.widen(k[row, off + s0:off + s0 + B], "bf16"), pos, base)
        vn[i, :B] = oracle.widen(v[row, off + s0:off + s0 + B], "bf16")
    dq, dkn, dvn = (bstep.to_device(synth.f32_to_bf16_bits(x), "bf16") for x in (qb, kn, vn))
    blk = torch.full(dq.shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    bs.bs_dual_cache_block_attention(ctx, w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 0.0, dq, dkn, dvn, dkc, dvc,
                                     w.R, w.W, 0, blk)
    torch.cuda.synchronize()
    got = oracle.widen(bstep.to_host(blk), "bf16")
    for i, (r, (s0, B, ln)) in enumerate(zip(w.reqs, w.spans())):
        row, off = int(r["row"]), int(r["off"])
        ref = out_h[row, off + s0:off + s0 + B]
        d = np.abs(got[i, :B] - ref).max()
        assert d <= ATT_TOL["bf16"] and d / np.abs(ref).max() <= 2 * ATT_REL, f"request {i}: {d:.3e}"


def test_rejects_unsupported_arguments(ctx):
    torch, bs, bstep = lazy()
    w = small_workload(4, 2)
    t = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(bs.BlockServeError, match="bf16 only"):
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, 4, 2, 128, bs.BS_F32, 0.0, 1e4, t, t, t, w.R, w.W, t, t, t)
    with pytest.raises(bs.BlockServeError, match="D = 128"):
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, 4, 2, 64, bs.BS_BF16, 0.0, 1e4, t, t, t, w.R, w.W, t, t, t)
    with pytest.raises(bs.BlockServeError, match="multiple"):
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, 3, 2, 128, bs.BS_BF16, 0.0, 1e4, t, t, t, w.R, w.W, t, t, t)
    with pytest.raises(bs.BlockServeError, match="NaN"):
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, 4, 2, 128, bs.BS_BF16, 0.0, float("nan"), t, t, t, w.R, w.W,
                                 t, t, t)
    with pytest.raises(bs.BlockServeError, match="exceeds W"):
        bs.bs_dual_cache_refresh(ctx, w.reqs, w.L, 4, 2, 128, bs.BS_BF16, 0.0, 1e4, t, t, t, w.R, 100, t, t, t)
