"""GPU parity of the fused step entry point (bs_mixed_state_step) against the
fp64 oracle's whole step, its equality with the separate K1/K2/K3/K1^-1
calls, multi-layer pointer arrays, the phase-timing ring and argument checks."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_attention, check_step_decode, lazy, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    torch, bs, _ = lazy()
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    c = bs.Context(0)
    yield c
    c.close()


def make_state(w, n_layers=None):
    """Device StepState plus the host inputs it was built from."""
    torch, bs, bstep = lazy()
    n_layers = w.layers if n_layers is None else n_layers
    tok, msk, blk = synth.gen_state(w)
    layers, host = [], []
    for l in range(n_layers):
        q = synth.gen_q(w, l)
        kn, vn = synth.gen_kv_new(w, l)
        kc, vc = synth.gen_cache(w, l)
        out = torch.full(q.shape, float("nan"), dtype=bstep.torch_dtype(w.dtype), device="cuda")
        layers.append(bstep.Layer(bstep.to_device(q, w.dtype), bstep.to_device(kn, w.dtype),
                                  bstep.to_device(vn, w.dtype), bstep.to_device(kc, w.dtype),
                                  bstep.to_device(vc, w.dtype), out))
        host.append(dict(q=q, k_new=kn, v_new=vn, k_cache=kc, v_cache=vc))
    logits = synth.gen_logits(w, blk)
    st = bstep.StepState(w.L, w.Hq, w.Hkv, w.D, w.V, w.dtype, w.R, w.W, bstep.to_device(tok), bstep.to_device(msk),
                         layers, bstep.to_device(logits, w.dtype), w.n, tau=w.tau, q_min=w.q_min,
                         eos_id=w.eos_id).alloc()
    return st, dict(tokens=tok, mask=msk, blk=blk, layers=host, logits=logits)


def snapshot(st):
    _, _, bstep = lazy()
    return dict(tokens=st.tokens.cpu().numpy(), mask=st.mask.cpu().numpy(), pos=st.pos.cpu().numpy(),
                conf=st.conf.cpu().numpy(), n_unmasked=st.n_unmasked.cpu().numpy(), done=st.done.cpu().numpy(),
                eos_seen=st.eos_seen.cpu().numpy(),
                layers=[dict(out=bstep.to_host(x.out), k_cache=bstep.to_host(x.k_cache),
                             v_cache=bstep.to_host(x.v_cache)) for x in st.layers])


def check_step(w, got, ref, host, label):
    """Attention per layer within tolerance, caches bit-exact, decode per
    position on the dense state (outside the 1e-3 band: bit-exact), cells of
    the dense boxes outside the active blocks untouched."""
    for l, (g, r) in enumerate(zip(got["layers"], ref["layers"])):
        check_attention(w, g["out"], r["out"], label=f"{label} layer {l}")
        np.testing.assert_array_equal(g["k_cache"], r["k_cache"])     # bf16: bit patterns on both sides
        np.testing.assert_array_equal(g["v_cache"], r["v_cache"])
    np.testing.assert_array_equal(got["pos"], ref["pos"])
    stats = check_step_decode(w, w.reqs, got, ref["decode"], host["tokens"], host["mask"], label)
    # every cell outside the active blocks (other columns, rows of no request) is untouched
    gtok, _ = oracle.gather_active_blocks(w.reqs, w.L, got["tokens"])
    gmsk, _ = oracle.gather_active_blocks(w.reqs, w.L, got["mask"])
    np.testing.assert_array_equal(oracle.scatter_active_blocks(w.reqs, w.L, gtok, host["tokens"]), got["tokens"])
    np.testing.assert_array_equal(oracle.scatter_active_blocks(w.reqs, w.L, gmsk, host["mask"]), got["mask"])
    return stats


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_fused_step_matches_oracle(ctx, cfg):
    torch, bs, bstep = lazy()
    w = synth.workload(cfg)
    say(f"[fused step cfg{cfg}] n={w.n} W={w.W} layers={w.layers}")
    st, host = make_state(w)
    bstep.run_step(ctx, st, w.reqs, want_conf=True)
    torch.cuda.synchronize()
    got = snapshot(st)
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                  tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    stats = check_step(w, got, ref, host, f"cfg{cfg}")
    say(f"  decode: {stats}")
    assert stats.band <= max(4, stats.positions // 50), stats


@pytest.mark.parametrize("seed", range(24))
def test_fused_step_random_geometries(ctx, seed):
    # seeded random batches: block length, head grouping, head dimension,
    # vocabulary, prompt and generation lengths, block indices (partial last
    # blocks, empty suffixes), row order with unused rows and padding slack;
    # the small ones leave CUs idle, so seeds 1-3, 11, 15, 19 and 20 (MHA)
    # run split-KV plans
    torch, bs, bstep = lazy()
    g_ = np.random.default_rng(9000 + seed)
    L = int(g_.choice([8, 16, 32, 64]))
    Hq, Hkv = [(4, 4), (8, 2), (14, 2), (8, 1)][seed % 4]
    D = 64 if seed % 3 == 0 else 128
    V = 8 * int(g_.integers(40, 700))                 # rows stay a multiple of 16 bytes
    n = int(g_.integers(1, 13))
    p = g_.integers(0, 200, n)
    gen = g_.integers(1, 200, n)
    k = np.array([int(g_.integers(0, -(-int(x) // L))) for x in gen])
    rows = g_.permutation(n + int(g_.integers(0, 4)))[:n]
    W = int((p + gen).max()) + int(g_.integers(0, 24))
    w = synth.custom(L, Hq, Hkv, D, V, "bf16", list(p), list(gen), list(k), W=W, rows=list(rows), variant=seed,
                     kv_sigma=1 / D ** 0.5)
    say(f"[fused step random {seed}] n={n} L={L} Hq={Hq} Hkv={Hkv} D={D} V={V} W={W} R={w.R}")
    st, host = make_state(w)
    bstep.run_step(ctx, st, w.reqs, want_conf=True)
    torch.cuda.synchronize()
    got = snapshot(st)
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                  tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    stats = check_step(w, got, ref, host, f"random {seed}")
    say(f"  decode: {stats}")


@pytest.mark.parametrize("cfg,L", [(2, 16), (2, 64), (3, 16), (3, 64)])
def test_fused_step_block_length_sweep(ctx, cfg, L):
    """The block-length ablation at kernel level: the same LLaDA- and
    Dream-shaped requests re-blocked at L = 16 and 64 (at L = 64 the Dream
    query groups are split into two row-block workgroups)."""
    torch, bs, bstep = lazy()
    w = synth.workload(cfg, block_length=L)
    say(f"[fused step {w.name}] n={w.n} W={w.W}")
    st, host = make_state(w)
    bstep.run_step(ctx, st, w.reqs, want_conf=True)
    torch.cuda.synchronize()
    got = snapshot(st)
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                  tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    stats = check_step(w, got, ref, host, w.name)
    say(f"  decode: {stats}")
    assert stats.band <= max(4, stats.positions // 50), stats


@pytest.mark.parametrize("Hq,Hkv", [(28, 4), (8, 8)])
def test_fused_step_split_kv_stragglers(ctx, Hq, Hkv):
    """A small batch with one long row, two layers: the fused step runs the
    split-KV plan (partial slots after the decode's part of its workspace)
    and matches the oracle; it equals the separate calls given the same
    workspace byte for byte, and the whole-row step within the attention
    bound (decode outputs identical)."""
    torch, bs, bstep = lazy()
    g_ = np.random.default_rng(77)
    n = 12
    p = g_.integers(40, 400, n)
    p[4] = 3000
    gen = np.full(n, 96)
    k = g_.integers(0, 3, n)
    w = synth.custom(32, Hq, Hkv, 128, 2048, "bf16", list(p), list(gen), list(k), variant=3, layers=2,
                     kv_sigma=128 ** -0.5)
    items, parts = bs.bs_attention_work_list(w.reqs, w.L, w.Hq, w.Hkv, w.D, bs.BS_BF16, 1)
    say(f"[fused step split-KV G={Hq // Hkv}] n={n} W={w.W}: {len(items)} work items, {parts} partial slots")
    assert parts > 0
    a, host = make_state(w)
    b, _ = make_state(w)
    c, _ = make_state(w)
    bstep.run_step(ctx, a, w.reqs, want_conf=True, fused=True)
    bstep.run_step(ctx, b, w.reqs, want_conf=True, fused=False)
    bstep.run_step(ctx, c, w.reqs, want_conf=True, fused=True, split=False)
    torch.cuda.synchronize()
    ga, gb, gc = snapshot(a), snapshot(b), snapshot(c)
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                  tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    stats = check_step(w, ga, ref, host, f"split-KV G={Hq // Hkv}")
    say(f"  decode: {stats}")
    for key in ("tokens", "mask", "pos", "conf", "n_unmasked", "done", "eos_seen"):
        np.testing.assert_array_equal(ga[key], gb[key], err_msg=key)
        np.testing.assert_array_equal(ga[key], gc[key], err_msg=key)
    for la, lb, lc in zip(ga["layers"], gb["layers"], gc["layers"]):
        for key in ("out", "k_cache", "v_cache"):
            np.testing.assert_array_equal(la[key], lb[key], err_msg=key)
        np.testing.assert_array_equal(la["k_cache"], lc["k_cache"])
        np.testing.assert_array_equal(la["v_cache"], lc["v_cache"])
        check_attention(w, la["out"], oracle.widen(lc["out"], w.dtype), label="split vs whole rows")


def test_fused_step_equals_separate_calls(ctx):
    """Same kernels, same order: the fused call and the K1/K2/K3/K1^-1
    sequence give identical bytes (GQA shapes, three layers)."""
    torch, bs, bstep = lazy()
    w = synth.workload(3, layers=3)
    say("[fused vs separate cfg3 x3 layers]")
    a, _ = make_state(w)
    b, _ = make_state(w)
    bstep.run_step(ctx, a, w.reqs, want_conf=True, fused=True)
    bstep.run_step(ctx, b, w.reqs, want_conf=True, fused=False)
    torch.cuda.synchronize()
    ga, gb = snapshot(a), snapshot(b)
    for key in ("tokens", "mask", "pos", "conf", "n_unmasked", "done", "eos_seen"):
        np.testing.assert_array_equal(ga[key], gb[key], err_msg=key)
    for la, lb in zip(ga["layers"], gb["layers"]):
        for key in ("out", "k_cache", "v_cache"):
            np.testing.assert_array_equal(la[key], lb[key], err_msg=key)


def test_fused_step_multi_layer_matches_oracle(ctx):
    """Layer l's pointers reach layer l's launch: four layers of distinct
    seeded tensors (fp32, tiny), each checked against the oracle."""
    torch, bs, bstep = lazy()
    w = synth.workload(1, layers=4)
    st, host = make_state(w)
    bstep.run_step(ctx, st, w.reqs, want_conf=True)
    torch.cuda.synchronize()
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], host["layers"], host["logits"],
                                  tau=w.tau, q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    check_step(w, snapshot(st), ref, host, "cfg1 x4 layers")


def test_fused_step_decode_only_and_empty_batch(ctx):
    torch, bs, bstep = lazy()
    w = synth.workload(1)
    st, host = make_state(w)
    bstep.run_step(ctx, st, w.reqs, want_conf=True, layers=[])     # n_layers = 0: K3 alone
    torch.cuda.synchronize()
    got = snapshot(st)
    ref = oracle.mixed_state_step(w.reqs, w.L, host["tokens"], host["mask"], [], host["logits"], tau=w.tau,
                                  q_min=w.q_min, eos_id=w.eos_id, dtype=w.dtype)
    got["layers"] = []
    check_step(w, got, ref, host, "decode only")
    bstep.run_step(ctx, st, w.reqs[:0])                               # n = 0: no-op
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.tokens.cpu().numpy(), got["tokens"])


def test_profile_ring_records_phases(ctx):
    torch, bs, bstep = lazy()
    w = synth.workload(2, layers=2)
    st, _ = make_state(w)
    tok0, msk0 = st.tokens.clone(), st.mask.clone()
    for rep in range(2):                       # the second round reuses the ring's events
        bs.bs_profile_begin(ctx, 4)
        for _ in range(6):                     # two more steps than the ring holds
            st.tokens.copy_(tok0)
            st.mask.copy_(msk0)
            bstep.run_step(ctx, st, w.reqs)
        ph = bs.bs_profile_end(ctx, 8)
        assert ph.shape == (4, len(bs.PROFILE_PHASES))
        assert (ph > 0).all() and (ph < 100).all(), ph
    with pytest.raises(bs.BlockServeError, match="not started"):
        bs.bs_profile_end(ctx, 4)


def test_fused_step_rejects_before_launch(ctx):
    torch, bs, bstep = lazy()
    w = synth.workload(1, layers=2)
    st, _ = make_state(w)
    tok = st.tokens.clone()
    lays = [(x.q, x.k_new, x.v_new, x.k_cache, x.v_cache, x.out) for x in st.layers]
    lays[1] = lays[1][:5] + (None,)
    with pytest.raises(bs.BlockServeError, match="layer 1"):
        bs.bs_mixed_state_step(ctx, w.reqs, w.L, w.R, w.W, lays, w.Hq, w.Hkv, w.D, bs.BS_F32, 0.0, 1, w.V,
                               bs.BS_F32, st.logits, st.logits.stride(1), st.tokens, w.W, st.mask, w.W, w.tau, 1, -1,
                               st.n_unmasked, st.done, st.eos_seen, None, None, st.dec_ws, st.dec_ws.numel())
    with pytest.raises(bs.BlockServeError, match="row strides"):
        bs.bs_mixed_state_step(ctx, w.reqs, w.L, w.R, w.W, [], w.Hq, w.Hkv, w.D, bs.BS_F32, 0.0, 1, w.V,
                               bs.BS_F32, st.logits, st.logits.stride(1), st.tokens, w.W - 1, st.mask, w.W, w.tau, 1,
                               -1, st.n_unmasked, st.done, st.eos_seen, None, None, st.dec_ws, st.dec_ws.numel())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.tokens.cpu().numpy(), tok.cpu().numpy())   # nothing ran
