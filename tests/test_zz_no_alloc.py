"""The allocation-free step (bs_mixed_state_step_noalloc) against the step
with a workspace (bs_mixed_state_step): the same kernels over the same
inputs, so every output byte must agree. Three calls in a row share the
library's static device array, each smaller than the one before (a stale
larger work list and stale partials stay behind in the array): the
LLaDA-8B-shaped layer (MHA, 32 requests), 16 requests of the Dream-7B-shaped
layer (GQA 28/4) over two layers, and the tiny fp32 step. The size limits
are rejected before anything is enqueued."""
import numpy as np
import pytest

import synth
from gpu_util import lazy, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    torch, bs, _ = lazy()
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    c = bs.Context(0)
    yield c
    c.close()


def state(w, n_layers):
    torch, bs, bstep = lazy()
    tok, msk, blk = synth.gen_state(w)
    layers = []
    for l in range(n_layers):
        q = synth.gen_q(w, l)
        kn, vn = synth.gen_kv_new(w, l)
        kc, vc = synth.gen_cache(w, l)
        layers.append(bstep.Layer(bstep.to_device(q, w.dtype), bstep.to_device(kn, w.dtype), bstep.to_device(vn, w.dtype),
                                  bstep.to_device(kc, w.dtype), bstep.to_device(vc, w.dtype),
                                  torch.full(q.shape, float("nan"), dtype=bstep.torch_dtype(w.dtype), device="cuda")))
    logits = synth.gen_logits(w, blk)
    return bstep.StepState(w.L, w.Hq, w.Hkv, w.D, w.V, w.dtype, w.R, w.W, bstep.to_device(tok), bstep.to_device(msk),
                           layers, bstep.to_device(logits, w.dtype), w.n, tau=w.tau, q_min=w.q_min,
                           eos_id=w.eos_id).alloc()


def clone(st):
    import dataclasses
    torch, bs, bstep = lazy()
    lays = [bstep.Layer(x.q, x.k_new, x.v_new, x.k_cache.clone(), x.v_cache.clone(), x.out.clone())
            for x in st.layers]
    return dataclasses.replace(st, tokens=st.tokens.clone(), mask=st.mask.clone(), layers=lays).alloc()


def outputs(st, n):
    torch, bs, bstep = lazy()
    d = dict(tokens=st.tokens, mask=st.mask, conf=st.conf[:n], pos=st.pos[:n], n_unmasked=st.n_unmasked[:n],
             done=st.done[:n], eos_seen=st.eos_seen[:n])
    out = {k: v.cpu().numpy() for k, v in d.items()}
    for l, x in enumerate(st.layers):
        out[f"out{l}"] = bstep.to_host(x.out[:n])
        out[f"k{l}"] = bstep.to_host(x.k_cache)
        out[f"v{l}"] = bstep.to_host(x.v_cache)
    return out


def noalloc_step(ctx, st, reqs):
    torch, bs, bstep = lazy()
    dt = bstep.dt_code(st.dtype)
    bs.bs_mixed_state_step_noalloc(ctx, reqs, st.L, st.R, st.W,
                                   [(x.q, x.k_new, x.v_new, x.k_cache, x.v_cache, x.out) for x in st.layers],
                                   st.Hq, st.Hkv, st.D, dt, st.scale, st.write_back, st.V, dt, st.logits,
                                   st.logits.stride(1), st.tokens, st.tokens.stride(0), st.mask, st.mask.stride(0),
                                   st.tau, st.q_min, st.eos_id, st.n_unmasked, st.done, st.eos_seen, st.conf, st.pos)


def test_noalloc_step_equals_step_with_workspace(ctx):
    torch, bs, bstep = lazy()
    cases = []
    w2 = synth.workload(2)
    cases.append((w2, w2.reqs, 1, "LLaDA-8B layer, 32 requests"))
    w3 = synth.workload(3)
    cases.append((w3, w3.reqs[:16], 2, "Dream-7B layer, 16 requests, 2 layers"))
    w1 = synth.workload(1)
    cases.append((w1, w1.reqs, 1, "tiny fp32, 4 requests"))
    for w, reqs, nl, label in cases:
        say(f"[no-alloc step] {label}")
        a = state(w, nl)
        b = clone(a)
        for x in b.layers + a.layers:
            x.out.fill_(float("nan"))
        torch.cuda.synchronize()
        # the no-alloc step runs every attention row whole (no room for
        # split-KV partials), like the step given only the decode's workspace
        bstep.run_step(ctx, a, reqs, want_conf=True, split=False)
        noalloc_step(ctx, b, reqs)
        torch.cuda.synchronize()
        ga, gb = outputs(a, len(reqs)), outputs(b, len(reqs))
        for key in ga:
            np.testing.assert_array_equal(ga[key], gb[key], err_msg=f"{label}: {key}")
        assert (ga["n_unmasked"] >= 1).all()
        del a, b
        torch.cuda.empty_cache()


def test_noalloc_step_rejects_sizes_beyond_the_array(ctx):
    torch, bs, bstep = lazy()
    # decode partials: 1024 requests x 64 positions x 8 parts of a 262144-entry bf16 row x 16 B = 8 MiB
    n = 1024
    reqs = np.zeros(n, bs.REQ_DTYPE)
    reqs["g"] = 64
    reqs["row"] = np.arange(n)
    with pytest.raises(bs.BlockServeError, match="decode partials") as e:
        bs.bs_mixed_state_step_noalloc(ctx, reqs, 64, n, 64, [], 32, 32, 128, bs.BS_BF16, 0.0, 1, 262144,
                                       bs.BS_BF16, None, 262144, None, 64, None, 64, 0.9, 1, -1, None, None, None,
                                       None, None)
    assert e.value.name == "BS_ERR_UNSUPPORTED"
    # work items: 2048 requests x 8 KV heads x 48 B = 768 KiB, plus the descriptors
    n = 2048
    reqs = np.zeros(n, bs.REQ_DTYPE)
    reqs["g"] = 32
    reqs["row"] = np.arange(n)
    kc = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    lay = [(kc, kc, kc, kc, kc, kc)]
    with pytest.raises(bs.BlockServeError, match="work items") as e:
        bs.bs_mixed_state_step_noalloc(ctx, reqs, 32, n, 32, lay, 8, 8, 128, bs.BS_BF16, 0.0, 1, 1000, bs.BS_BF16,
                                       None, 1000, None, 32, None, 32, 0.9, 1, -1, None, None, None, None, None)
    assert e.value.name == "BS_ERR_UNSUPPORTED"
