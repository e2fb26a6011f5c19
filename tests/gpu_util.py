"""Helpers shared by the GPU parity tests: run one entry point of the HIP
library on synthetic inputs and bring the results back to the host, plus the
comparison rules (exemption band for threshold decisions, attention
tolerances)."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
import synth

ATT_TOL = {"f32": 1e-5, "bf16": 1e-2}   # max abs error (fp32 / bf16 inputs, fp32 accumulation)
ATT_REL = 1e-2                           # bf16: max|d| / max|O_ref|
EXEMPT = 1e-3                            # |c - tau| or top-2 gap that exempts a decision
CONF_TOL = 2e-5                          # fp32 confidence vs fp64


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def lazy():
    import torch
    import paper_2607_08930_amd as bs
    from paper_2607_08930_amd import step as bstep
    return torch, bs, bstep


def widen_out(x, dtype):
    return oracle.widen(x, dtype)


def run_attention(ctx, w, layer=0, *, poison=False, write_back=True, reqs=None, q=None, kn=None, vn=None,
                  kc=None, vc=None, scale=0.0):
    """Returns (out, k_cache', v_cache', inputs) as host arrays."""
    torch, bs, bstep = lazy()
    reqs = w.reqs if reqs is None else reqs
    q = synth.gen_q(w, layer) if q is None else q
    if kn is None:
        kn, vn = synth.gen_kv_new(w, layer)
    if kc is None:
        kc, vc = synth.gen_cache(w, layer)
        if poison:
            kc, vc = synth.poison_cache(w, kc, vc)
    dq = bstep.to_device(q, w.dtype)
    dkn, dvn = bstep.to_device(kn, w.dtype), bstep.to_device(vn, w.dtype)
    dkc, dvc = bstep.to_device(kc, w.dtype), bstep.to_device(vc, w.dtype)
    out = torch.full(dq.shape, float("nan"), dtype=dq.dtype, device="cuda")
    bs.bs_dual_cache_block_attention(ctx, reqs, w.L, w.Hq, w.Hkv, w.D, bstep.dt_code(w.dtype), scale, dq, dkn,
                                     dvn, dkc, dvc, w.R, w.W, write_back, out)
    torch.cuda.synchronize()
    return (bstep.to_host(out), bstep.to_host(dkc), bstep.to_host(dvc),
            dict(q=q, k_new=kn, v_new=vn, k_cache=kc, v_cache=vc))


def check_attention(w, got, ref, reqs=None, label=""):
    """Element-wise: max abs error within ATT_TOL (and the relative bound for
    bf16); rows beyond each block must be exactly zero."""
    reqs = w.reqs if reqs is None else reqs
    g = widen_out(got, w.dtype)
    err = 0.0
    mx = 0.0
    for i, r in enumerate(reqs):
        t = oracle.geometry(r, w.L)
        d = np.abs(g[i, :t.B] - ref[i, :t.B])
        assert np.isfinite(g[i, :t.B]).all(), f"{label}: non-finite output in request {i}"
        err = max(err, float(d.max()))
        mx = max(mx, float(np.abs(ref[i, :t.B]).max()))
        assert (g[i, t.B:] == 0).all(), f"{label}: rows beyond the block not zero (request {i})"
    assert err <= ATT_TOL[w.dtype], f"{label}: max abs error {err:.3e} > {ATT_TOL[w.dtype]}"
    if w.dtype == "bf16":
        assert err / mx <= ATT_REL, f"{label}: relative error {err / mx:.3e} > {ATT_REL}"
    return err, mx


def run_decode(ctx, w, logits, tok_c, msk_c, *, tau=None, q_min=None, eos_id=None, reqs=None, dev_logits=None,
               ws=None):
    torch, bs, bstep = lazy()
    reqs = w.reqs if reqs is None else reqs
    n = len(reqs)
    tau = w.tau if tau is None else tau
    q_min = w.q_min if q_min is None else q_min
    eos_id = w.eos_id if eos_id is None else eos_id
    if dev_logits is None:
        # rows padded to a 16-byte multiple (the ABI requires it); the pad
        # holds NaN, so reading past V would show up in the results
        eb = 2 if w.dtype == "bf16" else 4
        vpad = -(-w.V * eb // 16) * 16 // eb
        if vpad != w.V:
            nanv = np.uint16(0x7FC0) if w.dtype == "bf16" else np.float32("nan")
            lp = np.full(logits.shape[:2] + (vpad,), nanv, dtype=logits.dtype)
            lp[:, :, :w.V] = logits
            logits = lp
        dl = bstep.to_device(logits, w.dtype)
    else:
        dl = dev_logits
    dt = bstep.to_device(tok_c)
    dm = bstep.to_device(msk_c)
    nun = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    done = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    eos = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    conf = torch.full((n, w.L), float("nan"), dtype=torch.float32, device="cuda")
    wsb = bs.bs_decode_workspace_bytes(n, w.L, w.V, bstep.dt_code(w.dtype))
    ws = torch.full((max(wsb, 16),), 0xAB, dtype=torch.uint8, device="cuda") if ws is None else ws
    bs.bs_parallel_decode(ctx, reqs, w.L, w.V, bstep.dt_code(w.dtype), dl, dl.stride(1), dt, dm, tau, q_min,
                          eos_id, nun, done, eos, conf, ws, wsb)
    torch.cuda.synchronize()
    return dict(tokens=dt.cpu().numpy(), masked=dm.cpu().numpy(), n_unmasked=nun.cpu().numpy(),
                done=done.cpu().numpy(), eos_seen=eos.cpu().numpy(), conf=conf.cpu().numpy(), ws=ws)


def exempt_requests(ref, reqs, L, tau, q_min=1):
    """Requests whose selection is not fixed at fp32 precision: the number
    selected changes when every confidence within EXEMPT of tau moves by
    EXEMPT either way, or the last selected and first unselected confidences
    are within EXEMPT of each other. (A confidence near tau that cannot change
    the count -- e.g. when the quota q_min decides it -- exempts nothing.)"""
    ex = set()
    for i, r in enumerate(reqs):
        t = oracle.geometry(r, L)
        cs = sorted((ref["conf"][i, j] for j in range(t.B) if ref["conf"][i, j] >= 0), reverse=True)
        if not cs:
            continue
        nm = len(cs)
        n_lo = min(nm, max(q_min, sum(c >= tau + EXEMPT for c in cs)))
        n_hi = min(nm, max(q_min, sum(c >= tau - EXEMPT for c in cs)))
        nsel = int(ref["n_unmasked"][i])
        if n_lo != n_hi:
            ex.add(i)
        elif 0 < nsel < nm and cs[nsel - 1] - cs[nsel] <= EXEMPT:
            ex.add(i)
    return ex


def check_decode(w, got, ref, reqs=None, tau=None, label="", q_min=None, conf_tol=CONF_TOL, also_exempt=()):
    reqs = w.reqs if reqs is None else reqs
    tau = w.tau if tau is None else tau
    ex = exempt_requests(ref, reqs, w.L, tau, w.q_min if q_min is None else q_min) | set(also_exempt)
    for i, r in enumerate(reqs):
        t = oracle.geometry(r, w.L)
        m = ref["conf"][i] >= 0
        assert np.array_equal(got["conf"][i] >= 0, m), f"{label}: conf_out mask differs (request {i})"
        if m.any():
            dc = np.abs(got["conf"][i][m] - ref["conf"][i][m]).max()
            assert dc <= conf_tol, f"{label}: confidence error {dc:.2e} (request {i})"
        assert (got["conf"][i][~m] == -1).all()
        if i in ex:
            continue
        assert np.array_equal(got["tokens"][i], ref["tokens"][i]), f"{label}: tokens differ (request {i})"
        assert np.array_equal(got["masked"][i], ref["masked"][i]), f"{label}: mask differs (request {i})"
        for key in ("n_unmasked", "done", "eos_seen"):
            assert got[key][i] == ref[key][i], f"{label}: {key} differs (request {i})"
    return len(ex)
