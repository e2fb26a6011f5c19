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
                  kc=None, vc=None, scale=0.0, split=True):
    """Returns (out, k_cache', v_cache', inputs) as host arrays. split: pass
    the workspace the descriptors' split-KV plan asks for (else none, so
    every row runs whole)."""
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
    dt = bstep.dt_code(w.dtype)
    nws = bs.bs_attention_workspace_bytes(reqs, w.L, w.Hq, w.Hkv, w.D, dt) if split else 0
    # garbage, not zeros: the partial slots need no initialisation
    ws = torch.full((nws,), 0xA5, dtype=torch.uint8, device="cuda") if nws else None
    bs.bs_dual_cache_block_attention(ctx, reqs, w.L, w.Hq, w.Hkv, w.D, dt, scale, dq, dkn,
                                     dvn, dkc, dvc, w.R, w.W, write_back, out, ws, nws)
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


class DecodeStats:
    """Counts of one decode comparison: masked positions compared, positions
    exempt because a confidence lies within EXEMPT of tau or of a
    neighbour at the selection boundary (the band), positions whose argmax
    is not fixed by the arithmetic (near ties, output head only), and
    requests whose selection count the band leaves open."""

    def __init__(self):
        self.positions = 0
        self.band = 0
        self.near_tie = 0
        self.open_requests = 0

    def add(self, o):
        for k in ("positions", "band", "near_tie", "open_requests"):
            setattr(self, k, getattr(self, k) + getattr(o, k))
        return self

    def __repr__(self):
        return (f"{self.positions} masked positions, {self.band} in the threshold/tie band, "
                f"{self.near_tie} near argmax ties, {self.open_requests} requests with an open count")


def selection_bands(conf_row, M, tau, q_min, eps=EXEMPT):
    """Per masked position j of one request: 'sel' when the decision rule
    selects j for every set of confidences within eps of conf_row, 'not' when
    it never does, 'band' otherwise; and the bounds (n_lo, n_hi) of the
    selection count over that set.

    The rule selects the n = min(|M|, max(q, #{c >= tau})) most confident
    positions (ties to the smaller j). Moving every confidence by at most eps
    keeps n in [n_lo, n_hi] (counts at tau + eps and tau - eps); at most
    #{k != j : c_k >= c_j - eps} positions can then rank ahead of j and at
    least #{k != j : c_k > c_j + eps} do."""
    c = np.array([conf_row[j] for j in M], np.float64)
    nm = len(M)
    n_lo = min(nm, max(q_min, int((c >= tau + eps).sum())))
    n_hi = min(nm, max(q_min, int((c >= tau - eps).sum())))
    status = {}
    for a, j in enumerate(M):
        others = np.delete(c, a)
        ahead_max = int((others >= c[a] - eps).sum())
        ahead_min = int((others > c[a] + eps).sum())
        status[j] = "sel" if ahead_max < n_lo else ("not" if ahead_min >= n_hi else "band")
    return status, n_lo, n_hi


def check_request_decode(label, i, B, tok_in, msk_in, got_tok, got_msk, got_conf, got_n, got_done, got_eos,
                         ref_conf, ref_pred, tau, q_min, eos_id, conf_tol, alt_ids=None):
    """One request's decode against the oracle, position by position.

    * confidences: computed exactly where the oracle computes them, within
      conf_tol; -1 elsewhere;
    * a position the rule decides the same way for every confidence within
      EXEMPT of the oracle's ('sel' / 'not') must be unmasked with the
      oracle's argmax, or left masked with its token unchanged; a 'band'
      position may do either (counted);
    * near argmax ties (alt_ids[j]: every id whose logit is within the tie
      gap of the largest) may take any of those ids (counted);
    * the GPU's own result must obey the rule on the GPU's own confidences:
      n = min(|M|, max(q, #{c >= tau})) positions, the n most confident
      (ties to the smaller j); and n_unmasked, done, eos_seen must describe
      its own tokens and mask;
    * positions outside M are untouched.
    Returns DecodeStats."""
    st = DecodeStats()
    alt_ids = alt_ids or {}
    M = [j for j in range(B) if msk_in[j]]
    assert CONF_TOL <= conf_tol < EXEMPT / 2, "the band argument needs conf_tol well below EXEMPT"
    for j in range(len(got_conf)):
        if j in M:
            assert ref_conf[j] >= 0, f"{label}: oracle lacks confidence at ({i},{j})"
            assert abs(float(got_conf[j]) - ref_conf[j]) <= conf_tol, \
                f"{label}: confidence error {abs(float(got_conf[j]) - ref_conf[j]):.2e} at ({i},{j})"
        else:
            assert got_conf[j] == -1, f"{label}: conf_out not -1 at unmasked ({i},{j})"
    for j in range(B, len(tok_in)):
        assert got_tok[j] == tok_in[j] and got_msk[j] == msk_in[j], f"{label}: cell past the block changed ({i},{j})"
    for j in range(B):
        if j not in M:
            assert got_tok[j] == tok_in[j] and got_msk[j] == msk_in[j], f"{label}: unmasked cell changed ({i},{j})"
    if not M:
        assert got_n == 0 and got_done == 1, f"{label}: empty request {i} not a no-op"
    else:
        status, n_lo, n_hi = selection_bands(ref_conf, M, tau, q_min)
        st.positions = len(M)
        st.open_requests = int(n_lo != n_hi)
        for j in M:
            ok_ids = alt_ids.get(j, {int(ref_pred[j])})
            if len(ok_ids) > 1:
                st.near_tie += 1
            if got_msk[j] == 0:
                assert int(got_tok[j]) in ok_ids, \
                    f"{label}: ({i},{j}) unmasked with {int(got_tok[j])}, oracle argmax {int(ref_pred[j])}"
                assert status[j] != "not", f"{label}: ({i},{j}) unmasked, the rule never selects it"
            else:
                assert got_msk[j] == 1 and got_tok[j] == tok_in[j], f"{label}: ({i},{j}) masked cell changed"
                assert status[j] != "sel", f"{label}: ({i},{j}) left masked, the rule always selects it"
            st.band += status[j] == "band"
        # the GPU's decision obeys the rule on its own confidences
        g = np.array([float(got_conf[j]) for j in M], np.float32)
        n_gpu = min(len(M), max(q_min, int((g >= np.float32(tau)).sum())))
        order = sorted(range(len(M)), key=lambda a: (-g[a], M[a]))
        chosen = {M[a] for a in order[:n_gpu]}
        unmasked = {j for j in M if got_msk[j] == 0}
        assert unmasked == chosen, f"{label}: request {i} selected {sorted(unmasked)}, its own rule {sorted(chosen)}"
        assert got_n == n_gpu and n_lo <= n_gpu <= n_hi, f"{label}: request {i} n_unmasked {got_n} ({n_lo}..{n_hi})"
        assert got_done == int(n_gpu == len(M)), f"{label}: request {i} done flag"
    eos = eos_id >= 0 and any(got_msk[j] == 0 and got_tok[j] == eos_id for j in range(B))
    assert got_eos == int(eos), f"{label}: request {i} eos_seen"
    return st


def check_decode(w, got, ref, reqs=None, tau=None, label="", q_min=None, conf_tol=CONF_TOL, alt_ids=None,
                 tok_in=None, msk_in=None, eos_id=None):
    """Compact-state decode results against the oracle's, per position (see
    check_request_decode). tok_in / msk_in: the compact state before the call
    (default: recovered from the oracle's result and its selections).
    alt_ids: {(i, j): ids} near argmax ties. Returns DecodeStats."""
    reqs = w.reqs if reqs is None else reqs
    tau = w.tau if tau is None else tau
    q_min = w.q_min if q_min is None else q_min
    eos_id = w.eos_id if eos_id is None else eos_id
    if msk_in is None:
        msk_in = (ref["masked"].astype(bool) | (ref["conf"] >= 0)).astype(np.uint8)
    if tok_in is None:
        raise ValueError("check_decode needs the input tokens")
    stats = DecodeStats()
    for i, r in enumerate(reqs):
        B = oracle.geometry(r, w.L).B
        alt = {j: ids for (ii, j), ids in (alt_ids or {}).items() if ii == i}
        stats.add(check_request_decode(label, i, B, tok_in[i], msk_in[i], got["tokens"][i], got["masked"][i],
                                       got["conf"][i], int(got["n_unmasked"][i]), int(got["done"][i]),
                                       int(got["eos_seen"][i]), ref["conf"][i], ref["pred"][i], tau, q_min,
                                       eos_id, conf_tol, alt))
    return stats


def check_step_decode(w, reqs, got, dec, tok_in, msk_in, label, only=None):
    """The fused step's decode, per position, on the dense boxes: each
    request's block cells are gathered from the result and from the input
    state and compared with the oracle's decode (check_request_decode)."""
    gtok, _ = oracle.gather_active_blocks(reqs, w.L, got["tokens"])
    gmsk, _ = oracle.gather_active_blocks(reqs, w.L, got["mask"])
    itok, _ = oracle.gather_active_blocks(reqs, w.L, tok_in)
    imsk, _ = oracle.gather_active_blocks(reqs, w.L, msk_in)
    stats = DecodeStats()
    for i in (range(len(reqs)) if only is None else only):
        B = oracle.geometry(reqs[i], w.L).B
        stats.add(check_request_decode(label, i, B, itok[i], imsk[i], gtok[i], gmsk[i], got["conf"][i],
                                       int(got["n_unmasked"][i]), int(got["done"][i]), int(got["eos_seen"][i]),
                                       dec["conf"][i], dec["pred"][i], w.tau, w.q_min, w.eos_id, 2e-5))
    return stats
