"""Closed-loop serving on the GPU (native scheduler + K4 + fused steps) against
a CPU replay of the same stream by the oracle's scheduler and step functions:
identical admissions and evictions per block-cycle, identical step counts and
bit-identical generated tokens for every request. The serving logits keep
every confidence >= 0.018 away from the threshold and from the others, so no
decision of the stream sits on an exemption boundary."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import lazy, say
from oracle import schedule as osch

pytestmark = pytest.mark.gpu

L, HQ, HKV, D, V = 8, 2, 2, 64, 1008      # fp32 rows of 4032 bytes (a multiple of 16)
MASK_ID, EOS_ID, TAU = 0, 1, 0.9


def eos_blocks(stream):
    """Every fourth request emits EOS in its first block (ending it early when
    it has more than one block)."""
    return {rid: 0 for rid, _, _ in stream if rid % 4 == 1}


class HostProvider:
    """Model stand-in: seeded logits and prompts from synth, random q / fresh
    KV / prefilled KV on the device (they do not influence the tokens)."""

    def __init__(self, layers, eos_block):
        torch, _, _ = lazy()
        self.torch = torch
        self.layers, self.eos_block = layers, eos_block
        self.gen = torch.Generator(device="cuda")
        self.gen.manual_seed(7)

    def _randn(self, shape):
        return self.torch.randn(shape, generator=self.gen, device="cuda", dtype=self.torch.float32)

    def prefill(self, ids, p, g, W):
        n, ws = len(ids), int((p + g).max())
        sk = self._randn((self.layers, n, HKV, ws, D)); sv = self._randn((self.layers, n, HKV, ws, D))
        rows = [synth.serve_prompt_row(int(r), int(pp), int(gg), W, V, MASK_ID) for r, pp, gg in zip(ids, p, g)]
        return sk, sv, np.stack([r[0] for r in rows]), np.stack([r[1] for r in rows])

    def step(self, ids, descs, cycle, step):
        n = len(ids)
        layers = [(self._randn((n, L, HQ, D)), self._randn((n, L, HKV, D)), self._randn((n, L, HKV, D)))
                  for _ in range(self.layers)]
        logits = synth.serve_logits(ids, descs, step, V, L, EOS_ID, self.eos_block)
        return layers, self.torch.from_numpy(logits).cuda()


def replay(cfg, stream, eos_block):
    s = osch.Scheduler(L=L, policy=cfg["policy"], budget=cfg["budget"], fixed_batch=cfg["fixed_batch"],
                       rows=cfg["rows"], width=cfg["width"], order=cfg["order"])
    s.submit(stream)
    R, W = cfg["rows"], cfg["width"]
    tok = np.zeros((R, W), np.int32); msk = np.zeros((R, W), np.uint8)
    out, admitted, evicted, steps = {}, [], [], 0
    while True:
        adm = s.admit()
        act = s.active_sorted()
        if not act:
            break
        admitted.append(adm)
        for r in act:
            if r.id in adm:
                tok[r.row], msk[r.row] = synth.serve_prompt_row(r.id, r.p, r.g, W, V, MASK_ID)
        descs = np.zeros(len(act), synth.REQ_DTYPE)
        descs["p"] = [r.p for r in act]; descs["g"] = [r.g for r in act]; descs["k"] = [r.b for r in act]
        descs["row"] = [r.row for r in act]; descs["off"] = [W - r.p - r.g for r in act]
        ids = [r.id for r in act]
        eos_any = np.zeros(len(act), bool)
        for step in range(L):
            logits = synth.serve_logits(ids, descs, step, V, L, EOS_ID, eos_block)
            tok_c, _ = oracle.gather_active_blocks(descs, L, tok)
            msk_c, _ = oracle.gather_active_blocks(descs, L, msk)
            dec = oracle.parallel_decode(descs, L, logits, tok_c, msk_c, tau=TAU, q_min=1, eos_id=EOS_ID, dtype="f32")
            tok = oracle.scatter_active_blocks(descs, L, dec["tokens"], tok)
            msk = oracle.scatter_active_blocks(descs, L, dec["masked"], msk)
            steps += 1
            eos_any |= dec["eos_seen"].astype(bool)
            if dec["done"].all():
                break
        gone = s.complete_cycle([i for i, e in zip(ids, eos_any) if e])
        for rid in gone:
            d = descs[ids.index(rid)]
            start = int(d["off"] + d["p"])
            out[rid] = tok[int(d["row"]), start:start + int(d["g"])].copy()
        evicted.append(gone)
    return dict(outputs=out, admitted=admitted, evicted=evicted, steps=steps, counts=s.active_counts)


@pytest.mark.parametrize("policy,order", [(osch.BUDGET, osch.ASCENDING), (osch.BUDGET, osch.ARRIVAL),
                                          (osch.FIXED, osch.ASCENDING)])
def test_closed_loop_serving_matches_replay(policy, order):
    torch, bs, bstep = lazy()
    from paper_2607_08930_amd import serve
    stream = synth.serve_stream(18, L)
    eos_block = eos_blocks(stream)
    cfg = dict(policy=policy, budget=220, fixed_batch=4, rows=6, width=80, order=order)
    say(f"[serve policy={policy} order={order}] {len(stream)} requests")
    ref = replay(cfg, stream, eos_block)
    with bs.Context(0) as ctx:
        sc = serve.ServeConfig(L=L, layers=2, Hq=HQ, Hkv=HKV, D=D, V=V, dtype="f32", rows=cfg["rows"],
                               width=cfg["width"], policy=policy, budget=cfg["budget"],
                               fixed_batch=cfg["fixed_batch"], order=order, tau=TAU, q_min=1, eos_id=EOS_ID,
                               mask_id=MASK_ID)
        srv = serve.Server(ctx, sc, HostProvider(2, eos_block))
        res = srv.run(stream)
        torch.cuda.synchronize()
    assert res.admitted == ref["admitted"]
    assert res.evicted == ref["evicted"]
    assert res.active_counts == ref["counts"]
    assert res.steps == ref["steps"]
    assert sorted(res.outputs) == sorted(ref["outputs"]) == sorted(r for r, _, _ in stream)
    for rid, toks in ref["outputs"].items():
        np.testing.assert_array_equal(res.outputs[rid], toks, err_msg=f"request {rid}")
    # EOS requests with several blocks left early; the others ran all K blocks
    for rid, p, g in stream:
        K = -(-g // L)
        assert res.blocks[rid] == (1 if rid in eos_block else K)
    say(f"  cycles={res.cycles} steps={res.steps} R={sum(res.active_counts) / (res.cycles * cfg['rows']):.2f}")


class RefreshProvider(HostProvider):
    """bf16, D = 128 stand-in with the refresh hook: box projections of every
    block start drawn on the device (kept for inspection)."""

    def __init__(self, layers, eos_block, hq, hkv, d, rows, width):
        super().__init__(layers, eos_block)
        self.hq, self.hkv, self.d, self.rows, self.width = hq, hkv, d, rows, width
        self.last, self.last_descs = None, None

    def prefill(self, ids, p, g, W):
        n, ws = len(ids), int((p + g).max())
        bf = self.torch.bfloat16
        sk = self._randn((self.layers, n, self.hkv, ws, self.d)).to(bf)
        sv = self._randn((self.layers, n, self.hkv, ws, self.d)).to(bf)
        rows = [synth.serve_prompt_row(int(r), int(pp), int(gg), W, V, MASK_ID) for r, pp, gg in zip(ids, p, g)]
        return sk, sv, np.stack([r[0] for r in rows]), np.stack([r[1] for r in rows])

    def step(self, ids, descs, cycle, step):
        n, bf = len(ids), self.torch.bfloat16
        layers = [(self._randn((n, L, self.hq, self.d)).to(bf), self._randn((n, L, self.hkv, self.d)).to(bf),
                   self._randn((n, L, self.hkv, self.d)).to(bf)) for _ in range(self.layers)]
        logits = synth.serve_logits(ids, descs, step, V, L, EOS_ID, self.eos_block)
        return layers, self.torch.from_numpy(logits).cuda().to(bf)

    def refresh(self, ids, descs, cycle):
        self.last_descs = descs.copy()
        bf, s = self.torch.bfloat16, 1.0 / np.sqrt(self.d)
        R, W = self.rows, self.width
        self.last = [(self._randn((R, W, self.hq, self.d)).to(bf), (self._randn((R, W, self.hkv, self.d)) * s).to(bf),
                      (self._randn((R, W, self.hkv, self.d)) * s).to(bf)) for _ in range(self.layers)]
        return self.last


def test_serving_with_dual_cache_refresh():
    # the refresh at every block start rebuilds the cache and leaves the
    # decisions (driven by the logits) unchanged; after one cycle the cache
    # cells outside the active blocks hold the rotated projections
    torch, bs, bstep = lazy()
    from paper_2607_08930_amd import serve
    stream = synth.serve_stream(10, L)
    eos_block = eos_blocks(stream)
    rows, width, hq, hkv, d, base = 5, 80, 4, 2, 128, 1e4

    def run(refresh, max_cycles=1_000_000):
        with bs.Context(0) as ctx:
            sc = serve.ServeConfig(L=L, layers=1, Hq=hq, Hkv=hkv, D=d, V=V, dtype="bf16", rows=rows, width=width,
                                   policy=osch.BUDGET, budget=220, fixed_batch=4, order=osch.ASCENDING, tau=TAU,
                                   q_min=1, eos_id=EOS_ID, mask_id=MASK_ID, refresh=refresh, rope_base=base)
            prov = RefreshProvider(1, eos_block, hq, hkv, d, rows, width)
            srv = serve.Server(ctx, sc, prov)
            res = srv.run(stream, max_cycles=max_cycles)
            torch.cuda.synchronize()
            return res, srv, prov

    plain, _, _ = run(False)
    with_ref, _, _ = run(True)
    assert with_ref.refreshes == with_ref.cycles
    assert with_ref.admitted == plain.admitted and with_ref.evicted == plain.evicted
    assert with_ref.steps == plain.steps
    for rid, toks in plain.outputs.items():
        np.testing.assert_array_equal(with_ref.outputs[rid], toks, err_msg=f"request {rid}")
    # one cycle: cache cells outside the active blocks (which the steps'
    # write-through replaced) against the oracle's rotation of the projections
    res, srv, prov = run(True, max_cycles=1)
    kbox = oracle.widen(bstep.to_host(srv.k_box[0]), "bf16")
    vbox = bstep.to_host(srv.v_box[0])
    _, kp, vp = (bstep.to_host(t) for t in prov.last[0])
    descs = prov.last_descs
    assert len(descs) > 0
    for r in descs:
        row, off, p_, g_, k_ = (int(r[f]) for f in ("row", "off", "p", "g", "k"))
        ln = p_ + g_
        s0, b0 = p_ + k_ * L, min(L, g_ - k_ * L)
        keep = np.ones(ln, bool)
        keep[s0:s0 + b0] = False
        kr = oracle.rope(oracle.widen(kp[row, off:off + ln], "bf16"), np.arange(ln)[:, None], base)
        got = kbox[row, :, off:off + ln].transpose(1, 0, 2)
        x = oracle.widen(kp[row, off:off + ln], "bf16")
        pair = np.sqrt(x[..., :d // 2] ** 2 + x[..., d // 2:] ** 2)
        pair = np.concatenate([pair, pair], axis=-1)
        bound = 2.0 ** -8 * np.abs(kr) + (2.5e-7 * np.arange(ln)[:, None, None] + 2e-6) * pair + 1e-7
        assert (np.abs(got - kr) <= bound)[keep].all(), f"row {row}: cached keys"
        np.testing.assert_array_equal(vbox[row, :, off:off + ln].transpose(1, 0, 2)[keep],
                                      vp[row, off:off + ln][keep])
