"""Seeded synthetic workloads for the mixed-state denoising step.

Input construction only. This module draws request geometries, attention
tensors, logits, token/mask states and block-boundary churn plans from
counter-keyed PCG64 streams. It performs none of the step's own arithmetic
(no gathering, attention, softmax, decoding or compaction): the CPU oracle and
the HIP library both consume what it produces, and neither imports the other.

Conventions
-----------
* Every tensor is drawn from ``Generator(PCG64(SeedSequence([ROOT_SEED, cfg,
  variant, stream, *keys])))``; keys index the request/row/layer so any single
  row can be regenerated alone (the oracle checks sampled rows at full size).
* bf16 tensors are returned as their raw bit patterns (``uint16``): an fp32
  draw rounded to nearest-even. ``bf16_bits_to_f32`` widens them exactly.
* Request descriptors use ``REQ_DTYPE`` = five little-endian int32 fields
  ``(p, g, k, row, off)``, byte-identical to the C struct ``bs_req_desc``.
  Copy segments use ``SEG_DTYPE``, byte-identical to ``bs_copy_seg``.

The five workloads mirror the shapes the paper evaluates (LLaDA-8B and Dream-7B,
block length 32, Section "Experimental setup"); the skewed prompt mix of
workload 4 follows the long-tailed prompt statistics of the benchmark table.
Stand-ins only: no dataset item is reproduced.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
import math
import numpy as np

ROOT_SEED = 260708930

REQ_DTYPE = np.dtype([("p", "<i4"), ("g", "<i4"), ("k", "<i4"), ("row", "<i4"), ("off", "<i4")])
SEG_DTYPE = np.dtype([("src_kind", "<i4"), ("src_row", "<i4"), ("src_col", "<i4"),
                      ("dst_row", "<i4"), ("dst_col", "<i4"), ("len", "<i4")])

# stream ids
S_DESC, S_Q, S_KC, S_VC, S_KN, S_VN, S_LOGITS, S_MASK, S_TOK, S_CHURN, S_ADMIT, S_STAGE, S_PAD = range(13)

BF16_NAN = np.uint16(0x7FC0)


def rng(cfg: int, variant: int, stream: int, *keys: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [ROOT_SEED, int(cfg), int(variant), int(stream)] + [int(k) for k in keys])))


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round fp32 to bf16 (nearest-even) and return the 16-bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[np.isnan(x)] = BF16_NAN
    return r


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _span(p: int, g: int, k: int, L: int):
    """(block start, block length, row length) used only to place inputs."""
    s = p + k * L
    return s, min(L, g - k * L), p + g


@dataclass
class Workload:
    cfg: int
    name: str
    L: int
    Hq: int
    Hkv: int
    D: int
    V: int
    dtype: str            # "f32" or "bf16" for attention and logits
    tau: float
    q_min: int
    eos_id: int
    mask_id: int
    layers: int
    reqs: np.ndarray      # REQ_DTYPE
    R: int
    W: int
    q_sigma: float = 1.0
    kv_sigma: float = 1.0
    logits: str = "spiked"   # "normal" (sigma = logit_sigma) or "spiked"
    logit_sigma: float = 1.0
    variant: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return len(self.reqs)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def elem(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def spans(self):
        return [_span(int(r["p"]), int(r["g"]), int(r["k"]), self.L) for r in self.reqs]


def make_reqs(p, g, k, *, W=None, rows=None) -> tuple[np.ndarray, int, int]:
    """Left-padded dense layout: row i holds request i right-aligned (off = W - len)."""
    p = np.asarray(p, dtype=np.int64); g = np.asarray(g, dtype=np.int64); k = np.asarray(k, dtype=np.int64)
    n = len(p)
    lens = p + g
    if W is None:
        W = int(lens.max()) if n else 1
    reqs = np.zeros(n, dtype=REQ_DTYPE)
    reqs["p"] = p; reqs["g"] = g; reqs["k"] = k
    reqs["row"] = np.arange(n) if rows is None else rows
    reqs["off"] = W - lens
    R = int(reqs["row"].max()) + 1 if n else 1
    return reqs, R, int(W)


def workload(cfg: int, variant: int = 0, block_length: int | None = None, **over) -> Workload:
    """Build one of the five step workloads (1: tiny fp32, 2: LLaDA-8B-shaped,
    3: Dream-7B-shaped, 4: token-budgeted skewed Dream batch, 5: LLaDA-8B-shaped
    32-layer churn). ``variant`` re-seeds every tensor; ``over`` overrides fields.

    ``block_length`` (workloads 2-5, a divisor or multiple of 32 up to 64)
    re-blocks the same requests at another L: block index k becomes
    floor(32 k / L), so each request's active block starts at the same
    position or the nearest block boundary below it."""
    r = rng(cfg, variant, S_DESC)
    if cfg == 1:
        reqs, R, W = make_reqs([5, 12, 7, 20], [16, 24, 8, 32], [1, 0, 0, 3])
        w = Workload(1, "tiny-fp32-L8-mha2-d64", 8, 2, 2, 64, 1000, "f32", 0.9, 1, -1, 0, 1,
                     reqs, R, W, q_sigma=1.0, kv_sigma=1.0, logits="normal", logit_sigma=3.0)
    elif cfg == 2:
        n = 32
        p = r.integers(64, 512, size=n, endpoint=True)
        g = np.full(n, 256)
        k = r.integers(0, 7, size=n, endpoint=True)
        reqs, R, W = make_reqs(p, g, k)
        w = Workload(2, "llada8b-layer-n32-mha32-d128-L32", 32, 32, 32, 128, 126464, "bf16", 0.9, 1, -1, 0, 1,
                     reqs, R, W, kv_sigma=1 / math.sqrt(128))
    elif cfg == 3:
        n = 64
        p = r.integers(128, 1024, size=n, endpoint=True)
        g = np.full(n, 512)
        k = r.integers(0, 15, size=n, endpoint=True)
        reqs, R, W = make_reqs(p, g, k)
        w = Workload(3, "dream7b-layer-n64-gqa28x4-d128-L32", 32, 28, 4, 128, 152064, "bf16", 0.9, 1, -1, 0, 1,
                     reqs, R, W, kv_sigma=1 / math.sqrt(128))
    elif cfg == 4:
        budget = 131072
        ps, gs = [], []
        total = 0
        while True:
            long_ = r.random() < 0.2
            pp = int(r.integers(1024, 2048, endpoint=True)) if long_ else int(r.integers(32, 128, endpoint=True))
            gg = int((128, 256, 512)[r.integers(0, 3)])
            if total + pp + gg > budget:
                break
            total += pp + gg
            ps.append(pp); gs.append(gg)
        K = [-(-gg // 32) for gg in gs]
        k = [int(r.integers(0, KK)) for KK in K]
        reqs, R, W = make_reqs(ps, gs, k)
        w = Workload(4, "dream7b-skewed-budget131072-gqa28x4-d128-L32", 32, 28, 4, 128, 152064, "bf16",
                     0.9, 1, -1, 0, 1, reqs, R, W, kv_sigma=1 / math.sqrt(128), meta={"budget": budget})
    elif cfg == 5:
        n = 256
        p = r.integers(32, 256, size=n, endpoint=True)
        g = np.full(n, 128)
        k = r.integers(0, 3, size=n, endpoint=True)
        reqs, R, W = make_reqs(p, g, k, W=256 + 128)
        w = Workload(5, "llada8b-churn-n256-32layers-mha32-d128-L32", 32, 32, 32, 128, 126464, "bf16",
                     0.9, 1, -1, 0, 32, reqs, R, W, kv_sigma=1 / math.sqrt(128))
    else:
        raise ValueError(f"unknown workload {cfg}")
    w.variant = variant
    if block_length is not None and block_length != w.L:
        if cfg == 1 or block_length not in (8, 16, 64):
            raise ValueError(f"block_length {block_length} not offered for workload {cfg}")
        w.reqs = w.reqs.copy()
        w.reqs["k"] = (w.reqs["k"] * w.L) // block_length
        w.name = w.name.replace(f"-L{w.L}", f"-L{block_length}")
        w.L = block_length
    for kk, vv in over.items():
        setattr(w, kk, vv)
    return w


def straggler(case: int) -> Workload:
    """Batches with a few rows far longer than the rest, the straggler mix a
    heterogeneous serving batch can hold. Cases 0 and 1 are Dream-7B-shaped
    (28 query / 4 KV heads, D = 128, L = 32, g = 512, p ~ U[128, 1024)): 24
    requests with one prompt of 8000 tokens, and 64 requests with prompts of
    16000 and 6000 tokens. Case 2 is LLaDA-8B-shaped (32 MHA heads, D = 128,
    L = 32, g = 256, p ~ U[64, 512)): 32 requests with one prompt of 16000
    tokens."""
    r = rng(200 + case, 0, S_DESC)
    if case == 2:
        n, longs, lo, hi, g, Hq, Hkv, V, K = 32, {7: 16000}, 64, 512, 256, 32, 32, 126464, 8
        tag = "llada8b", "mha32"
    else:
        n, longs = ((24, {8: 8000}), (64, {5: 16000, 40: 6000}))[case]
        lo, hi, g, Hq, Hkv, V, K = 128, 1024, 512, 28, 4, 152064, 16
        tag = "dream7b", "gqa28x4"
    p = r.integers(lo, hi, n)
    for i, v in longs.items():
        p[i] = v
    k = r.integers(0, K, n)
    w = custom(32, Hq, Hkv, 128, V, "bf16", p.tolist(), [g] * n, k.tolist(), cfg=200 + case,
               kv_sigma=1.0 / np.sqrt(128.0))
    w.name = f"{tag[0]}-stragglers-n{n}-" + "-".join(str(v) for v in longs.values()) + f"-{tag[1]}-d128-L32"
    return w


def custom(L, Hq, Hkv, D, V, dtype, p, g, k, *, W=None, rows=None, R=None, cfg=100, variant=0,
           tau=0.9, q_min=1, eos_id=-1, layers=1, q_sigma=1.0, kv_sigma=1.0, logits="spiked",
           logit_sigma=1.0) -> Workload:
    """Arbitrary small workload (edge cases: partial blocks, empty suffix, gaps)."""
    reqs, R0, W0 = make_reqs(p, g, k, W=W, rows=rows)
    return Workload(cfg, "custom", L, Hq, Hkv, D, V, dtype, tau, q_min, eos_id, 0, layers, reqs,
                    R if R is not None else R0, W0, q_sigma=q_sigma, kv_sigma=kv_sigma,
                    logits=logits, logit_sigma=logit_sigma, variant=variant)


# ---------------------------------------------------------------- tensors
def _normal(g: np.random.Generator, shape, sigma: float) -> np.ndarray:
    return (g.standard_normal(shape, dtype=np.float32) * np.float32(sigma)).astype(np.float32)


def _cast(w: Workload, x: np.ndarray) -> np.ndarray:
    return x if w.dtype == "f32" else f32_to_bf16_bits(x)


def gen_q(w: Workload, layer: int = 0) -> np.ndarray:
    """Block queries [n][L][Hq][D] (rows j >= block length are zero)."""
    out = np.zeros((w.n, w.L, w.Hq, w.D), np.float32)
    for i in range(w.n):
        out[i] = _normal(rng(w.cfg, w.variant, S_Q, layer, i), (w.L, w.Hq, w.D), w.q_sigma)
    return _cast(w, out)


def gen_kv_new(w: Workload, layer: int = 0):
    """Fresh block keys/values [n][L][Hkv][D]."""
    k = np.zeros((w.n, w.L, w.Hkv, w.D), np.float32)
    v = np.zeros_like(k)
    for i in range(w.n):
        k[i] = _normal(rng(w.cfg, w.variant, S_KN, layer, i), (w.L, w.Hkv, w.D), w.kv_sigma)
        v[i] = _normal(rng(w.cfg, w.variant, S_VN, layer, i), (w.L, w.Hkv, w.D), w.kv_sigma)
    return _cast(w, k), _cast(w, v)


def gen_cache_row(w: Workload, layer: int, row: int):
    """One dense cache row [Hkv][W][D] for K and V (padding and the stale block
    slot are drawn too: they hold values the step must not use)."""
    kc = _normal(rng(w.cfg, w.variant, S_KC, layer, row), (w.Hkv, w.W, w.D), w.kv_sigma)
    vc = _normal(rng(w.cfg, w.variant, S_VC, layer, row), (w.Hkv, w.W, w.D), w.kv_sigma)
    return _cast(w, kc), _cast(w, vc)


def gen_cache(w: Workload, layer: int = 0):
    """Dense dual cache [R][Hkv][W][D] for K and V."""
    dt = np.float32 if w.dtype == "f32" else np.uint16
    kc = np.zeros((w.R, w.Hkv, w.W, w.D), dt)
    vc = np.zeros_like(kc)
    for row in range(w.R):
        kc[row], vc[row] = gen_cache_row(w, layer, row)
    return kc, vc


def poison_cache(w: Workload, kc: np.ndarray, vc: np.ndarray):
    """NaN in every padding column and in each request's stale block slot."""
    nanv = np.float32("nan") if w.dtype == "f32" else BF16_NAN
    used = np.zeros((w.R, w.W), bool)
    for r, (s, B, ln) in zip(w.reqs, w.spans()):
        row, off = int(r["row"]), int(r["off"])
        used[row, off:off + ln] = True
        kc[row, :, off + s:off + s + B] = nanv
        vc[row, :, off + s:off + s + B] = nanv
    for row in range(w.R):
        kc[row, :, ~used[row]] = nanv
        vc[row, :, ~used[row]] = nanv
    return kc, vc


def gen_state(w: Workload, p_mask: float = 0.5):
    """Dense token ids [R][W] int32 and mask bitmap [R][W] uint8.

    Prompt and completed blocks are unmasked random ids in [1, V); the active
    block is Bernoulli(p_mask) masked with at least one masked position; the
    suffix is masked. Masked cells hold ``mask_id``. Padding cells hold random
    garbage (ids and mask bits) that the step must never read.
    Returns (tokens, mask, block_masked[n][L] bool)."""
    gp = rng(w.cfg, w.variant, S_PAD)
    tokens = gp.integers(-2**31, 2**31 - 1, size=(w.R, w.W), dtype=np.int32)
    mask = gp.integers(0, 255, size=(w.R, w.W), dtype=np.uint8, endpoint=True)
    blk = np.zeros((w.n, w.L), bool)
    for i, (r, (s, B, ln)) in enumerate(zip(w.reqs, w.spans())):
        row, off = int(r["row"]), int(r["off"])
        g = rng(w.cfg, w.variant, S_MASK, i)
        m = g.random(B) < p_mask
        if not m.any():
            m[g.integers(0, B)] = True
        blk[i, :B] = m
        gt = rng(w.cfg, w.variant, S_TOK, i)
        toks = gt.integers(1, w.V, size=ln, dtype=np.int32)
        mk = np.zeros(ln, np.uint8)
        mk[s:s + B] = m
        mk[s + B:] = 1
        toks[mk.astype(bool)] = w.mask_id
        tokens[row, off:off + ln] = toks
        mask[row, off:off + ln] = mk
    return tokens, mask, blk


def gen_logits_row(w: Workload, i: int, j: int) -> np.ndarray:
    """Logits of block position (i, j), [V] (fp32 values or bf16 bits).

    "normal": N(0, logit_sigma^2). "spiked": N(0,1) plus one spiked id in
    [1, V) whose logit is bf16(LSE(other logits) + m), m ~ U[0, 8): the max
    softmax probability then sits at sigmoid(m), spread around 0.9."""
    g = rng(w.cfg, w.variant, S_LOGITS, i, j)
    if w.logits == "normal":
        x = _normal(g, w.V, w.logit_sigma)
        return _cast(w, x)
    x = f32_to_bf16_bits(g.standard_normal(w.V, dtype=np.float32)) if w.dtype == "bf16" \
        else g.standard_normal(w.V, dtype=np.float32)
    sid = int(g.integers(1, w.V))
    m = float(g.uniform(0.0, 8.0))
    xf = (bf16_bits_to_f32(x) if w.dtype == "bf16" else x).astype(np.float64)
    xf[sid] = -np.inf
    mx = xf.max()
    lse = mx + math.log(np.exp(xf - mx).sum())
    spike = np.float32(lse + m)
    if w.dtype == "bf16":
        x[sid] = f32_to_bf16_bits(np.array([spike]))[0]
    else:
        x[sid] = spike
    return x


def gen_logits(w: Workload, blk: np.ndarray) -> np.ndarray:
    """Logits [n][L][V]; rows that are not masked block positions are NaN
    (the decode must never read them)."""
    if w.dtype == "f32":
        out = np.full((w.n, w.L, w.V), np.nan, np.float32)
    else:
        out = np.full((w.n, w.L, w.V), BF16_NAN, np.uint16)
    for i in range(w.n):
        for j in range(w.L):
            if blk[i, j]:
                out[i, j] = gen_logits_row(w, i, j)
    return out


def spike_margin(w: Workload, i: int, j: int) -> tuple[int, float]:
    """The (spiked id, margin m) drawn for row (i, j) of a spiked workload."""
    g = rng(w.cfg, w.variant, S_LOGITS, i, j)
    g.standard_normal(w.V, dtype=np.float32)
    return int(g.integers(1, w.V)), float(g.uniform(0.0, 8.0))


# ---------------------------------------------------------------- churn (workload 5)
@dataclass
class ChurnPlan:
    reqs: np.ndarray          # descriptors after the block boundary
    segs: np.ndarray          # SEG_DTYPE copy plan (staging -> freed rows)
    rows: np.ndarray          # rows whose token/mask contents are rewritten
    tokens_rows: np.ndarray   # [len(rows)][W] int32
    mask_rows: np.ndarray     # [len(rows)][W] uint8
    stage_reqs: np.ndarray    # REQ_DTYPE of admitted requests inside the staging box
    n_complete: int
    n_finish: int
    n_last_block: int


def churn_plan(w: Workload, reqs: np.ndarray, tok_mirror: np.ndarray, mask_mirror: np.ndarray,
               step: int, frac_complete=0.5, frac_finish=0.5) -> ChurnPlan:
    """Seeded block-boundary churn (stable-slot plan).

    A seeded half of the requests completes its block: its block cells become
    unmasked seeded ids (overwriting whatever was decoded). Half of those (all completers on their last block
    first, then a seeded choice of the others) finish and are evicted; a new
    prompt (k = 0, fully masked generation) takes each freed row, right-aligned,
    its staged KV copied in from staging row a (staging is left-aligned at
    column 0). The other completers advance k by one. Survivors never move.
    ``tok_mirror``/``mask_mirror`` are host copies of the dense state for the
    rewritten rows (updated in place)."""
    n = len(reqs)
    g = rng(w.cfg, w.variant, S_CHURN, step)
    comp = np.sort(g.choice(n, size=int(n * frac_complete), replace=False))
    K = -(-reqs["g"] // w.L)
    last = [int(i) for i in comp if reqs["k"][i] == K[i] - 1]
    others = [int(i) for i in comp if reqs["k"][i] != K[i] - 1]
    n_fin = int(len(comp) * frac_finish)
    if len(last) >= n_fin:
        fin = last
    else:
        extra = g.choice(len(others), size=n_fin - len(last), replace=False)
        fin = sorted(last + [others[e] for e in extra])
    fin_set = set(fin)
    new = reqs.copy()
    ga = rng(w.cfg, w.variant, S_ADMIT, step)
    segs = []
    stage = np.zeros(len(fin), REQ_DTYPE)
    rows = []
    for i in comp:
        i = int(i)
        row = int(new["row"][i])
        if i in fin_set:
            continue
        s, B, ln = _span(int(new["p"][i]), int(new["g"][i]), int(new["k"][i]), w.L)
        off = int(new["off"][i])
        cells = slice(off + s, off + s + B)
        gt = rng(w.cfg, w.variant, S_TOK, 1000 + step, i)
        # the whole block is committed with seeded ids, so the host copy of
        # this row is authoritative whatever the device decoded in it
        tok_mirror[row, cells] = gt.integers(1, w.V, size=B, dtype=np.int32)
        mask_mirror[row, cells] = 0
        new["k"][i] += 1
        rows.append(row)
    for a, i in enumerate(fin):
        row = int(new["row"][i])
        p = int(ga.integers(32, 256, endpoint=True))
        gg = 128
        ln = p + gg
        new["p"][i] = p; new["g"][i] = gg; new["k"][i] = 0; new["off"][i] = w.W - ln
        stage[a] = (p, gg, 0, a, 0)
        segs.append((1, a, 0, row, w.W - ln, ln))
        gt = rng(w.cfg, w.variant, S_TOK, 2000 + step, a)
        toks = gt.integers(1, w.V, size=ln, dtype=np.int32)
        toks[p:] = w.mask_id
        mk = np.zeros(ln, np.uint8); mk[p:] = 1
        tok_mirror[row, :] = gt.integers(-2**31, 2**31 - 1, size=w.W, dtype=np.int32)
        mask_mirror[row, :] = gt.integers(0, 255, size=w.W, dtype=np.uint8, endpoint=True)
        tok_mirror[row, w.W - ln:] = toks
        mask_mirror[row, w.W - ln:] = mk
        rows.append(row)
    rows = np.array(sorted(set(rows)), np.int64)
    return ChurnPlan(new, np.array(segs, SEG_DTYPE).reshape(-1), rows,
                     tok_mirror[rows].copy(), mask_mirror[rows].copy(), stage,
                     len(comp), len(fin), len(last))


def gen_stage_row(w: Workload, layer: int, step: int, a: int, Wst: int):
    """Staged (prefilled) KV of admitted request a: [Hkv][Wst][D] for K and V."""
    ks = _normal(rng(w.cfg, w.variant, S_STAGE, step, layer, a, 0), (w.Hkv, Wst, w.D), w.kv_sigma)
    vs = _normal(rng(w.cfg, w.variant, S_STAGE, step, layer, a, 1), (w.Hkv, Wst, w.D), w.kv_sigma)
    return _cast(w, ks), _cast(w, vs)


# ---------------------------------------------------------------- closed-loop serving streams
S_SERVE_LOGITS, S_SERVE_PROMPT, S_SERVE_STREAM = 20, 21, 22

# Spike margins of the serving logits: sigmoid(m) of consecutive entries differ
# by >= 0.018 and none lies within 0.019 of 0.9, so every selection decision of
# the serving stream is far from the threshold and from ties.
SERVE_MARGINS = np.array([0.2, 0.65, 1.1, 1.55, 2.0, 2.45, 2.9, 3.35], np.float64)


def serve_stream(n: int, L: int, *, variant: int = 0, p_range=(4, 40), blocks=(1, 2, 3, 4)):
    """Seeded request stream [(id, p, g)] with prompt lengths spread over
    p_range and generation lengths of 1..4 blocks (some ending mid-block)."""
    g_ = rng(900, variant, S_SERVE_STREAM)
    out = []
    for i in range(n):
        p = int(g_.integers(p_range[0], p_range[1], endpoint=True))
        k = int(g_.choice(blocks))
        g = k * L - (int(g_.integers(0, L // 2)) if g_.random() < 0.3 else 0)
        out.append((i, p, g))
    return out


def serve_prompt_row(rid: int, p: int, g: int, W: int, V: int, mask_id: int, variant: int = 0):
    """Token and mask rows of an admitted request, right-aligned in a row of W
    columns: prompt ids in [2, V), generation positions masked."""
    g_ = rng(901, variant, S_SERVE_PROMPT, rid)
    tok = np.zeros(W, np.int32)
    msk = np.zeros(W, np.uint8)
    off = W - (p + g)
    tok[off:off + p] = g_.integers(2, V, size=p, dtype=np.int32)
    tok[off + p:] = mask_id
    msk[off + p:] = 1
    return tok, msk


def serve_logits(ids, descs, step: int, V: int, L: int, eos_id: int, eos_block: dict,
                 variant: int = 0) -> np.ndarray:
    """Logits [n][L][V] fp32 for one denoising step of the active requests
    (descriptor k = block index). Every position gets N(0,1) logits plus a
    spiked id (LSE of the others + a margin from SERVE_MARGINS, a permutation
    per request, block and step, so no two positions of a block tie). A request
    listed in eos_block spikes eos_id at position 0 of that block."""
    out = np.zeros((len(ids), L, V), np.float32)
    for i, (rid, d) in enumerate(zip(ids, descs)):
        b = int(d["k"])
        g_ = rng(902, variant, S_SERVE_LOGITS, int(rid), b, step)
        x = g_.standard_normal((L, V)).astype(np.float32)
        perm = g_.permutation(len(SERVE_MARGINS))
        sid = g_.integers(2, V, size=L)
        for j in range(L):
            if eos_block.get(int(rid), -1) == b and j == 0:
                sid[j] = eos_id
            row = x[j].astype(np.float64)
            row[sid[j]] = -np.inf
            mx = row.max()
            lse = mx + math.log(np.exp(row - mx).sum())
            x[j, sid[j]] = np.float32(lse + SERVE_MARGINS[perm[j % len(perm)]])
        out[i] = x
    return out


# Prompt and generated lengths shaped like the benchmark statistics table
# (LLaDA tokenizer): (prompt avg, prompt max, generation limit, actual avg,
# actual max). Only these summary numbers are used; no benchmark item is.
TABLE_STREAMS = {
    "humaneval-256": (157, 423, 256, 231, 255),
    "gsm8k-256": (1020, 1632, 256, 231, 260),
    "mbpp-512": (750, 4332, 512, 284, 512),
    "truthfulqa-512": (198, 245, 512, 33, 510),
}


def _shaped(g: np.random.Generator, n: int, avg: float, mx: int, lo: int, sigma: float) -> np.ndarray:
    """n integers in [lo, mx] with mean close to avg: a lognormal spread around
    avg, clipped, then rescaled once so the clipped mean matches."""
    x = np.exp(g.normal(0.0, sigma, n) - sigma * sigma / 2.0) * avg
    x = np.clip(x, lo, mx)
    x = np.clip(x * (avg / x.mean()), lo, mx)
    return np.rint(x).astype(np.int64)


def table_stream(name: str, n: int, variant: int = 0):
    """[(id, p, g)]: g is the generated length (the request ends there, as
    CheckEOS would end it), at most the generation limit."""
    pa, pm, limit, ga, gm = TABLE_STREAMS[name]
    g_ = rng(903, variant, S_SERVE_STREAM, sum(map(ord, name)))
    p = _shaped(g_, n, pa, pm, 8, 0.6)
    sig = 1.2 if ga < 0.3 * limit else 0.25
    gen = _shaped(g_, n, ga, min(gm, limit), 1, sig)
    return [(i, int(p[i]), int(gen[i])) for i in range(n)]


# ---------------------------------------------------------------- output head
S_LM_W, S_LM_H = 30, 31
# model widths of the workloads' shapes (LLaDA-8B: 4096, Dream-7B: 3584)
LM_HEAD_DIM = {1: 64, 2: 4096, 3: 3584, 4: 3584, 5: 4096}


def gen_lm_weight(w: Workload, d: int, V: int | None = None) -> np.ndarray:
    """Output-head matrix [V][d] as bf16 bits with N(0, 1/d) entries (the
    logits of a unit-variance hidden state are then about N(0, 1)); rows are
    drawn in chunks of 8192 from per-chunk streams."""
    V = w.V if V is None else V
    out = np.empty((V, d), np.uint16)
    for c0 in range(0, V, 8192):
        g = rng(w.cfg, w.variant, S_LM_W, c0 // 8192)
        n = min(8192, V - c0)
        out[c0:c0 + n] = f32_to_bf16_bits(g.standard_normal((n, d), dtype=np.float32) / np.float32(math.sqrt(d)))
    return out


def gen_lm_hidden(w: Workload, wv: np.ndarray) -> np.ndarray:
    """Final hidden states [n][L][d] as bf16 bits: unit noise plus a component
    along the head row of a random target token that lifts its logit to
    ln(V) + 1/2 + m, m ~ U[-2, 6), about m above the log-sum-exp of the other
    logits, so the max softmax probability spreads over roughly (0.1, 1)."""
    V, d = wv.shape
    out = np.zeros((w.n, w.L, d), np.uint16)
    for i in range(w.n):
        g = rng(w.cfg, w.variant, S_LM_H, i)
        h = g.standard_normal((w.L, d), dtype=np.float32).astype(np.float64)
        tgt = g.integers(1, V, size=w.L)
        m = g.uniform(-2.0, 6.0, size=w.L)
        for j in range(w.L):
            wt = bf16_bits_to_f32(wv[tgt[j]]).astype(np.float64)
            h[j] += (math.log(V) + 0.5 + m[j] - h[j] @ wt) / (wt @ wt) * wt
        out[i] = f32_to_bf16_bits(h.astype(np.float32))
    return out


# ---------------------------------------------------------------- dual-cache refresh
S_RQ, S_RK, S_RV = 32, 33, 34
# rotary bases of the workloads' model shapes (LLaDA-8B: 5e5, Dream-7B: 1e6)
ROPE_BASE = {1: 10000.0, 2: 500000.0, 3: 1000000.0, 4: 1000000.0, 5: 500000.0}


def gen_refresh_row(w: Workload, layer: int, row: int):
    """Projections of one dense row for the refresh forward, token-major:
    q [W][Hq][D], k and v [W][Hkv][D] (fp32 values or bf16 bits). Padding
    cells are drawn too; ``gen_refresh`` can poison them."""
    q = _normal(rng(w.cfg, w.variant, S_RQ, layer, row), (w.W, w.Hq, w.D), w.q_sigma)
    k = _normal(rng(w.cfg, w.variant, S_RK, layer, row), (w.W, w.Hkv, w.D), w.kv_sigma)
    v = _normal(rng(w.cfg, w.variant, S_RV, layer, row), (w.W, w.Hkv, w.D), w.kv_sigma)
    return _cast(w, q), _cast(w, k), _cast(w, v)


def gen_refresh(w: Workload, layer: int = 0, poison: bool = True):
    """Box projections q [R][W][Hq][D], k/v [R][W][Hkv][D]; with ``poison``
    every cell outside the requests' logical rows holds NaN."""
    dt = np.float32 if w.dtype == "f32" else np.uint16
    q = np.zeros((w.R, w.W, w.Hq, w.D), dt)
    k = np.zeros((w.R, w.W, w.Hkv, w.D), dt)
    v = np.zeros_like(k)
    for row in range(w.R):
        q[row], k[row], v[row] = gen_refresh_row(w, layer, row)
    if poison:
        nanv = np.float32("nan") if w.dtype == "f32" else BF16_NAN
        used = np.zeros((w.R, w.W), bool)
        for r in w.reqs:
            used[int(r["row"]), int(r["off"]):int(r["off"]) + int(r["p"]) + int(r["g"])] = True
        q[~used] = nanv
        k[~used] = nanv
        v[~used] = nanv
    return q, k, v
