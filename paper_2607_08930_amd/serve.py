"""Closed-loop block-grained serving on one GPU (Algorithm 1 around the step).

Each iteration is one block-cycle:
1. the native scheduler refills the active set at the block boundary
   (compute-aware admission, Eq. 1) and returns the new descriptors;
2. admitted requests' prefilled KV rows are copied from a staging box into
   their rows of the dense KV box (K4, stable slots) and their token / mask
   rows are written;
3. with `refresh` on, the dual cache is rebuilt first: for every layer the
   provider's projections of the whole box go through the refresh entry
   point (rotary embedding at the rows' position ids, keys and values into
   the cache, full-row attention), which also prefills the admitted rows;
4. denoising steps run on the fused step entry point until every active
   request's block is fully unmasked (at most L steps, since every step
   unmasks at least one masked position of each block);
5. the scheduler advances every request by one block and evicts those that
   reached K_i blocks or reported EOS during the cycle; their rows are read
   back as the requests' outputs.

What a model would produce (queries, fresh block KV and logits at each step,
prefilled KV and prompt tokens at admission) comes from a provider object:

    provider.prefill(ids, p, g, W) -> (stg_k, stg_v, tok_rows, mask_rows)
        stg_k / stg_v: [layers][n][Hkv][Ws][D] device tensors (row a holds
        admitted request a's p + g positions from column 0); tok_rows [n][W]
        int32 and mask_rows [n][W] uint8 host arrays, right-aligned rows.
    provider.step(ids, descs, cycle, step) -> (layers, logits)
        layers: per layer (q, k_new, v_new) device tensors [n][L][H][D];
        logits: [n][L][V] device tensor (row stride a multiple of 16 bytes).
    provider.refresh(ids, descs, cycle) -> layers       (with `refresh` on)
        per layer (q, k, v) device tensors [R][W][H][D]: the projections of
        the whole box at the block start (bf16, D = 128).

PyTorch only supplies device memory and the stream; every step runs in the
library's kernels, and every scheduling decision in its native scheduler.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import (SCHED_BUDGET, Context, Scheduler, bs_decode_workspace_bytes, bs_dual_cache_refresh,
               bs_step_workspace_bytes,
               bs_kv_scatter_compact, bs_mixed_state_step)
from .step import dt_code, torch_dtype


@dataclass
class ServeConfig:
    L: int
    layers: int
    Hq: int
    Hkv: int
    D: int
    V: int
    dtype: str               # "bf16" or "f32" for attention and logits
    rows: int                # R: rows of the dense box
    width: int               # W: columns of the dense box
    policy: int = SCHED_BUDGET
    budget: int = 0
    fixed_batch: int = 0
    order: int = 0
    tau: float = 0.9
    q_min: int = 1
    eos_id: int = -1
    mask_id: int = 0
    refresh: bool = False    # rebuild the dual cache at every block start (bf16, D = 128)
    rope_base: float = 0.0   # rotary base of the refresh (<= 0: no rotation)


@dataclass
class ServeResult:
    outputs: dict = field(default_factory=dict)     # id -> generated token ids [g]
    blocks: dict = field(default_factory=dict)      # id -> block-cycles spent active
    cycles: int = 0
    steps: int = 0
    refreshes: int = 0                              # refresh calls (one per layer and cycle)
    active_counts: list = field(default_factory=list)
    admitted: list = field(default_factory=list)    # per cycle
    evicted: list = field(default_factory=list)     # per cycle


class Server:
    def __init__(self, ctx: Context, cfg: ServeConfig, provider, device="cuda"):
        self.ctx, self.cfg, self.provider = ctx, cfg, provider
        self.sched = Scheduler(cfg.L, policy=cfg.policy, budget=cfg.budget, fixed_batch=cfg.fixed_batch,
                               rows=cfg.rows, width=cfg.width, order=cfg.order)
        R, W = cfg.rows, cfg.width
        self.tokens = torch.zeros((R, W), dtype=torch.int32, device=device)
        self.mask = torch.zeros((R, W), dtype=torch.uint8, device=device)
        td = torch_dtype(cfg.dtype)
        self.k_box = torch.zeros((cfg.layers, R, cfg.Hkv, W, cfg.D), dtype=td, device=device)
        self.v_box = torch.zeros_like(self.k_box)
        self.out = [torch.empty((R, cfg.L, cfg.Hq, cfg.D), dtype=td, device=device) for _ in range(cfg.layers)]
        self.n_unmasked = torch.empty(R, dtype=torch.int32, device=device)
        # done and eos_seen side by side, so one small copy into pinned host
        # memory brings both back after every step
        self.flags = torch.zeros((2, R), dtype=torch.uint8, device=device)
        self.flags_host = torch.zeros((2, R), dtype=torch.uint8, pin_memory=True)
        self.done, self.eos_seen = self.flags[0], self.flags[1]
        self.ws = torch.empty(max(bs_decode_workspace_bytes(R, cfg.L, cfg.V, dt_code(cfg.dtype)), 16),
                              dtype=torch.uint8, device=device)
        self.info = {}      # id -> (p, g)
        if cfg.refresh:
            if cfg.dtype != "bf16" or cfg.D != 128:
                raise ValueError("the dual-cache refresh runs in bf16 with D = 128")
            self.ref_out = torch.empty((R, W, cfg.Hq, cfg.D), dtype=td, device=device)

    def _admit(self, plan):
        ids = plan["admitted"]
        if len(ids) == 0:
            return
        p = np.array([self.info[int(i)][0] for i in ids]); g = np.array([self.info[int(i)][1] for i in ids])
        stg_k, stg_v, tok_rows, mask_rows = self.provider.prefill(ids, p, g, self.cfg.width)
        cfg = self.cfg
        eb = stg_k.element_size()

        def lstride(t):
            return t.stride(0) * eb if t.shape[0] > 1 else t[0].numel() * eb

        bs_kv_scatter_compact(self.ctx, plan["segs"], cfg.layers, cfg.Hkv, cfg.D, dt_code(cfg.dtype), None, None, 0,
                              1, 1, stg_k, stg_v, lstride(stg_k), stg_k.shape[1], stg_k.shape[3], self.k_box,
                              self.v_box, lstride(self.k_box), cfg.rows, cfg.width)
        rows = torch.as_tensor(plan["segs"]["dst_row"].astype(np.int64), device=self.tokens.device)
        self.tokens[rows] = torch.from_numpy(np.ascontiguousarray(tok_rows, dtype=np.int32)).to(self.tokens.device)
        self.mask[rows] = torch.from_numpy(np.ascontiguousarray(mask_rows, dtype=np.uint8)).to(self.mask.device)

    def _collect(self, descs, ids, evicted, res):
        if len(evicted) == 0:
            return
        host_tok = self.tokens.cpu().numpy()
        for rid in evicted:
            i = int(np.nonzero(ids == rid)[0][0])
            d = descs[i]
            start = int(d["off"] + d["p"])
            res.outputs[int(rid)] = host_tok[int(d["row"]), start:start + int(d["g"])].copy()

    def run(self, requests, max_cycles=1_000_000) -> ServeResult:
        """requests: iterable of (id, p, g). Serves them to completion."""
        reqs = [(int(a), int(b), int(c)) for a, b, c in requests]
        for rid, p, g in reqs:
            self.info[rid] = (p, g)
        self.sched.submit(reqs)
        cfg = self.cfg
        res = ServeResult()
        dt = dt_code(cfg.dtype)
        while res.cycles < max_cycles:
            plan = self.sched.refill()
            descs, ids = plan["descs"], plan["ids"]
            n = len(ids)
            if n == 0:
                break
            self._admit(plan)
            if cfg.refresh:
                for l, (q, k, v) in enumerate(self.provider.refresh(ids, descs, res.cycles)):
                    bs_dual_cache_refresh(self.ctx, descs, cfg.L, cfg.Hq, cfg.Hkv, cfg.D, dt, 0.0, cfg.rope_base,
                                          q, k, v, cfg.rows, cfg.width, self.k_box[l], self.v_box[l], self.ref_out)
                    res.refreshes += 1
            res.admitted.append(plan["admitted"].tolist())
            res.active_counts.append(n)
            eos_any = np.zeros(n, np.uint8)
            # the cycle's descriptors are fixed: size the workspace for their
            # split-KV plan once
            need = bs_step_workspace_bytes(descs, cfg.L, cfg.Hq, cfg.Hkv, cfg.D, dt, cfg.V, dt)
            if need > self.ws.numel():
                self.ws = torch.empty(need, dtype=torch.uint8, device=self.ws.device)
            for step in range(cfg.L):
                layers, logits = self.provider.step(ids, descs, res.cycles, step)
                lay = [(q, kn, vn, self.k_box[l], self.v_box[l], self.out[l][:n])
                       for l, (q, kn, vn) in enumerate(layers)]
                bs_mixed_state_step(self.ctx, descs, cfg.L, cfg.rows, cfg.width, lay, cfg.Hq, cfg.Hkv, cfg.D, dt,
                                    0.0, 1, cfg.V, dt, logits, logits.stride(1), self.tokens, self.tokens.stride(0),
                                    self.mask, self.mask.stride(0), cfg.tau, cfg.q_min, cfg.eos_id,
                                    self.n_unmasked, self.done, self.eos_seen, None, None, self.ws,
                                    self.ws.numel())
                res.steps += 1
                self.flags_host.copy_(self.flags, non_blocking=True)
                torch.cuda.current_stream().synchronize()
                flags = self.flags_host.numpy()
                eos_any |= flags[1, :n]
                if flags[0, :n].all():
                    break
            evicted = self.sched.complete(eos_any)
            for rid in ids:
                res.blocks[int(rid)] = res.blocks.get(int(rid), 0) + 1
            self._collect(descs, ids, evicted, res)
            res.evicted.append(evicted.tolist())
            res.cycles += 1
        return res
