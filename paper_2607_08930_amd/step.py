"""One mixed-state denoising step on the GPU, sequenced over the C ABI.

Order (Algorithm 1's block-cycle, one denoising step): gather the active
blocks' token ids and mask bits -> dual-cache block attention for each layer
(with the in-place fresh-KV write) -> parallel decode -> scatter tokens and
mask back into the dense box. ``run_step`` enqueues the whole step with one
``bs_mixed_state_step`` call (decode then reads and writes the dense boxes
directly) or, with ``fused=False``, as the separate K1/K2/K3/K1^-1 calls. At a
block boundary ``compact`` first rewrites the KV boxes of every layer.
PyTorch only provides device memory and the stream; every step runs in
libblockserve's kernels.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import (BS_BF16, BS_F32, Context, bs_decode_workspace_bytes, bs_dual_cache_block_attention,
               bs_step_workspace_bytes,
               bs_gather_active_blocks_n, bs_kv_scatter_compact, bs_mixed_state_step, bs_parallel_decode,
               bs_scatter_active_blocks_n)


def dt_code(dtype: str) -> int:
    return BS_BF16 if dtype == "bf16" else BS_F32


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def to_device(x: np.ndarray, dtype: str | None = None, device="cuda") -> torch.Tensor:
    """numpy -> device tensor; bf16 arrives as uint16 bit patterns."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def to_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@dataclass
class Layer:
    q: torch.Tensor        # [n][L][Hq][D]
    k_new: torch.Tensor    # [n][L][Hkv][D]
    v_new: torch.Tensor
    k_cache: torch.Tensor  # [R][Hkv][W][D]
    v_cache: torch.Tensor
    out: torch.Tensor      # [n][L][Hq][D]


@dataclass
class StepState:
    L: int
    Hq: int
    Hkv: int
    D: int
    V: int
    dtype: str
    R: int
    W: int
    tokens: torch.Tensor   # [R][W] int32 (dense box)
    mask: torch.Tensor     # [R][W] uint8
    layers: list
    logits: torch.Tensor   # [n_max][L][V]
    n_max: int
    tau: float = 0.9
    q_min: int = 1
    eos_id: int = -1
    write_back: bool = True
    scale: float = 0.0
    # compact block state and decode outputs (allocated by ``alloc``)
    tok_c: torch.Tensor = None
    msk_c: torch.Tensor = None
    pos: torch.Tensor = None
    n_unmasked: torch.Tensor = None
    done: torch.Tensor = None
    eos_seen: torch.Tensor = None
    conf: torch.Tensor = None
    dec_ws: torch.Tensor = None      # the step's workspace: the decode's, then the attention's partials
    ws_key: bytes = None             # descriptors dec_ws was last sized for
    flags_host: torch.Tensor = None
    extra: dict = field(default_factory=dict)

    def alloc(self):
        dev = self.tokens.device
        n, L = self.n_max, self.L
        self.tok_c = torch.empty((n, L), dtype=torch.int32, device=dev)
        self.msk_c = torch.empty((n, L), dtype=torch.uint8, device=dev)
        self.pos = torch.empty((n, L), dtype=torch.int32, device=dev)
        self.n_unmasked = torch.empty(n, dtype=torch.int32, device=dev)
        self.done = torch.empty(n, dtype=torch.uint8, device=dev)
        self.eos_seen = torch.empty(n, dtype=torch.uint8, device=dev)
        self.conf = torch.empty((n, L), dtype=torch.float32, device=dev)
        ws = bs_decode_workspace_bytes(n, L, self.V, dt_code(self.dtype))
        self.dec_ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)
        return self

    def workspace_for(self, reqs: np.ndarray) -> torch.Tensor:
        """The step workspace, grown to what the descriptors' split-KV plan
        needs (queried again only when the descriptors change)."""
        key = reqs.tobytes()
        if key != self.ws_key:
            dt = dt_code(self.dtype)
            need = bs_step_workspace_bytes(reqs, self.L, self.Hq, self.Hkv, self.D, dt, self.V, dt)
            if need > self.dec_ws.numel():
                self.dec_ws = torch.empty(need, dtype=torch.uint8, device=self.dec_ws.device)
            self.ws_key = key
        return self.dec_ws


def run_step(ctx: Context, st: StepState, reqs: np.ndarray, *, stream=None, want_conf=False,
             layers=None, fused=True, split=True) -> None:
    """Enqueue one step for the requests ``reqs`` (REQ_DTYPE, n <= n_max).

    fused: one library call; the compact tok_c/msk_c are then not written.
    pos is written either way. split: give the attention room for its
    split-KV plan (else only the decode's workspace: every row whole)."""
    L, R, W = st.L, st.R, st.W
    dt = dt_code(st.dtype)
    lays = st.layers if layers is None else layers
    conf = st.conf if want_conf else None
    ws = st.workspace_for(reqs)
    ws_bytes = ws.numel() if split else bs_decode_workspace_bytes(len(reqs), L, st.V, dt)
    if fused:
        bs_mixed_state_step(ctx, reqs, L, R, W,
                            [(x.q, x.k_new, x.v_new, x.k_cache, x.v_cache, x.out) for x in lays],
                            st.Hq, st.Hkv, st.D, dt, st.scale, st.write_back, st.V, dt, st.logits,
                            st.logits.stride(1), st.tokens, st.tokens.stride(0), st.mask, st.mask.stride(0),
                            st.tau, st.q_min, st.eos_id, st.n_unmasked, st.done, st.eos_seen, conf, st.pos,
                            ws, ws_bytes, stream=stream)
        return
    strides = [st.tokens.stride(0) * 4, st.mask.stride(0)]
    bs_gather_active_blocks_n(ctx, reqs, L, R, W, [st.tokens, st.mask], strides, [4, 1], [st.tok_c, st.msk_c],
                              st.pos, stream=stream)
    for lay in lays:
        bs_dual_cache_block_attention(ctx, reqs, L, st.Hq, st.Hkv, st.D, dt, st.scale, lay.q, lay.k_new,
                                      lay.v_new, lay.k_cache, lay.v_cache, R, W, st.write_back, lay.out,
                                      ws if split else None, ws_bytes if split else 0, stream=stream)
    bs_parallel_decode(ctx, reqs, L, st.V, dt, st.logits, st.logits.stride(1), st.tok_c, st.msk_c, st.tau,
                       st.q_min, st.eos_id, st.n_unmasked, st.done, st.eos_seen, conf, ws,
                       ws_bytes, stream=stream)
    bs_scatter_active_blocks_n(ctx, reqs, L, R, W, [st.tok_c, st.msk_c], [4, 1], [st.tokens, st.mask], strides,
                               stream=stream)


def compact(ctx: Context, segs: np.ndarray, n_layers: int, Hkv: int, D: int, dtype: str,
            src_k: torch.Tensor, src_v: torch.Tensor, stg_k: torch.Tensor, stg_v: torch.Tensor,
            dst_k: torch.Tensor, dst_v: torch.Tensor, stream=None) -> None:
    """KV boxes are [layers][R][Hkv][W][D] tensors; strides come from them."""
    eb = src_k.element_size()

    def layer_stride(t):
        # a unit layer axis may carry any stride (NumPy gives a new axis
        # stride 0); with one layer the box size is the stride that matters
        return t.stride(0) * eb if t.shape[0] > 1 else t[0].numel() * eb

    bs_kv_scatter_compact(ctx, segs, n_layers, Hkv, D, dt_code(dtype), src_k, src_v, layer_stride(src_k),
                          src_k.shape[1], src_k.shape[3], stg_k, stg_v,
                          layer_stride(stg_k) if stg_k is not None else 0,
                          stg_k.shape[1] if stg_k is not None else 1, stg_k.shape[3] if stg_k is not None else 1,
                          dst_k, dst_v, layer_stride(dst_k), dst_k.shape[1], dst_k.shape[3], stream=stream)


def prefix_only(reqs: np.ndarray, L: int) -> np.ndarray:
    """Descriptors for the prefix-cache layout (no masked suffix in the keys):
    each request attends over its prompt, its decoded blocks and its active
    block only, i.e. the Eq. 1 row width p + (k + 1) L (capped at p + g for a
    partial last block). The dense box keeps its layout: g is cut to
    min(g, (k + 1) L) and off is unchanged, so the same cells hold the same
    positions and the kernels never read the cells past the active block."""
    out = np.array(reqs, copy=True)
    out["g"] = np.minimum(out["g"], (out["k"].astype(np.int64) + 1) * L).astype(out["g"].dtype)
    return out
