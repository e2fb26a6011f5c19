"""Python binding of libblockserve.so, the MI355X (gfx950) mixed-state
denoising step of BlockServe (block-grained continuous batching for diffusion
LLMs).

Argument marshalling only: every entry point forwards to the C ABI declared in
``include/blockserve.h`` under the same name; all work happens in the HIP
kernels of the library. Tensors are passed as torch device tensors (or raw
integer device addresses); descriptor and segment arrays as numpy structured
arrays with the C struct layouts ``REQ_DTYPE`` / ``SEG_DTYPE``. A nonzero
status raises ``BlockServeError``. There is no CPU implementation: importing
this package fails when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "REQ_DTYPE", "SEG_DTYPE", "BS_F32", "BS_BF16", "BlockServeError", "Context", "lib", "LIB_PATH",
    "bs_create", "bs_destroy", "bs_status_string", "bs_last_error", "bs_validate_requests",
    "bs_validate_segments",
    "bs_gather_active_blocks", "bs_scatter_active_blocks", "bs_gather_active_blocks_n",
    "bs_scatter_active_blocks_n", "bs_mixed_state_step", "bs_mixed_state_step_noalloc", "bs_profile_begin", "bs_profile_end",
    "bs_sched_create", "bs_sched_destroy", "bs_sched_submit", "bs_sched_refill", "bs_sched_complete",
    "bs_sched_counts", "bs_sched_last_error", "Scheduler",
    "bs_attention_workspace_bytes", "bs_step_workspace_bytes", "bs_attention_work_list",
    "bs_dual_cache_block_attention", "bs_decode_workspace_bytes", "bs_parallel_decode",
    "bs_kv_scatter_compact", "bs_lm_head_workspace_bytes", "bs_lm_head_decode", "bs_lm_head_pack_bytes",
    "bs_lm_head_pack", "bs_dual_cache_refresh",
    "PROFILE_PHASES", "LM_PROFILE_PHASES", "REFRESH_PROFILE_PHASES",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libblockserve.so")

REQ_DTYPE = np.dtype([("p", "<i4"), ("g", "<i4"), ("k", "<i4"), ("row", "<i4"), ("off", "<i4")])
SEG_DTYPE = np.dtype([("src_kind", "<i4"), ("src_row", "<i4"), ("src_col", "<i4"),
                      ("dst_row", "<i4"), ("dst_col", "<i4"), ("len", "<i4")])
BS_F32, BS_BF16 = 0, 1
STATUS = {0: "BS_OK", 1: "BS_ERR_INVALID_ARG", 2: "BS_ERR_UNSUPPORTED", 3: "BS_ERR_DESCRIPTOR",
          4: "BS_ERR_OVERLAP", 5: "BS_ERR_WORKSPACE", 6: "BS_ERR_HIP"}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2607_08930_amd.build)")

# PyTorch-ROCm ships its own libamdhip64.so with the same soname as ROCm's.
# Loading torch first makes the dynamic linker bind this library to torch's
# HIP runtime, so torch's streams, events and allocations are the ones the
# kernels see; two runtimes in one process would not share them.
import torch  # noqa: E402,F401


def _hip_runtimes() -> set:
    found = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                p = line.split()[-1] if line.strip() else ""
                if "libamdhip64" in p:
                    found.add(os.path.realpath(p))
    except OSError:
        pass
    return found


lib = ctypes.CDLL(LIB_PATH)
if len(_hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are loaded in this process (" + ", ".join(sorted(_hip_runtimes()))
                      + "): import torch before loading libblockserve.so")

_vp, _i32, _i64, _f32, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_SIGS = {
    "bs_create": (_i32, [ctypes.POINTER(_vp), _i32]),
    "bs_destroy": (_i32, [_vp]),
    "bs_status_string": (ctypes.c_char_p, [_i32]),
    "bs_last_error": (ctypes.c_char_p, [_vp]),
    "bs_validate_requests": (_i32, [_vp, _i32, _i32, _i32, _i32]),
    "bs_validate_segments": (_i32, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32]),
    "bs_gather_active_blocks": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _i64, _i32, _vp, _vp, _vp]),
    "bs_scatter_active_blocks": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _i32, _vp, _i64, _vp]),
    "bs_gather_active_blocks_n": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "bs_scatter_active_blocks_n": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "bs_mixed_state_step": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _i32,
                                   _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _i64, _vp, _i64, _vp, _i64,
                                   _f32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "bs_mixed_state_step_noalloc": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _f32,
                                           _i32, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _i64, _vp, _i64,
                                           _vp, _i64, _f32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "bs_profile_begin": (_i32, [_vp, _i32]),
    "bs_profile_end": (_i32, [_vp, _vp, _i32, ctypes.POINTER(_i32)]),
    "bs_sched_create": (_i32, [ctypes.POINTER(_vp), _vp]),
    "bs_sched_destroy": (_i32, [_vp]),
    "bs_sched_submit": (_i32, [_vp, _vp, _i32]),
    "bs_sched_refill": (_i32, [_vp, _vp]),
    "bs_sched_complete": (_i32, [_vp, _vp, _i32, _vp, ctypes.POINTER(_i32)]),
    "bs_sched_counts": (_i32, [_vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32), ctypes.POINTER(_i64),
                               ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
    "bs_sched_last_error": (ctypes.c_char_p, []),
    "bs_attention_workspace_bytes": (_sz, [_vp, _i32, _i32, _i32, _i32, _i32, _i32]),
    "bs_dual_cache_block_attention": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _vp, _vp,
                                             _vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _sz, _vp]),
    "bs_decode_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "bs_step_workspace_bytes": (_sz, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32]),
    "bs_attention_work_list": (_i32, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _i32,
                                      ctypes.POINTER(_i32), ctypes.POINTER(_i32)]),
    "bs_parallel_decode": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _i64, _vp, _vp, _f32, _i32, _i32,
                                  _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "bs_lm_head_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "bs_lm_head_decode": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _f32, _i32, _i32,
                                 _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "bs_lm_head_pack_bytes": (_sz, [_i32, _i32]),
    "bs_lm_head_pack": (_i32, [_vp, _vp, _i64, _i32, _i32, _i32, _vp, _sz, _vp]),
    "bs_dual_cache_refresh": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _f32, _vp, _vp, _vp,
                                     _i32, _i32, _vp, _vp, _vp, _vp]),
    "bs_kv_scatter_compact": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _i64, _i32, _i32, _vp,
                                     _vp, _i64, _i32, _i32, _vp, _vp, _i64, _i32, _i32, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class BlockServeError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        super().__init__(f"{self.name}: {detail}")


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, Context):
        return x.handle
    raise TypeError(f"cannot pass {type(x)} as a pointer")


def _host(arr, dtype):
    a = np.ascontiguousarray(arr)
    if a.dtype != dtype:
        a = a.astype(dtype)
    return a


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st: int, ctx=None):
    if st != 0:
        detail = lib.bs_last_error(_ptr(ctx) if ctx is not None else None)
        raise BlockServeError(st, detail.decode() if detail else "")
    return st


class Context:
    """Owns a bs_ctx (upload ring for descriptors); close() or use as a context manager."""

    def __init__(self, device: int = 0):
        h = _vp()
        _check(lib.bs_create(ctypes.byref(h), device))
        self.handle = h.value
        self.device = device

    def close(self):
        if self.handle:
            lib.bs_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def bs_create(device: int = 0) -> Context:
    return Context(device)


def bs_destroy(ctx: Context) -> None:
    ctx.close()


def bs_status_string(status: int) -> str:
    return lib.bs_status_string(status).decode()


def bs_last_error(ctx: Context | None = None) -> str:
    return lib.bs_last_error(_ptr(ctx) if ctx is not None else None).decode()


def bs_validate_requests(reqs, L: int, R: int, W: int) -> None:
    r = _host(reqs, REQ_DTYPE)
    _check(lib.bs_validate_requests(_ptr(r), len(r), L, R, W))


def bs_validate_segments(segs, R_src: int, W_src: int, R_stg: int, W_stg: int, R_dst: int, W_dst: int,
                         src_is_dst: bool = False, stg_is_dst: bool = False) -> None:
    g = _host(segs, SEG_DTYPE)
    _check(lib.bs_validate_segments(_ptr(g) if len(g) else None, len(g), R_src, W_src, R_stg, W_stg, R_dst, W_dst,
                                    int(bool(src_is_dst)), int(bool(stg_is_dst))))


def bs_gather_active_blocks(ctx, reqs, L, R, W, src, src_row_stride_bytes, elem_bytes, dst, pos_out=None,
                            stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_gather_active_blocks(_ptr(ctx), _ptr(r), len(r), L, R, W, _ptr(src),
                                              src_row_stride_bytes, elem_bytes, _ptr(dst), _ptr(pos_out),
                                              _stream(stream)), ctx)


def bs_scatter_active_blocks(ctx, reqs, L, R, W, src_compact, elem_bytes, dst_dense, dst_row_stride_bytes,
                             stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_scatter_active_blocks(_ptr(ctx), _ptr(r), len(r), L, R, W, _ptr(src_compact),
                                               elem_bytes, _ptr(dst_dense), dst_row_stride_bytes,
                                               _stream(stream)), ctx)


def _tensor_arrays(ptrs, strides, elem_bytes):
    k = len(ptrs)
    if not (len(strides) == len(elem_bytes) == k):
        raise ValueError("pointer, stride and element-size lists differ in length")
    P = (_vp * max(k, 1))(*[_ptr(x) for x in ptrs])
    S = (_i64 * max(k, 1))(*strides)
    E = (_i32 * max(k, 1))(*elem_bytes)
    return P, S, E


def bs_gather_active_blocks_n(ctx, reqs, L, R, W, src, src_row_stride_bytes, elem_bytes, dst, pos_out=None,
                              stream=None):
    """``src``/``dst``/``src_row_stride_bytes``/``elem_bytes`` are equal-length lists."""
    r = _host(reqs, REQ_DTYPE)
    P, S, E = _tensor_arrays(src, src_row_stride_bytes, elem_bytes)
    D = (_vp * max(len(dst), 1))(*[_ptr(x) for x in dst])
    return _check(lib.bs_gather_active_blocks_n(_ptr(ctx), _ptr(r), len(r), L, R, W, len(src), P, S, E, D,
                                                _ptr(pos_out), _stream(stream)), ctx)


def bs_scatter_active_blocks_n(ctx, reqs, L, R, W, src_compact, elem_bytes, dst_dense, dst_row_stride_bytes,
                               stream=None):
    r = _host(reqs, REQ_DTYPE)
    P, S, E = _tensor_arrays(dst_dense, dst_row_stride_bytes, elem_bytes)
    C = (_vp * max(len(src_compact), 1))(*[_ptr(x) for x in src_compact])
    return _check(lib.bs_scatter_active_blocks_n(_ptr(ctx), _ptr(r), len(r), L, R, W, len(src_compact), C, E,
                                                 P, S, _stream(stream)), ctx)


def bs_attention_workspace_bytes(reqs, L, Hq, Hkv, D, dt) -> int:
    r = _host(reqs, REQ_DTYPE)
    return int(lib.bs_attention_workspace_bytes(_ptr(r), len(r), L, Hq, Hkv, D, dt))


def bs_dual_cache_block_attention(ctx, reqs, L, Hq, Hkv, D, dt, scale, q, k_new, v_new, k_cache, v_cache, R,
                                  W, write_back, out, ws=None, ws_bytes=0, stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_dual_cache_block_attention(
        _ptr(ctx), _ptr(r), len(r), L, Hq, Hkv, D, dt, float(scale), _ptr(q), _ptr(k_new), _ptr(v_new),
        _ptr(k_cache), _ptr(v_cache), R, W, int(write_back), _ptr(out), _ptr(ws), int(ws_bytes),
        _stream(stream)), ctx)


def bs_attention_work_list(reqs, L, Hq, Hkv, D, dt, split):
    """(items [N][6] int32: request, KV head, row block, t0, t1, partial slot;
    number of partial slots) of the bf16 attention's work list."""
    r = _host(reqs, REQ_DTYPE)
    n_items, n_parts = _i32(0), _i32(0)
    _check(lib.bs_attention_work_list(_ptr(r), len(r), L, Hq, Hkv, D, dt, int(split), None, 0,
                                      ctypes.byref(n_items), ctypes.byref(n_parts)))
    out = np.zeros((n_items.value, 6), np.int32)
    _check(lib.bs_attention_work_list(_ptr(r), len(r), L, Hq, Hkv, D, dt, int(split), _ptr(out), len(out),
                                      ctypes.byref(n_items), ctypes.byref(n_parts)))
    return out, n_parts.value


def bs_decode_workspace_bytes(n, L, V, dt) -> int:
    return int(lib.bs_decode_workspace_bytes(n, L, V, dt))


def bs_step_workspace_bytes(reqs, L, Hq, Hkv, D, dt, V, logits_dt) -> int:
    r = _host(reqs, REQ_DTYPE)
    return int(lib.bs_step_workspace_bytes(_ptr(r), len(r), L, Hq, Hkv, D, dt, V, logits_dt))


def bs_parallel_decode(ctx, reqs, L, V, logits_dt, logits, logits_row_stride, tokens, masked, tau, q_min,
                       eos_id, n_unmasked, done, eos_seen, conf_out=None, ws=None, ws_bytes=0, stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_parallel_decode(
        _ptr(ctx), _ptr(r), len(r), L, V, logits_dt, _ptr(logits), int(logits_row_stride), _ptr(tokens),
        _ptr(masked), float(tau), int(q_min), int(eos_id), _ptr(n_unmasked), _ptr(done), _ptr(eos_seen),
        _ptr(conf_out), _ptr(ws), int(ws_bytes), _stream(stream)), ctx)


def bs_lm_head_workspace_bytes(n, L, V) -> int:
    return int(lib.bs_lm_head_workspace_bytes(n, L, V))


def bs_lm_head_decode(ctx, reqs, L, d, V, dt, hidden, w_packed, tokens, masked, tau, q_min, eos_id,
                      n_unmasked, done, eos_seen, conf_out=None, ws=None, ws_bytes=0, stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_lm_head_decode(
        _ptr(ctx), _ptr(r), len(r), L, d, V, dt, _ptr(hidden), _ptr(w_packed), _ptr(tokens), _ptr(masked),
        float(tau), int(q_min), int(eos_id), _ptr(n_unmasked), _ptr(done), _ptr(eos_seen), _ptr(conf_out),
        _ptr(ws), int(ws_bytes), _stream(stream)), ctx)


def bs_lm_head_pack_bytes(V, d) -> int:
    return int(lib.bs_lm_head_pack_bytes(V, d))


def bs_lm_head_pack(ctx, w_vocab, w_row_stride, V, d, dt, w_packed, packed_bytes, stream=None):
    return _check(lib.bs_lm_head_pack(_ptr(ctx), _ptr(w_vocab), int(w_row_stride), V, d, dt, _ptr(w_packed),
                                      int(packed_bytes), _stream(stream)), ctx)


def bs_dual_cache_refresh(ctx, reqs, L, Hq, Hkv, D, dt, scale, rope_base, q, k, v, R, W, k_cache, v_cache,
                          out, stream=None):
    r = _host(reqs, REQ_DTYPE)
    return _check(lib.bs_dual_cache_refresh(
        _ptr(ctx), _ptr(r), len(r), L, Hq, Hkv, D, dt, float(scale), float(rope_base), _ptr(q), _ptr(k), _ptr(v),
        R, W, _ptr(k_cache), _ptr(v_cache), _ptr(out), _stream(stream)), ctx)


def bs_kv_scatter_compact(ctx, segs, n_layers, Hkv, D, dt, src_k, src_v, src_layer_stride, R_src, W_src,
                          stg_k, stg_v, stg_layer_stride, R_stg, W_stg, dst_k, dst_v, dst_layer_stride,
                          R_dst, W_dst, stream=None):
    s = _host(segs, SEG_DTYPE)
    return _check(lib.bs_kv_scatter_compact(
        _ptr(ctx), _ptr(s), len(s), n_layers, Hkv, D, dt, _ptr(src_k), _ptr(src_v), int(src_layer_stride),
        R_src, W_src, _ptr(stg_k), _ptr(stg_v), int(stg_layer_stride), R_stg, W_stg, _ptr(dst_k),
        _ptr(dst_v), int(dst_layer_stride), R_dst, W_dst, _stream(stream)), ctx)


def bs_mixed_state_step(ctx, reqs, L, R, W, layers, Hq, Hkv, D, dt, scale, write_back, V, logits_dt, logits,
                        logits_row_stride, tokens, tokens_row_stride, masked, masked_row_stride, tau, q_min, eos_id,
                        n_unmasked, done, eos_seen, conf_out, pos_out, ws, ws_bytes, stream=None):
    """``layers``: sequence of (q, k_new, v_new, k_cache, v_cache, out) per layer.

    Row strides of tokens/masked are in elements."""
    r = _host(reqs, REQ_DTYPE)
    nl = len(layers)
    arrs = [(_vp * max(nl, 1))(*[_ptr(lay[t]) for lay in layers]) for t in range(6)]
    return _check(lib.bs_mixed_state_step(_ptr(ctx), _ptr(r), len(r), L, R, W, nl, Hq, Hkv, D, dt, scale,
                                          int(write_back), *arrs, V, logits_dt, _ptr(logits), logits_row_stride,
                                          _ptr(tokens), tokens_row_stride, _ptr(masked), masked_row_stride, tau,
                                          q_min, eos_id, _ptr(n_unmasked), _ptr(done), _ptr(eos_seen),
                                          _ptr(conf_out), _ptr(pos_out), _ptr(ws), ws_bytes, _stream(stream)), ctx)


def bs_mixed_state_step_noalloc(ctx, reqs, L, R, W, layers, Hq, Hkv, D, dt, scale, write_back, V, logits_dt,
                                logits, logits_row_stride, tokens, tokens_row_stride, masked, masked_row_stride, tau,
                                q_min, eos_id, n_unmasked, done, eos_seen, conf_out, pos_out, stream=None):
    """bs_mixed_state_step without a workspace; allocates nothing."""
    r = _host(reqs, REQ_DTYPE)
    nl = len(layers)
    arrs = [(_vp * max(nl, 1))(*[_ptr(lay[t]) for lay in layers]) for t in range(6)]
    return _check(lib.bs_mixed_state_step_noalloc(_ptr(ctx), _ptr(r), len(r), L, R, W, nl, Hq, Hkv, D, dt, scale,
                                                  int(write_back), *arrs, V, logits_dt, _ptr(logits),
                                                  logits_row_stride, _ptr(tokens), tokens_row_stride, _ptr(masked),
                                                  masked_row_stride, tau, q_min, eos_id, _ptr(n_unmasked),
                                                  _ptr(done), _ptr(eos_seen), _ptr(conf_out), _ptr(pos_out),
                                                  _stream(stream)), ctx)


PROFILE_PHASES = ("attention", "decode_rows", "decode_select")          # bs_mixed_state_step
LM_PROFILE_PHASES = ("rows", "gemm", "merge_select")                      # bs_lm_head_decode
REFRESH_PROFILE_PHASES = ("rope_kv", "attention", "none")                 # bs_dual_cache_refresh


def bs_profile_begin(ctx, max_steps: int) -> None:
    _check(lib.bs_profile_begin(_ptr(ctx), max_steps), ctx)


def bs_profile_end(ctx, max_steps: int) -> np.ndarray:
    """Per-step phase durations in ms, shape [steps][len(PROFILE_PHASES)]."""
    out = np.zeros((max(max_steps, 1), len(PROFILE_PHASES)), np.float32)
    n = _i32(0)
    _check(lib.bs_profile_end(_ptr(ctx), out.ctypes.data, max_steps, ctypes.byref(n)), ctx)
    return out[:n.value].copy()


# ---------------------------------------------------------------- host scheduler
SCHED_BUDGET, SCHED_FIXED = 0, 1
ORDER_ASCENDING, ORDER_DESCENDING, ORDER_ARRIVAL = 0, 1, 2


class _SchedConfig(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("policy", ctypes.c_int32), ("budget", ctypes.c_int64),
                ("fixed_batch", ctypes.c_int32), ("rows", ctypes.c_int32), ("width", ctypes.c_int32),
                ("order", ctypes.c_int32)]


class _SchedPlan(ctypes.Structure):
    _fields_ = [("n_active", ctypes.c_int32), ("descs", _vp), ("ids", _vp), ("n_admitted", ctypes.c_int32),
                ("admitted_ids", _vp), ("segs", _vp), ("cost", ctypes.c_int64), ("box_width", ctypes.c_int32)]


SCHED_REQ_DTYPE = np.dtype([("id", np.int32), ("p", np.int32), ("g", np.int32)])


def _sched_check(st):
    if st != 0:
        raise BlockServeError(st, lib.bs_sched_last_error().decode())


def _view(ptr, n, dtype):
    if n == 0:
        return np.zeros(0, dtype)
    buf = (ctypes.c_char * (n * np.dtype(dtype).itemsize)).from_address(ptr)
    return np.frombuffer(buf, dtype=dtype).copy()


class Scheduler:
    """Host block-grained scheduler (bs_sched_*); see include/blockserve.h."""

    def __init__(self, L, *, policy=SCHED_BUDGET, budget=0, fixed_batch=0, rows=1, width=1,
                 order=ORDER_ASCENDING):
        cfg = _SchedConfig(L, policy, budget, fixed_batch, rows, width, order)
        h = _vp()
        _sched_check(lib.bs_sched_create(ctypes.byref(h), ctypes.byref(cfg)))
        self.handle = h.value
        self.L, self.rows, self.width = L, rows, width

    def close(self):
        if self.handle:
            lib.bs_sched_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def submit(self, reqs):
        """reqs: iterable of (id, p, g)."""
        a = np.array([tuple(int(x) for x in r) for r in reqs], dtype=SCHED_REQ_DTYPE)
        _sched_check(lib.bs_sched_submit(self.handle, a.ctypes.data if len(a) else None, len(a)))

    def refill(self) -> dict:
        plan = _SchedPlan()
        _sched_check(lib.bs_sched_refill(self.handle, ctypes.byref(plan)))
        return dict(descs=_view(plan.descs, plan.n_active, REQ_DTYPE),
                    ids=_view(plan.ids, plan.n_active, np.int32),
                    admitted=_view(plan.admitted_ids, plan.n_admitted, np.int32),
                    segs=_view(plan.segs, plan.n_admitted, SEG_DTYPE),
                    cost=int(plan.cost), box_width=int(plan.box_width))

    def complete(self, eos=None) -> np.ndarray:
        """eos: per-request flags in the last plan's row order (its length must
        equal the active count), or None for no EOS."""
        e = None if eos is None else np.ascontiguousarray(eos, dtype=np.uint8)
        n = self.counts()["active"] if e is None else len(e)
        out = np.zeros(max(n, 1), np.int32)
        ne = _i32(0)
        _sched_check(lib.bs_sched_complete(self.handle, e.ctypes.data if e is not None else None, n,
                                           out.ctypes.data, ctypes.byref(ne)))
        return out[:ne.value].copy()

    def counts(self) -> dict:
        a, b = _i32(0), _i32(0)
        c, d, e = _i64(0), _i64(0), _i64(0)
        _sched_check(lib.bs_sched_counts(self.handle, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                         ctypes.byref(d), ctypes.byref(e)))
        return dict(pending=a.value, active=b.value, finished=c.value, cycles=d.value, sum_active=e.value)


def bs_sched_create(L, **kw) -> Scheduler:
    return Scheduler(L, **kw)


def bs_sched_destroy(s: Scheduler) -> None:
    s.close()


def bs_sched_submit(s: Scheduler, reqs) -> None:
    s.submit(reqs)


def bs_sched_refill(s: Scheduler) -> dict:
    return s.refill()


def bs_sched_complete(s: Scheduler, eos=None) -> np.ndarray:
    return s.complete(eos)


def bs_sched_counts(s: Scheduler) -> dict:
    return s.counts()


def bs_sched_last_error() -> str:
    return lib.bs_sched_last_error().decode()
