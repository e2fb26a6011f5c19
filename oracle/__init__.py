"""CPU oracle for BlockServe's mixed-state denoising step (test infrastructure).

This package is a plain, slow, fp64 NumPy statement of what the step computes,
written from the paper (Zhu et al., "BlockServe: Block-Grained Continuous
Batching for High-Throughput Diffusion LLM Serving"). It exists only to check
the HIP library: only the tests, the package smoke check and the benchmark's
CPU-baseline leg may import it. It shares no code with the library and imports
nothing from it; it does not import the synthetic input generators either
(they hand it plain arrays).

Modules and the passages they follow
------------------------------------
geometry   block decomposition K_i = ceil(g_i / L) and block index
           (Section "Problem formulation"); bounding-box cost (Eq. 1, Section
           "Compute-aware admission control"); left-padded layout and position
           ids from a cumulative sum over the attention mask (Section "Mixed-state
           memory management", paragraph "Logical positional alignment");
           per-step transfer quota (paragraph "Vectorized mixed-schedule
           execution"); effective compute ratio R (Eq. 2).
gather     gather of each request's active block into a compact tensor and the
           inverse scatter (paragraph "Vectorized mixed-schedule execution").
schedule   block-grained scheduling (Algorithm 1) and compute-aware admission
           (Eq. 1, sand filling, Fixed variant, Section "Compute-aware
           admission control"); effective compute ratio (Eq. 2).
attention  block attention of the active block against the request's dual
           cache (cached prefix + fresh block + cached masked suffix), with the
           in-place write of the fresh block KV at its physical offsets
           (paragraph "Vectorized mixed-schedule execution"; dual cache from the
           Fast-dLLM integration described in Sections "Experimental setup" and
           "Diffusion LLM Inference Optimization").
decode     confidence-aware parallel decoding with greedy (temperature 0)
           predictions and a per-step minimum quota (paragraph "Vectorized
           mixed-schedule execution"; "Implementation details").
lm_head    the same decoding step with its logits produced by the output head
           from the positions' hidden states (logits never stored).
refresh    the full-row attention of the dual-cache refresh at a block start
           (and the prefill of newly admitted rows), with rotary embedding at
           the explicit position ids of paragraph "Logical positional
           alignment"; the refreshed cache holds the rotated keys.
compact    KV scatter/compaction when requests are evicted and admitted at a
           block boundary (Algorithm 1; Eq. 1 discussion of the bounding box
           shrinking without explicit reclamation).
step       one mixed-state step composed of the above.

Numerics: every floating-point computation is fp64. bf16 inputs arrive as raw
16-bit patterns and are widened exactly. Every function is pinned by tests
under ``tests/`` against values fixed by the paper or by mathematics
(hand-enumerated geometry, closed forms, brute force, a textbook attention
special case, invariants).
"""
from .geometry import (geometry, validate_reqs, bbox_cost, position_ids, transfer_schedule,
                       effective_compute_ratio, widen)
from .gather import gather_active_blocks, scatter_active_blocks
from .attention import dual_cache_block_attention, attention_rows
from .decode import parallel_decode, row_stats
from .lm_head import lm_head_logits, lm_head_decode
from .refresh import rope, row_positions, refresh_row, dual_cache_refresh
from .compact import kv_scatter_compact
from .step import mixed_state_step
from . import schedule

__all__ = [
    "schedule",
    "geometry", "validate_reqs", "bbox_cost", "position_ids", "transfer_schedule",
    "effective_compute_ratio", "widen", "gather_active_blocks", "scatter_active_blocks",
    "dual_cache_block_attention", "attention_rows", "parallel_decode", "row_stats",
    "lm_head_logits", "lm_head_decode", "rope", "row_positions", "refresh_row",
    "dual_cache_refresh",
    "kv_scatter_compact", "mixed_state_step",
]
