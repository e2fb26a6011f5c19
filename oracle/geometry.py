"""Request geometry, layout and the host-side closed forms.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


def widen(x, dtype: str) -> np.ndarray:
    """Exact fp64 value of an fp32 array, or of bf16 raw bit patterns (uint16);
    an fp64 array ("f64": logits computed here, never stored) as it is."""
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    if dtype == "bf16":
        b = np.asarray(x, dtype=np.uint16)
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


@dataclass(frozen=True)
class Geo:
    p: int      # prompt length p_i
    g: int      # generation length g_i
    k: int      # current block index (b_i in the paper)
    row: int    # physical row of the dense box
    off: int    # physical column of logical position 0
    K: int      # number of blocks ceil(g / L)
    s: int      # first logical position of the active block
    B: int      # active block length (L except for a partial last block)
    e: int      # one past the active block
    len: int    # logical row length p + g (prompt, generation incl. masked suffix)


def geometry(req, L: int) -> Geo:
    """Section "Problem formulation": the generation of g_i tokens is split into
    K_i = ceil(g_i / L) blocks of L tokens and the request sits at block index
    k in {0, ..., K_i - 1}. Block k covers generated tokens [kL, (k+1)L), i.e.
    logical positions [p + kL, p + kL + L) after the p prompt tokens; the last
    block is shorter when L does not divide g_i (the ceiling)."""
    p, g, k, row, off = (int(req["p"]), int(req["g"]), int(req["k"]), int(req["row"]), int(req["off"]))
    K = math.ceil(g / L)
    s = p + k * L
    B = min(L, g - k * L)
    return Geo(p, g, k, row, off, K, s, B, s + B, p + g)


class DescriptorError(ValueError):
    pass


def validate_reqs(reqs, L: int, R: int, W: int) -> None:
    """Reject descriptors the step cannot serve: L < 1, p < 0, g < 1, k outside
    [0, K), a row outside [0, R), a row shared by two requests, off < 0, or a
    logical row that does not fit the W columns of the dense box."""
    if L < 1:
        raise DescriptorError("L < 1")
    seen = set()
    for r in reqs:
        p, g, k, row, off = (int(r["p"]), int(r["g"]), int(r["k"]), int(r["row"]), int(r["off"]))
        if p < 0 or g < 1:
            raise DescriptorError("p < 0 or g < 1")
        if not (0 <= k < math.ceil(g / L)):
            raise DescriptorError("block index outside [0, K)")
        if not (0 <= row < R):
            raise DescriptorError("row outside the box")
        if row in seen:
            raise DescriptorError("duplicate row")
        seen.add(row)
        if off < 0 or off + p + g > W:
            raise DescriptorError("row does not fit the box")


def bbox_cost(reqs, L: int) -> int:
    """Eq. 1: |A| * max_i (p_i + (b_i + 1) L), the bounding box the admission
    controller budgets (prompt plus completed and current blocks)."""
    if len(reqs) == 0:
        return 0
    return len(reqs) * max(int(r["p"]) + (int(r["k"]) + 1) * L for r in reqs)


def position_ids(attn_mask_row) -> np.ndarray:
    """Paragraph "Logical positional alignment": explicit position ids as a
    cumulative index over the attention (non-padding) mask, so that the first
    non-padding token is at position 0. Padding cells get -1."""
    m = np.asarray(attn_mask_row, dtype=np.int64)
    pos = np.cumsum(m) - 1
    return np.where(m > 0, pos, -1)


def transfer_schedule(n_masked: int, S: int) -> list[int]:
    """Per-step transfer quota: the block's masked tokens distributed uniformly
    over the S denoising steps (paragraph "Vectorized mixed-schedule
    execution"). Uniform integer split: floor(n/S) each, the remainder given to
    the earliest steps."""
    base, rem = divmod(int(n_masked), int(S))
    return [base + (1 if t < rem else 0) for t in range(S)]


def effective_compute_ratio(active_counts, B: int) -> float:
    """Eq. 2: R = (1 / (T B)) * sum_t a_t over the T block-cycles."""
    a = list(active_counts)
    return sum(a) / (len(a) * B)
