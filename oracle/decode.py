"""Confidence-aware parallel decoding of the active blocks.

Passages followed: paragraph "Vectorized mixed-schedule execution" (a per-step
transfer quota, the block's masked tokens spread uniformly over the S steps,
block-agnostic because every block starts fully masked); the confidence-aware
parallel decoding of Fast-dLLM that the paper integrates unchanged (Section
"Diffusion LLM Inference Optimization": high-confidence tokens are unmasked
selectively); greedy decoding at temperature 0 ("Implementation details").

Readings where the paper is silent or leaves the rule to Fast-dLLM:
* prediction x_j = argmax over the whole vocabulary, ties to the smallest id;
* confidence c_j = the softmax probability of x_j at temperature 1, i.e.
  1 / sum_v exp(l_v - l_max);
* a masked position qualifies when c_j >= tau;
* the number unmasked is n = min(|M|, max(q, #{c_j >= tau})): with q = 1 this
  is "every qualifying position, else the single most confident one", and
  with tau > 1 it is a fixed per-step quota of q;
* the n chosen positions are the n most confident, ties to the smallest j;
* the mask state is an explicit bitmap, so a predicted mask id is still an
  ordinary token; unmasked positions never change (no re-masking);
* eos_seen: some unmasked position of the block holds eos_id after the step.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import numpy as np

from .geometry import geometry, widen


def row_stats(logits_row, dtype: str):
    """(argmax with ties to the smallest id, max softmax probability) in fp64."""
    x = widen(logits_row, dtype)
    mx = x.max()
    # np.argmax returns the first maximal index; the pin tests check this
    # tie rule against an explicit scan.
    a = int(np.argmax(x))
    c = 1.0 / np.exp(x - mx).sum()
    return a, float(c)


def parallel_decode(reqs, L: int, logits, tokens, masked, *, tau: float, q_min: int = 1,
                    eos_id: int = -1, dtype: str = "f32", only=None):
    """One decoding step on the compact active blocks.

    logits [n][L][V] (rows of masked positions are read, others never);
    tokens [n][L] int32 and masked [n][L] uint8 are the gathered block state.
    Returns dict with tokens', masked', n_unmasked [n] int32, done [n] uint8,
    eos_seen [n] uint8, conf [n][L] fp64 (-1 where not computed), pred [n][L]
    int (-1 where not computed)."""
    n = len(reqs)
    tok = np.array(tokens, dtype=np.int32, copy=True)
    msk = np.array(masked, dtype=np.uint8, copy=True)
    n_un = np.zeros(n, np.int32)
    done = np.zeros(n, np.uint8)
    eos = np.zeros(n, np.uint8)
    conf = np.full((n, L), -1.0)
    pred = np.full((n, L), -1, np.int64)
    todo = range(n) if only is None else only
    for i in todo:
        t = geometry(reqs[i], L)
        M = [j for j in range(t.B) if msk[i, j]]
        for j in M:
            pred[i, j], conf[i, j] = row_stats(logits[i, j], dtype)
        n_sel = min(len(M), max(int(q_min), sum(1 for j in M if conf[i, j] >= tau)))
        ranked = sorted(M, key=lambda j: (-conf[i, j], j))
        U = ranked[:n_sel]
        for j in U:
            tok[i, j] = pred[i, j]
            msk[i, j] = 0
        n_un[i] = n_sel
        done[i] = 1 if n_sel == len(M) else 0
        eos[i] = 1 if (eos_id >= 0 and any(msk[i, j] == 0 and tok[i, j] == eos_id
                                           for j in range(t.B))) else 0
    return dict(tokens=tok, masked=msk, n_unmasked=n_un, done=done, eos_seen=eos,
                conf=conf, pred=pred)
