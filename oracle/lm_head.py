"""LM head fused with confidence-aware parallel decoding (reference).

Passages followed: paragraph "Vectorized mixed-schedule execution" and the
Fast-dLLM parallel decoding the paper integrates ("Implementation details":
greedy decoding): the model's output head turns the final hidden state of
each masked block position into one logit per vocabulary entry, and the
decoding rule of ``oracle.decode`` picks tokens from those logits.

Readings where the paper is silent:
* the logit of vocabulary entry v at a position with hidden state h is the
  inner product <h, w_v> of h with row v of the output-head matrix (no bias;
  a model with a bias or a final normalisation applies it before this call);
* logits are the exact inner products of the stored (bf16) inputs, computed
  here in fp64; they are never rounded to a storage precision;
* only masked positions of an active block are projected: the hidden states
  of other positions are never read.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import numpy as np

from .decode import parallel_decode
from .geometry import geometry, widen


def lm_head_logits(hidden_rows, w_vocab, dtype: str, chunk: int = 4096) -> np.ndarray:
    """fp64 logits [r][V] = hidden_rows [r][d] times w_vocab [V][d] transposed,
    one vocabulary chunk at a time (a library matmul per chunk)."""
    h = widen(hidden_rows, dtype)
    V = w_vocab.shape[0]
    out = np.empty((h.shape[0], V), np.float64)
    for v0 in range(0, V, chunk):
        out[:, v0:v0 + chunk] = h @ widen(w_vocab[v0:v0 + chunk], dtype).T
    return out


class _Rows:
    """logits[i, j] for the projected positions only."""

    def __init__(self, rows):
        self.rows = rows

    def __getitem__(self, ij):
        return self.rows[ij]


def lm_head_decode(reqs, L: int, hidden, w_vocab, tokens, masked, *, tau: float, q_min: int = 1,
                   eos_id: int = -1, dtype: str = "bf16", only=None):
    """One decoding step whose logits come from the output head.

    hidden [n][L][d] (rows of masked positions j < B_i are read, others
    never), w_vocab [V][d], tokens [n][L] int32 and masked [n][L] uint8 (the
    gathered block state). Returns what ``parallel_decode`` returns."""
    todo = range(len(reqs)) if only is None else only
    keys = [(i, j) for i in todo for j in range(geometry(reqs[i], L).B) if masked[i][j]]
    rows = {}
    if keys:
        lg = lm_head_logits(np.stack([hidden[i][j] for i, j in keys]), w_vocab, dtype)
        rows = {key: lg[a] for a, key in enumerate(keys)}
    return parallel_decode(reqs, L, _Rows(rows), tokens, masked, tau=tau, q_min=q_min, eos_id=eos_id,
                           dtype="f64", only=only)
