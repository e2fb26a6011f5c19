"""One mixed-state denoising step (Algorithm 1's ExecBlockCycle, one of its S
denoising steps, for one batch of requests at mixed block indices).

Order: (block-boundary KV compaction, when a plan is given) -> gather the
active blocks -> dual-cache block attention for every layer -> parallel decode
-> scatter the decoded tokens and mask back into the dense box. Each request's
result depends only on its own descriptor and data, so a request computed
alone equals the same request inside any batch.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

from .attention import dual_cache_block_attention
from .decode import parallel_decode
from .gather import gather_active_blocks, scatter_active_blocks


def mixed_state_step(reqs, L, tokens_dense, mask_dense, layers, logits, *, tau, q_min=1,
                     eos_id=-1, dtype="f32", scale=None):
    """``layers``: list of dicts with q, k_new, v_new, k_cache, v_cache.
    Returns dict with the new dense tokens/mask, per-layer attention outputs
    and updated caches, the decode results and the gathered positions."""
    tok_c, pos = gather_active_blocks(reqs, L, tokens_dense)
    msk_c, _ = gather_active_blocks(reqs, L, mask_dense)
    outs = []
    for lay in layers:
        o, kc, vc = dual_cache_block_attention(reqs, L, lay["q"], lay["k_new"], lay["v_new"],
                                               lay["k_cache"], lay["v_cache"], dtype=dtype,
                                               scale=scale, write_back=True)
        outs.append(dict(out=o, k_cache=kc, v_cache=vc))
    dec = parallel_decode(reqs, L, logits, tok_c, msk_c, tau=tau, q_min=q_min, eos_id=eos_id,
                          dtype=dtype)
    tokens2 = scatter_active_blocks(reqs, L, dec["tokens"], tokens_dense)
    mask2 = scatter_active_blocks(reqs, L, dec["masked"], mask_dense)
    return dict(tokens=tokens2, mask=mask2, layers=outs, decode=dec, pos=pos)
