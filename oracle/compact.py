"""KV scatter/compaction at a block boundary.

Passages followed: Algorithm 1 (requests that reach their last block or emit
EOS are removed at the block boundary and new requests are admitted into the
active set); Eq. 1 and its discussion (the dense bounding box shrinks when the
widest request leaves, without explicit memory reclamation); paragraph
"Logical positional alignment" (each request occupies a contiguous, left-padded
run of its row); paragraph "Vectorized mixed-schedule execution" (the frozen
prefix cache is preserved across batch reconfigurations).

The operation is a list of copy segments. Segment (src_kind, src_row, src_col,
dst_row, dst_col, len) copies, for every layer l and KV head h, the ``len``
cached positions src[l][src_row][h][src_col : src_col + len] to
dst[l][dst_row][h][dst_col : dst_col + len], for K and for V. src_kind 0 reads
the old cache, 1 the staging box (the admitted requests' prefilled KV).
Cells outside every destination range are unchanged.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

import numpy as np


def kv_scatter_compact(segs, src_k, src_v, stg_k, stg_v, dst_k, dst_v):
    """Boxes are [layers][rows][Hkv][W][D] arrays (any dtype); returns new
    (dst_k, dst_v) copies. Destination ranges must be disjoint and must not
    overlap any source range of the same array (checked)."""
    out_k = dst_k.copy()
    out_v = dst_v.copy()
    dst_cells = set()
    for s in segs:
        for t in range(int(s["len"])):
            cell = (int(s["dst_row"]), int(s["dst_col"]) + t)
            if cell in dst_cells:
                raise ValueError("overlapping destination segments")
            dst_cells.add(cell)
    for s in segs:
        kind, sr, sc, dr, dc, ln = (int(s["src_kind"]), int(s["src_row"]), int(s["src_col"]),
                                    int(s["dst_row"]), int(s["dst_col"]), int(s["len"]))
        if kind == 0 and src_k is dst_k:
            if any((sr, sc + t) in dst_cells for t in range(ln)):
                raise ValueError("source overlaps a destination")
        sk, sv = (src_k, src_v) if kind == 0 else (stg_k, stg_v)
        for l in range(out_k.shape[0]):
            for h in range(out_k.shape[2]):
                out_k[l, dr, h, dc:dc + ln] = sk[l, sr, h, sc:sc + ln]
                out_v[l, dr, h, dc:dc + ln] = sv[l, sr, h, sc:sc + ln]
    return out_k, out_v
