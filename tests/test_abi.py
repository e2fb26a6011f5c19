"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/blockserve.h declares, validates descriptors on the
host, and rejects bad arguments before touching a device."""
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2607_08930_amd as bs

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "blockserve.h")


def declared():
    src = open(HDR).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bs_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert len(names) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", bs.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(bs_\w+)", out))
    for n in names:
        assert n in exported, f"{n} declared but not exported"
        assert hasattr(bs.lib, n)
        assert hasattr(bs, n), f"binding lacks {n}"


def test_status_strings():
    assert [bs.bs_status_string(i) for i in range(7)] == [
        "BS_OK", "BS_ERR_INVALID_ARG", "BS_ERR_UNSUPPORTED", "BS_ERR_DESCRIPTOR", "BS_ERR_OVERLAP",
        "BS_ERR_WORKSPACE", "BS_ERR_HIP"]
    assert bs.bs_status_string(99) == "BS_UNKNOWN_STATUS"


@pytest.mark.parametrize("bad,msg", [
    ((5, 16, 2, 0, 0), "block index"), ((5, 16, -1, 0, 0), "block index"), ((5, 0, 0, 0, 0), "g >= 1"),
    ((-1, 16, 0, 0, 0), "p >= 0"), ((5, 16, 0, 9, 0), "row 9"), ((5, 16, 0, 0, 40), "exceeds W"),
    ((5, 16, 0, 0, -1), "exceeds W"),
])
def test_validate_rejects_each_class(bad, msg):
    with pytest.raises(bs.BlockServeError, match=msg) as e:
        bs.bs_validate_requests(np.array([bad], bs.REQ_DTYPE), 8, 4, 52)
    assert e.value.name == "BS_ERR_DESCRIPTOR"


def test_validate_duplicate_row_and_good_batch():
    with pytest.raises(bs.BlockServeError, match="used twice"):
        bs.bs_validate_requests(np.array([(5, 16, 0, 1, 0), (5, 16, 0, 1, 0)], bs.REQ_DTYPE), 8, 4, 52)
    good = np.array([(5, 16, 1, 0, 31), (12, 24, 0, 1, 16), (7, 8, 0, 2, 37), (20, 32, 3, 3, 0)], bs.REQ_DTYPE)
    bs.bs_validate_requests(good, 8, 4, 52)
    with pytest.raises(bs.BlockServeError, match="L < 1"):
        bs.bs_validate_requests(good, 0, 4, 52)


def test_calls_without_context_fail_before_any_device_work():
    null = None
    assert bs.lib.bs_gather_active_blocks(null, None, 0, 8, 1, 1, None, 0, 4, None, None, None) == 1
    assert bs.lib.bs_parallel_decode(null, None, 0, 8, 10, 0, None, 16, None, None, 0.9, 1, -1, None, None,
                                     None, None, None, 0, None) == 1
    assert bs.lib.bs_kv_scatter_compact(null, None, 0, 1, 1, 8, 0, None, None, 0, 1, 1, None, None, 0, 1, 1,
                                        None, None, 0, 1, 1, None) == 1
    assert bs.lib.bs_mixed_state_step(null, None, 0, 8, 1, 1, 0, 1, 1, 64, 0, 0.0, 1, None, None, None, None,
                                      None, None, 10, 0, None, 16, None, 1, None, 1, 0.9, 1, -1, None, None,
                                      None, None, None, None, 0, None) == 1
    assert bs.lib.bs_profile_begin(null, 4) == 1
    assert bs.lib.bs_lm_head_decode(null, None, 0, 8, 64, 10, 0, None, None, None, None, 0.9, 1, -1, None,
                                    None, None, None, None, 0, None) == 1
    assert bs.lib.bs_lm_head_pack(null, None, 64, 10, 64, 0, None, 0, None) == 1
    assert bs.lib.bs_dual_cache_refresh(null, None, 0, 32, 4, 2, 128, 1, 0.0, 1e4, None, None, None, 1, 1,
                                        None, None, None, None) == 1
    assert "ctx is NULL" in bs.bs_last_error()


def test_lm_head_workspace_query():
    # count (16 B) + row list (n L int32, 16-byte rounded) + one merged part
    # per row + one part per (row, 128-entry vocabulary slice)
    parts = 2 * -(-126464 // 256)
    assert parts == 988
    assert bs.bs_lm_head_workspace_bytes(32, 32, 126464) == 16 + 4096 + 1024 * 16 + 1024 * parts * 16
    assert bs.bs_lm_head_workspace_bytes(1, 3, 1) == 16 + 16 + 3 * 16 + 3 * 2 * 16
    assert bs.bs_lm_head_workspace_bytes(0, 8, 10) == 0
    # packed head: whole 256-row tiles of d bf16 each
    assert bs.bs_lm_head_pack_bytes(126464, 4096) == 494 * 256 * 4096 * 2
    assert bs.bs_lm_head_pack_bytes(1, 32) == 256 * 32 * 2


def test_workspace_queries():
    # a 126464-entry bf16 row is 8 chunks of 32 KiB, streamed as 4 parts of 2
    # chunks; the workspace holds one 16-byte part result per (i, j, part),
    # then one 8-byte block mask word per request
    assert bs.bs_decode_workspace_bytes(32, 32, 126464, bs.BS_BF16) == 32 * 32 * 4 * 16 + 32 * 8
    assert bs.bs_decode_workspace_bytes(2, 4, 16384, bs.BS_BF16) == 2 * 4 * 16 + 2 * 8      # exactly one chunk
    assert bs.bs_decode_workspace_bytes(2, 4, 16385, bs.BS_BF16) == 2 * 4 * 16 + 2 * 8      # two chunks, one part
    assert bs.bs_decode_workspace_bytes(2, 4, 32769, bs.BS_BF16) == 2 * 4 * 2 * 16 + 2 * 8  # three chunks
    assert bs.bs_decode_workspace_bytes(4, 8, 1000, bs.BS_F32) == 4 * 8 * 16 + 4 * 8
    assert bs.bs_decode_workspace_bytes(3, 5, 1000, bs.BS_F32) == 3 * 5 * 16 + 3 * 8
    assert bs.bs_decode_workspace_bytes(0, 8, 1000, bs.BS_F32) == 0
    reqs = np.array([(5, 16, 1, 0, 31)], bs.REQ_DTYPE)
    assert bs.bs_attention_workspace_bytes(reqs, 8, 2, 2, 64, bs.BS_F32) >= 0


def test_package_has_no_cpu_fallback():
    import inspect
    src = inspect.getsource(bs)
    assert "oracle" not in src.replace("oracle/", "")
    assert "import synth" not in src


def segs_of(rows):
    return np.array(rows, bs.SEG_DTYPE)


def test_validate_segments_zero_length_cannot_hide_an_overlap():
    # A = [0, 10) and C = [5, 6) on one destination row, with a zero-length
    # Z = [3, 3) that sorts between them
    a, z, c = (1, 0, 0, 2, 0, 10), (1, 1, 0, 2, 3, 0), (1, 2, 0, 2, 5, 1)
    for order in ([a, z, c], [z, a, c], [c, z, a], [a, c, z]):
        with pytest.raises(bs.BlockServeError, match="overlapping") as e:
            bs.bs_validate_segments(segs_of(order), 4, 16, 4, 16, 4, 16)
        assert e.value.name == "BS_ERR_OVERLAP"
    # a long range covering a later one past an intermediate disjoint one
    with pytest.raises(bs.BlockServeError, match="overlapping"):
        bs.bs_validate_segments(segs_of([(1, 0, 0, 0, 0, 12), (1, 1, 0, 0, 2, 1), (1, 2, 0, 0, 9, 2)]),
                                4, 16, 4, 16, 4, 16)
    # zero-length segments alone never overlap, even at a covered cell
    bs.bs_validate_segments(segs_of([(1, 0, 0, 2, 0, 10), (1, 1, 0, 2, 3, 0), (1, 2, 0, 2, 10, 4)]),
                            4, 16, 4, 16, 4, 16)
    bs.bs_validate_segments(segs_of([]), 4, 16, 4, 16, 4, 16)


def test_validate_segments_rules():
    ok = [(0, 0, 0, 1, 0, 8), (1, 0, 0, 0, 8, 8), (0, 3, 2, 3, 0, 4)]
    bs.bs_validate_segments(segs_of(ok), 4, 16, 2, 16, 4, 16)
    for bad, msg in [((0, 4, 0, 0, 0, 1), "source range"), ((1, 2, 0, 0, 0, 1), "source range"),
                     ((0, 0, 10, 0, 0, 7), "source range"), ((0, 0, 0, 0, 12, 5), "destination range"),
                     ((0, 0, 0, -1, 0, 1), "destination range"), ((2, 0, 0, 0, 0, 1), "src_kind"),
                     ((0, 0, 0, 0, 0, -1), "len < 0")]:
        with pytest.raises(bs.BlockServeError, match=msg) as e:
            bs.bs_validate_segments(segs_of([bad]), 4, 16, 2, 16, 4, 16)
        assert e.value.name == "BS_ERR_INVALID_ARG"
    # in place: a source range that another segment writes is rejected only
    # when the source box is the destination box
    alias = [(0, 1, 0, 2, 0, 4), (0, 3, 0, 1, 2, 4)]          # reads row 1 [0, 4), writes row 1 [2, 6)
    bs.bs_validate_segments(segs_of(alias), 4, 16, 2, 16, 4, 16)
    with pytest.raises(bs.BlockServeError, match="reads cells") as e:
        bs.bs_validate_segments(segs_of(alias), 4, 16, 2, 16, 4, 16, src_is_dst=True)
    assert e.value.name == "BS_ERR_OVERLAP"
    # touching ranges are disjoint; staging aliasing is checked for kind 1 only
    bs.bs_validate_segments(segs_of([(0, 1, 0, 2, 0, 4), (0, 3, 0, 1, 4, 4)]), 4, 16, 2, 16, 4, 16,
                            src_is_dst=True)
    bs.bs_validate_segments(segs_of(alias), 4, 16, 2, 16, 4, 16, stg_is_dst=True)


def test_validate_segments_against_brute_force():
    # random segment sets: the library's verdict equals a cell-by-cell check
    rng = np.random.default_rng(7)
    for trial in range(400):
        n = int(rng.integers(1, 7))
        rows = [(int(rng.integers(0, 2)), int(rng.integers(0, 3)), int(rng.integers(0, 8)),
                 int(rng.integers(0, 3)), int(rng.integers(0, 12)), int(rng.integers(0, 5))) for _ in range(n)]
        rows = [(k, r, min(c, 16 - ln), dr, min(dc, 16 - ln), ln) for k, r, c, dr, dc, ln in rows]
        in_place = bool(trial % 2)
        owner = {}
        expect = None
        for i, (k, r, c, dr, dc, ln) in enumerate(rows):
            for t in range(ln):
                if (dr, dc + t) in owner:
                    expect = "overlapping"
                owner[(dr, dc + t)] = i
        if expect is None and in_place:
            for k, r, c, dr, dc, ln in rows:
                if k == 0 and any((r, c + t) in owner for t in range(ln)):
                    expect = "reads cells"
        if expect is None:
            bs.bs_validate_segments(segs_of(rows), 3, 16, 3, 16, 3, 16, src_is_dst=in_place)
        else:
            with pytest.raises(bs.BlockServeError, match=expect):
                bs.bs_validate_segments(segs_of(rows), 3, 16, 3, 16, 3, 16, src_is_dst=in_place)
