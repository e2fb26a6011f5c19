"""Host-side logic of bench.py that needs no GPU: the refusal of more than one
GPU, the algorithmic byte and flop model of the step on a case worked out by
hand, and the rule that a committed counter summary only counts while the
kernel's sources are unchanged."""
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("mode", [[], ["--refresh"], ["--lm-head"], ["--config", "5"]])
def test_more_than_one_gpu_is_refused(mode):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"] + mode,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2, r.stderr
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_algorithmic_bytes_by_hand():
    # two requests, L = 8: (p, g, k) = (5, 16, 1) -> s = 13, B = 8, len = 21;
    # (3, 4, 0) -> s = 3, B = 4, len = 7. Hq = 4, Hkv = 2, D = 16, bf16.
    w = synth.custom(8, 4, 2, 16, 100, "bf16", [5, 3], [16, 4], [1, 0])
    ab = bench.algorithmic_bytes(w)
    eb, Hq, Hkv, D = 2, 4, 2, 16
    kv = (21 + 7) * Hkv * D * 2 * eb                    # every key and value of both rows, once
    qo = 2 * (8 + 4) * Hq * D * eb                      # queries in, outputs out
    wt = (8 + 4) * Hkv * D * 2 * eb                     # fresh block K/V written into the cache
    assert ab["kv"] == kv and ab["qo"] == qo and ab["write_through"] == wt
    assert ab["attn"] == ab["attn_per_layer"] == kv + qo + wt
    assert ab["positions"] == 12
    assert ab["attn_flops"] == 4 * (8 * 21 + 4 * 7) * Hq * D    # QK^T and PV, 2 flops per MAC


def test_algorithmic_bytes_scale_with_layers():
    w = synth.custom(8, 4, 2, 16, 100, "bf16", [5, 3], [16, 4], [1, 0])
    one = bench.algorithmic_bytes(w)
    w.layers = 3
    three = bench.algorithmic_bytes(w)
    assert three["attn"] == 3 * one["attn"] and three["attn_per_layer"] == one["attn_per_layer"]
    assert three["attn_flops"] == 3 * one["attn_flops"] and three["positions"] == one["positions"]


def test_traffic_counts_only_for_the_current_sources(tmp_path, monkeypatch):
    kernel = "k_decode_parts<unsigned short>"
    h = bench.source_hash("k_decode_parts")
    f = tmp_path / "traffic_x.md"
    monkeypatch.setattr(bench, "traffic_file", lambda workload: str(f))
    f.write_text(f"`traffic k_decode_parts 12345 {h}`  \n")
    assert bench.read_traffic("x", kernel) == 12345
    f.write_text(f"`traffic k_decode_parts 12345 {'0' * 16}`  \n")      # taken from other sources
    assert bench.read_traffic("x", kernel) is None
    f.unlink()
    assert bench.read_traffic("x", kernel) is None
