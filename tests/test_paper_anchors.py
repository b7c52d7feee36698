"""The bench's byte accounting against the KV sizes the paper states.

Fixture: tests/golden/paper_size_anchors.json (each entry cites its passage;
model shapes are the public Qwen3 configurations).  The paper quotes the
Qwen3-32B 8K cache as about 2 GB in BF16 and 1 GB in BFP8 (Sec. 2.3,
Challenge 1) and the per-request egress as at most 49 ms at 92.3 Gb/s
(Sec. 3.2).  The second figure also separates the block-size readings: one
exponent byte per 16 elements gives 49 ms, per 32 elements 48 ms, none 47 ms.
"""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (byte accounting only; nothing touches a GPU)

ANCHORS = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_size_anchors.json")))["anchors"]
GIB = 1 << 30


def _kv_bytes(a, per_token_layer):
    m = a["model"]
    return a["tokens"] * m["layers"] * per_token_layer(m["num_kv_heads"], m["head_dim"])


def test_qwen3_32b_8k_cache_sizes():
    a = ANCHORS[0]
    bf16 = _kv_bytes(a, bench.bf16_bytes_per_token_layer)
    bfp8 = _kv_bytes(a, bench.bfp8_bytes_per_token_layer)
    assert bf16 == 2 * GIB
    assert bfp8 == 1.0625 * GIB
    # the paper's rounded figures
    assert round(bf16 / GIB) == a["paper_bf16_GB"]
    assert round(bfp8 / GIB) == a["paper_bfp8_GB"]
    # BFP8 costs 1.0625 B per element against 2 B
    assert bfp8 / bf16 == pytest.approx(1.0625 / 2)


def test_egress_time_matches_the_16_element_block_reading():
    a = ANCHORS[1]
    rate = a["link_Gbps"] * 1e9 / 8                       # bytes per second
    ms = _kv_bytes(a, bench.bfp8_bytes_per_token_layer) / rate * 1e3
    assert round(ms) == a["paper_egress_ms_max"]
    m = a["model"]
    elems = a["tokens"] * m["layers"] * 2 * m["num_kv_heads"] * m["head_dim"]
    # other block sizes do not reproduce the paper's figure
    for bytes_per_elem in (1.0, 1.0 + 1.0 / 32):
        assert round(elems * bytes_per_elem / rate * 1e3) != a["paper_egress_ms_max"]


def test_attention_launch_bytes_for_the_headline_workload():
    import workloads as wl
    w = wl.WORKLOADS[3]
    ctx = wl.context_lens(w)
    # KV of one layer, Q in and BF16 out, page ids and lengths
    kv = int(ctx.sum()) * bench.bfp8_bytes_per_token_layer(w.num_kv_heads)
    assert kv == 285_212_672
    assert bench.attn_bytes(w, ctx) == kv + 2 * 16 * 64 * 128 * 2 + 16 * 512 * 4 + 16 * 4
