"""GPU parity of hma_bfp8_rebuild_tiled against the oracle: bit-exact.

The decoder's single pass (Sec. 3.3): tiled per-chip prefill shards ->
row-major BF16 pages, with the rotary key re-layout for keys.  Inputs are
random tile bytes (every exponent and byte value occurs); the oracle rebuilds
the same bytes.  Also: pages not named stay untouched, padding rows of the
last token tile are ignored, several pools at a byte stride, and a Qwen3-32B
8K request (64 layers, K and V, four prefill chips) in one launch."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_29986_amd as hma
from gpu_util import dev, note

pytestmark = pytest.mark.gpu

P, D = 16, 128
SENTINEL = 0x5A5A


def _case(rng, n_pools, n_shards, n_tokens, hkv, pool_pages, pad_stride=0):
    pool_bytes = n_shards * hma.tiled_shard_bytes(n_tokens, hkv // n_shards)
    stride = pool_bytes + pad_stride
    src = rng.integers(0, 256, n_pools * stride, dtype=np.uint8)
    n_req = (n_tokens + P - 1) // P
    dst_pages = rng.choice(pool_pages, n_req, replace=False).astype(np.int32)
    return src, stride, dst_pages


@pytest.mark.parametrize("rope", [False, True])
@pytest.mark.parametrize("n_shards,n_tokens,hkv", [(1, 1, 8), (2, 31, 8), (4, 100, 8), (8, 257, 8),
                                                   (1, 64, 1), (2, 48, 4)])
def test_tiled_rebuild_matches_oracle(rope, n_shards, n_tokens, hkv):
    note(f"tiled rebuild: shards={n_shards} tokens={n_tokens} hkv={hkv} rope={rope}")
    rng = np.random.default_rng(500 + n_tokens + 13 * n_shards + hkv)
    n_pools, pool_pages = 3, 40
    src, stride, dst_pages = _case(rng, n_pools, n_shards, n_tokens, hkv, pool_pages, pad_stride=48)
    want = np.full((n_pools * pool_pages, hkv, P, D), SENTINEL, np.uint16)
    oracle.rebuild_tiled(src, stride, n_pools, n_shards, n_tokens, hkv, want, dst_pages, pool_pages,
                         rope)
    out = torch.full(want.shape, SENTINEL, dtype=torch.int16, device="cuda")
    hma.bfp8_rebuild_tiled(dev(src), out, n_tokens, n_shards, dst_pages=dev(dst_pages),
                           n_pools=n_pools, src_pool_stride_bytes=stride,
                           dst_pool_stride_pages=pool_pages, rope_reorder=rope, num_kv_heads=hkv)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:4].tolist()}"


def test_tiled_rebuild_identity_pages():
    note("tiled rebuild: identity page list")
    rng = np.random.default_rng(77)
    n_tokens, hkv, n_shards = 90, 8, 2
    src, stride, _ = _case(rng, 1, n_shards, n_tokens, hkv, 6)
    n_req = (n_tokens + P - 1) // P
    want = np.full((n_req, hkv, P, D), SENTINEL, np.uint16)
    oracle.rebuild_tiled(src, 0, 1, n_shards, n_tokens, hkv, want, np.arange(n_req, dtype=np.int32), 0, True)
    out = torch.full(want.shape, SENTINEL, dtype=torch.int16, device="cuda")
    hma.bfp8_rebuild_tiled(dev(src), out, n_tokens, n_shards, rope_reorder=True, num_kv_heads=hkv)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint16), want)


def test_tiled_rebuild_qwen3_32b_8k_request():
    """64 layers x (K, V) of one 8K request from four prefill chips (Table 2:
    Qwen3-32B prefill at TP = 4): keys re-laid out, values not; sampled layers
    checked bitwise against the oracle."""
    note("tiled rebuild: Qwen3-32B 8K request, 4 shards, 64 layers")
    rng = np.random.default_rng(88)
    n_tokens, hkv, n_shards, layers = 8192, 8, 4, 64
    n_req = n_tokens // P
    pool_bytes = n_shards * hma.tiled_shard_bytes(n_tokens, hkv // n_shards)
    src = torch.randint(0, 256, (2, layers, pool_bytes), dtype=torch.uint8, device="cuda")
    out = torch.empty((2, layers, n_req, hkv, P, D), dtype=torch.int16, device="cuda")
    for kind in (0, 1):        # K pools (re-laid out), V pools
        hma.bfp8_rebuild_tiled(src[kind], out[kind], n_tokens, n_shards, n_pools=layers,
                               src_pool_stride_bytes=pool_bytes, dst_pool_stride_pages=n_req,
                               rope_reorder=(kind == 0), num_kv_heads=hkv)
    torch.cuda.synchronize()
    for kind in (0, 1):
        for layer in (0, 37, 63):
            s = src[kind, layer].cpu().numpy()
            want = np.empty((n_req, hkv, P, D), np.uint16)
            oracle.rebuild_tiled(s, 0, 1, n_shards, n_tokens, hkv, want,
                                 np.arange(n_req, dtype=np.int32), 0, kind == 0)
            assert np.array_equal(out[kind, layer].cpu().numpy().view(np.uint16), want), (kind, layer)
