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


@pytest.mark.parametrize("n_shards,n_tokens", [(1, 1), (2, 47), (4, 300), (8, 64)])
def test_pack_tiled_matches_oracle(n_shards, n_tokens):
    note(f"pack tiled: shards={n_shards} tokens={n_tokens}")
    rng = np.random.default_rng(900 + n_tokens + n_shards)
    hkv, n_pools, pool_pages = 8, 2, 30
    src, stride, dst_pages = _case(rng, n_pools, n_shards, n_tokens, hkv, pool_pages, pad_stride=16)
    wm = np.full((n_pools * pool_pages, hkv, P, D), 0xA5, np.uint8)
    we = np.full((n_pools * pool_pages, hkv, P, D // 16), 0xA5, np.uint8)
    oracle.pack_tiled(src, stride, n_pools, n_shards, n_tokens, hkv, wm, we, dst_pages, pool_pages)
    gm = torch.full(wm.shape, 0xA5, dtype=torch.uint8, device="cuda")
    ge = torch.full(we.shape, 0xA5, dtype=torch.uint8, device="cuda")
    hma.bfp8_pack_tiled(dev(src), gm, ge, n_tokens, n_shards, dst_pages=dev(dst_pages), n_pools=n_pools,
                        src_pool_stride_bytes=stride, dst_pool_stride_pages=pool_pages, num_kv_heads=hkv)
    torch.cuda.synchronize()
    assert np.array_equal(gm.cpu().numpy(), wm)
    assert np.array_equal(ge.cpu().numpy(), we)


def test_raw_pages_from_shards_through_fused_attention():
    """The deferred path end to end: prefill shards packed into BFP8 pages on
    the GPU, keys still in the interleaved rotary order, read by the fused
    attention with key_order = 1; against the oracle (which relabels the keys
    on read).  Both kernel shapes; also bitwise equal to the mixed-format
    kernel over BF16 pages that hold the same (stored-order) keys."""
    import workloads as wl
    from gpu_util import DevKV, assert_attn_close
    from oracle_fixtures import PagedKV
    rng = np.random.default_rng(4242)
    B, hq, hkv, n_shards = 4, 32, 8, 4
    ctx = np.array([70, 200, 1, 129], np.int32)
    pages_per = (ctx + P - 1) // P
    total = int(pages_per.sum())
    pt = np.zeros((B, int(pages_per.max())), np.int32)
    order = rng.permutation(total).astype(np.int32)
    k_mant = np.zeros((total, hkv, P, D), np.uint8)
    k_exp = np.zeros((total, hkv, P, D // 16), np.uint8)
    v_mant = np.zeros_like(k_mant)
    v_exp = np.zeros_like(k_exp)
    at = 0
    for b in range(B):
        ids = order[at:at + pages_per[b]]
        at += pages_per[b]
        pt[b, :pages_per[b]] = ids
        for mant, ex in ((k_mant, k_exp), (v_mant, v_exp)):
            # one request's shards: moderate exponents, random bytes
            pool_bytes = n_shards * hma.tiled_shard_bytes(int(ctx[b]), hkv // n_shards)
            src = rng.integers(0, 256, pool_bytes, dtype=np.uint8)
            tiles = src.reshape(-1, 1088)
            tiles[:, :64] = rng.integers(118, 132, (tiles.shape[0], 64), dtype=np.uint8)
            gm = torch.zeros(mant.shape, dtype=torch.uint8, device="cuda")
            ge = torch.zeros(ex.shape, dtype=torch.uint8, device="cuda")
            gm.copy_(torch.from_numpy(mant))
            ge.copy_(torch.from_numpy(ex))
            hma.bfp8_pack_tiled(dev(src), gm, ge, int(ctx[b]), n_shards, dst_pages=dev(ids),
                                num_kv_heads=hkv)
            torch.cuda.synchronize()
            mant[:] = gm.cpu().numpy()
            ex[:] = ge.cpu().numpy()
            # the GPU packing is pinned separately; check this request's pages anyway
            wm = np.zeros_like(mant)
            we = np.zeros_like(ex)
            oracle.pack_tiled(src, 0, 1, n_shards, int(ctx[b]), hkv, wm, we, ids, 0)
            for i, pid in enumerate(ids):
                n_valid = min(P, int(ctx[b]) - i * P)
                assert np.array_equal(mant[pid, :, :n_valid], wm[pid, :, :n_valid])
    q = wl.f32_to_bf16_bits(rng.standard_normal((B, hq, D)).astype(np.float32))
    kv = PagedKV(q, k_mant, k_exp, v_mant, v_exp, oracle.decode_blocks(k_mant, k_exp),
                 oracle.decode_blocks(v_mant, v_exp), pt, ctx, hkv, P, 1.0 / np.sqrt(D))
    ref, ref_lse = kv.oracle_attn(key_order=1)
    d = DevKV(kv)
    for tps in (0, 16):        # 32 workgroups (8 waves each) and 416 (the 4-wave shape)
        note(f"attn over packed shards, key_order=1, tps={tps}")
        out, lse = d.attn(tokens_per_split=tps, use_bf16_pools=False, key_order=1)
        assert_attn_close(out, lse, ref, ref_lse, what=f"interleaved keys tps={tps}")
        kv_bf = PagedKV(q, k_mant, k_exp, v_mant, v_exp, kv.k_bf16, kv.v_bf16, pt | wl.TAG_BF16, ctx,
                        hkv, P, kv.scale)
        out_b, lse_b = DevKV(kv_bf).attn(tokens_per_split=tps, key_order=1)
        assert torch.equal(out, out_b) and torch.equal(lse, lse_b)
    # and the interleaved keys do matter: reading them as half-split differs
    out0, _ = d.attn(use_bf16_pools=False, key_order=0)
    assert not torch.equal(out0, out)
