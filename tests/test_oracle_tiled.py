"""Pins of the oracle's tiled-shard rebuild (Sec. 3.3: the decoder's single
pass converts the prefill side's tiled layout to row-major pages, merges the
per-chip KV shards and moves keys from the interleaved to the half-split
rotary order).

* Tile order: shards built here from row-major pages with numpy reshapes and
  transposes (written from the documented layout, independently of the
  oracle's index arithmetic) must rebuild to the decode of those pages.
* Key re-layout: the channel permutation the oracle applies is read back from
  a tile whose values are the channel numbers, and checked against the rotary
  identity it must satisfy: rotating interleaved pairs (2i, 2i+1) and then
  relabelling equals relabelling and then rotating half-split pairs
  (i, i + D/2), for every position.
"""
import numpy as np
import pytest

import oracle
import workloads as wl

D, P = 128, 16


def _pages(rng, n_pages, hkv):
    mant = rng.integers(0, 256, (n_pages, hkv, P, D), dtype=np.uint8)
    ex = rng.integers(0, 256, (n_pages, hkv, P, D // 16), dtype=np.uint8)
    return mant, ex


def _shards_from_pages(mant, ex, page_list, n_tokens, n_shards, rng):
    """Tiled shards of one pool from row-major pages (test-side construction)."""
    hkv = mant.shape[1]
    hs = hkv // n_shards
    tt = (n_tokens + 31) // 32
    # token-major rows, padded to whole tiles with bytes the rebuild must ignore
    M = rng.integers(0, 256, (hkv, tt * 32, D), dtype=np.uint8)
    E = rng.integers(0, 256, (hkv, tt * 32, D // 16), dtype=np.uint8)
    for p in range(n_tokens):
        M[:, p] = mant[page_list[p // P], :, p % P]
        E[:, p] = ex[page_list[p // P], :, p % P]
    # mantissas: (head, tt, fr, row, ct, fc, col) -> (head, tt, ct, fr, fc, row, col)
    m6 = M.reshape(hkv, tt, 2, 16, D // 32, 2, 16).transpose(0, 1, 4, 2, 5, 3, 6)
    m_tiles = m6.reshape(hkv, tt, D // 32, 4 * 256)
    # exponents: block b = 2 ct + fc of token 32 tt + 16 fr + row
    e5 = E.reshape(hkv, tt, 2, 16, D // 32, 2).transpose(0, 1, 4, 2, 5, 3)
    e_tiles = e5.reshape(hkv, tt, D // 32, 64)
    tiles = np.concatenate([e_tiles, m_tiles], axis=-1)           # [head][tt][ct][1088]
    return np.concatenate([tiles[t * hs:(t + 1) * hs].reshape(-1) for t in range(n_shards)])


@pytest.mark.parametrize("n_shards", [1, 2, 4, 8])
@pytest.mark.parametrize("n_tokens", [1, 16, 31, 32, 33, 100, 256])
def test_tile_order_and_shard_merge_match_row_major_pages(n_shards, n_tokens):
    rng = np.random.default_rng(1000 + 7 * n_tokens + n_shards)
    hkv, pool_pages = 8, 40
    n_req = (n_tokens + P - 1) // P
    mant, ex = _pages(rng, pool_pages, hkv)
    src_list = rng.choice(pool_pages, n_req, replace=False)
    shards = _shards_from_pages(mant, ex, src_list, n_tokens, n_shards, rng)
    assert shards.size == n_shards * oracle.tiled_shard_bytes(n_tokens, hkv // n_shards)
    dst_pages = rng.choice(pool_pages, n_req, replace=False).astype(np.int32)
    out = np.full((pool_pages, hkv, P, D), 0x5A5A, np.uint16)
    oracle.rebuild_tiled(shards, 0, 1, n_shards, n_tokens, hkv, out, dst_pages, 0, False)
    want = oracle.decode_blocks(mant, ex)
    for p in range(n_tokens):
        assert np.array_equal(out[dst_pages[p // P], :, p % P], want[src_list[p // P], :, p % P]), p
    # slots past the last token and pages not named stay untouched
    last = n_tokens % P
    if last:
        assert (out[dst_pages[-1], :, last:] == 0x5A5A).all()
    others = np.setdiff1d(np.arange(pool_pages), dst_pages)
    assert (out[others] == 0x5A5A).all()


def test_several_pools_at_a_byte_stride():
    rng = np.random.default_rng(77)
    hkv, n_tokens, pools, shards = 4, 70, 3, 2
    n_req = (n_tokens + P - 1) // P
    stride = oracle.tiled_shard_bytes(n_tokens, hkv // shards) * shards + 512
    src = rng.integers(0, 256, pools * stride, dtype=np.uint8)
    want = []
    for q in range(pools):
        mant, ex = _pages(rng, n_req, hkv)
        src[q * stride:q * stride + stride - 512] = _shards_from_pages(mant, ex, np.arange(n_req),
                                                                       n_tokens, shards, rng)
        want.append(oracle.decode_blocks(mant, ex))
    out = np.zeros((pools * 10, hkv, P, D), np.uint16)
    oracle.rebuild_tiled(src, stride, pools, shards, n_tokens, hkv, out, np.arange(n_req, dtype=np.int32),
                         10, False)
    for q in range(pools):
        got = out[q * 10:q * 10 + n_req].transpose(0, 2, 1, 3).reshape(-1, hkv, D)[:n_tokens]
        exp = want[q].transpose(0, 2, 1, 3).reshape(-1, hkv, D)[:n_tokens]
        assert np.array_equal(got, exp), q


def _rotate(x, pairs, theta):
    y = x.copy()
    for (a, b), t in zip(pairs, theta):
        y[a] = x[a] * np.cos(t) - x[b] * np.sin(t)
        y[b] = x[a] * np.sin(t) + x[b] * np.cos(t)
    return y


def test_key_relayout_is_the_rotary_relabelling():
    # one token whose channel c holds the value c (E = 133: value = magnitude)
    n_tokens, hkv = 1, 1
    tiles = np.zeros(oracle.tiled_shard_bytes(n_tokens, hkv), np.uint8).reshape(D // 32, 1088)
    for ct in range(D // 32):
        tiles[ct, :64] = 133
        for cc in range(32):
            face = cc // 16
            tiles[ct, 64 + face * 256 + (cc % 16)] = 32 * ct + cc
    out = np.zeros((1, hkv, P, D), np.uint16)
    oracle.rebuild_tiled(tiles.reshape(-1), 0, 1, 1, n_tokens, hkv, out, np.zeros(1, np.int32), 0,
                         True)
    perm = oracle.bf16_to_f64(out[0, 0, 0]).astype(int)       # output position -> source channel
    assert sorted(perm) == list(range(D))
    ident = np.zeros_like(out)
    oracle.rebuild_tiled(tiles.reshape(-1), 0, 1, 1, n_tokens, hkv, ident, np.zeros(1, np.int32), 0,
                         False)
    assert np.array_equal(oracle.bf16_to_f64(ident[0, 0, 0]).astype(int), np.arange(D))
    rng = np.random.default_rng(5)
    theta_base = 10000.0 ** (-2.0 * np.arange(D // 2) / D)
    inter = [(2 * i, 2 * i + 1) for i in range(D // 2)]
    half = [(i, i + D // 2) for i in range(D // 2)]
    for pos in (0, 1, 7, 4095):
        x = rng.standard_normal(D)
        lhs = _rotate(x, inter, pos * theta_base)[perm]      # rotate on the prefill side, relabel
        rhs = _rotate(x[perm], half, pos * theta_base)       # relabel, rotate the decode-side way
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n_shards,n_tokens", [(1, 5), (2, 47), (4, 200), (8, 33)])
def test_pack_keeps_the_bytes_of_row_major_pages(n_shards, n_tokens):
    """Packing tiled shards back into BFP8 pages returns the page bytes that
    the numpy re-tiling started from (slots past the last token untouched)."""
    rng = np.random.default_rng(300 + n_tokens)
    hkv, pool_pages = 8, 30
    n_req = (n_tokens + P - 1) // P
    mant, ex = _pages(rng, pool_pages, hkv)
    src_list = rng.choice(pool_pages, n_req, replace=False)
    shards = _shards_from_pages(mant, ex, src_list, n_tokens, n_shards, rng)
    dst_pages = rng.choice(pool_pages, n_req, replace=False).astype(np.int32)
    pm = np.full((pool_pages, hkv, P, D), 0xA5, np.uint8)
    pe = np.full((pool_pages, hkv, P, D // 16), 0xA5, np.uint8)
    oracle.pack_tiled(shards, 0, 1, n_shards, n_tokens, hkv, pm, pe, dst_pages, 0)
    for p in range(n_tokens):
        assert np.array_equal(pm[dst_pages[p // P], :, p % P], mant[src_list[p // P], :, p % P])
        assert np.array_equal(pe[dst_pages[p // P], :, p % P], ex[src_list[p // P], :, p % P])
    if n_tokens % P:
        assert (pm[dst_pages[-1], :, n_tokens % P:] == 0xA5).all()


def _relayout_perm():
    """Output position -> source channel of the oracle's key re-layout (the
    permutation pinned by the rotary identity above)."""
    tiles = np.zeros(oracle.tiled_shard_bytes(1, 1), np.uint8).reshape(D // 32, 1088)
    for ct in range(D // 32):
        tiles[ct, :64] = 133
        for cc in range(32):
            tiles[ct, 64 + (cc // 16) * 256 + cc % 16] = 32 * ct + cc
    out = np.zeros((1, 1, P, D), np.uint16)
    oracle.rebuild_tiled(tiles.reshape(-1), 0, 1, 1, 1, 1, out, np.zeros(1, np.int32), 0, True)
    return oracle.bf16_to_f64(out[0, 0, 0]).astype(int)


def test_attention_over_interleaved_keys_matches_sdpa_on_relabelled_keys():
    """key_order = 1: K pages hold the rows as the prefill side leaves them.
    The result must equal float64 attention (torch SDPA) over the keys
    relabelled with the re-layout permutation, and attention over BF16 pages
    that already hold the relabelled keys."""
    import torch
    rng = np.random.default_rng(9)
    B, Hq, hkv, ctx = 2, 8, 2, 45
    n_pages = 2 * ((ctx + P - 1) // P)
    k_mant, k_exp = _pages(rng, n_pages, hkv)
    k_exp[:] = rng.integers(120, 134, k_exp.shape, dtype=np.uint8)
    v_mant, v_exp = _pages(rng, n_pages, hkv)
    v_exp[:] = rng.integers(120, 134, v_exp.shape, dtype=np.uint8)
    pt = np.arange(n_pages, dtype=np.int32).reshape(B, -1)
    cl = np.full(B, ctx, np.int32)
    q = wl.f32_to_bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    scale = 1.0 / np.sqrt(D)
    out, lse = oracle.decode_attn(q, k_mant, k_exp, v_mant, v_exp, None, None, pt, cl, hkv, P, scale,
                                  key_order=1)
    perm = _relayout_perm()
    kd = oracle.bf16_to_f64(oracle.decode_blocks(k_mant, k_exp))[..., perm]   # relabelled keys
    vd = oracle.bf16_to_f64(oracle.decode_blocks(v_mant, v_exp))
    s32 = float(np.float32(scale))
    for b in range(B):
        K = np.concatenate([kd[pt[b, i]] for i in range(pt.shape[1])], axis=1)[:, :ctx]  # [hkv][t][D]
        V = np.concatenate([vd[pt[b, i]] for i in range(pt.shape[1])], axis=1)[:, :ctx]
        qf = torch.from_numpy(oracle.bf16_to_f64(q[b])).view(hkv, Hq // hkv, 1, D)
        ref = torch.nn.functional.scaled_dot_product_attention(
            qf, torch.from_numpy(K)[:, None], torch.from_numpy(V)[:, None], scale=s32)
        np.testing.assert_allclose(out[b], ref.reshape(Hq, D).numpy(), rtol=0, atol=1e-12)
    # the same keys as BF16 pages already in half-split order, read without relabelling
    kb = oracle.decode_blocks(k_mant, k_exp)[..., perm].copy()
    vb = oracle.decode_blocks(v_mant, v_exp)
    out2, lse2 = oracle.decode_attn(q, k_mant, k_exp, v_mant, v_exp, kb, vb, pt | 0x40000000, cl,
                                    hkv, P, scale)
    np.testing.assert_allclose(out, out2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse2, rtol=0, atol=1e-12)
