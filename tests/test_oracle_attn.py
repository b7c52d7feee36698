"""Pins for the oracle's paged decode attention, split merge and page
reconstruction (CPU only).

The attention definition (softmax over scaled q.k, weighted mean of v) is the
standard one the paper's decode GPU runs over the paged BF16 cache (Sec. 3.3,
Fig. 2); the oracle is checked against:
  * torch's scaled_dot_product_attention in float64 and scipy's logsumexp
    (library routines) on a dense gather written separately,
  * closed forms: uniform softmax, a single token, one-hot dominance,
    empty context,
  * invariances: split partition, physical page placement, BF16-vs-BFP8 page
    format, identical queries within a GQA group, garbage past the context.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
import workloads as wl
from oracle_fixtures import dense_kv, make_paged, tiny_workload


def _sdpa_reference(kv, b):
    """float64 attention for sequence b via torch SDPA (GQA by repeat)."""
    K, V = dense_kv(kv, b)
    Hq = kv.q.shape[1]
    g = Hq // kv.num_kv_heads
    q = torch.from_numpy(oracle.bf16_to_f64(kv.q[b]))[:, None, :]        # [Hq][1][D]
    Kt = torch.from_numpy(K).repeat_interleave(g, dim=0)                 # [Hq][n][D]
    Vt = torch.from_numpy(V).repeat_interleave(g, dim=0)
    scale = float(np.float32(kv.scale))
    o = torch.nn.functional.scaled_dot_product_attention(q, Kt, Vt, scale=scale)[:, 0, :]
    s = scale * np.einsum("hd,hnd->hn", oracle.bf16_to_f64(kv.q[b]), Kt.numpy())
    return o.numpy(), logsumexp(s, axis=1)


@pytest.mark.parametrize("ctx", [[1, 17], [16, 40], [33, 5]])
def test_attn_matches_torch_sdpa_tiny(ctx):
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    kv = make_paged(w, ctx=ctx)
    out, lse = kv.oracle_attn()
    for b in range(2):
        ref, ref_lse = _sdpa_reference(kv, b)
        np.testing.assert_allclose(out[b], ref, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse[b], ref_lse, rtol=1e-12, atol=1e-12)


def test_attn_matches_torch_sdpa_smoke_workload_mixed_pages():
    w = wl.WORKLOADS[0]
    kv = make_paged(w, bf16_fraction=0.5)
    # half the pages now read the BF16 pool; make that pool differ from the
    # BFP8 pages so the tag is really followed
    kv.k_bf16 = kv.k_bf16 ^ np.uint16(0x0001)
    kv.v_bf16 = kv.v_bf16 ^ np.uint16(0x0001)
    out, lse = kv.oracle_attn()
    for b in range(w.batch):
        ref, ref_lse = _sdpa_reference(kv, b)
        np.testing.assert_allclose(out[b], ref, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(lse[b], ref_lse, rtol=1e-12, atol=1e-12)


def test_uniform_softmax_all_equal_keys():
    w = tiny_workload(Hq=4, Hkv=1, B=1)
    kv = make_paged(w, ctx=[37])
    # all keys equal: copy token 0's K row into every slot of every page
    k0m = kv.k_mant[kv.page_table[0, 0], 0, 0].copy()
    k0e = kv.k_exp[kv.page_table[0, 0], 0, 0].copy()
    kv.k_mant[:, :, :, :] = k0m
    kv.k_exp[:, :, :, :] = k0e
    out, lse = kv.oracle_attn()
    K, V = dense_kv(kv, 0)
    np.testing.assert_allclose(out[0], np.broadcast_to(V[0].mean(axis=0), out[0].shape),
                               rtol=1e-13, atol=1e-13)
    s = float(np.float32(kv.scale)) * oracle.bf16_to_f64(kv.q[0]) @ K[0, 0]
    np.testing.assert_allclose(lse[0], s + np.log(37.0), rtol=1e-13)


def test_single_token_returns_v0_exactly():
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    kv = make_paged(w, ctx=[1, 1])
    out, lse = kv.oracle_attn()
    for b in range(2):
        K, V = dense_kv(kv, b)
        for h in range(8):
            assert np.array_equal(out[b, h], V[h // 4, 0])
            s = float(np.float32(kv.scale)) * (oracle.bf16_to_f64(kv.q[b, h]) @ K[h // 4, 0])
            assert lse[b, h] == pytest.approx(s, rel=1e-15, abs=1e-15)


def test_empty_context():
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    kv = make_paged(w, ctx=[0, 20])
    out, lse = kv.oracle_attn()
    assert not out[0].any() and np.isneginf(lse[0]).all()
    assert np.isfinite(lse[1]).all()


def test_one_hot_dominance():
    """One key aligned with q far beyond the others (>= 60 nats): output is
    that token's value to within e^-60 relative weight."""
    w = tiny_workload(Hq=1, Hkv=1, B=1)
    kv = make_paged(w, ctx=[48])
    q = np.zeros(128)
    q[:16] = 1.0
    kv.q[0, 0] = (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    # every key: small; token 29: block 0 = +64 * 2^(E-133) with E = 140 (value 64*2^7)
    kv.k_exp[:] = 100
    pid, slot = kv.page_table[0, 29 // 16], 29 % 16
    kv.k_mant[pid, 0, slot, :16] = 64
    kv.k_exp[pid, 0, slot, 0] = 140
    out, lse = kv.oracle_attn()
    K, V = dense_kv(kv, 0)
    s = float(np.float32(kv.scale)) * (K[0] @ q)
    assert s[29] - np.delete(s, 29).max() > 60
    np.testing.assert_allclose(out[0, 0], V[0, 29], rtol=1e-20, atol=np.abs(V).max() * 48 * np.exp(-60))


def test_gqa_identical_queries_in_group():
    w = tiny_workload(Hq=8, Hkv=2, B=1)
    kv = make_paged(w, ctx=[45])
    kv.q[0, 1:4] = kv.q[0, 0]
    kv.q[0, 5:8] = kv.q[0, 4]
    out, _ = kv.oracle_attn()
    for h in (1, 2, 3):
        assert np.array_equal(out[0, h], out[0, 0])
    for h in (5, 6, 7):
        assert np.array_equal(out[0, h], out[0, 4])
    # heads of different groups read different kv heads
    kv.q[0, 4] = kv.q[0, 0]
    out2, _ = kv.oracle_attn()
    assert not np.allclose(out2[0, 4], out2[0, 0])


def test_garbage_past_context_is_ignored():
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    a = make_paged(w, ctx=[21, 39], garbage_tail=False)
    b = make_paged(w, ctx=[21, 39], garbage_tail=True)
    assert not np.array_equal(a.k_mant, b.k_mant)
    oa, la = a.oracle_attn()
    ob, lb = b.oracle_attn()
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)


def test_page_placement_invariance():
    """Moving pages to other physical ids (and updating the table) changes
    nothing, bit for bit."""
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    kv = make_paged(w, ctx=[50, 64])
    out, lse = kv.oracle_attn()
    n = kv.k_mant.shape[0]
    perm = np.random.default_rng(3).permutation(n)          # new id of old page i
    inv = np.argsort(perm)
    for name in ("k_mant", "k_exp", "v_mant", "v_exp", "k_bf16", "v_bf16"):
        setattr(kv, name, np.ascontiguousarray(getattr(kv, name)[inv]))
    kv.page_table = perm[kv.page_table].astype(np.int32)
    out2, lse2 = kv.oracle_attn()
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_bf16_pages_with_decoded_values_match_bfp8_pages():
    w = wl.WORKLOADS[0]
    a = make_paged(w, bf16_fraction=0.0)
    b = make_paged(w, bf16_fraction=0.5)
    assert (b.page_table & wl.TAG_BF16).any()
    oa, la = a.oracle_attn()
    ob, lb = b.oracle_attn()
    assert np.array_equal(oa, ob) and np.array_equal(la, lb)


@pytest.mark.parametrize("seed", range(6))
def test_split_merge_invariance(seed):
    w = tiny_workload(Hq=8, Hkv=2, B=2)
    ctx = [77, 130]
    kv = make_paged(w, ctx=ctx)
    out, lse = kv.oracle_attn()
    r = np.random.default_rng(seed)
    for b in range(2):
        n = ctx[b]
        cuts = np.sort(r.integers(0, n + 1, size=r.integers(1, 9)))
        bounds = np.concatenate([[0], cuts, [n]]).astype(np.int32)   # may hold empty ranges
        h = int(r.integers(0, 8))
        o, l, pm, pl, po = oracle.decode_attn_split_one(
            kv.q, kv.k_mant, kv.k_exp, kv.v_mant, kv.v_exp, kv.k_bf16, kv.v_bf16,
            kv.page_table, kv.ctx, kv.num_kv_heads, kv.page_size, kv.scale, b, h, bounds)
        np.testing.assert_allclose(o, out[b, h], rtol=1e-12, atol=1e-13)
        assert l == pytest.approx(lse[b, h], rel=1e-13)
        # each non-empty partial is itself the attention over its range
        for s in range(len(bounds) - 1):
            if bounds[s + 1] == bounds[s]:
                assert pl[s] == 0 and np.isneginf(pm[s]) and not po[s].any()


def test_merge_closed_form():
    # two partials with known values: o = (l1 e^{m1} o1 + l2 e^{m2} o2) / (l1 e^{m1} + l2 e^{m2})
    m = np.array([1.5, -0.25])
    l = np.array([3.0, 7.0])
    o = np.array([[1.0, -2.0], [4.0, 0.5]])
    out, lse = oracle.merge_partials(m, l, o)
    w1, w2 = 3.0 * np.exp(1.5), 7.0 * np.exp(-0.25)
    np.testing.assert_allclose(out, (w1 * o[0] + w2 * o[1]) / (w1 + w2), rtol=1e-15)
    assert lse == pytest.approx(np.log(w1 + w2), rel=1e-15)
    # empty partials are skipped; all-empty gives zeros and -inf
    out, lse = oracle.merge_partials(np.array([-np.inf, 2.0]), np.array([0.0, 5.0]), o)
    np.testing.assert_allclose(out, o[1])
    assert lse == pytest.approx(2.0 + np.log(5.0))
    out, lse = oracle.merge_partials(np.array([-np.inf]), np.array([0.0]), o[:1])
    assert not out.any() and np.isneginf(lse)


# ------------------------------------------------------------- dequant pages

def test_dequant_pages_multi_pool():
    r = np.random.default_rng(11)
    Hkv, P, D = 2, 16, 128
    n_src, n_dst, n_pools = 9, 12, 3
    mant = r.integers(0, 256, size=(n_pools * n_src, Hkv, P, D), dtype=np.uint8)
    exps = r.integers(0, 256, size=(n_pools * n_src, Hkv, P, D // 16), dtype=np.uint8)
    dst = np.full((n_pools * n_dst, Hkv, P, D), 0xABCD, dtype=np.uint16)
    src_pages = np.array([4, 0, 8, 3], dtype=np.int32)
    dst_pages = np.array([11, 2, 7, 0], dtype=np.int32)
    oracle.dequant_pages(mant, exps, dst, src_pages, dst_pages, n_pools, n_src, n_dst, Hkv, D, P)
    # independent statement via numpy's float32 ldexp, per page
    for p in range(n_pools):
        for s, d in zip(src_pages, dst_pages):
            m = mant[p * n_src + s]
            e = np.repeat(exps[p * n_src + s], 16, axis=-1).astype(np.int32)
            sign = np.where(m & 0x80, np.float32(-1), np.float32(1))
            with np.errstate(over="ignore"):
                v = np.ldexp(sign * (m & 0x7F).astype(np.float32), e - 133).astype(np.float32)
            assert np.array_equal(dst[p * n_dst + d], (v.view(np.uint32) >> 16).astype(np.uint16))
        untouched = sorted(set(range(n_dst)) - set(dst_pages.tolist()))
        assert (dst[p * n_dst + np.array(untouched)] == 0xABCD).all()
