"""GPU parity of hma_bfp8_dequant_pages against the oracle: bit-exact.

Paper: BFP8 pages kept raw in HBM and rebuilt to BF16 on the decode GPU
(Sec. 3.3).  Every comparison here is bitwise on the uint16 BF16 buffers."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_29986_amd as hma
import workloads as wl
from gpu_util import dev, note
from oracle_fixtures import make_paged

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A5A


def _run(src_mant, src_exp, n_dst_pages_per_pool, src_pages, dst_pages, n_pools, src_stride,
         dst_stride, hkv, naive=False):
    dm = dev(src_mant)
    de = dev(src_exp)
    dst = torch.full((n_pools * n_dst_pages_per_pool if n_pools > 1 else n_dst_pages_per_pool,
                      hkv, 16, 128), SENTINEL, dtype=torch.int16, device="cuda")
    hma.bfp8_dequant_pages(dm, de, dst, dev(np.asarray(src_pages, np.int32)),
                           dev(np.asarray(dst_pages, np.int32)), n_pools=n_pools,
                           src_pool_stride_pages=src_stride, dst_pool_stride_pages=dst_stride,
                           num_kv_heads=hkv, naive=naive)
    torch.cuda.synchronize()
    return dst.cpu().numpy().view(np.uint16)


def _oracle(src_mant, src_exp, n_dst, src_pages, dst_pages, n_pools, src_stride, dst_stride, hkv):
    ref = np.full((n_pools * n_dst if n_pools > 1 else n_dst, hkv, 16, 128), SENTINEL, np.uint16)
    oracle.dequant_pages(src_mant, src_exp, ref, src_pages, dst_pages, n_pools, src_stride,
                         dst_stride, hkv, 128, 16)
    return ref


@pytest.mark.parametrize("naive", [False, True])
def test_dequant_exhaustive_table(naive):
    """All 65,536 (exponent, byte) pairs: 4096 blocks of 16 = 4 pages of 8 heads
    (also through the one-thread-per-element baseline)."""
    note(f"dequant: exhaustive (E, byte) table, naive={naive}")
    E = np.repeat(np.arange(256, dtype=np.uint8), 256)
    B = np.tile(np.arange(256, dtype=np.uint8), 256)
    mant = B.reshape(4, 8, 16, 128)
    exps = E.reshape(4096, 16)[:, 0].reshape(4, 8, 16, 8).copy()
    got = _run(mant, exps, 4, [0, 1, 2, 3], [0, 1, 2, 3], 1, 0, 0, 8, naive=naive)
    want = oracle.decode_blocks(mant, exps).reshape(got.shape)
    bad = np.argwhere(got != want)
    assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:4].tolist()}"


def test_dequant_smoke_workload_subset_of_pages():
    note("dequant: 4B-shaped smoke workload, K and V pools, permuted page subset")
    w = wl.WORKLOADS[0]
    kv = make_paged(w, with_bf16_pool=False)
    n = kv.k_mant.shape[0]
    r = np.random.default_rng(5)
    src = r.permutation(n)[: n // 3].astype(np.int32)
    dst = r.permutation(n)[: n // 3].astype(np.int32)
    for mant, ex in ((kv.k_mant, kv.k_exp), (kv.v_mant, kv.v_exp)):
        got = _run(mant, ex, n, src, dst, 1, 0, 0, w.num_kv_heads)
        want = _oracle(mant, ex, n, src, dst, 1, 0, 0, w.num_kv_heads)
        assert np.array_equal(got, want)
        untouched = np.setdiff1d(np.arange(n), dst)
        assert (got[untouched] == SENTINEL).all()


@pytest.mark.parametrize("naive", [False, True])
def test_dequant_multi_pool_strides_and_ragged_counts(naive):
    r = np.random.default_rng(9)
    for n_pools, n_src, n_dst, n_pairs, hkv in ((3, 7, 11, 5, 8), (1, 1, 1, 1, 1), (5, 9, 9, 9, 2),
                                                 (2, 33, 40, 31, 4)):
        note(f"dequant: pools={n_pools} src_stride={n_src} dst_stride={n_dst} pairs={n_pairs} hkv={hkv}")
        mant = r.integers(0, 256, size=(n_pools * n_src, hkv, 16, 128), dtype=np.uint8)
        ex = r.integers(0, 256, size=(n_pools * n_src, hkv, 16, 8), dtype=np.uint8)
        src = r.choice(n_src, size=n_pairs, replace=False).astype(np.int32)
        dst = r.choice(n_dst, size=n_pairs, replace=False).astype(np.int32)
        got = _run(mant, ex, n_dst, src, dst, n_pools, n_src, n_dst, hkv, naive=naive)
        want = _oracle(mant, ex, n_dst, src, dst, n_pools, n_src, n_dst, hkv)
        assert np.array_equal(got, want)


def test_dequant_zero_pages_is_noop():
    note("dequant: zero pairs")
    dst = torch.full((2, 8, 16, 128), SENTINEL, dtype=torch.int16, device="cuda")
    e = torch.zeros(0, dtype=torch.int32, device="cuda")
    m = torch.zeros(16, dtype=torch.uint8, device="cuda")
    hma.bfp8_dequant_pages(m, m, dst, e, e)
    torch.cuda.synchronize()
    assert (dst.cpu().numpy().view(np.uint16) == SENTINEL).all()


def test_dequant_full_request_qwen3_32b_8k_all_layers():
    """The standalone rebuild of one 8K-token Qwen3-32B request: 64 layers x
    (K, V) = 128 pools of 512 pages in one call, as the benchmark times it.
    Bitwise against the oracle on every pool."""
    note("dequant: Qwen3-32B 8K request, 128 pools x 512 pages, one launch")
    w = wl.WORKLOADS[3]
    n_pages, n_pools, hkv = 512, 128, w.num_kv_heads
    stride = n_pages + 3          # pools sit at a stride larger than the request
    g = torch.Generator(device="cuda")
    g.manual_seed(1003)
    dm = torch.randint(0, 256, (n_pools * stride, hkv, 16, 128), dtype=torch.uint8, device="cuda",
                       generator=g)
    de = torch.randint(100, 160, (n_pools * stride, hkv, 16, 8), dtype=torch.uint8, device="cuda",
                       generator=g)
    src = torch.randperm(stride, generator=g, device="cuda")[:n_pages].to(torch.int32)
    dst_ids = torch.randperm(n_pages, generator=g, device="cuda").to(torch.int32)
    dst = torch.empty((n_pools * n_pages, hkv, 16, 128), dtype=torch.int16, device="cuda")
    hma.bfp8_dequant_pages(dm, de, dst, src, dst_ids, n_pools=n_pools, src_pool_stride_pages=stride,
                           dst_pool_stride_pages=n_pages, num_kv_heads=hkv)
    torch.cuda.synchronize()
    mant = dm.cpu().numpy()
    ex = de.cpu().numpy()
    s = src.cpu().numpy()
    d = dst_ids.cpu().numpy()
    got = dst.cpu().numpy().view(np.uint16).reshape(n_pools, n_pages, hkv, 16, 128)
    want = np.empty((n_pages, hkv, 16, 128), np.uint16)
    for p in range(n_pools):
        oracle.dequant_pages(mant[p * stride:(p + 1) * stride], ex[p * stride:(p + 1) * stride],
                             want, s, d, 1, 0, 0, hkv, 128, 16)
        assert np.array_equal(got[p], want), f"pool {p}"
