"""GPU parity of hma_decode_attn_bfp8_valu (the fused BFP8 decode attention
with both products on the vector ALU) against the float64 oracle.

Paper: decode attention reads raw BFP8 pages and rebuilds them inline in the
paged-attention kernel (Sec. 3.3, Fig. 2).  Same bar as the matrix-core
kernel: |gpu - oracle| <= 2e-3 + 1e-2 |oracle| elementwise on the BF16
output, the lse within its float32 bound, plus exact cases (single token,
repeat runs).  The workspace is filled with garbage before each call: every
slot is written before it is read."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_29986_amd as hma
import workloads as wl
from gpu_util import LSE_ATOL, LSE_RTOL, DevKV, assert_attn_close, note
from oracle_fixtures import PagedKV, make_paged, tiny_workload

pytestmark = pytest.mark.gpu


def valu_attn(d: DevKV, tokens_per_split=0, with_lse=True):
    B, Hq, D = d.B, d.Hq, d.D
    out = torch.full((B, Hq, D), 0x7FC0, dtype=torch.int16, device="cuda")
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device="cuda") if with_lse else None
    n = hma.valu_workspace_bytes(B, Hq, d.kv.num_kv_heads, d.max_ctx, tokens_per_split)
    ws = torch.full((max(n, 256),), 0xA5, dtype=torch.uint8, device="cuda")
    hma.decode_attn_bfp8_valu(d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, d.pt, d.ctx, d.max_ctx, out, ws,
                              lse=lse, scale=d.kv.scale, num_kv_heads=d.kv.num_kv_heads,
                              tokens_per_split=tokens_per_split)
    torch.cuda.synchronize()
    return out, lse


def test_smoke_workload_matches_oracle():
    w = wl.WORKLOADS[0]
    note(f"valu attn: {w.name}, auto split")
    kv = make_paged(w)
    ref, ref_lse = kv.oracle_attn()
    out, lse = valu_attn(DevKV(kv))
    assert_attn_close(out, lse, ref, ref_lse, what=w.name)


@pytest.mark.parametrize("tps", [16, 48, 256, 0])
def test_ragged_with_garbage_tails_and_splits(tps):
    w = tiny_workload(Hq=32, Hkv=8, B=9, index=0)
    ctx = [0, 1, 15, 16, 17, 31, 33, 300, 511]
    note(f"valu attn: ragged ctx={ctx} tps={tps}")
    kv = make_paged(w, ctx=ctx, garbage_tail=True)
    ref, ref_lse = kv.oracle_attn()
    out, lse = valu_attn(DevKV(kv), tokens_per_split=tps)
    assert_attn_close(out, lse, ref, ref_lse, what=f"ragged tps={tps}")
    assert not out[0].cpu().numpy().any() and np.isneginf(lse[0].cpu().numpy()).all()


@pytest.mark.parametrize("group", [1, 2, 3, 4, 5, 8])
def test_group_sizes(group):
    w = tiny_workload(Hq=2 * group, Hkv=2, B=3, index=1)
    ctx = [70, 129, 200]
    note(f"valu attn: group {group} ctx={ctx}")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    for tps in (64, 0):
        out, lse = valu_attn(DevKV(kv), tokens_per_split=tps)
        assert_attn_close(out, lse, ref, ref_lse, what=f"g={group} tps={tps}")


def test_single_token_is_v0_exactly():
    """ctx = 1: the weight is exactly 1, so the output is the decoded v_0 bit
    for bit, on both decode routes (E = 0 and 3 take the general route)."""
    w = tiny_workload(Hq=16, Hkv=2, B=5, index=2)
    note("valu attn: single-token contexts")
    kv = make_paged(w, ctx=[1] * 5)
    for b, E in zip(range(5), (0, 3, 100, 127, 200)):
        kv.v_exp[kv.page_table[b, 0], :, 0, :] = E
    ref, ref_lse = kv.oracle_attn()
    out, lse = valu_attn(DevKV(kv))
    got = out.cpu().numpy().view(np.uint16)
    vdec = oracle.decode_blocks(kv.v_mant, kv.v_exp)
    for b in range(5):
        pid = kv.page_table[b, 0]
        for h in range(16):
            assert np.array_equal(got[b, h], vdec[pid, h // 8, 0]), (b, h)
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_repeat_runs_are_bitwise_equal_and_lse_optional():
    w = tiny_workload(Hq=32, Hkv=8, B=4, index=4)
    kv = make_paged(w, ctx=[100, 700, 1, 1500])
    note("valu attn: repeat runs")
    d = DevKV(kv)
    a, la = valu_attn(d, tokens_per_split=128)
    b, lb = valu_attn(d, tokens_per_split=128)
    c, _ = valu_attn(d, tokens_per_split=128, with_lse=False)
    assert torch.equal(a, b) and torch.equal(la, lb) and torch.equal(a, c)


def _sample_seqs(w, n_seq, seed):
    r = np.random.default_rng(seed)
    return np.sort(r.choice(w.batch, size=min(n_seq, w.batch), replace=False))


@pytest.mark.parametrize("index,n_seq", [(1, 4), (2, 6), (3, 3)])
def test_full_size_workload_sampled(index, n_seq):
    """One layer of an evaluated workload at full size with the automatic
    ranges (as the benchmark launches it); the oracle checks a seeded sample
    of whole sequences."""
    w = wl.WORKLOADS[index]
    note(f"valu attn: full-size {w.name}")
    seqs = _sample_seqs(w, n_seq, seed=100 + index)
    kv = make_paged(w)
    out, lse = valu_attn(DevKV(kv))
    sub = PagedKV(np.ascontiguousarray(kv.q[seqs]), kv.k_mant, kv.k_exp, kv.v_mant, kv.v_exp, None, None,
                  np.ascontiguousarray(kv.page_table[seqs]), np.ascontiguousarray(kv.ctx[seqs]),
                  kv.num_kv_heads, kv.page_size, kv.scale)
    ref, ref_lse = sub.oracle_attn()
    err = assert_attn_close(out, lse, ref, ref_lse, rows=seqs, what=w.name)
    note(f"valu attn: {w.name} max abs err {err:.3g} on {len(seqs)} sequences")
