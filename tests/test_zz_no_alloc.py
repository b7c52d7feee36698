"""hma_decode_attn_bfp8_noalloc against hma_decode_attn_bfp8 (same kernels):
bitwise-equal outputs and log-sum-exps through the C ABI, on two calls in a
row on one GPU -- the second with a smaller input, so it runs on the scratch
the first one left behind.  For callers that cannot allocate (header)."""
import numpy as np
import pytest
import torch

import paper_2606_29986_amd as hma
from gpu_util import DevKV, assert_attn_close, note
from oracle_fixtures import make_paged, tiny_workload

pytestmark = pytest.mark.gpu


def _both(kv, tps=0):
    d = DevKV(kv)
    want, want_lse = d.attn(tokens_per_split=tps)
    out = torch.full_like(want, 0x7FC0)
    lse = torch.full_like(want_lse, float("nan"))
    # the same pools as the workspace call (with BF16 pools the mixed kernel
    # runs, whose occupancy -- and so page-balanced chunking -- differs)
    hma.decode_attn_bfp8_noalloc(d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, d.pt, d.ctx, d.max_ctx, out,
                                 k_bf16=d.k_bf16, v_bf16=d.v_bf16, lse=lse, scale=kv.scale,
                                 num_kv_heads=kv.num_kv_heads, tokens_per_split=tps)
    torch.cuda.synchronize()
    return out, lse, want, want_lse


def test_noalloc_matches_workspace_entry_on_two_calls():
    rng = np.random.default_rng(123)
    # call 1: a ragged batch of 48 sequences (4-wave shape, page-balanced
    # pieces, partials and counters in the scratch)
    big = make_paged(tiny_workload(Hq=64, Hkv=8, B=48, index=50),
                     ctx=rng.integers(0, 1200, 48).astype(np.int32), bf16_fraction=0.25)
    assert hma.workspace_bytes(48, 64, 8, int(big.ctx.max())) > 0
    note("noalloc: call 1, B=48 ragged")
    out, lse, want, want_lse = _both(big)
    assert torch.equal(out, want) and torch.equal(lse, want_lse)
    ref, ref_lse = big.oracle_attn()
    assert_attn_close(out, lse, ref, ref_lse, what="noalloc call 1")
    # call 2: smaller (3 sequences, one workgroup per CU, two splits each) on
    # the scratch call 1 left behind
    small = make_paged(tiny_workload(Hq=64, Hkv=8, B=3, index=51), ctx=np.array([2500, 700, 4000], np.int32),
                       with_bf16_pool=False)
    assert hma.workspace_bytes(3, 64, 8, 4000) > 0
    note("noalloc: call 2, B=3")
    out2, lse2, want2, want_lse2 = _both(small)
    assert torch.equal(out2, want2) and torch.equal(lse2, want_lse2)
    # and an explicit split length on the same scratch
    note("noalloc: call 3, B=3, 256-token splits")
    out3, lse3, want3, want_lse3 = _both(small, tps=256)
    assert torch.equal(out3, want3) and torch.equal(lse3, want_lse3)

