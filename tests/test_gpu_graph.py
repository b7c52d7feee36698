"""The fused attention captured in a HIP graph: every replay equals the eager
call bit for bit (the split counters are left at zero by each launch and no
memset is recorded), on the 8-wave split schedule and on the 4-wave
page-balanced schedule, through the workspace entry and through the
no-allocation entry (whose callers are the ones that capture graphs).
Eager work (refilling the outputs with NaN) and synchronisation sit between
the replays."""
import numpy as np
import pytest
import torch

import paper_2606_29986_amd as hma
from gpu_util import DevKV, note
from oracle_fixtures import make_paged, tiny_workload

pytestmark = pytest.mark.gpu

CASES = {
    # 16 (sequence, KV head) pairs: one pass of 8-wave workgroups, two splits each
    "split_8wave": dict(Hq=32, Hkv=8, B=2, ctx=[3000, 2100]),
    # 320 pairs: the persistent 4-wave page-balanced schedule, empty sequences included
    "balanced_4wave": dict(Hq=32, Hkv=8, B=40, ctx=None),
}


@pytest.mark.parametrize("entry", ["workspace", "noalloc"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_graph_replays_equal_the_eager_call(case, entry):
    c = CASES[case]
    rng = np.random.default_rng(77)
    ctx = np.array(c["ctx"], np.int32) if c["ctx"] else rng.integers(0, 1500, c["B"]).astype(np.int32)
    if c["ctx"] is None:
        ctx[[3, 17]] = 0
    kv = make_paged(tiny_workload(Hq=c["Hq"], Hkv=c["Hkv"], B=c["B"], index=60), ctx=ctx, bf16_fraction=0.2)
    d = DevKV(kv)
    want, want_lse = d.attn()
    out = torch.empty_like(want)
    lse = torch.empty_like(want_lse)
    ws = hma.alloc_workspace(d.B, d.Hq, kv.num_kv_heads, d.max_ctx, 0)

    def call():
        args = (d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, d.pt, d.ctx, d.max_ctx, out)
        kw = dict(k_bf16=d.k_bf16, v_bf16=d.v_bf16, lse=lse, scale=kv.scale, num_kv_heads=kv.num_kv_heads)
        if entry == "noalloc":
            hma.decode_attn_bfp8_noalloc(*args, **kw)
        else:
            hma.decode_attn_bfp8(*args, workspace=ws, **kw)

    note(f"graph: {case} {entry}, eager call")
    call()                                   # first use on the device happens outside the capture
    torch.cuda.synchronize()
    assert torch.equal(out, want) and torch.equal(lse, want_lse)
    note(f"graph: {case} {entry}, capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for rep in range(4):
        out.fill_(0x7FC0)
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        note(f"graph: {case} {entry}, replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"replay {rep}: output differs"
        assert torch.equal(lse, want_lse), f"replay {rep}: log-sum-exp differs"
