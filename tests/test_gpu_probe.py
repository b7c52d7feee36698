"""The read probes (measurement only) read every byte they claim, exactly
once: the XOR of their sink words equals numpy's XOR of the same bytes as
32-bit words -- for the paged probe, the K/V mantissa and exponent tiles of
every page the attention would read, per KV head, on ragged batches with
empty sequences, partial last pages and both decompositions."""
import numpy as np
import pytest
import torch

import paper_2606_29986_amd as hma
from gpu_util import note

pytestmark = pytest.mark.gpu


def _xor_words(a: np.ndarray) -> int:
    return int(np.bitwise_xor.reduce(np.ascontiguousarray(a).view(np.uint32).ravel(), initial=np.uint32(0)))


def _expected_paged(km, kx, vm, vx, pt, ctx, max_ctx):
    acc = 0
    for b in range(pt.shape[0]):
        n = -(-min(max(int(ctx[b]), 0), max_ctx) // 16)
        ids = pt[b, :n] & hma.PAGE_ID_MASK
        for arr in (km, kx, vm, vx):
            acc ^= _xor_words(arr[ids])
    return acc


@pytest.mark.parametrize("hkv,hpw,pps,max_ctx", [(8, 1, 8, 700), (8, 8, 4, 700), (2, 2, 64, 700),
                                                 (4, 1, 1024, 640)])
def test_paged_read_probe_reads_each_attention_byte_once(hkv, hpw, pps, max_ctx):
    rng = np.random.default_rng(hkv * 1000 + hpw * 10 + pps)
    B = 9
    maxp = -(-max_ctx // 16)
    ctx = rng.integers(0, max_ctx + 1, B).astype(np.int32)
    ctx[0], ctx[1], ctx[2] = 0, max_ctx, 17
    ctx[3] = max_ctx + 500                               # clamped to max_ctx, as the attention does
    n_pool = B * maxp + 5
    pt = rng.permutation(n_pool)[:B * maxp].astype(np.int32).reshape(B, maxp)
    pt[4, :3] |= hma.PAGE_BF16                           # the tag is ignored by the probe
    km = rng.integers(0, 256, (n_pool, hkv, 16, 128), dtype=np.uint8)
    vm = rng.integers(0, 256, (n_pool, hkv, 16, 128), dtype=np.uint8)
    kx = rng.integers(0, 256, (n_pool, hkv, 16, 8), dtype=np.uint8)
    vx = rng.integers(0, 256, (n_pool, hkv, 16, 8), dtype=np.uint8)
    ns = -(-maxp // pps)
    dev = lambda a: torch.from_numpy(a).cuda()
    sink = torch.full((B * (hkv // hpw) * ns * 8,), -1, dtype=torch.int32, device="cuda")
    note(f"paged probe hkv={hkv} hpw={hpw} pps={pps} ns={ns}")
    hma.paged_read_probe(dev(km), dev(kx), dev(vm), dev(vx), dev(pt), dev(ctx), max_ctx, sink,
                         num_kv_heads=hkv, pages_per_split=pps, n_splits=ns, heads_per_workgroup=hpw)
    torch.cuda.synchronize()
    got = _xor_words(sink.cpu().numpy())
    assert got == _expected_paged(km, kx, vm, vx, pt, ctx, max_ctx)


@pytest.mark.parametrize("nbytes,nwg", [(16, 1), (4096 * 16 + 48, 7), (3 << 20, 2048)])
def test_stream_read_probe_reads_each_byte_once(nbytes, nwg):
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 256, nbytes, dtype=np.uint8)
    sink = torch.full((nwg * 4,), -1, dtype=torch.int32, device="cuda")
    note(f"stream probe {nbytes} B over {nwg} workgroups")
    hma.stream_read_probe(torch.from_numpy(host).cuda(), sink, nwg)
    torch.cuda.synchronize()
    assert _xor_words(sink.cpu().numpy()) == _xor_words(host)


def test_issue_probe_counts_cycles_on_every_wave():
    """The issue probe: every wave reports a positive cycle count, for every
    instruction kind; one step of a matrix instruction plus 8 adds takes at
    least as long as either alone and no longer than both in sequence (plus a
    margin for the loop)."""
    wps, iters = 2, 400
    n = 1024 * wps
    cyc = torch.zeros(n, dtype=torch.int64, device="cuda")
    sink = torch.zeros(n * 64, dtype=torch.int32, device="cuda")
    per = {}
    cases = [(0, 0, 1), (0, 8, 0), (0, 8, 1)] + [(k, 16, 0) for k in range(1, len(hma.ISSUE_KINDS))]
    for kind, valu, mfma in cases:
        note(f"issue probe kind={kind} valu={valu} mfma={mfma}")
        cyc.zero_()
        hma.issue_probe(kind, valu, mfma, wps, iters, cyc, sink)
        torch.cuda.synchronize()
        c = cyc.cpu().numpy()
        assert (c > 0).all(), (kind, valu, mfma)
        per[(kind, valu, mfma)] = float(np.median(c)) / (iters * 8)
    assert per[(0, 8, 1)] >= 0.9 * max(per[(0, 0, 1)], per[(0, 8, 0)])
    assert per[(0, 8, 1)] <= 1.1 * (per[(0, 0, 1)] + per[(0, 8, 0)]) + 4
