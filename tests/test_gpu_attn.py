"""GPU parity of hma_decode_attn_bfp8 against the float64 oracle.

Paper: decode attention reads raw BFP8 pages and rebuilds them inline in the
paged-attention kernel (Sec. 3.3, Fig. 2).  Bar: |gpu - oracle| <= 2e-3 +
1e-2 |oracle| elementwise on the BF16 output, plus exact-equality invariants
(single token, page placement, page format, GQA, split count, repeat runs)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_29986_amd as hma
import workloads as wl
from gpu_util import LSE_ATOL, LSE_RTOL, DevKV, assert_attn_close, bf16_bits_to_f64, dev, note
from oracle_fixtures import PagedKV, make_paged, tiny_workload

pytestmark = pytest.mark.gpu


def test_smoke_workload_matches_oracle():
    w = wl.WORKLOADS[0]
    note(f"attn: {w.name} full, auto split")
    kv = make_paged(w)
    ref, ref_lse = kv.oracle_attn()
    d = DevKV(kv)
    out, lse = d.attn()
    assert_attn_close(out, lse, ref, ref_lse, what=w.name)


@pytest.mark.parametrize("tps", [16, 32, 48, 96, 256, 0])
def test_ragged_with_garbage_tails_and_splits(tps):
    w = tiny_workload(Hq=32, Hkv=8, B=9, index=0)
    ctx = [0, 1, 15, 16, 17, 31, 33, 300, 511]
    note(f"attn: ragged ctx={ctx} tps={tps}")
    kv = make_paged(w, ctx=ctx, garbage_tail=True)
    ref, ref_lse = kv.oracle_attn()
    out, lse = DevKV(kv).attn(tokens_per_split=tps)
    assert_attn_close(out, lse, ref, ref_lse, what=f"ragged tps={tps}")
    got = bf16_bits_to_f64(out)
    assert not got[0].any() and np.isneginf(lse[0].cpu().numpy()).all()


@pytest.mark.parametrize("group", [1, 2, 4, 5, 8, 16])
def test_group_sizes(group):
    w = tiny_workload(Hq=2 * group, Hkv=2, B=3, index=1)
    ctx = [70, 129, 200]
    note(f"attn: group {group} ctx={ctx}")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    for tps in (64, 0):
        out, lse = DevKV(kv).attn(tokens_per_split=tps)
        assert_attn_close(out, lse, ref, ref_lse, what=f"g={group} tps={tps}")


def test_single_token_is_v0_exactly():
    """ctx = 1: the softmax weight is exactly 1, so the BF16 output must equal
    the decoded v_0 bit for bit (pins the in-register decode of V), and the
    lse equals the single score."""
    w = tiny_workload(Hq=16, Hkv=2, B=5, index=2)
    note("attn: single-token contexts")
    kv = make_paged(w, ctx=[1] * 5)
    # make the V rows of the first tokens cover extreme exponents, incl. BF16 subnormals
    for b, E in zip(range(5), (0, 3, 100, 127, 200)):
        pid = kv.page_table[b, 0]
        kv.v_exp[pid, :, 0, :] = E
    kv.k_bf16 = oracle.decode_blocks(kv.k_mant, kv.k_exp)
    kv.v_bf16 = oracle.decode_blocks(kv.v_mant, kv.v_exp)
    ref, ref_lse = kv.oracle_attn()
    out, lse = DevKV(kv).attn()
    got = out.cpu().numpy().view(np.uint16)
    for b in range(5):
        pid = kv.page_table[b, 0]
        for h in range(16):
            want = kv.v_bf16[pid, h // 8, 0]
            assert np.array_equal(got[b, h], want), (b, h)
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_page_placement_invariance_bitwise():
    w = tiny_workload(Hq=32, Hkv=8, B=4, index=3)
    ctx = [100, 257, 64, 480]
    note("attn: physical page placement")
    kv = make_paged(w, ctx=ctx)
    out1, lse1 = DevKV(kv).attn(tokens_per_split=64)
    n = kv.k_mant.shape[0]
    perm = np.random.default_rng(4).permutation(n)
    inv = np.argsort(perm)
    kv2 = PagedKV(kv.q, *(np.ascontiguousarray(a[inv]) for a in
                          (kv.k_mant, kv.k_exp, kv.v_mant, kv.v_exp, kv.k_bf16, kv.v_bf16)),
                  perm[kv.page_table].astype(np.int32), kv.ctx, kv.num_kv_heads, kv.page_size,
                  kv.scale)
    out2, lse2 = DevKV(kv2).attn(tokens_per_split=64)
    assert torch.equal(out1, out2) and torch.equal(lse1, lse2)


def test_bf16_pages_equal_bfp8_pages_bitwise():
    """Pages tagged BF16 holding the decoded values give the same output as
    the BFP8 pages, bit for bit; and after hma_bfp8_dequant_pages rebuilds
    every page into the BF16 pool, an all-BF16 page table matches too."""
    w = wl.WORKLOADS[0]
    note("attn: mixed BF16/BFP8 pages")
    a = make_paged(w, bf16_fraction=0.0)
    b = make_paged(w, bf16_fraction=0.5)
    out_a, lse_a = DevKV(a).attn(use_bf16_pools=False)
    out_b, lse_b = DevKV(b).attn()
    assert torch.equal(out_a, out_b) and torch.equal(lse_a, lse_b)
    # rebuild all pages on the GPU, then read everything from the BF16 pool
    d = DevKV(a)
    n = a.k_mant.shape[0]
    ids = dev(np.arange(n, dtype=np.int32))
    kb = torch.empty((n, 8, 16, 128), dtype=torch.int16, device="cuda")
    vb = torch.empty_like(kb)
    hma.bfp8_dequant_pages(d.k_mant, d.k_exp, kb, ids, ids, num_kv_heads=8)
    hma.bfp8_dequant_pages(d.v_mant, d.v_exp, vb, ids, ids, num_kv_heads=8)
    d.k_bf16, d.v_bf16 = kb, vb
    d.pt = dev(a.page_table | wl.TAG_BF16)
    out_c, lse_c = d.attn()
    assert torch.equal(out_a, out_c) and torch.equal(lse_a, lse_c)


def test_gqa_identical_queries_bitwise():
    w = tiny_workload(Hq=32, Hkv=4, B=2, index=4)
    note("attn: identical queries within a group")
    kv = make_paged(w, ctx=[200, 333])
    for j in range(4):
        kv.q[:, 8 * j + 1: 8 * j + 8] = kv.q[:, 8 * j: 8 * j + 1]
    out, _ = DevKV(kv).attn(tokens_per_split=64)
    o = out.cpu().numpy()
    for j in range(4):
        for h in range(8 * j + 1, 8 * j + 8):
            assert np.array_equal(o[:, h], o[:, 8 * j])
    assert not np.array_equal(o[:, 0], o[:, 8])


def test_split_count_invariance_and_determinism():
    w = tiny_workload(Hq=64, Hkv=8, B=3, index=5)
    ctx = [1000, 777, 1500]
    note(f"attn: split invariance ctx={ctx}")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    d = DevKV(kv)
    first = None
    for tps in (16, 32, 128, 512, 1024, 1504):
        out, lse = d.attn(tokens_per_split=tps)
        assert_attn_close(out, lse, ref, ref_lse, what=f"tps={tps}")
        again, lse2 = d.attn(tokens_per_split=tps)
        assert torch.equal(out, again) and torch.equal(lse, lse2), f"tps={tps} not deterministic"
        first = out if first is None else first


def test_all_equal_keys_uniform_average():
    w = tiny_workload(Hq=8, Hkv=1, B=1, index=6)
    note("attn: all keys equal")
    kv = make_paged(w, ctx=[300])
    kv.k_mant[:] = kv.k_mant[kv.page_table[0, 0], 0, 0]
    kv.k_exp[:] = kv.k_exp[kv.page_table[0, 0], 0, 0]
    ref, ref_lse = kv.oracle_attn()
    vmean = np.stack([oracle.bf16_to_f64(oracle.decode_blocks(
        kv.v_mant[kv.page_table[0, t // 16], 0, t % 16], kv.v_exp[kv.page_table[0, t // 16], 0, t % 16]))
        for t in range(300)]).mean(axis=0)
    np.testing.assert_allclose(ref[0], np.broadcast_to(vmean, ref[0].shape), atol=1e-12)
    out, lse = DevKV(kv).attn(tokens_per_split=64)
    assert_attn_close(out, lse, ref, ref_lse, what="uniform")


# ---------------------------------------------------------- full-size cases

def _sample_seqs(w, n_seq, seed):
    r = np.random.default_rng(seed)
    return np.sort(r.choice(w.batch, size=min(n_seq, w.batch), replace=False))


def _oracle_rows(kv, seqs):
    """Oracle on a subset of sequences (the oracle's cost grows with context)."""
    sub = PagedKV(np.ascontiguousarray(kv.q[seqs]), kv.k_mant, kv.k_exp, kv.v_mant, kv.v_exp,
                  kv.k_bf16, kv.v_bf16, np.ascontiguousarray(kv.page_table[seqs]),
                  np.ascontiguousarray(kv.ctx[seqs]), kv.num_kv_heads, kv.page_size, kv.scale)
    return sub.oracle_attn()


@pytest.mark.parametrize("index,n_seq", [(1, 6), (2, 10), (3, 4), (4, 12)])
def test_full_size_workload_sampled(index, n_seq):
    """One layer of each evaluated workload at its full size, launched exactly
    as the benchmark launches it (automatic split); the oracle checks a
    seeded sample of whole sequences (every head, every channel).  For the
    200-sequence trace mix only the sampled sequences' pages carry drawn
    values (the rest are zeros) to keep the host-side draw short."""
    w = wl.WORKLOADS[index]
    note(f"attn: full-size {w.name}")
    seqs = _sample_seqs(w, n_seq, seed=index)
    kv = make_paged(w, bf16_fraction=w.bf16_page_fraction,
                    with_bf16_pool=w.bf16_page_fraction > 0,
                    value_seqs=seqs if index == 4 else None)
    out, lse = DevKV(kv).attn()
    ref, ref_lse = _oracle_rows(kv, seqs)
    err = assert_attn_close(out, lse, ref, ref_lse, rows=seqs, what=w.name)
    note(f"attn: {w.name} max abs err {err:.3g} on {len(seqs)} sequences")


def test_trace_mix_pure_bfp8_one_range_per_wave():
    """The 200-sequence trace mix with BFP8 pages only: the pure-BFP8 kernel
    under the page-balanced schedule at its one-range-per-wave granularity
    (taken for ranges of at least 64 pages; here T / (64 workgroups per KV
    head x 4 waves) pages each), where every piece is attended and published
    by one wave and the last wave to arrive folds.  Sampled sequences against
    the oracle, and a repeat call bitwise equal (the fold runs in piece order
    whichever wave arrives last)."""
    w = wl.WORKLOADS[4]
    seqs = _sample_seqs(w, 8, seed=40)
    kv = make_paged(w, bf16_fraction=0.0, with_bf16_pool=False, value_seqs=seqs)
    T = int(wl.pages_per_seq(kv.ctx, w.page_size).sum())
    assert -(-T // (512 // w.num_kv_heads * 4)) >= 64
    note(f"attn: trace mix, BFP8 only, {T} pages per KV head")
    d = DevKV(kv)
    out, lse = d.attn()
    out2, lse2 = d.attn()
    assert torch.equal(out, out2) and torch.equal(lse, lse2)
    ref, ref_lse = _oracle_rows(kv, seqs)
    err = assert_attn_close(out, lse, ref, ref_lse, rows=seqs, what="trace mix BFP8")
    note(f"attn: trace mix BFP8 max abs err {err:.3g} on {len(seqs)} sequences")


def test_single_long_sequence_many_splits():
    """One 32K-token sequence (Qwen3-32B heads): the automatic split gives 32
    splits of 1024 tokens on 256 one-per-CU workgroups, so the last workgroup
    of each KV head folds 32 partials."""
    w = tiny_workload(Hq=64, Hkv=8, B=1, index=6)
    ctx = [32768]
    assert hma.tokens_per_split(1, 64, 8, 32768) == 1024
    note(f"attn: single sequence ctx={ctx}")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    out, lse = DevKV(kv).attn()
    assert_attn_close(out, lse, ref, ref_lse, what="32K single sequence")


def _attn_with_bound(d, max_ctx, tps):
    """d.attn with a looser host bound on the context lengths (page table
    padded to match): the bound sizes the grid and the workspace, not the
    result."""
    kv = d.kv
    cols = (max_ctx + 15) // 16
    pt = np.zeros((kv.page_table.shape[0], max(cols, kv.page_table.shape[1])), np.int32)
    pt[:, :kv.page_table.shape[1]] = kv.page_table
    out = torch.full((d.B, d.Hq, d.D), 0x7FC0, dtype=torch.int16, device="cuda")
    lse = torch.full((d.B, d.Hq), float("nan"), dtype=torch.float32, device="cuda")
    ws = hma.alloc_workspace(d.B, d.Hq, kv.num_kv_heads, max_ctx, tps)
    hma.decode_attn_bfp8(d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, dev(pt), d.ctx, max_ctx, out, lse=lse,
                         scale=kv.scale, num_kv_heads=kv.num_kv_heads, tokens_per_split=tps, workspace=ws)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("lengths", ["ragged", "equal", "equal_whole"])
def test_length_aware_schedule_many_sequences_and_levels(lengths):
    """A batch the host sees only through its longest length: 70 sequences
    (more than one wave's worth) from empty to 4500 tokens, split every 32
    tokens (141 split levels); also 70 equal lengths (the schedule's
    table-free case), with and without a shorter last split.  Against the
    oracle, and bitwise equal to the direct one-workgroup-per-split schedule
    (reached through a looser length bound that gives 1024 splits per
    sequence)."""
    rng = np.random.default_rng(70)
    w = tiny_workload(Hq=16, Hkv=2, B=70, index=7)
    if lengths == "ragged":
        ctx = rng.integers(0, 300, 70).astype(np.int32)
        ctx[[3, 40]] = [4500, 2100]
        ctx[[5, 6, 7]] = [0, 1, 32]
    else:
        ctx = np.full(70, 300 if lengths == "equal" else 320, np.int32)
    tps = 32
    assert hma.tokens_per_split(70, 16, 2, int(ctx.max())) != tps        # a forced split length
    note(f"attn: length-aware schedule, B=70, {lengths}, max ctx {ctx.max()}, tps {tps}")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    d = DevKV(kv)
    out, lse = d.attn(tokens_per_split=tps)
    assert_attn_close(out, lse, ref, ref_lse, what="length-aware schedule")
    note("attn: direct schedule through a looser bound")
    out_d, lse_d = _attn_with_bound(d, 1024 * tps, tps)
    assert torch.equal(out, out_d) and torch.equal(lse, lse_d)


def test_batch_beyond_the_schedule_tables():
    """1030 sequences (more than the length-aware schedule's tables hold):
    the direct schedule runs; against the oracle."""
    rng = np.random.default_rng(1030)
    w = tiny_workload(Hq=8, Hkv=1, B=1030, index=8)
    ctx = rng.integers(0, 60, 1030).astype(np.int32)
    note("attn: batch of 1030 sequences")
    kv = make_paged(w, ctx=ctx)
    ref, ref_lse = kv.oracle_attn()
    for tps in (0, 16):
        out, lse = DevKV(kv).attn(tokens_per_split=tps)
        assert_attn_close(out, lse, ref, ref_lse, what=f"B=1030 tps={tps}")


@pytest.mark.parametrize("tps", [0, 16])
def test_lse_is_optional(tps):
    """lse = NULL changes nothing else: same output bits, with one split or
    several (both workgroup shapes)."""
    w = tiny_workload(Hq=32, Hkv=8, B=6, index=9)
    ctx = [1, 40, 300, 511, 16, 250]
    note(f"attn: optional lse, tps={tps}")
    kv = make_paged(w, ctx=ctx)
    d = DevKV(kv)
    out_a, _ = d.attn(tokens_per_split=tps)
    out_b, lse_b = d.attn(tokens_per_split=tps, with_lse=False)
    assert lse_b is None
    assert torch.equal(out_a, out_b)


def test_concurrent_calls_on_two_streams():
    """Calls that share no workspace may run concurrently on different
    streams: two batches (one per workgroup shape) enqueued on two streams
    without synchronisation in between give the bits of the same calls run
    alone."""
    note("attn: two streams")
    kv1 = make_paged(tiny_workload(Hq=64, Hkv=8, B=2, index=10), ctx=[3000, 4096])
    kv2 = make_paged(tiny_workload(Hq=16, Hkv=2, B=40, index=11),
                     ctx=np.random.default_rng(11).integers(1, 700, 40).astype(np.int32))
    d1, d2 = DevKV(kv1), DevKV(kv2)
    want1, lse1 = d1.attn()
    want2, lse2 = d2.attn(tokens_per_split=32)
    outs = []
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for d, s, tps in ((d1, streams[0], 0), (d2, streams[1], 32)):
        B, Hq = d.B, d.Hq
        out = torch.full((B, Hq, 128), 0x7FC0, dtype=torch.int16, device="cuda")
        lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device="cuda")
        ws = hma.alloc_workspace(B, Hq, d.kv.num_kv_heads, d.max_ctx, tps)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            for _ in range(3):
                hma.decode_attn_bfp8(d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, d.pt, d.ctx, d.max_ctx, out,
                                     lse=lse, scale=d.kv.scale, num_kv_heads=d.kv.num_kv_heads,
                                     tokens_per_split=tps, workspace=ws, stream=s)
        outs.append((out, lse))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], want1) and torch.equal(outs[0][1], lse1)
    assert torch.equal(outs[1][0], want2) and torch.equal(outs[1][1], lse2)


@pytest.mark.parametrize("tps", [0, 16])
def test_lengths_outside_the_bound_are_clamped(tps):
    """A length above max_context_len is read as max_context_len and a
    negative one as 0 (zero output, lse = -inf), on both workgroup shapes."""
    w = tiny_workload(Hq=16, Hkv=2, B=4, index=12)
    note(f"attn: lengths outside the bound, tps={tps}")
    kv_in = make_paged(w, ctx=[300, 640, 5, 640])
    kv_out = make_paged(w, ctx=[300, 640, 5, 640])
    want, want_lse = DevKV(kv_in).attn(tokens_per_split=tps)
    d = DevKV(kv_out)
    d.ctx = dev(np.array([300, 5000, -7, 640], np.int32))
    d.max_ctx = 640
    got, got_lse = d.attn(tokens_per_split=tps)
    for b in (0, 1, 3):
        assert torch.equal(got[b], want[b]) and torch.equal(got_lse[b], want_lse[b])
    assert not bf16_bits_to_f64(got[2]).any()
    assert np.isneginf(got_lse[2].cpu().numpy()).all()


@pytest.mark.parametrize("seed", range(6))
def test_random_batches(seed):
    """Random shapes against the oracle: batch 1..150, KV heads 1..8, group
    1..16, lengths 0..600 (some empty), a random split length or the
    library's; covers both workgroup shapes, both schedules and both
    kernel variants."""
    rng = np.random.default_rng(4000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.integers(1, 17))
    B = int(rng.integers(1, 151))
    w = tiny_workload(Hq=hkv * g, Hkv=hkv, B=B, index=20 + seed)
    ctx = rng.integers(0, 601, B).astype(np.int32)
    ctx[rng.random(B) < 0.1] = 0
    tps = int(rng.choice([0, 16, 48, 128, 512]))
    frac = float(rng.choice([0.0, 0.5]))
    note(f"attn: random batch seed={seed} B={B} hkv={hkv} g={g} tps={tps} bf16={frac} max ctx {ctx.max()}")
    kv = make_paged(w, ctx=ctx, bf16_fraction=frac)
    ref, ref_lse = kv.oracle_attn()
    out, lse = DevKV(kv).attn(tokens_per_split=tps)
    assert_attn_close(out, lse, ref, ref_lse, what=f"random batch {seed}")


@pytest.mark.parametrize("case", ["short_many", "mixed_lengths", "bf16_pages"])
def test_page_balanced_schedule_pieces_span_sequences(case):
    """The automatic split with more workgroups than one per CU cuts each KV
    head's concatenated page list into equal chunks on the device; a chunk
    spanning several sequences yields one piece per sequence and the pieces
    of a (sequence, KV head) are folded in chunk order.  Many short sequences
    (chunks of the 16-page minimum cover several of them), empty ones,
    ragged last pages, one sequence longer than a chunk, and pages of both
    formats: against the oracle, and bit-identical on a repeat."""
    rng = np.random.default_rng({"short_many": 71, "mixed_lengths": 72, "bf16_pages": 73}[case])
    if case == "short_many":
        B, hkv, g = 300, 8, 4
        ctx = rng.integers(0, 60, B).astype(np.int32)
    else:
        B, hkv, g = 90, 8, 8 if case == "mixed_lengths" else 5
        ctx = rng.integers(1, 400, B).astype(np.int32)
        ctx[[2, 50]] = [3000, 1500]
    ctx[[0, 7, 8]] = [0, 0, 1]
    w = tiny_workload(Hq=hkv * g, Hkv=hkv, B=B, index=30 + len(case))
    assert B * hkv > 256      # the 4-wave shape, so the page-balanced schedule
    frac = 0.5 if case == "bf16_pages" else 0.0
    note(f"attn: page-balanced schedule, {case}: B={B} hkv={hkv} g={g} max ctx {ctx.max()} total {ctx.sum()}")
    kv = make_paged(w, ctx=ctx, bf16_fraction=frac)
    ref, ref_lse = kv.oracle_attn()
    d = DevKV(kv)
    out, lse = d.attn()
    assert_attn_close(out, lse, ref, ref_lse, what=f"page-balanced {case}")
    again, lse2 = d.attn()
    assert torch.equal(out, again) and torch.equal(lse, lse2)


def test_workspace_reuse_contract():
    """One workspace serves repeated calls of one shape without a new zero
    fill: every call leaves its split-merge counters at zero.  Outputs are
    re-poisoned with NaN between the calls, so a missed merge would show.  A
    call with a larger batch * num_kv_heads gets the buffer zero-filled again
    first, as the header requires; a smaller one reuses it as it is."""
    rng = np.random.default_rng(77)
    big = make_paged(tiny_workload(Hq=64, Hkv=8, B=40, index=40),
                     ctx=rng.integers(1, 900, 40).astype(np.int32))
    small = make_paged(tiny_workload(Hq=64, Hkv=8, B=20, index=41),
                       ctx=rng.integers(1, 900, 20).astype(np.int32))
    nbytes = max(hma.workspace_bytes(40, 64, 8, int(big.ctx.max())),
                 hma.workspace_bytes(20, 64, 8, int(small.ctx.max())))
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")

    def run(kv):
        d = DevKV(kv)
        max_ctx = d.max_ctx
        out = torch.full((d.B, d.Hq, 128), 0x7FC0, dtype=torch.int16, device="cuda")
        lse = torch.full((d.B, d.Hq), float("nan"), dtype=torch.float32, device="cuda")
        hma.decode_attn_bfp8(d.q, d.k_mant, d.k_exp, d.v_mant, d.v_exp, d.pt, d.ctx, max_ctx, out, lse=lse,
                             scale=kv.scale, num_kv_heads=8, workspace=ws)
        torch.cuda.synchronize()
        return out, lse

    ref_s, lse_s = small.oracle_attn()
    ref_b, lse_b = big.oracle_attn()
    note("attn: workspace reuse, same shape twice")
    o1, l1 = run(small)
    o2, l2 = run(small)
    assert_attn_close(o2, l2, ref_s, lse_s, what="second call on a reused workspace")
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    note("attn: workspace reuse, larger batch after a zero fill")
    ws.zero_()
    o3, l3 = run(big)
    assert_attn_close(o3, l3, ref_b, lse_b, what="larger batch, zero-filled workspace")
    note("attn: workspace reuse, smaller batch without a zero fill")
    o4, l4 = run(small)
    assert torch.equal(o4, o1) and torch.equal(l4, l1)
