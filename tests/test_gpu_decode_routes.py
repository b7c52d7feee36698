"""Exhaustive check of the fused kernel's in-register BFP8 decode, both routes.

The attention kernel decodes a page either with a packed route (every block
exponent of the page in [7, 133]) or with the general route (v_ldexp_f32,
every exponent).  Single-token contexts make the decode observable exactly:

* V: with ctx = 1 the softmax weight is exactly 1, so the BF16 output row is
  the decoded v_0 bit for bit (up to the sign of zero: the accumulation starts
  from +0).  Every exponent 0..254 is combined with all 256 element bytes.
* K: with ctx = 1 the log-sum-exp is the single score; a one-hot query with a
  power-of-two weight turns it into scale * q * k_0[c] computed exactly up to
  the float32 roundings of the scale, so each channel's decoded value is read
  back through the lse.

  Every exponent 0..254 with all 256 bytes; for exponents above 252 the query
  weight is clamped to 2^-126 (a BF16 subnormal query would be flushed by the
  matrix cores), which keeps the score a small exact multiple of k.

Reference: the oracle's decode (Sec. 3.3 reading of the format).  Exponent 255
with m >= 64 (an infinity) is outside the attention call's contract (header:
non-finite inputs give non-finite outputs); test_infinite_elements_give_non_finite_results
checks exactly that documented behaviour, and exponent 255 with m < 64 (finite)
is decoded exactly like the rest.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DevKV, note
from oracle_fixtures import PagedKV

pytestmark = pytest.mark.gpu

HKV, P, D = 8, 16, 128
SCALE = 1.0 / np.sqrt(128.0)
# 32 sequences x 8 KV heads = 256 workgroups (one per CU: the 8-wave kernel);
# 64 sequences = 512 workgroups (the 4-wave kernel)
BATCHES = [32, 64]


def _kv(rng, B, Hq, sweep, half):
    """One page per sequence (ids permuted).  Token 0 of (sequence b, head j),
    t = 8 b + j, gets bytes 128 * ((t // 256 + half) % 2) .. + 127 and every
    block of that (page, head) tile of the swept stream gets exponent
    min(t % 256, cap); the other stream has exponent 127 and random bytes."""
    ids = rng.permutation(B).astype(np.int32)
    k_mant = rng.integers(0, 256, (B, HKV, P, D), dtype=np.uint8)
    v_mant = rng.integers(0, 256, (B, HKV, P, D), dtype=np.uint8)
    k_exp = np.full((B, HKV, P, D // 16), 127, np.uint8)
    v_exp = np.full((B, HKV, P, D // 16), 127, np.uint8)
    mant, ex, cap = (v_mant, v_exp, 254) if sweep == "v" else (k_mant, k_exp, 254)
    t = np.arange(B * HKV)
    exps = np.minimum(t % 256, cap)
    for b in range(B):
        for j in range(HKV):
            tt = 8 * b + j
            mant[ids[b], j, 0, :] = (128 * ((tt // 256 + half) % 2) + np.arange(D)) % 256
            ex[ids[b], j, :, :] = exps[tt]
    q = np.zeros((B, Hq, D), np.uint16)
    kv = PagedKV(q, k_mant, k_exp, v_mant, v_exp,
                 oracle.decode_blocks(k_mant, k_exp), oracle.decode_blocks(v_mant, v_exp),
                 ids.reshape(B, 1), np.ones(B, np.int32), HKV, P, SCALE)
    return kv, ids, exps


@pytest.mark.parametrize("B", BATCHES)
@pytest.mark.parametrize("mixed_kernel", [False, True])
def test_v_decode_exhaustive_through_single_token_output(mixed_kernel, B):
    for half in (0, 1):
        note(f"attn decode routes: V exhaustive, B={B} half={half}, mixed-format kernel={mixed_kernel}")
        rng = np.random.default_rng(11 + half)
        kv, ids, exps = _kv(rng, B, HKV, "v", half)
        kv.q[:] = 0x3F80                          # q = 1.0: scores are finite and irrelevant
        out, _ = DevKV(kv).attn(use_bf16_pools=mixed_kernel)
        got = out.cpu().numpy().view(np.uint16).copy()
        want = kv.v_bf16[ids, :, 0, :].copy()     # [B][Hkv][D] (g = 1: head j reads KV head j)
        # a weighted sum that starts from +0 turns -0 into +0: compare zeros unsigned
        got[got == 0x8000] = 0
        want[want == 0x8000] = 0
        bad = np.argwhere(got != want)
        assert bad.size == 0, (f"half {half}: {len(bad)} mismatches; first (b, h, c) {bad[:4].tolist()}, "
                               f"exponents {[int(exps[8 * b + h]) for b, h, _ in bad[:4]]}")


@pytest.mark.parametrize("B", BATCHES)
@pytest.mark.parametrize("mixed_kernel", [False, True])
def test_k_decode_exhaustive_through_single_token_lse(mixed_kernel, B):
    g = 16
    for half in (0, 1):
        note(f"attn decode routes: K exhaustive, B={B} half={half}, mixed-format kernel={mixed_kernel}")
        rng = np.random.default_rng(21 + half)
        kv, ids, exps = _kv(rng, B, HKV * g, "k", half)
        k_dec = oracle.bf16_to_f64(kv.k_bf16[ids, :, 0, :])      # [B][Hkv][D]
        d = DevKV(kv)
        for phase in range(8):
            # head h of group j probes channel 8 (h % 16) + phase with weight 2^(126 - E)
            q = np.zeros((B, HKV * g, D), np.uint16)
            chan = 8 * np.arange(g) + phase
            ref = np.zeros((B, HKV * g))
            for b in range(B):
                for j in range(HKV):
                    e = max(126 - int(exps[8 * b + j]), -126)     # a normal BF16 weight
                    q[b, j * g + np.arange(g), chan] = (e + 127) << 7
                    ref[b, j * g: (j + 1) * g] = float(np.float32(SCALE)) * 2.0 ** e * k_dec[b, j, chan]
            d.q = torch.from_numpy(q.view(np.int16)).cuda()
            _, lse = d.attn(use_bf16_pools=mixed_kernel)
            got = lse.cpu().numpy().astype(np.float64)
            err = np.abs(got - ref)
            bad = np.argwhere(err > 1e-6 * np.abs(ref))
            assert bad.size == 0, (f"half {half} phase {phase}: {len(bad)} mismatches; first (b, h) "
                                   f"{bad[:4].tolist()} got {got[tuple(bad[0])]} ref {ref[tuple(bad[0])]}")


@pytest.mark.parametrize("stream", ["k", "v"])
def test_infinite_elements_give_non_finite_results(stream):
    """Outside the contract, as documented in the header: one infinite element
    (E = 255, m >= 64) in a sequence's K or V makes the results of the query
    heads that read it non-finite (NaN or +-Inf) -- never a finite value that
    hides it -- and leaves every other (sequence, KV head) exact.  Single-token
    contexts; E = 255 with m < 64 is finite and decoded exactly."""
    rng = np.random.default_rng(91)
    B, g = 4, 2
    kv, ids, _ = _kv(rng, B, HKV * g, "v", 0)
    kv.q[:] = 0x3F80
    mant, ex = (kv.k_mant, kv.k_exp) if stream == "k" else (kv.v_mant, kv.v_exp)
    pid = ids[1]
    ex[pid, 3, 0, 2] = 255          # sequence 1, KV head 3, block 2 of token 0
    mant[pid, 3, 0, 32:48] = 5      # finite magnitudes (m < 64) ...
    mant[pid, 3, 0, 40] = 0x40      # ... and one infinity: m = 64, sign +
    kv.k_bf16 = oracle.decode_blocks(kv.k_mant, kv.k_exp)
    kv.v_bf16 = oracle.decode_blocks(kv.v_mant, kv.v_exp)
    note(f"attn: an infinite {stream} element, outside the contract")
    out, lse = DevKV(kv).attn(use_bf16_pools=False)
    got = oracle.bf16_to_f64(out.cpu().numpy().view(np.uint16))      # [B][Hq][D]
    heads = [3 * g + r for r in range(g)]
    if stream == "v":
        assert not np.isfinite(got[1, heads, 40]).any()
        rest = np.ones_like(got, dtype=bool)
        rest[1, heads, 40] = False
        assert np.isfinite(got[rest]).all()
    else:
        assert not np.isfinite(lse.cpu().numpy()[1, heads]).any() or not np.isfinite(got[1, heads]).all()
        other = [h for h in range(HKV * g) if h not in heads]
        assert np.isfinite(got[1, other]).all() and np.isfinite(got[[0, 2, 3]]).all()
