"""Pins for the oracle's BFP8 decode and encode (CPU only).

The paper (Sec. 3.3) states the format as a per-block shared exponent with a
7-bit mantissa per element, reconstructed to BF16 by bit manipulation.  The
readings used where it is silent: sign in bit 7, exponent byte with bias 127,
value = (-1)^s * m * 2^(E-133), 16-element blocks.

Each pin checks the oracle against something other than itself:
  * hand-derived values (tests/golden/bfp8_decode_examples.json),
  * numpy's float32 ldexp (a library route to the same exact value),
  * the independent bit-assembly twin, on all 65,536 (E, byte) pairs,
  * round-trip / idempotence / half-quantum error bound of the encoder.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

E_ALL = np.repeat(np.arange(256, dtype=np.uint8), 256)        # E-major
B_ALL = np.tile(np.arange(256, dtype=np.uint8), 256)


def _table(route):
    # the 65,536 pairs as 4096 blocks of 16: block k has exponent k // 16
    mant = B_ALL.reshape(4096, 16)
    exps = E_ALL.reshape(4096, 16)[:, 0].copy()
    return oracle.decode_blocks(mant, exps, route=route).reshape(-1)


def _numpy_route():
    """Decode through numpy's float32 ldexp: exact, subnormal-preserving,
    overflow to inf.  The BF16 pattern of an exactly representable float32 is
    its upper 16 bits."""
    m = (B_ALL & 0x7F).astype(np.float32)
    sign = np.where(B_ALL & 0x80, np.float32(-1.0), np.float32(1.0))
    with np.errstate(over="ignore"):
        v = np.ldexp(sign * m, E_ALL.astype(np.int32) - 133).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def test_decode_golden_examples():
    cases = json.load(open(os.path.join(GOLDEN, "bfp8_decode_examples.json")))["cases"]
    assert len(cases) >= 15
    for c in cases:
        E, byte, want = c["E"], int(c["byte"], 16), int(c["bf16"], 16)
        assert oracle.decode_scalar(E, byte) == want, c
        assert oracle.decode_bits_scalar(E, byte) == want, c


def test_decode_exhaustive_value_equals_bits():
    a = _table("value")
    b = _table("bits")
    bad = np.nonzero(a != b)[0]
    assert bad.size == 0, [(int(E_ALL[i]), int(B_ALL[i]), hex(a[i]), hex(b[i])) for i in bad[:8]]


def test_decode_exhaustive_equals_numpy_ldexp():
    a = _table("value")
    ref = _numpy_route()
    bad = np.nonzero(a != ref)[0]
    assert bad.size == 0, [(int(E_ALL[i]), int(B_ALL[i]), hex(a[i]), hex(ref[i])) for i in bad[:8]]


def test_decode_exhaustive_properties():
    a = _table("value")
    v = oracle.bf16_to_f64(a)
    m = (B_ALL & 0x7F).astype(np.int64)
    s = (B_ALL >> 7).astype(np.int64)
    # sign bit of the output is the element's sign bit, always (also for zero)
    assert np.array_equal((a >> 15).astype(np.int64), s)
    # no NaN is ever produced; Inf exactly for E = 255 and m >= 64
    assert not np.isnan(v).any()
    inf = np.isinf(v)
    assert np.array_equal(inf, (E_ALL == 255) & (m >= 64))
    # finite outputs equal the exact real value
    fin = ~inf
    exact = np.ldexp(m[fin].astype(np.float64), E_ALL[fin].astype(np.int64) - 133)
    assert np.array_equal(np.abs(v[fin]), exact)
    # monotone in m for a fixed exponent and sign
    mag = np.abs(v).reshape(256, 2, 128)
    assert (mag[:, :, 1:] >= mag[:, :, :-1]).all()


def test_f64_to_bf16_rounding_cases():
    f = oracle.f64_to_bf16_scalar
    assert f(1.0) == 0x3F80
    assert f(-2.0) == 0xC000
    # halfway between 1.0 and 1 + 2^-7 ties to even (1.0); just above rounds up
    assert f(1.0 + 2.0 ** -8) == 0x3F80
    assert f(1.0 + 2.0 ** -8 + 2.0 ** -30) == 0x3F81
    # halfway between 1 + 2^-7 (odd) and 1 + 2^-6 ties up to even
    assert f(1.0 + 3 * 2.0 ** -8) == 0x3F82
    # largest finite and overflow
    assert f(float.fromhex("0x1.fep127")) == 0x7F7F
    assert f(float.fromhex("0x1.ffp127")) == 0x7F80
    # subnormals: 2^-133 is fraction 1; 2^-134 is a tie to even (0)
    assert f(2.0 ** -133) == 0x0001
    assert f(2.0 ** -134) == 0x0000
    assert f(3 * 2.0 ** -134) == 0x0002
    assert f(-0.0) == 0x8000
    assert f(float("inf")) == 0x7F80
    assert (f(float("nan")) & 0x7FFF) > 0x7F80


# ----------------------------------------------------------------- encoder

def _bf16_from_f64(vals):
    return np.array([oracle.f64_to_bf16_scalar(x) for x in vals], dtype=np.uint16)


@st.composite
def representable_blocks(draw):
    """Blocks whose values are exactly (-1)^s m 2^(E-133) with the block
    maximum's leading bit (bit 6) set, so the encoding is unique."""
    E = draw(st.integers(min_value=1, max_value=254))
    ms = draw(st.lists(st.integers(0, 127), min_size=16, max_size=16))
    signs = draw(st.lists(st.booleans(), min_size=16, max_size=16))
    k = draw(st.integers(0, 15))
    ms[k] = draw(st.integers(64, 127))
    vals = [(-1.0 if s and m else 1.0) * m * 2.0 ** (E - 133) for m, s in zip(ms, signs)]
    return E, ms, signs, vals


@settings(max_examples=300, deadline=None)
@given(representable_blocks())
def test_encode_roundtrip_representable(blk):
    E, ms, signs, vals = blk
    x = _bf16_from_f64(vals)
    # representable values are exact in BF16 (at most 7 significant bits)
    assert np.array_equal(oracle.bf16_to_f64(x), np.array(vals))
    mant, exps = oracle.encode_blocks(x)
    assert int(exps[0]) == E
    assert [int(b) & 0x7F for b in mant] == ms
    back = oracle.decode_blocks(mant, exps)
    assert np.array_equal(oracle.bf16_to_f64(back), oracle.bf16_to_f64(x))
    # bit-identical except that a negative zero input has no sign in BFP8
    for xi, bi in zip(x, back):
        assert xi == bi or (xi == 0x8000 and bi == 0x0000)


finite_bf16 = st.integers(0, 0xFFFF).filter(lambda b: ((b >> 7) & 0xFF) != 0xFF)


@settings(max_examples=400, deadline=None)
@given(st.lists(finite_bf16, min_size=16, max_size=16))
def test_encode_error_bound_and_idempotence(block):
    x = np.array(block, dtype=np.uint16)
    mant, exps = oracle.encode_blocks(x)
    E = int(exps[0])
    assert E == max(((int(b) >> 7) & 0xFF) for b in block)
    xv = oracle.bf16_to_f64(x)
    back = oracle.bf16_to_f64(oracle.decode_blocks(mant, exps))
    # half a quantum: |x - x_hat| <= 2^(E-134) (the 127.5 -> 127 clamp is also half)
    assert (np.abs(xv - back) <= 2.0 ** (E - 134)).all()
    # the sign survives unless the element rounds to zero
    for xi, bi in zip(xv, back):
        if bi != 0:
            assert np.sign(xi) == np.sign(bi)
    # RNE on exact ties: |x| * 2^(133-E) = k + 1/2 rounds to the even k or k+1
    scaled = np.abs(xv) * 2.0 ** (133 - E)
    q = (mant & 0x7F).astype(np.float64)
    tie = scaled - np.floor(scaled) == 0.5
    ok_tie = (q[tie] % 2 == 0) | (q[tie] == 127)
    assert ok_tie.all()
    # idempotence: encode(decode(encode(x))) == encode(x)
    mant2, exps2 = oracle.encode_blocks(oracle.decode_blocks(mant, exps))
    assert np.array_equal(exps2, exps)
    assert np.array_equal(mant2, mant)


def test_encode_special_blocks():
    zeros = np.zeros(16, dtype=np.uint16)
    mant, exps = oracle.encode_blocks(zeros)
    assert exps[0] == 0 and not mant.any()
    negz = np.full(16, 0x8000, dtype=np.uint16)
    mant, exps = oracle.encode_blocks(negz)
    assert exps[0] == 0 and not mant.any()          # sign cleared when m = 0
    # all-ones significand maximum: 1.9921875 * 2^0 -> 127.5 -> clamps to 127
    blk = np.zeros(16, dtype=np.uint16)
    blk[3] = 0x3FFF
    mant, exps = oracle.encode_blocks(blk)
    assert exps[0] == 127 and mant[3] == 127
    # subnormal-only block: E = 0 and mantissas are the subnormal fractions
    blk = np.arange(16, dtype=np.uint16) * 7 + 0x8000 * (np.arange(16) % 2).astype(np.uint16)
    mant, exps = oracle.encode_blocks(blk)
    assert exps[0] == 0
    assert np.array_equal(oracle.decode_blocks(mant, exps)[2:], blk[2:])
    for bad in (0x7F80, 0xFF80, 0x7FC0):
        b = np.zeros(16, dtype=np.uint16)
        b[5] = bad
        with pytest.raises(ValueError):
            oracle.encode_blocks(b)


def test_encode_matches_independent_numpy_quantiser():
    """Encode a realistic draw and compare with a vectorised numpy statement
    of the same rule (max exponent field, RNE via np.rint, clamp, sign)."""
    r = np.random.default_rng(7)
    x = (r.standard_normal((512, 128)).astype(np.float32) * 3).astype(np.float32)
    xb = (x.view(np.uint32) >> 16).astype(np.uint16)         # truncation is fine for inputs
    mant, exps = oracle.encode_blocks(xb)
    blocks = xb.reshape(-1, 16)
    E = ((blocks >> 7) & 0xFF).max(axis=1).astype(np.int64)
    vals = oracle.bf16_to_f64(blocks)
    q = np.minimum(np.rint(np.abs(vals) * np.exp2(133 - E)[:, None]), 127).astype(np.int64)
    s = ((blocks >> 15) & 1).astype(np.int64) * (q != 0)
    assert np.array_equal(exps.reshape(-1).astype(np.int64), E)
    assert np.array_equal(mant.reshape(-1, 16).astype(np.int64), (s << 7) | q)
