"""C-ABI checks that need no GPU: the library loads, exports every function
include/hma.h declares, and rejects bad arguments on the host before any HIP
call (so nothing is launched)."""
import ctypes
import os
import re

import pytest

import paper_2606_29986_amd as hma

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hma.h")

# a non-NULL, 256-byte aligned fake device address: never dereferenced because
# every call below fails validation before any HIP call
FAKE = 0x10000
MISALIGNED = 0x10008


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"HMA_API\s+[\w\s\*]+?\b(hma_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    assert names == sorted(["hma_bfp8_dequant_pages", "hma_bfp8_dequant_pages_naive",
                            "hma_bfp8_pack_tiled", "hma_bfp8_rebuild_tiled", "hma_tiled_shard_bytes",
                            "hma_decode_attn_bfp8", "hma_decode_attn_bfp8_noalloc",
                            "hma_decode_attn_tokens_per_split", "hma_decode_attn_workspace_bytes",
                            "hma_ingress_rebuild", "hma_status_string", "hma_validate_page_table",
                            "hma_paged_read_probe", "hma_stream_read_probe",
                            "hma_decode_attn_bfp8_valu", "hma_decode_attn_valu_workspace_bytes",
                            "hma_issue_probe"])


def test_library_exports_every_declared_symbol():
    L = hma.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    # nothing but the C ABI is exported
    out = os.popen(f"nm -D --defined-only {hma.LIB_PATH}").read()
    exported = sorted(l.split()[-1] for l in out.splitlines() if " T " in l)
    assert exported == declared_functions()


def test_status_strings():
    for st in (0, -1, -2, -3, -4, 7):
        s = hma.status_string(st)
        assert isinstance(s, str) and s
    assert hma.status_string(0) == "ok"


def test_split_and_workspace_queries():
    tps = hma.tokens_per_split(16, 64, 8, 8192)
    assert tps > 0 and tps % 16 == 0
    S = -(-8192 // tps)
    ws = hma.workspace_bytes(16, 64, 8, 8192)
    pairs, g = 16 * 8, 8
    tickets = (pairs * 4 + 255) // 256 * 256
    ml = (pairs * S * g * 8 + 255) // 256 * 256
    assert ws == tickets + ml + pairs * S * g * 128 * 4
    # the 4-wave shape with the automatic split: page-balanced ranges, one per
    # wave, whose partial slots per KV head are bounded by the grid's share of
    # ranges (512 / Hkv workgroups x 4 waves) or by the ranges of the largest
    # size, plus one per sequence
    B, Hkv, g, ctx = 64, 8, 5, 15192
    assert hma.tokens_per_split(B, Hkv * g, Hkv, ctx) == 2048
    pages = -(-ctx // 16)
    slots = Hkv * (max(512 // Hkv * 4, -(-B * pages // 1024)) + B)
    assert hma.workspace_bytes(B, Hkv * g, Hkv, ctx) == (
        (B * Hkv * 4 + 255) // 256 * 256 + (slots * g * 8 + 255) // 256 * 256 + slots * g * 128 * 4)
    # the same shape with an explicit split: one slot per (sequence, head, split)
    S = -(-ctx // 2048)
    assert hma.workspace_bytes(B, Hkv * g, Hkv, ctx, 2048) == (
        (B * Hkv * 4 + 255) // 256 * 256 + (B * Hkv * S * g * 8 + 255) // 256 * 256 + B * Hkv * S * g * 512)
    # one split: no workspace
    assert hma.workspace_bytes(4, 32, 8, 512, 512) == 0
    assert hma.workspace_bytes(4, 32, 8, 0) == 0
    # explicit split sizes must be whole pages
    assert hma.workspace_bytes(4, 32, 8, 512, 48) > 0
    with pytest.raises(hma.HmaError):
        hma.workspace_bytes(4, 32, 8, 512, 40)
    with pytest.raises(hma.HmaError):
        hma.workspace_bytes(4, 30, 8, 512)
    assert hma.tokens_per_split(4, 30, 8, 512) == 0


def _dequant(naive=False, **kw):
    a = dict(src_mant=FAKE, src_exp=FAKE, dst=FAKE * 2, src_pages=FAKE, dst_pages=FAKE,
             n_pages=4, n_pools=1, src_stride=0, dst_stride=0, hkv=8, D=128, P=16)
    a.update(kw)
    fn = hma.lib().hma_bfp8_dequant_pages_naive if naive else hma.lib().hma_bfp8_dequant_pages
    return fn(a["src_mant"], a["src_exp"], a["dst"], a["src_pages"],
                                            a["dst_pages"], a["n_pages"], a["n_pools"],
                                            a["src_stride"], a["dst_stride"], a["hkv"], a["D"],
                                            a["P"], None)


@pytest.mark.parametrize("naive", [False, True])
def test_dequant_validation(naive):
    _dequant_validation(lambda **kw: _dequant(naive=naive, **kw))


def _dequant_validation(_dequant):
    assert _dequant(n_pages=0) == hma.HMA_OK             # no-op, nothing touched
    assert _dequant(n_pools=0) == hma.HMA_OK
    assert _dequant(n_pages=-1) == hma.HMA_EINVAL
    assert _dequant(hkv=0) == hma.HMA_EINVAL
    assert _dequant(D=64) == hma.HMA_EUNSUPPORTED
    assert _dequant(P=32) == hma.HMA_EUNSUPPORTED
    # (NULL page lists mean the identity and are valid: not probed here, since
    # with every other argument valid the call would launch on fake pointers)
    for k in ("src_mant", "src_exp", "dst"):
        assert _dequant(**{k: None}) == hma.HMA_EINVAL, k
    for k in ("src_mant", "src_exp", "dst"):
        assert _dequant(**{k: MISALIGNED}) == hma.HMA_EINVAL, k
    assert _dequant(dst=FAKE) == hma.HMA_EINVAL           # aliases the source
    # the span the host can bound: 4 pages of 8 x 2048 mantissa bytes from FAKE
    assert _dequant(dst=FAKE + 4 * 8 * 2048 - 256) == hma.HMA_EINVAL   # starts inside it
    assert _dequant(dst=FAKE - 256) == hma.HMA_EINVAL                  # ends inside it
    assert _dequant(src_exp=FAKE * 8, dst=FAKE * 8 + 4 * 8 * 128 - 16) == hma.HMA_EINVAL
    # two pools at a stride of 64 pages: the second pool's pages count too
    assert _dequant(n_pools=2, src_stride=64, dst_stride=4,
                    dst=FAKE + (64 + 3) * 8 * 2048) == hma.HMA_EINVAL
    assert _dequant(n_pools=2, src_stride=0, dst_stride=4) == hma.HMA_EINVAL
    assert _dequant(n_pools=2, src_stride=4, dst_stride=-1) == hma.HMA_EINVAL


def _ingress(**kw):
    a = dict(hm=FAKE, he=FAKE, sm=FAKE * 2, se=FAKE * 4, dst=FAKE * 8, dst_pages=None, n_pages=4,
             n_pools=2, dst_stride=64, hkv=8, D=128, P=16)
    a.update(kw)
    return hma.lib().hma_ingress_rebuild(a["hm"], a["he"], a["sm"], a["se"], a["dst"], a["dst_pages"],
                                         a["n_pages"], a["n_pools"], a["dst_stride"], a["hkv"],
                                         a["D"], a["P"], None)


def test_ingress_validation():
    assert _ingress(n_pages=0, hm=None) == hma.HMA_OK        # nothing to move
    assert _ingress(n_pools=0) == hma.HMA_OK
    assert _ingress(n_pages=-1) == hma.HMA_EINVAL
    assert _ingress(hkv=0) == hma.HMA_EINVAL
    assert _ingress(D=64) == hma.HMA_EUNSUPPORTED
    assert _ingress(P=8) == hma.HMA_EUNSUPPORTED
    for k in ("hm", "he", "sm", "se", "dst"):
        assert _ingress(**{k: None}) == hma.HMA_EINVAL, k
    for k in ("sm", "se", "dst"):
        assert _ingress(**{k: MISALIGNED}) == hma.HMA_EINVAL, k
    assert _ingress(dst_stride=0) == hma.HMA_EINVAL          # two pools need a stride
    assert _ingress(se=FAKE * 2 + 64) == hma.HMA_EINVAL      # staging buffers overlap
    assert _ingress(dst=FAKE * 2) == hma.HMA_EINVAL          # destination is the staging


def test_tiled_shard_bytes_matches_the_oracle():
    import oracle
    for n, hs in ((1, 1), (31, 2), (32, 2), (33, 8), (8192, 2)):
        assert hma.tiled_shard_bytes(n, hs) == oracle.tiled_shard_bytes(n, hs)
    with pytest.raises(hma.HmaError):
        hma.tiled_shard_bytes(-1, 2)
    with pytest.raises(hma.HmaError):
        hma.tiled_shard_bytes(32, 2, head_dim=64)


def _tiled(**kw):
    a = dict(src=FAKE, stride=0, pools=1, shards=4, n=100, dst=FAKE * 2, pages=None, dstride=0,
             hkv=8, D=128, P=16, rope=1)
    a.update(kw)
    return hma.lib().hma_bfp8_rebuild_tiled(a["src"], a["stride"], a["pools"], a["shards"], a["n"],
                                            a["dst"], a["pages"], a["dstride"], a["hkv"], a["D"],
                                            a["P"], a["rope"], None)


def test_tiled_rebuild_validation():
    assert _tiled(n=0) == hma.HMA_OK
    assert _tiled(pools=0) == hma.HMA_OK
    assert _tiled(n=-1) == hma.HMA_EINVAL
    assert _tiled(shards=0) == hma.HMA_EINVAL
    assert _tiled(shards=3) == hma.HMA_EINVAL            # 8 heads over 3 chips
    assert _tiled(rope=2) == hma.HMA_EINVAL
    assert _tiled(D=64) == hma.HMA_EUNSUPPORTED
    assert _tiled(src=None) == hma.HMA_EINVAL
    assert _tiled(dst=None) == hma.HMA_EINVAL
    assert _tiled(src=MISALIGNED) == hma.HMA_EINVAL
    assert _tiled(pools=2, stride=64, dstride=10) == hma.HMA_EINVAL      # pools overlap
    need = 4 * hma.tiled_shard_bytes(100, 2)
    assert _tiled(pools=2, stride=need + 8, dstride=10) == hma.HMA_EINVAL  # stride not 16-aligned
    assert _tiled(pools=2, stride=need, dstride=0) == hma.HMA_EINVAL


def test_pack_tiled_validation():
    def _pack(**kw):
        a = dict(src=FAKE, stride=0, pools=1, shards=4, n=100, dm=FAKE * 2, de=FAKE * 4, pages=None,
                 dstride=0, hkv=8, D=128, P=16)
        a.update(kw)
        return hma.lib().hma_bfp8_pack_tiled(a["src"], a["stride"], a["pools"], a["shards"], a["n"],
                                             a["dm"], a["de"], a["pages"], a["dstride"], a["hkv"],
                                             a["D"], a["P"], None)
    assert _pack(n=0) == hma.HMA_OK
    assert _pack(shards=3) == hma.HMA_EINVAL
    assert _pack(dm=None) == hma.HMA_EINVAL
    assert _pack(de=MISALIGNED) == hma.HMA_EINVAL
    assert _pack(de=FAKE * 2) == hma.HMA_EINVAL             # the two pools coincide
    assert _pack(P=32) == hma.HMA_EUNSUPPORTED


def _attn(**kw):
    a = dict(q=FAKE, km=FAKE, ke=FAKE, vm=FAKE, ve=FAKE, kb=None, vb=None, pt=FAKE, maxp=512,
             ctx=FAKE, maxctx=8192, B=16, Hq=64, Hkv=8, D=128, P=16, scale=0.088388346,
             tps=0, out=FAKE, lse=None, ws=None, wsb=0, korder=0)
    a.update(kw)
    return hma.lib().hma_decode_attn_bfp8(a["q"], a["km"], a["ke"], a["vm"], a["ve"], a["kb"],
                                          a["vb"], a["pt"], a["maxp"], a["ctx"], a["maxctx"],
                                          a["B"], a["Hq"], a["Hkv"], a["D"], a["P"], a["scale"],
                                          a["korder"], a["tps"], a["out"], a["lse"], a["ws"], a["wsb"],
                                          None)


def test_attn_validation():
    need = hma.workspace_bytes(16, 64, 8, 8192)
    assert need > 0
    # everything valid except the missing workspace
    assert _attn() == hma.HMA_EWORKSPACE
    assert _attn(ws=FAKE, wsb=need - 1) == hma.HMA_EWORKSPACE
    assert _attn(ws=MISALIGNED, wsb=need) == hma.HMA_EINVAL
    assert _attn(Hq=60) == hma.HMA_EINVAL                  # Hq % Hkv != 0
    assert _attn(Hq=8 * 17) == hma.HMA_EUNSUPPORTED        # group of 17
    assert _attn(D=64) == hma.HMA_EUNSUPPORTED
    assert _attn(P=32) == hma.HMA_EUNSUPPORTED
    assert _attn(tps=40) == hma.HMA_EINVAL                 # not whole pages
    assert _attn(tps=-32) == hma.HMA_EINVAL
    assert _attn(maxctx=-1) == hma.HMA_EINVAL
    assert _attn(maxp=100) == hma.HMA_EINVAL               # 8192 tokens need 512 pages
    assert _attn(scale=float("nan")) == hma.HMA_EINVAL
    assert _attn(korder=2) == hma.HMA_EINVAL
    assert _attn(B=0) == hma.HMA_OK                        # nothing to do
    for k in ("q", "km", "ke", "vm", "ve", "pt", "ctx", "out"):
        assert _attn(**{k: None}) == hma.HMA_EINVAL, k
    for k in ("q", "km", "ke", "vm", "ve", "out"):
        assert _attn(**{k: MISALIGNED}) == hma.HMA_EINVAL, k
    assert _attn(kb=FAKE, vb=None) == hma.HMA_EINVAL       # both BF16 pools or neither
    assert _attn(kb=MISALIGNED, vb=FAKE) == hma.HMA_EINVAL
    assert _attn(lse=0x10002) == hma.HMA_EINVAL


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(hma, "_lib", None)
    monkeypatch.setattr(hma, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        hma.lib()


def test_page_table_validator():
    """hma_validate_page_table checks, on host copies, exactly the entries the
    attention kernel reads: ceil(clamped length / 16) per row, ids below the
    pool sizes, the BF16 tag checked against the BF16 pool (or ignored when
    there is none), negative entries rejected."""
    import numpy as np
    B, W = 4, 8
    pt = np.arange(B * W, dtype=np.int32).reshape(B, W)
    ctx = np.array([0, 17, 128, 5], np.int32)
    assert hma.validate_page_table(pt, ctx, 128, num_bfp8_pages=B * W) == -1
    # row 1 reads 2 entries: an out-of-range third entry is never read
    pt2 = pt.copy()
    pt2[1, 2] = 10 ** 6
    assert hma.validate_page_table(pt2, ctx, 128, B * W) == -1
    pt2[1, 1] = B * W                                       # id == pool size
    assert hma.validate_page_table(pt2, ctx, 128, B * W) == 1 * W + 1
    pt3 = pt.copy()
    pt3[2, 7] = -5
    assert hma.validate_page_table(pt3, ctx, 128, B * W) == 2 * W + 7
    # lengths are clamped to the bound, negatives read nothing
    assert hma.validate_page_table(pt3, np.array([0, 17, 112, -3], np.int32), 112, B * W) == -1
    assert hma.validate_page_table(pt3, np.array([0, 17, 500, -3], np.int32), 112, B * W) == -1
    # BF16 tag: checked against the BF16 pool when one is given
    pt4 = pt.copy()
    pt4[3, 0] = 3 | hma.PAGE_BF16
    assert hma.validate_page_table(pt4, ctx, 128, B * W, num_bf16_pages=4) == -1
    assert hma.validate_page_table(pt4, ctx, 128, B * W, num_bf16_pages=3) == 3 * W
    assert hma.validate_page_table(pt4, ctx, 128, B * W) == -1     # no BF16 pools: tag ignored
    pt4[3, 0] = (B * W) | hma.PAGE_BF16
    assert hma.validate_page_table(pt4, ctx, 128, B * W) == 3 * W
    # sizes
    with pytest.raises(hma.HmaError):
        hma.validate_page_table(pt, ctx, 129, B * W)       # more tokens than the table holds
    with pytest.raises(hma.HmaError):
        hma.validate_page_table(pt, ctx, 128, B * W, page_size=32)


def test_noalloc_validation():
    """hma_decode_attn_bfp8_noalloc validates like hma_decode_attn_bfp8 and
    rejects, before any HIP call, problems larger than its fixed scratch:
    1000 sequences x 8 KV heads x 16 query heads at 32K tokens need far more
    than 16 MiB of partials."""
    L = hma.lib()

    def call(B=1000, Hq=128, maxctx=32768, maxp=2048, q=FAKE):
        return L.hma_decode_attn_bfp8_noalloc(q, FAKE, FAKE, FAKE, FAKE, None, None, FAKE, maxp, FAKE, maxctx,
                                              B, Hq, 8, 128, 16, 0.088388346, 0, 0, FAKE, None, None)
    assert hma.workspace_bytes(1000, 128, 8, 32768) > (16 << 20)
    assert call() == hma.HMA_ESCRATCH
    assert "scratch" in hma.status_string(hma.HMA_ESCRATCH)
    assert call(q=None) == hma.HMA_EINVAL
    assert call(maxp=100) == hma.HMA_EINVAL
    assert call(Hq=60) == hma.HMA_EINVAL
    assert call(B=0) == hma.HMA_OK


def test_read_probe_validation():
    """The read probes reject bad shapes, pools and sinks before any HIP call."""
    L = hma.lib()

    def paged(B=4, maxp=64, maxctx=1000, hkv=8, hpw=1, pps=32, ns=2, sink_words=None, k=FAKE, pt=FAKE):
        words = B * (hkv // hpw) * ns * 8 if sink_words is None else sink_words
        return L.hma_paged_read_probe(k, FAKE, FAKE, FAKE, pt, maxp, FAKE, maxctx, B, hkv, hpw, pps, ns,
                                      FAKE, words, None)
    assert paged(k=None) == hma.HMA_EINVAL
    assert paged(k=MISALIGNED) == hma.HMA_EINVAL
    assert paged(pt=None) == hma.HMA_EINVAL
    assert paged(hpw=3) == hma.HMA_EINVAL                 # not 1, 2, 4 or 8
    assert paged(hkv=4, hpw=8) == hma.HMA_EINVAL          # does not divide the KV heads
    assert paged(pps=0) == hma.HMA_EINVAL
    assert paged(pps=1025) == hma.HMA_EINVAL              # beyond the staged page-table slice
    assert paged(ns=1) == hma.HMA_EINVAL                  # 32 pages do not cover 1000 tokens
    assert paged(maxctx=1025, maxp=64) == hma.HMA_EINVAL  # more tokens than the table holds
    assert paged(sink_words=4 * 8 * 2 * 8 - 1) == hma.HMA_EINVAL
    assert paged(B=0) == hma.HMA_OK                       # nothing to read

    def stream(buf=FAKE, nbytes=1 << 20, nwg=64, sink_words=None):
        return L.hma_stream_read_probe(buf, nbytes, nwg, FAKE, 4 * nwg if sink_words is None else sink_words,
                                       None)
    assert stream(buf=None) == hma.HMA_EINVAL
    assert stream(buf=MISALIGNED) == hma.HMA_EINVAL
    assert stream(nbytes=0) == hma.HMA_EINVAL
    assert stream(nbytes=1000) == hma.HMA_EINVAL          # not a multiple of 16
    assert stream(nwg=0) == hma.HMA_EINVAL
    assert stream(nwg=(1 << 20) + 1) == hma.HMA_EINVAL
    assert stream(sink_words=255) == hma.HMA_EINVAL


def test_valu_attn_validation_and_workspace():
    """The vector-ALU comparison kernel: BFP8 pools only, groups up to 8, a
    workspace of (2 + 128) floats per (sequence, query head, range) with the
    (max, sum) region padded to 256 bytes; every check before any HIP call."""
    L = hma.lib()
    # automatic ranges: one workgroup per compute unit (256) over the batch at
    # max_context_len, whole pages, at most 4096 tokens
    def auto_splits(B, Hkv, ctx):
        tps = min(-(-B * Hkv * ctx // 256), ctx, 4096)
        return -(-ctx // (-(-tps // 16) * 16))
    B, Hq, Hkv, ctx = 16, 64, 8, 8192
    S = auto_splits(B, Hkv, ctx)
    assert S == 2
    assert hma.valu_workspace_bytes(B, Hq, Hkv, ctx) == (B * Hq * S * 8 + 255) // 256 * 256 + B * Hq * S * 512
    # as many pairs as compute units: one range per sequence up to 4096 tokens
    assert hma.valu_workspace_bytes(64, 64, 8, 2400) == 64 * 64 * 8 + 64 * 64 * 512
    assert hma.valu_workspace_bytes(64, 64, 8, 9000) == 3 * (64 * 64 * 8 + 64 * 64 * 512)
    # a small batch: ranges of ceil(B * Hkv * ctx / 256) tokens rounded up to whole pages
    assert auto_splits(1, 8, 8000) == 32
    assert hma.valu_workspace_bytes(1, 64, 8, 8000) == (64 * 32 * 8 + 255) // 256 * 256 + 64 * 32 * 512
    # explicit ranges
    assert hma.valu_workspace_bytes(B, Hq, Hkv, ctx, 1024) == B * Hq * 8 * 8 + B * Hq * 8 * 512
    assert hma.valu_workspace_bytes(0, Hq, Hkv, ctx) == 0
    for bad in ((B, 60, Hkv, ctx, 0), (B, 16 * 9, 16, ctx, 0), (B, Hq, Hkv, ctx, 40), (B, Hq, Hkv, -1, 0),
                (B, Hq, Hkv, ctx, 16400)):
        with pytest.raises(hma.HmaError):
            hma.valu_workspace_bytes(*bad)

    need = hma.valu_workspace_bytes(B, Hq, Hkv, ctx)

    def call(q=FAKE, maxp=512, maxctx=ctx, Hq=Hq, Hkv=Hkv, D=128, P=16, tps=0, ws=FAKE, wsb=need, lse=None,
             scale=0.088388346, Bn=B):
        return L.hma_decode_attn_bfp8_valu(q, FAKE, FAKE, FAKE, FAKE, FAKE, maxp, FAKE, maxctx, Bn, Hq, Hkv, D, P,
                                           scale, tps, FAKE, lse, ws, wsb, None)
    assert call(ws=None) == hma.HMA_EWORKSPACE
    assert call(wsb=need - 1) == hma.HMA_EWORKSPACE
    assert call(ws=MISALIGNED) == hma.HMA_EINVAL
    assert call(Hq=16 * 9, Hkv=16) == hma.HMA_EUNSUPPORTED      # group of 9
    assert call(Hq=60) == hma.HMA_EINVAL
    assert call(D=64) == hma.HMA_EUNSUPPORTED
    assert call(P=32) == hma.HMA_EUNSUPPORTED
    assert call(tps=40) == hma.HMA_EINVAL
    assert call(maxp=100) == hma.HMA_EINVAL
    assert call(scale=float("nan")) == hma.HMA_EINVAL
    assert call(q=None) == hma.HMA_EINVAL
    assert call(q=MISALIGNED) == hma.HMA_EINVAL
    assert call(lse=0x10002) == hma.HMA_EINVAL
    assert call(Bn=0) == hma.HMA_OK


def test_issue_probe_validation():
    """hma_issue_probe rejects unsupported mixes and short buffers before any HIP call."""
    L = hma.lib()

    def call(kind=0, valu=8, mfma=1, wps=2, iters=100, cyc=FAKE, cw=None, sink=FAKE, sw=None):
        n = 1024 * wps
        return L.hma_issue_probe(kind, valu, mfma, wps, iters, cyc, n if cw is None else cw, sink,
                                 n * 64 if sw is None else sw, None)
    assert call(valu=3) == hma.HMA_EINVAL
    assert call(valu=4) == hma.HMA_EINVAL
    assert call(kind=-1) == hma.HMA_EINVAL
    assert call(kind=5) == hma.HMA_EINVAL
    assert call(valu=0, mfma=0) == hma.HMA_EINVAL
    assert call(mfma=2) == hma.HMA_EINVAL
    assert call(wps=0) == hma.HMA_EINVAL
    assert call(wps=5) == hma.HMA_EINVAL
    assert call(iters=0) == hma.HMA_EINVAL
    assert call(cyc=None) == hma.HMA_EINVAL
    assert call(cyc=FAKE + 4) == hma.HMA_EINVAL           # 8-byte words
    assert call(cw=2047) == hma.HMA_EINVAL
    assert call(sw=2048 * 64 - 1) == hma.HMA_EINVAL
