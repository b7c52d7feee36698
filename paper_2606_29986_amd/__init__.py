"""paper_2606_29986_amd -- MI355X (gfx950) deferred-dequantization decode path.

Thin Python binding over ``libhma.so`` (C ABI in ``include/hma.h``): argument
marshalling only.  Every step of the path runs in the library's HIP kernels;
torch supplies device memory and the current HIP stream.  If the library is
missing the import still succeeds but every call raises -- there is no
fallback of any kind.

Paper: "HBM Is Not All You Need" (HMA-Serve), arXiv 2606.29986, Sec. 3.3.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhma.so")

HMA_OK = 0
HMA_EINVAL = -1
HMA_EUNSUPPORTED = -2
HMA_EWORKSPACE = -3
HMA_EHIP = -4
HMA_ESCRATCH = -5
PAGE_BF16 = 0x40000000
PAGE_ID_MASK = 0x3FFFFFFF
HEAD_DIM = 128
PAGE_SIZE = 16

_lib = None


class HmaError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


def lib() -> ctypes.CDLL:
    """Load libhma.so; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libhma.so not built at {LIB_PATH}; run "
                           "`python -m paper_2606_29986_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.hma_bfp8_dequant_pages.argtypes = [vp, vp, vp, vp, vp, i32, i32, i64, i64, i32, i32, i32, vp]
    L.hma_bfp8_dequant_pages.restype = ctypes.c_int
    L.hma_bfp8_dequant_pages_naive.argtypes = L.hma_bfp8_dequant_pages.argtypes
    L.hma_bfp8_dequant_pages_naive.restype = ctypes.c_int
    L.hma_bfp8_rebuild_tiled.argtypes = [vp, i64, i32, i32, i32, vp, vp, i64, i32, i32, i32, i32, vp]
    L.hma_bfp8_rebuild_tiled.restype = ctypes.c_int
    L.hma_bfp8_pack_tiled.argtypes = [vp, i64, i32, i32, i32, vp, vp, vp, i64, i32, i32, i32, vp]
    L.hma_bfp8_pack_tiled.restype = ctypes.c_int
    L.hma_tiled_shard_bytes.argtypes = [i32, i32, i32]
    L.hma_tiled_shard_bytes.restype = i64
    L.hma_ingress_rebuild.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i64, i32, i32, i32, vp]
    L.hma_ingress_rebuild.restype = ctypes.c_int
    L.hma_decode_attn_bfp8.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32, i32, i32,
                                       i32, i32, i32, ctypes.c_float, i32, i32, vp, vp, vp, sz,
                                       vp]
    L.hma_decode_attn_bfp8.restype = ctypes.c_int
    L.hma_decode_attn_bfp8_noalloc.argtypes = L.hma_decode_attn_bfp8.argtypes[:21] + [vp]
    L.hma_decode_attn_bfp8_noalloc.restype = ctypes.c_int
    L.hma_decode_attn_tokens_per_split.argtypes = [i32, i32, i32, i32]
    L.hma_decode_attn_tokens_per_split.restype = i32
    L.hma_decode_attn_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    L.hma_decode_attn_workspace_bytes.restype = sz
    L.hma_validate_page_table.argtypes = [vp, i32, i32, vp, i32, i64, i64, i32, vp]
    L.hma_validate_page_table.restype = ctypes.c_int
    L.hma_paged_read_probe.argtypes = [vp, vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32, vp, sz, vp]
    L.hma_paged_read_probe.restype = ctypes.c_int
    L.hma_stream_read_probe.argtypes = [vp, sz, i32, vp, sz, vp]
    L.hma_stream_read_probe.restype = ctypes.c_int
    L.hma_decode_attn_bfp8_valu.argtypes = [vp, vp, vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32,
                                            ctypes.c_float, i32, vp, vp, vp, sz, vp]
    L.hma_decode_attn_bfp8_valu.restype = ctypes.c_int
    L.hma_decode_attn_valu_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    L.hma_decode_attn_valu_workspace_bytes.restype = sz
    L.hma_issue_probe.argtypes = [i32, i32, i32, i32, i32, vp, sz, vp, sz, vp]
    L.hma_issue_probe.restype = ctypes.c_int
    L.hma_status_string.argtypes = [ctypes.c_int]
    L.hma_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().hma_status_string(int(status)).decode()


def _ptr(t):
    """Device pointer of a torch tensor (or None -> NULL).  Raw ints pass through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check_dev(*ts):
    for t in ts:
        if t is not None and not isinstance(t, int):
            if not t.is_cuda:
                raise ValueError("libhma takes device tensors only")
            if not t.is_contiguous():
                raise ValueError("libhma takes contiguous tensors only")


def tokens_per_split(batch: int, num_q_heads: int, num_kv_heads: int, max_context_len: int) -> int:
    """Split length the library picks when tokens_per_split = 0."""
    return int(lib().hma_decode_attn_tokens_per_split(batch, num_q_heads, num_kv_heads,
                                                      max_context_len))


def workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int, max_context_len: int,
                    tokens_per_split: int = 0) -> int:
    n = int(lib().hma_decode_attn_workspace_bytes(batch, num_q_heads, num_kv_heads,
                                                  max_context_len, tokens_per_split))
    if n == (1 << 64) - 1:
        raise HmaError(HMA_EINVAL, "hma_decode_attn_workspace_bytes")
    return n


def alloc_workspace(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split=0,
                    device="cuda"):
    """Zero-filled workspace tensor of the size the library needs (or None)."""
    import torch
    n = workspace_bytes(batch, num_q_heads, num_kv_heads, max_context_len, tokens_per_split)
    if n == 0:
        return None
    return torch.zeros(n, dtype=torch.uint8, device=device)


def validate_page_table(page_table, context_lens, max_context_len, num_bfp8_pages, num_bf16_pages=-1,
                        page_size=PAGE_SIZE) -> int:
    """hma_validate_page_table on host (numpy) copies: returns -1 when every
    entry the attention kernel would read is in range, else the flat index
    (b * max_pages_per_seq + i) of the first bad entry.  num_bf16_pages < 0:
    no BF16 pools (the tag bit is ignored)."""
    import numpy as np
    pt = np.ascontiguousarray(page_table, dtype=np.int32)
    ctx = np.ascontiguousarray(context_lens, dtype=np.int32)
    if pt.ndim != 2 or ctx.ndim != 1 or ctx.shape[0] != pt.shape[0]:
        raise ValueError("page_table is [batch][max_pages], context_lens [batch]")
    bad = ctypes.c_int64(-2)
    rc = lib().hma_validate_page_table(pt.ctypes.data, pt.shape[0], pt.shape[1], ctx.ctypes.data,
                                       int(max_context_len), int(num_bfp8_pages), int(num_bf16_pages),
                                       int(page_size), ctypes.byref(bad))
    if rc == HMA_OK:
        return -1
    if rc == HMA_EINVAL and bad.value >= 0:
        return int(bad.value)
    raise HmaError(rc, "hma_validate_page_table")


def bfp8_dequant_pages(src_mant, src_exp, dst_bf16, src_pages, dst_pages, n_pools=1,
                       src_pool_stride_pages=0, dst_pool_stride_pages=0, num_kv_heads=8,
                       head_dim=HEAD_DIM, page_size=PAGE_SIZE, n_pages=None, stream=None,
                       naive=False) -> None:
    """hma_bfp8_dequant_pages: rebuild BFP8 pages into the BF16 pool dst_bf16.

    src_mant uint8, src_exp uint8, dst_bf16 int16/uint16/bfloat16 device
    tensors; src_pages / dst_pages int32 device tensors of equal length, or
    None for the identity (then n_pages gives the count).  naive=True runs
    hma_bfp8_dequant_pages_naive (one thread per element; a baseline)."""
    _check_dev(src_mant, src_exp, dst_bf16, src_pages, dst_pages)
    lens = {int(t.numel()) for t in (src_pages, dst_pages) if t is not None}
    if n_pages is not None:
        lens.add(int(n_pages))
    if len(lens) != 1:
        raise ValueError("src_pages, dst_pages and n_pages must agree on the page count")
    n = lens.pop()
    fn = lib().hma_bfp8_dequant_pages_naive if naive else lib().hma_bfp8_dequant_pages
    rc = fn(_ptr(src_mant), _ptr(src_exp), _ptr(dst_bf16), _ptr(src_pages), _ptr(dst_pages), n,
            n_pools, src_pool_stride_pages, dst_pool_stride_pages, num_kv_heads, head_dim,
            page_size, _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_bfp8_dequant_pages" + ("_naive" if naive else ""))


def tiled_shard_bytes(n_tokens: int, heads_per_shard: int, head_dim: int = HEAD_DIM) -> int:
    """Bytes of one prefill shard in the tiled source layout."""
    n = int(lib().hma_tiled_shard_bytes(n_tokens, heads_per_shard, head_dim))
    if n < 0:
        raise HmaError(HMA_EINVAL, "hma_tiled_shard_bytes")
    return n


def bfp8_rebuild_tiled(src, dst_bf16, n_tokens, n_shards, dst_pages=None, n_pools=1,
                       src_pool_stride_bytes=0, dst_pool_stride_pages=0, rope_reorder=False,
                       num_kv_heads=8, head_dim=HEAD_DIM, page_size=PAGE_SIZE, stream=None) -> None:
    """hma_bfp8_rebuild_tiled: tiled per-chip prefill shards (uint8 device
    tensor) -> BF16 pages of dst_bf16, with the rotary key re-layout when
    rope_reorder is set."""
    _check_dev(src, dst_bf16, dst_pages)
    if dst_pages is not None and int(dst_pages.numel()) != (n_tokens + page_size - 1) // page_size:
        raise ValueError("dst_pages must name one page per 16 tokens")
    rc = lib().hma_bfp8_rebuild_tiled(_ptr(src), src_pool_stride_bytes, n_pools, n_shards, n_tokens,
                                      _ptr(dst_bf16), _ptr(dst_pages), dst_pool_stride_pages,
                                      num_kv_heads, head_dim, page_size, int(bool(rope_reorder)),
                                      _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_bfp8_rebuild_tiled")


def bfp8_pack_tiled(src, dst_mant, dst_exp, n_tokens, n_shards, dst_pages=None, n_pools=1,
                    src_pool_stride_bytes=0, dst_pool_stride_pages=0, num_kv_heads=8,
                    head_dim=HEAD_DIM, page_size=PAGE_SIZE, stream=None) -> None:
    """hma_bfp8_pack_tiled: tiled per-chip prefill shards -> BFP8 pages,
    bytes unchanged (keys stay in the interleaved rotary order)."""
    _check_dev(src, dst_mant, dst_exp, dst_pages)
    if dst_pages is not None and int(dst_pages.numel()) != (n_tokens + page_size - 1) // page_size:
        raise ValueError("dst_pages must name one page per 16 tokens")
    rc = lib().hma_bfp8_pack_tiled(_ptr(src), src_pool_stride_bytes, n_pools, n_shards, n_tokens,
                                   _ptr(dst_mant), _ptr(dst_exp), _ptr(dst_pages),
                                   dst_pool_stride_pages, num_kv_heads, head_dim, page_size,
                                   _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_bfp8_pack_tiled")


def ingress_rebuild(host_mant, host_exp, stage_mant, stage_exp, dst_bf16, dst_pages=None,
                    n_pools=1, dst_pool_stride_pages=0, num_kv_heads=8, head_dim=HEAD_DIM,
                    page_size=PAGE_SIZE, stream=None) -> None:
    """hma_ingress_rebuild: copy raw BFP8 pages from host memory to the device
    staging buffers and rebuild them into the BF16 pools, in order on
    ``stream``.  host_mant / host_exp are CPU uint8 tensors shaped
    [n_pools][n_pages][Hkv][16][128] and [...][8] (pinned, for an asynchronous
    copy); the staging tensors are device tensors of the same sizes."""
    for t in (host_mant, host_exp):
        if t.is_cuda or not t.is_contiguous():
            raise ValueError("host_mant and host_exp must be contiguous CPU tensors")
    _check_dev(stage_mant, stage_exp, dst_bf16, dst_pages)
    if host_mant.dim() != 5 or host_exp.dim() != 5:
        raise ValueError("host buffers are [n_pools][n_pages][Hkv][page_size][...]")
    pools, n = int(host_mant.shape[0]), int(host_mant.shape[1])
    if pools != n_pools or host_exp.shape[:2] != host_mant.shape[:2]:
        raise ValueError("host buffer shapes disagree with n_pools")
    if stage_mant.numel() < host_mant.numel() or stage_exp.numel() < host_exp.numel():
        raise ValueError("staging buffers smaller than the host buffers")
    if dst_pages is not None and int(dst_pages.numel()) != n:
        raise ValueError("dst_pages must name one page per staged page")
    rc = lib().hma_ingress_rebuild(host_mant.data_ptr(), host_exp.data_ptr(), _ptr(stage_mant),
                                   _ptr(stage_exp), _ptr(dst_bf16), _ptr(dst_pages), n, n_pools,
                                   dst_pool_stride_pages, num_kv_heads, head_dim, page_size,
                                   _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_ingress_rebuild")


def decode_attn_bfp8(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, max_context_len,
                     out, k_bf16=None, v_bf16=None, lse=None, scale=None, num_kv_heads=None,
                     tokens_per_split=0, workspace=None, head_dim=HEAD_DIM, page_size=PAGE_SIZE,
                     key_order=0, stream=None) -> None:
    """hma_decode_attn_bfp8: fused BFP8 paged decode attention into ``out``.

    q, out: [B][Hq][128] 16-bit tensors (BF16 bits); pools as in hma.h;
    page_table int32 [B][max_pages]; context_lens int32 [B];
    max_context_len: host int bound.  num_kv_heads defaults to k_mant.shape[1].
    key_order=1: K pages hold channels in the interleaved rotary order."""
    _check_dev(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, out, k_bf16, v_bf16,
               lse, workspace)
    B, Hq, D = q.shape
    hkv = int(num_kv_heads if num_kv_heads is not None else k_mant.shape[1])
    if scale is None:
        scale = 1.0 / (D ** 0.5)
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    rc = lib().hma_decode_attn_bfp8(
        _ptr(q), _ptr(k_mant), _ptr(k_exp), _ptr(v_mant), _ptr(v_exp), _ptr(k_bf16),
        _ptr(v_bf16), _ptr(page_table), int(page_table.shape[1]), _ptr(context_lens),
        int(max_context_len), B, Hq, hkv, D, page_size, float(scale), int(key_order),
        int(tokens_per_split),
        _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_decode_attn_bfp8")


def decode_attn_bfp8_noalloc(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, max_context_len,
                             out, k_bf16=None, v_bf16=None, lse=None, scale=None, num_kv_heads=None,
                             tokens_per_split=0, head_dim=HEAD_DIM, page_size=PAGE_SIZE, key_order=0,
                             stream=None) -> None:
    """hma_decode_attn_bfp8_noalloc: decode_attn_bfp8 without a workspace (the
    library's fixed device scratch holds the split-merge state)."""
    _check_dev(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, out, k_bf16, v_bf16, lse)
    B, Hq, D = q.shape
    hkv = int(num_kv_heads if num_kv_heads is not None else k_mant.shape[1])
    if scale is None:
        scale = 1.0 / (D ** 0.5)
    rc = lib().hma_decode_attn_bfp8_noalloc(
        _ptr(q), _ptr(k_mant), _ptr(k_exp), _ptr(v_mant), _ptr(v_exp), _ptr(k_bf16),
        _ptr(v_bf16), _ptr(page_table), int(page_table.shape[1]), _ptr(context_lens),
        int(max_context_len), B, Hq, hkv, D, page_size, float(scale), int(key_order),
        int(tokens_per_split), _ptr(out), _ptr(lse), _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_decode_attn_bfp8_noalloc")


ISSUE_KINDS = ("v_add_u32", "v_perm_b32", "v_cvt_f32_ubyte1", "v_pk_sub_u16", "v_fma_f32")


def issue_probe(valu_kind, valu_ops, with_mfma, waves_per_simd, iters, cycles, sink, stream=None) -> None:
    """hma_issue_probe: cycles (int64/uint64 device tensor, 1024 * waves_per_simd
    words) receives each wave's shader-clock cycles over `iters` steps of
    eight (matrix instruction + valu_ops instructions of ISSUE_KINDS[valu_kind])
    groups; sink holds 64 words per wave."""
    _check_dev(cycles, sink)
    rc = lib().hma_issue_probe(int(valu_kind), int(valu_ops), int(with_mfma), int(waves_per_simd), int(iters),
                               _ptr(cycles), int(cycles.numel()), _ptr(sink), int(sink.numel()), _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_issue_probe")


def valu_workspace_bytes(batch: int, num_q_heads: int, num_kv_heads: int, max_context_len: int,
                         tokens_per_split: int = 0) -> int:
    """hma_decode_attn_valu_workspace_bytes."""
    n = int(lib().hma_decode_attn_valu_workspace_bytes(batch, num_q_heads, num_kv_heads,
                                                       max_context_len, tokens_per_split))
    if n == (1 << 64) - 1:
        raise HmaError(HMA_EINVAL, "hma_decode_attn_valu_workspace_bytes")
    return n


def decode_attn_bfp8_valu(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, max_context_len,
                          out, workspace, lse=None, scale=None, num_kv_heads=None, tokens_per_split=0,
                          head_dim=HEAD_DIM, page_size=PAGE_SIZE, stream=None) -> None:
    """hma_decode_attn_bfp8_valu: decode_attn_bfp8 over BFP8 pages with both
    products on the vector ALU (a measured comparison point, not for
    production).  workspace: uint8 device tensor of valu_workspace_bytes()."""
    _check_dev(q, k_mant, k_exp, v_mant, v_exp, page_table, context_lens, out, lse, workspace)
    B, Hq, D = q.shape
    hkv = int(num_kv_heads if num_kv_heads is not None else k_mant.shape[1])
    if scale is None:
        scale = 1.0 / (D ** 0.5)
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    rc = lib().hma_decode_attn_bfp8_valu(
        _ptr(q), _ptr(k_mant), _ptr(k_exp), _ptr(v_mant), _ptr(v_exp), _ptr(page_table),
        int(page_table.shape[1]), _ptr(context_lens), int(max_context_len), B, Hq, hkv, D, page_size,
        float(scale), int(tokens_per_split), _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes,
        _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_decode_attn_bfp8_valu")


def paged_read_probe(k_mant, k_exp, v_mant, v_exp, page_table, context_lens, max_context_len, sink,
                     num_kv_heads, pages_per_split, n_splits, heads_per_workgroup=1, stream=None) -> None:
    """hma_paged_read_probe: read (and XOR) the BFP8 bytes of an attention call
    in its decomposition; sink is a uint32/int32 device tensor of
    batch * (num_kv_heads / heads_per_workgroup) * n_splits * 8 words."""
    _check_dev(k_mant, k_exp, v_mant, v_exp, page_table, context_lens, sink)
    B = int(page_table.shape[0])
    rc = lib().hma_paged_read_probe(
        _ptr(k_mant), _ptr(k_exp), _ptr(v_mant), _ptr(v_exp), _ptr(page_table), int(page_table.shape[1]),
        _ptr(context_lens), int(max_context_len), B, int(num_kv_heads), int(heads_per_workgroup),
        int(pages_per_split), int(n_splits), _ptr(sink), int(sink.numel()), _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_paged_read_probe")


def stream_read_probe(buf, sink, n_workgroups, stream=None) -> None:
    """hma_stream_read_probe: read (and XOR) a contiguous device buffer;
    sink holds n_workgroups * 4 words."""
    _check_dev(buf, sink)
    nbytes = int(buf.numel()) * int(buf.element_size())
    rc = lib().hma_stream_read_probe(_ptr(buf), nbytes, int(n_workgroups), _ptr(sink), int(sink.numel()),
                                     _stream(stream))
    if rc != HMA_OK:
        raise HmaError(rc, "hma_stream_read_probe")
