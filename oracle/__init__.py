"""Plain float64 CPU oracle for the BFP8 deferred-dequantization decode path.

TEST INFRASTRUCTURE ONLY.  The product library never imports, links or calls
anything in this package; only the tests, the package smoke check and the
CPU-baseline leg of the benchmark do.  The arithmetic lives in
``hma_oracle.c`` (plain C, float64, scalar, OpenMP over independent rows);
this module compiles it with gcc and marshals numpy arrays through ctypes.

Paper: "HBM Is Not All You Need" (HMA-Serve), arXiv 2606.29986.
  - BFP8 block-float decode and the BF16 paged cache: Sec. 3.3 (Deferred
    Dequantization) and Sec. 2.3 (Challenge 2).
  - Paged single-token decode attention over BFP8/BF16 pages: Sec. 3.3, Fig. 2.
Parity status of each function is listed in the design notes; every function
here is pinned by a ``-m "not gpu"`` test (closed forms, library routines,
invariants), except agreement with Tenstorrent's own BFP8 bit layout, which
the paper does not give ("parity unpinned" for that reading only).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hma_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

TAG_BF16 = 0x40000000
ID_MASK = 0x3FFFFFFF
BLOCK = 16

_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile hma_oracle.c into oracle/liboracle.so with gcc (-O2, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _p(ctype):
    return ctypes.POINTER(ctype)


def lib():
    """Load (building first if absent) the oracle shared library."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(_LIB_PATH)
        u8, u16, i32, i64, f64 = (ctypes.c_uint8, ctypes.c_uint16, ctypes.c_int32,
                                  ctypes.c_int64, ctypes.c_double)
        L.ora_bf16_to_f64.argtypes = [u16]
        L.ora_bf16_to_f64.restype = f64
        L.ora_f64_to_bf16.argtypes = [f64]
        L.ora_f64_to_bf16.restype = u16
        L.ora_bfp8_decode_value.argtypes = [u8, u8]
        L.ora_bfp8_decode_value.restype = u16
        L.ora_bfp8_decode_bits.argtypes = [u8, u8]
        L.ora_bfp8_decode_bits.restype = u16
        L.ora_bfp8_encode_block.argtypes = [_p(u16), _p(u8), _p(u8)]
        L.ora_bfp8_encode_block.restype = ctypes.c_int
        L.ora_bfp8_encode_blocks.argtypes = [_p(u16), i64, _p(u8), _p(u8)]
        L.ora_bfp8_encode_blocks.restype = ctypes.c_int
        L.ora_bfp8_decode_blocks.argtypes = [_p(u8), _p(u8), i64, _p(u16)]
        L.ora_bfp8_decode_blocks.restype = None
        L.ora_bfp8_decode_blocks_bits.argtypes = [_p(u8), _p(u8), i64, _p(u16)]
        L.ora_bfp8_decode_blocks_bits.restype = None
        L.ora_dequant_pages.argtypes = [_p(u8), _p(u8), _p(u16), _p(i32), _p(i32), i32, i32,
                                        i64, i64, i32, i32, i32]
        L.ora_dequant_pages.restype = None
        L.ora_rebuild_tiled.argtypes = [_p(u8), i64, i32, i32, i32, i32, i32, i32, i32, _p(u16),
                                        _p(i32), i64]
        L.ora_rebuild_tiled.restype = None
        L.ora_pack_tiled.argtypes = [_p(u8), i64, i32, i32, i32, i32, i32, i32, _p(u8), _p(u8),
                                     _p(i32), i64]
        L.ora_pack_tiled.restype = None
        L.ora_merge_partials.argtypes = [i32, _p(f64), _p(f64), _p(f64), i32, _p(f64), _p(f64)]
        L.ora_merge_partials.restype = None
        L.ora_decode_attn.argtypes = [_p(u16), _p(u8), _p(u8), _p(u8), _p(u8), _p(u16), _p(u16),
                                      _p(i32), i32, _p(i32), i32, i32, i32, i32, i32, f64, i32,
                                      _p(f64), _p(f64)]
        L.ora_decode_attn.restype = ctypes.c_int
        L.ora_decode_attn_split_one.argtypes = [_p(u16), _p(u8), _p(u8), _p(u8), _p(u8), _p(u16),
                                                _p(u16), _p(i32), i32, _p(i32), i32, i32, i32, i32,
                                                f64, i32, i32, _p(i32), i32, _p(f64), _p(f64),
                                                _p(f64), _p(f64), _p(f64)]
        L.ora_decode_attn_split_one.restype = ctypes.c_int
        _lib = L
        return L


def _ptr(a, ctype):
    if a is None:
        return ctypes.POINTER(ctype)()
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ BF16

def bf16_to_f64(bits) -> np.ndarray:
    """BF16 bit patterns (uint16 array) -> float64, exactly."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_scalar(v: float) -> int:
    """float64 -> BF16 bits with round-to-nearest-even (scalar)."""
    return int(lib().ora_f64_to_bf16(float(v)))


# ------------------------------------------------------------------ BFP8

def decode_scalar(E: int, byte: int) -> int:
    """Value-level BFP8 decode of one element -> BF16 bits."""
    return int(lib().ora_bfp8_decode_value(E, byte))


def decode_bits_scalar(E: int, byte: int) -> int:
    """Bit-assembly BFP8 decode of one element -> BF16 bits."""
    return int(lib().ora_bfp8_decode_bits(E, byte))


def decode_blocks(mant: np.ndarray, exps: np.ndarray, route: str = "value") -> np.ndarray:
    """Decode consecutive 16-element blocks; mant.size == 16 * exps.size.

    Returns uint16 BF16 bits with mant's shape.  route = "value" (definition)
    or "bits" (bit-assembly twin)."""
    m = _c(mant, np.uint8)
    e = _c(exps, np.uint8)
    if m.size != BLOCK * e.size:
        raise ValueError("mantissa count must be 16 x exponent count")
    out = np.empty(m.shape, dtype=np.uint16)
    fn = lib().ora_bfp8_decode_blocks if route == "value" else lib().ora_bfp8_decode_blocks_bits
    fn(_ptr(m, ctypes.c_uint8), _ptr(e, ctypes.c_uint8), e.size, _ptr(out, ctypes.c_uint16))
    return out


def encode_blocks(x_bf16: np.ndarray):
    """Encode BF16 bits (size multiple of 16) into (mantissa bytes, exponents).

    mant has x's shape; exps has shape x.shape[:-1] + (x.shape[-1] // 16,).
    Raises ValueError on NaN/Inf inputs."""
    x = _c(x_bf16, np.uint16)
    if x.shape[-1] % BLOCK:
        raise ValueError("last dimension must be a multiple of 16")
    mant = np.empty(x.shape, dtype=np.uint8)
    exps = np.empty(x.shape[:-1] + (x.shape[-1] // BLOCK,), dtype=np.uint8)
    rc = lib().ora_bfp8_encode_blocks(_ptr(x, ctypes.c_uint16), x.size // BLOCK,
                                      _ptr(mant, ctypes.c_uint8), _ptr(exps, ctypes.c_uint8))
    if rc != 0:
        raise ValueError("BFP8 encode: non-finite input")
    return mant, exps


# ---------------------------------------------------- page reconstruction

def dequant_pages(src_mant, src_exp, dst, src_pages, dst_pages, n_pools,
                  src_pool_stride_pages, dst_pool_stride_pages,
                  num_kv_heads, head_dim, page_size) -> np.ndarray:
    """Reconstruct BFP8 pages into the BF16 pool ``dst`` (modified in place).

    Same argument meaning as the library call hma_bfp8_dequant_pages; pools
    are flat numpy arrays addressed by page strides."""
    assert dst.dtype == np.uint16 and dst.flags["C_CONTIGUOUS"]
    m = _c(src_mant, np.uint8)
    e = _c(src_exp, np.uint8)
    sp = _c(src_pages, np.int32)
    dp = _c(dst_pages, np.int32)
    lib().ora_dequant_pages(_ptr(m, ctypes.c_uint8), _ptr(e, ctypes.c_uint8),
                            _ptr(dst, ctypes.c_uint16), _ptr(sp, ctypes.c_int32),
                            _ptr(dp, ctypes.c_int32), sp.size, n_pools,
                            src_pool_stride_pages, dst_pool_stride_pages,
                            num_kv_heads, head_dim, page_size)
    return dst


TILE_BYTES = 64 + 32 * 32     # one 32x32 BFP8 tile of a prefill shard


def tiled_shard_bytes(n_tokens, heads_per_shard, head_dim=128):
    """Bytes of one shard: heads x ceil(tokens/32) x head_dim/32 tiles."""
    return heads_per_shard * ((n_tokens + 31) // 32) * (head_dim // 32) * TILE_BYTES


def rebuild_tiled(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens, num_kv_heads, dst,
                  dst_pages, dst_pool_stride_pages, rope_reorder, head_dim=128, page_size=16):
    """Tiled prefill shards -> BF16 pages (``dst`` modified in place); see
    ora_rebuild_tiled for the tile byte order."""
    assert dst.dtype == np.uint16 and dst.flags["C_CONTIGUOUS"]
    s = _c(src, np.uint8)
    dp = _c(dst_pages, np.int32)
    lib().ora_rebuild_tiled(_ptr(s, ctypes.c_uint8), src_pool_stride_bytes, n_pools, n_shards,
                            n_tokens, num_kv_heads, head_dim, page_size, int(bool(rope_reorder)),
                            _ptr(dst, ctypes.c_uint16), _ptr(dp, ctypes.c_int32),
                            dst_pool_stride_pages)
    return dst


def pack_tiled(src, src_pool_stride_bytes, n_pools, n_shards, n_tokens, num_kv_heads, dst_mant,
               dst_exp, dst_pages, dst_pool_stride_pages, head_dim=128, page_size=16):
    """Tiled shards -> BFP8 pages, bytes unchanged (dst_* modified in place)."""
    assert dst_mant.dtype == np.uint8 and dst_exp.dtype == np.uint8
    assert dst_mant.flags["C_CONTIGUOUS"] and dst_exp.flags["C_CONTIGUOUS"]
    s = _c(src, np.uint8)
    dp = _c(dst_pages, np.int32)
    lib().ora_pack_tiled(_ptr(s, ctypes.c_uint8), src_pool_stride_bytes, n_pools, n_shards,
                         n_tokens, num_kv_heads, head_dim, page_size,
                         _ptr(dst_mant, ctypes.c_uint8), _ptr(dst_exp, ctypes.c_uint8),
                         _ptr(dp, ctypes.c_int32), dst_pool_stride_pages)
    return dst_mant, dst_exp


# ---------------------------------------------------------- attention

def decode_attn(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table, context_lens,
                num_kv_heads, page_size, scale, key_order=0):
    """float64 paged decode attention.

    q: uint16 [B][Hq][D] BF16 bits.  Pools as in the library (flat or shaped).
    page_table: int32 [B][max_pages]; context_lens: int32 [B].
    scale: float; it is first rounded to float32 (the library takes a float)
    and then widened, so both sides use the same scale value.
    key_order=1: K rows are stored in the interleaved rotary order and are
    relabelled to the queries' half-split order on read.
    Returns (out float64 [B][Hq][D], lse float64 [B][Hq])."""
    q = _c(q, np.uint16)
    B, Hq, D = q.shape
    pt = _c(page_table, np.int32)
    cl = _c(context_lens, np.int32)
    assert pt.shape[0] == B and cl.shape == (B,)
    out = np.zeros((B, Hq, D), dtype=np.float64)
    lse = np.zeros((B, Hq), dtype=np.float64)
    arrs = [_c(a, t) for a, t in ((k_mant, np.uint8), (k_exp, np.uint8), (v_mant, np.uint8),
                                  (v_exp, np.uint8), (k_bf16, np.uint16), (v_bf16, np.uint16))]
    rc = lib().ora_decode_attn(
        _ptr(q, ctypes.c_uint16),
        _ptr(arrs[0], ctypes.c_uint8), _ptr(arrs[1], ctypes.c_uint8),
        _ptr(arrs[2], ctypes.c_uint8), _ptr(arrs[3], ctypes.c_uint8),
        _ptr(arrs[4], ctypes.c_uint16), _ptr(arrs[5], ctypes.c_uint16),
        _ptr(pt, ctypes.c_int32), pt.shape[1], _ptr(cl, ctypes.c_int32),
        B, Hq, num_kv_heads, D, page_size, float(np.float32(scale)), int(key_order),
        _ptr(out, ctypes.c_double), _ptr(lse, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle decode_attn: bad arguments")
    return out, lse


def decode_attn_split_one(q, k_mant, k_exp, v_mant, v_exp, k_bf16, v_bf16, page_table,
                          context_lens, num_kv_heads, page_size, scale, b, h, bounds):
    """One (b, h) row computed as separate contiguous token ranges, merged.

    bounds: nondecreasing ints from 0 to context_lens[b].  Returns
    (out [D], lse, part_m [S], part_l [S], part_o [S][D])."""
    q = _c(q, np.uint16)
    B, Hq, D = q.shape
    pt = _c(page_table, np.int32)
    cl = _c(context_lens, np.int32)
    bd = _c(bounds, np.int32)
    S = bd.size - 1
    pm = np.zeros(S, dtype=np.float64)
    pl = np.zeros(S, dtype=np.float64)
    po = np.zeros((S, D), dtype=np.float64)
    out = np.zeros(D, dtype=np.float64)
    lse = np.zeros(1, dtype=np.float64)
    arrs = [_c(a, t) for a, t in ((k_mant, np.uint8), (k_exp, np.uint8), (v_mant, np.uint8),
                                  (v_exp, np.uint8), (k_bf16, np.uint16), (v_bf16, np.uint16))]
    rc = lib().ora_decode_attn_split_one(
        _ptr(q, ctypes.c_uint16),
        _ptr(arrs[0], ctypes.c_uint8), _ptr(arrs[1], ctypes.c_uint8),
        _ptr(arrs[2], ctypes.c_uint8), _ptr(arrs[3], ctypes.c_uint8),
        _ptr(arrs[4], ctypes.c_uint16), _ptr(arrs[5], ctypes.c_uint16),
        _ptr(pt, ctypes.c_int32), pt.shape[1], _ptr(cl, ctypes.c_int32),
        Hq, num_kv_heads, D, page_size, float(np.float32(scale)), b, h,
        _ptr(bd, ctypes.c_int32), S, _ptr(pm, ctypes.c_double), _ptr(pl, ctypes.c_double),
        _ptr(po, ctypes.c_double), _ptr(out, ctypes.c_double), _ptr(lse, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle split attention: bad partition")
    return out, float(lse[0]), pm, pl, po


def merge_partials(m, l, o):
    """Log-sum-exp merge of partials (m [S], l [S], o [S][D]) -> (out [D], lse)."""
    m = _c(m, np.float64)
    l = _c(l, np.float64)
    o = _c(o, np.float64)
    S, D = o.shape
    out = np.zeros(D, dtype=np.float64)
    lse = np.zeros(1, dtype=np.float64)
    lib().ora_merge_partials(S, _ptr(m, ctypes.c_double), _ptr(l, ctypes.c_double),
                             _ptr(o, ctypes.c_double), D, _ptr(out, ctypes.c_double),
                             _ptr(lse, ctypes.c_double))
    return out, float(lse[0])
