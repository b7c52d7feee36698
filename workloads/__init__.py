"""Seeded synthetic workloads for the BFP8 decode path (shared input generators).

This module only draws random numbers and arranges them into the shapes of
the evaluated workloads; it holds none of the method's arithmetic (no BFP8
encode or decode, no attention).  Tests turn the BF16 draws into BFP8 pages
with the oracle's encoder; the benchmark draws BFP8 byte streams directly
(``bfp8_codes_device``), since its throughput does not depend on values.

Shapes follow the paper's evaluated models and traces (Table 2; Sec. 4):
Qwen3-4B/8B/14B/32B attention shapes (head_dim 128, 8 KV heads), paged KV
with 16-token pages, and ShareGPT / LongBench / arXiv-like length mixes stood
in for by seeded log-normal length draws.  None of those datasets is used.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
HEAD_DIM = 128
TAG_BF16 = 0x40000000


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    layers: int
    num_q_heads: int
    num_kv_heads: int
    batch: int
    ctx: tuple                     # ("uniform", n) | ("lognormal", median, sigma, lo, hi)
                                   # | ("bimodal", p_short, med_short, med_long, sigma, cap, floor)
    kv_dist: str                   # "outlier" | "channel_lognormal"
    bf16_page_fraction: float = 0.0
    head_dim: int = HEAD_DIM
    page_size: int = PAGE_SIZE
    notes: str = field(default="", compare=False)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


WORKLOADS = {
    0: Workload(0, "qwen3-4b-smoke-1layer-b4-ctx512", 1, 32, 8, 4, ("uniform", 512), "outlier",
                notes="tiny smoke case the oracle finishes in seconds"),
    1: Workload(1, "qwen3-8b-b32-ctx4096", 36, 32, 8, 32, ("uniform", 4096), "channel_lognormal"),
    2: Workload(2, "qwen3-14b-ragged-b64-ln2048", 40, 40, 8, 64,
                ("lognormal", 2048.0, 0.8, 64, 16384), "channel_lognormal"),
    3: Workload(3, "qwen3-32b-b16-ctx8192", 64, 64, 8, 16, ("uniform", 8192), "outlier",
                notes="headline long-context configuration"),
    4: Workload(4, "qwen3-32b-trace-mix-200seq", 64, 64, 8, 200,
                ("bimodal", 0.7, 1024.0, 12288.0, 0.8, 32768, 64), "outlier",
                bf16_page_fraction=0.5),
}

# named sub-streams of one workload's seed
_STREAMS = {"q": 0, "k": 1, "v": 2, "outlier": 3, "chanscale": 4, "lens": 5, "perm": 6, "fresh": 7,
            "garbage": 8, "codes": 9}


def rng(workload_index: int, stream: str, *sub: int) -> np.random.Generator:
    """Independent generator for (workload, stream, sub-keys...).

    Root entropy is 1000 + workload index; sub-streams are spawn keys, so a
    draw never depends on which other draws were made first."""
    key = (_STREAMS[stream],) + tuple(int(s) for s in sub)
    return np.random.default_rng(np.random.SeedSequence(1000 + workload_index, spawn_key=key))


# ----------------------------------------------------------------- lengths

def context_lens(w: Workload) -> np.ndarray:
    """Per-sequence context lengths (int32 [batch])."""
    kind = w.ctx[0]
    r = rng(w.index, "lens")
    if kind == "uniform":
        return np.full(w.batch, w.ctx[1], dtype=np.int32)
    if kind == "lognormal":
        _, median, sigma, lo, hi = w.ctx
        x = r.lognormal(math.log(median), sigma, size=w.batch)
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    if kind == "bimodal":
        _, p_short, med_s, med_l, sigma, cap, floor = w.ctx
        short = r.random(w.batch) < p_short
        xs = r.lognormal(math.log(med_s), sigma, size=w.batch)
        xl = r.lognormal(math.log(med_l), sigma, size=w.batch)
        x = np.where(short, xs, xl)
        return np.clip(np.rint(x), floor, cap).astype(np.int32)
    raise ValueError(kind)


def pages_per_seq(ctx: np.ndarray, page_size: int = PAGE_SIZE) -> np.ndarray:
    return (np.asarray(ctx, dtype=np.int64) + page_size - 1) // page_size


def page_table(w: Workload, ctx: np.ndarray, max_pages: int | None = None):
    """Page table with physical ids drawn from a seeded permutation.

    Returns (pt int32 [batch][max_pages], total_pages).  Logical page i of
    sequence b maps to physical page pt[b][i]; unused entries hold 0."""
    npg = pages_per_seq(ctx, w.page_size)
    total = int(npg.sum())
    if max_pages is None:
        max_pages = max(1, int(npg.max()) if npg.size else 1)
    perm = rng(w.index, "perm").permutation(total).astype(np.int32)
    pt = np.zeros((len(ctx), max_pages), dtype=np.int32)
    off = 0
    for b, n in enumerate(npg):
        pt[b, :n] = perm[off:off + n]
        off += n
    return pt, total


def bf16_page_mask(w: Workload, total_pages: int, fraction: float | None = None) -> np.ndarray:
    """Exactly round(fraction * total) pages (seeded choice) marked True."""
    f = w.bf16_page_fraction if fraction is None else fraction
    n = int(round(f * total_pages))
    mask = np.zeros(total_pages, dtype=bool)
    mask[rng(w.index, "fresh").choice(total_pages, size=n, replace=False)] = True
    return mask


# ------------------------------------------------------------------ values

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> BF16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    flat = u.reshape(-1)
    out = np.empty(flat.size, np.uint16)
    # in chunks, in place: large fresh temporaries dominate the cost otherwise
    step = 1 << 18
    tmp = np.empty(min(step, flat.size), np.uint32)
    for s in range(0, flat.size, step):
        c = flat[s:s + step]
        t = tmp[:c.size]
        np.right_shift(c, 16, out=t)
        t &= 1
        t += np.uint32(0x7FFF)
        t += c
        t >>= 16
        out[s:s + step] = t
    return out.reshape(u.shape)


def kv_values_bf16(w: Workload, layer: int, kind: str, num_pages: int) -> np.ndarray:
    """K or V values as BF16 bits, shape [num_pages][Hkv][page_size][head_dim].

    "outlier": N(0,1) with 4 distinct channels per (layer, kv head, K/V)
    multiplied by 20.  "channel_lognormal": N(0,1) times a per-(layer, kv
    head, K/V, channel) LogNormal(0, 0.5) scale."""
    assert kind in ("k", "v")
    kv_id = 0 if kind == "k" else 1
    shape = (num_pages, w.num_kv_heads, w.page_size, w.head_dim)
    x = rng(w.index, kind, layer).standard_normal(size=shape, dtype=np.float32)
    if w.kv_dist == "outlier":
        r = rng(w.index, "outlier", layer, kv_id)
        for j in range(w.num_kv_heads):
            ch = r.choice(w.head_dim, size=4, replace=False)
            for c in ch:           # distinct channels; strided views, no temporaries
                x[:, j, :, c] *= np.float32(20.0)
    elif w.kv_dist == "channel_lognormal":
        r = rng(w.index, "chanscale", layer, kv_id)
        s = r.lognormal(0.0, 0.5, size=(w.num_kv_heads, w.head_dim)).astype(np.float32)
        x *= s[None, :, None, :]
    else:
        raise ValueError(w.kv_dist)
    return f32_to_bf16_bits(x)


def q_bf16(w: Workload, layer: int = 0) -> np.ndarray:
    """Queries as BF16 bits, N(0,1), shape [batch][Hq][head_dim]."""
    x = rng(w.index, "q", layer).standard_normal(size=(w.batch, w.num_q_heads, w.head_dim),
                                                 dtype=np.float32)
    return f32_to_bf16_bits(x)


def softmax_scale(w: Workload) -> float:
    """1/sqrt(head_dim) as a float32 value."""
    return float(np.float32(1.0 / math.sqrt(w.head_dim)))


def garbage_bytes(w: Workload, n: int, salt: int = 0) -> np.ndarray:
    """Uniform random bytes for slots no result may depend on."""
    return rng(w.index, "garbage", salt).integers(0, 256, size=n, dtype=np.uint8)


# ----------------------------------------------- bulk device draws (bench)

def bfp8_codes_device(w: Workload, layer: int, kind: str, num_pages: int, device, route: str = "packed"):
    """Random BFP8 byte streams drawn directly on the device (benchmark only).

    Mantissa bytes are uniform over all 256 sign/magnitude codes; exponent
    bytes are uniform over 124..131, the range the BF16 draws above produce.
    The fused attention's work per page depends on the data in two places:
    it picks one of two exact decode routes per (page, KV head) -- the packed
    16-bit route when every block exponent of the page lies in 7..133, the
    ldexp route otherwise -- and it skips the rescale of its accumulators
    when a page does not raise the running maximum.  Exponents in 124..131
    always take the packed route.  route="ldexp" forces the other one: the
    first block exponent of token 0 of every (page, KV head) is set to 134
    (elements up to 254, still finite).  Encoder-produced values of the
    outlier workloads mix both routes.  Returns (mant uint8, exp uint8)
    tensors of shapes [pages][Hkv][P][D] and [pages][Hkv][P][D/16]."""
    import torch
    if route not in ("packed", "ldexp"):
        raise ValueError(route)
    g = torch.Generator(device=device)
    g.manual_seed(int(np.random.SeedSequence(
        1000 + w.index, spawn_key=(_STREAMS["codes"], layer, 0 if kind == "k" else 1)
    ).generate_state(1)[0]))
    shp = (num_pages, w.num_kv_heads, w.page_size, w.head_dim)
    mant = torch.randint(0, 256, shp, dtype=torch.uint8, device=device, generator=g)
    exp = torch.randint(124, 132, shp[:-1] + (w.head_dim // 16,), dtype=torch.uint8,
                        device=device, generator=g)
    if route == "ldexp":
        exp[:, :, 0, 0] = 134
    return mant, exp
