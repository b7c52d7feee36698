"""Shared host-side helpers for the tests: seeded paged workloads encoded by
the oracle's BFP8 encoder.  Test infrastructure; not part of the library."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

import oracle
import workloads as wl


@dataclass
class PagedKV:
    """One layer of paged KV (host arrays) and everything needed to attend."""
    q: np.ndarray            # uint16 [B][Hq][D]
    k_mant: np.ndarray       # uint8  [pages][Hkv][P][D]
    k_exp: np.ndarray        # uint8  [pages][Hkv][P][D/16]
    v_mant: np.ndarray
    v_exp: np.ndarray
    k_bf16: np.ndarray       # uint16 [pages][Hkv][P][D]  (decoded values, or None)
    v_bf16: np.ndarray
    page_table: np.ndarray   # int32 [B][max_pages]  (tag bit 30 on BF16 pages)
    ctx: np.ndarray          # int32 [B]
    num_kv_heads: int
    page_size: int
    scale: float

    def oracle_attn(self, key_order=0):
        return oracle.decode_attn(self.q, self.k_mant, self.k_exp, self.v_mant, self.v_exp,
                                  self.k_bf16, self.v_bf16, self.page_table, self.ctx,
                                  self.num_kv_heads, self.page_size, self.scale, key_order=key_order)


def make_paged(w: wl.Workload, layer: int = 0, ctx=None, bf16_fraction: float = 0.0,
               garbage_tail: bool = True, with_bf16_pool: bool = True,
               value_seqs=None) -> PagedKV:
    """Build one layer of workload w with the oracle's encoder.

    ctx overrides the workload's length draw.  bf16_fraction of the pages
    (seeded) are tagged as BF16 pages whose BF16 pool holds the exact decoded
    values.  garbage_tail fills the slots past each sequence's end with random
    bytes that no result may depend on.  value_seqs (for the very large
    workloads) restricts the value draws to the pages of those sequences;
    every other page holds zeros, and only those sequences may be checked."""
    ctx = wl.context_lens(w) if ctx is None else np.asarray(ctx, dtype=np.int32)
    pt, total = wl.page_table(w, ctx)
    total = max(total, 1)
    if value_seqs is None:
        k_mant, k_exp = oracle.encode_blocks(wl.kv_values_bf16(w, layer, "k", total))
        v_mant, v_exp = oracle.encode_blocks(wl.kv_values_bf16(w, layer, "v", total))
    else:
        npg_all = wl.pages_per_seq(ctx, w.page_size)
        ids = np.concatenate([pt[b, :npg_all[b]] for b in value_seqs]).astype(np.int64)
        shape = (total, w.num_kv_heads, w.page_size, w.head_dim)
        k_mant = np.zeros(shape, np.uint8)
        v_mant = np.zeros(shape, np.uint8)
        k_exp = np.zeros(shape[:-1] + (w.head_dim // 16,), np.uint8)
        v_exp = np.zeros_like(k_exp)
        for kind, mant, ex in (("k", k_mant, k_exp), ("v", v_mant, v_exp)):
            m_sub, e_sub = oracle.encode_blocks(wl.kv_values_bf16(w, layer, kind, ids.size))
            mant[ids] = m_sub
            ex[ids] = e_sub
    if garbage_tail:
        npg = wl.pages_per_seq(ctx, w.page_size)
        salt = 0
        for b in range(len(ctx)):
            used = int(ctx[b]) - (int(npg[b]) - 1) * w.page_size
            if npg[b] == 0 or used == w.page_size:
                continue
            pid = int(pt[b, npg[b] - 1])
            for arr in (k_mant, k_exp, v_mant, v_exp):
                tail = arr[pid, :, used:, :]
                tail[...] = wl.garbage_bytes(w, tail.size, salt).reshape(tail.shape)
                salt += 1
    k_bf = oracle.decode_blocks(k_mant, k_exp) if with_bf16_pool else None
    v_bf = oracle.decode_blocks(v_mant, v_exp) if with_bf16_pool else None
    if bf16_fraction > 0:
        mask = wl.bf16_page_mask(w, total, bf16_fraction)
        tagged = pt.copy()
        npg = wl.pages_per_seq(ctx, w.page_size)
        for b in range(len(ctx)):
            for i in range(int(npg[b])):
                if mask[pt[b, i]]:
                    tagged[b, i] = pt[b, i] | wl.TAG_BF16
        pt = tagged
    return PagedKV(wl.q_bf16(w, layer), k_mant, k_exp, v_mant, v_exp, k_bf, v_bf, pt, ctx,
                   w.num_kv_heads, w.page_size, wl.softmax_scale(w))


def dense_kv(kv: PagedKV, b: int):
    """Decoded K and V of sequence b as float64 [Hkv][ctx][D] (dense gather
    written independently of the oracle's page walk)."""
    n = int(kv.ctx[b])
    P = kv.page_size
    D = kv.q.shape[-1]
    Hkv = kv.num_kv_heads
    K = np.zeros((Hkv, n, D))
    V = np.zeros((Hkv, n, D))
    kdec = oracle.bf16_to_f64(oracle.decode_blocks(kv.k_mant, kv.k_exp))
    vdec = oracle.bf16_to_f64(oracle.decode_blocks(kv.v_mant, kv.v_exp))
    for t in range(n):
        e = int(kv.page_table[b, t // P])
        pid = e & oracle.ID_MASK
        if e & oracle.TAG_BF16:
            K[:, t] = oracle.bf16_to_f64(kv.k_bf16[pid, :, t % P])
            V[:, t] = oracle.bf16_to_f64(kv.v_bf16[pid, :, t % P])
        else:
            K[:, t] = kdec[pid, :, t % P]
            V[:, t] = vdec[pid, :, t % P]
    return K, V


def tiny_workload(Hq=8, Hkv=2, B=2, index=0):
    """A small custom shape used by the brute-force pins (head_dim 128)."""
    return wl.Workload(index=index, name="tiny", layers=1, num_q_heads=Hq, num_kv_heads=Hkv,
                       batch=B, ctx=("uniform", 1), kv_dist="outlier")
