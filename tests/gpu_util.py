"""Helpers for the GPU parity tests: move oracle-built inputs to the device,
run the library through its C ABI, compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2606_29986_amd as hma

# tolerance for the BF16 attention output against the float64 oracle (absolute + relative)
ATOL = 2e-3
RTOL = 1e-2
# LSE (float32): scores are exact products summed in float32 and the softmax
# weights carry ~2^-17 relative error, so |d lse| stays far below 1e-4 for
# |lse| < 100; the bound below leaves an order of magnitude of room
LSE_ATOL = 1e-3
LSE_RTOL = 1e-5


def note(msg):
    """Name the case on stdout before a GPU step (survives a lost box)."""
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.cuda()


def bf16_bits_to_f64(t):
    return oracle.bf16_to_f64(t.cpu().numpy().view(np.uint16))


class DevKV:
    """Device copy of a tests.oracle_fixtures.PagedKV."""

    def __init__(self, kv):
        self.kv = kv
        self.q = dev(kv.q.view(np.int16))
        self.k_mant = dev(kv.k_mant)
        self.k_exp = dev(kv.k_exp)
        self.v_mant = dev(kv.v_mant)
        self.v_exp = dev(kv.v_exp)
        self.k_bf16 = None if kv.k_bf16 is None else dev(kv.k_bf16.view(np.int16))
        self.v_bf16 = None if kv.v_bf16 is None else dev(kv.v_bf16.view(np.int16))
        self.pt = dev(kv.page_table)
        self.ctx = dev(kv.ctx)
        self.max_ctx = int(kv.ctx.max()) if kv.ctx.size else 0
        B, Hq, D = kv.q.shape
        self.B, self.Hq, self.D = B, Hq, D

    def attn(self, tokens_per_split=0, use_bf16_pools=None, with_lse=True, out=None, key_order=0):
        B, Hq, D = self.B, self.Hq, self.D
        if out is None:
            out = torch.full((B, Hq, D), 0x7FC0, dtype=torch.int16, device="cuda")
        lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device="cuda") if with_lse else None
        ws = hma.alloc_workspace(B, Hq, self.kv.num_kv_heads, self.max_ctx, tokens_per_split)
        use = (self.k_bf16 is not None) if use_bf16_pools is None else use_bf16_pools
        hma.decode_attn_bfp8(self.q, self.k_mant, self.k_exp, self.v_mant, self.v_exp, self.pt,
                             self.ctx, self.max_ctx, out,
                             k_bf16=self.k_bf16 if use else None,
                             v_bf16=self.v_bf16 if use else None, lse=lse,
                             scale=self.kv.scale, num_kv_heads=self.kv.num_kv_heads,
                             tokens_per_split=tokens_per_split, workspace=ws, key_order=key_order)
        torch.cuda.synchronize()
        return out, lse


def assert_attn_close(out_dev, lse_dev, ref_out, ref_lse, rows=None, what=""):
    """Elementwise |gpu - ref| <= ATOL + RTOL |ref| on the BF16 output."""
    got = bf16_bits_to_f64(out_dev)
    if rows is not None:
        got = got[rows]
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref_out)
    bound = ATOL + RTOL * np.abs(ref_out)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; max err "
                             f"{err.max():.3g}; first {idx.tolist()} got "
                             f"{[got[tuple(i)] for i in idx]} ref {[ref_out[tuple(i)] for i in idx]}")
    if lse_dev is not None:
        gl = lse_dev.cpu().numpy().astype(np.float64)
        if rows is not None:
            gl = gl[rows]
        fin = np.isfinite(ref_lse)
        assert np.array_equal(np.isneginf(gl), np.isneginf(ref_lse)), what
        np.testing.assert_allclose(gl[fin], ref_lse[fin], rtol=LSE_RTOL, atol=LSE_ATOL, err_msg=what)
    return float(err.max()) if err.size else 0.0
