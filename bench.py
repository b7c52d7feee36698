#!/usr/bin/env python3
"""Benchmark of the BFP8 deferred-dequantization decode path on one MI355X.

One step = the whole hot path over one batch of synthetic input, on one HIP
stream, inputs resident in HBM:
  * hma_decode_attn_bfp8 for every layer of the model (one decode token's
    attention over the paged BFP8 KV of the whole batch), then
  * hma_bfp8_dequant_pages rebuilding one request's K and V of every layer
    into the paged BF16 cache (a single launch over all 2 x layers pools).
For the trace mix (workload 4) every layer launch reads a page table in
which half the pages are already BF16, and each attention launch is
followed by the rebuild of that layer's freshly arrived BFP8 pages.

Prints ONE JSON line.  value = effective KV GB/s of the step: the bytes the
method must move (BFP8 pages at 1.0625 B/element, BF16 pages at 2 B/element,
plus Q, output and page table; for the rebuild, BFP8 read + BF16 written)
divided by the step time.  Per-kernel figures come from HIP events recorded
on the launch stream.  For the uniform workloads the attention launches of
all layers are captured once in a HIP graph and each step replays it between
one event pair (average launch duration, dispatch gaps included); the same
launches issued one by one are timed too (attn_us_per_layer_eager).
attn_us_p50/p99 come from a separate untimed pass with an event pair around
each launch.

Beside the step the line carries, for the uniform BFP8 workloads:
  read_ceiling  the read-only probes of libhma: the attention's BFP8 bytes
                read in the attention's decomposition and with the heads of a
                page read together, and a flat 1 GiB streaming read;
  route_legs    one layer timed on codes that force the ldexp decode route,
                on the headline's codes (packed route) under the same
                repetition scheme, and (with the CPU baseline) on the oracle
                encoder's codes of the workload's value distribution.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload 3] [--eager]
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

HBM_PEAK_GBPS = 8000.0
PAGE_ID_MASK = 0x3FFFFFFF
KERNEL_SOURCES = ["paper_2606_29986_amd/csrc/decode_attn.hip",
                  "paper_2606_29986_amd/csrc/bfp8_dequant.hip",
                  "paper_2606_29986_amd/csrc/hma_device.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_hash(path: str) -> str:
    h = hashlib.sha256()
    for p in (path, "paper_2606_29986_amd/csrc/hma_device.h"):
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


# ------------------------------------------------------------ byte accounting

def bfp8_bytes_per_token_layer(hkv: int, d: int = 128) -> int:
    """K + V bytes of one token of one layer in BFP8 (1 + 1/16 B per element)."""
    return 2 * hkv * (d + d // 16)


def bf16_bytes_per_token_layer(hkv: int, d: int = 128) -> int:
    return 2 * hkv * d * 2


def attn_bytes(w: wl.Workload, ctx: np.ndarray, bf16_tokens: int = 0) -> int:
    """Algorithmic bytes of one attention launch: KV pages read (by format),
    Q read, output written, page-table entries and context lengths read."""
    tokens = int(ctx.sum())
    kv = (tokens - bf16_tokens) * bfp8_bytes_per_token_layer(w.num_kv_heads, w.head_dim) \
        + bf16_tokens * bf16_bytes_per_token_layer(w.num_kv_heads, w.head_dim)
    qo = 2 * w.batch * w.num_q_heads * w.head_dim * 2
    pt = int(wl.pages_per_seq(ctx, w.page_size).sum()) * 4 + w.batch * 4
    return kv + qo + pt


def dequant_bytes(w: wl.Workload, n_pages: int, n_pools: int) -> int:
    """BFP8 read + BF16 written + page ids, for n_pages pages of n_pools pools."""
    tile = w.page_size * w.head_dim
    per_page = w.num_kv_heads * (tile + tile // 16 + 2 * tile)
    return n_pools * n_pages * per_page + 2 * 4 * n_pages


# -------------------------------------------------------------- CPU baseline

def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _omp_threads(n: int) -> bool:
    """Set the OpenMP thread count of this thread's later parallel regions
    (the oracle's libgomp is the process's)."""
    import ctypes
    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))
        return True
    except OSError:
        return False


def _time_loop(fn, budget_s: float, min_reps: int = 1):
    reps, t0 = 0, time.perf_counter()
    while True:
        fn()
        reps += 1
        elapsed = time.perf_counter() - t0
        if reps >= min_reps and elapsed >= budget_s:
            return reps, elapsed


def cpu_baseline(w: wl.Workload, budget_s: float = 12.0, one_thread_budget_s: float = 5.0,
                 rebuild_budget_s: float = 3.0):
    """Time the float64 oracle (as it stands) on a bounded sample of the same
    workload: one layer of the whole batch, run repeatedly for ~budget_s with
    every host thread, then the first sequence of that layer with one thread,
    then the oracle's page rebuild of request 0's K pages.  Returns the report
    and the encoded layer (the oracle encoder's codes of the workload's value
    distribution, reused by the encoded-values leg)."""
    import oracle
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from oracle_fixtures import make_paged  # test infrastructure (value draws + encode)
    kv = make_paged(w, with_bf16_pool=False)
    cores = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))

    def attn(nseq):
        oracle.decode_attn(kv.q[:nseq], kv.k_mant, kv.k_exp, kv.v_mant, kv.v_exp, None, None,
                           kv.page_table[:nseq], kv.ctx[:nseq], kv.num_kv_heads, kv.page_size, kv.scale)

    reps, elapsed = _time_loop(lambda: attn(w.batch), budget_s)
    nbytes = reps * attn_bytes(w, kv.ctx)
    res = {"value": round(nbytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": cores,
           "kind": "oracle",
           "sample": f"float64 oracle attention over one layer of the full batch "
                     f"({int(kv.ctx.sum())} tokens, {w.num_q_heads} heads), {reps} runs "
                     f"in {elapsed:.1f} s; same byte accounting as the GPU figure",
           "cpu_model": cpu_model()}
    if _omp_threads(1):
        try:
            sub = dataclasses.replace(w, batch=1)
            r1, e1 = _time_loop(lambda: attn(1), one_thread_budget_s)
            res["one_thread_value"] = round(r1 * attn_bytes(sub, kv.ctx[:1]) / e1 / 1e9, 4)
            res["one_thread_sample"] = (f"sequence 0 of the same layer ({int(kv.ctx[0])} tokens), "
                                        f"{r1} runs in {e1:.1f} s, one OpenMP thread")
        finally:
            _omp_threads(cores)
    n0 = int(wl.pages_per_seq(kv.ctx[:1], w.page_size)[0])
    ids = kv.page_table[0, :n0] & PAGE_ID_MASK
    km, kx = kv.k_mant[ids], kv.k_exp[ids]
    rr, er = _time_loop(lambda: oracle.decode_blocks(km, kx), rebuild_budget_s)
    res["rebuild_value"] = round(rr * dequant_bytes(w, n0, 1) / er / 1e9, 4)
    res["rebuild_sample"] = (f"oracle page rebuild of request 0's K pages of one layer ({n0} pages), "
                             f"{rr} runs in {er:.1f} s, {cores} threads; byte accounting of the "
                             f"GPU rebuild")
    return res, kv


def packed_route_share(kv) -> float:
    """Share of the (page, KV head) tiles read by the attention whose block
    exponents all lie in 7..133 (the packed decode route)."""
    used = np.concatenate([kv.page_table[b, :n] for b, n in
                           enumerate(wl.pages_per_seq(kv.ctx, kv.page_size))]) & PAGE_ID_MASK
    ok = np.ones((used.size, kv.num_kv_heads), dtype=bool)
    for ex in (kv.k_exp, kv.v_exp):
        e = ex[used].reshape(used.size, kv.num_kv_heads, -1)
        ok &= ((e >= 7) & (e <= 133)).all(axis=-1)
    return float(ok.mean())


def copy_probe(mib: int, reps: int = 5) -> None:
    """Plain device copy of a known size, for scaling HBM byte counters."""
    import torch
    n = mib << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "reps": reps}))


def ingress_experiment(w, ctx, n_requests, attn_launch, resident, stream, steps):
    """Decode steps (attention over every layer, on `stream`) alone, then
    while n_requests new requests of the workload's longest context arrive
    (the decode side of the layer-wise transfer pipeline): per layer, their
    raw BFP8 K and V pages are copied from pinned host memory and rebuilt
    into a BF16 cache, (a) by hma_ingress_rebuild on a side stream running
    concurrently with decode, and (b) by copies on a copy stream with each
    layer's rebuild slotted between two decode launches once its bytes have
    landed."""
    import torch
    import paper_2606_29986_amd as hma
    dev = torch.device("cuda", 0)
    n_pages = int(wl.pages_per_seq(np.array([int(ctx.max())]), w.page_size)[0])
    shape = (2, n_pages, w.num_kv_heads, w.page_size, w.head_dim)
    eshape = shape[:-1] + (w.head_dim // 16,)
    g = torch.Generator().manual_seed(7)
    host = []
    for layer in range(w.layers):          # one request's bytes, as the network delivers them
        m = torch.randint(0, 256, shape, dtype=torch.uint8, generator=g).pin_memory()
        e = torch.randint(124, 132, eshape, dtype=torch.uint8, generator=g).pin_memory()
        host.append((m, e))
    stage_m = torch.empty(shape, dtype=torch.uint8, device=dev)
    stage_e = torch.empty(eshape, dtype=torch.uint8, device=dev)
    dst = torch.empty((w.layers,) + shape, dtype=torch.int16, device=dev)
    side = torch.cuda.Stream(device=dev)
    req_bytes = w.layers * sum(int(t.numel()) for t in host[0])

    def decode_steps(k):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(k):
            for layer in range(w.layers):
                attn_launch(layer % resident)
        e1.record(stream)
        return e0, e1

    for _ in range(2):
        decode_steps(1)
    torch.cuda.synchronize()
    a0, a1 = decode_steps(steps)
    torch.cuda.synchronize()
    alone = a0.elapsed_time(a1) / steps
    # ingress alone
    i0 = torch.cuda.Event(enable_timing=True)
    i1 = torch.cuda.Event(enable_timing=True)
    i0.record(side)
    for layer in range(w.layers):
        hma.ingress_rebuild(host[layer][0], host[layer][1], stage_m, stage_e, dst[layer], None,
                            n_pools=2, dst_pool_stride_pages=n_pages,
                            num_kv_heads=w.num_kv_heads, stream=side)
    i1.record(side)
    torch.cuda.synchronize()
    ingress_alone_ms = i0.elapsed_time(i1)
    # (a) side stream: hma_ingress_rebuild (copy + rebuild) for n_requests
    #     requests runs concurrently with decode
    s0 = torch.cuda.Event(enable_timing=True)
    s0.record(side)
    for _ in range(n_requests):
        for layer in range(w.layers):
            hma.ingress_rebuild(host[layer][0], host[layer][1], stage_m, stage_e, dst[layer], None,
                                n_pools=2, dst_pool_stride_pages=n_pages,
                                num_kv_heads=w.num_kv_heads, stream=side)
    s1 = torch.cuda.Event(enable_timing=True)
    s1.record(side)
    overlap_steps = max(1, int(n_requests * ingress_alone_ms / alone))
    b0, b1 = decode_steps(overlap_steps)
    torch.cuda.synchronize()
    both = b0.elapsed_time(b1) / overlap_steps
    side_res = {"decode_ms_per_step": round(both, 4), "decode_steps": overlap_steps,
                "decode_slowdown": round(both / alone - 1.0, 4),
                "ingress_ms_total": round(s0.elapsed_time(s1), 3)}
    del stage_m, stage_e

    # (b) interleaved: the copy engine moves every layer's bytes on a copy
    #     stream (no compute units); the decode loop rebuilds a layer between
    #     two attention launches once the host sees that layer's copy done
    copy = side
    stage_all_m = torch.empty((w.layers,) + shape, dtype=torch.uint8, device=dev)
    stage_all_e = torch.empty((w.layers,) + eshape, dtype=torch.uint8, device=dev)
    landed = [torch.cuda.Event() for _ in range(w.layers)]
    total_steps, step_ms, rebuilt = 0, [], 0
    for _ in range(n_requests):
        with torch.cuda.stream(copy):
            for layer in range(w.layers):
                stage_all_m[layer].copy_(host[layer][0], non_blocking=True)
                stage_all_e[layer].copy_(host[layer][1], non_blocking=True)
                landed[layer].record(copy)
        nxt = 0
        while nxt < w.layers:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for layer in range(w.layers):
                attn_launch(layer % resident)
                if nxt < w.layers and landed[nxt].query():
                    stream.wait_event(landed[nxt])
                    hma.bfp8_dequant_pages(stage_all_m[nxt], stage_all_e[nxt], dst[nxt], None, None,
                                           n_pages=n_pages, n_pools=2,
                                           src_pool_stride_pages=n_pages,
                                           dst_pool_stride_pages=n_pages,
                                           num_kv_heads=w.num_kv_heads, stream=stream)
                    nxt += 1
                    rebuilt += 1
            e1.record(stream)
            step_ms.append((e0, e1))
            total_steps += 1
    torch.cuda.synchronize()
    inter = float(np.mean([a.elapsed_time(b) for a, b in step_ms]))
    inter_res = {"decode_ms_per_step": round(inter, 4), "decode_steps": total_steps,
                 "layers_rebuilt": rebuilt, "decode_slowdown": round(inter / alone - 1.0, 4)}
    return {"requests": n_requests, "request_bytes": req_bytes,
            "ingress_ms_per_request_alone": round(ingress_alone_ms, 3),
            "ingress_GBps_alone": round(req_bytes / (ingress_alone_ms * 1e-3) / 1e9, 2),
            "decode_ms_per_step_alone": round(alone, 4),
            "side_stream": side_res, "interleaved": inter_res}


# --------------------------------------------------------------------- main

def _time_launches(torch, stream, fn, n, warm=2):
    """Average duration (us) of n back-to-back calls of fn(i) between one
    event pair on `stream`."""
    for i in range(warm):
        fn(i)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(n):
        fn(i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n


def read_ceiling(w, hma, torch, mant, expo, pt_d, ctx_d, max_ctx, tps, resident, stream, attn_us):
    """libhma's read-only probes: the BFP8 bytes of one attention launch read
    as one contiguous stream (every workload), and -- for the uniform-length
    workloads, whose attention runs the static split grid -- read from the
    pools in the attention's decomposition (one KV head per workgroup, the
    same splits) and with the KV heads of a page read together; plus a flat
    1 GiB read.  attn_over_* = attention launch time / probe time over the
    same bytes (the ragged batches run a page-balanced schedule that no
    static grid reproduces, so they get the stream figure only)."""
    kv_bytes = int(wl.pages_per_seq(wl.context_lens(w), w.page_size).sum()) * w.page_size \
        * bfp8_bytes_per_token_layer(w.num_kv_heads, w.head_dim)
    maxp = -(-max_ctx // w.page_size)
    dev = mant.device
    out = {"bytes_per_launch": kv_bytes}
    n16 = -(-kv_bytes // 16) * 16
    buf = torch.empty(3 * n16, dtype=torch.uint8, device=dev)
    buf.fill_(3)
    nwg = 4096
    sink = torch.empty(nwg * 4, dtype=torch.int32, device=dev)
    us = _time_launches(torch, stream, lambda i: hma.stream_read_probe(
        buf[(i % 3) * n16:(i % 3 + 1) * n16], sink, nwg, stream=stream), 30)
    out["stream_same_bytes"] = {"us": round(us, 3), "GBps": round(kv_bytes / (us * 1e-6) / 1e9, 1)}
    out["attn_over_stream_same_bytes"] = round(attn_us / us, 4)
    del buf
    if w.ctx[0] == "uniform":
        for name, hpw, pps in (("attn_decomposition", 1, tps // w.page_size),
                               ("heads_together", w.num_kv_heads, None)):
            if pps is None:                     # about one workgroup per CU
                ns = max(1, -(-256 // w.batch))
                pps = min(1024, -(-maxp // ns))
            ns = -(-maxp // pps)
            sink = torch.empty(w.batch * (w.num_kv_heads // hpw) * ns * 8, dtype=torch.int32, device=dev)

            def probe(i, hpw=hpw, pps=pps, ns=ns, sink=sink):
                slot = i % resident
                hma.paged_read_probe(mant[2 * slot], expo[2 * slot], mant[2 * slot + 1], expo[2 * slot + 1],
                                     pt_d, ctx_d, max_ctx, sink, num_kv_heads=w.num_kv_heads,
                                     pages_per_split=pps, n_splits=ns, heads_per_workgroup=hpw, stream=stream)
            us = _time_launches(torch, stream, probe, min(64, max(resident, 16)))
            out[name] = {"us": round(us, 3), "GBps": round(kv_bytes / (us * 1e-6) / 1e9, 1),
                         "heads_per_workgroup": hpw, "pages_per_split": pps, "splits": ns}
            out["attn_over_" + name] = round(attn_us / us, 4)
    buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    buf.fill_(3)
    sink = torch.empty(nwg * 4, dtype=torch.int32, device=dev)
    us = _time_launches(torch, stream, lambda i: hma.stream_read_probe(buf, sink, nwg, stream=stream), 10)
    out["stream_1GiB"] = {"us": round(us, 1), "GBps": round((1 << 30) / (us * 1e-6) / 1e9, 1)}
    del buf
    return out


def issue_ceiling(hma, torch, waves_per_simd=2, iters=2000):
    """libhma's issue probe with waves_per_simd waves on every SIMD.  A SIMD's
    time is its last wave's (the older wave is favoured and finishes first),
    so each figure is the largest per-wave cycle count over all the work the
    SIMD's waves issued: SIMD cycles per step of one 16x16x32 BF16 matrix
    instruction, of 8 plain adds, and of both; and SIMD cycles per
    instruction of each VALU kind the decode and softmax issue."""
    dev = torch.device("cuda", 0)
    n = 1024 * waves_per_simd
    cyc = torch.zeros(n, dtype=torch.int64, device=dev)
    sink = torch.zeros(n * 64, dtype=torch.int32, device=dev)

    def run(kind, valu, mfma):
        hma.issue_probe(kind, valu, mfma, waves_per_simd, 200, cyc, sink)     # warm-up
        hma.issue_probe(kind, valu, mfma, waves_per_simd, iters, cyc, sink)
        torch.cuda.synchronize()
        return float(cyc.max().item()) / (iters * 8) / waves_per_simd
    out = {"waves_per_simd": waves_per_simd, "unit": "SIMD shader cycles (last wave)"}
    out["mfma"] = round(run(0, 0, 1), 2)
    out["valu8"] = round(run(0, 8, 0), 2)
    out["mfma_plus_valu8"] = round(run(0, 8, 1), 2)
    out["per_instruction"] = {name: round(run(k, 16, 0) / 16, 2) for k, name in enumerate(hma.ISSUE_KINDS)}
    return out


def route_legs(w, hma, torch, total_pages, pt_d, ctx_d, max_ctx, q, tps, scale, stream, a_bytes):
    """One attention layer timed on codes that force the ldexp decode route
    (every page carries one block exponent of 134), against the headline's
    codes (exponents 124..131: packed route), both cycling over 4 resident
    layers so that no layer is re-read from the caches."""
    dev = q.device
    out = {}
    ws = hma.alloc_workspace(w.batch, w.num_q_heads, w.num_kv_heads, max_ctx, tps, device=dev)
    o = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.int16, device=dev)
    for route in ("packed", "ldexp"):
        pools = []
        for layer in range(4):
            km, kx = wl.bfp8_codes_device(w, layer, "k", total_pages, dev, route=route)
            vm, vx = wl.bfp8_codes_device(w, layer, "v", total_pages, dev, route=route)
            pools.append((km, kx, vm, vx))

        def launch(i, pools=pools):
            km, kx, vm, vx = pools[i % 4]
            hma.decode_attn_bfp8(q[i % q.shape[0]], km, kx, vm, vx, pt_d, ctx_d, max_ctx, o, scale=scale,
                                 num_kv_heads=w.num_kv_heads, tokens_per_split=tps, workspace=ws,
                                 stream=stream)
        us = _time_launches(torch, stream, launch, 32)
        out[route + "_route_us"] = round(us, 3)
        out[route + "_route_GBps"] = round(a_bytes / (us * 1e-6) / 1e9, 1)
        del pools
    out["ldexp_over_packed"] = round(out["ldexp_route_us"] / out["packed_route_us"], 4)
    return out


def encoded_values_leg(w, hma, torch, kv, tps, stream, a_bytes):
    """The layer the CPU baseline encoded (the oracle encoder's codes of the
    workload's value distribution, outlier channels included), uploaded as 4
    copies and timed like the route legs; with the share of its (page, KV
    head) tiles that take the packed route."""
    dev = torch.device("cuda", 0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    pools = [(t(kv.k_mant), t(kv.k_exp), t(kv.v_mant), t(kv.v_exp)) for _ in range(4)]
    qd = t(kv.q.view(np.int16))
    ptd, cd = t(kv.page_table), t(kv.ctx)
    max_ctx = int(kv.ctx.max())
    ws = hma.alloc_workspace(w.batch, w.num_q_heads, w.num_kv_heads, max_ctx, tps, device=dev)
    o = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.int16, device=dev)

    def launch(i):
        km, kx, vm, vx = pools[i % 4]
        hma.decode_attn_bfp8(qd, km, kx, vm, vx, ptd, cd, max_ctx, o, scale=kv.scale,
                             num_kv_heads=w.num_kv_heads, tokens_per_split=tps, workspace=ws, stream=stream)
    us = _time_launches(torch, stream, launch, 32)
    return {"encoded_values_us": round(us, 3), "encoded_values_GBps": round(a_bytes / (us * 1e-6) / 1e9, 1),
            "encoded_packed_route_share": round(packed_route_share(kv), 4)}


def valu_leg(w, hma, torch, mant, expo, pt_d, ctx_d, max_ctx, q, scale, resident, stream, a_bytes, attn_us):
    """The same attention launches (resident layers cycled, automatic ranges)
    through libhma's vector-ALU comparison kernel, which runs both products on
    v_dot2c / FMA instead of the matrix cores; valu_over_mfma = its time per
    launch / the fused kernel's."""
    dev = q.device
    n = hma.valu_workspace_bytes(w.batch, w.num_q_heads, w.num_kv_heads, max_ctx)
    ws = torch.empty(max(n, 256), dtype=torch.uint8, device=dev)
    o = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.int16, device=dev)

    def launch(i):
        s = i % resident
        hma.decode_attn_bfp8_valu(q[s], mant[2 * s], expo[2 * s], mant[2 * s + 1], expo[2 * s + 1], pt_d, ctx_d,
                                  max_ctx, o, ws, scale=scale, num_kv_heads=w.num_kv_heads, stream=stream)
    us = _time_launches(torch, stream, launch, min(64, max(resident, 16)))
    return {"valu_us": round(us, 3), "valu_GBps": round(a_bytes / (us * 1e-6) / 1e9, 1),
            "valu_over_mfma": round(us / attn_us, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--tokens-per-split", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="time the attention launches issued one by one (no HIP graph)")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the read-ceiling probes and the decode-route legs")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--kv-format", choices=["bfp8", "bf16"], default="bfp8",
                    help="bf16: every page is already BF16 and the step is attention only "
                         "(the dequant-free baseline)")
    ap.add_argument("--ingress-requests", type=int, default=0,
                    help="also measure decode steps while this many new requests' raw BFP8 "
                         "pages stream in from pinned host memory and are rebuilt on a side "
                         "stream (hma_ingress_rebuild, one call per layer)")
    ap.add_argument("--resident-layers", type=int, default=0,
                    help="layers kept resident (0 = all that the workload defines, 8 for the trace mix)")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the batch of a uniform-length workload (capacity comparisons)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return

    import torch
    import paper_2606_29986_amd as hma

    w = wl.WORKLOADS[args.workload]
    if args.batch:
        if w.ctx[0] != "uniform":
            print(json.dumps({"error": "--batch applies to the uniform-length workloads"}))
            sys.exit(2)
        w = dataclasses.replace(w, batch=args.batch, name="%s-batch%d" % (w.name, args.batch))
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = wl.context_lens(w)
    pt_np, total_pages = wl.page_table(w, ctx)
    max_ctx = int(ctx.max())
    mixed = w.bf16_page_fraction > 0
    all_bf16 = args.kv_format == "bf16"
    if all_bf16 and mixed:
        print(json.dumps({"error": "--kv-format bf16 applies to the uniform-format workloads"}))
        sys.exit(2)
    resident = args.resident_layers or (8 if mixed else w.layers)
    n_pools = 2 * resident

    # ---- resident inputs: one allocation per stream, pool p = 2*layer + (0: K, 1: V)
    # (the all-BF16 baseline never reads BFP8 pools: one page of each stands in)
    bfp8_pages = 1 if all_bf16 else total_pages
    mant = torch.empty((n_pools, bfp8_pages, w.num_kv_heads, w.page_size, w.head_dim),
                       dtype=torch.uint8, device=dev)
    expo = torch.empty((n_pools, bfp8_pages, w.num_kv_heads, w.page_size, w.head_dim // 16),
                       dtype=torch.uint8, device=dev)
    for layer in range(0 if all_bf16 else resident):
        for kind, off in (("k", 0), ("v", 1)):
            m, e = wl.bfp8_codes_device(w, layer, kind, total_pages, dev)
            mant[2 * layer + off].copy_(m)
            expo[2 * layer + off].copy_(e)
            del m, e
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + w.index)
    q = torch.randn((resident, w.batch, w.num_q_heads, w.head_dim), generator=g, device=dev)
    q = q.to(torch.bfloat16).view(torch.int16).contiguous()
    out = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.int16, device=dev)
    ctx_d = torch.from_numpy(ctx).to(dev)

    bf16_tokens = 0
    if all_bf16:
        bf16 = torch.empty((n_pools, total_pages, w.num_kv_heads, w.page_size, w.head_dim),
                           dtype=torch.int16, device=dev)
        bf16.random_(-32768, 32767, generator=g)
        bf16 &= 0x3FFF                       # finite BF16 patterns
        tagged = pt_np | wl.TAG_BF16
        pt_d = torch.from_numpy(tagged.astype(np.int32)).to(dev)
        bf16_tokens = int(ctx.sum())
        dq_pages = 0
    elif mixed:
        # BF16 pool per resident layer and stream; tagged pages read it
        mask = wl.bf16_page_mask(w, total_pages)
        bf16 = torch.empty((n_pools, total_pages, w.num_kv_heads, w.page_size, w.head_dim),
                           dtype=torch.int16, device=dev)
        bf16.random_(-32768, 32767, generator=g)
        bf16 &= 0x3FFF                       # finite BF16 patterns
        tagged = pt_np.copy()
        npg = wl.pages_per_seq(ctx, w.page_size)
        for b in range(w.batch):
            sel = mask[pt_np[b, :npg[b]]]
            tagged[b, :npg[b]][sel] |= wl.TAG_BF16
            last_full = ctx[b] - (npg[b] - 1) * w.page_size
            tok = np.full(npg[b], w.page_size)
            tok[-1] = last_full
            bf16_tokens += int(tok[sel].sum())
        pt_d = torch.from_numpy(tagged).to(dev)
        fresh = np.nonzero(~mask)[0].astype(np.int32)
        fresh_d = torch.from_numpy(fresh).to(dev)
        dq_pages = len(fresh)
    else:
        pt_d = torch.from_numpy(pt_np).to(dev)
        # standalone rebuild of request 0 of every layer into a BF16 cache
        req_pages = pt_np[0, :int(wl.pages_per_seq(ctx[:1], w.page_size)[0])].astype(np.int32)
        src_d = torch.from_numpy(req_pages).to(dev)
        dst_d = torch.arange(len(req_pages), dtype=torch.int32, device=dev)
        dq_pages = len(req_pages)
        bf16_dst = torch.empty((n_pools, dq_pages, w.num_kv_heads, w.page_size, w.head_dim),
                               dtype=torch.int16, device=dev)
    # the library's own choice (0) unless a split length is forced; tps is the
    # split length that choice amounts to (the ragged batches run the
    # page-balanced schedule instead)
    tps_arg = args.tokens_per_split
    tps = tps_arg or hma.tokens_per_split(w.batch, w.num_q_heads, w.num_kv_heads, max_ctx)
    ws = hma.alloc_workspace(w.batch, w.num_q_heads, w.num_kv_heads, max_ctx, tps_arg, device=dev)
    scale = wl.softmax_scale(w)
    stream = torch.cuda.current_stream()

    def attn_launch(layer_slot):
        hma.decode_attn_bfp8(
            q[layer_slot], mant[2 * layer_slot], expo[2 * layer_slot], mant[2 * layer_slot + 1],
            expo[2 * layer_slot + 1], pt_d, ctx_d, max_ctx, out,
            k_bf16=bf16[2 * layer_slot] if (mixed or all_bf16) else None,
            v_bf16=bf16[2 * layer_slot + 1] if (mixed or all_bf16) else None,
            scale=scale, num_kv_heads=w.num_kv_heads, tokens_per_split=tps_arg, workspace=ws)

    def dequant_launch(layer_slot=None):
        if mixed:       # this layer's fresh pages, K and V (two pools at stride total_pages)
            hma.bfp8_dequant_pages(mant[2 * layer_slot], expo[2 * layer_slot], bf16[2 * layer_slot],
                                   fresh_d, fresh_d, n_pools=2, src_pool_stride_pages=total_pages,
                                   dst_pool_stride_pages=total_pages, num_kv_heads=w.num_kv_heads,
                                   stream=stream)
        else:           # request 0 of every layer, K and V: one launch over all pools
            hma.bfp8_dequant_pages(mant, expo, bf16_dst, src_d, dst_d, n_pools=n_pools,
                                   src_pool_stride_pages=total_pages,
                                   dst_pool_stride_pages=dq_pages, num_kv_heads=w.num_kv_heads,
                                   stream=stream)

    n_launch = w.layers
    events = []

    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record(stream)
        return e

    def step(record, per_launch=False):
        """One pass of the path.  Uniform workloads: the attention launches of
        all layers run back to back and are bracketed by one event pair (their
        average is the per-launch duration, dispatch gaps included), then the
        rebuild launch has its own pair.  With per_launch (a separate,
        untimed pass) every attention launch gets its own pair, for the
        latency distribution.  Mixed workload: attention and rebuild alternate
        per layer, each launch bracketed."""
        evs = []
        if mixed:
            for layer in range(n_launch):
                slot = layer % resident
                e0 = ev() if record else None
                attn_launch(slot)
                e1 = ev() if record else None
                dequant_launch(slot)
                if record:
                    evs.append(("attn", e0, e1, 1))
                    evs.append(("dq", e1, ev(), 1))
        else:
            if record and not per_launch:
                e0 = ev()
            if graph is not None and not per_launch:
                graph.replay()
            else:
                for layer in range(n_launch):
                    if per_launch:
                        a0 = ev()
                    attn_launch(layer % resident)
                    if per_launch:
                        evs.append(("attn", a0, ev(), 1))
            if record and not per_launch:
                e1 = ev()
                evs.append(("attn", e0, e1, n_launch))
            if not all_bf16:
                dequant_launch()
                if record and not per_launch:
                    evs.append(("dq", e1, ev(), 1))
        return evs

    graph = None
    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    if not mixed and not args.eager:
        # the attention launches of all layers, captured once (they allocate
        # nothing and clear nothing: the split counters are left at zero by
        # every launch) and replayed by every step
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for layer in range(n_launch):
                attn_launch(layer % resident)
        torch.cuda.synchronize()
        for _ in range(max(1, args.warmup)):
            step(False)
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        events.append(step(True))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    attn_us, dq_us = [], []
    for evs in events:
        for kind, e0, e1, n in evs:
            (attn_us if kind == "attn" else dq_us).append(e0.elapsed_time(e1) * 1e3 / n)
    attn_us = np.array(attn_us)
    dq_us = np.array(dq_us)
    eager_us = None
    if graph is not None:
        # the same launches issued one by one (outside the timed region)
        pairs = []
        for _ in range(max(3, args.steps // 2)):
            e0 = ev()
            for layer in range(n_launch):
                attn_launch(layer % resident)
            pairs.append((e0, ev()))
        torch.cuda.synchronize()
        eager_us = float(np.mean([a.elapsed_time(b) * 1e3 / n_launch for a, b in pairs]))
    # latency distribution over single launches (outside the timed region)
    if mixed:
        single = attn_us
    else:
        evs = step(True, per_launch=True)
        torch.cuda.synchronize()
        single = np.array([e0.elapsed_time(e1) * 1e3 for _, e0, e1, _ in evs])

    a_bytes = attn_bytes(w, ctx, bf16_tokens)
    if all_bf16:
        d_bytes = 0
        step_bytes = n_launch * a_bytes
    elif mixed:
        d_bytes = dequant_bytes(w, dq_pages, 2)
        step_bytes = n_launch * (a_bytes + d_bytes)
    else:
        d_bytes = dequant_bytes(w, dq_pages, n_pools)
        step_bytes = n_launch * a_bytes + d_bytes
    ms_per_step = wall / args.steps * 1e3
    value = step_bytes / (wall / args.steps) / 1e9
    attn_mean = float(attn_us.mean())
    attn_gbps = a_bytes / (attn_mean * 1e-6) / 1e9

    traffic = None
    try:
        tf = json.load(open(TRAFFIC_FILE))
        ent = tf.get("decode_attn_bfp8", {}).get(w.name)
        if ent and ent.get("kernel_hash") == kernel_hash(KERNEL_SOURCES[0]) and not all_bf16:
            traffic = ent["bytes_per_launch"]
    except (OSError, ValueError):
        pass

    res = {
        "metric": "effective KV GB/s (fraction of HBM peak) + decode-attention us/layer, "
                  "Qwen3-32B 8K",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded BFP8 codes drawn on the device; no dataset)",
        "config": {
            "workload": w.name, "batch": w.batch, "context": "uniform %d" % max_ctx
            if w.ctx[0] == "uniform" else "ragged, max %d, total %d" % (max_ctx, int(ctx.sum())),
            "layers": w.layers, "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim, "page_size": w.page_size,
            "tokens_per_split": tps_arg if tps_arg else "automatic (%d)" % tps,
            "resident_layers": resident, "bf16_page_fraction": w.bf16_page_fraction,
            "kv_format": "bf16 (every page already BF16)" if all_bf16 else
                         ("mixed" if mixed else "bfp8"),
            "step": ("attention over %d layers, every page already BF16 (dequant-free baseline)"
                     % n_launch) if all_bf16 else
                    ("attention over %d layers (mixed BF16/BFP8 pages) + per-layer rebuild of "
                     "fresh pages" % n_launch) if mixed else
                    ("attention over %d layers + one launch rebuilding request 0's K/V of all "
                     "%d layers (%d pages each)" % (n_launch, w.layers, dq_pages)),
        },
        "attn_us_per_layer": round(attn_mean, 3),
        "attn_launch": "hip graph of the %d layer launches, replayed per step" % n_launch
                       if graph is not None else "launched one by one",
        "attn_us_per_layer_eager": round(eager_us, 3) if eager_us is not None else round(attn_mean, 3),
        "attn_us_p50": round(float(np.percentile(single, 50)), 3),
        "attn_us_p99": round(float(np.percentile(single, 99)), 3),
        "attn_GBps": round(attn_gbps, 2),
        "attn_frac_hbm_peak": round(attn_gbps / HBM_PEAK_GBPS, 4),
        "dequant_us": round(float(dq_us.mean()), 3) if dq_us.size else None,
        "dequant_us_p99": round(float(np.percentile(dq_us, 99)), 3) if dq_us.size else None,
        "dequant_GBps": round(d_bytes / (float(dq_us.mean()) * 1e-6) / 1e9, 2) if dq_us.size else None,
        "roofline": {"bound": "hbm", "achieved": round(attn_gbps, 2), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": traffic,
                     "kernel": "decode_attn_bfp8_kernel",
                     "algorithmic_bytes_per_launch": a_bytes},
    }
    if not mixed and not all_bf16:
        # the same rebuild through the one-thread-per-element baseline (Sec. 3.3
        # sets a naive elementwise reconstruction against the fused pass)
        n0 = torch.cuda.Event(enable_timing=True)
        n1 = torch.cuda.Event(enable_timing=True)
        n0.record(stream)
        hma.bfp8_dequant_pages(mant, expo, bf16_dst, src_d, dst_d, n_pools=n_pools,
                               src_pool_stride_pages=total_pages, dst_pool_stride_pages=dq_pages,
                               num_kv_heads=w.num_kv_heads, stream=stream, naive=True)
        n1.record(stream)
        torch.cuda.synchronize()
        naive_us = n0.elapsed_time(n1) * 1e3
        res["naive_rebuild_us"] = round(naive_us, 1)
        res["naive_over_fused_rebuild"] = round(naive_us / float(dq_us.mean()), 2)
        # the same request from tiled per-chip shards (4 prefill chips), keys
        # re-laid out from interleaved to half-split rotary order
        n_req_tok = int(ctx[0])
        shards = 4 if w.num_kv_heads % 4 == 0 else 1
        pool_bytes = shards * hma.tiled_shard_bytes(n_req_tok, w.num_kv_heads // shards)
        tiled_src = torch.randint(0, 256, (2, resident, pool_bytes), dtype=torch.uint8, device=dev)
        t_us = []
        for _ in range(3):
            t0_ = torch.cuda.Event(enable_timing=True)
            t1_ = torch.cuda.Event(enable_timing=True)
            t0_.record(stream)
            for kind in (0, 1):
                hma.bfp8_rebuild_tiled(tiled_src[kind], bf16_dst[kind], n_req_tok, shards,
                                       n_pools=resident, src_pool_stride_bytes=pool_bytes,
                                       dst_pool_stride_pages=2 * dq_pages, rope_reorder=(kind == 0),
                                       num_kv_heads=w.num_kv_heads, stream=stream)
            t1_.record(stream)
            torch.cuda.synchronize()
            t_us.append(t0_.elapsed_time(t1_) * 1e3)
        tiled_bytes = 2 * resident * (pool_bytes + n_req_tok * w.num_kv_heads * w.head_dim * 2)
        res["tiled_rebuild_us"] = round(float(np.median(t_us)), 1)
        res["tiled_rebuild_GBps"] = round(tiled_bytes / (float(np.median(t_us)) * 1e-6) / 1e9, 2)
        del tiled_src
    legs = not mixed and not all_bf16 and not args.no_legs
    if legs:
        res["read_ceiling"] = read_ceiling(w, hma, torch, mant, expo, pt_d, ctx_d, max_ctx, tps, resident,
                                           stream, attn_mean)
        res["issue_ceiling"] = issue_ceiling(hma, torch)
        res["route_legs"] = route_legs(w, hma, torch, total_pages, pt_d, ctx_d, max_ctx, q, tps_arg, scale,
                                       stream, a_bytes)
        if w.num_q_heads // w.num_kv_heads <= 8:
            res["valu_leg"] = valu_leg(w, hma, torch, mant, expo, pt_d, ctx_d, max_ctx, q, scale, resident,
                                       stream, a_bytes, attn_mean)
    # a plain 1 GiB device copy on the same box: the attention rate as a
    # fraction of what a copy (read + write) reaches here
    cp_a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    cp_a.fill_(1)
    cp_b = torch.empty_like(cp_a)
    cp_us = []
    for rep in range(6):
        c0_, c1_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            c0_.record(stream)
            cp_b.copy_(cp_a)
            c1_.record(stream)
        torch.cuda.synchronize()
        if rep:
            cp_us.append(c0_.elapsed_time(c1_) * 1e3)
    copy_gbps = 2 * (1 << 30) / (float(np.median(cp_us)) * 1e-6) / 1e9
    res["copy_GBps"] = round(copy_gbps, 1)
    res["attn_frac_copy"] = round(attn_gbps / copy_gbps, 4)
    del cp_a, cp_b
    if args.ingress_requests and not mixed and not all_bf16:
        res["ingress"] = ingress_experiment(w, ctx, args.ingress_requests, attn_launch, resident,
                                            stream, max(args.steps, 10))
    if not args.no_cpu_baseline and not all_bf16:
        res["cpu_baseline"], enc = cpu_baseline(w)
        if legs:
            res["route_legs"].update(encoded_values_leg(w, hma, torch, enc, tps_arg, stream, a_bytes))
        del enc
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
