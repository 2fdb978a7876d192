#!/usr/bin/env python3
"""Benchmark of one device's share of an ATP transformer layer on MI355X.

A step is one pass of the whole hot path on one batch: the block forward
(QKV, out-proj, fc1+GeLU, fc2 local GEMMs with chunked Partial(SUM)
reductions overlapping the next chunk's GEMM, Sec. 3.2.1 / Sec. 4.1) and the
block backward (dX chunks with overlapped reductions, dW, db; Sec. 4.2).
The other group members' partial buffers are seeded inputs resident in
HBM (one GPU stands in for the mesh).  Default workload: h = 20480,
4096 tokens, DeviceMesh(8, 1), column-first block, 8 chunks.

Prints ONE JSON line on stdout; diagnostics go to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)

METRIC = "TFLOP/s per GPU, chunked 2D-TP shard MLP+attn-proj block; MFMA util %"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
DEFAULT_WORKLOAD = "wide_h20480_col_8x1"
LIN = ("qkv", "out", "fc1", "fc2")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--chunks", type=int, default=None, help="override the chunk count")
    ap.add_argument("--bwd-chunks", type=int, default=1,
                    help="chunk count of the backward call.  The paper chunks the forward "
                         "only (Sec. 4.1); in the backward each linear's dX all-reduce "
                         "overlaps the dW products (Sec. 4.2), which is 1 here")
    ap.add_argument("--mesh", default=None,
                    help="override the workload's mesh, as D1xD2 (one device's share of it)")
    ap.add_argument("--fwd-only", action="store_true", help="time the forward only")
    ap.add_argument("--serial", action="store_true",
                    help="run reductions on the compute stream (no overlap)")
    ap.add_argument("--no-workspace", action="store_true",
                    help="no workspace: chunk products are never split over k")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step as a captured HIP graph (measured slower than "
                         "launching it: the replay loses part of the reduce/GEMM overlap)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=384,
                    help="token rows in the oracle's timed CPU sample")
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(reference kernel for scaling HBM counters)")
    ap.add_argument("--attention", action="store_true",
                    help="time the attention core (fwd+bwd) of one device's heads instead of "
                         "the linear block: sequences of min(2048, tokens), head dim 128")
    ap.add_argument("--attention-block", action="store_true",
                    help="time the attention block of one device instead: QKV and out-proj "
                         "with their chunked reductions around the causal core, fwd+bwd")
    ap.add_argument("--linear", action="store_true",
                    help="time one reduced linear of the block (fc2: the largest reduction) "
                         "as the chunked pipeline with f32 and with bf16 partials, serialized, "
                         "unchunked, and with the reduction fused into the GEMM epilogue")
    ap.add_argument("--weight-layout", choices=("kn", "nk"), default="kn",
                    help="local weights stored [k, n] (the paper's Y = XW) or [n, k] "
                         "(torch.nn.Linear's order)")
    ap.add_argument("--partials", choices=("f32", "bf16"), default="f32",
                    help="Partial(SUM) buffers in fp32 or bf16 (Sec. 5's 16-bit all-reduce)")
    ap.add_argument("--comm-cus", type=int, default=0,
                    help="run the reductions on a comm stream restricted to this many CUs "
                         "(hipExtStreamCreateWithCUMask; 0 = all CUs)")
    ap.add_argument("--pad", type=int, default=0,
                    help="elements added to the row pitch of every activation, gradient, "
                         "weight and partial buffer")
    ap.add_argument("--seed", type=int, default=21)
    ap.add_argument("--profile-detail", action="store_true",
                    help="also print per-shape kernel timings to stderr")
    return ap.parse_args()


def setup(torch, atp, S, wl, chunks, seed, layout="kn", partials="f32", pad=0):
    """Device-resident seeded inputs and outputs of one device's share; every
    2-D buffer's rows are `pad` elements longer than its columns."""
    dev = "cuda:0"
    d1, d2 = wl["mesh"]
    m = atp.mesh(d1, d2, 0, 0)
    bm = atp.ATP_BLOCK_COL if wl["mode"] == "col" else atp.ATP_BLOCK_ROW
    h, T, sw = wl["h"], wl["tokens"], wl["sigma_w"]
    G = atp.block_geometry(m, bm, h)
    def padded(r, c, dt):
        return torch.empty((r, c + pad), dtype=dt, device=dev)[:, :c]

    def rnd(shape, std, tid, dt=torch.bfloat16):
        t = S.randn_device(shape, std, seed, tid, dev, dtype=dt)
        if pad == 0 or len(shape) != 2:
            return t
        out = padded(shape[0], shape[1], dt)
        out.copy_(t)
        return out
    kn = layout == "kn"
    pdt = torch.float32 if partials == "f32" else torch.bfloat16
    st = dict(m=m, bm=bm, G=G, T=T, h=h, chunks=chunks,
              layout=atp.ATP_W_KN if kn else atp.ATP_W_NK)
    st["x"] = rnd((T, G[0].k_loc), 1.0, S.TID["x"])
    st["a"] = rnd((T, G[1].k_loc), 1.0, S.TID["a"])
    st["w"] = [rnd((g.k_loc, g.n_loc), sw, S.TID["w_" + n]) for g, n in zip(G, LIN)]
    if not kn:
        st["w"] = [padded(w.shape[1], w.shape[0], w.dtype).copy_(w.t()) for w in st["w"]]
    st["b"] = [torch.zeros(g.n_loc, dtype=torch.bfloat16, device=dev) for g in G]
    emp = lambda r, c, dt=torch.bfloat16: padded(r, c, dt)  # noqa: E731
    st["fwd_tabs"], st["bwd_tabs"] = [], []
    for i, g in enumerate(G):
        if g.red_size > 1:
            sp = S.peer_sigma(g.k_loc, sw, 1.0)
            tab = [padded(T, g.n_loc, pdt).copy_(
                       rnd((T, g.n_loc), sp, S.PEER_TID_BASE + 100 * i + j, torch.float32))
                   for j in range(g.red_size)]
            st["fwd_tabs"].append(tab)        # entry red_index is overwritten (own)
        else:
            st["fwd_tabs"].append(None)
        if g.bwd_size > 1:
            sp = S.peer_sigma(g.n_loc, sw, 1.0)
            tab = [padded(T, g.k_loc, pdt).copy_(
                       rnd((T, g.k_loc), sp, S.BWD_PEER_TID_BASE + 100 * i + j, torch.float32))
                   for j in range(g.bwd_size)]
            st["bwd_tabs"].append(tab)
        else:
            st["bwd_tabs"].append(None)
    st["qkv"], st["o"] = emp(T, G[0].n_loc), emp(T, G[1].n_loc)
    st["hh"], st["pre"], st["z"] = emp(T, G[2].n_loc), emp(T, G[2].n_loc), emp(T, G[3].n_loc)
    st["dz"] = rnd((T, G[3].n_loc), 1.0, S.TID["dz"])
    st["dqkv"] = rnd((T, G[0].n_loc), 1.0, S.TID["dqkv"])
    st["do"] = rnd((T, G[1].n_loc), 1.0, S.TID["do"])
    st["dh_pre"] = emp(T, G[2].n_loc)
    st["dx_qkv"], st["dx_fc1"] = emp(T, G[0].k_loc), emp(T, G[2].k_loc)
    st["d_attn"] = emp(T, G[1].k_loc)
    st["dw"] = [padded(*((g.k_loc, g.n_loc) if kn else (g.n_loc, g.k_loc)), torch.float32)
                for g in G]
    st["db"] = [torch.empty((g.n_loc,), dtype=torch.float32, device=dev) for g in G]
    return st


def linear_bench(torch, atp, S, args, wl, chunks):
    """fc2 of the workload's block on one device (Sec. 3.2: row-first in the
    column-first block, reduced over its group with the bias): the paper's
    chunked overlap (Sec. 4.1) with f32 partials and with bf16 partials (the
    16-bit all-reduce of Sec. 5), the same serialized and unchunked, and the
    fused GEMM + reduction that Sec. 4.1 contrasts it with.  All variants
    run the product from W as given (no transposed copy)."""
    dev = "cuda:0"
    d1, d2 = wl["mesh"]
    m = atp.mesh(d1, d2, 0, 0)
    bm = atp.ATP_BLOCK_COL if wl["mode"] == "col" else atp.ATP_BLOCK_ROW
    T, h, sw = wl["tokens"], wl["h"], wl["sigma_w"]
    G = atp.block_geometry(m, bm, h)
    L = 3
    g = G[L]
    mode = atp.ATP_ROW_FIRST if bm == atp.ATP_BLOCK_COL else atp.ATP_COL_FIRST
    K, N = 4 * h, h
    if g.red_size < 2:
        raise SystemExit(f"bench.py --linear: fc2 of {args.workload} has no reduction")
    rnd = lambda shape, std, tid, dt=torch.bfloat16: S.randn_device(  # noqa: E731
        shape, std, args.seed, tid, dev, dtype=dt)
    x = rnd((T, g.k_loc), 1.0, S.TID["h"])
    w = rnd((g.k_loc, g.n_loc), sw, S.TID["w_fc2"])
    bias = rnd((g.n_loc,), 0.02, S.TID["b_fc2"])
    sp = S.peer_sigma(g.k_loc, sw, 1.0)
    tab = [rnd((T, g.n_loc), sp, S.PEER_TID_BASE + 100 * L + j, torch.float32)
           for j in range(g.red_size)]
    tab16 = [t.to(torch.bfloat16) for t in tab]
    out = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=dev)
    evs = [atp.HipEvent() for _ in range(chunks)]
    side = torch.cuda.Stream()
    flops = 2.0 * T * g.k_loc * g.n_loc
    own = g.red_index

    def chunked(c, parts16, serial):
        def run():
            cs = torch.cuda.current_stream()
            ms = cs if serial else side
            t = tab16 if parts16 else tab
            atp.atp_shard_linear_fwd(m, mode, T, K, N, c, x, w, None, atp.ATP_EPI_NONE, t[own],
                                     stream=cs, chunk_done=None if serial else evs[:c])
            red = atp.atp_chunked_partial_reduce_bf16 if parts16 else \
                atp.atp_chunked_partial_reduce
            red(g.red_size, T, g.n_loc, c, t, bias, atp.ATP_EPI_BIAS, out, stream=ms,
                chunk_ready=None if serial else evs[:c])
            if not serial:
                e = torch.cuda.Event()
                e.record(ms)
                cs.wait_event(e)
        return run

    def fused():
        peers = [None if j == own else tab[j] for j in range(g.red_size)]
        atp.atp_shard_linear_fwd_fused(m, mode, T, K, N, x, w, peers, bias, atp.ATP_EPI_BIAS,
                                       out, stream=torch.cuda.current_stream())

    variants = [("chunked_f32", chunked(chunks, False, False)),
                ("chunked_f32_serial", chunked(chunks, False, True)),
                ("unchunked_f32", chunked(1, False, True)),
                ("chunked_bf16_partials", chunked(chunks, True, False)),
                ("fused_epilogue", fused)]
    res = {}
    for name, run in variants:
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            run()
        e1.record()
        torch.cuda.synchronize()
        ms_ = e0.elapsed_time(e1) / args.steps
        res[name] = dict(ms=round(ms_, 4), tflops=round(flops / (ms_ * 1e-3) / 1e12, 1))
        log(f"[linear] {name}: {res[name]}")
    base = res["chunked_f32"]["ms"]
    out_line = dict(
        metric="fc2 forward of one device (GEMM + reduction of its group), ms", value=base,
        unit="ms", n_gpus=1, steps=args.steps, warmup=args.warmup, higher_is_better=False,
        scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload=args.workload, linear="fc2", mesh=[d1, d2], tokens=T, h=h,
                    chunks=chunks, red_size=g.red_size, gemm=[T, g.k_loc, g.n_loc],
                    gflop=round(flops / 1e9, 1)),
        variants=res)
    print(json.dumps(out_line), flush=True)


def attention_bench(torch, atp, S, args, wl):
    """The attention core of one device (Sec. 3.2.1): its run of heads of
    the reduced QKV block, causal, forward then backward, K timed steps."""
    dev = "cuda:0"
    d1, d2 = wl["mesh"]
    m = atp.mesh(d1, d2, 0, 0)
    bm = atp.ATP_BLOCK_COL if wl["mode"] == "col" else atp.ATP_BLOCK_ROW
    h, T = wl["h"], wl["tokens"]
    heads = h // 128
    seq = min(2048, T)
    batch = T // seq
    T = batch * seq
    g = atp.block_geometry(m, bm, h)[0]
    first, hd, per_block = atp.attention_heads(m, bm, h, heads)
    rnd = lambda shape, tid: S.randn_device(shape, 1.0, args.seed, tid, dev)  # noqa: E731
    qkv = rnd((T, g.n_loc), 401)
    d_out = rnd((T, g.n_loc // 3), 402)
    out = torch.empty((T, g.n_loc // 3), dtype=torch.bfloat16, device=dev)
    d_qkv = torch.empty((T, g.n_loc), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((hd, T), dtype=torch.float32, device=dev)
    delta = torch.empty((hd * T,), dtype=torch.float32, device=dev)

    def step():
        atp.atp_attention_fwd(m, bm, batch, seq, h, heads, qkv, out, lse)
        atp.atp_attention_bwd(m, bm, batch, seq, h, heads, qkv, out, lse, d_out, d_qkv, delta)

    pairs = batch * hd * seq * (seq + 1) / 2.0
    flops = 2.0 * 128 * pairs * (2 + 5)       # forward QK^T, PV; backward five products
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = max(e0.elapsed_time(e1), (time.perf_counter() - t0) * 1e3) / args.steps
    value = flops / (ms_step * 1e-3) / 1e12
    atp.atp_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    atp.atp_profile_enable(False)
    kernels = []
    for r in atp.atp_profile_collect(16):
        kernels.append(dict(name=r["name"], avg_us=round(r["total_ms"] / r["launches"] * 1e3, 2),
                            tflops=round(r["flops"] / (r["total_ms"] * 1e-3) / 1e12, 1)))
    dom = max(kernels, key=lambda k: k["avg_us"])
    cpu = None
    if not args.no_cpu_baseline:
        import oracle as O
        import numpy as np
        q = qkv[:seq, first * 384:first * 384 + 384].float().cpu().numpy()
        t1 = time.perf_counter()
        o_ref, _ = O.attention_fwd(q[:, :128], q[:, 128:256], q[:, 256:])
        O.attention_bwd(q[:, :128], q[:, 128:256], q[:, 256:], np.ones_like(o_ref))
        sec = time.perf_counter() - t1
        cpu = dict(value=round(2.0 * 128 * seq * (seq + 1) / 2.0 * 7 / sec / 1e12, 6),
                   unit="TFLOP/s", cores=O.num_threads(), kind="oracle",
                   sample=f"one head, one {seq}-token sequence, forward and backward",
                   seconds=round(sec, 3))
    out_line = dict(
        metric="TFLOP/s, attention core fwd+bwd of one device's heads (causal)",
        value=round(value, 2), unit="TFLOP/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=round(ms_step, 4), higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="bf16", data="synthetic",
        config=dict(workload=args.workload, part="attention", mode=wl["mode"], mesh=[d1, d2],
                    coord=[0, 0], h=h, heads=heads, heads_per_device=hd, batch=batch, seq=seq,
                    gflop_per_step=round(flops / 1e9, 1)),
        roofline=dict(bound="mfma", kernel=dom["name"], achieved=dom["tflops"],
                      peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                      frac=round(dom["tflops"] / PEAK_BF16_TFLOPS, 4), traffic=None),
        kernels=kernels, cpu_baseline=cpu)
    print(json.dumps(out_line), flush=True)


def attention_block_bench(torch, atp, S, args, wl, chunks):
    """The attention block of one device (Sec. 3.2.1): QKV, its Partial(SUM)
    reduced over the group in chunks beside the next chunk's product
    (Sec. 4.1), the causal core on the device's heads, the out-proj reduced
    the same way; then the backward (Sec. 4.2).  The other members' partials
    and gathered columns are seeded inputs resident in HBM."""
    dev = "cuda:0"
    d1, d2 = wl["mesh"]
    m = atp.mesh(d1, d2, 0, 0)
    bm = atp.ATP_BLOCK_COL if wl["mode"] == "col" else atp.ATP_BLOCK_ROW
    h, T, sw = wl["h"], wl["tokens"], wl["sigma_w"]
    heads = h // 128
    seq = min(2048, T)
    batch = T // seq
    T = batch * seq
    gq, go = atp.block_geometry(m, bm, h)[:2]
    _, hd, _ = atp.attention_heads(m, bm, h, heads)
    bf = torch.bfloat16

    def rnd(shape, std, tid, dt=bf):
        return S.randn_device(shape, std, args.seed, tid, dev, dtype=dt)

    def table(size, cols, sigma, tid0):
        if size == 1:
            return None
        return [rnd((T, cols), sigma, tid0 + j, torch.float32) for j in range(size)]

    x = rnd((T, gq.k_loc), 1.0, 411)
    w = [rnd((gq.k_loc, gq.n_loc), sw, 412), rnd((go.k_loc, go.n_loc), sw, 413)]
    b = [torch.zeros(gq.n_loc, dtype=bf, device=dev), torch.zeros(go.n_loc, dtype=bf, device=dev)]
    qtab = table(gq.red_size, gq.n_loc, S.peer_sigma(gq.k_loc, sw, 1.0), 420)
    otab = table(go.red_size, go.n_loc, S.peer_sigma(go.k_loc, sw, 1.0), 440)
    atab = table(go.bwd_size, go.k_loc, S.peer_sigma(go.n_loc, sw, 1.0), 460)
    xtab = table(gq.bwd_size, gq.k_loc, S.peer_sigma(gq.n_loc, sw, 1.0), 480)
    qkv = torch.empty((T, gq.n_loc), dtype=bf, device=dev)
    attn = rnd((T, go.k_loc), 1.0, 414)        # the other members' gathered columns
    lse = torch.empty((hd, T), dtype=torch.float32, device=dev)
    o = torch.empty((T, go.n_loc), dtype=bf, device=dev)
    d_o = rnd((T, go.n_loc), 1.0, 415)
    d_attn = torch.empty((T, go.k_loc), dtype=bf, device=dev)
    delta = torch.empty((hd * T,), dtype=torch.float32, device=dev)
    d_qkv = rnd((T, gq.n_loc), 1.0, 416)       # the other members' columns
    dx = torch.empty((T, gq.k_loc), dtype=bf, device=dev)
    dw = [torch.empty((g.k_loc, g.n_loc), dtype=torch.float32, device=dev) for g in (gq, go)]
    db = [torch.empty((g.n_loc,), dtype=torch.float32, device=dev) for g in (gq, go)]
    comm = torch.cuda.Stream()
    bwd_chunks = args.bwd_chunks or chunks
    ws = None
    if not args.no_workspace:
        nb = atp.atp_block_workspace_bytes(m, bm, T, h, chunks, atp.ATP_W_KN)
        ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)

    def step():
        cs = torch.cuda.current_stream()
        atp.atp_attention_block_fwd(m, bm, batch, seq, h, heads, chunks, w, b, x, qtab, qkv,
                                    attn, lse, otab, o, workspace=ws, compute_stream=cs,
                                    comm_stream=comm)
        atp.atp_attention_block_bwd(m, bm, batch, seq, h, heads, bwd_chunks, w, b, x, qkv, attn,
                                    lse, d_o, atab, d_attn, delta, d_qkv, xtab, dx, dw, db,
                                    workspace=ws, compute_stream=cs, comm_stream=comm)

    pairs = batch * hd * seq * (seq + 1) / 2.0
    lin = sum(2.0 * T * g.k_loc * g.n_loc for g in (gq, go))
    flops = 3.0 * lin + 2.0 * 128 * pairs * (2 + 5)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = max(e0.elapsed_time(e1), (time.perf_counter() - t0) * 1e3) / args.steps
    value = flops / (ms_step * 1e-3) / 1e12
    atp.atp_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    atp.atp_profile_enable(False)
    kernels = []
    for r in atp.atp_profile_collect(32):
        k = dict(name=r["name"], launches_per_step=r["launches"] // args.steps,
                 avg_us=round(r["total_ms"] / r["launches"] * 1e3, 2),
                 ms_per_step=round(r["total_ms"] / args.steps, 4))
        if r["flops"] > 0:
            k["tflops"] = round(r["flops"] / (r["total_ms"] * 1e-3) / 1e12, 1)
        if r["bytes"] > 0:
            k["gbs"] = round(r["bytes"] / (r["total_ms"] * 1e-3) / 1e9, 1)
        kernels.append(k)
    dom = max((k for k in kernels if "tflops" in k), key=lambda k: k["ms_per_step"])
    out_line = dict(
        metric="TFLOP/s, attention block fwd+bwd of one device (QKV, causal core, out-proj)",
        value=round(value, 2), unit="TFLOP/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=round(ms_step, 4), higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="bf16", data="synthetic",
        config=dict(workload=args.workload, part="attention_block", mode=wl["mode"],
                    mesh=[d1, d2], coord=[0, 0], h=h, heads=heads, heads_per_device=hd,
                    batch=batch, seq=seq, chunks=chunks, bwd_chunks=bwd_chunks,
                    workspace=ws is not None, gflop_per_step=round(flops / 1e9, 1)),
        roofline=dict(bound="mfma", kernel=dom["name"], achieved=dom["tflops"],
                      peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                      frac=round(dom["tflops"] / PEAK_BF16_TFLOPS, 4), traffic=None),
        kernels=kernels, cpu_baseline=None)
    print(json.dumps(out_line), flush=True)


def step_flops(st, fwd_only):
    f = sum(2.0 * st["T"] * g.k_loc * g.n_loc for g in st["G"])
    return f if fwd_only else 3.0 * f


def make_step(torch, atp, st, fwd_only, serial, comm=None):
    bwd_chunks = st.get("bwd_chunks") or st["chunks"]
    ms = None if serial else (comm if comm is not None else torch.cuda.Stream())

    def step():
        # the stream current at call time (the capture stream inside a graph)
        cs = torch.cuda.current_stream()
        ms_ = cs if serial else ms
        atp.atp_block_fwd(st["m"], st["bm"], st["T"], st["h"], st["chunks"], st["w"], st["b"],
                          st["x"], st["a"], st["fwd_tabs"], st["qkv"], st["o"], st["hh"],
                          st["pre"], st["z"], workspace=st["ws"], compute_stream=cs,
                          comm_stream=ms_, weight_layout=st["layout"])
        if fwd_only:
            return
        atp.atp_block_bwd(st["m"], st["bm"], st["T"], st["h"], bwd_chunks, st["w"], st["b"],
                          st["x"], st["a"], st["hh"], st["pre"], st["dz"], st["dqkv"], st["do"],
                          st["bwd_tabs"], st["dh_pre"], st["dx_qkv"], st["dx_fc1"],
                          st["d_attn"], st["dw"], st["db"], workspace=st["ws"], compute_stream=cs,
                          comm_stream=ms_, weight_layout=st["layout"])
    return step


def cu_masked_stream(torch, n_cus, total=256):
    """A stream whose kernels may only use `n_cus` of the chip's CUs: the
    lowest n_cus / 8 of every 32-bit word of the mask, i.e. the same number
    in each 32-CU group (hipExtStreamCreateWithCUMask), wrapped for torch.
    The stream lives until the process ends."""
    import ctypes
    per = n_cus // (total // 32)
    if n_cus % (total // 32) or not 0 < per <= 32:
        raise SystemExit(f"bench.py: --comm-cus must be a multiple of {total // 32} up to {total}")
    hip = ctypes.CDLL("libamdhip64.so")
    words = (ctypes.c_uint32 * (total // 32))(*([(1 << per) - 1] * (total // 32)))
    handle = ctypes.c_void_p()
    rc = hip.hipExtStreamCreateWithCUMask(ctypes.byref(handle), ctypes.c_uint32(total // 32),
                                          words)
    if rc != 0:
        raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
    return torch.cuda.ExternalStream(handle.value)


def capture(torch, step):
    """One step recorded as a HIP graph (hipStreamBeginCapture through torch):
    the same kernels, events and stream joins, replayed without host launches."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, or None if there is none for this kernel and workload
    or the GEMM source changed since the counters were taken."""
    import hashlib
    path = os.path.join(HERE, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = os.path.join(HERE, "paper_2301_08658_amd", "csrc", "gemm.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if rec.get("kernel") != kernel or rec.get("gemm_source_sha256") != sha:
        return None
    return rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]


def cpu_baseline(st, rows_n, fwd_only, seed):
    """The oracle, as it stands, timed on a bounded sample of the same
    workload: the block forward (and input-gradient backward) for a few
    token rows, and dW / db for one column of each linear."""
    import numpy as np
    import torch
    import oracle as O

    G, T = st["G"], st["T"]
    rng = np.random.default_rng(seed)
    rows = sorted(rng.choice(T, size=rows_n, replace=False).tolist())
    cpu = lambda t: t.detach().cpu()  # noqa: E731
    W = [O._f64(cpu(w)) for w in st["w"]]
    Wt = [np.ascontiguousarray(w.T) for w in W]
    x, a = O._f64(cpu(st["x"][rows])), O._f64(cpu(st["a"][rows]))
    bias = [O._f64(cpu(b)) for b in st["b"]]
    ftab = [[O._f64(cpu(p[rows])) for p in t] if t else None for t in st["fwd_tabs"]]
    btab = [[O._f64(cpu(p[rows])) for p in t] if t else None for t in st["bwd_tabs"]]
    dz, dq, do = (O._f64(cpu(st[k][rows])) for k in ("dz", "dqkv", "do"))
    xs_full = O._f64(cpu(st["x"]))
    dq_col = O._f64(cpu(st["dqkv"][:, :1]))
    torch.set_num_threads(max(1, os.cpu_count() or 1))
    flops = 0.0

    def red(i, own, tab, idx, epi, b=None, pre=None):
        parts = [own] if tab is None else tab[:idx] + [own] + tab[idx + 1:]
        return O.partial_reduce(parts, b, epi, pre)

    t0 = time.perf_counter()
    # forward, sampled rows
    qkv, _ = red(0, O.matmul(x, W[0]), ftab[0], G[0].red_index, O.EPI_BIAS, bias[0])
    o, _ = red(1, O.matmul(a, W[1]), ftab[1], G[1].red_index, O.EPI_BIAS, bias[1])
    hh, pre = red(2, O.matmul(x, W[2]), ftab[2], G[2].red_index, O.EPI_BIAS_GELU, bias[2])
    z, _ = red(3, O.matmul(hh, W[3]), ftab[3], G[3].red_index, O.EPI_BIAS, bias[3])
    flops += sum(2.0 * rows_n * g.k_loc * g.n_loc for g in G)
    if not fwd_only:
        # input gradients, sampled rows
        dh, _ = red(3, O.matmul(dz, Wt[3]), btab[3], G[3].bwd_index, O.EPI_GELU_BWD, None, pre)
        red(2, O.matmul(dh, Wt[2]), btab[2], G[2].bwd_index, O.EPI_NONE)
        red(1, O.matmul(do, Wt[1]), btab[1], G[1].bwd_index, O.EPI_NONE)
        red(0, O.matmul(dq, Wt[0]), btab[0], G[0].bwd_index, O.EPI_NONE)
        flops += sum(2.0 * rows_n * g.k_loc * g.n_loc for g in G)
        # one dW column (all tokens) of the qkv linear
        O.matmul(xs_full.T, dq_col)
        O.colsum(dq_col)
        flops += 2.0 * T * G[0].k_loc
    dt = time.perf_counter() - t0
    sample = (f"{rows_n} token rows of the block forward" +
              ("" if fwd_only else " and input-gradient backward, plus one dW column of qkv") +
              f" ({flops / 1e9:.1f} GFLOP)")
    model, avail = cpu_host()
    return dict(value=flops / dt / 1e12, unit="TFLOP/s", cores=O.num_threads(), kind="oracle",
                sample=sample, seconds=round(dt, 3), cpu_model=model, cpus_available=avail,
                per_config=cpu_per_config(seed))


def cpu_host():
    """The host CPU's model string and the logical CPUs this process may use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def cpu_per_config(seed, rows=256, cols=512):
    """The oracle on one bounded sample of every workload: each of the four
    linears of the device's share, `rows` token rows by the first `cols`
    output columns over the linear's whole contraction, reduced with its
    group's (seeded) peer partials and the linear's epilogue.  Inputs are
    drawn on the CPU (synth_inputs), so no GPU value is involved."""
    import oracle as O
    import paper_2301_08658_amd as atp
    import synth_inputs as S

    res = []
    for name, wl in S.WORKLOADS.items():
        if name.startswith("tiny"):
            continue
        d1, d2 = wl["mesh"]
        bm = atp.ATP_BLOCK_COL if wl["mode"] == "col" else atp.ATP_BLOCK_ROW
        G = atp.block_geometry(atp.mesh(d1, d2, 0, 0), bm, wl["h"])
        flops, dt = 0.0, 0.0
        for i, g in enumerate(G):
            nc = min(cols, g.n_loc)
            x = S.randn_bf16((rows, g.k_loc), 1.0, seed, 50 + i)
            w = S.randn_bf16((g.k_loc, nc), wl["sigma_w"], seed, 60 + i)
            peers = [S.randn_f32((rows, nc), 1.0, seed, 70 + 10 * i + j)
                     for j in range(g.red_size - 1)]
            b = S.randn_bf16((nc,), 0.02, seed, 90 + i)
            t0 = time.perf_counter()
            own = O.matmul(x, w)
            O.partial_reduce([own] + peers, b, O.EPI_BIAS_GELU if i == 2 else O.EPI_BIAS)
            dt += time.perf_counter() - t0
            flops += 2.0 * rows * g.k_loc * nc
        res.append(dict(workload=name, value=round(flops / dt / 1e12, 5), unit="TFLOP/s",
                        seconds=round(dt, 3),
                        sample=f"{rows} token rows x first {cols} output columns of each linear"))
    return res


def reduce_alone(torch, atp, st, reps):
    """The largest reduction of the step (one chunk), timed with nothing else
    running: its group's partial buffers, the bias epilogue, bf16 output."""
    cand = [(len(t), i) for i, t in enumerate(st["fwd_tabs"]) if t]
    if not cand:
        return None
    _, L = max(cand, key=lambda c: (c[0], st["G"][c[1]].n_loc))
    g, T, c = st["G"][L], st["T"], st["chunks"]
    rows = T // c
    tab = [p[:rows] for p in st["fwd_tabs"][L]]
    out = torch.empty((rows, g.n_loc), dtype=torch.bfloat16, device="cuda:0")
    b16 = tab[0].dtype == torch.bfloat16
    red = atp.atp_chunked_partial_reduce_bf16 if b16 else atp.atp_chunked_partial_reduce
    run = lambda: red(len(tab), rows, g.n_loc, 1, tab, st["b"][L], atp.ATP_EPI_BIAS, out)  # noqa
    for _ in range(3):
        run()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = len(tab) * rows * g.n_loc * (2 if b16 else 4) + rows * g.n_loc * 2 + g.n_loc * 2
    gbs = nbytes / (ms * 1e-3) / 1e9
    return dict(linear=LIN[L], red_size=len(tab), rows=rows, n_loc=g.n_loc,
                avg_us=round(ms * 1e3, 2), achieved=round(gbs, 1), peak=PEAK_HBM_GBS,
                frac=round(gbs / PEAK_HBM_GBS, 4))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this library runs one device's share on one GPU; --gpus {args.gpus} "
              "is not supported (the multi-GPU exchange is not part of it).", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2301_08658_amd as atp
    import synth_inputs as S

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(3)
    wl = dict(S.WORKLOADS[args.workload])
    if args.mesh:
        wl["mesh"] = tuple(int(v) for v in args.mesh.lower().split("x"))
    chunks = args.chunks or wl["chunks"]
    fwd_only = args.fwd_only or not wl.get("bwd", False)
    atp.load_library()
    # a CU-masked stream needs a hardware queue of its own: made first
    comm = cu_masked_stream(torch, args.comm_cus) if args.comm_cus else None
    if args.attention:
        attention_bench(torch, atp, S, args, wl)
        return
    if args.attention_block:
        attention_block_bench(torch, atp, S, args, wl, chunks)
        return
    if args.linear:
        linear_bench(torch, atp, S, args, wl, chunks)
        return
    log(f"[bench] {atp.atp_version()} workload={args.workload} chunks={chunks} "
        f"pass={'fwd' if fwd_only else 'fwd+bwd'}")
    st = setup(torch, atp, S, wl, chunks, args.seed, args.weight_layout, args.partials,
               args.pad)
    st["bwd_chunks"] = args.bwd_chunks
    st["ws"] = None
    if not args.no_workspace:
        nb = atp.atp_block_workspace_bytes(st["m"], st["bm"], st["T"], st["h"], chunks,
                                           st["layout"])
        st["ws"] = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda:0")
    torch.cuda.synchronize()
    step = make_step(torch, atp, st, fwd_only, args.serial, comm)
    flops = step_flops(st, fwd_only)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")
    run = step
    # the direct path (no workspace) is not captured: the library refuses it
    if args.graph and not args.no_workspace:
        graph = capture(torch, step)
        run = graph.replay
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        log("[bench] step captured as a HIP graph")

    # timed region: inputs resident, K steps between two device-wide syncs;
    # an event after each step (on the stream the block joins into) gives the
    # per-step distribution
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        run()
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = max(evs[0].elapsed_time(evs[-1]), wall * 1e3) / args.steps
    value = flops / (ms_step * 1e-3) / 1e12
    per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    q = lambda f: per[min(len(per) - 1, int(round(f * (len(per) - 1))))]  # noqa: E731
    step_ms = dict(median=round(q(0.5), 4), p10=round(q(0.1), 4), p90=round(q(0.9), 4),
                   min=round(per[0], 4), max=round(per[-1], 4))
    log(f"[bench] {args.steps} steps, {ms_step:.3f} ms/step, {value:.1f} TFLOP/s "
        f"(per step median {step_ms['median']:.3f} p10 {step_ms['p10']:.3f} p90 {step_ms['p90']:.3f} ms)")

    # same K steps again, launched eagerly with every library launch bracketed
    # by HIP events on its own stream: per-kernel durations for the roofline
    atp.atp_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    atp.atp_profile_enable(False)
    stats = atp.atp_profile_collect(64)
    kernels = []
    for s in stats:
        avg = s["total_ms"] / max(1, s["launches"])
        ent = dict(name=s["name"], launches=s["launches"] // args.steps,
                   avg_us=round(avg * 1e3, 2), ms_per_step=round(s["total_ms"] / args.steps, 4))
        if s["flops"] and s["name"].startswith("gemm"):
            ent["tflops"] = round(s["flops"] / (s["total_ms"] * 1e-3) / 1e12, 1)
        if s["name"] in ("partial_reduce", "colsum", "transpose"):
            ent["gbs"] = round(s["bytes"] / (s["total_ms"] * 1e-3) / 1e9, 1)
        kernels.append(ent)
    gemms = [s for s in stats if s["name"].startswith("gemm")]
    dom = max(gemms, key=lambda s: s["total_ms"])
    achieved = dom["flops"] / (dom["total_ms"] * 1e-3) / 1e12
    traffic = measured_traffic(dom["name"], args.workload)
    roofline = dict(bound="mfma", kernel=dom["name"], achieved=round(achieved, 1),
                    peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=round(achieved / PEAK_BF16_TFLOPS, 4), traffic=traffic,
                    algorithmic_bytes_per_launch=dom["bytes"] / dom["launches"],
                    flops_per_launch=dom["flops"] / dom["launches"],
                    avg_launch_us=round(dom["total_ms"] / dom["launches"] * 1e3, 2))
    overlap = None
    if not args.serial:
        # the same launches with nothing beside them: the step with every
        # launch serialized on the compute stream, timed like the pipelined
        # step, then once more with per-launch events
        solo = make_step(torch, atp, st, fwd_only, True)
        solo()
        sev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        sev[0].record()
        for _ in range(args.steps):
            solo()
        sev[1].record()
        torch.cuda.synchronize()
        serial_ms = sev[0].elapsed_time(sev[1]) / args.steps
        atp.atp_profile_enable(True)
        for _ in range(args.steps):
            solo()
        torch.cuda.synchronize()
        atp.atp_profile_enable(False)
        solo_stats = atp.atp_profile_collect(64)
        red_solo = sum(s["total_ms"] for s in solo_stats if s["name"] == "partial_reduce")
        red_solo /= args.steps
        if red_solo > 0:
            # Sec. 4.1's overlap: the share of the reductions' own time that
            # the pipelined step hides behind the GEMMs
            overlap = dict(serial_ms=round(serial_ms, 4), pipelined_ms=round(ms_step, 4),
                           reduce_ms=round(red_solo, 4),
                           hidden=round((serial_ms - ms_step) / red_solo, 4),
                           note="(serial - pipelined) / reduction kernel time of the serialized "
                                "step; serial: every launch on the compute stream")
            log(f"[bench] overlap: {overlap}")
        alone = [s for s in solo_stats if s["name"] == dom["name"]]
        if alone:
            a = alone[0]
            tf = a["flops"] / (a["total_ms"] * 1e-3) / 1e12
            roofline["alone"] = dict(achieved=round(tf, 1), frac=round(tf / PEAK_BF16_TFLOPS, 4),
                                     avg_launch_us=round(a["total_ms"] / a["launches"] * 1e3, 2))
            roofline["note"] = ("achieved: launches of the pipelined step, which share the chip "
                                "with the other compute lane and the reductions; alone: the same "
                                "launches of a serialized pass of the step")
    red = [s for s in stats if s["name"] == "partial_reduce"]
    reduce_info = None
    if red:
        r = red[0]
        gbs = r["bytes"] / (r["total_ms"] * 1e-3) / 1e9
        reduce_info = dict(achieved=round(gbs, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                           frac=round(gbs / PEAK_HBM_GBS, 4),
                           bytes_per_step=r["bytes"] / args.steps,
                           note="durations measured while overlapping the GEMMs")
    for k in kernels:
        log(f"[bench]   {k}")
    alone = reduce_alone(torch, atp, st, args.steps)
    if alone and reduce_info is not None:
        reduce_info["alone"] = alone
        log(f"[bench] partial reduce alone: {alone}")

    if args.profile_detail:
        atp.atp_profile_enable(2)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        atp.atp_profile_enable(False)
        for s in sorted(atp.atp_profile_collect(128), key=lambda s: -s["total_ms"]):
            us = s["total_ms"] / s["launches"] * 1e3
            tf = s["flops"] / (s["total_ms"] * 1e-3) / 1e12 if s["flops"] else 0.0
            gb = s["bytes"] / (s["total_ms"] * 1e-3) / 1e9
            log(f"[detail] {s['name']:<44} n={s['launches'] // args.steps:<3} "
                f"avg={us:9.1f}us  {tf:7.1f} TFLOP/s  {gb:7.1f} GB/s")

    if args.copy_calib_mb:
        n = args.copy_calib_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.copy_calib_mb} MiB done")

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        cpu = cpu_baseline(st, args.cpu_rows, fwd_only, args.seed)
        log(f"[bench] cpu baseline: {cpu}")

    d1, d2 = wl["mesh"]
    out = dict(
        metric=METRIC, value=round(value, 2), unit="TFLOP/s", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(ms_step, 4), higher_is_better=True,
        scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload=args.workload, mode=wl["mode"], mesh=[d1, d2], coord=[0, 0],
                    tokens=wl["tokens"], h=wl["h"], chunks=chunks,
                    bwd_chunks=None if fwd_only else st["bwd_chunks"],
                    **{"pass": "fwd" if fwd_only else "fwd+bwd"},
                    serial=bool(args.serial), workspace=not args.no_workspace,
                    weight_layout=args.weight_layout, partials=args.partials,
                    comm_cus=args.comm_cus or None,
                    hip_graph=bool(args.graph and not args.no_workspace),
                    gflop_per_step=round(flops / 1e9, 1)),
        step_ms=step_ms, mfma_util=round(value / PEAK_BF16_TFLOPS, 4),
        roofline=roofline, reduce=reduce_info, overlap=overlap, kernels=kernels,
        cpu_baseline=cpu)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
