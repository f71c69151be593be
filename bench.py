"""Benchmark of block-causal streaming attention on one MI355X.

Headline workload (the largest single-GPU configuration): one streaming
step of 4 concurrent streams, GQA 64 query / 8 KV heads x 128, each
appending a 512-token block (committed in the same launch, WS_FUSE_APPEND)
and attending to its own paged cache of 131072 tokens (64-token pages in
seeded random order).  A "step" is one ws_block_causal_attn_fwd call:
plan/validate, append, K/V tile fetch, QK^T, online softmax, PV, split
merge (none here: the work items fill the chip) and epilogue.

Timing: W warm-up steps, then K timed steps bracketed by
torch.cuda.synchronize() (the wall clock gives `value`) and by two HIP events
recorded on the stream the kernels run on (torch's current stream), which
give the average kernel time per step used for the roofline.  Nothing else
runs inside the timed region.  Afterwards a separate loop puts each step
between two events for the per-block latency.  Inputs of small workloads
rotate over enough device-resident copies (> 512 MB in total) that no copy
is still in the 256 MB last-level cache when it is used again.

Also reported: the single 256-token step over a 4096-token cache (its HBM
roofline), the prefill workloads, KV-length sweeps, the streaming replay of
the prefill workloads block by block, the practical MFMA and HBM-read
ceilings measured in the same job, and the fp64 oracle timed on the host
cores on a stated row sample of every workload.

Prints one JSON line (see the metric/roofline/cpu_baseline fields).
Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-extra]
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2606_25041_amd as ws  # noqa: E402
from paper_2606_25041_amd import inputs  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2516.6   # 256 CU x 4096 flop/clk x 2.4 GHz, dense
ROTATE_BYTES = 600 << 20    # rotation set larger than the 256 MB MALL
METRIC = "block-causal attn TFLOP/s + per-block step latency (ms) vs KV cache length"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for p in ws._build.KERNEL_SOURCES:
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# algorithmic work of a workload

def visible_pairs(wl):
    """Visible (query, key) pairs per (stream, query head).  With token-causal
    segments (text_starts), token i of a block with segment start ts sees
    max(ts, i + 1) keys (step: after the stream's cache).  Steps over padded
    blocks (new_lens) count the real tokens only."""
    ts_all = getattr(wl, "text_starts", None)
    if wl.kind == "step":
        out = []
        for b, c in enumerate(wl.cache_lens):
            nls = getattr(wl, "new_lens", None)
            lq = int(wl.Lq) if nls is None else int(nls[b])
            ts = lq if ts_all is None else min(int(ts_all[b]), lq)
            # sum over t < lq of max(ts, t + 1)
            own = ts * ts + (lq * (lq + 1) - ts * (ts + 1)) // 2
            out.append(lq * int(c) + own)
        return out
    out = []
    for b, off in enumerate(wl.offsets):
        off = off.astype(np.int64)
        s, e = off[:-1], off[1:]
        if ts_all is None:
            out.append(int(np.sum((e - s) * e)))
        else:
            t = np.asarray(ts_all[b], dtype=np.int64)
            # rows [s, t) see t keys; rows i in [t, e) see i + 1
            out.append(int(np.sum((t - s) * t + (e * (e + 1) - t * (t + 1)) // 2)))
    return out


def algorithmic_flops(wl):
    return 4.0 * wl.D * wl.Hq * float(sum(visible_pairs(wl)))


def algorithmic_bytes(wl):
    """Q, K, V and O moved once (K/V once per KV head), plus the appended
    block's writes when it is committed."""
    e = 2  # bf16
    out_e = 4 if wl.out_f32 else 2
    if wl.kind == "step":
        # real tokens only when the blocks are padded
        nls = getattr(wl, "new_lens", None)
        n_new = [int(wl.Lq)] * wl.B if nls is None else [int(n) for n in nls]
        q = sum(n_new) * wl.Hq * wl.D * e
        o = sum(n_new) * wl.Hq * wl.D * out_e
        kv = 2 * sum(int(c) + n for c, n in zip(wl.cache_lens, n_new)) * wl.Hkv * wl.D * e
        app = 2 * sum(n_new) * wl.Hkv * wl.D * e if wl.fuse_append else 0
        return q + kv + o + app
    q = wl.B * wl.Lq * wl.Hq * wl.D * e
    o = wl.B * wl.Lq * wl.Hq * wl.D * out_e
    kv = 2 * wl.B * wl.Lq * wl.Hkv * wl.D * e
    return q + kv + o


# ---------------------------------------------------------------------------
# device setup

class DeviceCase:
    """Device-resident inputs of one workload (one rotation copy)."""

    def __init__(self, wl, dev):
        self.wl = wl
        self.q = wl.q.to(dev)
        self.out = torch.empty((wl.B, wl.Lq, wl.Hq, wl.D),
                               dtype=torch.float32 if wl.out_f32 else torch.bfloat16, device=dev)
        self.lse = torch.empty((wl.B, wl.Hq, wl.Lq), dtype=torch.float32, device=dev)
        if wl.kind == "step":
            self.k_new = wl.k_new.contiguous().to(dev)
            self.v_new = wl.v_new.contiguous().to(dev)
            self.cache = ws.PagedCache.allocate(wl.num_pages, wl.Hkv, wl.D,
                                                torch.from_numpy(wl.page_table), device=dev,
                                                fill_bits=0x7FC1)
            lens = torch.from_numpy(wl.cache_lens.astype(np.int32))
            self.lens = (lens, lens.to(dev))
            self.text = None
            if wl.text_starts is not None:
                th = torch.from_numpy(np.ascontiguousarray(wl.text_starts, dtype=np.int32))
                self.text = (th, th.to(dev))
            self.new_lens = None
            if wl.new_lens is not None:
                nh = torch.from_numpy(np.ascontiguousarray(wl.new_lens, dtype=np.int32))
                self.new_lens = (nh, nh.to(dev))
            kc = wl.k_cache.contiguous().to(dev)
            vc = wl.v_cache.contiguous().to(dev)
            n = int(wl.cache_lens.min())
            assert all(int(c) == n for c in wl.cache_lens)
            zero = torch.zeros(wl.B, dtype=torch.int32)
            ws.kv_append(self.cache, (zero, zero.to(dev)), kc[:, :n], vc[:, :n])
            del kc, vc
            if wl.new_lens is None:
                need = ws.workspace_bytes(ws.WS_OP_STEP, wl.B, wl.Hq, wl.Hkv, wl.Lq,
                                          int(wl.cache_lens.max()) + wl.Lq)
            else:
                need = ws.step_workspace_bytes_varlen(wl.B, wl.Hq, wl.Hkv, wl.Lq, wl.cache_lens, wl.new_lens)
            self.workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
        else:
            off = torch.from_numpy(wl.offsets.astype(np.int32))
            self.offsets = (off, off.to(dev))
            self.text = None
            if wl.text_starts is not None:
                th = torch.from_numpy(np.ascontiguousarray(wl.text_starts, dtype=np.int32))
                self.text = (th, th.to(dev))
            if wl.paged:
                self.cache = ws.PagedCache.allocate(wl.num_pages, wl.Hkv, wl.D,
                                                    torch.from_numpy(wl.page_table), device=dev,
                                                    fill_bits=0x7FC1)
                zero = torch.zeros(wl.B, dtype=torch.int32)
                ws.kv_append(self.cache, (zero, zero.to(dev)), wl.k.contiguous().to(dev),
                             wl.v.contiguous().to(dev))
                self.k = self.v = None
            else:
                self.cache = None
                self.k = wl.k.to(dev)
                self.v = wl.v.to(dev)

    def run(self):
        wl = self.wl
        if wl.kind == "step":
            ws.block_causal_attn_fwd(self.q, self.k_new, self.v_new, self.cache, self.lens,
                                     scale=wl.scale, fuse_append=wl.fuse_append, out=self.out,
                                     lse=self.lse, want_lse=True, workspace=self.workspace,
                                     text_starts=self.text, new_lens=self.new_lens)
        else:
            ws.block_causal_prefill(self.q, self.k, self.v, self.offsets, scale=wl.scale,
                                    cache=self.cache, num_kv_heads=wl.Hkv, out=self.out,
                                    lse=self.lse, want_lse=True, text_starts=self.text)


def time_workload(wl, steps, warmup, dev, rotate=True, latency_steps=None, stats=None, graph_stats=None):
    """Returns (ms per step from the synchronised wall clock over the K timed
    steps, ms per step from HIP events recorded on the launch stream at the
    two ends of the same timed region, median per-step latency in ms, one
    case).  The timed region has no per-step instrumentation; the per-step
    latency comes from a separate loop afterwards, each step between two
    events.  graph_stats (a dict): also the per-step latency with each step
    (fused append, attention and merge) launched from a captured HIP graph,
    median / p10 / p90 in ms."""
    nbytes = algorithmic_bytes(wl)
    copies = max(1, math.ceil(ROTATE_BYTES / nbytes)) if rotate else 1
    copies = min(copies, 16)
    log(f"[bench] {wl.name}: building {copies} device copies")
    cases = [DeviceCase(wl, dev) for _ in range(copies)]
    torch.cuda.synchronize()
    for i in range(warmup):
        cases[i % copies].run()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for i in range(steps):
        cases[i % copies].run()
    e1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    ev_ms = e0.elapsed_time(e1) / steps
    n_lat = latency_steps if latency_steps is not None else steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_lat)]
    for i in range(n_lat):
        ev[i][0].record()
        cases[i % copies].run()
        ev[i][1].record()
    torch.cuda.synchronize()
    lats = [a.elapsed_time(b) for a, b in ev]
    lat = float(np.median(lats)) if n_lat else ev_ms
    if stats is not None:   # p10 / p90 of the per-step latency
        stats["p10"] = float(np.percentile(lats, 10)) if n_lat else ev_ms
        stats["p90"] = float(np.percentile(lats, 90)) if n_lat else ev_ms
    log(f"[bench] {wl.name}: wall {wall_ms:.4f} ms/step, events over the timed region {ev_ms:.4f} "
        f"ms/step, per-step latency median {lat:.4f} ms")
    if graph_stats is not None and n_lat:
        graph_latency(cases, n_lat, graph_stats)
        log(f"[bench] {wl.name}: per-step latency from HIP graph launches, median {graph_stats['median']:.4f} ms")
    return wall_ms, ev_ms, lat, cases[0]


def graph_latency(cases, n, stats):
    """Each case's step captured once into a HIP graph (after a warm-up on a
    side stream); then n graph launches, each between two events."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for c in cases:
            c.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = []
    for c in cases:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            c.run()
        graphs.append(g)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for i in range(n):
        ev[i][0].record()
        graphs[i % len(graphs)].replay()
        ev[i][1].record()
    torch.cuda.synchronize()
    lats = [a.elapsed_time(b) for a, b in ev]
    stats["median"] = float(np.median(lats))
    stats["p10"] = float(np.percentile(lats, 10))
    stats["p90"] = float(np.percentile(lats, 90))
    del graphs


# ---------------------------------------------------------------------------
# KV-length sweeps: the step at growing cache lengths and small query blocks

class SweepPoint:
    """A streaming step of B streams (Hq query / Hkv KV heads x 128) with a
    block of Lq new tokens against Lc cached tokens per stream, committed in
    the same launch.  Inputs are N(0,1) bf16 drawn on the device from a
    seeded generator (only their shape matters for timing); the pool pages
    are a seeded random permutation, as in the headline workload."""

    kind = "step"
    D = 128
    out_f32 = False
    fuse_append = True

    def __init__(self, sweep, B, Hq, Hkv, Lq, Lc, token_causal=False):
        self.sweep, self.B, self.Hq, self.Hkv, self.Lq, self.Lc = sweep, B, Hq, Hkv, Lq, Lc
        self.cache_lens = np.full(B, Lc, dtype=np.int64)
        # token-causal block (segment start 0): the thinker's decode step
        self.text_starts = np.zeros(B, np.int32) if token_causal else None
        self.name = f"{sweep}_b{B}_h{Hq}x{Hkv}_q{Lq}_c{Lc}" + ("_tokcausal" if token_causal else "")


SWEEPS = ([SweepPoint("S1", 1, 24, 24, 256, c) for c in (0, 1024, 4096, 16384, 65536, 131072)]
          + [SweepPoint("S2", 4, 64, 8, 512, c) for c in (4096, 16384, 32768, 65536, 131072)]
          + [SweepPoint("S3", 4, 64, 8, lq, 131072) for lq in (16, 64)]
          + [SweepPoint("S3", 1, 24, 24, lq, 131072) for lq in (16, 64)]
          + [SweepPoint("S5", 4, 64, 8, lq, c, token_causal=True) for lq in (1, 4, 8) for c in (32768, 131072)])


class SweepCase:
    def __init__(self, pt, dev, seed):
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        B, Lq, Hq, Hkv, D = pt.B, pt.Lq, pt.Hq, pt.Hkv, pt.D
        self.pt = pt
        self.q = torch.randn((B, Lq, Hq, D), generator=g, device=dev).to(torch.bfloat16)
        self.k_new = torch.randn((B, Lq, Hkv, D), generator=g, device=dev).to(torch.bfloat16)
        self.v_new = torch.randn((B, Lq, Hkv, D), generator=g, device=dev).to(torch.bfloat16)
        per = (pt.Lc + Lq + ws.PAGE_SIZE - 1) // ws.PAGE_SIZE
        gh = torch.Generator()
        gh.manual_seed(seed)
        table = torch.randperm(B * per, generator=gh).to(torch.int32).reshape(B, per)
        shape = (B * per, Hkv, ws.PAGE_SIZE, D)
        kp = torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)
        vp = torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)
        self.cache = ws.PagedCache(kp, vp, table)
        lens = torch.full((B,), pt.Lc, dtype=torch.int32)
        self.lens = (lens, lens.to(dev))
        self.out = torch.empty((B, Lq, Hq, D), dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((B, Hq, Lq), dtype=torch.float32, device=dev)
        need = ws.workspace_bytes(ws.WS_OP_STEP, B, Hq, Hkv, Lq, pt.Lc + Lq)
        self.workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
        self.text = None
        if pt.text_starts is not None:
            th = torch.from_numpy(pt.text_starts)
            self.text = (th, th.to(dev))

    def run(self):
        ws.block_causal_attn_fwd(self.q, self.k_new, self.v_new, self.cache, self.lens,
                                 fuse_append=True, out=self.out, lse=self.lse, want_lse=True,
                                 workspace=self.workspace, text_starts=self.text)


def run_sweeps(dev, steps, points=None):
    """Median HIP-event time per point, over device copies rotated so that
    more than the 256 MB last-level cache is touched between reuses."""
    todo = SWEEPS if points is None else points
    points = []
    for i, pt in enumerate(todo):
        nbytes = algorithmic_bytes(pt)
        copies = min(64, max(1, math.ceil(ROTATE_BYTES / nbytes)))
        cases = [SweepCase(pt, dev, 7000 + 100 * i + c) for c in range(copies)]
        torch.cuda.synchronize()
        n = max(5, min(steps, int(2e5 / max(1.0, nbytes / 1e6))))   # ~ a fixed byte budget per point
        for c in range(min(3, n)):
            cases[c % copies].run()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for k in range(n):
            ev[k][0].record()
            cases[k % copies].run()
            ev[k][1].record()
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
        flops = algorithmic_flops(pt)
        tf = flops / (ms * 1e-3) / 1e12
        gbs = nbytes / (ms * 1e-3) / 1e9
        ai = flops / nbytes
        attain = min(BF16_PEAK_TFLOPS, ai * HBM_PEAK_GBS / 1e3)
        points.append({"sweep": pt.sweep, "workload": pt.name, "batch": pt.B, "q_heads": pt.Hq,
                       "kv_heads": pt.Hkv, "block_tokens": pt.Lq, "cache_tokens": pt.Lc,
                       "ms": round(ms, 5), "TFLOP/s": round(tf, 1), "GB/s": round(gbs, 1),
                       "flop_per_byte": round(ai, 1),
                       "bound": "hbm" if ai * HBM_PEAK_GBS / 1e3 < BF16_PEAK_TFLOPS else "mfma",
                       "frac_of_bound": round(tf / attain, 4),
                       "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)})
        log(f"[bench] sweep {pt.name}: {ms * 1e3:.1f} us, {tf:.0f} TFLOP/s, {gbs:.0f} GB/s")
        del cases
        torch.cuda.empty_cache()
    return points


def solver_loop_timing(dev, steps=8, reps=40):
    """The performer's loop for one streaming unit at the headline shape
    (MHA 24 x 128, 256-token block, 4096 cached tokens, paged): ``steps`` - 1
    solver steps of a changing noisy block against the fixed cache, then a
    step that commits the clean block.  Timed eagerly and as one captured
    HIP graph replay (events on the launch stream; median over ``reps``).
    The same cache is read by every step of a unit, so after the first step
    it is served from the 256 MB last-level cache, as in the real loop."""
    wl = inputs.config(2)
    case = DeviceCase(wl, dev)
    g = torch.Generator(device=dev)
    g.manual_seed(9100)
    shp_q, shp_kv = tuple(case.q.shape), tuple(case.k_new.shape)
    qs = [torch.randn(shp_q, generator=g, device=dev).to(torch.bfloat16) for _ in range(steps)]
    ks = [torch.randn(shp_kv, generator=g, device=dev).to(torch.bfloat16) for _ in range(steps)]
    vs = [torch.randn(shp_kv, generator=g, device=dev).to(torch.bfloat16) for _ in range(steps)]
    outs = [torch.empty_like(case.out) for _ in range(steps)]

    def loop():
        for s in range(steps):
            ws.block_causal_attn_fwd(qs[s], ks[s], vs[s], case.cache, case.lens, scale=wl.scale,
                                     fuse_append=(s == steps - 1), out=outs[s], workspace=case.workspace)

    def timed(fn):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    for _ in range(3):
        loop()
    torch.cuda.synchronize()
    eager = timed(loop)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        loop()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        loop()
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    replay = timed(graph.replay)
    flops = algorithmic_flops(wl) * steps
    log(f"[bench] solver loop x{steps}: eager {eager * 1e3:.1f} us, graph replay {replay * 1e3:.1f} us per unit")
    out = {"workload": f"solver_loop_b1_mha24_d128_q256_c4096_x{steps}", "steps_per_unit": steps,
           "eager_ms_per_unit": round(eager, 5), "graph_ms_per_unit": round(replay, 5),
           "eager_TFLOP/s": round(flops / (eager * 1e-3) / 1e12, 1),
           "graph_TFLOP/s": round(flops / (replay * 1e-3) / 1e12, 1)}
    del case, qs, ks, vs, outs, graph
    torch.cuda.empty_cache()
    return out


def backward_timing(dev, steps=5):
    """Gradients of the whole-sequence workload (2 x 16384 tokens, GQA 32/8,
    64 blocks of 256): dQ, dK and dV from dO, the forward's output and lse.
    Algorithmic work 10 d flops per visible pair (recomputed S^T, dP, dV, dK,
    dQ: 2.5 x the forward's), although the kernels recompute S and dP once
    more (14 d)."""
    wl = inputs.config(3)
    q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
    off = torch.from_numpy(wl.offsets.astype(np.int32))
    offs = (off, off.to(dev))
    o, lse = ws.block_causal_prefill(q, k, v, offs, want_lse=True)
    g = torch.Generator(device=dev)
    g.manual_seed(9200)
    dout = torch.randn(tuple(q.shape), generator=g, device=dev).to(torch.bfloat16)
    dq = torch.empty(tuple(q.shape), dtype=torch.float32, device=dev)
    dk = torch.empty(tuple(k.shape), dtype=torch.float32, device=dev)
    dv = torch.empty_like(dk)
    work = torch.empty(ws.workspace_bytes(ws.WS_OP_PREFILL_BWD, wl.B, wl.Hq, wl.Hkv, wl.Lq, wl.Lq),
                       dtype=torch.uint8, device=dev)

    def run():
        ws.block_causal_prefill_bwd(q, k, v, o, dout, lse, offs, dq=dq, dk=dk, dv=dv, workspace=work)

    for _ in range(2):
        run()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    flops = 2.5 * algorithmic_flops(wl)
    tf = flops / (ms * 1e-3) / 1e12
    log(f"[bench] prefill backward: {ms:.3f} ms, {tf:.0f} TFLOP/s")
    out = {"workload": "prefill_bwd_b2_gqa32x8_d128_64x256", "ms": round(ms, 4), "TFLOP/s": round(tf, 1),
           "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4), "flops": flops}
    del q, k, v, o, lse, dout, dq, dk, dv, work
    torch.cuda.empty_cache()
    return out


def row_key_counts(wl, rows):
    """Keys each sampled (b, h, i) row sees (block-causal, no segments): a
    prefill row sees every token up to the end of its block, a step row its
    stream's cache and the whole new block."""
    rows = np.asarray(rows)
    if wl.kind == "step":
        return np.array([int(wl.cache_lens[b]) + wl.Lq for b in rows[:, 0]], dtype=np.int64)
    out = np.empty(len(rows), dtype=np.int64)
    for n, (b, _, i) in enumerate(rows):
        off = wl.offsets[b]
        out[n] = off[np.searchsorted(off, i, side="right")]
    return out


# pairs of (query, key) per oracle sample: ~5 s of fp64 work on 16 host cores
ORACLE_PAIRS = 2.0e8


def oracle_sample(wl, seed=11):
    """The fp64 oracle (as it stands) on a bounded sample of a workload's
    query rows: the whole workload when it has at most ORACLE_PAIRS visible
    pairs, else distinct (stream, head, token) rows drawn uniformly from the
    seed until the sample holds about that many.  Returns the timing record
    (TFLOP/s of the sampled rows' algorithmic work)."""
    import oracle  # test infrastructure: only this baseline leg uses it
    threads = oracle.default_threads()
    total_pairs = float(sum(visible_pairs(wl))) * wl.Hq
    rows = None
    if total_pairs > ORACLE_PAIRS:
        per_row = total_pairs / (wl.B * wl.Hq * wl.Lq)
        n = int(ORACLE_PAIRS / per_row)
        rows = inputs.sample_rows(np.random.default_rng(seed), wl.B, wl.Hq, wl.Lq, n)
        pairs = float(row_key_counts(wl, rows).sum())
        sample = (f"{len(rows)} of {wl.B * wl.Hq * wl.Lq} query rows (stream, head, token) drawn "
                  f"uniformly with seed {seed}, {pairs:.3g} visible pairs, fp64, {threads} threads")
    else:
        pairs = total_pairs
        sample = f"the whole workload ({wl.B * wl.Hq * wl.Lq} query rows, {pairs:.3g} visible pairs), fp64, " \
                 f"{threads} threads"
    q = inputs.bf16_bits(wl.q)
    t0 = time.perf_counter()
    if wl.kind == "step":
        oracle.step(q, inputs.bf16_bits(wl.k_cache), inputs.bf16_bits(wl.v_cache), wl.cache_lens,
                    inputs.bf16_bits(wl.k_new), inputs.bf16_bits(wl.v_new), wl.scale, rows=rows, nthreads=threads)
    else:
        oracle.prefill(q, inputs.bf16_bits(wl.k), inputs.bf16_bits(wl.v), wl.offsets, wl.scale, rows=rows,
                       nthreads=threads)
    dt = time.perf_counter() - t0
    log(f"[bench] oracle {wl.name}: {dt:.2f} s for {pairs:.3g} pairs")
    return {"workload": wl.name, "value": 4.0 * wl.D * pairs / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 3), "sample": sample, "cpu_model": cpu_model()}


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def replay_timing(idx, dev, reps=5):
    """Streaming replay (the prefill workloads run block by block): for block
    j of every stream, one step whose cache is blocks < j (already committed)
    and whose new block is block j, committed in the same launch.  The
    cache sits in a paged pool (the workload's page table, or a seeded
    random one for contiguous workloads).  Per-block latency = median over
    ``reps`` replays of the events around each step; the whole pool is
    reused by every step, as in the streaming loop (it fits the last-level
    cache for these workloads)."""
    wl = inputs.config(idx)
    B, Hq, Hkv, D = wl.B, wl.Hq, wl.Hkv, wl.D
    offs = wl.offsets
    assert all(np.array_equal(offs[0], o) for o in offs), "streams share block offsets"
    off = offs[0].astype(np.int64)
    table, npages = wl.page_table, wl.num_pages
    if table is None:
        table, npages = inputs.page_table(inputs.rng(wl.seed, inputs.S_PAGES), B, max(1, -(-wl.Lq // 64)))
    cache = ws.PagedCache.allocate(npages, Hkv, D, torch.from_numpy(table), device=dev, fill_bits=0x7FC1)
    q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
    odt = torch.float32 if wl.out_f32 else torch.bfloat16
    steps, need = [], 16
    for j in range(len(off) - 1):
        s0, e0 = int(off[j]), int(off[j + 1])
        if e0 == s0:
            continue
        lq = e0 - s0
        lens = torch.full((B,), s0, dtype=torch.int32)
        need = max(need, ws.workspace_bytes(ws.WS_OP_STEP, B, Hq, Hkv, lq, s0 + lq))
        steps.append(dict(q=q[:, s0:e0], k=k[:, s0:e0], v=v[:, s0:e0], lens=(lens, lens.to(dev)),
                          out=torch.empty((B, lq, Hq, D), dtype=odt, device=dev), c=s0, n=lq))
    work = torch.empty(need, dtype=torch.uint8, device=dev)   # one workspace, reused by every step
    for st in steps:
        st["work"] = work

    def run(st):
        ws.block_causal_attn_fwd(st["q"], st["k"], st["v"], cache, st["lens"], scale=wl.scale,
                                 fuse_append=True, out=st["out"], workspace=st["work"])

    for st in steps:   # warm-up replay (also fills the cache)
        run(st)
    torch.cuda.synchronize()
    ms = np.zeros((reps, len(steps)))
    for r in range(reps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in steps]
        for (a, b), st in zip(ev, steps):
            a.record()
            run(st)
            b.record()
        torch.cuda.synchronize()
        ms[r] = [a.elapsed_time(b) for a, b in ev]
    med = np.median(ms, axis=0)
    flops = 0.0
    for st in steps:
        flops += 4.0 * D * Hq * B * st["n"] * (st["c"] + st["n"])
    total = float(med.sum())
    log(f"[bench] replay {wl.name}: {len(steps)} blocks, {total:.3f} ms per replay "
        f"({flops / (total * 1e-3) / 1e12:.0f} TFLOP/s)")
    out = {"workload": f"replay_{wl.name}", "blocks": len(steps), "ms_per_replay": round(total, 4),
           "TFLOP/s": round(flops / (total * 1e-3) / 1e12, 1),
           "cache_tokens": [st["c"] for st in steps], "block_tokens": [st["n"] for st in steps],
           "ms_per_block_median": [round(float(x), 4) for x in med],
           "ms_per_block_p10": [round(float(x), 4) for x in np.percentile(ms, 10, axis=0)],
           "ms_per_block_p90": [round(float(x), 4) for x in np.percentile(ms, 90, axis=0)]}
    del cache, q, k, v, steps, work
    torch.cuda.empty_cache()
    return out


def _ceil_lib():
    import ctypes
    lib = ctypes.CDLL(ws._build.CEIL_LIB)
    lib.wsc_mfma_loop.restype = ctypes.c_int
    lib.wsc_mfma_loop.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_void_p]
    lib.wsc_stream_read.restype = ctypes.c_int
    lib.wsc_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_void_p]
    return lib


def ceilings(dev, reps=10):
    """Practical ceilings measured in the same job (libwsceil.so): the dense
    bf16 MFMA rate of 8-wave work-groups issuing register-operand MFMAs
    (4 work-groups per CU, 16384 MFMAs per wave into 2, 3 or 4 independent
    accumulators: the best of the three), and the rate of reading a 4 GiB
    buffer once with 16-byte non-temporal loads (8 work-groups of 256
    threads per CU).  Median of ``reps`` event-timed launches each."""
    lib = _ceil_lib()
    stream = torch.cuda.current_stream().cuda_stream

    def timed(fn):
        fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]))

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ng = 4 * cus
    out = torch.empty(ng, dtype=torch.float32, device=dev)
    rates = {}
    for chains in (2, 3, 4):
        iters = 16384 // (4 * chains)   # 16384 MFMAs per wave whatever the chain count

        def mf():
            rc = lib.wsc_mfma_loop(out.data_ptr(), ng, iters, chains, stream)
            assert rc == 0, rc
        ms = timed(mf)
        rates[chains] = ng * 8 * iters * 4 * chains * 32768 / (ms * 1e-3) / 1e12
    best = max(rates, key=rates.get)
    mfma_tf = rates[best]
    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(3)
    ng2 = 8 * cus
    out2 = torch.empty(ng2, dtype=torch.int32, device=dev)

    def rd():
        rc = lib.wsc_stream_read(buf.data_ptr(), nbytes, out2.data_ptr(), ng2, stream)
        assert rc == 0, rc
    ms2 = timed(rd)
    read_gbs = nbytes / (ms2 * 1e-3) / 1e9
    log(f"[bench] ceilings: MFMA {mfma_tf:.0f} TFLOP/s, streaming read {read_gbs:.0f} GB/s")
    del buf
    torch.cuda.empty_cache()
    return {"mfma_bf16_TFLOP/s": round(mfma_tf, 1), "mfma_frac_of_peak": round(mfma_tf / BF16_PEAK_TFLOPS, 4),
            "hbm_read_GB/s": round(read_gbs, 1), "hbm_read_frac_of_peak": round(read_gbs / HBM_PEAK_GBS, 4),
            "mfma_kernel": f"{ng} work-groups x 8 waves x 16384 v_mfma_f32_32x32x16_bf16, best of "
                           f"2 / 3 / 4 accumulators per wave ({best}: "
                           + ", ".join(f"{c}: {r:.0f}" for c, r in rates.items()) + " TFLOP/s)",
            "read_kernel": f"{nbytes >> 30} GiB read once, {ng2} work-groups x 256 threads, 16-byte loads"}


def roofline_of(wl, ev_ms, flops, nbytes):
    """Roofline block of a workload from its average kernel time per step."""
    ai = flops / nbytes
    bound = "hbm" if ai < BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9) else "mfma"
    if bound == "hbm":
        gbs = nbytes / (ev_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    else:
        tf = flops / (ev_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / BF16_PEAK_TFLOPS, 4)}
    roof["traffic"] = load_traffic(wl.name)
    roof["algorithmic_bytes"] = nbytes
    roof["algorithmic_flops"] = flops
    roof["step_ms_events"] = round(ev_ms, 5)
    return roof


def load_traffic(workload_name):
    """HBM bytes per step measured with rocprofv3 counters (FETCH_SIZE and
    WRITE_SIZE, scaled by a copy-kernel calibration), if the committed summary
    was taken on the current kernel source; None otherwise."""
    p = os.path.join(ROOT, "profiles", f"traffic_attn_{workload_name}.txt")
    if not os.path.exists(p):
        return None
    for line in open(p):
        if line.startswith("machine-readable:"):
            d = json.loads(line.split(":", 1)[1])
            if d.get("kernel_source_hash") == kernel_source_hash():
                return d.get("bytes_per_launch")
    return None


def step_record(wl, wall_ms, ev_ms, lat, stats=None):
    flops, nbytes = algorithmic_flops(wl), algorithmic_bytes(wl)
    rec = {"workload": wl.name, "ms": round(ev_ms, 5), "wall_ms": round(wall_ms, 5),
           "TFLOP/s": round(flops / (ev_ms * 1e-3) / 1e12, 1),
           "mfma_frac": round(flops / (ev_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
           "GB/s": round(nbytes / (ev_ms * 1e-3) / 1e9, 1), "flops": flops, "bytes": nbytes,
           "latency_ms_per_block": round(lat, 5)}
    if stats:
        rec["latency_ms_p10_p90"] = [round(stats["p10"], 5), round(stats["p90"], 5)]
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-extra", action="store_true", help="headline workload only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-sweep", action="store_true", help="skip the KV-length sweeps")
    ap.add_argument("--config", type=int, default=5, help="headline workload index (1-5)")
    ap.add_argument("--sweep-only", default=None, metavar="NAME",
                    help="only time the named KV-length sweep point(s), comma-separated (for profiling)")
    ap.add_argument("--varlen-only", action="store_true",
                    help="only time the four-stream step over units of different lengths (for profiling)")
    ap.add_argument("--bwd-only", action="store_true",
                    help="only time the gradients of the whole-sequence workload (for profiling)")
    ap.add_argument("--replay-only", type=int, default=0, metavar="IDX",
                    help="only time the streaming replay of workload IDX (1, 3 or 4; for profiling)")
    ap.add_argument("--solver-only", action="store_true",
                    help="only time the solver loop, eager and replayed from a HIP graph (for profiling)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (to calibrate "
                         "the FETCH_SIZE / WRITE_SIZE counters against known bytes)")
    args = ap.parse_args()
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 5}), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: there is no multi-GPU path (streams, KV-head groups "
              "and cache slices would shard with no exchange but one LSE merge); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    ws.library()
    if args.bwd_only:
        print(json.dumps(backward_timing(dev, steps=args.steps)), flush=True)
        return
    if args.replay_only:
        print(json.dumps(replay_timing(args.replay_only, dev)), flush=True)
        return
    if args.solver_only:
        print(json.dumps(solver_loop_timing(dev)), flush=True)
        return
    if args.varlen_only:
        w2 = inputs.streams_varlen()
        f2, b2 = algorithmic_flops(w2), algorithmic_bytes(w2)
        _, emean, _, _ = time_workload(w2, args.steps, args.warmup, dev, latency_steps=0)
        print(json.dumps({"workload": w2.name, "new_lens": [int(x) for x in w2.new_lens], "ms": round(emean, 4),
                          "TFLOP/s": round(f2 / (emean * 1e-3) / 1e12, 1), "flops": f2, "bytes": b2}), flush=True)
        return
    if args.sweep_only:
        names = set(args.sweep_only.split(","))
        pts = [p for p in SWEEPS if p.name in names]
        if not pts:
            print(f"no sweep point named {args.sweep_only}", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(run_sweeps(dev, args.steps, points=pts)), flush=True)
        return

    def workload(idx):
        w = inputs.config(idx)
        if w.kind == "step":
            w.fuse_append = True  # every per-block step commits its block
        return w

    wl = workload(args.config)
    flops, nbytes = algorithmic_flops(wl), algorithmic_bytes(wl)
    torch.cuda.synchronize()
    lat_stats, graph_stats = {}, {}
    wall_ms, ev_mean, ev_med, _ = time_workload(wl, args.steps, args.warmup, dev, stats=lat_stats,
                                                graph_stats=graph_stats if wl.kind == "step" else None)
    tflops = flops / (wall_ms * 1e-3) / 1e12
    roof = roofline_of(wl, ev_mean, flops, nbytes)

    extra, oracle_runs = [], []
    if not args.no_extra:
        for idx in (2, 3, 4, "thinker", "varlen"):
            if idx == args.config:
                continue
            # "thinker": the interleaved workload with each unit's text
            # segment token-causal; "varlen": four streams each ingesting an
            # interleaved unit of its own length in one step
            w2 = (inputs.thinker_prefill() if idx == "thinker" else inputs.streams_varlen() if idx == "varlen"
                  else workload(idx))
            st, gst = {}, {}
            n_steps = args.steps if w2.kind == "step" and idx == 2 else max(3, args.steps // 5)
            wms, emean, emed, _ = time_workload(w2, n_steps, 2, dev, latency_steps=n_steps if idx == 2 else 0,
                                                stats=st if idx == 2 else None,
                                                graph_stats=gst if idx == 2 else None)
            rec = step_record(w2, wms, emean, emed, st if idx == 2 else None)
            if idx == 2:   # the single-block step: HBM-bound, reported with its roofline
                rec["roofline"] = roofline_of(w2, emean, algorithmic_flops(w2), algorithmic_bytes(w2))
                rec["latency_ms_per_block_graph"] = round(gst["median"], 5)
                rec["latency_ms_p10_p90_graph"] = [round(gst["p10"], 5), round(gst["p90"], 5)]
            extra.append(rec)
            del w2
            torch.cuda.empty_cache()
        extra.append(solver_loop_timing(dev))
        extra.append(backward_timing(dev))
    sweeps = [] if (args.no_extra or args.no_sweep) else run_sweeps(dev, 200)
    replays = [] if (args.no_extra or args.no_sweep) else [replay_timing(i, dev) for i in (1, 3, 4)]
    ceil = None if args.no_extra else ceilings(dev)
    if ceil is not None:
        # the headline against the measured ceiling too
        roof["frac_of_measured_ceiling"] = round(roof["achieved"] / (
            ceil["mfma_bf16_TFLOP/s"] if roof["bound"] == "mfma" else ceil["hbm_read_GB/s"]), 4)
        for rec in extra:
            r2 = rec.get("roofline")
            if r2:
                r2["frac_of_measured_ceiling"] = round(r2["achieved"] / (
                    ceil["mfma_bf16_TFLOP/s"] if r2["bound"] == "mfma" else ceil["hbm_read_GB/s"]), 4)
        for pt in sweeps:   # the binding roof rebuilt from the two measured ceilings
            attain = min(ceil["mfma_bf16_TFLOP/s"], pt["flop_per_byte"] * ceil["hbm_read_GB/s"] / 1e3)
            pt["frac_of_measured_bound"] = round(pt["TFLOP/s"] / attain, 4)
    cpu = None
    if not args.no_cpu:
        cpu = oracle_sample(wl)
        if not args.no_extra:
            for idx in (1, 2, 3, 4):
                if idx != args.config:
                    oracle_runs.append(oracle_sample(inputs.config(idx)))
            oracle_runs.append(cpu)
    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.B, "q_heads": wl.Hq, "kv_heads": wl.Hkv,
                   "head_dim": wl.D, "block_tokens": wl.Lq,
                   "cache_tokens": int(wl.cache_lens[0]) if wl.kind == "step" else 0,
                   "page_size": 64, "fused_append": bool(wl.fuse_append), "seed": wl.seed,
                   "parallelism": "none (1 GPU)"},
        "latency_ms_per_block": round(ev_med, 5),
        "latency_ms_p10_p90": [round(lat_stats["p10"], 5), round(lat_stats["p90"], 5)],
        "latency_ms_per_block_graph": round(graph_stats["median"], 5) if graph_stats else None,
        "latency_ms_p10_p90_graph": ([round(graph_stats["p10"], 5), round(graph_stats["p90"], 5)]
                                     if graph_stats else None),
        "roofline": roof,
        "cpu_baseline": cpu,
        "ceilings": ceil,
        "extra": extra,
        "sweeps": sweeps,
        "replays": replays,
        "oracle_by_workload": oracle_runs,
        "gpu": torch.cuda.get_device_name(0),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
