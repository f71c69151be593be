"""Shared helpers of the GPU tests: move a synthetic workload to the device,
run the HIP path through the C ABI, run the fp64 oracle on the same inputs,
and compare.

Tolerance (bf16 inputs, fp32 accumulation, P rounded to bf16 before P.V,
bf16 output): max-abs <= 2e-2 and mean-abs <= 2e-3 against the fp64 oracle.
lse is fp32 end to end: |err| <= 1e-3.
"""
import sys

import numpy as np
import torch

import oracle
import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_ABS = 1e-3
NAN_BITS = 0x7FC1  # bf16 quiet NaN: unused pool slots hold it, so a stray read shows up


def say(msg):
    """Names the case before a GPU step (flushed, so it survives a crash)."""
    print(msg, file=sys.stderr, flush=True)


def dev():
    return torch.device("cuda:0")


def to_dev_bf16(t):
    return t.contiguous().to(dev())


def bits_to_dev(a):
    """uint16 bf16 bit array -> device bf16 tensor."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev())


def cpu_pool(wl, counts):
    """Pools filled on the CPU by the oracle's append: stream b holds its
    first counts[b] logical tokens; every other slot is NaN."""
    shape = (wl.num_pages, wl.Hkv, inputs.PAGE, wl.D)
    pk = np.full(shape, NAN_BITS, np.uint16)
    pv = np.full(shape, NAN_BITS, np.uint16)
    kb, vb = inputs.bf16_bits(wl.k), inputs.bf16_bits(wl.v)
    for b in range(wl.B):
        n = int(counts[b])
        oracle.kv_append(pk, pv, wl.page_table[b:b + 1], [0], kb[b:b + 1, :n], vb[b:b + 1, :n])
    return pk, pv


def device_cache(wl, counts, fill_on_gpu=False):
    """PagedCache on the device holding each stream's first counts[b] tokens.
    fill_on_gpu: fill with ws_kv_append instead of the CPU oracle (large
    workloads; the append kernel is checked bit-exactly elsewhere)."""
    if not fill_on_gpu:
        pk, pv = cpu_pool(wl, counts)
        return ws.PagedCache(bits_to_dev(pk), bits_to_dev(pv), torch.from_numpy(wl.page_table))
    cache = ws.PagedCache.allocate(wl.num_pages, wl.Hkv, wl.D, torch.from_numpy(wl.page_table),
                                   device=dev(), fill_bits=NAN_BITS)
    kd, vd = to_dev_bf16(wl.k), to_dev_bf16(wl.v)
    n = int(min(counts))
    assert all(int(c) == n for c in counts), "GPU fill needs equal counts"
    ws.kv_append(cache, [0] * wl.B, kd[:, :n], vd[:, :n])
    torch.cuda.synchronize()
    return cache


def run_gpu(wl, cache=None, out_dtype=None, want_lse=True, fuse=None):
    """The HIP path through the C ABI.  Returns (out, lse) on the device."""
    out_dtype = out_dtype or (torch.float32 if wl.out_f32 else torch.bfloat16)
    q = to_dev_bf16(wl.q)
    if wl.kind == "prefill":
        if wl.paged:
            return ws.block_causal_prefill(q, None, None, wl.offsets, scale=wl.scale, cache=cache,
                                           num_kv_heads=wl.Hkv, out_dtype=out_dtype, want_lse=want_lse,
                                           text_starts=wl.text_starts)
        return ws.block_causal_prefill(q, to_dev_bf16(wl.k), to_dev_bf16(wl.v), wl.offsets,
                                       scale=wl.scale, out_dtype=out_dtype, want_lse=want_lse,
                                       text_starts=wl.text_starts)
    fuse = wl.fuse_append if fuse is None else fuse
    return ws.block_causal_attn_fwd(q, to_dev_bf16(wl.k_new), to_dev_bf16(wl.v_new), cache,
                                    wl.cache_lens, scale=wl.scale, fuse_append=fuse,
                                    out_dtype=out_dtype, want_lse=want_lse, text_starts=wl.text_starts,
                                    new_lens=wl.new_lens)


def run_oracle(wl, rows=None):
    """fp64 oracle on the same bf16 inputs.  rows: optional (b, h, i) list."""
    if wl.kind == "prefill":
        return oracle.prefill(inputs.bf16_bits(wl.q), inputs.bf16_bits(wl.k), inputs.bf16_bits(wl.v),
                              wl.offsets, wl.scale, rows=rows, text_starts=wl.text_starts)
    return oracle.step(inputs.bf16_bits(wl.q), inputs.bf16_bits(wl.k_cache), inputs.bf16_bits(wl.v_cache),
                       wl.cache_lens, inputs.bf16_bits(wl.k_new), inputs.bf16_bits(wl.v_new), wl.scale,
                       rows=rows, text_starts=wl.text_starts, new_lens=wl.new_lens)


def compare(out, lse, ref_out, ref_lse, rows=None):
    """Element-wise errors of the device results against the oracle."""
    o = out.detach().to(torch.float64).cpu().numpy()
    l = lse.detach().to(torch.float64).cpu().numpy() if lse is not None else None
    if rows is not None:
        o = np.stack([o[b, i, h] for b, h, i in rows])
        if l is not None:
            l = np.array([l[b, h, i] for b, h, i in rows])
    err = np.abs(o - ref_out)
    stats = {"max_abs": float(err.max()) if err.size else 0.0,
             "mean_abs": float(err.mean()) if err.size else 0.0,
             "finite": bool(np.all(np.isfinite(o)))}
    if l is not None:
        stats["lse_max_abs"] = float(np.abs(l - ref_lse).max()) if l.size else 0.0
    return stats


def run_block_oracle(wl, groups=None):
    """Every output and lse of a workload from the block-wise fp64 oracle
    (``oracle.blocks``, pinned to the loop oracle): float64 numpy (out, lse);
    groups: optional (b, KV head) list to compute, the rest NaN (as are a
    step's padding rows)."""
    from oracle import blocks
    bits = inputs.bf16_bits
    if wl.kind == "step":
        return blocks.step(bits(wl.q), bits(wl.k_cache), bits(wl.v_cache), wl.cache_lens, bits(wl.k_new),
                           bits(wl.v_new), wl.scale, text_starts=wl.text_starts,
                           new_lens=getattr(wl, "new_lens", None), groups=groups)
    return blocks.prefill(bits(wl.q), bits(wl.k), bits(wl.v), wl.offsets, wl.scale,
                          text_starts=wl.text_starts, groups=groups)


def compare_all(out, lse, ref_out, ref_lse):
    """Element-wise errors over every output (and lse) the oracle computed
    (entries it left NaN are skipped)."""
    o = out.detach().to(torch.float64).cpu().numpy()
    sel = ~np.isnan(ref_out)
    err = np.abs(o[sel] - ref_out[sel])
    stats = {"elements": int(sel.sum()), "max_abs": float(err.max()), "mean_abs": float(err.mean()),
             "finite": bool(np.all(np.isfinite(o)))}
    if lse is not None:
        l = lse.detach().to(torch.float64).cpu().numpy()
        ls = ~np.isnan(ref_lse)
        stats["lse_max_abs"] = float(np.abs(l[ls] - ref_lse[ls]).max())
    return stats


def assert_close(stats):
    assert stats["finite"], stats
    assert stats["max_abs"] <= MAX_ABS, stats
    assert stats["mean_abs"] <= MEAN_ABS, stats
    if "lse_max_abs" in stats:
        assert stats["lse_max_abs"] <= LSE_ABS, stats


def coverage_rows_prefill(g, B, Hq, L, must=()):
    """(b, h, i) rows for a full-size prefill check: one row of every 32-row
    block of every (stream, query head), which is every wave of every work
    item (a work item is one query head's 256-row tile): the first row of a
    tile's first block, the last row of its last block, a random row of the
    others; plus the given rows."""
    rows = {tuple(int(x) for x in r) for r in must}
    for b in range(B):
        for h in range(Hq):
            for k in range(-(-L // 32)):
                lo, hi = 32 * k, min(32 * k + 32, L)
                if k % 8 == 0:
                    i = lo
                elif k % 8 == 7 or hi == L:
                    i = hi - 1
                else:
                    i = int(g.integers(lo, hi))
                rows.add((b, h, i))
    return np.array(sorted(rows), dtype=np.int32)


def coverage_rows_step(g, B, Hq, Hkv, Lq, must=(), new_lens=None):
    """(b, h, t) rows for a full-size step check.  A step packs the G query
    heads of a KV head into one row space, row p = t * G + hh; one row of
    every 32-row block of it per (stream, KV head), chosen as in
    ``coverage_rows_prefill`` (each 256-row tile's first and last row).
    Every such row sees every KV split.  new_lens: only real tokens."""
    G = Hq // Hkv
    rows = {tuple(int(x) for x in r) for r in must}
    for b in range(B):
        n = G * (Lq if new_lens is None else int(new_lens[b]))
        for kvh in range(Hkv):
            for k in range(-(-n // 32)):
                lo, hi = 32 * k, min(32 * k + 32, n)
                if k % 8 == 0:
                    p = lo
                elif k % 8 == 7 or hi == n:
                    p = hi - 1
                else:
                    p = int(g.integers(lo, hi))
                rows.add((b, kvh * G + p % G, p // G))
    return np.array(sorted(rows), dtype=np.int32)
