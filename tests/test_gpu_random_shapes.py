"""GPU parity on seeded random shapes.  Each case draws, from its own seed,
the head counts (GQA ratio 1, 2, 3, 4 or 8 over 1-3 KV heads), the head dim
(64 or 128), the stream count, the block lengths (empty blocks included) or
the cache and new-block lengths (empty caches and one-token blocks
included), token-causal segments, paged or contiguous keys, bf16 or f32
output, blocks of different lengths and the fused append, so combinations
that no hand-picked case names are compared with the fp64 oracle on every
output row and lse (a step's padding rows aside), and a fused append's pool
with the oracle's append bit for bit.  Sizes keep the loop oracle near a
second per case.  Tolerance: max-abs 2e-2, mean-abs 2e-3, lse 1e-3."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _heads(g):
    hkv = int(g.integers(1, 4))
    return hkv * int(g.choice([1, 2, 3, 4, 8])), hkv


def _draw_prefill(seed):
    g = np.random.default_rng([seed, 2024])
    Hq, Hkv = _heads(g)
    D = int(g.choice([64, 128]))
    B = int(g.integers(1, 3))
    L = int(g.integers(1, 1201))
    nb = int(g.integers(1, min(L, 30) + 1))
    lens = []
    for _ in range(B):
        cuts = np.sort(g.integers(0, L + 1, size=nb - 1))   # repeated cuts give empty blocks
        lens.append(np.diff(np.concatenate([[0], cuts, [L]])))
    paged = bool(g.random() < 0.5)
    wl = inputs.prefill_workload(f"rand_prefill_{seed}", B, Hq, Hkv, D, lens, seed, paged=paged,
                                 out_f32=bool(g.random() < 0.3))
    if g.random() < 0.4:
        off = wl.offsets.astype(np.int64)
        wl.text_starts = np.array([[g.integers(off[b, n], off[b, n + 1] + 1) for n in range(nb)]
                                   for b in range(B)], np.int32)
    return wl


def _draw_step(seed):
    g = np.random.default_rng([seed, 2025])
    Hq, Hkv = _heads(g)
    D = int(g.choice([64, 128]))
    B = int(g.integers(1, 4))
    Lq = int(g.choice([int(g.integers(1, 9)), int(g.integers(1, 201))]))
    lens = [int(x) for x in g.integers(0, 4001, size=B)]
    if g.random() < 0.3:
        lens[int(g.integers(0, B))] = 0
    fuse = bool(g.random() < 0.5)
    wl = inputs.step_workload(f"rand_step_{seed}", B, Hq, Hkv, D, Lq, lens, seed, fuse_append=fuse)
    if g.random() < 0.3:
        wl.text_starts = g.integers(0, Lq + 1, size=B).astype(np.int32)
    if g.random() < 0.3 and Lq > 1:
        wl.new_lens = g.integers(1, Lq + 1, size=B).astype(np.int32)
        for b, n in enumerate(wl.new_lens):      # padding is never read: poison it
            wl.k[b, wl.Lc_max + int(n):] = float("nan")
            wl.v[b, wl.Lc_max + int(n):] = float("nan")
    out_dtype = torch.float32 if g.random() < 0.3 else torch.bfloat16
    return wl, out_dtype


def _describe(wl):
    extra = f" text={wl.text_starts is not None}"
    if wl.kind == "step":
        extra += f" cache={wl.cache_lens.tolist()} fuse={wl.fuse_append} new_lens={getattr(wl, 'new_lens', None)}"
    else:
        extra += f" paged={wl.paged} out_f32={wl.out_f32}"
    return f"[gpu] {wl.name}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Lq={wl.Lq}" + extra


@pytest.mark.parametrize("seed", range(24))
def test_random_prefill_shapes(seed):
    wl = _draw_prefill(seed)
    cache = gs.device_cache(wl, [wl.Lq] * wl.B) if wl.paged else None
    gs.say(_describe(wl))
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse))


@pytest.mark.parametrize("seed", range(24))
def test_random_step_shapes(seed):
    wl, out_dtype = _draw_step(seed)
    cache = gs.device_cache(wl, wl.cache_lens)
    gs.say(_describe(wl) + f" out={out_dtype}")
    out, lse = gs.run_gpu(wl, cache=cache, out_dtype=out_dtype)
    torch.cuda.synchronize()
    nl = getattr(wl, "new_lens", None)
    rows = None
    if nl is not None:
        rows = np.array([(b, h, t) for b in range(wl.B) for h in range(wl.Hq) for t in range(int(nl[b]))],
                        np.int32)
    ref, ref_lse = gs.run_oracle(wl, rows=rows)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse, rows=rows))
    if wl.fuse_append:
        # the pool as the oracle's append leaves it: each stream's real new
        # tokens after its cache, every other slot unchanged
        pk, pv = gs.cpu_pool(wl, wl.cache_lens)
        kb, vb = inputs.bf16_bits(wl.k_new), inputs.bf16_bits(wl.v_new)
        for b in range(wl.B):
            n = int(nl[b]) if nl is not None else wl.Lq
            oracle.kv_append(pk, pv, wl.page_table[b:b + 1], wl.cache_lens[b:b + 1], kb[b:b + 1, :n], vb[b:b + 1, :n])
        assert np.array_equal(cache.k_pool.view(torch.int16).cpu().numpy().view(np.uint16), pk)
        assert np.array_equal(cache.v_pool.view(torch.int16).cpu().numpy().view(np.uint16), pv)


@pytest.mark.parametrize("Hq,Hkv,D", [(16, 1, 128), (32, 2, 64), (64, 1, 128)])
def test_large_gqa_ratio_step_and_prefill(Hq, Hkv, D):
    """GQA ratios of 16, 32 and 64: a step packs (token, query head) rows of
    a KV group into 256-row tiles (64 heads fill a tile with 4 tokens), the
    prefill runs one query head per work item; full outputs against the
    oracle, and the step split across KV tiles."""
    g = np.random.default_rng([Hq, D, 2029])
    wl = inputs.step_workload(f"gqa{Hq // Hkv}_step", 2, Hq, Hkv, D, 37, [1500, 3100], seed=Hq + D)
    cache = gs.device_cache(wl, wl.cache_lens)
    gs.say(_describe(wl))
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse))
    L = 400
    cuts = np.sort(g.choice(np.arange(1, L), size=5, replace=False))
    lens = [np.diff(np.concatenate([[0], cuts, [L]]))]
    wp = inputs.prefill_workload(f"gqa{Hq // Hkv}_prefill", 1, Hq, Hkv, D, lens, seed=Hq + D + 1)
    gs.say(_describe(wp))
    out, lse = gs.run_gpu(wp)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wp)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse))
