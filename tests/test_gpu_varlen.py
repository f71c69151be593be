"""GPU parity of steps over new blocks of different lengths: concurrent
streams, each at its own unit (units hold varying numbers of visual, audio
and text tokens, Sec. 2.2 and Sec. 2.4), padded to one new_len and run in one
launch through the *_varlen entry points, against the fp64 oracle.  Padding
tokens hold NaN, so a padding key that were read would show up.  Tolerance
as for the block-causal path: max-abs 2e-2, mean-abs 2e-3 (bf16 outputs),
lse 1e-3; cache contents bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _varlen(name, B, Hq, Hkv, D, Lq, lens, new_lens, seed, starts=None, fuse=False):
    wl = inputs.step_workload(name, B, Hq, Hkv, D, Lq, lens, seed, fuse_append=fuse)
    wl.new_lens = np.asarray(new_lens, np.int32)
    if starts is not None:
        wl.text_starts = np.asarray(starts, np.int32)
    for b, n in enumerate(wl.new_lens):
        wl.k[b, wl.Lc_max + int(n):] = float("nan")
        wl.v[b, wl.Lc_max + int(n):] = float("nan")
    return wl


def _real_rows(wl, heads=None):
    """Every (b, h, t) with t a real token of stream b (padding rows'
    outputs are unspecified)."""
    heads = range(wl.Hq) if heads is None else heads
    return np.array([(b, h, t) for b in range(wl.B) for h in heads for t in range(int(wl.new_lens[b]))],
                    np.int32)


def _real(out, lse, wl):
    """The real rows' outputs and lse, flattened (for bitwise comparisons)."""
    n = [int(x) for x in wl.new_lens]
    return (torch.cat([out[b, :n[b]].reshape(-1) for b in range(wl.B)]),
            torch.cat([lse[b, :, :n[b]].reshape(-1) for b in range(wl.B)]))


def _check_full(wl, cache, **kw):
    gs.say(f"[gpu] {wl.name}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Lq={wl.Lq} "
           f"new_lens={wl.new_lens.tolist()[:8]} text={None if wl.text_starts is None else wl.text_starts.tolist()[:8]}")
    out, lse = gs.run_gpu(wl, cache=cache, **kw)
    torch.cuda.synchronize()
    rows = _real_rows(wl)
    ref, ref_lse = gs.run_oracle(wl, rows=rows)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse, rows=rows))
    return out, lse


def _expected_pools(wl):
    """Pools after committing each stream's real new tokens (oracle append)."""
    pk, pv = gs.cpu_pool(wl, wl.cache_lens)
    kb, vb = inputs.bf16_bits(wl.k_new), inputs.bf16_bits(wl.v_new)
    for b in range(wl.B):
        n = int(wl.new_lens[b])
        oracle.kv_append(pk, pv, wl.page_table[b:b + 1], wl.cache_lens[b:b + 1], kb[b:b + 1, :n], vb[b:b + 1, :n])
    return pk, pv


def _pool_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("Lq,lens,new_lens,starts", [
    (100, [0, 333, 4100], [100, 37, 1], None),
    (100, [0, 333, 4100], [100, 37, 1], [0, 20, 1]),
    (300, [129, 0, 1000], [1, 300, 150], [0, 299, 150]),
])
def test_step_varlen_ragged(D, Lq, lens, new_lens, starts):
    wl = _varlen(f"varlen_step_d{D}_q{Lq}", 3, 8, 2, D, Lq, lens, new_lens, seed=71 + Lq + D, starts=starts)
    _check_full(wl, gs.device_cache(wl, wl.cache_lens))


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_step_varlen_token_causal_decode_gqa8(out_dtype):
    """Decode steps of 1 to 8 tokens over split caches (GQA 16/2)."""
    wl = _varlen("varlen_decode_gqa8", 3, 16, 2, 128, 8, [4100, 2500, 9000], [8, 3, 1], seed=73,
                 starts=[0, 0, 0])
    _check_full(wl, gs.device_cache(wl, wl.cache_lens), out_dtype=out_dtype)


def test_step_varlen_many_streams_from_memory():
    """More than 32 streams: lengths and starts are read from the device."""
    g = np.random.default_rng(75)
    lens = [int(x) for x in g.integers(0, 700, size=40)]
    wl = _varlen("varlen_step_b40", 40, 2, 1, 64, 8, lens, g.integers(1, 9, size=40), seed=75,
                 starts=g.integers(0, 9, size=40))
    _check_full(wl, gs.device_cache(wl, wl.cache_lens))


def test_fused_append_commits_only_real_tokens():
    """With WS_FUSE_APPEND the attention result (real rows) is bitwise that
    of the plain call, and the cache holds exactly the real tokens (padding
    slots keep their NaN fill).  In streams 1 and 2 (1 and 50 of 70 tokens)
    the second query tile (tokens 64..69) holds padding only and is skipped,
    while its work items' share of the append (from token 35 on) still
    holds real tokens of stream 2."""
    wl = _varlen("varlen_fused", 3, 8, 2, 128, 70, [10, 200, 640], [70, 1, 50], seed=77, starts=[70, 0, 5])
    cache = gs.device_cache(wl, wl.cache_lens)
    a, la = gs.run_gpu(wl, cache=cache, fuse=False)
    torch.cuda.synchronize()
    pk0 = _pool_bits(cache.k_pool)
    gs.say("[gpu] varlen fused append")
    b, lb = gs.run_gpu(wl, cache=cache, fuse=True)
    torch.cuda.synchronize()
    ra, rla = _real(a, la, wl)
    rb, rlb = _real(b, lb, wl)
    assert torch.equal(ra, rb) and torch.equal(rla, rlb)
    ek, ev = _expected_pools(wl)
    assert np.array_equal(_pool_bits(cache.k_pool), ek)
    assert np.array_equal(_pool_bits(cache.v_pool), ev)
    assert not np.array_equal(pk0, ek)


def test_kv_append_varlen_bit_exact():
    """ws_kv_append_varlen commits t < new_lens[b] only (a zero length too)."""
    wl = _varlen("varlen_append", 4, 4, 2, 64, 90, [0, 63, 64, 700], [90, 0, 1, 65], seed=79)
    cache = gs.device_cache(wl, wl.cache_lens)
    gs.say("[gpu] kv_append_varlen")
    ws.kv_append(cache, wl.cache_lens, gs.to_dev_bf16(wl.k_new), gs.to_dev_bf16(wl.v_new), new_lens=wl.new_lens)
    torch.cuda.synchronize()
    ek, ev = _expected_pools(wl)
    assert np.array_equal(_pool_bits(cache.k_pool), ek)
    assert np.array_equal(_pool_bits(cache.v_pool), ev)


def test_full_lengths_match_plain_bitwise():
    """new_lens all equal to new_len: bitwise the plain and _text entry points."""
    wl = inputs.step_workload("varlen_full", 2, 8, 2, 128, 40, [3000, 77], seed=81)
    cache = gs.device_cache(wl, wl.cache_lens)
    a, la = gs.run_gpu(wl, cache=cache)
    wl.new_lens = np.full(2, 40, np.int32)
    b, lb = gs.run_gpu(wl, cache=cache)
    wl.text_starts = np.array([5, 40], np.int32)
    c, lc = gs.run_gpu(wl, cache=cache)
    wl.new_lens = None
    d, ld = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)
    assert torch.equal(c, d) and torch.equal(lc, ld)


def test_varlen_equals_truncated_steps():
    """Each stream's real rows match a step over its real tokens alone (a
    different launch shape, so compared within the tolerance)."""
    wl = _varlen("varlen_vs_truncated", 3, 8, 2, 128, 64, [500, 64, 3000], [64, 9, 40], seed=83,
                 starts=[64, 3, 0])
    cache = gs.device_cache(wl, wl.cache_lens)
    out, lse = gs.run_gpu(wl, cache=cache)
    q, kn, vn = gs.to_dev_bf16(wl.q), gs.to_dev_bf16(wl.k_new), gs.to_dev_bf16(wl.v_new)
    for b in range(wl.B):
        n = int(wl.new_lens[b])
        one = ws.PagedCache(cache.k_pool, cache.v_pool, torch.from_numpy(wl.page_table[b:b + 1].copy()))
        o1, l1 = ws.block_causal_attn_fwd(q[b:b + 1, :n], kn[b:b + 1, :n], vn[b:b + 1, :n], one,
                                          [int(wl.cache_lens[b])], scale=wl.scale, want_lse=True,
                                          text_starts=[min(int(wl.text_starts[b]), n)])
        torch.cuda.synchronize()
        err = (o1.float() - out[b:b + 1, :n].float()).abs()
        assert err.max().item() <= 2e-2 and err.mean().item() <= 2e-3, b
        assert (l1 - lse[b:b + 1, :, :n]).abs().max().item() <= 1e-3, b


def test_thinker_decode_varlen_full_size():
    """The thinker's decode step at full size (4 x 131072 cache, GQA 64/8,
    blocks of 8) with streams at 8, 5, 1 and 3 new tokens, committed in the
    same launch; sampled rows, and the committed slots bit-exact."""
    wl = inputs.thinker_step()
    wl.new_lens = np.array([8, 5, 1, 3], np.int32)
    for b, n in enumerate(wl.new_lens):
        wl.k[b, wl.Lc_max + int(n):] = float("nan")
        wl.v[b, wl.Lc_max + int(n):] = float("nan")
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    rows = _real_rows(wl, heads=range(wl.Hq))
    gs.say(f"[gpu] {wl.name} varlen {wl.new_lens.tolist()}: full size, all {len(rows)} real rows")
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl, rows=rows)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse, rows=rows))
    # committed slots: real tokens bit-exact, the slot after them untouched (NaN)
    kb = inputs.bf16_bits(wl.k_new)
    pk = cache.k_pool
    for b in range(wl.B):
        for t in range(int(wl.new_lens[b]) + 1):
            pos = int(wl.cache_lens[b]) + t
            page = int(wl.page_table[b, pos // inputs.PAGE])
            got = pk[page, :, pos % inputs.PAGE].view(torch.int16).cpu().numpy().view(np.uint16)
            if t < wl.new_lens[b]:
                assert np.array_equal(got, kb[b, t]), (b, t)
            else:
                assert np.all(got == gs.NAN_BITS), (b, t)


def test_streams_varlen_full_size():
    """The bench's mixed-unit workload at full size: 4 streams over 131072
    cached tokens (GQA 64/8), each ingesting one interleaved unit of its own
    length (text segment token-causal), padded to the longest; sampled rows
    including each unit's first, segment-start and last token."""
    wl = inputs.streams_varlen()
    for b, n in enumerate(wl.new_lens):
        wl.k[b, wl.Lc_max + int(n):] = float("nan")
        wl.v[b, wl.Lc_max + int(n):] = float("nan")
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    must = []
    for b in range(wl.B):
        n, ts = int(wl.new_lens[b]), int(wl.text_starts[b])
        must += [(b, 0, 0), (b, 63, n - 1), (b, 17, ts), (b, 40, max(ts - 1, 0))]
    rows = gs.coverage_rows_step(np.random.default_rng(9), wl.B, wl.Hq, wl.Hkv, wl.Lq, must=must,
                                 new_lens=wl.new_lens)
    gs.say(f"[gpu] {wl.name} new_lens {wl.new_lens.tolist()}: full size, {len(rows)} rows")
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl, rows=rows)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse, rows=rows))


def test_many_streams_padding_tiles_fused_from_memory():
    """40 streams (lengths and cache lengths read from device memory), GQA 8
    (8 x 40 packed rows: two query tiles, the second starting at token 32),
    d = 64, committed in the same launch: streams of at most 32 tokens skip
    their second tile, whose work items still commit tokens from 20 on."""
    g = np.random.default_rng(85)
    lens = [int(x) for x in g.integers(0, 700, size=40)]
    n_new = [int(x) for x in g.integers(1, 41, size=40)]
    n_new[:4] = [21, 32, 33, 40]
    wl = _varlen("varlen_b40_fused", 40, 8, 1, 64, 40, lens, n_new, seed=85, starts=g.integers(0, 41, size=40),
                 fuse=True)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache)
    torch.cuda.synchronize()
    ek, ev = _expected_pools(wl)
    assert np.array_equal(_pool_bits(cache.k_pool), ek)
    assert np.array_equal(_pool_bits(cache.v_pool), ev)
