"""GPU invariants of the block-causal path and bit-exact cache indexing."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _interleaved(name, nblocks, seed, Hq=4, Hkv=2, paged=False, B=1):
    g = inputs.rng(seed, inputs.S_LENGTHS)
    lens = inputs.interleaved_block_lengths(g, nblocks)
    return inputs.prefill_workload(name, B, Hq, Hkv, 128, [lens] * B, seed, paged=paged)


def test_append_bit_exact_through_page_table():
    """ws_kv_append in uneven slices equals the oracle's per-token append,
    bit for bit, on a shuffled pool; slots nobody owns keep their sentinel."""
    B, Hkv, D = 3, 2, 128
    final = np.array([37, 300, 69])
    wl = inputs.step_workload("append", B, 2, Hkv, D, 1, final, seed=3)
    cache = ws.PagedCache.allocate(wl.num_pages, Hkv, D, torch.from_numpy(wl.page_table),
                                   device=gs.dev(), fill_bits=gs.NAN_BITS)
    pk = np.full((wl.num_pages, Hkv, 64, D), gs.NAN_BITS, np.uint16)
    pv = pk.copy()
    kb, vb = inputs.bf16_bits(wl.k), inputs.bf16_bits(wl.v)
    kd, vd = gs.to_dev_bf16(wl.k), gs.to_dev_bf16(wl.v)
    cur = np.zeros(B, np.int32)
    # (streams appended together, slice length): ragged slices, pages
    # crossed mid-slice, sub-batches once the shorter streams are complete
    schedule = [([0, 1, 2], 5), ([0, 1, 2], 0), ([0, 1, 2], 17), ([0, 1, 2], 15),
                ([1, 2], 32), ([1], 64), ([1], 167)]
    for streams, n in schedule:
        gs.say(f"[gpu] append {n} tokens to streams {streams} at {cur[streams].tolist()}")
        sub = ws.PagedCache(cache.k_pool, cache.v_pool, torch.from_numpy(wl.page_table[streams]))
        lens = cur[streams].copy()
        knew = torch.stack([kd[b, int(cur[b]):int(cur[b]) + n] for b in streams])
        vnew = torch.stack([vd[b, int(cur[b]):int(cur[b]) + n] for b in streams])
        ws.kv_append(sub, lens, knew, vnew)
        oracle.kv_append(pk, pv, wl.page_table[streams], lens,
                         np.stack([kb[b, int(cur[b]):int(cur[b]) + n] for b in streams]),
                         np.stack([vb[b, int(cur[b]):int(cur[b]) + n] for b in streams]))
        cur[streams] += n
    assert np.array_equal(cur, final)
    torch.cuda.synchronize()
    gk = cache.k_pool.cpu().view(torch.int16).numpy().view(np.uint16)
    gv = cache.v_pool.cpu().view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(gk, pk)
    assert np.array_equal(gv, pv)
    for b in range(B):
        n = int(cur[b])
        assert np.array_equal(oracle.gather(gk, wl.page_table[b], n), kb[b, :n])
        assert np.array_equal(oracle.gather(gv, wl.page_table[b], n), vb[b, :n])
    # untouched slots still hold the sentinel
    assert int((gk == gs.NAN_BITS).sum()) == gk.size - int(final.sum()) * Hkv * D


def test_fused_append_matches_unfused():
    """WS_FUSE_APPEND commits the block exactly as ws_kv_append does and the
    attention output is bitwise the same."""
    wl = inputs.step_workload("fused", 3, 8, 2, 128, 200, [64, 1000, 5], seed=17)
    c1 = gs.device_cache(wl, wl.cache_lens)
    c2 = gs.device_cache(wl, wl.cache_lens)
    gs.say("[gpu] fused vs unfused step")
    out1, lse1 = gs.run_gpu(wl, cache=c1, fuse=False)
    ws.kv_append(c1, wl.cache_lens, gs.to_dev_bf16(wl.k_new), gs.to_dev_bf16(wl.v_new))
    out2, lse2 = gs.run_gpu(wl, cache=c2, fuse=True)
    torch.cuda.synchronize()
    assert torch.equal(out1, out2) and torch.equal(lse1, lse2)
    assert torch.equal(c1.k_pool.view(torch.int16), c2.k_pool.view(torch.int16))
    assert torch.equal(c1.v_pool.view(torch.int16), c2.v_pool.view(torch.int16))


def test_deterministic():
    wl = inputs.step_workload("det", 1, 8, 8, 128, 256, [3000], seed=19)
    cache = gs.device_cache(wl, wl.cache_lens)
    gs.say("[gpu] determinism")
    a, la = gs.run_gpu(wl, cache=cache)
    b, lb = gs.run_gpu(wl, cache=cache)
    wp = _interleaved("det_prefill", 8, 20)
    c, lc = gs.run_gpu(wp)
    d, ld = gs.run_gpu(wp)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)
    assert torch.equal(c, d) and torch.equal(lc, ld)


def test_paged_prefill_equals_contiguous():
    wl = _interleaved("paged_vs_contig", 9, 23, paged=True)
    cache = gs.device_cache(wl, [wl.Lq])
    gs.say("[gpu] paged vs contiguous prefill")
    a, la = gs.run_gpu(wl, cache=cache)
    wl.paged = False
    b, lb = gs.run_gpu(wl)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_streaming_replay_equals_prefill():
    """Sec. 2.3: training and inference share one causal format.  Block by
    block (step, then commit) reproduces the prefill rows of every block."""
    wl = _interleaved("replay", 6, 29, paged=True)
    gs.say("[gpu] streaming replay vs prefill")
    cache = gs.device_cache(wl, [wl.Lq])
    full, full_lse = gs.run_gpu(wl, cache=cache)
    sc = ws.PagedCache.allocate(wl.num_pages, wl.Hkv, wl.D, torch.from_numpy(wl.page_table),
                                device=gs.dev(), fill_bits=gs.NAN_BITS)
    q, k, v = gs.to_dev_bf16(wl.q), gs.to_dev_bf16(wl.k), gs.to_dev_bf16(wl.v)
    offs = wl.offsets[0]
    for j in range(len(offs) - 1):
        s, e = int(offs[j]), int(offs[j + 1])
        if e == s:
            continue
        out, lse = ws.block_causal_attn_fwd(q[:, s:e], k[:, s:e], v[:, s:e], sc, [s], scale=wl.scale,
                                            fuse_append=True, want_lse=True)
        err = (out.float() - full[:, s:e].float()).abs()
        assert err.max().item() <= 2e-2 and err.mean().item() <= 2e-3, j
        assert (lse - full_lse[:, :, s:e]).abs().max().item() <= 1e-3, j
    torch.cuda.synchronize()
    assert torch.equal(sc.k_pool.view(torch.int16), cache.k_pool.view(torch.int16))


def test_later_block_leaves_earlier_rows_bitwise():
    """Adding a later block, which no earlier row may see, leaves every
    earlier row's output and lse bitwise unchanged."""
    grown = _interleaved("grown", 6, 31)
    L5 = int(grown.offsets[0][5])
    prefix = inputs.Workload("prefix", "prefill", 1, grown.Hq, grown.Hkv, 128, grown.scale,
                             grown.q[:, :L5], grown.k[:, :L5], grown.v[:, :L5], L5,
                             offsets=grown.offsets[:, :6].copy())
    gs.say(f"[gpu] grow by one block: {L5} -> {grown.Lq} tokens")
    b, lb = gs.run_gpu(grown)
    c, lc = gs.run_gpu(prefix)
    torch.cuda.synchronize()
    assert torch.equal(b[:, :L5], c) and torch.equal(lb[:, :, :L5], lc)


def test_rejected_call_changes_nothing():
    """A call that fails validation leaves output, lse and pool untouched."""
    wl = inputs.step_workload("reject", 1, 4, 2, 128, 64, [200], seed=37)
    cache = gs.device_cache(wl, wl.cache_lens)
    out = torch.full((1, 64, 4, 128), 7.0, dtype=torch.bfloat16, device=gs.dev())
    lse = torch.full((1, 4, 64), 3.0, dtype=torch.float32, device=gs.dev())
    pool_before = cache.k_pool.clone()
    bad = ws.PagedCache(cache.k_pool, cache.v_pool, torch.from_numpy(wl.page_table))
    bad.page_table_host[0, 4] = wl.num_pages + 5  # page of positions 256.., only the append writes it
    with pytest.raises(ws.WsError) as exc:
        ws.block_causal_attn_fwd(gs.to_dev_bf16(wl.q), gs.to_dev_bf16(wl.k_new), gs.to_dev_bf16(wl.v_new),
                                 bad, wl.cache_lens, fuse_append=True, out=out, lse=lse, want_lse=True)
    assert exc.value.name == "WS_ERR_PAGE"
    torch.cuda.synchronize()
    assert (out == 7.0).all() and (lse == 3.0).all()
    assert torch.equal(cache.k_pool.view(torch.int16), pool_before.view(torch.int16))



def test_workspace_reuse():
    """One workspace serves consecutive split-KV steps: every call gives the
    same bits as a call with a freshly allocated workspace."""
    wl = inputs.step_workload("ws_reuse", 2, 8, 2, 128, 40, [3000, 1800], seed=29)
    cache = gs.device_cache(wl, wl.cache_lens)
    gs.say("[gpu] workspace reuse over 4 steps")
    host = torch.as_tensor(wl.cache_lens, dtype=torch.int32)
    lens = (host, host.to(gs.dev()))
    need = ws.workspace_bytes(ws.WS_OP_STEP, wl.B, wl.Hq, wl.Hkv, wl.Lq, int(host.max()) + wl.Lq)
    assert need > 0
    work = torch.full((need,), 0x5A, dtype=torch.uint8, device=gs.dev())   # contents are ignored
    q, kn, vn = gs.to_dev_bf16(wl.q), gs.to_dev_bf16(wl.k_new), gs.to_dev_bf16(wl.v_new)
    ref, ref_lse = ws.block_causal_attn_fwd(q, kn, vn, cache, lens, want_lse=True)
    for _ in range(4):
        out, lse = ws.block_causal_attn_fwd(q, kn, vn, cache, lens, want_lse=True, workspace=work)
        torch.cuda.synchronize()
        assert torch.equal(out, ref) and torch.equal(lse, ref_lse)


def test_solver_loop_then_commit():
    """The performer's loop (Sec. 2.4, Sec. 2.1): several solver steps of a
    noisy block attend to a fixed cache without changing it, then the clean
    block is committed.  Every step matches the oracle, the pool is bitwise
    unchanged until the commit, and the commit equals the oracle's append."""
    B, Hq, Hkv, D, Lq = 2, 8, 2, 128, 48
    lens = [700, 333]
    base = inputs.step_workload("solver_cache", B, Hq, Hkv, D, Lq, lens, seed=43)
    cache = gs.device_cache(base, base.cache_lens)
    pool_k0 = cache.k_pool.clone()
    pool_v0 = cache.v_pool.clone()
    gs.say("[gpu] solver loop: 3 uncommitted steps, then a committing step")
    wl = inputs.step_workload("solver_step", B, Hq, Hkv, D, Lq, lens, seed=43)
    for s in range(4):
        # the noisy block changes every step (its queries, keys and values);
        # the cached keys and values stay the same
        wl.q = inputs.bf16_normal(inputs.rng(500 + s, inputs.S_Q), tuple(wl.q.shape))
        wl.k[:, wl.Lc_max:] = inputs.bf16_normal(inputs.rng(500 + s, inputs.S_K), tuple(wl.k_new.shape))
        wl.v[:, wl.Lc_max:] = inputs.bf16_normal(inputs.rng(500 + s, inputs.S_V), tuple(wl.v_new.shape))
        commit = s == 3
        out, lse = gs.run_gpu(wl, cache=cache, fuse=commit)
        torch.cuda.synchronize()
        ref, ref_lse = gs.run_oracle(wl)
        gs.assert_close(gs.compare(out, lse, ref, ref_lse))
        if not commit:
            assert torch.equal(cache.k_pool.view(torch.int16), pool_k0.view(torch.int16))
            assert torch.equal(cache.v_pool.view(torch.int16), pool_v0.view(torch.int16))
    # the committed pool: the oracle appends the last step's block after each stream's cache
    pk = pool_k0.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    pv = pool_v0.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    oracle.kv_append(pk, pv, wl.page_table, np.asarray(lens), inputs.bf16_bits(wl.k_new), inputs.bf16_bits(wl.v_new))
    assert np.array_equal(cache.k_pool.view(torch.int16).cpu().numpy().view(np.uint16), pk)
    assert np.array_equal(cache.v_pool.view(torch.int16).cpu().numpy().view(np.uint16), pv)
