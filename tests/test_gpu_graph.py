"""The performer's solver loop (Sec. 2.4: per streaming unit, several
flow-matching solver steps of the noisy unit against the fixed full-history
cache, then the clean unit is committed; Sec. 1 and Sec. 2.4 mention graph
capture) recorded once into a HIP graph and replayed.  The entry points
enqueue kernels only (no allocation, synchronisation or memset), so the
whole loop can be captured; every replay, with eager work and
synchronisations in between, must give bitwise the eager results."""
import numpy as np
import pytest
import torch

import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _pair(a):
    h = torch.as_tensor(np.asarray(a), dtype=torch.int32).contiguous()
    return h, h.to(gs.dev())


def _loop_buffers(wl, steps, new_lens=None):
    """Device inputs of every solver step (a fresh noisy block each step) and
    preallocated outputs, lse and workspace."""
    qs, ks, vs = [], [], []
    for s in range(steps):
        qs.append(gs.to_dev_bf16(inputs.bf16_normal(inputs.rng(700 + s, inputs.S_Q), tuple(wl.q.shape))))
        ks.append(gs.to_dev_bf16(inputs.bf16_normal(inputs.rng(700 + s, inputs.S_K), tuple(wl.k_new.shape))))
        vs.append(gs.to_dev_bf16(inputs.bf16_normal(inputs.rng(700 + s, inputs.S_V), tuple(wl.v_new.shape))))
    outs = [torch.empty(tuple(wl.q.shape), dtype=torch.bfloat16, device=gs.dev()) for _ in range(steps)]
    lses = [torch.empty((wl.B, wl.Hq, wl.Lq), dtype=torch.float32, device=gs.dev()) for _ in range(steps)]
    if new_lens is None:
        need = ws.workspace_bytes(ws.WS_OP_STEP, wl.B, wl.Hq, wl.Hkv, wl.Lq, int(max(wl.cache_lens)) + wl.Lq)
    else:
        need = ws.step_workspace_bytes_varlen(wl.B, wl.Hq, wl.Hkv, wl.Lq, wl.cache_lens, new_lens)
    work = torch.empty(max(need, 16), dtype=torch.uint8, device=gs.dev())
    return qs, ks, vs, outs, lses, work


def _run_loop(cache, lens, text, bufs, new_lens=None):
    """steps - 1 uncommitted solver steps, then a step that commits its block."""
    qs, ks, vs, outs, lses, work = bufs
    n = len(qs)
    for s in range(n):
        ws.block_causal_attn_fwd(qs[s], ks[s], vs[s], cache, lens, fuse_append=(s == n - 1),
                                 out=outs[s], lse=lses[s], want_lse=True, workspace=work,
                                 text_starts=text, new_lens=new_lens)


def _real(t, n_real, tok_dim):
    """Rows of real tokens only (padding rows' outputs are unspecified)."""
    if n_real is None:
        return t
    return torch.cat([t[b].narrow(tok_dim - 1, 0, int(n)).reshape(-1) for b, n in enumerate(n_real)])


@pytest.mark.parametrize("mode", ["performer", "thinker", "mixed"])
def test_solver_loop_graph_replays_match_eager(mode):
    """performer: plain blocks; thinker: token-causal segments; mixed: new
    blocks of 48 and 21 tokens padded to 48, with segments."""
    starts = {"performer": None, "thinker": [0, 20], "mixed": [40, 5]}[mode]
    n_real = [48, 21] if mode == "mixed" else None
    _check_graph_loop(2, 8, 2, 128, 48, [700, 333], 71, starts, n_real, mode)


@pytest.mark.parametrize("seed", range(6))
def test_graph_replays_random_shapes(seed):
    """The same loop on seeded random shapes: GQA ratio 1-8 over 1-3 KV
    heads, head dim 64 or 128, 1-3 streams, blocks of 1-200 tokens over
    caches of 0-4000 (empty ones included), segments and blocks of
    different lengths in some."""
    g = np.random.default_rng([seed, 2028])
    Hkv = int(g.integers(1, 4))
    Hq = Hkv * int(g.choice([1, 2, 3, 4, 8]))
    D = int(g.choice([64, 128]))
    B = int(g.integers(1, 4))
    Lq = int(g.integers(1, 201))
    lens = [int(x) for x in g.integers(0, 4001, size=B)]
    if g.random() < 0.3:
        lens[int(g.integers(0, B))] = 0
    starts = [int(x) for x in g.integers(0, Lq + 1, size=B)] if g.random() < 0.4 else None
    n_real = [int(x) for x in g.integers(1, Lq + 1, size=B)] if g.random() < 0.3 and Lq > 1 else None
    _check_graph_loop(B, Hq, Hkv, D, Lq, lens, 7100 + seed, starts, n_real, f"random {seed}")


def _check_graph_loop(B, Hq, Hkv, D, Lq, lens, seed, starts, n_real, tag):
    """Eager loop against the oracle, then three replays of the captured
    loop (eager work and synchronisations in between), each bitwise the
    eager results: outputs, lse and the pool after the commit."""
    wl = inputs.step_workload("graph_loop", B, Hq, Hkv, D, Lq, lens, seed=seed)
    cache = gs.device_cache(wl, wl.cache_lens)
    k0, v0 = cache.k_pool.clone(), cache.v_pool.clone()
    lens_p = _pair(wl.cache_lens)
    text = _pair(np.array(starts)) if starts is not None else None
    nl = _pair(np.array(n_real)) if n_real is not None else None
    bufs = _loop_buffers(wl, 4, n_real)
    gs.say(f"[gpu] solver loop eager, {tag}: B={B} Hq={Hq} Hkv={Hkv} D={D} Lq={Lq} cache={lens} "
           f"starts={starts} new_lens={n_real}")
    _run_loop(cache, lens_p, text, bufs, nl)
    torch.cuda.synchronize()
    ref = [_real(o, n_real, 1).clone() for o in bufs[3]] + [_real(l, n_real, 2).clone() for l in bufs[4]]
    ref_k, ref_v = cache.k_pool.clone(), cache.v_pool.clone()
    # the eager loop matches the oracle (the last step sees its own block)
    wl.q = bufs[0][3].cpu()
    wl.k[:, wl.Lc_max:] = bufs[1][3].cpu()
    wl.v[:, wl.Lc_max:] = bufs[2][3].cpu()
    wl.text_starts = np.array(starts, np.int32) if starts is not None else None
    wl.new_lens = np.array(n_real, np.int32) if n_real is not None else None
    rows = None
    if n_real is not None:
        rows = np.array([(b, h, t) for b in range(B) for h in range(Hq) for t in range(n_real[b])], np.int32)
    o_ref, l_ref = gs.run_oracle(wl, rows=rows)
    gs.assert_close(gs.compare(bufs[3][3], bufs[4][3], o_ref, l_ref, rows=rows))

    gs.say("[gpu] capture")
    cache.k_pool.copy_(k0)
    cache.v_pool.copy_(v0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):      # warm-up on a side stream before capture
        _run_loop(cache, lens_p, text, bufs, nl)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _run_loop(cache, lens_p, text, bufs, nl)
    torch.cuda.synchronize()
    other = inputs.prefill_workload("graph_other", 1, 4, 2, 128, [np.array([100, 60])], 72)
    for rep in range(3):
        gs.say(f"[gpu] replay {rep}")
        cache.k_pool.copy_(k0)
        cache.v_pool.copy_(v0)
        for o in bufs[3] + bufs[4]:
            o.fill_(7.0)
        torch.cuda.synchronize()
        graph.replay()
        # eager work between replays
        gs.run_gpu(other)
        torch.cuda.synchronize()
        got = [_real(o, n_real, 1) for o in bufs[3]] + [_real(l, n_real, 2) for l in bufs[4]]
        for a, b in zip(got, ref):
            assert torch.equal(a, b), rep
        assert torch.equal(cache.k_pool.view(torch.int16), ref_k.view(torch.int16)), rep
        assert torch.equal(cache.v_pool.view(torch.int16), ref_v.view(torch.int16)), rep
