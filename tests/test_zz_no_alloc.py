"""The allocation-free step entry point (ws_block_causal_attn_fwd_noalloc)
against the workspace entry point it mirrors (ws_block_causal_attn_fwd):
same plan, same kernels, so the outputs and lse must agree bit for bit.
Two calls in a row share the library's scratch array, the second on a
smaller step; a step whose partials exceed the array is rejected before
anything is enqueued."""
import numpy as np
import pytest
import torch

import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _case(name, B, Hq, Hkv, Lq, lens, seed, D=128):
    wl = inputs.step_workload(name, B, Hq, Hkv, D, Lq, lens, seed=seed)
    cache = gs.device_cache(wl, wl.cache_lens)
    dev = gs.dev()
    lens_h = torch.from_numpy(wl.cache_lens.astype(np.int32))
    bufs = dict(q=gs.to_dev_bf16(wl.q), k=gs.to_dev_bf16(wl.k_new), v=gs.to_dev_bf16(wl.v_new),
                lens=(lens_h, lens_h.to(dev)),
                out=torch.full((B, Lq, Hq, D), float("nan"), dtype=torch.bfloat16, device=dev),
                lse=torch.full((B, Hq, Lq), float("nan"), dtype=torch.float32, device=dev))
    return wl, cache, bufs


def _reference(wl, cache, b):
    return ws.block_causal_attn_fwd(b["q"], b["k"], b["v"], cache, b["lens"], scale=wl.scale, want_lse=True)


def _noalloc(wl, cache, b):
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    ws.block_causal_attn_fwd_noalloc(b["q"], b["k"], b["v"], cache, b["lens"], b["out"], lse=b["lse"],
                                     scale=wl.scale)
    assert torch.cuda.memory_allocated() == before   # nothing allocated on the way
    torch.cuda.synchronize()
    return b["out"], b["lse"]


def test_noalloc_matches_workspace_entry_point_twice():
    # first call: the single-block step shape (10 KV splits, 8 MB of partials)
    wl1, c1, b1 = _case("noalloc_step_big", 1, 24, 24, 256, [4096], seed=501)
    ns1, need1 = ws.step_plan(1, 24, 24, 256, wl1.cache_lens)
    assert ns1 > 1 and 0 < need1 <= ws.NOALLOC_SCRATCH_BYTES
    gs.say(f"[gpu] noalloc call 1: {wl1.name}, {ns1} splits, {need1} bytes of partials")
    o1, l1 = _noalloc(wl1, c1, b1)
    r1, rl1 = _reference(wl1, c1, b1)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), r1.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), rl1.view(torch.int32))
    # second call, smaller: GQA, 3 streams, ragged caches, fewer partials
    wl2, c2, b2 = _case("noalloc_step_small", 3, 8, 2, 37, [100, 2000, 0], seed=502)
    ns2, need2 = ws.step_plan(3, 8, 2, 37, wl2.cache_lens)
    assert ns2 > 1 and 0 < need2 < need1
    gs.say(f"[gpu] noalloc call 2: {wl2.name}, {ns2} splits, {need2} bytes of partials")
    o2, l2 = _noalloc(wl2, c2, b2)
    r2, rl2 = _reference(wl2, c2, b2)
    torch.cuda.synchronize()
    assert torch.equal(o2.view(torch.int16), r2.view(torch.int16))
    assert torch.equal(l2.view(torch.int32), rl2.view(torch.int32))
    # and both agree with the oracle within the output tolerance
    ref, ref_lse = gs.run_oracle(wl2)
    gs.assert_close(gs.compare(o2, l2, ref, ref_lse))


@pytest.mark.parametrize("seed", range(8))
def test_noalloc_random_shapes_match_workspace_entry_point(seed):
    """Seeded random steps (GQA ratio 1-8, head dim 64 or 128, 1-3 streams,
    blocks of 1-300 tokens over caches of 0-6000, so the split count varies
    from call to call on the shared scratch array), each bitwise the
    workspace entry point's result."""
    g = np.random.default_rng([seed, 2027])
    Hkv = int(g.integers(1, 4))
    Hq = Hkv * int(g.choice([1, 2, 3, 4, 8]))
    D = int(g.choice([64, 128]))
    B = int(g.integers(1, 4))
    Lq = int(g.integers(1, 301))
    lens = [int(x) for x in g.integers(0, 6001, size=B)]
    ns, need = ws.step_plan(B, Hq, Hkv, Lq, np.asarray(lens, np.int32))
    assert need <= ws.NOALLOC_SCRATCH_BYTES
    wl, cache, b = _case(f"noalloc_rand_{seed}", B, Hq, Hkv, Lq, lens, seed=600 + seed, D=D)
    gs.say(f"[gpu] {wl.name}: B={B} Hq={Hq} Hkv={Hkv} D={D} Lq={Lq} cache={lens}, {ns} splits")
    o, l = _noalloc(wl, cache, b)
    r, rl = _reference(wl, cache, b)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), r.view(torch.int16))
    assert torch.equal(l.view(torch.int32), rl.view(torch.int32))


def test_noalloc_rejects_steps_beyond_its_scratch():
    """MHA 32 x 128 with a 512-token block over 4096 cached tokens plans 4
    splits of 34 MB of partials, more than the scratch array: rejected on
    the host, outputs untouched."""
    wl, cache, b = _case("noalloc_too_big", 1, 32, 32, 512, [4096], seed=503)
    _, need = ws.step_plan(1, 32, 32, 512, wl.cache_lens)
    assert need > ws.NOALLOC_SCRATCH_BYTES
    with pytest.raises(ws.WsError) as e:
        ws.block_causal_attn_fwd_noalloc(b["q"], b["k"], b["v"], cache, b["lens"], b["out"], lse=b["lse"])
    assert e.value.name == "WS_ERR_WORKSPACE"
    torch.cuda.synchronize()
    assert torch.isnan(b["out"].float()).all() and torch.isnan(b["lse"]).all()
