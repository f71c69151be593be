"""GPU parity with the layouts a Transformer layer produces: q, k and v as
strided views into one fused QKV projection output [B][L][Hq + 2 Hkv][d],
outputs and gradients written into views of larger buffers.  The C ABI takes
element strides, so these calls must match the contiguous ones bit for bit
and leave the rest of the buffers untouched."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _fused(B, L, Hq, Hkv, D, seed):
    qkv = inputs.bf16_normal(inputs.rng(seed, 7), (B, L, Hq + 2 * Hkv, D)).to(gs.dev())
    return qkv, qkv[:, :, :Hq], qkv[:, :, Hq:Hq + Hkv], qkv[:, :, Hq + Hkv:]


def test_prefill_fused_qkv_and_output_view():
    B, L, Hq, Hkv, D = 2, 500, 8, 2, 128
    qkv, q, k, v = _fused(B, L, Hq, Hkv, D, 101)
    offs = np.array([[0, 100, 101, 300, 500], [0, 250, 260, 261, 500]], np.int32)
    big = torch.full((B, L, Hq + 3, D), 5.0, dtype=torch.bfloat16, device=gs.dev())
    out = big[:, :, 2:2 + Hq]
    lse = torch.empty((B, Hq, L), dtype=torch.float32, device=gs.dev())
    gs.say("[gpu] prefill on fused-QKV views")
    ws.block_causal_prefill(q, k, v, offs, out=out, lse=lse, want_lse=True)
    ref_out, ref_lse = ws.block_causal_prefill(q.contiguous(), k.contiguous(), v.contiguous(), offs,
                                               want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
    assert (big[:, :, :2] == 5.0).all() and (big[:, :, 2 + Hq:] == 5.0).all()
    o64, l64 = oracle.prefill(inputs.bf16_bits(q.cpu()), inputs.bf16_bits(k.cpu()), inputs.bf16_bits(v.cpu()),
                              offs, 1.0 / np.sqrt(D))
    gs.assert_close(gs.compare(out, lse, o64, l64))


def test_step_fused_qkv_commit():
    B, Lq, Hq, Hkv, D = 2, 40, 8, 2, 128
    wl = inputs.step_workload("layout_step", B, Hq, Hkv, D, Lq, [300, 129], seed=103)
    qkv, q, kn, vn = _fused(B, Lq, Hq, Hkv, D, 103)
    c1 = gs.device_cache(wl, wl.cache_lens)
    c2 = gs.device_cache(wl, wl.cache_lens)
    gs.say("[gpu] step on fused-QKV views, committed")
    a = ws.block_causal_attn_fwd(q, kn, vn, c1, wl.cache_lens, fuse_append=True)
    b = ws.block_causal_attn_fwd(q.contiguous(), kn.contiguous(), vn.contiguous(), c2, wl.cache_lens,
                                 fuse_append=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(c1.k_pool.view(torch.int16), c2.k_pool.view(torch.int16))
    assert torch.equal(c1.v_pool.view(torch.int16), c2.v_pool.view(torch.int16))
    wl.q = q.cpu()
    wl.k[:, wl.Lc_max:] = kn.cpu()
    wl.v[:, wl.Lc_max:] = vn.cpu()
    ref, ref_lse = gs.run_oracle(wl)
    gs.assert_close(gs.compare(a, None, ref, ref_lse))


def test_backward_fused_qkv_gradient_views():
    """Gradients written straight into the slices of one fused dQKV buffer
    equal the contiguous call bit for bit."""
    B, L, Hq, Hkv, D = 1, 400, 8, 2, 64
    qkv, q, k, v = _fused(B, L, Hq, Hkv, D, 105)
    offs = np.array([[0, 64, 200, 201, 400]], np.int32)
    o, lse = ws.block_causal_prefill(q, k, v, offs, want_lse=True)
    dout = inputs.bf16_normal(inputs.rng(105, 9), (B, L, Hq, D)).to(gs.dev())
    dqkv = torch.full((B, L, Hq + 2 * Hkv, D), 3.0, dtype=torch.float32, device=gs.dev())
    gs.say("[gpu] backward into fused dQKV views")
    ws.block_causal_prefill_bwd(q, k, v, o, dout, lse, offs, dq=dqkv[:, :, :Hq], dk=dqkv[:, :, Hq:Hq + Hkv],
                                dv=dqkv[:, :, Hq + Hkv:])
    rq, rk, rv = ws.block_causal_prefill_bwd(q.contiguous(), k.contiguous(), v.contiguous(), o, dout, lse, offs)
    torch.cuda.synchronize()
    assert torch.equal(dqkv[:, :, :Hq], rq)
    assert torch.equal(dqkv[:, :, Hq:Hq + Hkv], rk)
    assert torch.equal(dqkv[:, :, Hq + Hkv:], rv)
