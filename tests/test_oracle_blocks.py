"""Pins of the block-wise fp64 oracle (``oracle.blocks``), used to check
full-size workloads on every output element and the full-size backward
element by element.  Forward and gradients must agree with the plain-loop
oracle (itself pinned by brute force, textbook cases, autograd, central
differences and planted mistakes) within 1e-12, and the gradients with
autograd of an explicitly masked softmax attention, on ragged, empty, unit,
single-block, token-causal, grouped-query and padded cases (Abstract, Fig.
1; Sec. 2.3 and Sec. 2.4)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import blocks


def _case(seed, B, L, Hq, Hkv, d, nb, empty=False):
    g = np.random.default_rng([seed, 5])
    offs = []
    for _ in range(B):
        cuts = np.sort(g.integers(0 if empty else 1, L + (1 if empty else 0), size=nb - 1))
        offs.append(np.concatenate([[0], cuts, [L]]))
    offs = np.asarray(offs, np.int32)
    q = g.standard_normal((B, L, Hq, d))
    k = 0.7 * g.standard_normal((B, L, Hkv, d))
    v = g.standard_normal((B, L, Hkv, d))
    do = g.standard_normal((B, L, Hq, d))
    return q, k, v, do, offs


def _text_starts(g, offs):
    B, nb = offs.shape[0], offs.shape[1] - 1
    ts = np.empty((B, nb), np.int32)
    for b in range(B):
        for n in range(nb):
            ts[b, n] = g.integers(offs[b, n], offs[b, n + 1] + 1)
    return ts


CASES = [
    dict(seed=1, B=2, L=97, Hq=4, Hkv=2, d=64, nb=5),
    dict(seed=2, B=1, L=130, Hq=6, Hkv=2, d=128, nb=7, empty=True),
    dict(seed=3, B=2, L=40, Hq=3, Hkv=3, d=64, nb=40),     # mostly unit blocks
    dict(seed=4, B=1, L=64, Hq=2, Hkv=1, d=64, nb=1),      # one block: bidirectional
]


@pytest.mark.parametrize("text", [False, True])
@pytest.mark.parametrize("c", CASES, ids=lambda c: f"s{c['seed']}")
def test_blocks_match_loop_oracle(c, text):
    q, k, v, do, offs = _case(**c)
    ts = _text_starts(np.random.default_rng([c["seed"], 6]), offs) if text else None
    scale = 0.11
    ref = oracle.prefill_bwd(q, k, v, do, offs, scale, text_starts=ts)
    got = blocks.prefill_bwd(q, k, v, do, offs, scale, text_starts=ts)
    for name, a, r in zip(("dq", "dk", "dv"), got, ref):
        err = np.abs(a - r).max()
        assert err <= 1e-12 * max(1.0, np.abs(r).max()), (name, err)


def test_blocks_match_autograd_of_a_dense_mask():
    """Autograd through softmax(scale Q K^T + mask) V with the mask written
    out entry by entry from the rule (own block and earlier blocks; inside a
    block with a segment starting at t, key j is visible to query i iff
    j < t or j <= i)."""
    q, k, v, do, offs = _case(seed=9, B=1, L=50, Hq=4, Hkv=2, d=64, nb=4)
    ts = np.array([[offs[0, 1], offs[0, 1] + 3, offs[0, 3] - 1, offs[0, 3]]], np.int32)
    scale = 0.2
    L = q.shape[1]
    blk = np.searchsorted(offs[0], np.arange(L), side="right") - 1
    mask = np.zeros((L, L), bool)
    for i in range(L):
        for j in range(L):
            vis = blk[j] <= blk[i]
            if vis and blk[j] == blk[i]:
                t = ts[0, blk[i]]
                vis = j < t or j <= i
            mask[i, j] = vis
    Q = torch.tensor(q[0], requires_grad=True)              # [L][Hq][d]
    K = torch.tensor(k[0], requires_grad=True)
    V = torch.tensor(v[0], requires_grad=True)
    Kx, Vx = K.repeat_interleave(2, dim=1), V.repeat_interleave(2, dim=1)
    S = scale * torch.einsum("ihc,jhc->hij", Q, Kx)
    S = S.masked_fill(~torch.from_numpy(mask), float("-inf"))
    O = torch.einsum("hij,jhc->ihc", torch.softmax(S, dim=-1), Vx)
    O.backward(torch.from_numpy(do[0]))
    got = blocks.prefill_bwd(q, k, v, do, offs, scale, text_starts=ts)
    for a, r in zip(got, (Q.grad, K.grad, V.grad)):
        assert np.abs(a[0] - r.numpy()).max() <= 1e-12


def test_partial_groups_are_exact_where_stated():
    q, k, v, do, offs = _case(seed=11, B=2, L=120, Hq=4, Hkv=2, d=64, nb=6, empty=True)
    ts = _text_starts(np.random.default_rng([11, 6]), offs)
    scale = 0.09
    full = blocks.prefill_bwd(q, k, v, do, offs, scale, text_starts=ts)
    for b, g, n0 in ((0, 1, 0), (1, 0, 4), (1, 1, 6)):
        lo = offs[b, n0]
        dq, dk, dv = blocks.prefill_bwd_group(q, k, v, do, offs, scale, b, g, n0, text_starts=ts)
        np.testing.assert_allclose(dq, full[0][b, lo:, 2 * g:2 * g + 2], rtol=0, atol=1e-13)
        np.testing.assert_allclose(dk, full[1][b, lo:, g], rtol=0, atol=1e-13)
        np.testing.assert_allclose(dv, full[2][b, lo:, g], rtol=0, atol=1e-13)


def test_dq_rows_match_the_full_gradient():
    q, k, v, do, offs = _case(seed=13, B=2, L=90, Hq=6, Hkv=3, d=64, nb=5, empty=True)
    ts = _text_starts(np.random.default_rng([13, 6]), offs)
    scale = 0.13
    dq = blocks.prefill_bwd(q, k, v, do, offs, scale, text_starts=ts)[0]
    g = np.random.default_rng(14)
    rows = np.stack([g.integers(0, 2, 40), g.integers(0, 6, 40), g.integers(0, 90, 40)], axis=1)
    got = blocks.prefill_dq_rows(q, k, v, do, offs, scale, rows, text_starts=ts)
    np.testing.assert_allclose(got, dq[rows[:, 0], rows[:, 2], rows[:, 1]], rtol=0, atol=1e-13)


@pytest.mark.parametrize("text", [False, True])
@pytest.mark.parametrize("c", CASES, ids=lambda c: f"s{c['seed']}")
def test_block_forward_matches_loop_oracle(c, text):
    q, k, v, _, offs = _case(**c)
    ts = _text_starts(np.random.default_rng([c["seed"], 6]), offs) if text else None
    ro, rl = oracle.prefill(q, k, v, offs, 0.11, text_starts=ts)
    go, gl = blocks.prefill(q, k, v, offs, 0.11, text_starts=ts)
    assert np.abs(go - ro).max() <= 1e-12 * max(1.0, np.abs(ro).max())
    assert np.abs(gl - rl).max() <= 1e-12 * max(1.0, np.abs(rl).max())


@pytest.mark.parametrize("text,padded", [(False, False), (True, False), (False, True), (True, True)])
def test_block_step_matches_loop_oracle(text, padded):
    g = np.random.default_rng([21, int(text), int(padded)])
    B, Lq, Hq, Hkv, d = 3, 37, 8, 2, 64
    lens = np.array([0, 130, 301])
    Lc = int(lens.max())
    q = g.standard_normal((B, Lq, Hq, d))
    kc = g.standard_normal((B, Lc, Hkv, d))
    vc = g.standard_normal((B, Lc, Hkv, d))
    kn = g.standard_normal((B, Lq, Hkv, d))
    vn = g.standard_normal((B, Lq, Hkv, d))
    ts = np.array([0, 17, Lq], np.int32) if text else None
    nl = np.array([Lq, 20, 1], np.int32) if padded else None
    ro, rl = oracle.step(q, kc, vc, lens, kn, vn, 0.125, text_starts=ts, new_lens=nl)
    go, gl = blocks.step(q, kc, vc, lens, kn, vn, 0.125, text_starts=ts, new_lens=nl, row_chunk=50)
    for b in range(B):
        n = Lq if nl is None else int(nl[b])
        assert np.abs(go[b, :n] - ro[b, :n]).max() <= 1e-12 * max(1.0, np.abs(ro[b, :n]).max())
        assert np.abs(gl[b, :, :n] - rl[b, :, :n]).max() <= 1e-12 * max(1.0, np.abs(rl[b, :, :n]).max())
        assert np.isnan(go[b, n:]).all()
