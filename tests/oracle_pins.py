"""Pins for the fp64 oracle: checks against what the definition of
block-causal attention fixes, none of which reuses the oracle's own code.

Every pin is a function ``pin_*(lib)`` that raises AssertionError when the
oracle library ``lib`` disagrees with it.  ``test_oracle_pins.py`` runs them
on the real oracle; ``test_oracle_mutants.py`` runs them on deliberately
broken builds of the oracle and requires each broken build to fail at least
one pin.

The rule being pinned (Wan-Streamer v0.1, Abstract, Sec. 1 with Fig. 1 and
Sec. 5: block-causal attention over the interleaved stream; Sec. 2.1, Eq. 1:
unit k is conditioned on inputs of units <= k and responses of units < k):
a token sees every token of its own block and of every earlier block, and
nothing later (and, for the gradients, the chain rule through that
softmax).  With a token-causal segment at the end of a block (the
thinker's language and state slots, decoded token by token: Sec. 1 and
Sec. 2.4; next-token prediction of language, Sec. 2.1), the block's
observation tokens (before the segment) see each other but not the segment,
and a segment token sees the observations and the segment tokens up to
itself.
"""
import itertools
import math

import numpy as np
import torch

import oracle

ATOL_TIGHT = 1e-12


def _rng(*key):
    return np.random.default_rng(list(key))


def _offsets_from_lengths(lengths):
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


# --------------------------------------------------------------------------
# brute force: 1 head, 8 tokens, all 2^7 block compositions

def _brute_force_row(q, k, v, ids, i, scale):
    """Independent pure-Python definition for one query row."""
    visible = [j for j in range(len(ids)) if ids[j] <= ids[i]]
    logits = {j: scale * math.fsum(q[i][c] * k[j][c] for c in range(len(q[i])))
              for j in visible}
    m = max(logits.values())
    w = {j: math.exp(logits[j] - m) for j in visible}
    z = math.fsum(w.values())
    out = [math.fsum(w[j] * v[j][c] for j in visible) / z for c in range(len(v[0]))]
    return out, m + math.log(z)


def pin_bruteforce_all_compositions(lib, seeds=(0, 1, 2), n=8, d=4):
    scale = 0.7
    for seed in seeds:
        rng = _rng(11, seed)
        q = rng.standard_normal((1, n, 1, d))
        k = rng.standard_normal((1, n, 1, d))
        v = rng.standard_normal((1, n, 1, d))
        ql, kl, vl = q[0, :, 0].tolist(), k[0, :, 0].tolist(), v[0, :, 0].tolist()
        for comp in range(2 ** (n - 1)):
            # a boundary after token g when bit g is set
            ids = [bin(comp & ((1 << t) - 1)).count("1") for t in range(n)]
            cuts = [g + 1 for g in range(n - 1) if comp >> g & 1]
            offs = np.array([0] + cuts + [n], np.int32)[None]
            out, lse = oracle.prefill(q, k, v, offs, scale, nthreads=1, lib=lib)
            for i in range(n):
                ref_o, ref_lse = _brute_force_row(ql, kl, vl, ids, i, scale)
                assert np.all(np.isfinite(out[0, i, 0])), (comp, i)
                assert np.max(np.abs(out[0, i, 0] - ref_o)) <= ATOL_TIGHT, (seed, comp, i)
                assert abs(lse[0, 0, i] - ref_lse) <= ATOL_TIGHT, (seed, comp, i)


# --------------------------------------------------------------------------
# textbook special cases through an independent library routine (fp64 SDPA)

def _sdpa(q, k, v, scale, causal):
    """torch fp64 scaled_dot_product_attention on [B][L][H][d] arrays (MHA)."""
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)
    tk = torch.from_numpy(k).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v).permute(0, 2, 1, 3)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=causal, scale=scale)
    return o.permute(0, 2, 1, 3).numpy()


def _lse_ref(q, k, scale, causal):
    s = np.einsum("bihc,bjhc->bhij", q, k) * scale
    if causal:
        L = s.shape[-1]
        s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
    return torch.logsumexp(torch.from_numpy(s), dim=-1).numpy()


def pin_single_block_is_full_attention(lib):
    rng = _rng(12)
    B, L, H, d = 2, 37, 3, 16
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    scale = 1.0 / math.sqrt(d)
    offs = np.array([[0, L]] * B, np.int32)
    out, lse = oracle.prefill(q, k, v, offs, scale, lib=lib)
    ref = _sdpa(q, k, v, scale, causal=False)
    assert np.max(np.abs(out - ref)) <= 1e-12
    assert np.max(np.abs(lse - _lse_ref(q, k, scale, False))) <= 1e-12


def pin_unit_blocks_are_causal_attention(lib):
    rng = _rng(13)
    B, L, H, d = 2, 29, 2, 8
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    scale = 0.31
    offs = np.tile(np.arange(L + 1, dtype=np.int32), (B, 1))
    out, lse = oracle.prefill(q, k, v, offs, scale, lib=lib)
    ref = _sdpa(q, k, v, scale, causal=True)
    assert np.max(np.abs(out - ref)) <= 1e-12
    assert np.max(np.abs(lse - _lse_ref(q, k, scale, True))) <= 1e-12


# --------------------------------------------------------------------------
# closed forms and invariants

def _random_offsets(rng, L, nb):
    cuts = np.sort(rng.choice(np.arange(1, L), size=nb - 1, replace=False))
    return np.concatenate([[0], cuts, [L]]).astype(np.int32)


def pin_zero_query_is_mean_of_visible_values(lib):
    """Q = 0 makes every logit 0, so o_i is the plain mean of the visible
    values and lse_i = ln(#visible): counts the mask extent at every row."""
    rng = _rng(14)
    B, L, H, d = 1, 40, 1, 6
    q = np.zeros((B, L, H, d))
    k = rng.standard_normal((B, L, H, d))
    v = rng.standard_normal((B, L, H, d))
    offs = np.array([[0, 3, 4, 11, 11, 25, 40]], np.int32)  # includes an empty block
    out, lse = oracle.prefill(q, k, v, offs, 0.9, lib=lib)
    for i in range(L):
        end = next(int(e) for e in offs[0][1:] if e > i)  # end of i's block
        assert np.max(np.abs(out[0, i, 0] - v[0, :end, 0].mean(axis=0))) <= 1e-13, i
        assert abs(lse[0, 0, i] - math.log(end)) <= 1e-13, i


def pin_constant_values(lib):
    rng = _rng(15)
    B, L, H, d = 1, 33, 2, 5
    q = rng.standard_normal((B, L, H, d)) * 3
    k = rng.standard_normal((B, L, H, d)) * 3
    c = rng.standard_normal(d)
    v = np.broadcast_to(c, (B, L, H, d)).copy()
    offs = _random_offsets(rng, L, 5)[None]
    out, _ = oracle.prefill(q, k, v, offs, 0.5, lib=lib)
    assert np.max(np.abs(out - c)) <= 1e-13


def pin_probability_rows(lib):
    """Each probability row sums to 1; later blocks get exactly 0 weight and
    every visible key gets positive weight."""
    rng = _rng(16)
    B, L, H, d = 1, 24, 2, 4
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    offs = np.array([[0, 5, 6, 13, 24]], np.int32)
    rows = [(0, h, i) for h in range(H) for i in range(L)]
    _, _, P = oracle.prefill(q, k, v, offs, 0.8, rows=rows, want_probs=True, lib=lib)
    for r, (_, h, i) in enumerate(rows):
        end = next(int(e) for e in offs[0][1:] if e > i)
        assert abs(math.fsum(P[r]) - 1.0) <= 1e-12
        assert np.all(P[r, end:] == 0.0), (h, i)
        assert np.all(P[r, :end] > 0.0), (h, i)


def pin_appending_masked_block_keeps_earlier_rows(lib):
    """Adding a later block (which no earlier row may see) leaves every
    earlier row bitwise unchanged."""
    rng = _rng(17)
    B, L, H, d, extra = 2, 30, 2, 8, 9
    q, k, v = (rng.standard_normal((B, L + extra, H, d)) for _ in range(3))
    base = _random_offsets(rng, L, 4)
    o1, l1 = oracle.prefill(q[:, :L], k[:, :L], v[:, :L], np.stack([base] * B), 0.4, lib=lib)
    o2, l2 = oracle.prefill(q, k, v, np.stack([np.append(base, L + extra)] * B).astype(np.int32),
                            0.4, lib=lib)
    assert np.array_equal(o1, o2[:, :L])
    assert np.array_equal(l1, l2[:, :, :L])


def pin_permutation_symmetry(lib):
    """Permuting the tokens of one block permutes that block's output rows
    the same way; permuting the (k, v) pairs of earlier blocks leaves later
    rows unchanged (up to summation order)."""
    rng = _rng(18)
    B, L, H, d = 1, 30, 2, 6
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    offs = np.array([[0, 10, 18, 30]], np.int32)
    out, _ = oracle.prefill(q, k, v, offs, 0.6, lib=lib)
    perm = np.arange(L)
    perm[10:18] = 10 + rng.permutation(8)
    out2, _ = oracle.prefill(q[:, perm], k[:, perm], v[:, perm], offs, 0.6, lib=lib)
    assert np.max(np.abs(out2 - out[:, perm])) <= 1e-13
    perm = np.arange(L)
    perm[:18] = rng.permutation(18)
    k3, v3 = k.copy(), v.copy()
    k3[:, :18], v3[:, :18] = k[:, perm[:18]], v[:, perm[:18]]
    out3, _ = oracle.prefill(q, k3, v3, offs, 0.6, lib=lib)
    assert np.max(np.abs(out3[:, 18:] - out[:, 18:])) <= 1e-13
    # the first two blocks do see the permuted pairs
    assert np.max(np.abs(out3[:, :18] - out[:, :18])) > 1e-6


def pin_key_shift(lib):
    """Adding one vector c to every key shifts row i's logits by the
    constant scale*<q_i, c>: outputs unchanged, lse shifted by that constant."""
    rng = _rng(19)
    B, L, H, d = 1, 21, 1, 7
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    c = rng.standard_normal(d)
    offs = np.array([[0, 4, 9, 21]], np.int32)
    scale = 0.45
    o1, l1 = oracle.prefill(q, k, v, offs, scale, lib=lib)
    o2, l2 = oracle.prefill(q, k + c, v, offs, scale, lib=lib)
    assert np.max(np.abs(o1 - o2)) <= 1e-12
    shift = scale * np.einsum("bihc,c->bhi", q, c)
    assert np.max(np.abs(l2 - l1 - shift)) <= 1e-12


def pin_gqa_is_mha_with_repeated_kv(lib):
    """Query head h reads KV head floor(h / G)."""
    rng = _rng(20)
    B, L, Hkv, G, d = 1, 19, 3, 4, 5
    q = rng.standard_normal((B, L, Hkv * G, d))
    k = rng.standard_normal((B, L, Hkv, d))
    v = rng.standard_normal((B, L, Hkv, d))
    offs = np.array([[0, 7, 8, 19]], np.int32)
    o1, l1 = oracle.prefill(q, k, v, offs, 0.5, lib=lib)
    o2, l2 = oracle.prefill(q, np.repeat(k, G, axis=2), np.repeat(v, G, axis=2), offs, 0.5, lib=lib)
    assert np.array_equal(o1, o2)
    assert np.array_equal(l1, l2)


def pin_streaming_equals_prefill(lib):
    """Training and inference share one causal format (Sec. 2.3): prefill rows
    of block j equal a streaming step whose cache holds blocks < j."""
    rng = _rng(21)
    B, H, Hkv, d = 2, 4, 2, 8
    lengths = [5, 3, 7, 6]
    L = sum(lengths)
    q = rng.standard_normal((B, L, H, d))
    k = rng.standard_normal((B, L, Hkv, d))
    v = rng.standard_normal((B, L, Hkv, d))
    offs = _offsets_from_lengths(lengths)
    out, lse = oracle.prefill(q, k, v, np.stack([offs] * B), 0.7, lib=lib)
    for j in range(len(lengths)):
        s, e = int(offs[j]), int(offs[j + 1])
        so, sl = oracle.step(q[:, s:e], k[:, :s], v[:, :s], [s] * B, k[:, s:e], v[:, s:e],
                             0.7, lib=lib)
        assert np.array_equal(so, out[:, s:e]), j
        assert np.array_equal(sl, lse[:, :, s:e]), j


def pin_step_ragged_cache_lengths(lib):
    """Streams with different cache lengths: only the first cache_lens[b]
    cache tokens count (poisoning the rest changes nothing)."""
    rng = _rng(22)
    B, Lq, Lc, H, d = 3, 4, 9, 2, 4
    q = rng.standard_normal((B, Lq, H, d))
    kc = rng.standard_normal((B, Lc, H, d))
    vc = rng.standard_normal((B, Lc, H, d))
    kn = rng.standard_normal((B, Lq, H, d))
    vn = rng.standard_normal((B, Lq, H, d))
    lens = [0, 5, 9]
    o1, l1 = oracle.step(q, kc, vc, lens, kn, vn, 0.6, lib=lib)
    kc2, vc2 = kc.copy(), vc.copy()
    for b, n in enumerate(lens):
        kc2[b, n:] = 1e6
        vc2[b, n:] = np.nan
    o2, l2 = oracle.step(q, kc2, vc2, lens, kn, vn, 0.6, lib=lib)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    # stream with an empty cache is full attention over the new block
    ref = _sdpa(q[:1], kn[:1], vn[:1], 0.6, causal=False)
    assert np.max(np.abs(o1[:1] - ref)) <= 1e-12


def pin_bf16_inputs_are_widened_exactly(lib):
    """uint16 bf16 bit patterns give the same result as their exact fp64
    values passed directly."""
    rng = _rng(23)
    B, L, H, d = 1, 12, 2, 8
    f32 = [rng.standard_normal((B, L, H, d)).astype(np.float32) for _ in range(3)]
    bits = [torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
            for a in f32]
    vals = [torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy() for a in f32]
    offs = np.array([[0, 5, 12]], np.int32)
    o1, l1 = oracle.prefill(*bits, offs, 0.35, lib=lib)
    o2, l2 = oracle.prefill(*vals, offs, 0.35, lib=lib)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def pin_row_subset_matches_all_rows(lib):
    rng = _rng(24)
    B, L, H, Hkv, d = 2, 17, 4, 2, 6
    q = rng.standard_normal((B, L, H, d))
    k = rng.standard_normal((B, L, Hkv, d))
    v = rng.standard_normal((B, L, Hkv, d))
    offs = np.array([[0, 6, 17], [0, 1, 17]], np.int32)
    out, lse = oracle.prefill(q, k, v, offs, 0.5, lib=lib)
    rows = [(1, 3, 0), (0, 2, 16), (1, 0, 9), (0, 1, 5)]
    o2, l2 = oracle.prefill(q, k, v, offs, 0.5, rows=rows, lib=lib)
    for r, (b, h, i) in enumerate(rows):
        assert np.array_equal(o2[r], out[b, i, h]) and l2[r] == lse[b, h, i]


# --------------------------------------------------------------------------
# token-causal segments at the end of blocks

def _brute_force_text_row(q, k, v, ids, starts, i, scale):
    """Independent pure-Python rule for one query row: a token is an
    observation of its block before the block's segment start and a segment
    (text) token from there on; earlier blocks are always visible, and inside
    the block observations are visible to everyone there while segment
    tokens are visible only to segment tokens at or after them."""
    role = ["text" if j >= starts[ids[j]] else "obs" for j in range(len(ids))]
    visible = {j for j in range(len(ids))
               if ids[j] < ids[i] or (ids[j] == ids[i] and (role[j] == "obs" or (role[i] == "text" and j <= i)))}
    logits = {j: scale * math.fsum(q[i][c] * k[j][c] for c in range(len(q[i]))) for j in visible}
    m = max(logits.values())
    w = {j: math.exp(logits[j] - m) for j in visible}
    z = math.fsum(w.values())
    out = [math.fsum(w[j] * v[j][c] for j in sorted(visible)) / z for c in range(len(v[0]))]
    return out, m + math.log(z)


def pin_bruteforce_text_segments(lib, n=8, d=3):
    """Every block composition of 8 tokens with every choice of segment
    start in every block (11144 cases) against the pure-Python rule."""
    rng = _rng(31)
    q = rng.standard_normal((1, n, 1, d))
    k = rng.standard_normal((1, n, 1, d))
    v = rng.standard_normal((1, n, 1, d))
    ql, kl, vl = q[0, :, 0].tolist(), k[0, :, 0].tolist(), v[0, :, 0].tolist()
    scale = 0.8
    cases = 0
    for comp in range(2 ** (n - 1)):
        cuts = [g + 1 for g in range(n - 1) if comp >> g & 1]
        offs = [0] + cuts + [n]
        ids = [sum(1 for c in cuts if c <= t) for t in range(n)]
        choices = [range(offs[b], offs[b + 1] + 1) for b in range(len(offs) - 1)]
        for starts in itertools.product(*choices):
            out, lse = oracle.prefill(q, k, v, np.array([offs], np.int32), scale, nthreads=1, lib=lib,
                                      text_starts=np.array([starts], np.int32))
            for i in range(n):
                ref_o, ref_lse = _brute_force_text_row(ql, kl, vl, ids, starts, i, scale)
                assert np.max(np.abs(out[0, i, 0] - ref_o)) <= ATOL_TIGHT, (comp, starts, i)
                assert abs(lse[0, 0, i] - ref_lse) <= ATOL_TIGHT, (comp, starts, i)
            cases += 1
    assert cases == 11144


def pin_text_everywhere_is_causal_attention(lib):
    """Blocks that are all segment (start = block start) make every token
    see exactly the tokens up to itself: standard causal attention, whatever
    the block boundaries (fp64 SDPA is_causal)."""
    rng = _rng(32)
    B, L, H, d = 2, 31, 2, 8
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    offs = np.stack([_random_offsets(rng, L, 6) for _ in range(B)])
    out, lse = oracle.prefill(q, k, v, offs, 0.45, lib=lib, text_starts=offs[:, :-1])
    assert np.max(np.abs(out - _sdpa(q, k, v, 0.45, causal=True))) <= 1e-12
    assert np.max(np.abs(lse - _lse_ref(q, k, 0.45, True))) <= 1e-12


def pin_empty_segments_are_block_causal(lib):
    """Segments that start at the block end are empty: bitwise the plain
    block-causal result."""
    rng = _rng(33)
    B, L, H, Hkv, d = 2, 27, 4, 2, 5
    q = rng.standard_normal((B, L, H, d))
    k = rng.standard_normal((B, L, Hkv, d))
    v = rng.standard_normal((B, L, Hkv, d))
    offs = np.stack([_random_offsets(rng, L, 5) for _ in range(B)])
    o1, l1 = oracle.prefill(q, k, v, offs, 0.6, lib=lib)
    o2, l2 = oracle.prefill(q, k, v, offs, 0.6, lib=lib, text_starts=offs[:, 1:])
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def pin_zero_query_text_counts(lib):
    """Q = 0: o_i is the mean of the visible values and lse_i = ln(#visible).
    An observation token of block b sees [0, start_b); a segment token at i
    sees [0, i]."""
    rng = _rng(34)
    B, L, H, d = 1, 40, 1, 4
    q = np.zeros((B, L, H, d))
    k = rng.standard_normal((B, L, H, d))
    v = rng.standard_normal((B, L, H, d))
    offs = np.array([[0, 3, 4, 11, 11, 25, 40]], np.int32)
    starts = np.array([[1, 4, 8, 11, 25, 33]], np.int32)   # empty, whole, inner, empty block, empty, inner
    out, lse = oracle.prefill(q, k, v, offs, 0.9, lib=lib, text_starts=starts)
    for i in range(L):
        blk = next(b for b in range(6) if offs[0, b] <= i < offs[0, b + 1])
        n = int(starts[0, blk]) if i < starts[0, blk] else i + 1
        assert np.max(np.abs(out[0, i, 0] - v[0, :n, 0].mean(axis=0))) <= 1e-13, i
        assert abs(lse[0, 0, i] - math.log(n)) <= 1e-13, i


def pin_streaming_equals_prefill_text(lib):
    """Prefill rows of block j equal a streaming step of block j (its segment
    start given relative to the block) over a cache of blocks < j."""
    rng = _rng(35)
    B, H, Hkv, d = 2, 4, 2, 6
    lengths = [6, 4, 9, 5]
    rel = [[2, 4, 0, 5], [6, 1, 9, 3]]    # per stream, segment start within each block
    L = sum(lengths)
    q = rng.standard_normal((B, L, H, d))
    k = rng.standard_normal((B, L, Hkv, d))
    v = rng.standard_normal((B, L, Hkv, d))
    offs = _offsets_from_lengths(lengths)
    starts = np.array([[offs[j] + r[j] for j in range(4)] for r in rel], np.int32)
    out, lse = oracle.prefill(q, k, v, np.stack([offs] * B), 0.7, lib=lib, text_starts=starts)
    for j in range(len(lengths)):
        s, e = int(offs[j]), int(offs[j + 1])
        so, sl = oracle.step(q[:, s:e], k[:, :s], v[:, :s], [s] * B, k[:, s:e], v[:, s:e], 0.7,
                             lib=lib, text_starts=[r[j] for r in rel])
        assert np.array_equal(so, out[:, s:e]), j
        assert np.array_equal(sl, lse[:, :, s:e]), j


# --------------------------------------------------------------------------
# gradients (training uses the same causal format, Sec. 2.3)

def _visible(ids, starts, L):
    """Boolean [L][L] visibility from block ids and segment starts, written
    from the rule: earlier blocks, and inside the block observations (before
    the segment start) plus segment tokens up to the query."""
    vis = np.zeros((L, L), bool)
    for i in range(L):
        for j in range(L):
            same = ids[j] == ids[i]
            vis[i, j] = ids[j] < ids[i] or (same and (j < starts[ids[i]] or j <= i))
    return vis


def pin_bwd_matches_autograd(lib):
    """fp64 autograd through torch's scaled_dot_product_attention with the
    boolean mask of random block/segment layouts (GQA by repeating K/V)."""
    rng = _rng(41)
    for trial in range(4):
        B, L, Hkv, G, d = 1, 23, 2, 2, 6
        Hq = Hkv * G
        offs = _random_offsets(rng, L, 5)
        starts = np.array([rng.integers(offs[n], offs[n + 1] + 1) for n in range(5)], np.int32)
        text = None if trial == 0 else starts[None]
        q, do = (rng.standard_normal((B, L, Hq, d)) for _ in range(2))
        k, v = (rng.standard_normal((B, L, Hkv, d)) for _ in range(2))
        scale = 0.45
        dq, dk, dv = oracle.prefill_bwd(q, k, v, do, offs[None], scale, text_starts=text, lib=lib)
        ids = [int(np.searchsorted(offs, t, side="right") - 1) for t in range(L)]
        ids = [min(x, 4) for x in ids]
        vis = _visible(ids, starts if text is not None else offs[1:], L)
        tq, tk, tv = (torch.from_numpy(a.copy()).requires_grad_(True) for a in (q, k, v))
        kk = tk.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
        vv = tv.repeat_interleave(G, dim=2).permute(0, 2, 1, 3)
        o = torch.nn.functional.scaled_dot_product_attention(
            tq.permute(0, 2, 1, 3), kk, vv, attn_mask=torch.from_numpy(vis), scale=scale)
        o.permute(0, 2, 1, 3).backward(torch.from_numpy(do))
        assert np.max(np.abs(dq - tq.grad.numpy())) <= 1e-11, trial
        assert np.max(np.abs(dk - tk.grad.numpy())) <= 1e-11, trial
        assert np.max(np.abs(dv - tv.grad.numpy())) <= 1e-11, trial


def pin_bwd_finite_differences(lib):
    """Central differences of the oracle's own forward: d<O, dO>/dx."""
    rng = _rng(42)
    B, L, Hq, Hkv, d = 1, 7, 2, 1, 3
    q, do = (rng.standard_normal((B, L, Hq, d)) for _ in range(2))
    k, v = (rng.standard_normal((B, L, Hkv, d)) for _ in range(2))
    offs = np.array([[0, 2, 3, 7]], np.int32)
    starts = np.array([[1, 3, 5]], np.int32)
    scale = 0.7
    grads = oracle.prefill_bwd(q, k, v, do, offs, scale, text_starts=starts, lib=lib)

    def loss(q_, k_, v_):
        o, _ = oracle.prefill(q_, k_, v_, offs, scale, lib=lib, text_starts=starts)
        return float(np.sum(o * do))

    h = 1e-6
    for which, (x, g) in enumerate(zip((q, k, v), grads)):
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p[which], args_m[which] = xp, xm
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - g[idx]) <= 1e-7, (which, idx, fd, g[idx])


def pin_bwd_closed_forms(lib):
    """Rows of P sum to 1, so the dV of all keys sums to the sum of dO over
    the group's query rows and heads; rows of dS sum to 0, so the dK of all
    keys sums to 0; constant values make dS = 0, so dQ = dK = 0."""
    rng = _rng(43)
    B, L, Hkv, G, d = 2, 19, 2, 3, 4
    Hq = Hkv * G
    q, do = (rng.standard_normal((B, L, Hq, d)) for _ in range(2))
    k, v = (rng.standard_normal((B, L, Hkv, d)) for _ in range(2))
    offs = np.stack([_random_offsets(rng, L, 4) for _ in range(B)])
    dq, dk, dv = oracle.prefill_bwd(q, k, v, do, offs, 0.6, lib=lib)
    for g in range(Hkv):
        sum_do = do[:, :, g * G:(g + 1) * G].sum(axis=(1, 2))
        assert np.max(np.abs(dv[:, :, g].sum(axis=1) - sum_do)) <= 1e-12
    assert np.max(np.abs(dk.sum(axis=1))) <= 1e-12
    c = rng.standard_normal(d)
    vc = np.broadcast_to(c, v.shape).copy()
    dq, dk, dv = oracle.prefill_bwd(q, k, vc, do, offs, 0.6, lib=lib)
    assert np.max(np.abs(dq)) <= 1e-13 and np.max(np.abs(dk)) <= 1e-13


def pin_bwd_later_block_keeps_earlier_dq(lib):
    """A later block (invisible to earlier rows) leaves the earlier rows'
    dQ bitwise unchanged."""
    rng = _rng(44)
    B, L, H, d, extra = 1, 20, 2, 5, 6
    q, k, v, do = (rng.standard_normal((B, L + extra, H, d)) for _ in range(4))
    base = _random_offsets(rng, L, 3)
    dq1, _, _ = oracle.prefill_bwd(q[:, :L], k[:, :L], v[:, :L], do[:, :L], base[None], 0.5, lib=lib)
    dq2, _, _ = oracle.prefill_bwd(q, k, v, do, np.append(base, L + extra)[None].astype(np.int32), 0.5, lib=lib)
    assert np.array_equal(dq1, dq2[:, :L])


def pin_step_varlen_is_truncated_block(lib):
    """A step whose new blocks are padded to a common length equals, row for
    row, the step over each stream's real tokens only (bitwise): padding is
    never a key.  With a token-causal segment as well."""
    rng = _rng(45)
    B, Lq, Lc, H, Hkv, d = 3, 7, 9, 4, 2, 5
    q = rng.standard_normal((B, Lq, H, d))
    kc, vc = (rng.standard_normal((B, Lc, Hkv, d)) for _ in range(2))
    kn, vn = (rng.standard_normal((B, Lq, Hkv, d)) for _ in range(2))
    lens, new_lens, ts = [9, 0, 4], [7, 3, 1], [7, 1, 0]
    for text in (None, ts):
        o, l = oracle.step(q, kc, vc, lens, kn, vn, 0.6, lib=lib, new_lens=new_lens, text_starts=text)
        for b in range(B):
            n = new_lens[b]
            tb = None if text is None else [min(text[b], n)]
            o1, l1 = oracle.step(q[b:b + 1, :n], kc[b:b + 1], vc[b:b + 1], [lens[b]], kn[b:b + 1, :n],
                                 vn[b:b + 1, :n], 0.6, lib=lib, text_starts=tb)
            assert np.array_equal(o[b:b + 1, :n], o1), (b, text)
            assert np.array_equal(l[b:b + 1, :, :n], l1), (b, text)
    # padding values never matter (poisoned: same results)
    kn2, vn2 = kn.copy(), vn.copy()
    for b, n in enumerate(new_lens):
        kn2[b, n:] = 1e6
        vn2[b, n:] = np.nan
    o2, l2 = oracle.step(q, kc, vc, lens, kn2, vn2, 0.6, lib=lib, new_lens=new_lens)
    o3, l3 = oracle.step(q, kc, vc, lens, kn, vn, 0.6, lib=lib, new_lens=new_lens)
    assert np.array_equal(o2, o3) and np.array_equal(l2, l3)


ALL_PINS = [
    pin_bruteforce_all_compositions,
    pin_single_block_is_full_attention,
    pin_unit_blocks_are_causal_attention,
    pin_zero_query_is_mean_of_visible_values,
    pin_constant_values,
    pin_probability_rows,
    pin_appending_masked_block_keeps_earlier_rows,
    pin_permutation_symmetry,
    pin_key_shift,
    pin_gqa_is_mha_with_repeated_kv,
    pin_streaming_equals_prefill,
    pin_step_ragged_cache_lengths,
    pin_bf16_inputs_are_widened_exactly,
    pin_row_subset_matches_all_rows,
    pin_bruteforce_text_segments,
    pin_text_everywhere_is_causal_attention,
    pin_empty_segments_are_block_causal,
    pin_zero_query_text_counts,
    pin_streaming_equals_prefill_text,
    pin_bwd_matches_autograd,
    pin_bwd_finite_differences,
    pin_bwd_closed_forms,
    pin_bwd_later_block_keeps_earlier_dq,
    pin_step_varlen_is_truncated_block,
]

# the deliberately broken oracle builds (see WSO_MUTANT in ws_oracle.c)
MUTANTS = {
    1: "own block masked out",
    2: "softmax scale dropped",
    3: "GQA head map h % Hkv instead of h / G",
    4: "key index shifted by one",
    5: "lse missing ln(l)",
    6: "block boundary off by one",
    7: "output not normalised",
    8: "mask direction reversed",
    9: "segment token sees the next segment token",
    10: "observation tokens see their block's segment",
    11: "gradient: D_i term dropped from dS",
    12: "gradient: scale dropped from dK",
    13: "first padding token of a short new block used as a key",
    14: "gradient: dQ sums the values instead of the keys",
    15: "gradient: dV weighted by the unnormalised weights",
    16: "gradient: D_i sums dP without the softmax weights",
}
