"""Block-causal attention and its gradients, one query block at a time, with
fp64 matmuls on the CPU (TEST INFRASTRUCTURE ONLY, like the rest of this
package).

The results are the ones ``oracle.prefill`` / ``oracle.step`` /
``oracle.prefill_bwd`` compute with plain per-pair loops.  Those loops take
minutes to hours on full-size workloads; here the queries of one block share
their visible keys, so each block is a handful of dense fp64 products (a
library matmul as a step; no other reordering).  Only the summation order
differs from the loop oracle; the tests hold the two within 1e-12 of each
other on ragged, empty, unit, token-causal, grouped-query and padded cases.

Visibility (Abstract and Fig. 1: a token sees every token of its own block
and of earlier blocks; token-causal segment, Sec. 1 and Sec. 2.4): the
queries of block n = [s, e) see keys [0, e); when the block has a segment
starting at t, a key j of the block itself is visible to query i only if
j < t or j <= i.  A streaming step (Sec. 2.4) is the last block of such a
sequence: its queries see the cached keys and the new block's keys (with a
segment start: new key j visible to new query i iff j < t or j <= i; keys
past a stream's new-block length are padding, never visible).

Forward, per (stream, KV head g) and query block, with the G query heads of
g stacked:
    S = scale * Q K^T (masked entries -> -inf),  m = rowmax(S),
    P = exp(S - m),  l = rowsum(P),  O = (P V) / l,  lse = m + ln l.
Gradients, per (stream, KV head g) and query block n:
    S  = scale * Q_n K_{<e}^T             masked entries -> -inf
    P  = softmax over each row of S
    dP = dO_n V_{<e}^T,  D = rowsum(P * dP),  dS = P * (dP - D)
    dQ_n      = scale * dS K_{<e}
    dK_{<e}  += scale * dS^T Q_n   (summed over the G heads)
    dV_{<e}  += P^T dO_n           (summed over the G heads)
"""
import numpy as np
import torch


def _f64(a):
    """float64 tensor of a float64 array, or of uint16 bf16 bit patterns
    widened exactly."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.float64:
        return torch.from_numpy(a)
    if a.dtype == np.uint16:
        return torch.from_numpy((a.astype(np.uint32) << 16).view(np.float32)).double()
    raise TypeError(f"oracle inputs must be float64 or uint16 (bf16 bits), got {a.dtype}")


def _check(q, k, v, dout, offsets, text_starts):
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape
    assert Hkv > 0 and Hq % Hkv == 0
    assert q.dtype == k.dtype == v.dtype
    assert dout is None or (dout.shape == q.shape and dout.dtype == q.dtype)
    off = np.asarray(offsets, dtype=np.int64).reshape(B, -1)
    nb = off.shape[1] - 1
    for b in range(B):
        assert off[b, 0] == 0 and off[b, nb] == L and np.all(np.diff(off[b]) >= 0)
    ts = None if text_starts is None else np.asarray(text_starts, dtype=np.int64).reshape(B, nb)
    return off, ts


def _grads(Q, dO, pos, K, V, s, e, scale, t):
    """Gradients of queries Q, dO [.][r][d] at key positions pos (all in the
    block [s, e)) against their visible keys K, V [e][d].  Returns dQ
    [.][r][d], and dK, dV [e][d] summed over the leading axis."""
    S = scale * torch.matmul(Q, K.T)                              # [.][r][e]
    if t is not None and s <= t < e:
        j = torch.arange(s, e).view(1, -1)
        hidden = ~((j < t) | (j <= pos.view(-1, 1)))              # keys of the block itself
        S[:, :, s:e].masked_fill_(hidden, float("-inf"))
    P = torch.softmax(S, dim=-1)
    dP = torch.matmul(dO, V.T)
    Dn = (P * dP).sum(dim=-1, keepdim=True)
    dS = P * (dP - Dn)
    dQ = scale * torch.matmul(dS, K)
    dK = scale * torch.matmul(dS.transpose(1, 2), Q).sum(dim=0)
    dV = torch.matmul(P.transpose(1, 2), dO).sum(dim=0)
    return dQ, dK, dV


def prefill_bwd_group(q, k, v, dout, offsets, scale, b, g, n0=0, text_starts=None):
    """Gradients of stream b, KV head g, from query block n0 on.  Keys of
    block m are seen by the queries of blocks m and later only, so with
    lo = offsets[b][n0] the dK, dV of keys [lo, L) and the dQ of queries
    [lo, L) (the G query heads of g) are exact.  Inputs as ``prefill_bwd``.
    Returns float64 numpy (dq [L-lo][G][d], dk [L-lo][d], dv [L-lo][d])."""
    off, ts = _check(q, k, v, dout, offsets, text_starts)
    L, Hq, d = q.shape[1], q.shape[2], q.shape[3]
    G = Hq // k.shape[2]
    nb = off.shape[1] - 1
    heads = slice(g * G, (g + 1) * G)
    lo = int(off[b, n0])
    Qg = _f64(q[b, lo:, heads]).permute(1, 0, 2)       # [G][L-lo][d]
    dOg = _f64(dout[b, lo:, heads]).permute(1, 0, 2)
    Kg, Vg = _f64(k[b, :, g]), _f64(v[b, :, g])         # [L][d]
    dq = torch.empty((G, L - lo, d), dtype=torch.float64)
    dk = torch.zeros((L - lo, d), dtype=torch.float64)
    dv = torch.zeros((L - lo, d), dtype=torch.float64)
    for n in range(n0, nb):
        s, e = int(off[b, n]), int(off[b, n + 1])
        if e == s:
            continue
        t = None if ts is None else int(ts[b, n])
        dQ, dK, dV = _grads(Qg[:, s - lo:e - lo], dOg[:, s - lo:e - lo], torch.arange(s, e),
                            Kg[:e], Vg[:e], s, e, scale, t)
        dq[:, s - lo:e - lo] = dQ
        dk[:e - lo] += dK[lo:]
        dv[:e - lo] += dV[lo:]
    return dq.permute(1, 0, 2).numpy(), dk.numpy(), dv.numpy()


def prefill_bwd(q, k, v, dout, offsets, scale, text_starts=None):
    """Same arguments and results as ``oracle.prefill_bwd``: q, dout
    [B][L][Hq][d]; k, v [B][L][Hkv][d] (float64, or uint16 bf16 bits);
    offsets [B][nb+1]; optional text_starts [B][nb].  Returns float64
    (dq, dk, dv) numpy arrays."""
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    dq = np.empty((B, L, Hq, d))
    dk = np.empty((B, L, Hkv, d))
    dv = np.empty((B, L, Hkv, d))
    for b in range(B):
        for g in range(Hkv):
            dq[b, :, g * G:(g + 1) * G], dk[b, :, g], dv[b, :, g] = prefill_bwd_group(
                q, k, v, dout, offsets, scale, b, g, 0, text_starts)
    return dq, dk, dv


def prefill_dq_rows(q, k, v, dout, offsets, scale, rows, text_starts=None):
    """dQ of the query rows ``rows`` ([n][3] of (b, h, i)) only, as the
    matching rows of ``prefill_bwd``'s dq: returns float64 [n][d]."""
    off, ts = _check(q, k, v, dout, offsets, text_starts)
    G = q.shape[2] // k.shape[2]
    rows = np.asarray(rows, dtype=np.int64).reshape(-1, 3)
    out = np.empty((rows.shape[0], q.shape[3]), np.float64)
    by_block = {}
    for x, (b, h, i) in enumerate(rows):
        n = int(np.searchsorted(off[b], i, side="right")) - 1
        by_block.setdefault((int(b), int(h) // G, n), []).append(x)
    for (b, g, n), xs in by_block.items():
        s, e = int(off[b, n]), int(off[b, n + 1])
        t = None if ts is None else int(ts[b, n])
        h, pos = rows[xs, 1], rows[xs, 2]
        Q = _f64(q[b, pos, h])[None]                        # [1][m][d]
        dO = _f64(dout[b, pos, h])[None]
        dQ, _, _ = _grads(Q, dO, torch.from_numpy(pos), _f64(k[b, :e, g]), _f64(v[b, :e, g]), s, e,
                          scale, t)
        out[xs] = dQ[0].numpy()
    return out


def _softmax_out(S, V):
    """O = softmax(S) V and lse over the last axis of S (rows of -inf only
    where a row sees no key, which no valid input has)."""
    m = S.max(dim=-1, keepdim=True).values
    P = torch.exp(S - m)
    l = P.sum(dim=-1, keepdim=True)
    O = torch.matmul(P, V) / l
    return O, (m + torch.log(l)).squeeze(-1)


def prefill(q, k, v, offsets, scale, text_starts=None, groups=None):
    """Same arguments and results as ``oracle.prefill`` over all rows: q
    [B][L][Hq][d]; k, v [B][L][Hkv][d] (float64, or uint16 bf16 bits);
    offsets [B][nb+1]; optional text_starts [B][nb].  Returns float64 numpy
    (out [B][L][Hq][d], lse [B][Hq][L]).  groups: optional list of (b, g)
    to compute (the other entries are NaN)."""
    off, ts = _check(q, k, v, None, offsets, text_starts)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    nb = off.shape[1] - 1
    fill = 0.0 if groups is None else float("nan")
    out = np.full((B, L, Hq, d), fill)
    lse = np.full((B, Hq, L), fill)
    for b, g in (groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]):
        heads = slice(g * G, (g + 1) * G)
        Kg, Vg = _f64(k[b, :, g]), _f64(v[b, :, g])
        for n in range(nb):
            s, e = int(off[b, n]), int(off[b, n + 1])
            if e == s:
                continue
            Q = _f64(q[b, s:e, heads]).permute(1, 0, 2)          # [G][r][d]
            S = scale * torch.matmul(Q, Kg[:e].T)                # [G][r][e]
            t = None if ts is None else int(ts[b, n])
            if t is not None and s <= t < e:
                i = torch.arange(s, e).view(-1, 1)
                j = torch.arange(s, e).view(1, -1)
                S[:, :, s:e].masked_fill_(~((j < t) | (j <= i)), float("-inf"))
            O, ls = _softmax_out(S, Vg[:e])
            out[b, s:e, heads] = O.permute(1, 0, 2).numpy()
            lse[b, heads, s:e] = ls.numpy()
    return out, lse


def step(q, k_cache, v_cache, cache_lens, k_new, v_new, scale, text_starts=None, new_lens=None,
         groups=None, row_chunk=512):
    """Same arguments and results as ``oracle.step`` over all rows: q
    [B][Lq][Hq][d]; k_cache, v_cache [B][Lc_max][Hkv][d] (stream b's first
    cache_lens[b] tokens); k_new, v_new [B][Lq][Hkv][d]; optional text_starts
    [B] (segment start within the new block) and new_lens [B] (tokens of the
    new block; rows past it are padding and left NaN).  Returns float64 numpy
    (out [B][Lq][Hq][d], lse [B][Hq][Lq]).  groups: optional list of (b, g)
    to compute (the other entries are NaN).  The G heads x Lq rows of a KV
    head are taken row_chunk at a time."""
    B, Lq, Hq, d = q.shape
    Hkv = k_new.shape[2]
    assert Hkv > 0 and Hq % Hkv == 0 and k_new.shape == (B, Lq, Hkv, d) and v_new.shape == k_new.shape
    assert k_cache.shape[0] == B and k_cache.shape[2:] == (Hkv, d) and v_cache.shape == k_cache.shape
    G = Hq // Hkv
    out = np.full((B, Lq, Hq, d), np.nan)
    lse = np.full((B, Hq, Lq), np.nan)
    for b, g in (groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]):
        lc = int(cache_lens[b])
        nl = Lq if new_lens is None else int(new_lens[b])
        assert 0 <= lc <= k_cache.shape[1] and 1 <= nl <= Lq
        t = nl if text_starts is None else int(text_starts[b])
        assert 0 <= t <= Lq
        K = torch.cat([_f64(k_cache[b, :lc, g]), _f64(k_new[b, :nl, g])])    # [lc + nl][d]
        V = torch.cat([_f64(v_cache[b, :lc, g]), _f64(v_new[b, :nl, g])])
        Q = _f64(q[b, :nl, g * G:(g + 1) * G])                             # [nl][G][d]
        rows = Q.reshape(nl * G, d)                                        # row = token * G + head
        tok = torch.arange(nl).repeat_interleave(G)
        for r0 in range(0, nl * G, row_chunk):
            r1 = min(r0 + row_chunk, nl * G)
            S = scale * torch.matmul(rows[r0:r1], K.T)                      # [rows][lc + nl]
            i = tok[r0:r1].view(-1, 1)
            j = torch.arange(nl).view(1, -1)
            S[:, lc:].masked_fill_(~((j < t) | (j <= i)), float("-inf"))
            O, ls = _softmax_out(S, V)
            x = np.arange(r0, r1)
            tt, hh = x // G, g * G + x % G
            out[b, tt, hh] = O.numpy()
            lse[b, hh, tt] = ls.numpy()
    return out, lse
