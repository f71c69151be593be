"""Gradients of whole-sequence block-causal attention, one query block at a
time, with fp64 matmuls on the CPU (TEST INFRASTRUCTURE ONLY, like the rest
of this package).

The result is the one ``oracle.prefill_bwd`` computes with plain per-pair
loops (training uses the same causal format as generation, Sec. 2.3).  Those
loops take tens of minutes on a full-size sequence; here the rows of one
query block share their visible keys, so each block is a handful of dense
fp64 products.  Only the summation order
differs from the loop oracle; the tests hold the two within 1e-12 of each
other on ragged, empty, unit, token-causal and grouped-query cases.

Visibility (Abstract and Fig. 1: a token sees every token of its own block
and of earlier blocks; token-causal segment, Sec. 1 and Sec. 2.4): the
queries of block n = [s, e) see keys [0, e); when the block has a segment
starting at t, a key j of the block itself is visible to query i only if
j < t or j <= i.

Per (stream, KV head g) and query block n, with the G query heads of g
stacked:
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
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape and dout.shape == q.shape
    assert Hkv > 0 and Hq % Hkv == 0
    assert q.dtype == k.dtype == v.dtype == dout.dtype
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
