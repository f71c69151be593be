"""fp64 CPU oracle for block-causal attention and for paged-cache append.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg may use this package; the GPU library and its
Python binding never import it.

* ``prefill`` / ``step`` wrap the plain C triple loop in ``ws_oracle.c``
  (block-causal attention, Wan-Streamer v0.1 Abstract, Sec. 1 and Fig. 1;
  conditioning set of Sec. 2.1, Eq. 1), optionally with a token-causal
  segment at the end of each block (the thinker's language and state slots,
  Sec. 1 and Sec. 2.4).
* ``prefill_bwd``: gradients dQ, dK, dV of the whole-sequence path for an
  upstream output gradient (training uses the same causal format, Sec. 2.3).
* ``kv_append`` / ``gather`` are the paged full-history cache written out as
  plain per-token loops (the performer appends each received KV slice to its
  own full-history cache, Sec. 2.4).
* ``oracle.blocks`` computes the same outputs, lse and gradients one query
  block at a time with fp64 matmuls, for full-size checks of every element
  (pinned to the loops above).

Inputs are numpy arrays: float64, or uint16 holding bf16 bit patterns (which
the C code widens exactly).  All token tensors are contiguous [B][L][H][d].
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


def load(path=None):
    """Load (building it first if missing) the oracle shared library."""
    global _LIB
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _LIB is None:
        if not os.path.exists(_build.LIB) or (
                os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC)):
            _build.build()
        _LIB = _bind(ctypes.CDLL(_build.LIB))
    return _LIB


def _bind(lib):
    P = ctypes.c_void_p
    I = ctypes.c_int
    I64 = ctypes.c_int64
    D = ctypes.c_double
    lib.wso_prefill.argtypes = [P, P, P, I, I, I, I, I, I, P, I, D, P, I64, P, P, P, I]
    lib.wso_prefill.restype = I
    lib.wso_step.argtypes = [P, P, P, P, P, I, I, I, I, P, I, I, I, D, P, I64, P, P, P, I]
    lib.wso_step.restype = I
    lib.wso_prefill_text.argtypes = [P, P, P, I, I, I, I, I, I, P, I, P, D, P, I64, P, P, P, I]
    lib.wso_prefill_text.restype = I
    lib.wso_step_text.argtypes = [P, P, P, P, P, I, I, I, I, P, P, I, I, I, D, P, I64, P, P, P, I]
    lib.wso_step_text.restype = I
    lib.wso_step_varlen.argtypes = [P, P, P, P, P, I, I, I, I, P, P, P, I, I, I, D, P, I64, P, P, P, I]
    lib.wso_step_varlen.restype = I
    lib.wso_prefill_bwd.argtypes = [P, P, P, P, I, I, I, I, I, I, P, I, P, D, P, P, P, I]
    lib.wso_prefill_bwd.restype = I
    lib.wso_mutant.restype = I
    return lib


def default_threads():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _as_input(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.float64:
        return a, 0
    if a.dtype == np.uint16:
        return a, 1
    raise TypeError(f"oracle inputs must be float64 or uint16 (bf16 bits), got {a.dtype}")


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def prefill(q, k, v, offsets, scale, rows=None, want_probs=False, nthreads=None, lib=None,
            text_starts=None):
    """Block-causal attention over whole sequences.

    q: [B][L][Hq][d]; k, v: [B][L][Hkv][d]; offsets: [B][nb+1] int block
    boundaries (first 0, non-decreasing, last L).  text_starts: optional
    [B][nb] start of each block's token-causal segment (its block end: no
    segment; Sec. 1, Sec. 2.4).  rows: optional int array
    [n][3] of (b, h, i).  Returns (out, lse[, probs]): with rows=None,
    out [B][L][Hq][d] and lse [B][Hq][L]; with rows, out [n][d], lse [n] and
    probs [n][L].
    """
    lib = lib or load()
    q, dt = _as_input(q)
    k, dtk = _as_input(k)
    v, dtv = _as_input(v)
    assert dt == dtk == dtv
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape
    offsets = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32).reshape(B, -1))
    nb = offsets.shape[1] - 1
    if rows is None:
        out = np.empty((B, L, Hq, d), np.float64)
        lse = np.empty((B, Hq, L), np.float64)
        rows_a, n, probs = None, 0, None
    else:
        rows_a = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, 3))
        n = rows_a.shape[0]
        out = np.empty((n, d), np.float64)
        lse = np.empty((n,), np.float64)
        probs = np.zeros((n, L), np.float64) if want_probs else None
    ts = None
    if text_starts is not None:
        ts = np.ascontiguousarray(np.asarray(text_starts, dtype=np.int32).reshape(B, nb))
    rc = lib.wso_prefill_text(_ptr(q), _ptr(k), _ptr(v), dt, B, L, Hq, Hkv, d,
                              _ptr(offsets), nb, _ptr(ts), float(scale), _ptr(rows_a), n,
                              _ptr(out), _ptr(lse), _ptr(probs),
                              int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError(f"oracle prefill rejected its arguments (rc={rc})")
    return (out, lse, probs) if want_probs else (out, lse)


def step(q, k_cache, v_cache, cache_lens, k_new, v_new, scale, rows=None,
         want_probs=False, nthreads=None, lib=None, text_starts=None, new_lens=None):
    """One streaming step: the new block attends to its stream's cache
    (tokens [0, cache_lens[b])) and bidirectionally to itself, except for an
    optional token-causal segment starting at text_starts[b] within the
    block (Lq: none).  new_lens (optional, [B], 1..Lq): stream b's block has
    new_lens[b] tokens; the rest of its Lq positions are padding, never keys.

    q: [B][Lq][Hq][d]; k_cache, v_cache: [B][Lc_max][Hkv][d] logical cache;
    k_new, v_new: [B][Lq][Hkv][d].  Returns like ``prefill``; probs rows have
    length Lc_max + Lq, keys ordered cache then new.
    """
    lib = lib or load()
    q, dt = _as_input(q)
    kc, _ = _as_input(k_cache)
    vc, _ = _as_input(v_cache)
    kn, _ = _as_input(k_new)
    vn, _ = _as_input(v_new)
    B, Lq, Hq, d = q.shape
    Lc_max, Hkv = kc.shape[1], kc.shape[2]
    for a in (kc, vc, kn, vn):
        assert a.dtype == q.dtype
    assert kc.shape == (B, Lc_max, Hkv, d) and vc.shape == kc.shape
    assert kn.shape == (B, Lq, Hkv, d) and vn.shape == kn.shape
    lens = np.ascontiguousarray(np.asarray(cache_lens, dtype=np.int32).reshape(B))
    if rows is None:
        out = np.empty((B, Lq, Hq, d), np.float64)
        lse = np.empty((B, Hq, Lq), np.float64)
        rows_a, n, probs = None, 0, None
    else:
        rows_a = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, 3))
        n = rows_a.shape[0]
        out = np.empty((n, d), np.float64)
        lse = np.empty((n,), np.float64)
        probs = np.zeros((n, Lc_max + Lq), np.float64) if want_probs else None
    ts = None
    if text_starts is not None:
        ts = np.ascontiguousarray(np.asarray(text_starts, dtype=np.int32).reshape(B))
    nl = None
    if new_lens is not None:
        nl = np.ascontiguousarray(np.asarray(new_lens, dtype=np.int32).reshape(B))
    rc = lib.wso_step_varlen(_ptr(q), _ptr(kc), _ptr(vc), _ptr(kn), _ptr(vn), dt,
                             B, Lq, Lc_max, _ptr(lens), _ptr(nl), _ptr(ts), Hq, Hkv, d, float(scale),
                             _ptr(rows_a), n, _ptr(out), _ptr(lse), _ptr(probs),
                             int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError(f"oracle step rejected its arguments (rc={rc})")
    return (out, lse, probs) if want_probs else (out, lse)


def prefill_bwd(q, k, v, dout, offsets, scale, text_starts=None, nthreads=None, lib=None):
    """Gradients of ``prefill`` for an upstream output gradient dout
    [B][L][Hq][d] (training uses the same causal format, Sec. 2.3).
    Returns (dq [B][L][Hq][d], dk [B][L][Hkv][d], dv [B][L][Hkv][d]) in
    float64."""
    lib = lib or load()
    q, dt = _as_input(q)
    k, dtk = _as_input(k)
    v, dtv = _as_input(v)
    do, dto = _as_input(dout)
    assert dt == dtk == dtv == dto
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape and do.shape == q.shape
    offsets = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32).reshape(B, -1))
    nb = offsets.shape[1] - 1
    ts = None
    if text_starts is not None:
        ts = np.ascontiguousarray(np.asarray(text_starts, dtype=np.int32).reshape(B, nb))
    dq = np.empty((B, L, Hq, d), np.float64)
    dk = np.empty((B, L, Hkv, d), np.float64)
    dv = np.empty((B, L, Hkv, d), np.float64)
    rc = lib.wso_prefill_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(do), dt, B, L, Hq, Hkv, d,
                             _ptr(offsets), nb, _ptr(ts), float(scale), _ptr(dq), _ptr(dk), _ptr(dv),
                             int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError(f"oracle prefill_bwd rejected its arguments (rc={rc})")
    return dq, dk, dv


def kv_append(k_pool, v_pool, page_table, cache_lens, k_new, v_new):
    """Append a block of new tokens to a paged full-history cache, in place.

    Pools: [num_pages][Hkv][page_size][d] (any dtype, copied bit for bit);
    page_table: [B][max_pages] physical page of each logical page;
    k_new, v_new: [B][Ln][Hkv][d].  Token t of stream b lands at logical
    position p = cache_lens[b] + t, i.e. page page_table[b][p // page_size],
    slot p % page_size.
    """
    page_size = k_pool.shape[2]
    B, Ln = k_new.shape[0], k_new.shape[1]
    for b in range(B):
        for t in range(Ln):
            p = int(cache_lens[b]) + t
            phys = int(page_table[b][p // page_size])
            slot = p % page_size
            k_pool[phys, :, slot, :] = k_new[b, t]
            v_pool[phys, :, slot, :] = v_new[b, t]


def gather(pool, page_table_row, length):
    """Logical [length][Hkv][d] view of one stream read back through its
    page-table row (token p sits in page row[p // page_size], slot
    p % page_size)."""
    page_size = pool.shape[2]
    out = np.empty((length, pool.shape[1], pool.shape[3]), dtype=pool.dtype)
    for p in range(length):
        out[p] = pool[int(page_table_row[p // page_size]), :, p % page_size, :]
    return out
