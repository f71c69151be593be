"""Block-causal streaming attention on MI355X (gfx950).

Thin ctypes binding over libwsattn.so (C ABI in include/ws_attn.h).  Python
only marshals arguments: every step of the computation runs in the HIP
kernels of csrc/.  PyTorch supplies device memory and the current stream.
If the library is missing this module raises; there is no fallback.

Entry points (same names as the C ABI, without the ``ws_`` prefix):
  kv_append(cache, cache_lens, k_new, v_new, new_lens=None)
  block_causal_attn_fwd(q, k_new, v_new, cache, cache_lens, ..., text_starts=None,
                        new_lens=None)
  block_causal_attn_fwd_noalloc(q, k_new, v_new, cache, (lens_host, lens_dev), out, ...)
  block_causal_prefill(q, k, v, block_offsets, ..., text_starts=None)
(with text_starts: the *_text entry points, blocks ending in a token-causal
segment; with new_lens: the *_varlen entry points, new blocks of different
lengths padded to a common one)
  block_causal_prefill_bwd(q, k, v, o, dout, lse, block_offsets, ...)
  workspace_bytes(op, batch, num_q_heads, num_kv_heads, max_q, max_k)
  step_workspace_bytes_varlen(batch, num_q_heads, num_kv_heads, new_len, cache_lens, new_lens)
  step_plan(batch, num_q_heads, num_kv_heads, new_len, cache_lens, new_lens=None, num_cus=0)
"""
import ctypes
import math
import os

import torch  # loads the HIP runtime that libwsattn.so then shares

from . import build as _build

__all__ = ["WsError", "PagedCache", "kv_append", "block_causal_attn_fwd", "block_causal_attn_fwd_noalloc",
           "block_causal_prefill", "block_causal_prefill_bwd", "workspace_bytes",
           "step_workspace_bytes_varlen", "step_plan", "library",
           "abi_version", "WS_OP_STEP", "WS_OP_PREFILL", "WS_OP_PREFILL_BWD", "PAGE_SIZE"]

WS_DTYPE_BF16, WS_DTYPE_F32 = 1, 2
WS_FUSE_APPEND = 1
WS_OP_STEP, WS_OP_PREFILL, WS_OP_PREFILL_BWD = 1, 2, 3
PAGE_SIZE = 64
NOALLOC_SCRATCH_BYTES = 32 << 20   # WS_NOALLOC_SCRATCH_BYTES of the C header
STATUS = {0: "WS_OK", 1: "WS_ERR_NULL", 2: "WS_ERR_SHAPE", 3: "WS_ERR_UNSUPPORTED",
          4: "WS_ERR_ALIGN", 5: "WS_ERR_OFFSETS", 6: "WS_ERR_PAGE", 7: "WS_ERR_CAPACITY",
          8: "WS_ERR_HEADS", 9: "WS_ERR_WORKSPACE", 10: "WS_ERR_HIP"}


class WsError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        self.name = STATUS.get(status, "WS_ERR_UNKNOWN")
        super().__init__(f"{self.name}: {detail}")


class Tensor4(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("stride_b", ctypes.c_int64), ("stride_t", ctypes.c_int64),
                ("stride_h", ctypes.c_int64)]


class PagedKVDesc(ctypes.Structure):
    _fields_ = [("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p),
                ("page_table_dev", ctypes.c_void_p), ("page_table_host", ctypes.c_void_p),
                ("num_pages", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pages_per_seq", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32)]


_LIB = None


def library():
    """The loaded libwsattn.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            raise RuntimeError(f"{_build.LIB} is not built; run `python -m paper_2606_25041_amd.build`")
        lib = ctypes.CDLL(_build.LIB)
        P, I32, I64, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        lib.ws_abi_version.restype = ctypes.c_int
        lib.ws_status_string.restype = ctypes.c_char_p
        lib.ws_status_string.argtypes = [ctypes.c_int]
        lib.ws_last_error.restype = ctypes.c_char_p
        lib.ws_workspace_bytes.restype = ctypes.c_size_t
        lib.ws_workspace_bytes.argtypes = [I32, I32, I32, I32, I32, I32]
        lib.ws_kv_append.restype = ctypes.c_int
        lib.ws_kv_append.argtypes = [ctypes.POINTER(PagedKVDesc), I32, P, P, I32, Tensor4, Tensor4, P]
        lib.ws_block_causal_attn_fwd.restype = ctypes.c_int
        lib.ws_block_causal_attn_fwd.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, I32, I32, I32, F, I32,
            Tensor4, P, P, ctypes.c_size_t, P]
        lib.ws_block_causal_prefill.restype = ctypes.c_int
        lib.ws_block_causal_prefill.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, I32, I32, I32, I32, I32,
            I32, F, Tensor4, P, P]
        lib.ws_block_causal_attn_fwd_text.restype = ctypes.c_int
        lib.ws_block_causal_attn_fwd_text.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, P, P, I32, I32, I32, F, I32,
            Tensor4, P, P, ctypes.c_size_t, P]
        lib.ws_block_causal_attn_fwd_varlen.restype = ctypes.c_int
        lib.ws_block_causal_attn_fwd_varlen.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, P, P, P, P, I32, I32, I32, F, I32,
            Tensor4, P, P, ctypes.c_size_t, P]
        lib.ws_step_workspace_bytes_varlen.restype = ctypes.c_size_t
        lib.ws_step_workspace_bytes_varlen.argtypes = [I32, I32, I32, I32, P, P]
        lib.ws_kv_append_varlen.restype = ctypes.c_int
        lib.ws_kv_append_varlen.argtypes = [ctypes.POINTER(PagedKVDesc), I32, P, P, P, P, I32, Tensor4, Tensor4, P]
        lib.ws_block_causal_prefill_text.restype = ctypes.c_int
        lib.ws_block_causal_prefill_text.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, P, P, I32, I32, I32, I32, I32,
            I32, F, Tensor4, P, P]
        lib.ws_block_causal_prefill_bwd.restype = ctypes.c_int
        lib.ws_block_causal_prefill_bwd.argtypes = [
            Tensor4, Tensor4, Tensor4, Tensor4, Tensor4, P, P, P, P, P, I32, I32, I32, I32, I32, I32, F,
            Tensor4, Tensor4, Tensor4, P, ctypes.c_size_t, P]
        lib.ws_block_causal_attn_fwd_noalloc.restype = ctypes.c_int
        lib.ws_block_causal_attn_fwd_noalloc.argtypes = [
            Tensor4, Tensor4, Tensor4, ctypes.POINTER(PagedKVDesc), P, P, I32, I32, I32, F, I32,
            Tensor4, P, P]
        lib.ws_step_plan.restype = ctypes.c_int
        lib.ws_step_plan.argtypes = [I32, I32, I32, I32, I32, P, P, ctypes.POINTER(I32),
                                     ctypes.POINTER(ctypes.c_size_t)]
        if lib.ws_abi_version() != 5:
            raise RuntimeError("libwsattn.so ABI version mismatch")
        _LIB = lib
    return _LIB


def abi_version():
    return library().ws_abi_version()


def _check(rc):
    if rc != 0:
        raise WsError(rc, library().ws_last_error().decode())


def _t4(t):
    """Tensor4 descriptor of a [B][L][H][d] tensor (None -> NULL)."""
    if t is None:
        return Tensor4(None, WS_DTYPE_BF16, 0, 0, 0)
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("token tensors must be 4-d [B][L][H][d] with a contiguous last dim")
    if t.dtype == torch.bfloat16:
        dt = WS_DTYPE_BF16
    elif t.dtype == torch.float32:
        dt = WS_DTYPE_F32
    else:
        raise ValueError(f"unsupported dtype {t.dtype}")
    return Tensor4(t.data_ptr(), dt, t.stride(0), t.stride(1), t.stride(2))


def _shape(name, t, shape):
    """Shapes are checked here because the C ABI only sees pointers and
    strides: a tensor smaller than the call implies would be read past its end."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t is not None and not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


class PagedCache:
    """Caller-owned paged full-history KV cache.

    k_pool, v_pool: bf16 device [num_pages][num_kv_heads][64][head_dim];
    page_table: int32 [batch][max_pages_per_seq] (kept on host and device).
    """

    def __init__(self, k_pool, v_pool, page_table):
        assert k_pool.shape == v_pool.shape and k_pool.dim() == 4
        assert k_pool.shape[2] == PAGE_SIZE
        self.k_pool, self.v_pool = k_pool, v_pool
        self.page_table_host = page_table.to(torch.int32).cpu().contiguous()
        self.page_table = self.page_table_host.to(k_pool.device)
        self.num_pages, self.num_kv_heads, _, self.head_dim = k_pool.shape

    @classmethod
    def allocate(cls, num_pages, num_kv_heads, head_dim, page_table, device="cuda", fill_bits=None):
        """New pools; fill_bits: optional 16-bit pattern written to every slot."""
        shape = (num_pages, num_kv_heads, PAGE_SIZE, head_dim)
        k = torch.empty(shape, dtype=torch.bfloat16, device=device)
        v = torch.empty(shape, dtype=torch.bfloat16, device=device)
        if fill_bits is not None:
            bits = int(fill_bits) - 0x10000 if int(fill_bits) >= 0x8000 else int(fill_bits)
            k.view(torch.int16).fill_(bits)
            v.view(torch.int16).fill_(bits)
        return cls(k, v, page_table)

    def desc(self):
        return PagedKVDesc(self.k_pool.data_ptr(), self.v_pool.data_ptr(),
                           self.page_table.data_ptr(), self.page_table_host.data_ptr(),
                           self.num_pages, PAGE_SIZE, self.page_table_host.shape[1],
                           self.num_kv_heads, self.head_dim)


def _lens(cache_lens, device):
    """(host int32 tensor, device int32 tensor) from a list / tensor / pair."""
    if isinstance(cache_lens, tuple):
        host, dev = cache_lens
        return host, dev
    host = torch.as_tensor(cache_lens, dtype=torch.int32).cpu().contiguous()
    return host, host.to(device)


def _check_lens(host, dev, B):
    if host.shape != (B,) or dev.shape != (B,) or host.dtype != torch.int32 or dev.dtype != torch.int32:
        raise ValueError("cache_lens must be int32 [B] on host and device")


def _check_table(cache, B):
    if cache.page_table_host.shape[0] < B or cache.page_table.shape != cache.page_table_host.shape:
        raise ValueError("page table has fewer rows than the batch")


def workspace_bytes(op, batch, num_q_heads, num_kv_heads, max_q, max_k):
    return library().ws_workspace_bytes(op, batch, num_q_heads, num_kv_heads, max_q, max_k)


def step_workspace_bytes_varlen(batch, num_q_heads, num_kv_heads, new_len, cache_lens, new_lens):
    """Workspace bytes of a step over blocks of different lengths (host
    int32 arrays or tensors of [batch])."""
    ch = torch.as_tensor(cache_lens, dtype=torch.int32).cpu().contiguous()
    nh = torch.as_tensor(new_lens, dtype=torch.int32).cpu().contiguous()
    return library().ws_step_workspace_bytes_varlen(batch, num_q_heads, num_kv_heads, new_len, ch.data_ptr(),
                                                    nh.data_ptr())


def step_plan(batch, num_q_heads, num_kv_heads, new_len, cache_lens, new_lens=None, num_cus=0):
    """(KV split count, workspace bytes) of a step planned for num_cus
    compute units (0: the current device's)."""
    ch = torch.as_tensor(cache_lens, dtype=torch.int32).cpu().contiguous()
    nh = None if new_lens is None else torch.as_tensor(new_lens, dtype=torch.int32).cpu().contiguous()
    ns, nbytes = ctypes.c_int32(0), ctypes.c_size_t(0)
    _check(library().ws_step_plan(num_cus, batch, num_q_heads, num_kv_heads, new_len, ch.data_ptr(),
                                  _ptr(nh), ctypes.byref(ns), ctypes.byref(nbytes)))
    return ns.value, nbytes.value


def kv_append(cache, cache_lens, k_new, v_new, new_lens=None):
    """Commit k_new/v_new [B][Ln][Hkv][d] at positions cache_lens[b] + t
    (only t < new_lens[b] when new_lens, [B], is given)."""
    host, dev = _lens(cache_lens, k_new.device)
    B, Ln = k_new.shape[0], k_new.shape[1]
    _shape("k_new", k_new, (B, Ln, cache.num_kv_heads, cache.head_dim))
    _shape("v_new", v_new, (B, Ln, cache.num_kv_heads, cache.head_dim))
    _check_lens(host, dev, B)
    _check_table(cache, B)
    desc = cache.desc()
    if new_lens is None:
        _check(library().ws_kv_append(ctypes.byref(desc), B, host.data_ptr(), dev.data_ptr(),
                                      Ln, _t4(k_new), _t4(v_new), _stream()))
    else:
        nh, nd = _int32_pair(new_lens, (B,), k_new.device)
        _check(library().ws_kv_append_varlen(ctypes.byref(desc), B, host.data_ptr(), dev.data_ptr(),
                                             nh.data_ptr(), nd.data_ptr(), Ln, _t4(k_new), _t4(v_new),
                                             _stream()))


def _int32_pair(x, shape, device):
    """(host, device) int32 tensors of the given shape from an array-like or
    a (host, device) pair."""
    if isinstance(x, tuple):
        host, dev = x
    else:
        host = torch.as_tensor(x, dtype=torch.int32).cpu().contiguous()
        dev = host.to(device)
    host = host.reshape(shape)
    dev = dev.reshape(shape)
    if host.dtype != torch.int32 or dev.dtype != torch.int32 or not host.is_contiguous() or not dev.is_contiguous():
        raise ValueError("int32 contiguous arrays expected")
    return host, dev


def block_causal_attn_fwd(q, k_new, v_new, cache, cache_lens, scale=None, fuse_append=False,
                          out=None, out_dtype=torch.bfloat16, want_lse=False, lse=None,
                          workspace=None, text_starts=None, new_lens=None):
    """One streaming step: q [B][Lq][Hq][d] of the new block attends to
    cache tokens [0, cache_lens[b]) and to its own block (k_new/v_new).
    text_starts (optional, [B]): the new block ends in a token-causal segment
    starting at that token of the block; new token t then sees new tokens
    [0, max(text_starts[b], t + 1)).
    new_lens (optional, [B], 1..Lq): stream b's block is its first
    new_lens[b] tokens; the rest is padding, never a key and never committed,
    and its rows' out and lse are unspecified.
    Returns out (and lse [B][Hq][Lq] f32 when want_lse)."""
    B, Lq, Hq, D = q.shape
    host, dev = _lens(cache_lens, q.device)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty((B, Lq, Hq, D), dtype=out_dtype, device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((B, Hq, Lq), dtype=torch.float32, device=q.device)
    _shape("k_new", k_new, (B, Lq, cache.num_kv_heads, D))
    _shape("v_new", v_new, (B, Lq, cache.num_kv_heads, D))
    _shape("out", out, (B, Lq, Hq, D))
    _shape("lse", lse, (B, Hq, Lq))
    if D != cache.head_dim:
        raise ValueError("q head_dim differs from the cache's")
    _check_lens(host, dev, B)
    _check_table(cache, B)
    nl = None if new_lens is None else _int32_pair(new_lens, (B,), q.device)
    if B == 0 or Lq == 0:
        need = 0
    elif nl is None:
        need = workspace_bytes(WS_OP_STEP, B, Hq, cache.num_kv_heads, Lq, int(host.max().item()) + Lq)
    else:
        need = step_workspace_bytes_varlen(B, Hq, cache.num_kv_heads, Lq, host, nl[0])
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_ptr = _ptr(workspace)
    ws_len = workspace.numel() if workspace is not None else 0
    desc = cache.desc()
    flags = WS_FUSE_APPEND if fuse_append else 0
    if nl is not None:
        th, td = _int32_pair(text_starts, (B,), q.device) if text_starts is not None else (None, None)
        _check(library().ws_block_causal_attn_fwd_varlen(
            _t4(q), _t4(k_new), _t4(v_new), ctypes.byref(desc), host.data_ptr(), dev.data_ptr(),
            nl[0].data_ptr(), nl[1].data_ptr(), _ptr(th), _ptr(td), B, Lq, Hq, float(scale), flags,
            _t4(out), _ptr(lse), ws_ptr, ws_len, _stream()))
    elif text_starts is None:
        _check(library().ws_block_causal_attn_fwd(
            _t4(q), _t4(k_new), _t4(v_new), ctypes.byref(desc), host.data_ptr(), dev.data_ptr(),
            B, Lq, Hq, float(scale), flags, _t4(out), _ptr(lse), ws_ptr, ws_len, _stream()))
    else:
        th, td = _int32_pair(text_starts, (B,), q.device)
        _check(library().ws_block_causal_attn_fwd_text(
            _t4(q), _t4(k_new), _t4(v_new), ctypes.byref(desc), host.data_ptr(), dev.data_ptr(),
            th.data_ptr(), td.data_ptr(), B, Lq, Hq, float(scale), flags, _t4(out), _ptr(lse),
            ws_ptr, ws_len, _stream()))
    return (out, lse) if want_lse else out


def block_causal_attn_fwd_noalloc(q, k_new, v_new, cache, cache_lens, out, lse=None, scale=None,
                                  fuse_append=False):
    """``block_causal_attn_fwd`` through the allocation-free entry point: the
    split partials live in the library's per-device scratch array, and this
    wrapper allocates nothing either, so every buffer comes from the caller:
    cache_lens is a (host, device) pair of int32 [B] tensors, out the
    [B][Lq][Hq][d] output (bf16 or f32), lse None or f32 [B][Hq][Lq].
    Calls on one device must be ordered (they share the scratch array)."""
    B, Lq, Hq, D = q.shape
    if not isinstance(cache_lens, tuple):
        raise ValueError("cache_lens must be a (host, device) pair of int32 tensors")
    host, dev = cache_lens
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    _shape("k_new", k_new, (B, Lq, cache.num_kv_heads, D))
    _shape("v_new", v_new, (B, Lq, cache.num_kv_heads, D))
    _shape("out", out, (B, Lq, Hq, D))
    _shape("lse", lse, (B, Hq, Lq))
    if D != cache.head_dim:
        raise ValueError("q head_dim differs from the cache's")
    _check_lens(host, dev, B)
    _check_table(cache, B)
    desc = cache.desc()
    _check(library().ws_block_causal_attn_fwd_noalloc(
        _t4(q), _t4(k_new), _t4(v_new), ctypes.byref(desc), host.data_ptr(), dev.data_ptr(),
        B, Lq, Hq, float(scale), WS_FUSE_APPEND if fuse_append else 0, _t4(out), _ptr(lse), _stream()))
    return out


def block_causal_prefill(q, k, v, block_offsets, scale=None, cache=None, num_kv_heads=None,
                         out=None, out_dtype=torch.bfloat16, want_lse=False, lse=None,
                         text_starts=None):
    """Whole-sequence block-causal attention.  q [B][L][Hq][d]; k, v
    [B][L][Hkv][d] or None to read them from ``cache``; block_offsets
    [B][nb+1] (host tensor, or a (host, device) pair).  text_starts
    (optional, [B][nb], absolute positions): block n ends in a token-causal
    segment starting there; its token i then sees keys
    j < max(text_starts[b][n], i + 1)."""
    B, L, Hq, D = q.shape
    if isinstance(block_offsets, tuple):
        off_h, off_d = block_offsets
    else:
        off_h = torch.as_tensor(block_offsets, dtype=torch.int32).cpu().contiguous()
        off_d = off_h.to(q.device)
    nb = off_h.shape[-1] - 1
    if k is not None:
        hkv = k.shape[2]
    else:
        hkv = num_kv_heads if num_kv_heads is not None else cache.num_kv_heads
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty((B, L, Hq, D), dtype=out_dtype, device=q.device)
    if want_lse and lse is None:
        lse = torch.empty((B, Hq, L), dtype=torch.float32, device=q.device)
    if k is not None or v is not None:
        _shape("k", k, (B, L, hkv, D))
        _shape("v", v, (B, L, hkv, D))
    else:
        _check_table(cache, B)
    _shape("out", out, (B, L, Hq, D))
    _shape("lse", lse, (B, Hq, L))
    if tuple(off_h.shape) != (B, nb + 1) or tuple(off_d.shape) != (B, nb + 1):
        raise ValueError("block_offsets must be [B][num_blocks + 1]")
    desc = cache.desc() if cache is not None else None
    kvp = ctypes.byref(desc) if desc is not None else None
    if text_starts is None:
        _check(library().ws_block_causal_prefill(
            _t4(q), _t4(k), _t4(v), kvp, off_h.data_ptr(), off_d.data_ptr(), B, L, nb, Hq, hkv, D,
            float(scale), _t4(out), _ptr(lse), _stream()))
    else:
        th, td = _int32_pair(text_starts, (B, nb), q.device)
        _check(library().ws_block_causal_prefill_text(
            _t4(q), _t4(k), _t4(v), kvp, off_h.data_ptr(), off_d.data_ptr(), th.data_ptr(), td.data_ptr(),
            B, L, nb, Hq, hkv, D, float(scale), _t4(out), _ptr(lse), _stream()))
    return (out, lse) if want_lse else out


def block_causal_prefill_bwd(q, k, v, o, dout, lse, block_offsets, scale=None, text_starts=None,
                             dq=None, dk=None, dv=None, workspace=None):
    """Gradients of ``block_causal_prefill`` (contiguous K/V) for an upstream
    output gradient dout: returns f32 (dq [B][L][Hq][d], dk, dv
    [B][L][Hkv][d]).  o and lse are the forward's output and lse;
    text_starts as in ``block_causal_prefill``."""
    B, L, Hq, D = q.shape
    hkv = k.shape[2]
    if isinstance(block_offsets, tuple):
        off_h, off_d = block_offsets
    else:
        off_h = torch.as_tensor(block_offsets, dtype=torch.int32).cpu().contiguous()
        off_d = off_h.to(q.device)
    nb = off_h.shape[-1] - 1
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    for name, t, shp in (("k", k, (B, L, hkv, D)), ("v", v, (B, L, hkv, D)), ("o", o, (B, L, Hq, D)),
                         ("dout", dout, (B, L, Hq, D)), ("lse", lse, (B, Hq, L))):
        _shape(name, t, shp)
    if tuple(off_h.shape) != (B, nb + 1) or tuple(off_d.shape) != (B, nb + 1):
        raise ValueError("block_offsets must be [B][num_blocks + 1]")
    if dq is None:
        dq = torch.empty((B, L, Hq, D), dtype=torch.float32, device=q.device)
    if dk is None:
        dk = torch.empty((B, L, hkv, D), dtype=torch.float32, device=q.device)
    if dv is None:
        dv = torch.empty((B, L, hkv, D), dtype=torch.float32, device=q.device)
    _shape("dq", dq, (B, L, Hq, D))
    _shape("dk", dk, (B, L, hkv, D))
    _shape("dv", dv, (B, L, hkv, D))
    need = workspace_bytes(WS_OP_PREFILL_BWD, B, Hq, hkv, L, L) if B > 0 and L > 0 else 0
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    th = td = None
    if text_starts is not None:
        th, td = _int32_pair(text_starts, (B, nb), q.device)
    _check(library().ws_block_causal_prefill_bwd(
        _t4(q), _t4(k), _t4(v), _t4(o), _t4(dout), _ptr(lse), off_h.data_ptr(), off_d.data_ptr(),
        _ptr(th), _ptr(td), B, L, nb, Hq, hkv, D, float(scale), _t4(dq), _t4(dk), _t4(dv),
        _ptr(workspace), workspace.numel() if workspace is not None else 0, _stream()))
    return dq, dk, dv
