"""C-ABI checks that need no GPU: the library loads, exports every function
include/ws_attn.h declares, and rejects bad arguments with the documented
status before touching any device memory (all "device" pointers below are
fake and never dereferenced, because validation fails first)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import paper_2606_25041_amd as ws
from paper_2606_25041_amd import build as wsbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ws_attn.h")
FAKE = 0x10000  # 16-byte aligned, never dereferenced


# Every call below must fail validation: the pointers are fake, so a call
# that passed would launch a kernel on them.  Never run this module where a
# GPU is visible.
if torch.cuda.device_count() > 0:
    pytest.skip("uses fake device pointers; CPU-only module", allow_module_level=True)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(wsbuild.LIB):
        wsbuild.build()
    return ws.library()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ws_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert {"ws_kv_append", "ws_block_causal_attn_fwd", "ws_block_causal_prefill",
            "ws_block_causal_attn_fwd_text", "ws_block_causal_prefill_text", "ws_block_causal_prefill_bwd",
            "ws_block_causal_attn_fwd_varlen", "ws_kv_append_varlen", "ws_step_workspace_bytes_varlen",
            "ws_workspace_bytes", "ws_step_plan", "ws_block_causal_attn_fwd_noalloc", "ws_abi_version",
            "ws_status_string",
            "ws_last_error"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    assert lib.ws_abi_version() == 5
    assert lib.ws_status_string(0) == b"WS_OK"
    assert lib.ws_status_string(10) == b"WS_ERR_HIP"


def test_ceilings_library_exports_every_declared_symbol():
    """libwsceil.so (the benchmark's MFMA and HBM-read ceilings) loads and
    exports what include/ws_ceilings.h declares."""
    if not os.path.exists(wsbuild.CEIL_LIB):
        wsbuild.build_ceilings()
    lib = ctypes.CDLL(wsbuild.CEIL_LIB)
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "ws_ceilings.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(wsc_[a-z0-9_]+)\s*\(", text)))
    assert names == ["wsc_mfma_loop", "wsc_stream_read"]
    for name in names:
        assert hasattr(lib, name), name
    # argument checks fail before anything is launched
    lib.wsc_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_void_p]
    lib.wsc_mfma_loop.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
    assert lib.wsc_stream_read(FAKE, 17, FAKE, 1, None) != 0
    assert lib.wsc_mfma_loop(None, 1, 1, 2, None) != 0
    assert lib.wsc_mfma_loop(FAKE, 1, 1, 0, None) != 0
    assert lib.wsc_mfma_loop(FAKE, 1, 1, 5, None) != 0


def t4(ptr=FAKE, dtype=ws.WS_DTYPE_BF16, sb=0, st=0, sh=0, d=128, L=16, H=4):
    if sb == 0 and st == 0 and sh == 0:
        sh, st, sb = d, H * d, L * H * d
    return ws.Tensor4(ptr, dtype, sb, st, sh)


class Host:
    """Host arrays the library validates (kept alive by this object)."""

    def __init__(self, B=2, max_pages=4, num_pages=10, lens=(10, 100)):
        self.table = np.arange(B * max_pages, dtype=np.int32).reshape(B, max_pages) % num_pages
        self.lens = np.array(lens, dtype=np.int32)
        self.num_pages, self.max_pages = num_pages, max_pages

    def desc(self, **kw):
        d = dict(k_pool=FAKE, v_pool=FAKE, page_table_dev=FAKE,
                 page_table_host=self.table.ctypes.data, num_pages=self.num_pages,
                 page_size=64, max_pages_per_seq=self.max_pages, num_kv_heads=2, head_dim=128)
        d.update(kw)
        return ws.PagedKVDesc(**d)


def step_call(lib, h, desc=None, q=None, kn=None, vn=None, out=None, B=2, Lq=16, Hq=4,
              scale=0.088, flags=0, lse=None, wsp=FAKE, wsb=1 << 30, lens_ptr="host"):
    desc = desc or h.desc()
    q = q or t4(H=Hq, L=Lq)
    kn = kn or t4(H=2, L=Lq)
    vn = vn or t4(H=2, L=Lq)
    out = out or t4(H=Hq, L=Lq)
    lh = h.lens.ctypes.data if lens_ptr == "host" else lens_ptr
    return lib.ws_block_causal_attn_fwd(q, kn, vn, ctypes.byref(desc), lh, FAKE, B, Lq, Hq,
                                        scale, flags, out, lse, wsp, wsb, None)


def test_step_errors(lib):
    h = Host()
    assert step_call(lib, h, q=t4(ptr=None)) == 1                      # NULL q
    assert step_call(lib, h, lens_ptr=None) == 1                       # NULL cache_lens
    assert step_call(lib, h, desc=h.desc(k_pool=None)) == 1            # NULL pool
    assert step_call(lib, h, desc=h.desc(page_table_host=None)) == 1   # NULL host table
    assert step_call(lib, h, B=-1) == 2                                # negative batch
    assert step_call(lib, h, Hq=0) == 2
    assert step_call(lib, h, desc=h.desc(head_dim=96)) == 3            # head_dim
    assert step_call(lib, h, desc=h.desc(page_size=32)) == 3           # page size
    assert step_call(lib, h, q=t4(dtype=ws.WS_DTYPE_F32)) == 3         # f32 input
    assert step_call(lib, h, flags=4) == 3                             # unknown flag
    assert step_call(lib, h, scale=0.0) == 3
    assert step_call(lib, h, scale=float("nan")) == 3
    assert step_call(lib, h, q=t4(ptr=FAKE + 2)) == 4                  # misaligned pointer
    assert step_call(lib, h, q=t4(sb=16 * 4 * 128, st=4 * 128, sh=130)) == 4  # stride % 8
    assert step_call(lib, h, lse=FAKE + 2) == 4
    big = 1 << 24                                                      # K/V token stride limit
    assert step_call(lib, h, kn=t4(H=2, sb=big, st=big, sh=128)) == 2
    assert step_call(lib, h, vn=t4(H=2, sb=big, st=big, sh=128)) == 2
    # just below the limit passes the stride check and fails a later one
    assert step_call(lib, h, kn=t4(H=2, sb=big, st=big - 8, sh=128), lse=FAKE + 2) == 4
    assert step_call(lib, h, Hq=3, q=t4(H=3), out=t4(H=3)) == 8        # Hq % Hkv
    h2 = Host(lens=(10, 300))                                          # 300 > 4 pages * 64
    assert step_call(lib, h2) == 7
    h4 = Host()
    h4.table[1, 1] = 99                                                # page id out of range
    assert step_call(lib, h4) == 6
    h5 = Host(lens=(10, -1))
    assert step_call(lib, h5) == 2
    # A call that passes every argument check plans for the device's compute
    # units next; with no device here that query fails (the workspace checks
    # that follow run in the GPU tests).
    hw = Host(lens=(10, 200))            # 216 keys: the plan splits the KV range
    assert plan(lib, 256, 2, 4, 2, 16, [10, 200])[1] > 0
    assert step_call(lib, hw, wsp=None) == 10
    assert b"compute units" in lib.ws_last_error()


def test_step_noalloc_validates_like_the_workspace_entry_point(lib):
    h = Host()

    def call(q=None, B=2, Lq=16, Hq=4, flags=0, lse=None, lens_ptr="host"):
        desc = h.desc()
        lh = h.lens.ctypes.data if lens_ptr == "host" else lens_ptr
        return lib.ws_block_causal_attn_fwd_noalloc(q or t4(H=Hq, L=Lq), t4(H=2, L=Lq), t4(H=2, L=Lq),
                                                    ctypes.byref(desc), lh, FAKE, B, Lq, Hq, 0.088, flags,
                                                    t4(H=Hq, L=Lq), lse, None)
    assert call(q=t4(ptr=None)) == 1
    assert call(lens_ptr=None) == 1
    assert call(B=-1) == 2
    assert call(flags=4) == 3
    assert call(lse=FAKE + 2) == 4
    assert call(Hq=3) == 8
    assert call(B=0) == 0                      # nothing to do
    # valid arguments reach the device plan (no device here)
    assert call() == 10


def test_step_capacity_counts_fused_append(lib):
    # cache of 250 tokens fits 4 pages, but committing 16 more does not
    h = Host(lens=(10, 250))
    assert step_call(lib, h, flags=ws.WS_FUSE_APPEND) == 7
    h.table[1, 3] = -5  # the 4th page is only read for the append
    assert step_call(lib, h, flags=ws.WS_FUSE_APPEND) in (6, 7)


def append_call(lib, h, desc=None, B=2, Ln=16, kn=None, vn=None, lens_ptr="host"):
    desc = desc or h.desc()
    lh = h.lens.ctypes.data if lens_ptr == "host" else lens_ptr
    return lib.ws_kv_append(ctypes.byref(desc), B, lh, FAKE, Ln, kn or t4(H=2, L=Ln),
                            vn or t4(H=2, L=Ln), None)


def test_append_errors(lib):
    h = Host()
    assert append_call(lib, h, lens_ptr=None) == 1
    assert append_call(lib, h, kn=t4(ptr=None)) == 1
    assert append_call(lib, h, B=-2) == 2
    assert append_call(lib, h, Ln=-1) == 2
    assert append_call(lib, h, desc=h.desc(head_dim=32)) == 3
    assert append_call(lib, h, kn=t4(ptr=FAKE + 8)) == 4
    assert append_call(lib, h, Ln=200) == 7          # 100 + 200 > 256
    h.table[0, 0] = 10                               # == num_pages
    assert append_call(lib, h) == 6


def prefill_call(lib, offs, B=1, L=None, nb=None, Hq=4, Hkv=2, d=128, q=None, k=None, v=None,
                 out=None, desc=None, scale=0.1):
    offs = np.ascontiguousarray(np.asarray(offs, np.int32))
    L = int(offs.reshape(B, -1)[0, -1]) if L is None else L
    nb = offs.reshape(B, -1).shape[1] - 1 if nb is None else nb
    q = q or t4(H=Hq, L=L, d=d)
    k = k if k is not None else t4(H=Hkv, L=L, d=d)
    v = v if v is not None else t4(H=Hkv, L=L, d=d)
    out = out or t4(H=Hq, L=L, d=d)
    return lib.ws_block_causal_prefill(q, k, v, ctypes.byref(desc) if desc else None,
                                       offs.ctypes.data, FAKE, B, L, nb, Hq, Hkv, d, scale, out,
                                       None, None)


def test_prefill_errors(lib):
    assert prefill_call(lib, [[1, 5, 9]]) == 5                    # first offset != 0
    assert prefill_call(lib, [[0, 6, 5, 9]]) == 5                 # decreasing
    assert prefill_call(lib, [[0, 5, 9]], L=10) == 5              # last != seq_len
    assert prefill_call(lib, [[0, 4, 8], [0, 2, 7]], B=2, L=8) == 5
    assert prefill_call(lib, [[0, 8]], Hq=6, Hkv=4) == 8
    assert prefill_call(lib, [[0, 8]], d=80) == 3
    assert prefill_call(lib, [[0, 8]], q=t4(ptr=None)) == 1
    null = ws.Tensor4(None, 1, 0, 0, 0)
    assert prefill_call(lib, [[0, 8]], k=null, v=null) == 1       # paged without a cache
    assert prefill_call(lib, [[0, 8]], Hq=0) == 2
    big = 1 << 24
    assert prefill_call(lib, [[0, 8]], k=t4(H=2, L=8, sb=big, st=big, sh=128)) == 2
    assert prefill_call(lib, [[0, 8]], v=t4(H=2, L=8, sb=big, st=big, sh=128)) == 2
    h = Host(B=1, lens=(0,))
    assert prefill_call(lib, [[0, 300]], k=null, v=null, desc=h.desc()) == 7
    h.table[0, 2] = 77
    assert prefill_call(lib, [[0, 150]], k=null, v=null, desc=h.desc()) == 6
    assert prefill_call(lib, [[0, 150]], k=null, v=null, desc=h.desc(num_kv_heads=4)) == 8


def step_text_call(lib, h, starts, B=2, Lq=16, Hq=4, lse=None, starts_dev=FAKE):
    desc = h.desc()
    st = np.ascontiguousarray(np.asarray(starts, np.int32)) if starts is not None else None
    return lib.ws_block_causal_attn_fwd_text(t4(H=Hq, L=Lq), t4(H=2, L=Lq), t4(H=2, L=Lq), ctypes.byref(desc),
                                             h.lens.ctypes.data, FAKE,
                                             st.ctypes.data if st is not None else None, starts_dev,
                                             B, Lq, Hq, 0.088, 0, t4(H=Hq, L=Lq), lse, FAKE, 1 << 30, None)


def test_step_text_errors(lib):
    h = Host()
    assert step_text_call(lib, h, None) == 1                  # NULL host starts
    assert step_text_call(lib, h, [0, 3], starts_dev=None) == 1
    assert step_text_call(lib, h, [0, 17]) == 5               # start past new_len (16)
    assert step_text_call(lib, h, [-1, 3]) == 5
    # valid starts (0 and new_len) pass to the next check: a misaligned lse
    assert step_text_call(lib, h, [0, 16], lse=FAKE + 2) == 4


def step_varlen_call(lib, h, new_lens, starts=None, B=2, Lq=16, Hq=4, flags=0, lse=None, wsb=1 << 30,
                     nl_dev=FAKE, starts_dev=FAKE):
    desc = h.desc()
    nl = np.ascontiguousarray(np.asarray(new_lens, np.int32)) if new_lens is not None else None
    st = np.ascontiguousarray(np.asarray(starts, np.int32)) if starts is not None else None
    return lib.ws_block_causal_attn_fwd_varlen(
        t4(H=Hq, L=Lq), t4(H=2, L=Lq), t4(H=2, L=Lq), ctypes.byref(desc), h.lens.ctypes.data, FAKE,
        nl.ctypes.data if nl is not None else None, nl_dev,
        st.ctypes.data if st is not None else None, starts_dev if st is not None else None,
        B, Lq, Hq, 0.088, flags, t4(H=Hq, L=Lq), lse, FAKE, wsb, None)


def test_step_varlen_errors(lib):
    h = Host()
    assert step_varlen_call(lib, h, None) == 1                  # NULL host lengths
    assert step_varlen_call(lib, h, [16, 3], nl_dev=None) == 1
    assert step_varlen_call(lib, h, [16, 0]) == 2               # an empty block
    assert step_varlen_call(lib, h, [17, 3]) == 2               # longer than new_len
    assert step_varlen_call(lib, h, [16, 3], starts=[0, 17]) == 5
    # valid lengths (1 and new_len) pass to the next check: a misaligned lse
    assert step_varlen_call(lib, h, [16, 1], starts=[0, 16], lse=FAKE + 2) == 4
    assert step_varlen_call(lib, h, [16, 1], lse=FAKE + 2) == 4
    # host starts without device starts
    desc = h.desc()
    nl = np.array([16, 3], np.int32)
    st = np.array([0, 3], np.int32)
    assert lib.ws_block_causal_attn_fwd_varlen(
        t4(), t4(H=2), t4(H=2), ctypes.byref(desc), h.lens.ctypes.data, FAKE, nl.ctypes.data, FAKE,
        st.ctypes.data, None, 2, 16, 4, 0.088, 0, t4(), None, FAKE, 1 << 30, None) == 1


def test_step_varlen_capacity_counts_real_tokens(lib):
    # 4 pages hold 256 tokens: stream 1 (250 cached) can commit 6 new tokens, not 7
    h = Host(lens=(10, 250))
    assert step_varlen_call(lib, h, [16, 7], flags=ws.WS_FUSE_APPEND) == 7
    # 6 fits and passes every argument check (it then plans for the device)
    assert step_varlen_call(lib, h, [16, 6], flags=ws.WS_FUSE_APPEND, wsb=16) == 10


def plan(lib, cus, B, hq, hkv, lq, lens, nls=None):
    """(status, workspace bytes, splits) from ws_step_plan."""
    ch = np.ascontiguousarray(np.asarray(lens, np.int32))
    nh = None if nls is None else np.ascontiguousarray(np.asarray(nls, np.int32))
    ns, nbytes = ctypes.c_int32(-1), ctypes.c_size_t(0)
    rc = lib.ws_step_plan(cus, B, hq, hkv, lq, ch.ctypes.data, None if nh is None else nh.ctypes.data,
                          ctypes.byref(ns), ctypes.byref(nbytes))
    return rc, nbytes.value, ns.value


def test_step_plan_workspace_and_errors(lib):
    lens = [131072] * 4
    ws_of = lambda *a, **k: plan(lib, 256, *a, **k)[1]
    # equal lengths given as lengths: the plain step's plan
    for lq, c in ((512, 131072), (243, 131072), (8, 131072), (256, 4096)):
        assert ws_of(4, 64, 8, lq, [c] * 4, [lq] * 4) == ws_of(4, 64, 8, lq, [c] * 4)
    # four long streams padded to 243 tokens fill the CUs exactly (no split,
    # no workspace); with their real lengths 72 of the 256 work-groups hold
    # padding only, and the KV range is split instead
    assert ws_of(4, 64, 8, 243, lens, [243] * 4) == 0
    assert ws_of(4, 64, 8, 243, lens, [145, 110, 163, 243]) > 0
    # a batch of 3 long 512-token blocks (384 work-groups: 1.5 rounds) splits too
    assert ws_of(3, 64, 8, 512, lens[:3]) > 0
    assert ws_of(4, 64, 8, 512, lens) == 0
    # invalid arguments
    assert plan(lib, 256, 4, 64, 8, 243, lens, [145, 0, 163, 243])[0] == 2
    assert plan(lib, 256, 4, 64, 8, 243, lens, [145, 244, 163, 243])[0] == 2
    assert plan(lib, 256, 4, 64, 8, 243, [131072, -1, 5, 5], [145, 110, 163, 243])[0] == 2
    assert plan(lib, 256, 4, 64, 7, 243, lens)[0] == 8
    assert plan(lib, -1, 4, 64, 8, 243, lens)[0] == 2
    ns, nb = ctypes.c_int32(0), ctypes.c_size_t(0)
    assert lib.ws_step_plan(256, 4, 64, 8, 243, None, None, ctypes.byref(ns), ctypes.byref(nb)) == 1
    # no device here: planning for "the current device" fails, and the
    # device-planned workspace queries return 0
    assert plan(lib, 0, 1, 24, 24, 256, [4096])[0] == 10
    assert lib.ws_workspace_bytes(ws.WS_OP_STEP, 1, 24, 24, 256, 4352) == 0
    ch = np.array([4096], np.int32)
    nh = np.array([256], np.int32)
    assert lib.ws_step_workspace_bytes_varlen(1, 24, 24, 256, ch.ctypes.data, nh.ctypes.data) == 0


def append_varlen_call(lib, h, new_lens, Ln=16, nl_dev=FAKE, kn=None):
    desc = h.desc()
    nl = np.ascontiguousarray(np.asarray(new_lens, np.int32)) if new_lens is not None else None
    return lib.ws_kv_append_varlen(ctypes.byref(desc), 2, h.lens.ctypes.data, FAKE,
                                   nl.ctypes.data if nl is not None else None, nl_dev, Ln,
                                   kn or t4(H=2, L=Ln), t4(H=2, L=Ln), None)


def test_append_varlen_errors(lib):
    h = Host(lens=(10, 250))
    assert append_varlen_call(lib, h, None) == 1
    assert append_varlen_call(lib, h, [1, 2], nl_dev=None) == 1
    assert append_varlen_call(lib, h, [-1, 2]) == 2
    assert append_varlen_call(lib, h, [17, 2]) == 2
    assert append_varlen_call(lib, h, [16, 7]) == 7              # 250 + 7 > 256
    assert append_varlen_call(lib, h, [16, 6], kn=t4(ptr=FAKE + 8)) == 4


def prefill_text_call(lib, offs, starts, B=1, starts_dev=FAKE, lse=None):
    offs = np.ascontiguousarray(np.asarray(offs, np.int32))
    L = int(offs.reshape(B, -1)[0, -1])
    nb = offs.reshape(B, -1).shape[1] - 1
    st = np.ascontiguousarray(np.asarray(starts, np.int32)) if starts is not None else None
    return lib.ws_block_causal_prefill_text(t4(H=4, L=L), t4(H=2, L=L), t4(H=2, L=L), None,
                                            offs.ctypes.data, FAKE, st.ctypes.data if st is not None else None,
                                            starts_dev, B, L, nb, 4, 2, 128, 0.1, t4(H=4, L=L), lse, None)


def test_prefill_text_errors(lib):
    assert prefill_text_call(lib, [[0, 5, 9]], None) == 1
    assert prefill_text_call(lib, [[0, 5, 9]], [[0, 5]], starts_dev=None) == 1
    assert prefill_text_call(lib, [[0, 5, 9]], [[6, 7]]) == 5     # start past its block's end
    assert prefill_text_call(lib, [[0, 5, 9]], [[0, 4]]) == 5     # start before its block
    assert prefill_text_call(lib, [[0, 5, 5, 9]], [[2, 6, 9]]) == 5   # empty block: start must be 5
    assert prefill_text_call(lib, [[0, 4, 8], [0, 2, 8]], [[1, 8], [2, 9]], B=2) == 5
    # starts at the block bounds are valid: the call reaches a later check
    assert prefill_text_call(lib, [[0, 5, 5, 9]], [[5, 5, 5]], lse=FAKE + 2) == 4
    assert prefill_text_call(lib, [[0, 5, 9]], [[0, 9]], lse=FAKE + 2) == 4


def bwd_call(lib, offs, B=1, Hq=4, Hkv=2, d=128, lse=FAKE, wsp=FAKE, wsb=1 << 30, dq_dtype=ws.WS_DTYPE_F32,
             text=None, text_dev=None):
    offs = np.ascontiguousarray(np.asarray(offs, np.int32))
    L = int(offs.reshape(B, -1)[0, -1])
    nb = offs.reshape(B, -1).shape[1] - 1
    f32 = lambda H: t4(dtype=dq_dtype, H=H, L=L, d=d, sh=d, st=H * d, sb=L * H * d)
    tx = np.ascontiguousarray(np.asarray(text, np.int32)) if text is not None else None
    return lib.ws_block_causal_prefill_bwd(t4(H=Hq, L=L, d=d), t4(H=Hkv, L=L, d=d), t4(H=Hkv, L=L, d=d),
                                           t4(H=Hq, L=L, d=d), t4(H=Hq, L=L, d=d), lse, offs.ctypes.data, FAKE,
                                           tx.ctypes.data if tx is not None else None, text_dev, B, L, nb, Hq, Hkv,
                                           d, 0.1, f32(Hq), f32(Hkv), f32(Hkv), wsp, wsb, None)


def test_bwd_errors(lib):
    assert bwd_call(lib, [[0, 5, 9]], lse=None) == 1
    assert bwd_call(lib, [[0, 5, 9]], text=[[0, 5]]) == 1          # host starts without device copy
    assert bwd_call(lib, [[0, 5, 9]], dq_dtype=ws.WS_DTYPE_BF16) == 3
    assert bwd_call(lib, [[0, 5, 9]], d=96) == 3
    assert bwd_call(lib, [[0, 5, 9]], Hq=3) == 8
    assert bwd_call(lib, [[1, 5, 9]]) == 5
    assert bwd_call(lib, [[0, 5, 9]], text=[[6, 7]], text_dev=FAKE) == 5
    assert bwd_call(lib, [[0, 5, 9]], wsp=None) == 9
    assert bwd_call(lib, [[0, 5, 9]], wsb=16) == 9
    assert bwd_call(lib, [[0, 5, 9]], lse=FAKE + 2) == 4
    n = lib.ws_workspace_bytes(ws.WS_OP_PREFILL_BWD, 2, 32, 8, 16384, 16384)
    assert n == 2 * 32 * 16384 * 8 + 2 * 16384 * 4


def test_empty_calls_are_ok(lib):
    h = Host(B=0, lens=())
    assert step_call(lib, h, B=0) == 0
    assert prefill_call(lib, [[0]], L=0, nb=0) == 0
    assert prefill_call(lib, np.zeros((0, 3), np.int32), B=0, L=5, nb=2) == 0


def test_workspace_bytes(lib):
    # a single 256-row tile per head needs KV splits (and partials) to fill the chip
    n = plan(lib, 256, 1, 24, 24, 256, [4096])[1]
    assert n > 0 and n % (24 * 256 * 130 * 4) == 0
    # enough work items already: no splits, no workspace
    assert plan(lib, 256, 4, 64, 8, 512, [131072] * 4)[1] == 0
    # a 16-token block of 8 query heads per KV head packs into one 128-row
    # tile per (stream, KV head): 32 tiles, so the long cache is split
    n16 = plan(lib, 256, 4, 64, 8, 16, [131072] * 4)[1]
    assert n16 > 0 and n16 % (4 * 8 * 128 * 130 * 4) == 0
    # on a partition of 32 compute units the 24 tiles of the headline step
    # need fewer splits
    assert 1 < plan(lib, 32, 1, 24, 24, 256, [4096])[2] < plan(lib, 256, 1, 24, 24, 256, [4096])[2]
    # 256 query tiles fill exactly one round of 256 CUs: one split (the GPU
    # test of a split longer than the staged page ids relies on it)
    assert plan(lib, 256, 1, 8, 1, 8192, [170000])[2] == 1
    assert lib.ws_workspace_bytes(ws.WS_OP_PREFILL, 2, 32, 8, 16384, 16384) == 0
    assert lib.ws_workspace_bytes(ws.WS_OP_STEP, 0, 24, 24, 256, 4352) == 0
    assert lib.ws_workspace_bytes(ws.WS_OP_STEP, 1, 24, 5, 256, 4352) == 0   # 24 % 5 != 0
    assert lib.ws_workspace_bytes(ws.WS_OP_STEP, 1, 24, 0, 256, 4352) == 0


def _split_model(B, hq, hkv, lq, lens, nls, slots=256):
    """The documented split rule, written out by brute force: the default
    (the largest split count whose work-groups fit one round of the CUs), and
    rounds(s) x (ceil(tiles / s) + 4) counted per XCD over the real items of
    the launch order (groups KV-head-major for blocks of different lengths),
    the fewest splits within 2 % of its minimum taking over when that is
    more than 10 % cheaper than the default.  Returns the split count."""
    qt, xcds, fixed = 256, 8, 4
    G = hq // hkv
    nqt = -(-G * lq // qt)
    real = [-(-G * n // qt) for n in nls] if nls is not None else [nqt] * B
    base = hkv * sum(real)
    ntiles = -(-max(c + (n if nls is not None else lq) for c, n in zip(lens, nls or [lq] * B)) // 64)
    cap = max(1, min(ntiles // 2, 32))

    def cost(s):
        per_split = -(-ntiles // s) + fixed
        if nls is None:
            return -(-base * s // slots) * per_split
        P = nqt * s
        n_work = B * hkv * P
        per = -(-n_work // xcds)
        cnt = [0] * xcds
        for g in range(B * hkv):
            lo, hi = g * P, g * P + real[g % B] * s
            for x in range(xcds):
                cnt[x] += max(0, min(hi, (x + 1) * per) - max(lo, x * per))
        return max(-(-c // max(1, slots // xcds)) for c in cnt) * per_split

    ns = min(slots // base if base < slots else 1, cap)
    lo = min(cost(s) for s in range(1, cap + 1))
    best = 1
    while 50 * cost(best) > 51 * lo:
        best += 1
    return best if 10 * cost(best) < 9 * cost(ns) else ns


@pytest.mark.parametrize("cus", [256, 32])
def test_split_planner_matches_its_rule(lib, cus):
    """The library's split count and workspace equal the rule computed by
    brute force, for equal and for different new-block lengths, on random
    shapes, for the full chip (256 compute units) and a 32-unit partition."""
    rng = np.random.default_rng(17)
    for _ in range(150):
        hkv = int(rng.choice([1, 2, 4, 8, 16]))
        G = int(rng.choice([1, 2, 4, 8]))
        B = int(rng.integers(1, 9))
        lq = int(rng.integers(1, 600))
        lens = [int(rng.choice([0, 100, 4096, 30000, 131072])) for _ in range(B)]
        nls = [int(x) for x in rng.integers(1, lq + 1, size=B)]
        rows = -(-G * lq // 32) * 32
        unit = B * hkv * rows * 130 * 4
        for var in (False, True):
            rc, got, ns_lib = plan(lib, cus, B, hkv * G, hkv, lq, lens, nls if var else None)
            assert rc == 0
            ns = _split_model(B, hkv * G, hkv, lq, lens, nls if var else None, slots=cus)
            assert ns_lib == ns, (cus, B, hkv * G, hkv, lq, lens, nls, var, ns, ns_lib)
            assert got == (0 if ns == 1 else ns * unit), (B, hkv * G, hkv, lq, lens, nls, var, ns, got)
