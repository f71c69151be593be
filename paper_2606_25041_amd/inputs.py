"""Seeded synthetic inputs shaped like Wan-Streamer's streaming workloads.

Holds random draws, shapes and page permutations only -- none of the
attention arithmetic -- so the GPU path and the fp64 oracle can both be fed
from it without sharing any computation.

Streams of one seed (``np.random.default_rng([seed, k])``): k = 0 block
lengths, 1 page permutation, 2 Q, 3 K, 4 V.  Values are fp32 N(0, 1) rounded
to bf16 (round-to-nearest-even); a K scale is applied after rounding (exact
for powers of two).

The five named workloads are the interleaved-stream shapes of the paper
(Abstract and Sec. 3: streaming units of 160 ms = 4 frames at 25 fps mixing
visual, audio and text tokens; Sec. 2.4: a full-history cache grown by one
slice per unit).  The paper gives no token counts or model sizes; the sizes
below are the chosen synthetic stand-ins.
"""
import dataclasses
from typing import List, Optional

import numpy as np
import torch

PAGE = 64
S_LENGTHS, S_PAGES, S_Q, S_K, S_V = 0, 1, 2, 3, 4


def rng(seed, stream):
    return np.random.default_rng([seed, stream])


def bf16_normal(g, shape, scale=1.0):
    """fp32 N(0,1) draws rounded to bf16 (CPU tensor), times ``scale``."""
    t = torch.from_numpy(g.standard_normal(size=shape, dtype=np.float32)).to(torch.bfloat16)
    if scale != 1.0:
        t = t * scale
    return t


def bf16_bits(t):
    """uint16 numpy view of a bf16 CPU tensor (for the oracle)."""
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def interleaved_segments(g, nblocks):
    """Per-unit segment token counts of an interleaved stream, in block order
    [visual, audio, text]: a 4-frame visual segment of U{64..256} tokens in
    total, an audio segment of U{4..16} and a text segment of U{0..8}
    (inclusive bounds).  Returns (vis, aud, txt) int64 arrays."""
    vis = g.integers(64, 257, size=nblocks)
    aud = g.integers(4, 17, size=nblocks)
    txt = g.integers(0, 9, size=nblocks)
    return vis.astype(np.int64), aud.astype(np.int64), txt.astype(np.int64)


def interleaved_block_lengths(g, nblocks):
    """Per-unit token counts of an interleaved stream (sum of the segments of
    ``interleaved_segments``)."""
    vis, aud, txt = interleaved_segments(g, nblocks)
    return vis + aud + txt


def text_starts_of(offsets, text_lens):
    """Absolute start of each block's trailing text segment: [B][nb] from
    block offsets [B][nb+1] and per-block text lengths [B][nb]."""
    offsets = np.asarray(offsets, dtype=np.int64)
    return (offsets[:, 1:] - np.asarray(text_lens, dtype=np.int64)).astype(np.int32)


def interleaved_block_lengths_per_frame(g, nblocks):
    """Literal alternative: each of the 4 frames draws U{64..256} tokens."""
    vis = g.integers(64, 257, size=(nblocks, 4)).sum(axis=1)
    aud = g.integers(4, 17, size=nblocks)
    txt = g.integers(0, 9, size=nblocks)
    return (vis + aud + txt).astype(np.int64)


def page_table(g, batch, pages_per_seq, spare=2):
    """Seeded random physical order: one permutation of the whole pool;
    stream b owns the next pages_per_seq entries in logical order.  Returns
    (table [batch][pages_per_seq] int32, num_pages)."""
    num_pages = batch * pages_per_seq + spare
    perm = g.permutation(num_pages).astype(np.int32)
    return perm[: batch * pages_per_seq].reshape(batch, pages_per_seq).copy(), num_pages


@dataclasses.dataclass
class Workload:
    name: str
    kind: str                      # "prefill" or "step"
    B: int
    Hq: int
    Hkv: int
    D: int
    scale: float
    q: torch.Tensor                # bf16 CPU [B][Lq][Hq][D]
    k: torch.Tensor                # bf16 CPU logical keys  [B][Lk][Hkv][D]
    v: torch.Tensor                # bf16 CPU logical values
    Lq: int
    offsets: Optional[np.ndarray] = None     # prefill: [B][nb+1] int32
    cache_lens: Optional[np.ndarray] = None  # step: [B] int32 (cache tokens before the block)
    Lc_max: int = 0
    paged: bool = False
    page_table: Optional[np.ndarray] = None  # [B][max_pages] int32
    num_pages: int = 0
    out_f32: bool = False
    fuse_append: bool = False
    seed: int = 0
    # token-causal segments: prefill [B][nb] absolute starts; step [B]
    # starts within the new block (None: plain block-causal)
    text_starts: Optional[np.ndarray] = None
    # step: tokens of each stream's new block [B] (None: all Lq); the rest
    # of the Lq positions is padding
    new_lens: Optional[np.ndarray] = None

    # step views: the cache part and the new block of the logical K/V
    @property
    def k_cache(self):
        return self.k[:, : self.Lc_max]

    @property
    def v_cache(self):
        return self.v[:, : self.Lc_max]

    @property
    def k_new(self):
        return self.k[:, self.Lc_max:]

    @property
    def v_new(self):
        return self.v[:, self.Lc_max:]

    @property
    def num_blocks(self):
        return None if self.offsets is None else self.offsets.shape[1] - 1


def prefill_workload(name, B, Hq, Hkv, D, block_lens: List[np.ndarray], seed, paged=False,
                     k_scale=1.0, out_f32=False, spare_pages=2):
    """Whole-sequence workload; block_lens[b] are stream b's block lengths
    (every stream must total the same L)."""
    L = int(np.sum(block_lens[0]))
    offs = np.stack([np.concatenate([[0], np.cumsum(bl)]) for bl in block_lens]).astype(np.int32)
    assert np.all(offs[:, -1] == L), "streams must have equal total length"
    q = bf16_normal(rng(seed, S_Q), (B, L, Hq, D))
    k = bf16_normal(rng(seed, S_K), (B, L, Hkv, D), k_scale)
    v = bf16_normal(rng(seed, S_V), (B, L, Hkv, D))
    table, npages = (None, 0)
    if paged:
        table, npages = page_table(rng(seed, S_PAGES), B, max(1, -(-L // PAGE)), spare_pages)
    return Workload(name, "prefill", B, Hq, Hkv, D, 1.0 / np.sqrt(D), q, k, v, L, offsets=offs,
                    paged=paged, page_table=table, num_pages=npages, out_f32=out_f32, seed=seed)


def step_workload(name, B, Hq, Hkv, D, Lq, cache_lens, seed, fuse_append=False, spare_pages=2,
                  k_scale=1.0):
    """One streaming step of a new Lq-token block per stream; stream b has
    cache_lens[b] cached tokens (all earlier blocks)."""
    lens = np.asarray(cache_lens, dtype=np.int32).reshape(B)
    Lc = int(lens.max()) if B else 0
    q = bf16_normal(rng(seed, S_Q), (B, Lq, Hq, D))
    k = bf16_normal(rng(seed, S_K), (B, Lc + Lq, Hkv, D), k_scale)
    v = bf16_normal(rng(seed, S_V), (B, Lc + Lq, Hkv, D))
    # room for the committed block after the cache
    table, npages = page_table(rng(seed, S_PAGES), B, max(1, -(-(Lc + Lq) // PAGE)), spare_pages)
    return Workload(name, "step", B, Hq, Hkv, D, 1.0 / np.sqrt(D), q, k, v, Lq, cache_lens=lens,
                    Lc_max=Lc, paged=True, page_table=table, num_pages=npages,
                    fuse_append=fuse_append, seed=seed)


def config(idx, seed=None, c4_reading="B"):
    """The five named workloads; seed defaults to 1000 + idx."""
    seed = 1000 + idx if seed is None else seed
    if idx == 1:  # tiny: 4 blocks x 32 tokens, MHA 2 x 64, fp32 output
        return prefill_workload("tiny_b1_h2_d64_4x32", 1, 2, 2, 64, [np.full(4, 32)], seed,
                                out_f32=True)
    if idx == 2:  # one streaming step against a 4096-token cache
        return step_workload("step_b1_mha24_d128_q256_c4096", 1, 24, 24, 128, 256, [4096], seed)
    if idx == 3:  # whole-sequence prefill, 64 blocks of 256
        return prefill_workload("prefill_b2_gqa32x8_d128_64x256", 2, 32, 8, 128, [np.full(64, 256)] * 2,
                                seed, k_scale=0.5)
    if idx == 4:  # interleaved-modality variable blocks, paged
        g = rng(seed, S_LENGTHS)
        lens = (interleaved_block_lengths(g, 128) if c4_reading == "B"
                else interleaved_block_lengths_per_frame(g, 128))
        return prefill_workload(f"interleaved_b1_gqa40x8_d128_128blk_{int(lens.sum())}tok", 1, 40, 8, 128,
                                [lens], seed, paged=True)
    if idx == 5:  # 4 concurrent streams, 512-token block, 131072-token caches, fused append
        return step_workload("streams_b4_gqa64x8_d128_q512_c131072", 4, 64, 8, 128, 512, [131072] * 4,
                             seed, fuse_append=True)
    raise ValueError(f"no workload {idx}")


def thinker_prefill(seed=1006, nblocks=128):
    """The interleaved workload (1 stream, GQA 40/8 x 128, 128 variable
    blocks, paged) with each block's text segment token-causal: the
    thinker's pass over the language and state slots."""
    g = rng(seed, S_LENGTHS)
    vis, aud, txt = interleaved_segments(g, nblocks)
    wl = prefill_workload(f"thinker_prefill_b1_gqa40x8_d128_{nblocks}blk_{int((vis + aud + txt).sum())}tok",
                          1, 40, 8, 128, [vis + aud + txt], seed, paged=True)
    wl.text_starts = text_starts_of(wl.offsets, txt[None])
    return wl


def thinker_step(B=4, Hq=64, Hkv=8, Lq=8, Lc=131072, seed=1007):
    """A token-causal decode step of the thinker: B streams append Lq
    language/state tokens, all token-causal (segment start 0), to caches of
    Lc tokens (GQA Hq/Hkv x 128), committed in the same launch."""
    wl = step_workload(f"thinker_step_b{B}_gqa{Hq}x{Hkv}_d128_q{Lq}_c{Lc}", B, Hq, Hkv, 128, Lq,
                       [Lc] * B, seed, fuse_append=True)
    wl.text_starts = np.zeros(B, np.int32)
    return wl


def streams_varlen(B=4, Hq=64, Hkv=8, Lc=131072, seed=1008):
    """B concurrent streams, each ingesting its next interleaved unit (token
    counts from ``interleaved_segments``, the unit's text segment token-causal
    at its end) in one step, padded to the longest unit, over Lc cached
    tokens (GQA Hq/Hkv x 128), committed in the same launch."""
    vis, aud, txt = interleaved_segments(rng(seed, S_LENGTHS), B)
    lens = vis + aud + txt
    Lq = int(lens.max())
    wl = step_workload(f"streams_varlen_b{B}_gqa{Hq}x{Hkv}_d128_q{Lq}_c{Lc}", B, Hq, Hkv, 128, Lq, [Lc] * B,
                       seed, fuse_append=True)
    wl.new_lens = lens.astype(np.int32)
    wl.text_starts = (vis + aud).astype(np.int32)
    return wl


def sample_rows(g, B, Hq, L, n, must=()):
    """n distinct (b, h, i) rows (plus the given ones) for sampled checks."""
    rows = {tuple(int(x) for x in r) for r in must}
    while len(rows) < n + len(must):
        rows.add((int(g.integers(B)), int(g.integers(Hq)), int(g.integers(L))))
    return np.array(sorted(rows), dtype=np.int32)
