"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle,
element by element on seeded inputs.  Small cases span several 64-key tiles,
several query tiles and ragged tails; the five named workloads run at full
size and are checked on sampled rows that the loop oracle computes one by
one (one in every 32-row block of every work item) and, for the larger ones,
on every output against the block-wise fp64 oracle.
Tolerance: max-abs 2e-2, mean-abs 2e-3 (bf16 outputs), lse 1e-3."""
import numpy as np
import pytest
import torch

import paper_2606_25041_amd as ws
from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu


def _prefill_case(name, B, Hq, Hkv, D, L, nb, seed, paged=False, out_f32=False):
    g = np.random.default_rng([seed, 99])
    lens = []
    for _ in range(B):
        cuts = np.sort(g.choice(np.arange(1, L), size=nb - 1, replace=False))
        lens.append(np.diff(np.concatenate([[0], cuts, [L]])))
    return inputs.prefill_workload(name, B, Hq, Hkv, D, lens, seed, paged=paged, out_f32=out_f32)


def _check_full(wl, cache=None, **kw):
    gs.say(f"[gpu] {wl.name}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Lq={wl.Lq}")
    out, lse = gs.run_gpu(wl, cache=cache, **kw)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl)
    stats = gs.compare(out, lse, ref, ref_lse)
    gs.assert_close(stats)
    return out, lse, stats


def test_tiny_config_full():
    wl = inputs.config(1)
    out, _, stats = _check_full(wl)
    assert out.dtype == torch.float32


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("L,nb", [(777, 9), (100, 3), (1300, 40)])
def test_prefill_contiguous_ragged(D, L, nb):
    wl = _prefill_case(f"prefill_c_d{D}_L{L}", 2, 4, 2, D, L, nb, seed=7 + L + D)
    _check_full(wl)


def test_prefill_unit_and_empty_blocks():
    # blocks of length 1 (token-causal stretch), empty blocks, one long block
    lens = [np.array([1, 1, 1, 0, 5, 0, 1, 200, 1, 1, 0, 90])]
    wl = inputs.prefill_workload("prefill_unit_empty", 1, 2, 1, 128, lens, 31)
    _check_full(wl)


def test_prefill_single_block_and_f32_out():
    wl = inputs.prefill_workload("prefill_single_block", 1, 2, 2, 128, [np.array([700])], 32,
                                 out_f32=True)
    _check_full(wl)


def test_prefill_paged_interleaved():
    g = inputs.rng(41, inputs.S_LENGTHS)
    lens = inputs.interleaved_block_lengths(g, 10)
    wl = inputs.prefill_workload("prefill_paged_interleaved", 1, 5, 1, 128, [lens], 41, paged=True)
    cache = gs.device_cache(wl, [wl.Lq])
    _check_full(wl, cache=cache)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("Lq,lens", [(100, [0, 333, 64]), (1, [5, 700, 64]), (300, [129, 0, 1000])])
def test_step_ragged(D, Lq, lens):
    wl = inputs.step_workload(f"step_d{D}_q{Lq}", 3, 8, 2, D, Lq, lens, seed=11 + Lq + D)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache=cache)


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("Lq", [1, 16, 37])
def test_step_small_block_gqa8(Lq, out_dtype):
    """Small blocks of a GQA-8 model: the 8 query heads of a KV head share one
    packed query tile (8 x Lq rows), and the long caches are split."""
    wl = inputs.step_workload(f"step_gqa8_q{Lq}", 2, 16, 2, 128, Lq, [4100, 2500], seed=23 + Lq)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache=cache, out_dtype=out_dtype)


def test_step_many_streams_lengths_from_memory():
    """More streams than the cache lengths passed by value (32): the kernel
    reads them from the device array; ragged lengths, GQA 2, d = 64."""
    g = np.random.default_rng(31)
    lens = [int(x) for x in g.integers(0, 700, size=40)]
    wl = inputs.step_workload("step_b40", 40, 2, 1, 64, 8, lens, seed=31)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache=cache)


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_step_most_splits(out_dtype):
    """One head, a 16-token block and an 8192-token cache: the plan uses the
    largest split count (32), so the merge sees every split slot."""
    wl = inputs.step_workload("step_s32", 1, 1, 1, 128, 16, [8192], seed=37)
    cache = gs.device_cache(wl, wl.cache_lens)
    assert ws.workspace_bytes(ws.WS_OP_STEP, 1, 1, 1, 16, 8192 + 16) == 32 * 1 * 32 * 130 * 4
    _check_full(wl, cache=cache, out_dtype=out_dtype)


def test_step_one_token_empty_cache():
    """The smallest step: one new token, nothing cached (it sees itself)."""
    wl = inputs.step_workload("step_min", 2, 4, 2, 128, 1, [0, 0], seed=41)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache=cache)


def test_step_mha_f32_out():
    wl = inputs.step_workload("step_mha_f32", 1, 6, 6, 128, 256, [1000], seed=13)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_full(wl, cache=cache, out_dtype=torch.float32)


# ---------------------------------------------------------------------------
# the five named workloads at full size

def _covered(wl, cache, rows):
    """Full-size run against the oracle on the given rows (computed one by
    one by the oracle); every output must be finite (NaN-filled unused pool
    pages never leak)."""
    gs.say(f"[gpu] {wl.name}: full size, {len(rows)} rows")
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl, rows=rows)
    stats = gs.compare(out, lse, ref, ref_lse, rows=rows)
    gs.assert_close(stats)
    assert torch.isfinite(out).all()
    return out, stats


def test_config2_step_full_size():
    """The headline step at full size (MHA 24 x 128, 256 new tokens, 4096
    cached, 10 KV splits), committed in the same launch as the benchmark
    runs it: every output element against the oracle."""
    wl = inputs.config(2)
    wl.fuse_append = True
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    ns, _ = ws.step_plan(wl.B, wl.Hq, wl.Hkv, wl.Lq, wl.cache_lens)
    gs.say(f"[gpu] {wl.name}: full size, every output ({ns} KV splits)")
    _check_full(wl, cache=cache)


def test_config3_prefill_full_size():
    wl = inputs.config(3)
    rows = gs.coverage_rows_prefill(np.random.default_rng(5), wl.B, wl.Hq, wl.Lq,
                                    must=[(1, 31, 16383), (0, 7, 255), (1, 8, 256), (0, 16, 8191)])
    _covered(wl, None, rows)


def test_config4_interleaved_full_size():
    wl = inputs.config(4)
    cache = gs.device_cache(wl, [wl.Lq], fill_on_gpu=True)
    offs = wl.offsets[0]
    # every block's first and last row in some head, on top of the coverage
    must = [(0, j % wl.Hq, int(offs[j])) for j in range(wl.num_blocks) if offs[j + 1] > offs[j]]
    must += [(0, (3 * j + 1) % wl.Hq, int(offs[j + 1]) - 1) for j in range(wl.num_blocks) if offs[j + 1] > offs[j]]
    rows = gs.coverage_rows_prefill(np.random.default_rng(5), wl.B, wl.Hq, wl.Lq, must=must)
    _covered(wl, cache, rows)


def test_config5_streams_full_size():
    wl = inputs.config(5)
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    rows = gs.coverage_rows_step(np.random.default_rng(5), wl.B, wl.Hq, wl.Hkv, wl.Lq,
                                 must=[(3, 63, 511), (1, 8, 256), (2, 7, 255)])
    _covered(wl, cache, rows)
    # the fused append committed the new block at positions 131072 ..
    kn = wl.k_new
    for b, t in [(0, 0), (3, 511), (2, 300)]:
        pos = int(wl.cache_lens[b]) + t
        page = int(wl.page_table[b][pos // 64])
        got = cache.k_pool[page, :, pos % 64].cpu()
        assert torch.equal(got.view(torch.int16), kn[b, t].view(torch.int16))


def _every_output(wl, cache=None, groups=None):
    """Full-size run against the block-wise fp64 oracle on every output
    element and lse (of the given (stream, KV head) groups, if any)."""
    gs.say(f"[gpu] {wl.name}: full size, every output" + (f" of groups {groups}" if groups else ""))
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_block_oracle(wl, groups=groups)
    stats = gs.compare_all(out, lse, ref, ref_lse)
    gs.say(f"[gpu]   {stats}")
    gs.assert_close(stats)
    assert torch.isfinite(out).all()


def test_config3_prefill_every_output():
    _every_output(inputs.config(3))


def test_config4_interleaved_every_output():
    wl = inputs.config(4)
    _every_output(wl, cache=gs.device_cache(wl, [wl.Lq], fill_on_gpu=True))


def test_config5_streams_every_output_of_four_groups():
    """Every output of one KV group per stream (KV heads 0, 3, 5, 7: 64 of the
    512 work items); the other groups are covered row by row above."""
    wl = inputs.config(5)
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    _every_output(wl, cache=cache, groups=[(0, 0), (1, 3), (2, 5), (3, 7)])


def test_long_streams_split_by_round_model_full_size():
    """3 streams of 512-token blocks over 131072 cached tokens (GQA 64/8):
    the 384 work-groups fill 1.5 rounds, so the planner splits the KV range
    in two (workspace > 0); one row of every packed 32-row block."""
    B = 3
    wl = inputs.step_workload(f"streams_b{B}_gqa64x8_d128_q512_c131072", B, 64, 8, 128, 512, [131072] * B,
                              seed=1020 + B, fuse_append=True)
    ns, need = ws.step_plan(B, 64, 8, 512, wl.cache_lens)
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert ns == 2 and need > 0
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    rows = gs.coverage_rows_step(np.random.default_rng(7), wl.B, wl.Hq, wl.Hkv, wl.Lq)
    _covered(wl, cache, rows)


def test_long_split_reads_page_ids_from_memory():
    """One long KV split: 170000 cached tokens (2657 pages) in shuffled
    pages, one KV head shared by 8 query heads, 8192 new tokens (65536
    packed rows = 256 query tiles, exactly one round of work-groups on 256
    compute units, so the plan keeps one split); every page id is read from
    the device page table one loop step before its tile's loads.  One row of
    every packed 32-row block (each sees every key)."""
    wl = inputs.step_workload("step_long_split_b1_gqa8x1_q8192_c170000", 1, 8, 1, 128, 8192, [170000],
                              seed=77, fuse_append=True)
    ns, _ = ws.step_plan(1, 8, 1, 8192, wl.cache_lens)
    if ns != 1:
        pytest.skip(f"the device plan splits this step in {ns}")
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    rows = gs.coverage_rows_step(np.random.default_rng(8), wl.B, wl.Hq, wl.Hkv, wl.Lq, must=[(0, 7, 8191)])
    _covered(wl, cache, rows)


def test_million_token_cache():
    """One stream over 1048576 cached tokens (16384 shuffled pages, 512 MiB
    of K/V), 8 query heads on one KV head, a 16-token block committed in the
    same launch: positions, page indices and tile counts at that scale, the
    keys split across up to 32 work-groups.  Every output and lse against
    the oracle."""
    n = 1 << 20
    wl = inputs.step_workload("step_b1_gqa8x1_q16_c1048576", 1, 8, 1, 128, 16, [n], seed=79, fuse_append=True)
    ns, _ = ws.step_plan(1, 8, 1, 16, wl.cache_lens)
    cache = gs.device_cache(wl, wl.cache_lens, fill_on_gpu=True)
    gs.say(f"[gpu] {wl.name}: {ns} splits")
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl)
    gs.assert_close(gs.compare(out, lse, ref, ref_lse))


def test_device_plan_matches_its_compute_units():
    """Steps are planned for the compute units the device reports."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for args in ((1, 24, 24, 256, [4096]), (4, 64, 8, 16, [131072] * 4), (3, 64, 8, 512, [131072] * 3)):
        assert ws.step_plan(*args) == ws.step_plan(*args, num_cus=cus)
        assert ws.step_plan(*args)[1] == ws.workspace_bytes(ws.WS_OP_STEP, *args[:4], max(args[4]) + args[3])
