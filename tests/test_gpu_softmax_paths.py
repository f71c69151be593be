"""GPU parity on inputs shaped to drive every branch of the kernels' online
softmax (running max in the log2 domain, lazily rescaled; the tile max is
only taken when a row may need a larger running max).  Every query row points
along one direction u and key j carries a chosen score level along u, so
the scores of a whole 64-key tile sit near a level picked per tile:

* rising levels: the running max must grow on every tile;
* a plateau a few units above the first tile's max: many moderate weights
  (their lane sum passes the rescale bound while no single weight does);
* a tile far below the running max (every weight underflows to 0);
* a first tile far below zero (rows that have seen no key yet must take
  the tile's max, or all their weights would underflow);
* a jump far above the running max after all of these.

Both the whole-sequence path (one pass over the keys) and a step whose
keys are split across work-groups (each split starts from an empty running
max) are compared with the fp64 oracle on every output.
Tolerance: max-abs 2e-2, mean-abs 2e-3 (bf16 outputs), lse 1e-3."""
import numpy as np
import pytest
import torch

from paper_2606_25041_amd import inputs
from tests import gpu_support as gs

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634


def _tile_levels(n_keys, profile, seed):
    """Score level (log2 units) of every key: one level per 64-key tile."""
    g = np.random.default_rng([seed, 5])
    nt = -(-n_keys // 64)
    if profile == "rising":
        lv = 12.0 * np.arange(nt)
    elif profile == "mixed":
        pattern = [-150.0, 0.0, 5.0, 5.0, -300.0, 5.0, 40.0, 44.0, 44.0, -100.0]
        lv = np.array([pattern[t % len(pattern)] + 60.0 * (t // len(pattern)) for t in range(nt)])
    else:
        raise ValueError(profile)
    lv = np.repeat(lv, 64)[:n_keys]
    return lv + g.uniform(-0.5, 0.5, n_keys)   # spread within a tile


def _shape(wl, profile, key_pos):
    """Rewrite q and k in place: q rows = u + small noise, key j = its level
    along u (so scale * q.k * log2(e) is about the level) + small noise."""
    D = wl.D
    g = np.random.default_rng([wl.seed, 6])
    u = np.zeros(D)
    u[0] = 1.0
    q = u + 0.02 * g.standard_normal(wl.q.shape)
    wl.q = torch.from_numpy(q.astype(np.float32)).to(torch.bfloat16)
    k = 0.02 * g.standard_normal(wl.k.shape)
    for b in range(wl.B):
        pos = key_pos(b)                       # logical key index -> its position in the sequence
        levels = _tile_levels(int(pos.max()) + 1, profile, wl.seed + b)
        k[b, : len(pos), :, 0] = (levels[pos] / (wl.scale * LOG2E))[:, None]
    wl.k = torch.from_numpy(k.astype(np.float32)).to(torch.bfloat16)
    return wl


def _check_every_output(wl, cache=None):
    gs.say(f"[gpu] {wl.name}: B={wl.B} Hq={wl.Hq} Hkv={wl.Hkv} D={wl.D} Lq={wl.Lq}")
    out, lse = gs.run_gpu(wl, cache=cache)
    torch.cuda.synchronize()
    ref, ref_lse = gs.run_oracle(wl)
    stats = gs.compare(out, lse, ref, ref_lse)
    gs.assert_close(stats)
    assert np.isfinite(out.float().cpu().numpy()).all()
    return stats


@pytest.mark.parametrize("profile,D", [("rising", 128), ("mixed", 128), ("mixed", 64)])
def test_prefill_running_max_paths(profile, D):
    # stream 1's first block lies inside the first tile: its rows see no
    # key above the first tile's level
    lens = [np.array([100, 300, 77, 400, 223]), np.array([40, 600, 60, 300, 100])]
    wl = inputs.prefill_workload(f"softmax_paths_prefill_{profile}_d{D}", 2, 4, 2, D, lens, 5101)
    _shape(wl, profile, lambda b: np.arange(wl.Lq))
    _check_every_output(wl)


@pytest.mark.parametrize("profile", ["rising", "mixed"])
def test_split_step_running_max_paths(profile):
    cache_lens = [3000, 1800]
    wl = inputs.step_workload(f"softmax_paths_step_{profile}", 2, 16, 2, 128, 48, cache_lens, 5102)
    Lc = wl.Lc_max

    def key_pos(b):
        # logical keys: the stream's cache rows, unused rows up to Lc, then
        # the new block (which follows the cache in the sequence)
        pos = np.zeros(Lc + wl.Lq, dtype=np.int64)
        pos[: cache_lens[b]] = np.arange(cache_lens[b])
        pos[cache_lens[b]: Lc] = 0
        pos[Lc:] = cache_lens[b] + np.arange(wl.Lq)
        return pos

    _shape(wl, profile, key_pos)
    cache = gs.device_cache(wl, wl.cache_lens)
    _check_every_output(wl, cache=cache)
