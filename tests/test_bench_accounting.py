"""The benchmark's work accounting (CPU only): the visible (query, key)
pairs behind every TFLOP/s figure, counted by brute force from the masking
rule row by row, and the algorithmic bytes written out term by term."""
import numpy as np
import pytest

import bench
from paper_2606_25041_amd import inputs


def _pairs_brute(wl):
    """Per stream: sum over real query rows of the keys they see."""
    out = []
    if wl.kind == "step":
        for b in range(wl.B):
            c = int(wl.cache_lens[b])
            n = int(wl.Lq) if getattr(wl, "new_lens", None) is None else int(wl.new_lens[b])
            tau = n if getattr(wl, "text_starts", None) is None else int(wl.text_starts[b])
            total = 0
            for t in range(n):
                # cache tokens, then the block's own tokens j < n with
                # j < tau or j <= t
                total += c + sum(1 for j in range(n) if j < tau or j <= t)
            out.append(total)
        return out
    for b in range(wl.B):
        off = [int(x) for x in wl.offsets[b]]
        total = 0
        for blk in range(len(off) - 1):
            s, e = off[blk], off[blk + 1]
            tau = e if getattr(wl, "text_starts", None) is None else int(wl.text_starts[b][blk])
            for i in range(s, e):
                total += s + sum(1 for j in range(s, e) if j < tau or j <= i)
        out.append(total)
    return out


def _small_cases():
    st = inputs.step_workload("acc_step", 3, 4, 2, 64, 37, [0, 100, 5], seed=1)
    st_text = inputs.step_workload("acc_step_text", 3, 4, 2, 64, 37, [0, 100, 5], seed=1)
    st_text.text_starts = np.array([0, 20, 37], np.int32)
    st_var = inputs.step_workload("acc_step_var", 3, 4, 2, 64, 37, [0, 100, 5], seed=1)
    st_var.new_lens = np.array([37, 1, 20], np.int32)
    st_var.text_starts = np.array([5, 0, 30], np.int32)
    pf = inputs.prefill_workload("acc_prefill", 2, 4, 2, 64, [np.array([3, 0, 50, 7]), np.array([20, 20, 0, 20])], seed=2)
    pf_text = inputs.prefill_workload("acc_prefill_text", 1, 4, 2, 64, [np.array([10, 0, 40, 9])], seed=2)
    pf_text.text_starts = np.array([[4, 10, 30, 59]], np.int32)
    return [st, st_text, st_var, pf, pf_text]


@pytest.mark.parametrize("i", range(5))
def test_visible_pairs_match_brute_force(i):
    wl = _small_cases()[i]
    assert bench.visible_pairs(wl) == _pairs_brute(wl), wl.name


def test_visible_pairs_of_the_measured_step_workloads():
    wls = [inputs.config(2), inputs.thinker_step(Lc=4096), inputs.streams_varlen(Lc=4096)]
    for wl in wls:
        assert bench.visible_pairs(wl) == _pairs_brute(wl), wl.name
    # the headline: 256 rows x (4096 cached + 256 own keys)
    assert bench.visible_pairs(inputs.config(2)) == [256 * 4352]
    assert bench.algorithmic_flops(inputs.config(2)) == 4.0 * 128 * 24 * 256 * 4352


def test_algorithmic_bytes_terms():
    wl = inputs.streams_varlen(Lc=4096)
    n = [int(x) for x in wl.new_lens]
    e = 2
    want = (sum(n) * wl.Hq * wl.D * e * 2                                   # q read, o written (bf16)
            + 2 * sum(4096 + k for k in n) * wl.Hkv * wl.D * e              # K and V once per KV head
            + 2 * sum(n) * wl.Hkv * wl.D * e)                               # the committed real tokens
    assert bench.algorithmic_bytes(wl) == want
    h = inputs.config(2)
    h.fuse_append = True
    assert bench.algorithmic_bytes(h) == 59768832


def test_oracle_sample_row_keys_match_brute_force():
    """The per-row key counts behind the oracle sample's TFLOP/s equal the
    masking rule counted key by key (block-causal, no segments)."""
    pf = _small_cases()[3]
    rows = inputs.sample_rows(np.random.default_rng(3), pf.B, pf.Hq, pf.Lq, 40)
    got = bench.row_key_counts(pf, rows)
    for (b, h, i), n in zip(rows, got):
        off = [int(x) for x in pf.offsets[b]]
        blk = max(k for k in range(len(off) - 1) if off[k] <= i < off[k + 1])
        assert n == sum(1 for j in range(pf.Lq) if j < off[blk + 1]), (b, h, i)
    st = _small_cases()[0]
    rows = inputs.sample_rows(np.random.default_rng(4), st.B, st.Hq, st.Lq, 20)
    assert list(bench.row_key_counts(st, rows)) == [int(st.cache_lens[b]) + st.Lq for b, _, _ in rows]
    # a whole workload's rows sum to its visible pairs
    all_rows = np.array([(b, h, i) for b in range(pf.B) for h in range(pf.Hq) for i in range(pf.Lq)])
    assert int(bench.row_key_counts(pf, all_rows).sum()) == pf.Hq * sum(bench.visible_pairs(pf))
