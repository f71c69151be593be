"""The paged-cache append oracle against a hand-worked example and against
the round-trip property (gathering through the page table returns the
logical token sequence; pages nobody owns keep their sentinel bits)."""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "kv_append_worked_example.json")


def test_worked_example():
    g = json.load(open(GOLDEN))
    P, N = g["page_size"], g["num_pages"]
    pool_k = np.full((N, 1, P, 1), g["sentinel"], np.float64)
    pool_v = pool_k.copy()
    kn = np.array(g["k_new_values"], np.float64)[:, :, None, None]
    oracle.kv_append(pool_k, pool_v, np.array(g["page_table"]), g["cache_lens"], kn, -kn)
    expected = np.array(g["expected_pool"], np.float64)
    assert np.array_equal(pool_k[:, 0, :, 0], expected)
    exp_v = np.where(expected == g["sentinel"], g["sentinel"], -expected)
    assert np.array_equal(pool_v[:, 0, :, 0], exp_v)


def test_round_trip_and_sentinels():
    rng = np.random.default_rng(5)
    B, Hkv, d, P = 3, 2, 8, 16
    lens_final = [0, 37, 64]
    max_pages = 5
    num_pages = B * max_pages + 4
    perm = rng.permutation(num_pages).astype(np.int32)
    table = perm[: B * max_pages].reshape(B, max_pages)
    sentinel = np.uint16(0x7FC1)  # a NaN bit pattern in bf16
    pool_k = np.full((num_pages, Hkv, P, d), sentinel, np.uint16)
    pool_v = pool_k.copy()
    logical_k = rng.integers(0, 0x7F00, size=(B, 64, Hkv, d), dtype=np.uint16)
    logical_v = rng.integers(0, 0x7F00, size=(B, 64, Hkv, d), dtype=np.uint16)
    # grow the cache in uneven slices: every stream appends the same slice
    # count, and each slice length is capped by that stream's final length
    cur = [0] * B
    for piece in (5, 0, 17, 42):
        for b in range(B):
            n = min(piece, lens_final[b] - cur[b])
            if n <= 0:
                continue
            oracle.kv_append(pool_k, pool_v, table[b:b + 1], [cur[b]],
                             logical_k[b:b + 1, cur[b]:cur[b] + n], logical_v[b:b + 1, cur[b]:cur[b] + n])
            cur[b] += n
    assert cur == lens_final
    touched = np.zeros((num_pages, P), bool)
    for b in range(B):
        n = lens_final[b]
        assert np.array_equal(oracle.gather(pool_k, table[b], n), logical_k[b, :n])
        assert np.array_equal(oracle.gather(pool_v, table[b], n), logical_v[b, :n])
        for p in range(n):
            touched[table[b][p // P], p % P] = True
    for page in range(num_pages):
        for slot in range(P):
            if not touched[page, slot]:
                assert np.all(pool_k[page, :, slot] == sentinel)
                assert np.all(pool_v[page, :, slot] == sentinel)
