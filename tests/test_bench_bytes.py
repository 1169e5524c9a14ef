"""The byte counts bench.py divides by: a hand-worked plain count, and the prefix-shared count
against a brute-force count of the distinct pages a GRPO-like batch references."""
import numpy as np
import pytest

import bench
from paper_2504_15930_amd import inputs


def test_algorithmic_bytes_hand_worked():
    # lengths 17, 0, 32 -> 49 tokens on 2 + 0 + 2 pages; Hq 4, Hkv 2, D 64
    L = np.array([17, 0, 32])
    qo = 3 * 2 * 4 * 64 * 2
    assert bench.algorithmic_bytes(L, 4, 2, 64, 2) == 49 * 2 * 2 * 64 * 2 + qo + 4 * 4
    assert bench.algorithmic_bytes(L, 4, 2, 64, 1) == 49 * 2 * 2 * 64 * 1 + 4 * 2 * 2 * 4 + qo + 4 * 4


@pytest.mark.parametrize("kv", ["bf16", "e4m3"])
@pytest.mark.parametrize("prompts,samples,prompt_len", [(3, 4, 40), (2, 8, 16), (5, 2, 100)])
def test_prefix_unique_bytes_brute_force(kv, prompts, samples, prompt_len):
    b, starts, shared = inputs.make_grpo_batch(prompts, samples, prompt_len, seed=prompts + samples, device="cpu",
                                               num_q_heads=8, num_kv_heads=2, head_dim=64, gen_median=30.0,
                                               gen_cap=200, kv_dtype=kv)
    L = b.seq_lens.numpy().astype(np.int64)
    bt = b.block_table.numpy()
    kvb = 1 if kv == "e4m3" else 2
    live = {}   # distinct page id -> live tokens in it (the same for every row that reads it)
    for r in range(len(L)):
        for i in range(-(-int(L[r]) // 16)):
            n = min(16, int(L[r]) - 16 * i)
            assert live.setdefault(int(bt[r, i]), n) == n
    tokens, pages = sum(live.values()), len(live)
    want = (tokens * 2 * 2 * 64 * kvb + len(L) * 2 * 8 * 64 * 2 + pages * 4
            + (pages * 2 * 2 * 4 if kvb == 1 else 0))
    assert bench.prefix_unique_bytes(L, prompts, prompt_len // 16, 8, 2, 64, kvb) == want
    assert bench.prefix_unique_bytes(L, prompts, 0, 8, 2, 64, kvb) == bench.algorithmic_bytes(L, 8, 2, 64, kvb)


def test_subset_rows():
    L = np.array([5, 90, 3, 40, 7, 1, 60, 8] * 10)
    rows = bench.subset_rows(L, 32)
    assert len(rows) == 32 and rows == sorted(set(rows))
    assert int(np.argmax(L)) in rows and int(np.argmin(L)) in rows
    assert bench.subset_rows(L[:20], 32) == list(range(20))
    assert bench.subset_rows(L, 32) == rows   # seeded


def test_ptl_at_hand_worked():
    pb, ps = [1, 4, 8], [10.0, 16.0, 24.0]
    assert bench.ptl_at(0, pb, ps) == 10.0 and bench.ptl_at(1, pb, ps) == 10.0   # flat below
    assert bench.ptl_at(2, pb, ps) == 12.0                                       # 10 + 6 * 1/3
    assert bench.ptl_at(6, pb, ps) == 20.0
    assert bench.ptl_at(12, pb, ps) == 32.0                                      # last segment continued
    assert bench.ptl_at(5, [3], [7.0]) == 7.0


def test_prefix_subgroups():
    assert bench.prefix_subgroups(8, 7) == 1 and bench.prefix_subgroups(16, 7) == 2   # M = 9
    assert bench.prefix_subgroups(20, 7) == 3 and bench.prefix_subgroups(16, 4) == 1  # M = 16
    assert bench.prefix_subgroups(33, 8) == 5 and bench.prefix_subgroups(1, 16) == 1  # M = 8, 4
