"""Seeded workload generator: the recipe, its sizes and its poison filling (CPU only)."""
import numpy as np
import pytest
import torch

from paper_2504_15930_amd import inputs

# Seed-0 totals of the length recipe (sum of lengths, longest, pages of 16 tokens).
SEED0 = {
    "tiny": (698, 218, None),
    "qwen7b_longtail": (957_219, 16_896, 59_942),
    "straggler": (329_407, 32_049, 20_596),
    "qwen72b_longtail": (4_184_821, 33_792, 261_787),
    "fp8_qwen7b_longtail": (1_923_430, 33_280, 120_453),
}


@pytest.mark.parametrize("name", list(SEED0))
def test_seed0_lengths(name):
    w = inputs.WORKLOADS[name]
    L = inputs.draw_lengths(w, np.random.default_rng(0))
    total, longest, pages = SEED0[name]
    assert L.shape == (w.batch,)
    assert int(L.sum()) == total and int(L.max()) == longest
    if pages is not None:
        assert int((-(-L // 16)).sum()) == pages
    if w.lengths == "uniform":
        lo, hi = w.params
    else:
        lo, hi = w.params[0] + 1, w.params[0] + w.params[3]
    assert L.min() >= lo and L.max() <= hi


def test_tiny_batch_structure():
    b = inputs.make_batch("tiny", seed=0)
    assert b.q.shape == (8, 4, 64) and b.q.dtype == torch.bfloat16
    assert b.k_pages.shape == (160, 2, 16, 64)
    bt = b.block_table.numpy()
    assert bt.shape == (8, 20) and sorted(bt.ravel().tolist()) == list(range(160))
    assert b.scale == float(np.float32(1 / 8))
    L = b.seq_lens.numpy()
    k = b.k_pages.float()
    for s in range(8):
        nb = -(-int(L[s]) // 16)
        for i in range(nb):
            page = bt[s, i]
            live = min(16, int(L[s]) - 16 * i)
            assert torch.isfinite(k[page, :, :live]).all()
            assert torch.isnan(k[page, :, live:]).all()
        for i in range(nb, 20):
            assert torch.isnan(k[bt[s, i]]).all()


def test_exact_pool_and_poison_padding():
    b = inputs.make_paged_batch([5, 40, 16], 4, 2, 64, seed=3)
    N = 1 + 3 + 1
    assert b.k_pages.shape[0] == N + 1 and b.poison_page == N
    bt = b.block_table.numpy()
    assert bt.shape == (3, 3)
    assert sorted(bt[bt != N].tolist()) == list(range(N))
    assert torch.isnan(b.k_pages[N].float()).all() and torch.isnan(b.v_pages[N].float()).all()


def test_values_are_deterministic():
    a = inputs.make_paged_batch([33, 7], 8, 2, 128, seed=5)
    c = inputs.make_paged_batch([33, 7], 8, 2, 128, seed=5)
    d = inputs.make_paged_batch([33, 7], 8, 2, 128, seed=6)
    assert torch.equal(a.q, c.q) and torch.equal(a.block_table, c.block_table)
    assert torch.equal(a.k_pages.view(torch.int16), c.k_pages.view(torch.int16))
    assert not torch.equal(a.q, d.q)


def test_fp8_quantisation():
    b = inputs.make_paged_batch([20, 3], 4, 2, 64, seed=1, kv_dtype="e4m3")
    ref = inputs.make_paged_batch([20, 3], 4, 2, 64, seed=1)
    assert b.k_pages.dtype == torch.uint8 and b.k_scales.shape == (b.k_pages.shape[0], 2)
    vals = b.k_pages.view(torch.float8_e4m3fn).float() * b.k_scales[:, :, None, None]
    live = torch.isfinite(ref.k_pages.float())
    x = ref.k_pages.float()
    # E4M3 keeps 3 mantissa bits: relative error <= 2^-4 for normal codes
    err = (vals - x).abs()[live]
    assert (err <= x.abs()[live] * 2 ** -4 + b.k_scales.max() * 2 ** -9).all()
    assert (b.k_pages[~live] == 0x7F).all()
    # the scale maps the largest live magnitude of each (page, head) to 448
    amax = torch.where(live, x.abs(), torch.zeros(())).amax(dim=(2, 3))
    used = amax > 0
    assert torch.allclose(b.k_scales[used] * 448, amax[used], rtol=1e-6)
