"""Helpers shared by the GPU parity tests: tolerance check and oracle calls on a batch."""
from __future__ import annotations

import numpy as np
import torch

import oracle

# Tolerance for bf16 inputs with fp32 accumulation and a bf16 output: absolute
# 1e-2 and relative 2e-2, applied per element as |gpu - ref| <= ATOL + RTOL |ref|
# (the bf16 output alone is rounded by up to 2^-9 |ref|, which exceeds 1e-2 once
# |ref| > 5, so a bare 1e-2 bound cannot hold for large outputs), and per
# (sequence, head) row as ||gpu - ref||_2 <= RTOL ||ref||_2.
ATOL = 1e-2
RTOL = 2e-2


def assert_parity(gpu: torch.Tensor, ref: np.ndarray, what: str = "", atol=ATOL, rtol=RTOL):
    g = gpu.detach().float().cpu().double().numpy()
    ref = np.asarray(ref, dtype=np.float64)
    assert g.shape == ref.shape, f"{what}: shape {g.shape} vs {ref.shape}"
    assert np.isfinite(g).all(), f"{what}: non-finite GPU output at {np.argwhere(~np.isfinite(g))[:5]}"
    err = np.abs(g - ref)
    excess = err - (atol + rtol * np.abs(ref))
    worst = np.unravel_index(np.argmax(excess), err.shape)
    assert excess.max() <= 0, (f"{what}: |err| {err[worst]:.3g} > {atol} + {rtol}|ref| "
                               f"(ref {ref[worst]:.3g}) at {worst}; max abs err {err.max():.3g}")
    num = np.sqrt(((g - ref) ** 2).sum(axis=-1))
    den = np.sqrt((ref ** 2).sum(axis=-1))
    zero = den == 0
    assert np.all(num[zero] == 0), f"{what}: nonzero output where the reference row is zero"
    rel = num[~zero] / den[~zero]
    if rel.size:
        assert rel.max() <= rtol, f"{what}: max row relative L2 err {rel.max():.3g}"


def oracle_full(batch, threads: int = 0) -> np.ndarray:
    """The oracle on every sequence of ``batch`` (host copies of all inputs)."""
    h = batch.host_arrays()
    return oracle.decode_attn(h["q"], h["k_pages"], h["v_pages"], h["block_table"], h["seq_lens"],
                              h["scale"], k_scales=h.get("k_scales"), v_scales=h.get("v_scales"),
                              threads=threads)


def oracle_rows(batch, rows, threads: int = 0) -> np.ndarray:
    """The oracle on the sequences ``rows`` of a (possibly huge) device batch.

    Only the pages those sequences reference are copied to the host: the pool
    is compacted on the device with ``index_select`` and the block-table rows are
    renumbered, which leaves every cached token where the definition reads it.
    """
    rows = [int(r) for r in rows]
    bt = batch.block_table[rows].cpu().numpy()
    lens = batch.seq_lens[rows].cpu().numpy()
    nb = -(-np.maximum(lens, 0) // 16)
    used = np.unique(np.concatenate([bt[i, :nb[i]] for i in range(len(rows))] + [np.zeros(0, np.int32)]))
    remap = {int(p): i for i, p in enumerate(used)}
    new_bt = np.zeros_like(bt)
    for i in range(len(rows)):
        new_bt[i, :nb[i]] = [remap[int(p)] for p in bt[i, :nb[i]]]
    idx = torch.as_tensor(used.astype(np.int64), device=batch.k_pages.device)
    if idx.numel() == 0:
        idx = torch.zeros(1, dtype=torch.int64, device=batch.k_pages.device)

    def bits(t):
        t = t.detach().cpu().contiguous()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    k = bits(batch.k_pages.index_select(0, idx))
    v = bits(batch.v_pages.index_select(0, idx))
    q = bits(batch.q[rows])
    ks = vs = None
    if batch.k_scales is not None:
        ks = batch.k_scales.index_select(0, idx).cpu().numpy()
        vs = batch.v_scales.index_select(0, idx).cpu().numpy()
    return oracle.decode_attn(q, k, v, new_bt.astype(np.int32), lens.astype(np.int32), batch.scale,
                              k_scales=ks, v_scales=vs, threads=threads)


def sample_rows(seq_lens, n: int, seed: int = 0) -> list[int]:
    """n sequences of a batch: always the longest and the shortest, the rest seeded-random."""
    L = np.asarray(seq_lens.cpu() if isinstance(seq_lens, torch.Tensor) else seq_lens)
    rng = np.random.default_rng(seed)
    pick = {int(np.argmax(L)), int(np.argmin(L))}
    rest = [i for i in rng.permutation(len(L)) if i not in pick]
    return sorted(pick | set(int(i) for i in rest[: max(0, n - len(pick))]))
