"""Helpers shared by the GPU parity tests: tolerance check and oracle calls on a batch."""
from __future__ import annotations

import numpy as np
import torch

import oracle

# Tolerance for bf16 inputs with fp32 accumulation and a bf16 output: absolute
# 1e-2 and relative 2e-2, applied per element as |gpu - ref| <= ATOL + RTOL |ref|
# (the bf16 output alone is rounded by up to 2^-9 |ref|, which exceeds 1e-2 once
# |ref| > 5, so a bare 1e-2 bound cannot hold for large outputs), and per
# (sequence, head) row as ||gpu - ref||_2 <= RTOL ||ref||_2. Where |ref| < STRICT_BELOW
# the bare absolute bound |gpu - ref| <= ATOL must hold as well: there the bf16
# output rounding is at most half an ulp of [2, 4), 2^-7 = 7.8e-3, so the stated
# 1e-2 is reachable, and the relative term cannot hide an arithmetic error of up
# to 2-7x the stated bound for outputs of magnitude 0.5-3.
ATOL = 1e-2
RTOL = 2e-2
STRICT_BELOW = 4.0


def assert_parity(gpu, ref: np.ndarray, what: str = "", atol=ATOL, rtol=RTOL, strict_below=STRICT_BELOW,
                  value_scale=None):
    """Elementwise and row-wise parity of a bf16 GPU result with the fp64 oracle.

    ``value_scale``: for inputs whose values are not of unit scale, the RMS of the cached value
    rows each output row averages (array broadcastable to ref.shape[:-1] + (1,), see
    ``value_rms_rows``). The absolute terms are stated for unit-scale data (the workloads draw
    K and V from N(0, 1)); scaling V by s scales the output and every rounding error in it by s,
    so there both the absolute bound and the |ref| range it covers are multiplied by max(1, s).
    One such error is inherent to the method's arithmetic: softmax weights enter the value
    product rounded to bf16 (relative error up to 2^-8 each), which moves the output by up to
    2^-8 times the spread of the value rows around it, not of the output itself.
    """
    g = gpu.detach().float().cpu().double().numpy() if isinstance(gpu, torch.Tensor) else np.asarray(gpu, np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert g.shape == ref.shape, f"{what}: shape {g.shape} vs {ref.shape}"
    assert np.isfinite(g).all(), f"{what}: non-finite GPU output at {np.argwhere(~np.isfinite(g))[:5]}"
    err = np.abs(g - ref)
    s = np.ones(ref.shape[:-1] + (1,)) if value_scale is None else np.maximum(1.0, np.asarray(value_scale, float))
    s = np.broadcast_to(s, ref.shape)
    atol = atol * s
    strict_below = strict_below * s
    excess = err - (atol + rtol * np.abs(ref))
    worst = np.unravel_index(np.argmax(excess), err.shape)
    assert excess.max() <= 0, (f"{what}: |err| {err[worst]:.3g} > {atol[worst]:.3g} + {rtol}|ref| "
                               f"(ref {ref[worst]:.3g}) at {worst}; max abs err {err.max():.3g}")
    small = np.abs(ref) < strict_below
    if small.any():
        es = np.where(small, err - atol, -np.inf)
        ws = np.unravel_index(np.argmax(es), err.shape)
        assert es.max() <= 0, (f"{what}: |err| {err[ws]:.3g} > {atol[ws]:.3g} where |ref| < {strict_below[ws]:.3g} "
                               f"(ref {ref[ws]:.3g}) at {ws}")
    num = np.sqrt(((g - ref) ** 2).sum(axis=-1))
    den = np.sqrt((ref ** 2).sum(axis=-1))
    zero = den == 0
    assert np.all(num[zero] == 0), f"{what}: nonzero output where the reference row is zero"
    rel = num[~zero] / den[~zero]
    if rel.size:
        assert rel.max() <= rtol, f"{what}: max row relative L2 err {rel.max():.3g}"


def value_rms_rows(v_pages: np.ndarray, block_table: np.ndarray, seq_lens: np.ndarray, num_q_heads: int):
    """[B, Hq, 1]: RMS of the live cached value rows that each output row (sequence b, query head
    h) averages, from float64 value pages [N, Hkv, P, D] (dequantised by the caller)."""
    B = len(seq_lens)
    N, Hkv, P, D = v_pages.shape
    G = num_q_heads // Hkv
    out = np.ones((B, num_q_heads, 1))
    for b in range(B):
        L = int(seq_lens[b])
        if L <= 0:
            continue
        nb = -(-L // P)
        rows = v_pages[block_table[b, :nb]].transpose(1, 0, 2, 3).reshape(Hkv, nb * P, D)[:, :L]
        rms = np.sqrt((rows ** 2).mean(axis=(1, 2)))
        out[b, :, 0] = np.repeat(rms, G)
    return out


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
