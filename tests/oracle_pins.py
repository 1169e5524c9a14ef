"""Checks that pin the CPU oracle to facts outside itself.

Each ``pin_*`` function takes the path of an oracle shared library and raises
AssertionError when the library disagrees with what the definition of decode
attention (softmax(q K^T * scale) V over the sequence's cached tokens, read
through the block table) fixes independently of the oracle's code:

* a library routine: ``torch.nn.functional.scaled_dot_product_attention`` in
  float64 on dense per-sequence tensors that the *test* scatters into pages
  (the inverse of the oracle's gather), with the GQA grouping of
  ``enable_gqa=True``; ``torch.float8_e4m3fn`` for the FP8 code table;
* closed forms: one cached token returns its value row; identical keys (or
  scale 0) return the mean of the value rows; constant values come back
  unchanged; a token whose score exceeds all others by thousands returns its
  own value row exactly; hand-derived fixtures in ``tests/golden``;
* invariants: physical page order, aliasing block-table rows (prefix sharing),
  and head permutations inside a KV group.

The same functions run against deliberately broken copies of the oracle (see
``test_oracle_mutants.py``) to show that each plausible mistake trips one of
them.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
BF16_NAN = np.uint16(0x7FC0)


def bf16_bits(x) -> np.ndarray:
    """Round a float tensor/array to bf16 and return the bit patterns (uint16)."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bits_f64(bits) -> torch.Tensor:
    """bf16 bit patterns -> float64 tensor (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(b.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64)


def scatter_pages(logical: np.ndarray, lengths, P: int, rng: np.random.Generator,
                  fill, extra_pages: int = 3, table=None, num_pages=None):
    """Place per-sequence tokens ``logical[b, t, g, :]`` into a shuffled page pool.

    Returns (pool [N, Hkv, P, D], block_table [B, max_blocks]). Pages that hold
    no token, slots past a sequence's end and the padding column are ``fill``.
    With ``table`` given, that table is used (it may alias pages) with a pool of
    ``num_pages`` pages (default: largest id + 1 + extra_pages); tokens of later
    sequences then overwrite shared slots, so callers sharing pages must give
    equal tokens there.
    """
    B, _, H, D = logical.shape
    lengths = np.asarray(lengths)
    nb = -(-lengths // P)
    if table is None:
        n_live = int(nb.sum())
        N = n_live + extra_pages
        ids = rng.permutation(N)
        pad = ids[-1]
        table = np.full((B, int(max(nb.max(initial=0), 1)) + 1), pad, dtype=np.int32)
        c = 0
        for b in range(B):
            table[b, :nb[b]] = ids[c:c + nb[b]]
            c += nb[b]
    else:
        table = np.asarray(table, dtype=np.int32)
        N = num_pages if num_pages is not None else int(table.max()) + 1 + extra_pages
    pool = np.empty((N, H, P, D), dtype=logical.dtype)
    pool[...] = fill
    for b in range(B):
        for t in range(int(lengths[b])):
            pool[table[b, t // P], :, t % P, :] = logical[b, t]
    return pool, table


def sdpa_reference(q_f64, k_log_f64, v_log_f64, lengths, scale):
    """float64 SDPA per sequence on dense [B, Lmax, Hkv, D] tensors; zero rows for L=0."""
    B, Hq, D = q_f64.shape
    out = torch.zeros((B, Hq, D), dtype=torch.float64)
    for b in range(B):
        L = int(lengths[b])
        if L == 0:
            continue
        qb = q_f64[b][None, :, None, :]
        kb = k_log_f64[b, :L].permute(1, 0, 2)[None]
        vb = v_log_f64[b, :L].permute(1, 0, 2)[None]
        out[b] = F.scaled_dot_product_attention(qb, kb, vb, scale=float(np.float32(scale)),
                                                enable_gqa=True)[0, :, 0, :]
    return out.numpy()


def _close(a, b, rtol, what):
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.abs(a - b)
    bound = rtol * np.maximum(1.0, np.abs(b))
    assert np.all(err <= bound), f"{what}: max err {np.nanmax(err)} (nan: {np.isnan(a).any()})"


def random_case(rng, B, Hq, Hkv, D, P, lengths, scale=None, table=None):
    """Random bf16 q/K/V; returns dict of oracle inputs plus the dense float64 tensors."""
    lengths = np.asarray(lengths, dtype=np.int32)
    Lmax = max(int(lengths.max(initial=0)), 1)
    q = bf16_bits(rng.standard_normal((B, Hq, D)))
    k_log = bf16_bits(rng.standard_normal((B, Lmax, Hkv, D)))
    v_log = bf16_bits(rng.standard_normal((B, Lmax, Hkv, D)))
    if table is not None:
        # sequences sharing a page share its tokens: copy from the first owner
        owner = {}
        for b in range(B):
            for t in range(int(lengths[b])):
                key = (int(table[b, t // P]), t % P)
                if key in owner:
                    ob, ot = owner[key]
                    k_log[b, t] = k_log[ob, ot]
                    v_log[b, t] = v_log[ob, ot]
                else:
                    owner[key] = (b, t)
    sub = np.random.default_rng(int(rng.integers(1 << 31)))
    k_pages, bt = scatter_pages(k_log, lengths, P, sub, BF16_NAN, table=table)
    v_pages, _ = scatter_pages(v_log, lengths, P, sub, BF16_NAN, table=bt,
                               num_pages=k_pages.shape[0])
    if scale is None:
        scale = float(np.float32(1.0 / np.sqrt(D)))
    return dict(q=q, k_pages=k_pages, v_pages=v_pages, block_table=bt, seq_lens=lengths,
                scale=scale), dict(q=bits_f64(q), k=bits_f64(k_log), v=bits_f64(v_log))


def run(lib, case, **kw):
    return oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"],
                              case["seq_lens"], case["scale"], lib=lib, **kw)


# --------------------------------------------------------------------------- pins

def pin_sdpa_random(lib):
    """Random shapes (G = 1, 2, 4, 7; D = 32, 64, 128; page 4 and 16) vs float64 SDPA."""
    rng = np.random.default_rng(11)
    shapes = [
        (5, 8, 2, 64, 16, [1, 15, 16, 17, 40]),
        (3, 6, 6, 128, 16, [33, 2, 64]),
        (2, 7, 1, 32, 16, [50, 9]),
        (4, 4, 2, 64, 4, [7, 0, 13, 4]),
        (1, 16, 4, 64, 16, [200]),
    ]
    for B, Hq, Hkv, D, P, lengths in shapes:
        case, dense = random_case(rng, B, Hq, Hkv, D, P, lengths)
        ref = sdpa_reference(dense["q"], dense["k"], dense["v"], lengths, case["scale"])
        _close(run(lib, case), ref, 1e-12, f"sdpa B={B} Hq={Hq} Hkv={Hkv} D={D} P={P}")


def pin_sdpa_large_scores(lib):
    """Scores in the hundreds (scale 40): a softmax without max-subtraction overflows."""
    rng = np.random.default_rng(12)
    case, dense = random_case(rng, 3, 4, 2, 64, 16, [30, 17, 5], scale=40.0)
    ref = sdpa_reference(dense["q"], dense["k"], dense["v"], case["seq_lens"], 40.0)
    _close(run(lib, case), ref, 1e-10, "sdpa large scores")


def pin_prefix_sharing(lib):
    """Rows of the block table alias pages (shared prompt prefix) vs float64 SDPA."""
    rng = np.random.default_rng(13)
    P = 16
    table = np.array([[0, 1, 2, 9],
                      [0, 1, 3, 9],      # shares the first two pages with sequence 0
                      [0, 4, 5, 9],
                      [6, 7, 8, 9]], dtype=np.int32)
    lengths = [40, 35, 48, 20]
    case, dense = random_case(rng, 4, 4, 2, 64, P, lengths, table=table)
    ref = sdpa_reference(dense["q"], dense["k"], dense["v"], lengths, case["scale"])
    _close(run(lib, case), ref, 1e-12, "prefix sharing")
    # identical rows when two sequences alias all pages and share q
    case["block_table"] = np.array([[0, 1, 2, 9], [0, 1, 2, 9]], dtype=np.int32)
    case["seq_lens"] = np.array([37, 37], dtype=np.int32)
    case["q"] = np.stack([case["q"][0], case["q"][0]])
    out = run(lib, case)
    assert np.array_equal(out[0], out[1]), "aliased sequences differ"


def pin_single_token(lib):
    """One cached token: the output is that token's value row, exactly."""
    rng = np.random.default_rng(14)
    case, dense = random_case(rng, 4, 8, 2, 64, 16, [1, 1, 1, 1])
    out = run(lib, case)
    G = 4
    for b in range(4):
        for h in range(8):
            assert np.array_equal(out[b, h], dense["v"][b, 0, h // G].numpy()), "single token"


def pin_identical_keys(lib):
    """All keys of a sequence equal: uniform weights, so the output is the mean value row."""
    rng = np.random.default_rng(15)
    B, Hq, Hkv, D, P = 3, 4, 2, 64, 16
    lengths = np.array([5, 16, 33], dtype=np.int32)
    case, dense = random_case(rng, B, Hq, Hkv, D, P, lengths)
    k_log = np.repeat(bf16_bits(rng.standard_normal((B, 1, Hkv, D))), lengths.max(), axis=1)
    sub = np.random.default_rng(1)
    case["k_pages"], _ = scatter_pages(k_log, lengths, P, sub, BF16_NAN, table=case["block_table"],
                                       num_pages=case["k_pages"].shape[0])
    out = run(lib, case)
    for b in range(B):
        mean = dense["v"][b, :lengths[b]].mean(dim=0).numpy()       # [Hkv, D]
        for h in range(Hq):
            _close(out[b, h], mean[h // 2], 1e-14, "identical keys")
    # scale 0 gives the same uniform weights whatever the keys
    case2, dense2 = random_case(rng, B, Hq, Hkv, D, P, lengths, scale=0.0)
    out2 = run(lib, case2)
    for b in range(B):
        mean = dense2["v"][b, :lengths[b]].mean(dim=0).numpy()
        for h in range(Hq):
            _close(out2[b, h], mean[h // 2], 1e-14, "scale zero")


def pin_constant_values(lib):
    """Softmax weights sum to one: constant value rows come back unchanged."""
    rng = np.random.default_rng(16)
    case, _ = random_case(rng, 3, 6, 3, 64, 16, [9, 31, 64])
    for pages in ("v_pages",):
        live = case[pages] != BF16_NAN
        case[pages] = np.where(live, bf16_bits(np.full(case[pages].shape, 1.5)), BF16_NAN)
    out = run(lib, case)
    _close(out, np.full(out.shape, 1.5), 1e-14, "constant values")


def pin_dominant_token(lib):
    """One token's score exceeds the rest by 4096: output = its value row, at every position.

    Value rows encode (sequence, position, kv head) as small integers, so a read of
    the wrong page, slot or head returns a different row.
    """
    B, Hq, Hkv, D, P = 2, 4, 2, 64, 16
    lengths = np.array([37, 20], dtype=np.int32)
    Lmax = int(lengths.max())
    rng = np.random.default_rng(17)
    v_log = np.zeros((B, Lmax, Hkv, D), dtype=np.float32)
    for b in range(B):
        for t in range(Lmax):
            for g in range(Hkv):
                v_log[b, t, g, :] = (b * 64 + t) + g / 2.0 + np.arange(D) % 3 * 0.25
    v_bits = bf16_bits(v_log)
    q = np.zeros((B, Hq, D), dtype=np.float32)
    q[:, :, 0] = 64.0
    q_bits = bf16_bits(q)
    for b in range(B):
        for t in range(int(lengths[b])):
            k_log = np.zeros((B, Lmax, Hkv, D), dtype=np.float32)
            k_log[b, t, :, 0] = 64.0          # score 4096 at (b, t); 0 elsewhere
            k_bits = bf16_bits(k_log)
            sub = np.random.default_rng(1000 + t)
            k_pages, table = scatter_pages(k_bits, lengths, P, sub, BF16_NAN)
            v_pages, _ = scatter_pages(v_bits, lengths, P, sub, BF16_NAN, table=table,
                                       num_pages=k_pages.shape[0])
            case = dict(q=q_bits, k_pages=k_pages, v_pages=v_pages, block_table=table,
                        seq_lens=lengths, scale=1.0)
            out = run(lib, case, rows=[b])
            want = bits_f64(v_bits[b, t]).numpy()        # [Hkv, D]
            for h in range(Hq):
                assert np.array_equal(out[0, h], want[h // (Hq // Hkv)]), \
                    f"dominant token b={b} t={t} h={h}"
    _ = rng


def pin_page_permutation(lib):
    """Physical page order is irrelevant: permuting the pool and remapping the table is exact."""
    rng = np.random.default_rng(18)
    case, _ = random_case(rng, 4, 8, 4, 64, 16, [3, 70, 16, 33])
    base = run(lib, case)
    N = case["k_pages"].shape[0]
    perm = rng.permutation(N)
    new = dict(case)
    new["k_pages"] = np.empty_like(case["k_pages"])
    new["v_pages"] = np.empty_like(case["v_pages"])
    new["k_pages"][perm] = case["k_pages"]
    new["v_pages"][perm] = case["v_pages"]
    new["block_table"] = perm[case["block_table"]].astype(np.int32)
    assert np.array_equal(run(lib, new), base), "page permutation changed the result"


def pin_head_permutation(lib):
    """Permuting q heads inside one KV group permutes the outputs; other groups are untouched."""
    rng = np.random.default_rng(19)
    case, _ = random_case(rng, 2, 8, 2, 64, 16, [21, 40])
    base = run(lib, case)
    perm = np.array([2, 0, 3, 1, 4, 5, 6, 7])
    new = dict(case)
    new["q"] = case["q"][:, perm]
    assert np.array_equal(run(lib, new), base[:, perm]), "head permutation"
    # moving a head across groups changes its output (the grouping is contiguous)
    cross = np.array([4, 1, 2, 3, 0, 5, 6, 7])
    new["q"] = case["q"][:, cross]
    assert not np.allclose(run(lib, new)[:, 0], base[:, 4]), "head grouping"


def pin_zero_length(lib):
    """A sequence with no cached token yields a zero row; others are unaffected."""
    rng = np.random.default_rng(20)
    case, dense = random_case(rng, 3, 4, 2, 64, 16, [0, 12, 0])
    out = run(lib, case)
    assert np.array_equal(out[0], np.zeros_like(out[0])) and np.array_equal(out[2], out[0])
    ref = sdpa_reference(dense["q"], dense["k"], dense["v"], case["seq_lens"], case["scale"])
    _close(out[1], ref[1], 1e-12, "zero length neighbour")


def pin_rows_subset(lib):
    """Computing a subset of sequences returns exactly those rows of the full result."""
    rng = np.random.default_rng(21)
    case, _ = random_case(rng, 5, 4, 1, 64, 16, [5, 50, 17, 1, 30])
    full = run(lib, case)
    part = run(lib, case, rows=[3, 1, 1])
    assert np.array_equal(part, full[[3, 1, 1]]), "row subset"


def pin_e4m3_table(lib):
    """All 256 FP8 E4M3 codes decode as torch.float8_e4m3fn does (NaN for 0x7F/0xFF)."""
    ref = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn)
    ref = ref.to(torch.float64).numpy()
    got = np.array([oracle.e4m3_to_double(c, lib=lib) for c in range(256)])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan), "e4m3 NaN codes"
    assert np.array_equal(got[~nan], ref[~nan]), "e4m3 values"


def pin_sdpa_fp8(lib):
    """FP8 pages with per-(page, head) scales vs float64 SDPA on dequantised values."""
    rng = np.random.default_rng(22)
    B, Hq, Hkv, D, P = 3, 8, 2, 64, 16
    lengths = np.array([17, 40, 3], dtype=np.int32)
    Lmax = int(lengths.max())
    q = bf16_bits(rng.standard_normal((B, Hq, D)))
    codes_k = rng.integers(0, 256, (B, Lmax, Hkv, D)).astype(np.uint8)
    codes_v = rng.integers(0, 256, (B, Lmax, Hkv, D)).astype(np.uint8)
    for c in (codes_k, codes_v):          # keep NaN codes out of live slots
        c[(c & 0x7F) == 0x7F] = 0x3C
    sub = np.random.default_rng(5)
    k_pages, table = scatter_pages(codes_k, lengths, P, sub, np.uint8(0x7F))
    v_pages, _ = scatter_pages(codes_v, lengths, P, sub, np.uint8(0x7F), table=table,
                               num_pages=k_pages.shape[0])
    N = k_pages.shape[0]
    k_scales = (2.0 ** rng.integers(-8, 4, (N, Hkv)) * rng.uniform(0.5, 1.0, (N, Hkv))).astype(np.float32)
    v_scales = (2.0 ** rng.integers(-8, 4, (N, Hkv)) * rng.uniform(0.5, 1.0, (N, Hkv))).astype(np.float32)

    def deq(codes_log, scales):
        vals = torch.from_numpy(codes_log).view(torch.float8_e4m3fn).to(torch.float64)
        s = torch.zeros((B, Lmax, Hkv, 1), dtype=torch.float64)
        for b in range(B):
            for t in range(int(lengths[b])):
                s[b, t, :, 0] = torch.from_numpy(scales[table[b, t // P]].astype(np.float64))
        return vals * s

    ref = sdpa_reference(bits_f64(q), deq(codes_k, k_scales), deq(codes_v, v_scales), lengths,
                         float(np.float32(1 / 8)))
    out = oracle.decode_attn(q, k_pages, v_pages, table, lengths, float(np.float32(1 / 8)),
                             k_scales=k_scales, v_scales=v_scales, lib=lib)
    _close(out, ref, 1e-12, "fp8 vs sdpa")


def pin_golden_hand_worked(lib):
    """Hand-derived closed-form examples stored in tests/golden/hand_worked.json."""
    with open(os.path.join(GOLDEN, "hand_worked.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        q = bf16_bits(np.array(c["q"], dtype=np.float32))
        P = c["page_size"]
        k = bf16_bits(np.array(c["k_pages"], dtype=np.float32))
        v = bf16_bits(np.array(c["v_pages"], dtype=np.float32))
        for bits, vals in ((k, c["k_pages"]), (v, c["v_pages"])):
            assert np.array_equal(bits_f64(bits).numpy(), np.array(vals, dtype=np.float64),
                                  equal_nan=True), "fixture values must be exact in bf16"
        assert k.shape[2] == P
        out = oracle.decode_attn(q, k, v, np.array(c["block_table"], dtype=np.int32),
                                 np.array(c["seq_lens"], dtype=np.int32),
                                 float(np.float32(c["scale"])), lib=lib)
        _close(out, np.array(c["expected"]), c["rtol"], c["name"])


ALL_PINS = [
    pin_sdpa_random, pin_sdpa_large_scores, pin_prefix_sharing, pin_single_token,
    pin_identical_keys, pin_constant_values, pin_dominant_token, pin_page_permutation,
    pin_head_permutation, pin_zero_length, pin_rows_subset, pin_e4m3_table, pin_sdpa_fp8,
    pin_golden_hand_worked,
]
