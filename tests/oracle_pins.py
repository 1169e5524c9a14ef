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


# ------------------------------------------------------------- KV append pins
#
# The append step (oracle/append.c) is pinned the same way: torch's own
# float8_e4m3fn conversion for the encoder, float64 SDPA over dense sequences
# for where a bf16 row lands, torch-quantised whole pages for the FP8 scale
# rule, an error bound for re-encoding, and a hand-derived fixture.

E4M3_FN = torch.float8_e4m3fn


def torch_e4m3(y: np.ndarray) -> np.ndarray:
    """torch's float32 -> float8_e4m3fn codes after clamping to +-448 (saturation)."""
    t = torch.from_numpy(np.asarray(y, dtype=np.float32)).clamp(-448.0, 448.0)
    return t.to(E4M3_FN).view(torch.uint8).numpy().copy()


def _e4m3_probe_values() -> np.ndarray:
    finite = np.array([oracle.e4m3_to_double(c) for c in range(256)], dtype=np.float64)
    finite = np.unique(finite[np.isfinite(finite)])                   # sorted, -448 .. 448
    mids = (finite[:-1] + finite[1:]) / 2                             # exact ties
    f32 = lambda x: np.asarray(x, dtype=np.float32)
    around = np.concatenate([np.nextafter(f32(mids), f32(np.inf)), np.nextafter(f32(mids), f32(-np.inf))])
    rng = np.random.default_rng(5)
    rand = f32(np.exp(rng.uniform(np.log(2.0 ** -13), np.log(600.0), 3000)) * rng.choice([-1, 1], 3000))
    big = f32([448.0, 449.0, 463.99, 464.0, 465.0, 480.0, 1e6, 3e38, np.inf, -np.inf, -470.0])
    small = f32([0.0, -0.0, 2.0 ** -9, 2.0 ** -10, 3 * 2.0 ** -11, 2.0 ** -12, 1e-30, -1e-30, 2.0 ** -6, 0.015624])
    return np.concatenate([f32(finite), f32(mids), around, rand, big, small])


def pin_e4m3_encode_torch(lib):
    """The encoder equals torch's float8_e4m3fn conversion (after +-448 clamping) on every
    code, every tie, both neighbours of every tie, subnormals, saturation and random values."""
    y = _e4m3_probe_values()
    got = oracle.e4m3_encode(y, lib=oracle.load(lib))
    want = torch_e4m3(y)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, f"encode differs from torch at {y[bad[:5]]}: {got[bad[:5]]} vs {want[bad[:5]]}"
    assert oracle.e4m3_encode(np.array([np.nan], np.float32), lib=oracle.load(lib))[0] == 0x7F


def _append_case(rng, lengths, Hkv, D, P, fp8):
    """Pages holding each sequence's first L-1 tokens, plus the step's new rows."""
    lengths = np.asarray(lengths, dtype=np.int32)
    B = len(lengths)
    Lmax = max(int(lengths.max(initial=0)), 1)
    k_log = bf16_bits(rng.standard_normal((B, Lmax, Hkv, D)) * rng.uniform(0.2, 5.0, (B, Lmax, 1, 1)))
    v_log = bf16_bits(rng.standard_normal((B, Lmax, Hkv, D)) * rng.uniform(0.2, 5.0, (B, Lmax, 1, 1)))
    before = np.maximum(lengths - 1, 0)
    sub = np.random.default_rng(int(rng.integers(1 << 31)))
    k_pages, bt = scatter_pages(k_log, lengths, P, sub, BF16_NAN)
    v_pages, _ = scatter_pages(v_log, lengths, P, sub, BF16_NAN, table=bt, num_pages=k_pages.shape[0])
    # the new token's slot is not written yet: poison it
    for b in range(B):
        if lengths[b] >= 1:
            t = lengths[b] - 1
            k_pages[bt[b, t // P], :, t % P, :] = BF16_NAN
            v_pages[bt[b, t // P], :, t % P, :] = BF16_NAN
    idx = np.maximum(lengths - 1, 0)
    k_new = k_log[np.arange(B), idx]                                  # [B, Hkv, D]
    v_new = v_log[np.arange(B), idx]
    return dict(lengths=lengths, before=before, bt=bt, k_pages=k_pages, v_pages=v_pages,
                k_new=k_new, v_new=v_new, k_log=k_log, v_log=v_log)


def pin_append_bf16_dense(lib):
    """After appending the new rows, attention over the pages equals float64 SDPA over the
    dense sequences that end with those rows, and no other slot changed."""
    rng = np.random.default_rng(21)
    P, Hkv, D, G = 16, 2, 64, 3
    lengths = [1, 15, 16, 17, 33, 0, 48, 2]
    c = _append_case(rng, lengths, Hkv, D, P, fp8=False)
    kp, vp = oracle.kv_append(c["k_new"], c["v_new"], c["bt"], c["lengths"], c["k_pages"],
                              c["v_pages"], lib=oracle.load(lib))
    changed = np.any(kp != c["k_pages"], axis=-1) | np.any(vp != c["v_pages"], axis=-1)
    expect = np.zeros_like(changed)
    for b, L in enumerate(lengths):
        if L >= 1:
            expect[c["bt"][b, (L - 1) // P], :, (L - 1) % P] = True
    assert np.array_equal(changed, expect), "append wrote outside the new tokens' slots"
    q = bf16_bits(rng.standard_normal((len(lengths), Hkv * G, D)))
    scale = float(np.float32(1 / 8))
    out = oracle.decode_attn(q, kp, vp, c["bt"], c["lengths"], scale, lib=lib)
    ref = sdpa_reference(bits_f64(q), bits_f64(c["k_log"]), bits_f64(c["v_log"]), lengths, scale)
    _close(out, ref, 1e-12, "append then attend vs dense sdpa")


def _fp8_pages_from(c, P):
    """E4M3 pages holding the first L-1 tokens quantised per (page, head) by torch."""
    kp = c["k_pages"]
    N, Hkv, _, D = kp.shape
    out = []
    for pages in (c["k_pages"], c["v_pages"]):
        vals = bits_f64(pages).to(torch.float32)
        live = torch.zeros((N, 1, P, 1), dtype=torch.bool)
        for b, L in enumerate(c["lengths"]):
            for t in range(max(int(L) - 1, 0)):
                live[c["bt"][b, t // P], 0, t % P, 0] = True
        amax = torch.where(live, vals.abs(), torch.zeros(())).amax(dim=(2, 3))
        sc = torch.where(amax > 0, amax / 448.0, torch.ones(()))
        codes = (vals / sc[:, :, None, None]).clamp(-448, 448).to(E4M3_FN).view(torch.uint8)
        codes = torch.where(live, codes, torch.full((), 0x7F, dtype=torch.uint8))
        out += [codes.numpy().copy(), sc.numpy().copy()]
    return out


def pin_append_fp8_fresh_page(lib):
    """A row that opens a page gets scale amax/448 and torch's codes of row/scale; K and V
    keep separate scales; nothing else changes."""
    rng = np.random.default_rng(22)
    P, Hkv, D = 16, 3, 64
    lengths = [1, 17, 33, 49, 1]
    c = _append_case(rng, lengths, Hkv, D, P, fp8=True)
    kc, ks, vc, vs = _fp8_pages_from(c, P)
    kp, vp, ks2, vs2 = oracle.kv_append(c["k_new"], c["v_new"], c["bt"], c["lengths"], kc, vc,
                                        k_scales=ks, v_scales=vs, lib=oracle.load(lib))
    for new, pages, scales, pages0, scales0, what in ((c["k_new"], kp, ks2, kc, ks, "K"),
                                                     (c["v_new"], vp, vs2, vc, vs, "V")):
        x = bits_f64(new).to(torch.float32)                           # [B, Hkv, D]
        amax = x.abs().amax(-1)
        sc = torch.where(amax > 0, amax / 448.0, torch.ones(())).numpy()
        want = torch_e4m3((x / torch.from_numpy(sc)[..., None]).numpy())
        mask = np.ones(pages.shape[:3], dtype=bool)
        for b, L in enumerate(lengths):
            pg = c["bt"][b, (L - 1) // P]
            assert np.array_equal(scales[pg], sc[b]), f"{what} scale of a fresh page"
            assert np.array_equal(pages[pg, :, 0, :], want[b]), f"{what} codes of a fresh page"
            mask[pg, :, 0] = False
        assert np.array_equal(pages[mask], pages0[mask]), f"{what}: other slots changed"


def pin_append_fp8_largest_first(lib):
    """Filling a page one row at a time, largest row first, never re-encodes: the result equals
    torch quantising the whole page with scale = page amax / 448."""
    rng = np.random.default_rng(23)
    P, Hkv, D = 16, 2, 32
    for trial in range(3):
        x = rng.standard_normal((P, Hkv, D)) * np.exp(-np.arange(P) * 0.15)[:, None, None]
        x[0] *= 3.0
        xb = bf16_bits(x)
        codes = np.full((1, Hkv, P, D), 0x7F, np.uint8)
        sc = np.ones((1, Hkv), np.float32)
        kc, vc, ks, vs = codes, codes.copy(), sc, sc.copy()
        bt = np.zeros((1, 1), np.int32)
        for t in range(P):
            kc, vc, ks, vs = oracle.kv_append(xb[t][None], xb[t][None], bt, np.array([t + 1], np.int32),
                                              kc, vc, k_scales=ks, v_scales=vs, lib=oracle.load(lib))
        vals = bits_f64(xb).to(torch.float32).permute(1, 0, 2)        # [Hkv, P, D]
        amax = vals.abs().amax(dim=(1, 2))
        want_sc = torch.where(amax > 0, amax / 448.0, torch.ones(()))
        want = torch_e4m3((vals / want_sc[:, None, None]).numpy())
        assert np.array_equal(ks[0], want_sc.numpy()), f"trial {trial}: page scale"
        assert np.array_equal(kc[0], want), f"trial {trial}: page codes"
        assert np.array_equal(vc, kc) and np.array_equal(vs, ks)


def pin_append_fp8_growing_rows(lib):
    """Rows of growing magnitude force a re-encode on every append: the final scale is the last
    row's amax/448 and every dequantised value stays within the rounding error of the encodes
    it went through (one half step of the 3-bit mantissa per encode, or half the smallest
    subnormal step at the final scale)."""
    rng = np.random.default_rng(24)
    P, D = 16, 64
    mags = 0.01 * 1.7 ** np.arange(P)
    x = rng.standard_normal((P, 1, D)) * mags[:, None, None]
    for t in range(P):
        x[t, 0, t % D] = 3.0 * mags[t] * (1 if t % 2 else -1)          # a clear maximum per row
    xb = bf16_bits(x)
    kc = np.full((1, 1, P, D), 0x7F, np.uint8)
    ks = np.ones((1, 1), np.float32)
    bt = np.zeros((1, 1), np.int32)
    for t in range(P):
        kc, _, ks, _ = oracle.kv_append(xb[t][None], xb[t][None], bt, np.array([t + 1], np.int32), kc,
                                        kc.copy(), k_scales=ks, v_scales=ks.copy(), lib=oracle.load(lib))
        s_t = np.float32(np.abs(bits_f64(xb[t]).numpy()).max()) / np.float32(448)
        assert ks[0, 0] == s_t, f"scale after row {t}: {ks[0, 0]} vs {s_t}"
    vals = bits_f64(xb).numpy()[:, 0, :]
    deq = np.array([[oracle.e4m3_to_double(c) for c in row] for row in kc[0, 0]]) * float(ks[0, 0])
    encodes = (P - np.arange(P))[:, None]                              # row t: 1 + (P-1-t) re-encodes
    bound = encodes * (2.0 ** -4 * np.abs(vals) * 1.001 + 2.0 ** -10 * float(ks[0, 0])) + 1e-30
    err = np.abs(deq - vals)
    assert np.all(err <= bound), f"re-encode error {np.max(err / bound):.3f} x bound"


def pin_golden_append(lib):
    """Hand-derived quantise-on-write steps in tests/golden/append_worked.json."""
    with open(os.path.join(GOLDEN, "append_worked.json")) as f:
        g = json.load(f)
    P, D = g["page_size"], g["head_dim"]
    kc = np.full((1, 1, P, D), 0x7F, np.uint8)
    vc = kc.copy()
    ks = np.ones((1, 1), np.float32)
    vs = ks.copy()
    bt = np.zeros((1, 1), np.int32)
    num = lambda v: np.array([float(x) for x in v], dtype=np.float32)
    for st in g["steps"]:
        kn = bf16_bits(num(st["k_new"]))[None, None]
        vn = bf16_bits(num(st["v_new"]))[None, None]
        assert np.array_equal(bits_f64(kn).numpy(), num(st["k_new"]).astype(np.float64)[None, None],
                              equal_nan=True), "fixture rows must be exact in bf16"
        kc, vc, ks, vs = oracle.kv_append(kn, vn, bt, np.array([st["seq_len"]], np.int32), kc, vc,
                                          k_scales=ks, v_scales=vs, lib=oracle.load(lib))
        n = st["seq_len"]
        assert np.array_equal(kc[0, 0, :n], np.array(st["k_codes"], np.uint8)), f"K codes at {n}"
        assert np.array_equal(vc[0, 0, :n], np.array(st["v_codes"], np.uint8)), f"V codes at {n}"
        assert ks[0, 0] == np.float32(st["k_scale"]) and vs[0, 0] == np.float32(st["v_scale"]), f"scales at {n}"


ALL_PINS = [
    pin_sdpa_random, pin_sdpa_large_scores, pin_prefix_sharing, pin_single_token,
    pin_identical_keys, pin_constant_values, pin_dominant_token, pin_page_permutation,
    pin_head_permutation, pin_zero_length, pin_rows_subset, pin_e4m3_table, pin_sdpa_fp8,
    pin_golden_hand_worked,
    pin_e4m3_encode_torch, pin_append_bf16_dense, pin_append_fp8_fresh_page,
    pin_append_fp8_largest_first, pin_append_fp8_growing_rows, pin_golden_append,
]
