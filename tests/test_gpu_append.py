"""GPU parity of the KV append step (sl_kv_append / sl_kv_append_fp8) against the oracle.

Everything here is integer or byte work decided in binary32 on both sides, so
the bar is bit-exact: pages (all bytes, untouched slots included) and scales
must equal the oracle's. The chain test then runs attention over the appended
cache and compares it with the oracle to the bf16 attention tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import oracle_pins as pins
import parity
from paper_2504_15930_amd import inputs, sl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _bf16(bits):
    return _dev(np.asarray(bits, np.uint16).view(np.int16)).view(torch.bfloat16)


def _u16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def gpu_append(k_new, v_new, bt, lens, kp, vp, ks=None, vs=None, num_q_heads=None):
    """Run the library's append on device copies; returns host arrays."""
    fp8 = kp.dtype == np.uint8
    Kp = _dev(kp) if fp8 else _bf16(kp)
    Vp = _dev(vp) if fp8 else _bf16(vp)
    Ks = _dev(ks) if fp8 else None
    Vs = _dev(vs) if fp8 else None
    sl.kv_append(_bf16(k_new), _bf16(v_new), _dev(bt), _dev(lens), Kp, Vp, k_scales=Ks, v_scales=Vs,
                 num_q_heads=num_q_heads)
    torch.cuda.synchronize()
    if fp8:
        return Kp.cpu().numpy(), Vp.cpu().numpy(), Ks.cpu().numpy(), Vs.cpu().numpy()
    return _u16(Kp), _u16(Vp)


def assert_same(got, want, what):
    for i, (g, w) in enumerate(zip(got, want)):
        g = np.asarray(g)
        w = np.asarray(w)
        if g.dtype == np.float32:
            g, w = g.view(np.uint32), w.view(np.uint32)
        bad = np.argwhere(g != w)
        assert bad.size == 0, f"{what}: array {i} differs at {bad[:4].tolist()} ({g[tuple(bad[0])]} vs {w[tuple(bad[0])]})"


def test_encoder_every_bf16_value():
    """Every bf16 value in [-448, 448] (and NaN) through the fresh-page path with scale 1."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = pins.bits_f64(bits).numpy()
    keep = np.isnan(vals) | (np.abs(vals) <= 448.0)
    bits = bits[keep]
    D = 128
    per = D - 1
    rows = -(-bits.size // per)
    x = np.zeros((rows, D), np.uint16)
    x[:, 0] = pins.bf16_bits(np.float32(448.0))                       # amax 448 -> scale exactly 1
    flat = np.zeros(rows * per, np.uint16)
    flat[:bits.size] = bits
    x[:, 1:] = flat.reshape(rows, per)
    B = rows
    k_new = x[:, None, :]
    v_new = x[::-1][:, None, :].copy()
    bt = np.arange(B, dtype=np.int32)[:, None]
    lens = np.ones(B, np.int32)
    kp = np.full((B, 1, 16, D), 0x7F, np.uint8)
    sc = np.full((B, 1), 7.0, np.float32)
    got = gpu_append(k_new, v_new, bt, lens, kp, kp.copy(), sc, sc.copy())
    want = oracle.kv_append(k_new, v_new, bt, lens, kp, kp.copy(), k_scales=sc, v_scales=sc.copy())
    assert_same(got, want, "every bf16 value")
    assert np.all(got[2] == 1.0)


CASES = [
    # (lengths, Hkv, D)
    ([1, 2, 15, 16, 17, 31, 32, 33, 100, 0, 5], 2, 128),
    ([1, 16, 17, 3, 48, 49, 7], 4, 64),
    ([200, 1, 33, 17], 1, 128),
]


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "e4m3"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_append_random(case, fp8):
    lengths, Hkv, D = CASES[case]
    rng = np.random.default_rng(100 + case)
    c = pins._append_case(rng, lengths, Hkv, D, 16, fp8)
    if fp8:
        kc, ks, vc, vs = pins._fp8_pages_from(c, 16)
        # grow some new rows past their page's scale, shrink others
        mult = rng.choice([0.1, 1.0, 5.0, 40.0], size=(len(lengths), 1, 1))
        k_new = pins.bf16_bits(pins.bits_f64(c["k_new"]).numpy() * mult)
        v_new = pins.bf16_bits(pins.bits_f64(c["v_new"]).numpy() * mult[::-1])
        got = gpu_append(k_new, v_new, c["bt"], c["lengths"], kc, vc, ks, vs)
        want = oracle.kv_append(k_new, v_new, c["bt"], c["lengths"], kc, vc, k_scales=ks, v_scales=vs)
    else:
        got = gpu_append(c["k_new"], c["v_new"], c["bt"], c["lengths"], c["k_pages"], c["v_pages"])
        want = oracle.kv_append(c["k_new"], c["v_new"], c["bt"], c["lengths"], c["k_pages"], c["v_pages"])
    assert_same(got, want, f"case {case}")


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "e4m3"])
def test_append_chain_then_attend(fp8):
    """40 decode steps of appends from empty pages, bit-exact after every step; then attention
    over the appended cache against the oracle."""
    rng = np.random.default_rng(7)
    B, Hkv, G, D, steps = 6, 2, 4, 128, 40
    start = np.array([0, 1, 15, 16, 30, 5], np.int32)
    max_blocks = (int(start.max()) + steps) // 16 + 1
    N = B * max_blocks + 2
    bt = rng.permutation(N)[:B * max_blocks].astype(np.int32).reshape(B, max_blocks)
    if fp8:
        kp = np.full((N, Hkv, 16, D), 0x7F, np.uint8)
        ks = np.ones((N, Hkv), np.float32)
        state = [kp, kp.copy(), ks, ks.copy()]
    else:
        kp = np.full((N, Hkv, 16, D), pins.BF16_NAN, np.uint16)
        state = [kp, kp.copy()]
    # every token of every sequence is appended one step at a time, from empty
    lens = np.zeros(B, np.int32)
    for step in range(int(start.max()) + steps):
        active = lens < start + steps
        new_lens = np.where(active, lens + 1, lens)
        step_lens = np.where(active, new_lens, 0).astype(np.int32)    # L = 0: no append this step
        mag = np.exp(rng.uniform(-3, 3, (B, Hkv, 1)))
        k_new = pins.bf16_bits(rng.standard_normal((B, Hkv, D)) * mag)
        v_new = pins.bf16_bits(rng.standard_normal((B, Hkv, D)) * mag[::-1])
        want = oracle.kv_append(k_new, v_new, bt, step_lens, *state[:2],
                                **(dict(k_scales=state[2], v_scales=state[3]) if fp8 else {}))
        got = gpu_append(k_new, v_new, bt, step_lens, *state)
        assert_same(got, want, f"step {step}")
        state = list(want)
        lens = new_lens
    q = pins.bf16_bits(rng.standard_normal((B, Hkv * G, D)))
    scale = float(np.float32(1 / np.sqrt(D)))
    ref = oracle.decode_attn(q, state[0], state[1], bt, lens, scale,
                             **(dict(k_scales=state[2], v_scales=state[3]) if fp8 else {}))
    if fp8:
        out = sl.decode_attn_fp8(_bf16(q), _dev(state[0]), _dev(state[1]), _dev(state[2]), _dev(state[3]),
                                 _dev(bt), _dev(lens), scale)
    else:
        out = sl.decode_attn(_bf16(q), _bf16(state[0]), _bf16(state[1]), _dev(bt), _dev(lens), scale)
    torch.cuda.synchronize()
    # Values were drawn at scales e^-3 .. e^3 (to drive the E4M3 scales up and down), so the
    # absolute bound is taken at each row's value scale.
    if fp8:
        v64 = torch.from_numpy(state[1]).view(torch.float8_e4m3fn).double().numpy() * state[3][:, :, None, None]
    else:
        v64 = pins.bits_f64(state[1]).numpy()
    parity.assert_parity(out, ref, "attention over appended cache",
                         value_scale=parity.value_rms_rows(v64, bt, lens, Hkv * G))


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "e4m3"])
def test_append_edge_cases(fp8):
    """Empty, negative and too-long lengths and out-of-pool pages leave the cache untouched;
    NaN, inf and all-zero rows follow the oracle bit for bit."""
    rng = np.random.default_rng(9)
    Hkv, D, N, mb = 2, 128, 12, 2
    lens = np.array([0, -3, 40, 5, 17, 1, 2, 9], np.int32)          # 40 > mb * 16
    B = len(lens)
    # receiving pages: row 3 -> 99 (outside the pool), row 4 -> 8, row 5 -> 9, row 6 -> -1, row 7 -> 11
    bt = np.array([[0, 1], [2, 3], [4, 5], [99, 6], [7, 8], [9, 10], [-1, 11], [11, 10]], np.int32)
    k_new = pins.bf16_bits(rng.standard_normal((B, Hkv, D)))
    v_new = pins.bf16_bits(rng.standard_normal((B, Hkv, D)))
    k_new[4, 0, 3] = pins.bf16_bits(np.float32(np.nan))
    k_new[4, 1, :] = pins.bf16_bits(np.float32(np.nan))               # all-NaN row
    v_new[5, 0, :] = 0                                                # all-zero row on a fresh page
    k_new[7, 1, 5] = pins.bf16_bits(np.float32(np.inf))
    if fp8:
        kp = rng.integers(0, 0x7E, (N, Hkv, 16, D), dtype=np.uint8)
        ks = rng.uniform(0.01, 0.1, (N, Hkv)).astype(np.float32)
        base = [kp, kp.copy(), ks, ks.copy()]
    else:
        kp = pins.bf16_bits(rng.standard_normal((N, Hkv, 16, D)))
        base = [kp, kp.copy()]
    got = gpu_append(k_new, v_new, bt, lens, *base)
    # the oracle rejects invalid rows, so it runs on the valid ones only
    valid = (lens >= 1) & (lens <= mb * 16)
    ok = np.array([valid[b] and 0 <= bt[b, (lens[b] - 1) // 16] < N for b in range(B)])
    keep_lens = np.where(ok, lens, 0).astype(np.int32)
    want = oracle.kv_append(k_new, v_new, np.where(bt < 0, 0, np.minimum(bt, N - 1)).astype(np.int32),
                            keep_lens, *base[:2], **(dict(k_scales=base[2], v_scales=base[3]) if fp8 else {}))
    assert_same(got, want, "edge cases")


@pytest.mark.parametrize("name", ["qwen7b_longtail", "fp8_qwen7b_longtail"])
def test_append_full_workload(name):
    """One append over a full-size batch; the receiving tiles of sampled sequences (the
    longest and shortest included) match the oracle run on just those tiles."""
    b = inputs.make_batch(name, seed=0, device=DEV)
    torch.cuda.synchronize()
    B, Hq, D = b.q.shape
    Hkv = b.k_pages.shape[1]
    fp8 = b.kv_dtype == "e4m3"
    gen = torch.Generator(device=DEV).manual_seed(5)
    k_new = (torch.randn((B, Hkv, D), generator=gen, device=DEV) * 3).to(torch.bfloat16)
    v_new = (torch.randn((B, Hkv, D), generator=gen, device=DEV) * 0.5).to(torch.bfloat16)
    lens = b.seq_lens.cpu().numpy()
    rows = parity.sample_rows(lens, 24)
    pages = torch.tensor([int(b.block_table[r, (lens[r] - 1) // 16]) for r in rows], device=DEV)
    before = [b.k_pages.index_select(0, pages).cpu(), b.v_pages.index_select(0, pages).cpu()]
    if fp8:
        before += [b.k_scales.index_select(0, pages).cpu(), b.v_scales.index_select(0, pages).cpu()]
    sl.kv_append(k_new, v_new, b.block_table, b.seq_lens, b.k_pages, b.v_pages,
                 k_scales=b.k_scales if fp8 else None, v_scales=b.v_scales if fp8 else None, num_q_heads=Hq)
    torch.cuda.synchronize()
    if fp8:
        after = [b.k_pages.index_select(0, pages).cpu().numpy(), b.v_pages.index_select(0, pages).cpu().numpy(),
                 b.k_scales.index_select(0, pages).cpu().numpy(), b.v_scales.index_select(0, pages).cpu().numpy()]
    else:
        after = [_u16(b.k_pages.index_select(0, pages)), _u16(b.v_pages.index_select(0, pages))]
    # mini problem: sequence i of the sample owns mini page i
    n = len(rows)
    L = lens[rows].astype(np.int32)
    mb = int(((L - 1) // 16).max()) + 1
    bt = np.zeros((n, mb), np.int32)
    bt[np.arange(n), (L - 1) // 16] = np.arange(n)
    kn = _u16(k_new)[rows]
    vn = _u16(v_new)[rows]
    if fp8:
        want = oracle.kv_append(kn, vn, bt, L, before[0].numpy(), before[1].numpy(),
                                k_scales=before[2].numpy(), v_scales=before[3].numpy())
    else:
        want = oracle.kv_append(kn, vn, bt, L, before[0].view(torch.int16).numpy().view(np.uint16),
                                before[1].view(torch.int16).numpy().view(np.uint16))
    assert_same(after, want, name)
