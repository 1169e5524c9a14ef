"""GPU path (libsl through the C ABI) against the fp64 oracle and the attention invariants."""
import numpy as np
import pytest
import torch

from paper_2504_15930_amd import inputs, sl
from parity import assert_parity, oracle_full, oracle_rows, sample_rows
import oracle_pins

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")]
DEV = "cuda:0"


def _bits(t):
    return t.detach().cpu().view(torch.int16)


def _say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_workload(seed):
    _say("tiny workload seed", seed)
    b = inputs.make_batch("tiny", seed=seed, device=DEV)
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    assert_parity(out, oracle_full(b), f"tiny seed {seed}")


SHAPES = [
    # (B, Hq, Hkv, D, lengths or (lo, hi) for seeded-uniform)
    (1, 8, 1, 128, [1]),
    (3, 8, 2, 64, [15, 16, 17]),
    (5, 28, 4, 128, [1, 33, 100, 16, 250]),
    (17, 16, 16, 64, (1, 300)),       # G = 1
    (33, 40, 8, 128, (1, 500)),       # G = 5
    (9, 14, 2, 64, (1, 200)),         # G = 7
    (6, 32, 2, 128, (1, 400)),        # G = 16
    (4, 64, 8, 128, [1000, 2000, 17, 3000]),
    (4, 4, 4, 128, [0, 5, 0, 32]),    # empty sequences
]


def _lengths(spec, B, seed):
    if isinstance(spec, tuple):
        lo, hi = spec
        return np.random.default_rng(seed).integers(lo, hi + 1, B)
    return np.array(spec)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"B{s[0]}_Hq{s[1]}_Hkv{s[2]}_D{s[3]}")
@pytest.mark.parametrize("workers", [0, 1, 7, 1000])
@pytest.mark.parametrize("kv", ["bf16", "e4m3"])
def test_random_shapes(shape, workers, kv):
    B, Hq, Hkv, D, spec = shape
    L = _lengths(spec, B, seed=B * 31 + D)
    _say("random shape", shape, "workers", workers, kv)
    b = inputs.make_paged_batch(L, Hq, Hkv, D, seed=B + Hq, device=DEV, kv_dtype=kv)
    out = sl.run_batch(b, num_workers=workers)
    torch.cuda.synchronize()
    assert_parity(out, oracle_full(b), f"{shape} workers={workers} {kv}")


def _sweep_case(i):
    """Configuration i of the seeded sweep: head layout, head size, batch, a length mix with the
    edge values (0, 1, 15, 16, 17, whole pages, long tails), worker count and cache type."""
    rng = np.random.default_rng(1000 + i)
    D = int(rng.choice([64, 128]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 16]))
    B = int(rng.choice([1, 2, 3, 8, 31, 64, 130, 257]))
    kind = rng.integers(0, 4, B)   # 0: edge value, 1: short, 2: lognormal tail, 3: whole pages
    L = np.where(kind == 0, rng.choice([0, 1, 15, 16, 17, 31, 32, 33], B),
         np.where(kind == 1, rng.integers(1, 64, B),
         np.where(kind == 2, np.minimum(np.exp(rng.normal(np.log(300), 1.2, B)).astype(np.int64) + 1, 6000),
                  16 * rng.integers(1, 40, B))))
    workers = int(rng.choice([0, 0, 1, 2, 5, 33, 256, 1000]))
    kv = str(rng.choice(["bf16", "e4m3"]))
    return L.astype(np.int64), G * Hkv, Hkv, D, workers, kv


@pytest.mark.parametrize("i", range(40))
def test_seeded_sweep(i):
    L, Hq, Hkv, D, workers, kv = _sweep_case(i)
    what = f"sweep {i}: B={len(L)} Hq={Hq} Hkv={Hkv} D={D} workers={workers} {kv} total={int(L.sum())}"
    _say(what)
    b = inputs.make_paged_batch(L, Hq, Hkv, D, seed=2000 + i, device=DEV, kv_dtype=kv)
    out = sl.run_batch(b, num_workers=workers)
    torch.cuda.synchronize()
    assert_parity(out, oracle_full(b), what)


@pytest.mark.parametrize("workers", [1, 3, 16, 97, 1000, 0])
def test_sparse_batch_with_empty_runs(workers):
    """Mostly empty sequences, including the first and the last, with the non-empty ones far apart:
    every worker locates its first tile by binary search over runs of equal page prefix sums and
    walks across the empty sequences between units."""
    _say("sparse batch workers", workers)
    L = np.zeros(64, np.int64)
    L[[5, 6, 31, 47, 62]] = [33, 1, 700, 16, 257]
    b = inputs.make_paged_batch(L, 28, 4, 128, seed=11, device=DEV)
    out = sl.run_batch(b, num_workers=workers)
    torch.cuda.synchronize()
    assert_parity(out, oracle_full(b), f"sparse workers={workers}")


@pytest.mark.parametrize("workers", [1, 2, 3, 7, 16, 64, 1000, 0])
def test_worker_count_independence(workers):
    _say("worker count", workers)
    b = inputs.make_paged_batch([700, 5, 1300, 64, 17], 16, 2, 128, seed=7, device=DEV)
    ref = oracle_full(b)
    out = sl.run_batch(b, num_workers=workers)
    torch.cuda.synchronize()
    assert_parity(out, ref, f"workers={workers}")


def test_back_to_back_calls_share_the_workspace():
    """Partial states of one call must never leak into the next (same shapes, new values)."""
    _say("back to back calls")
    a = inputs.make_paged_batch([900, 40, 1500, 333], 16, 2, 128, seed=21, device=DEV)
    b = inputs.make_paged_batch([900, 40, 1500, 333], 16, 2, 128, seed=22, device=DEV)
    ra, rb = oracle_full(a), oracle_full(b)
    for workers in (0, 7, 64, 0):
        for _ in range(3):
            oa = sl.run_batch(a, num_workers=workers)
            ob = sl.run_batch(b, num_workers=workers)
        torch.cuda.synchronize()
        assert_parity(oa, ra, f"first of pair, workers={workers}")
        assert_parity(ob, rb, f"second of pair, workers={workers}")


@pytest.mark.parametrize("kv", ["bf16", "e4m3"])
def test_single_token_returns_value_row_exactly(kv):
    _say("single token", kv)
    b = inputs.make_paged_batch([1] * 6, 8, 2, 128, seed=3, device=DEV, kv_dtype=kv)
    if kv == "e4m3":
        # bf16-exact value scales: the probability (1) times the scale is then exact in bf16
        b.v_scales = b.v_scales.to(torch.bfloat16).float()
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    bt = b.block_table.cpu().numpy()
    for s in range(6):
        for h in range(8):
            g = h // 4
            if kv == "bf16":
                want = b.v_pages[bt[s, 0], g, 0]
            else:
                want = (b.v_pages[bt[s, 0], g, 0].view(torch.float8_e4m3fn).float()
                        * b.v_scales[bt[s, 0], g]).to(torch.bfloat16)
            assert torch.equal(_bits(out[s, h]), _bits(want)), (s, h)


def test_constant_values_come_back_unchanged():
    _say("constant values")
    b = inputs.make_paged_batch([1, 17, 300, 4000], 28, 4, 128, seed=4, device=DEV)
    b.v_pages = torch.where(torch.isnan(b.v_pages), b.v_pages, torch.ones((), dtype=torch.bfloat16,
                                                                           device=DEV))
    for workers in (0, 3):
        out = sl.run_batch(b, num_workers=workers)
        torch.cuda.synchronize()
        assert torch.equal(out.float().cpu(), torch.ones(out.shape)), workers


@pytest.mark.parametrize("D", [64, 128])
def test_dominant_token_bit_exact_at_every_position(D):
    """Score gap 256 makes every other weight underflow to 0: out is that token's V row."""
    _say("dominant token D", D)
    B, Hq, Hkv, P = 3, 8, 2, 16
    lengths = np.array([40, 17, 33], dtype=np.int32)
    Lmax = int(lengths.max())
    v_log = np.zeros((B, Lmax, Hkv, D), dtype=np.float32)
    for s in range(B):
        for t in range(Lmax):
            for g in range(Hkv):
                v_log[s, t, g] = (s * 16 + t) % 50 + g / 2.0 + (np.arange(D) % 3) * 0.25
    v_bits = oracle_pins.bf16_bits(v_log)
    q = np.zeros((B, Hq, D), dtype=np.float32)
    q[:, :, 0] = 16.0
    q_bits = torch.from_numpy(oracle_pins.bf16_bits(q).view(np.int16)).view(torch.bfloat16).to(DEV)
    rng = np.random.default_rng(0)
    for t in range(Lmax):
        k_log = np.zeros((B, Lmax, Hkv, D), dtype=np.float32)
        k_log[:, t, :, 0] = 16.0
        k_bits = oracle_pins.bf16_bits(k_log)
        k_pages, table = oracle_pins.scatter_pages(k_bits, lengths, P, rng, oracle_pins.BF16_NAN)
        v_pages, _ = oracle_pins.scatter_pages(v_bits, lengths, P, rng, oracle_pins.BF16_NAN,
                                               table=table, num_pages=k_pages.shape[0])
        tb = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(DEV)
        for workers in (0, 5):
            out = sl.decode_attn(q_bits, tb(k_pages), tb(v_pages), torch.from_numpy(table).to(DEV),
                                 torch.from_numpy(lengths).to(DEV), 1.0, num_workers=workers)
            torch.cuda.synchronize()
            for s in range(B):
                if t >= lengths[s]:
                    continue
                want = torch.from_numpy(v_bits[s, t].view(np.int16))       # [Hkv, D]
                got = _bits(out[s]).reshape(Hkv, Hq // Hkv, D)
                assert torch.equal(got, want[:, None, :].expand_as(got)), (t, s, workers)


def test_page_permutation_is_bit_exact():
    _say("page permutation")
    b = inputs.make_paged_batch([3, 700, 16, 33, 1500], 28, 4, 128, seed=8, device=DEV)
    base = sl.run_batch(b).clone()
    N = b.k_pages.shape[0]
    perm = torch.randperm(N, generator=torch.Generator().manual_seed(1)).to(DEV)
    k2 = torch.empty_like(b.k_pages)
    v2 = torch.empty_like(b.v_pages)
    k2[perm] = b.k_pages
    v2[perm] = b.v_pages
    bt2 = perm[b.block_table.long()].int()
    out = sl.decode_attn(b.q, k2, v2, bt2, b.seq_lens, b.scale)
    torch.cuda.synchronize()
    assert torch.equal(_bits(out), _bits(base))


def test_prefix_sharing_aliased_pages():
    _say("prefix sharing")
    P = 16
    table = np.array([[0, 1, 2, 3, 10],
                      [0, 1, 4, 5, 10],     # shares two pages with sequence 0
                      [0, 1, 2, 3, 10],     # aliases every page of sequence 0
                      [6, 7, 8, 9, 10]], dtype=np.int32)
    lengths = np.array([60, 50, 60, 64], dtype=np.int32)
    b = inputs.make_paged_batch(lengths, 8, 2, 128, seed=9, device=DEV, block_table=table,
                                num_pages=11)
    b.q[2] = b.q[0]
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    assert_parity(out, oracle_full(b), "prefix sharing")
    assert torch.equal(_bits(out[0]), _bits(out[2]))


def test_zero_length_rows_are_zero():
    _say("zero lengths")
    b = inputs.make_paged_batch([0, 0, 0], 8, 2, 64, seed=10, device=DEV)
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    assert torch.equal(out.float().cpu(), torch.zeros(out.shape))


def test_invalid_device_data_gives_nan_rows_not_faults():
    _say("invalid device data")
    b = inputs.make_paged_batch([40, 20, 33, 18], 8, 2, 128, seed=11, device=DEV)
    N = b.k_pages.shape[0]
    bt = b.block_table.clone()
    lens = b.seq_lens.clone()
    bt[0, 1] = N + 5            # page id past the pool
    bt[3, 0] = -2               # negative page id
    lens[1] = 16 * bt.shape[1] + 1   # longer than the block table allows
    lens[2] = -4                # negative length
    for workers in (0, 3):
        out = sl.decode_attn(b.q, b.k_pages, b.v_pages, bt, lens, b.scale, num_workers=workers)
        torch.cuda.synchronize()
        assert torch.isnan(out.float()).all(), workers


def test_max_batch_short_sequences():
    _say("max batch 8192")
    L = np.random.default_rng(12).integers(1, 65, 8192)
    b = inputs.make_paged_batch(L, 8, 2, 64, seed=12, device=DEV)
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    rows = sample_rows(b.seq_lens, 64)
    assert_parity(out[rows], oracle_rows(b, rows), "batch 8192")


def test_fp8_every_code_decodes_exactly():
    """One dominant token whose value row holds every E4M3 code; unit value scale."""
    _say("fp8 code coverage")
    D, Hq, Hkv = 128, 4, 2
    codes = np.arange(256, dtype=np.uint8)
    live_codes = codes[(codes & 0x7F) != 0x7F]                 # 254 finite codes
    rows = [live_codes[i:i + D] for i in range(0, len(live_codes), D)]
    rows[-1] = np.concatenate([rows[-1], np.zeros(D - len(rows[-1]), np.uint8)])
    for r, vrow in enumerate(rows):
        L = 20
        lengths = np.array([L], dtype=np.int32)
        k_codes = np.zeros((1, L, Hkv, D), np.uint8)
        k_codes[0, 7, :, 0] = 0x70                             # 2^7 = 128: score gap 128*16
        v_codes = np.full((1, L, Hkv, D), 0x38, np.uint8)      # 1.0 elsewhere
        v_codes[0, 7, :, :] = vrow
        rng = np.random.default_rng(r)
        kp, table = oracle_pins.scatter_pages(k_codes, lengths, 16, rng, np.uint8(0x7F))
        vp, _ = oracle_pins.scatter_pages(v_codes, lengths, 16, rng, np.uint8(0x7F), table=table,
                                          num_pages=kp.shape[0])
        q = torch.zeros(1, Hq, D, dtype=torch.bfloat16, device=DEV)
        q[:, :, 0] = 16.0
        ones = torch.ones(kp.shape[0], Hkv, dtype=torch.float32, device=DEV)
        out = sl.decode_attn_fp8(q, torch.from_numpy(kp).to(DEV), torch.from_numpy(vp).to(DEV),
                                 ones, ones, torch.from_numpy(table).to(DEV),
                                 torch.from_numpy(lengths).to(DEV), 1.0)
        torch.cuda.synchronize()
        # exact values (-0 and +0 compare equal: the sum of +0 weights times -0 is +0)
        want = torch.from_numpy(vrow).view(torch.float8_e4m3fn).to(torch.float32)
        for h in range(Hq):
            assert torch.equal(out[0, h].float().cpu(), want), (r, h)
            assert torch.equal(out[0, h].float().cpu(), want.to(torch.bfloat16).float()), (r, h)


@pytest.mark.parametrize("name", ["qwen7b_longtail", "straggler", "qwen72b_longtail",
                                  "fp8_qwen7b_longtail"])
def test_full_workload_sampled_rows(name):
    """Full-size decode step in the default launch configuration; 24 sampled sequences
    (always the longest and the shortest) checked against the oracle."""
    _say("full workload", name)
    b = inputs.make_batch(name, seed=0, device=DEV)
    out = sl.run_batch(b)
    torch.cuda.synchronize()
    rows = sample_rows(b.seq_lens, 24)
    assert_parity(out[rows], oracle_rows(b, rows), name)
    assert torch.isfinite(out.float()).all()
    del b
    torch.cuda.empty_cache()
