"""GPU parity of prefix-shared decode attention (sl_decode_attn_prefix) against the oracle.

Sharing pages changes how often a page is read, not the result: every output
row must match the attention oracle (the same definition as sl_decode_attn) to
the bf16 tolerance. Batches are GRPO-like: several samples of one prompt share
the prompt's full pages and continue on pages of their own.
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


def grpo_layout(rng, members, prompts, gen_max, extra=0):
    """Groups of `members[k]` sequences whose first floor(prompts[k] / 16) pages are the same
    page ids (and tokens); each member continues with `gen` tokens on pages of its own; `extra`
    unshared sequences follow. Returns (lengths, block table, pool size, group_start,
    shared_pages)."""
    lengths, starts, shared = [], [0], []
    for m, p in zip(members, prompts):
        lengths += [p + int(g) for g in rng.integers(0, gen_max + 1, m)]
        starts.append(starts[-1] + m)
        shared.append(p // 16)
    lengths += [int(x) for x in rng.integers(1, 300, extra)]
    B = len(lengths)
    mb = max(-(-L // 16) for L in lengths) + 1
    N = B * mb + 8
    perm = list(rng.permutation(N))
    table = np.zeros((B, mb), np.int32)
    for k, m in enumerate(members):
        sp = shared[k]
        common = [perm.pop() for _ in range(sp)]
        for b in range(starts[k], starts[k] + m):
            table[b, :sp] = common
            for i in range(sp, mb):
                table[b, i] = perm.pop()
    for b in range(starts[-1], B):
        for i in range(mb):
            table[b, i] = perm.pop()
    return lengths, table, N, np.array(starts, np.int32), np.array(shared, np.int32)


def grpo_case(rng, members, prompts, gen_max, Hq, Hkv, D, extra=0):
    """A bf16 oracle case over grpo_layout's groups."""
    lengths, table, N, starts, shared = grpo_layout(rng, members, prompts, gen_max, extra)
    case, dense = pins.random_case(rng, len(lengths), Hq, Hkv, D, 16, lengths, table=table)
    return case, starts, shared


def grpo_fp8_batch(rng, members, prompts, gen_max, Hq, Hkv, D, extra=0, seed=0):
    """An E4M3 device batch over grpo_layout's groups (codes and per-(page, KV head) scales)."""
    lengths, table, N, starts, shared = grpo_layout(rng, members, prompts, gen_max, extra)
    b = inputs.make_paged_batch(np.array(lengths), Hq, Hkv, D, seed=seed, device=DEV, kv_dtype="e4m3",
                                block_table=table, num_pages=N)
    return b, torch.from_numpy(starts).to(DEV), torch.from_numpy(shared).to(DEV)


def run_prefix_fp8(b, starts, shared, num_workers=0):
    out = sl.decode_attn_prefix_fp8(b.q, b.k_pages, b.v_pages, b.k_scales, b.v_scales, b.block_table, b.seq_lens,
                                    b.scale, starts, shared, num_workers=num_workers)
    torch.cuda.synchronize()
    return out


def _bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def run_prefix(case, starts, shared, num_workers=0):
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = sl.decode_attn_prefix(_bf16(case["q"]), _bf16(case["k_pages"]), _bf16(case["v_pages"]),
                                d(case["block_table"]), d(case["seq_lens"]), case["scale"], d(starts), d(shared),
                                num_workers=num_workers)
    torch.cuda.synchronize()
    return out


CASES = [
    # members, prompt lengths, max generated, Hq, Hkv, D, extra unshared sequences
    ([8, 8, 1, 9], [100, 512, 40, 17], 200, 28, 4, 128, 3),
    ([16, 3, 2], [64, 160, 300], 50, 16, 4, 64, 0),
    ([4, 4], [1000, 33], 0, 8, 8, 128, 2),          # nothing generated: some contexts are all shared
    ([2], [16], 5, 64, 8, 128, 1),                   # G = 8, one shared page
]


@pytest.mark.parametrize("case_id", range(len(CASES)))
@pytest.mark.parametrize("workers", [0, 1, 7, 1000])
def test_prefix_matches_oracle(case_id, workers):
    members, prompts, gen, Hq, Hkv, D, extra = CASES[case_id]
    rng = np.random.default_rng(40 + case_id)
    case, starts, shared = grpo_case(rng, members, prompts, gen, Hq, Hkv, D, extra)
    out = run_prefix(case, starts, shared, workers)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, f"case {case_id} workers {workers}")


def test_no_groups_is_plain_attention():
    rng = np.random.default_rng(50)
    case, _, _ = grpo_case(rng, [3], [70], 30, 28, 4, 128, extra=4)
    out = run_prefix(case, np.zeros(1, np.int32), np.zeros(0, np.int32))
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "no groups")


def test_oversized_and_zero_share_groups_stay_exact():
    """A group with more members than fit the 64 query rows (read as sub-groups), and groups
    sharing no page (attended without sharing), stay exact."""
    rng = np.random.default_rng(51)
    case, starts, shared = grpo_case(rng, [10, 3, 2], [48, 33, 5], 40, 28, 4, 128)   # 10 * 7 = 70 > 64 rows
    out = run_prefix(case, starts, shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "oversized group")


def test_member_shorter_than_shared_prefix_gets_nan():
    """A group whose page count fits the block table but exceeds its members' lengths: NaN rows
    for the members (an invalid request), exact rows for everyone else."""
    rng = np.random.default_rng(52)
    case, starts, shared = grpo_case(rng, [4, 2], [64, 32], 20, 28, 4, 128)
    shared = shared.copy()
    mb = case["block_table"].shape[1]               # one more than any sequence's page count
    assert (case["seq_lens"][:4] < 16 * mb).all()
    shared[0] = mb                                  # in bounds, but longer than every member
    out = run_prefix(case, starts, shared).float().cpu().numpy()
    assert np.isnan(out[:4]).all()
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(torch.from_numpy(out[4:]).to(torch.bfloat16), ref[4:], "other group")


def test_full_size_grpo_batch():
    """32 prompts x 8 samples, 7B-like heads, 1024-token prompts (64 shared pages), generated
    lengths lognormal (median 512, capped at 4096): sampled rows against the oracle."""
    b, starts, shared = inputs.make_grpo_batch(32, 8, 1024, seed=3, device=DEV)
    torch.cuda.synchronize()
    out = sl.decode_attn_prefix(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale, starts, shared)
    torch.cuda.synchronize()
    rows = parity.sample_rows(b.seq_lens.cpu().numpy(), 24)
    parity.assert_parity(out[rows], parity.oracle_rows(b, rows), "grpo")
    plain = sl.run_batch(b)
    torch.cuda.synchronize()
    parity.assert_parity(out[rows], parity.oracle_rows(b, rows), "grpo")
    assert (out.float() - plain.float()).abs().max().item() < 0.05


def test_page_count_beyond_block_table_is_unshared():
    """A shared page count larger than the block table's width is out of bounds: that group is
    attended without sharing, exactly."""
    rng = np.random.default_rng(53)
    case, starts, shared = grpo_case(rng, [4, 3], [64, 40], 20, 28, 4, 128)
    shared = shared.copy()
    shared[0] = case["block_table"].shape[1] + 1
    out = run_prefix(case, starts, shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "page count beyond the table")


def test_max_prefix_batch_many_groups():
    """The largest batch prefix sharing accepts (4096 sequences), in 2048 groups of two: every
    workgroup keeps 3 B + 2 NG + 2 ints of stream description in LDS, and the shared-page
    stream crosses a group boundary every few tiles. Every row against the oracle."""
    rng = np.random.default_rng(54)
    ng = 2048
    case, starts, shared = grpo_case(rng, [2] * ng, list(rng.integers(16, 49, ng)), 40, 8, 2, 64)
    assert len(case["seq_lens"]) == 4096
    out = run_prefix(case, starts, shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "batch 4096, 2048 groups")


def _prefix_sweep_case(i):
    """Configuration i of the seeded prefix sweep: head layout, group sizes (some too large to
    share), prompt lengths (some under one page), generated lengths, extra unshared sequences and
    worker count."""
    rng = np.random.default_rng(3000 + i)
    D = int(rng.choice([64, 128]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 7, 8]))
    ng = int(rng.integers(1, 9))
    members = [int(rng.choice([1, 2, 3, 5, 8, 16, 20])) for _ in range(ng)]
    prompts = [int(rng.choice([5, 16, 40, 100, 256, 700])) for _ in range(ng)]
    gen = int(rng.choice([0, 20, 200]))
    extra = int(rng.integers(0, 4))
    workers = int(rng.choice([0, 0, 1, 7, 100, 1000]))
    return members, prompts, gen, G * Hkv, Hkv, D, extra, workers


@pytest.mark.parametrize("i", range(16))
def test_prefix_seeded_sweep(i):
    members, prompts, gen, Hq, Hkv, D, extra, workers = _prefix_sweep_case(i)
    what = f"prefix sweep {i}: members={members} prompts={prompts} gen<={gen} Hq={Hq} Hkv={Hkv} D={D} " \
           f"extra={extra} workers={workers}"
    print(what, flush=True)
    rng = np.random.default_rng(4000 + i)
    case, starts, shared = grpo_case(rng, members, prompts, gen, Hq, Hkv, D, extra)
    out = run_prefix(case, starts, shared, workers)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, what)


@pytest.mark.parametrize("case_id", range(len(CASES)))
@pytest.mark.parametrize("workers", [0, 1, 7, 1000])
def test_prefix_fp8_matches_oracle(case_id, workers):
    """sl_decode_attn_prefix_fp8: E4M3 pages with per-(page, KV head) scales, every row against
    the oracle on the same codes and scales."""
    members, prompts, gen, Hq, Hkv, D, extra = CASES[case_id]
    what = f"fp8 case {case_id} workers {workers}"
    print(what, flush=True)
    rng = np.random.default_rng(60 + case_id)
    b, starts, shared = grpo_fp8_batch(rng, members, prompts, gen, Hq, Hkv, D, extra, seed=70 + case_id)
    out = run_prefix_fp8(b, starts, shared, workers)
    parity.assert_parity(out, parity.oracle_full(b), what)


def test_prefix_fp8_oversized_and_no_groups():
    """E4M3 cache: a group too large for the 64 query rows and a group sharing nothing stay exact,
    and no groups at all is plain attention."""
    rng = np.random.default_rng(61)
    b, starts, shared = grpo_fp8_batch(rng, [10, 3, 2], [48, 33, 5], 40, 28, 4, 128, seed=71)
    parity.assert_parity(run_prefix_fp8(b, starts, shared), parity.oracle_full(b), "fp8 oversized group")
    none_s = torch.zeros(1, dtype=torch.int32, device=DEV)
    none_p = torch.zeros(0, dtype=torch.int32, device=DEV)
    parity.assert_parity(run_prefix_fp8(b, none_s, none_p), parity.oracle_full(b), "fp8 no groups")


def test_full_size_grpo_batch_fp8():
    """32 prompts x 8 samples of 1024-token prompts over an E4M3 cache: sampled rows against the
    oracle, and the whole output against the plain E4M3 kernel."""
    b, starts, shared = inputs.make_grpo_batch(32, 8, 1024, seed=4, device=DEV, kv_dtype="e4m3")
    torch.cuda.synchronize()
    out = run_prefix_fp8(b, starts, shared)
    rows = parity.sample_rows(b.seq_lens.cpu().numpy(), 24)
    parity.assert_parity(out[rows], parity.oracle_rows(b, rows), "grpo fp8")
    plain = sl.run_batch(b)
    torch.cuda.synchronize()
    assert (out.float() - plain.float()).abs().max().item() < 0.05


@pytest.mark.parametrize("i", range(8))
def test_prefix_fp8_seeded_sweep(i):
    members, prompts, gen, Hq, Hkv, D, extra, workers = _prefix_sweep_case(100 + i)
    what = f"fp8 prefix sweep {i}: members={members} prompts={prompts} gen<={gen} Hq={Hq} Hkv={Hkv} D={D} " \
           f"extra={extra} workers={workers}"
    print(what, flush=True)
    rng = np.random.default_rng(5000 + i)
    b, starts, shared = grpo_fp8_batch(rng, members, prompts, gen, Hq, Hkv, D, extra, seed=5100 + i)
    out = run_prefix_fp8(b, starts, shared, workers)
    parity.assert_parity(out, parity.oracle_full(b), what)


def test_max_prefix_batch_many_groups_fp8():
    """The largest accepted batch (4096 sequences in 2048 groups of two) over an E4M3 cache, every row."""
    rng = np.random.default_rng(55)
    ng = 2048
    b, starts, shared = grpo_fp8_batch(rng, [2] * ng, list(rng.integers(16, 49, ng)), 40, 8, 2, 64, seed=56)
    assert b.seq_lens.shape[0] == 4096
    print("fp8 batch 4096, 2048 groups", flush=True)
    parity.assert_parity(run_prefix_fp8(b, starts, shared), parity.oracle_full(b), "fp8 batch 4096, 2048 groups")


SPLIT_CASES = [
    # members, prompt lengths, max generated, Hq, Hkv, D, extra: groups beyond M = min(16, 64 / G)
    ([16, 20, 9, 1], [300, 64, 100, 48], 60, 28, 4, 128, 2),   # G = 7, M = 9: 8+8, 7+7+6, 9, 1
    ([40, 17], [130, 16], 30, 16, 16, 64, 0),                  # G = 1, M = 16: 14+14+12, 9+8
    ([33], [200], 10, 64, 8, 128, 1),                          # G = 8, M = 8: 7+7+7+7+5
]


@pytest.mark.parametrize("case_id", range(len(SPLIT_CASES)))
@pytest.mark.parametrize("workers", [0, 1, 7, 1000])
def test_large_groups_split_into_subgroups(case_id, workers):
    """Groups with more members than one shared unit holds are read as consecutive sub-groups,
    each over the shared pages once: every row against the oracle."""
    members, prompts, gen, Hq, Hkv, D, extra = SPLIT_CASES[case_id]
    what = f"split case {case_id} workers {workers}"
    print(what, flush=True)
    rng = np.random.default_rng(90 + case_id)
    case, starts, shared = grpo_case(rng, members, prompts, gen, Hq, Hkv, D, extra)
    out = run_prefix(case, starts, shared, workers)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, what)


def test_whole_batch_one_group():
    """All 300 sequences in one group (G = 4, M = 16: 18 sub-groups of 16 and one of 12)."""
    rng = np.random.default_rng(95)
    case, starts, shared = grpo_case(rng, [300], [520], 40, 16, 4, 128)
    out = run_prefix(case, starts, shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "one group of 300")


def test_non_ascending_group_start_stays_exact():
    """group_start [0, 4, 0, 2, 7]: group 1 is empty (4 > 0), group 2 ([0, 2)) starts before the end
    of group 0 ([0, 4)) and overlaps it, so it must not be shared (sharing both would let two
    shared units claim the same sequences); group 3 ([2, 7)) overlaps group 0 too. Only group 0 is
    shared; every row stays exact."""
    rng = np.random.default_rng(96)
    case, starts, shared = grpo_case(rng, [4, 3], [96, 40], 30, 28, 4, 128, extra=2)
    bad_starts = np.array([0, 4, 0, 2, 7], np.int32)
    bad_shared = np.array([shared[0], 1, 2, 1], np.int32)
    out = run_prefix(case, bad_starts, bad_shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "non-ascending group_start")
    for workers in (1, 1000):
        parity.assert_parity(run_prefix(case, bad_starts, bad_shared, workers), ref, f"non-ascending w={workers}")


def test_large_groups_split_fp8():
    """E4M3 cache: the first split case (16, 20, 9, 1 members at G = 7), every row against the oracle."""
    members, prompts, gen, Hq, Hkv, D, extra = SPLIT_CASES[0]
    rng = np.random.default_rng(97)
    b, starts, shared = grpo_fp8_batch(rng, members, prompts, gen, Hq, Hkv, D, extra, seed=98)
    for workers in (0, 7):
        parity.assert_parity(run_prefix_fp8(b, starts, shared, workers), parity.oracle_full(b),
                             f"fp8 split workers={workers}")


def test_max_prefix_batch_one_group():
    """The largest accepted batch (4096 sequences) as one group: 256 sub-groups of 16 (G = 4)."""
    rng = np.random.default_rng(99)
    case, starts, shared = grpo_case(rng, [4096], [40], 20, 8, 2, 64)
    out = run_prefix(case, starts, shared)
    ref = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"], case["seq_lens"],
                             case["scale"])
    parity.assert_parity(out, ref, "batch 4096, one group")


def _prefix_ws_bytes(B, Hq, Hkv, D, max_blocks, num_pages, ng, workers):
    import ctypes
    desc = sl.make_desc(B, Hq, Hkv, D, 16, max_blocks, num_pages, workers, 0)
    need = ctypes.c_size_t(0)
    sl._check(sl.load().sl_decode_attn_prefix_workspace_size(ctypes.byref(desc), ng, ctypes.byref(need)), "size")
    return need.value


def test_workspace_contents_and_reuse_do_not_matter():
    """Nothing the workspace held before may matter: a workspace of random bytes, reused by calls
    with other batches, group layouts, worker counts and both caches, gives the oracle's rows every
    time, and repeating a call gives the same bits."""
    rng = np.random.default_rng(77)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    plan = [(0, 0), (1, 7), (2, 1000), (0, 3), (3, 0)]
    cases = {}
    need = 0
    for case_id, workers in plan:
        members, prompts, gen, Hq, Hkv, D, extra = CASES[case_id]
        if case_id not in cases:
            cases[case_id] = grpo_case(np.random.default_rng(140 + case_id), members, prompts, gen, Hq, Hkv, D,
                                       extra)
        case, starts, shared = cases[case_id]
        B, mb = case["block_table"].shape
        need = max(need, _prefix_ws_bytes(B, Hq, Hkv, D, mb, case["k_pages"].shape[0], len(shared), workers))
    b, starts8, shared8 = grpo_fp8_batch(np.random.default_rng(5), [8, 3], [200, 40], 90, 28, 4, 128, extra=2,
                                         seed=3)
    need = max(need, _prefix_ws_bytes(b.q.shape[0], 28, 4, 128, b.block_table.shape[1], b.k_pages.shape[0], 2, 0))
    ws = torch.randint(0, 256, (need + 4096,), dtype=torch.uint8, device=DEV)
    ws = ws[(-ws.data_ptr()) % 256:][:need]   # 256-byte aligned view of random bytes
    for case_id, workers in plan:
        case, starts, shared = cases[case_id]
        print("workspace reuse: case", case_id, "workers", workers, flush=True)
        want = oracle.decode_attn(case["q"], case["k_pages"], case["v_pages"], case["block_table"],
                                  case["seq_lens"], case["scale"])
        outs = []
        for rep in range(2):
            out = sl.decode_attn_prefix(_bf16(case["q"]), _bf16(case["k_pages"]), _bf16(case["v_pages"]),
                                        d(case["block_table"]), d(case["seq_lens"]), case["scale"], d(starts),
                                        d(shared), num_workers=workers, workspace=ws)
            torch.cuda.synchronize()
            outs.append(out.clone())
        parity.assert_parity(outs[0], want, f"random workspace, case {case_id}, workers {workers}")
        assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16)), "repeated call differs"
    # E4M3 on the same workspace
    out8 = sl.decode_attn_prefix_fp8(b.q, b.k_pages, b.v_pages, b.k_scales, b.v_scales, b.block_table, b.seq_lens,
                                     b.scale, starts8, shared8, workspace=ws)
    torch.cuda.synchronize()
    parity.assert_parity(out8, parity.oracle_full(b), "E4M3 after the bf16 calls")
