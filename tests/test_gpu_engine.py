"""GPU tests of the decode engine (include/sl_engine.h) against the scheduling oracle.

The schedule, the per-step sequence lengths and the live block-table entries
are integers and must equal the oracle's exactly. At checkpoint steps the
cache on the device is checked too: every generated token's K/V row holds the
row appended in its step, and the step's attention output matches the
attention oracle run on that cache.
"""
import numpy as np
import pytest
import torch

import oracle
import parity
from oracle import schedule as S
from paper_2504_15930_amd import engine as E

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _host_u16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _case(seed, M, lo_p=0, hi_p=100, med_o=40):
    rng = np.random.default_rng(seed)
    prompt = rng.integers(lo_p, hi_p + 1, M).astype(np.int32)
    out = np.clip(np.exp(rng.normal(np.log(med_o), 1.0, M)), 1, 300).astype(np.int32)
    est = np.maximum(1, (out * rng.uniform(0.7, 1.3, M)).astype(np.int32))   # a noisy predictor
    return prompt, out, est


@pytest.mark.parametrize("mode", ["bf16", "bf16-two-launch", "e4m3", "e4m3-two-launch"])
@pytest.mark.parametrize("lpt", [True, False], ids=["lpt", "fifo"])
def test_engine_matches_oracle(lpt, mode):
    fp8 = mode.startswith("e4m3")
    prompt, out, est = _case(11 if lpt else 12, M=30)
    BS, Hq, Hkv, D = 6, 8, 2, 128
    eng = E.Engine(prompt, out, est, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
                   kv_fp8=fp8, lpt=lpt, seed=3, two_launch=mode.endswith("two-launch"))
    ref = S.simulate(prompt, out, est, BS, eng.num_pages, eng.max_blocks, "lpt" if lpt else "fifo",
                     checkpoints=range(0, 10000))
    checks = [0, 1, 2, 7, 16, 33, ref.makespan // 2, ref.makespan - 1]
    done = 0
    for c in sorted(set(checks)):
        done += eng.run(c + 1 - done)
        assert done == c + 1
        torch.cuda.synchronize()
        lens = eng.seq_lens.cpu().numpy()
        table = eng.block_table.cpu().numpy()
        want_lens, want_table = ref.checkpoints[c]
        assert lens.tolist() == want_lens, f"step {c}: lengths"
        for b in range(BS):
            n = -(-int(lens[b]) // 16)
            assert table[b, :n].tolist() == want_table[b][:n], f"step {c}: block table of slot {b}"
        # generated tokens hold the appended row of their slot (bf16 pages store it verbatim)
        if not fp8:
            kp = _host_u16(eng.k_pages)
            kn = _host_u16(eng.k_new)
            slot_of = {int(ref.slot[i]): i for i in range(len(out))
                       if ref.admit_step[i] <= c and (ref.finish_step[i] >= c)}
            for b, i in slot_of.items():
                for t in range(int(prompt[i]), int(lens[b])):
                    pg = table[b, t // 16]
                    assert np.array_equal(kp[pg, :, t % 16, :], kn[b]), f"step {c}: slot {b} token {t}"
        # this step's attention output against the oracle on the device cache
        q = _host_u16(eng.q)
        kw = dict(k_scales=eng.k_scales.cpu().numpy(), v_scales=eng.v_scales.cpu().numpy()) if fp8 else {}
        kp_all = eng.k_pages.cpu().numpy() if fp8 else _host_u16(eng.k_pages)
        vp_all = eng.v_pages.cpu().numpy() if fp8 else _host_u16(eng.v_pages)
        want = oracle.decode_attn(q, kp_all, vp_all, table, lens, eng.scale, **kw)
        parity.assert_parity(eng.out, want, f"attention at step {c}")
    eng.run()
    slot, adm, fin, steps, active = eng.schedule()
    assert steps == ref.makespan
    assert slot.tolist() == ref.slot and adm.tolist() == ref.admit_step and fin.tolist() == ref.finish_step
    assert active.sum() == int(out.sum())
    eng.close()


def test_engine_lpt_beats_fifo_on_long_tail():
    """On a long-tailed batch with the longest samples last in index order, LPT needs fewer
    steps than FIFO (the makespans equal the oracle's)."""
    rng = np.random.default_rng(5)
    M, BS = 64, 8
    out = np.clip(np.exp(rng.normal(np.log(30), 1.2, M)), 1, 600).astype(np.int32)
    out = np.sort(out)                                  # longest last: the worst case for FIFO
    prompt = np.full(M, 20, np.int32)
    spans = {}
    for lpt in (True, False):
        eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=4, num_kv_heads=1, head_dim=64, lpt=lpt)
        eng.run()
        torch.cuda.synchronize()
        spans[lpt] = eng.schedule()[3]
        ref = S.simulate(prompt, out, out, BS, eng.num_pages, eng.max_blocks, "lpt" if lpt else "fifo")
        assert spans[lpt] == ref.makespan
        eng.close()
    assert spans[True] < spans[False]


def test_engine_one_launch_long_contexts():
    """bf16 cache, 32 slots of 7B-like heads with prompts of 300-1500 tokens: the one-launch step
    gives every unit several workgroups, whose pieces the last one to arrive merges. Checked at
    checkpoints against the oracle, after runs of one and of many steps."""
    rng = np.random.default_rng(21)
    M, BS, Hq, Hkv, D = 48, 32, 28, 4, 128
    prompt = rng.integers(300, 1500, M).astype(np.int32)
    out = np.clip(np.exp(rng.normal(np.log(60), 0.8, M)), 1, 200).astype(np.int32)
    eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, lpt=True,
                   seed=4)
    ref = S.simulate(prompt, out, out, BS, eng.num_pages, eng.max_blocks, "lpt", checkpoints=range(0, 10000))
    done = 0
    for c in [0, 1, 2, 3, 9, 10, 40, ref.makespan // 2, ref.makespan - 2, ref.makespan - 1]:
        print("one-launch engine checkpoint", c, flush=True)
        done += eng.run(c + 1 - done)
        assert done == c + 1
        torch.cuda.synchronize()
        lens = eng.seq_lens.cpu().numpy()
        table = eng.block_table.cpu().numpy()
        want_lens, want_table = ref.checkpoints[c]
        assert lens.tolist() == want_lens, f"step {c}: lengths"
        want = oracle.decode_attn(_host_u16(eng.q), _host_u16(eng.k_pages), _host_u16(eng.v_pages), table, lens,
                                  eng.scale)
        parity.assert_parity(eng.out, want, f"one-launch attention at step {c}")
    eng.close()


@pytest.mark.parametrize("queries", ["zero", "random"])
@pytest.mark.parametrize("Hq,Hkv,D", [(8, 2, 128), (16, 1, 64)], ids=["G4-D128", "G16-D64"])
@pytest.mark.parametrize("kv", ["bf16", "e4m3"])
def test_engine_one_launch_every_step_matches_two_launch(kv, Hq, Hkv, D, queries):
    """Every step's output of a whole generation, kept in the engine's output history, with one
    launch per step against split + merge (whose steps the oracle checks above). The samples finish
    often, open pages often (prompts of 0, 16, 32 tokens among them) and include one 3000-token
    prompt, so the steps cover units of one and of many workgroups, empty slots, admissions beside
    finishes, and next-step appends that take a page freed in the same step (those run in a launch
    of their own). With an E4M3 cache the one-launch step's units append their own next rows (the
    single workgroup of a unit, or the last of its workgroups to arrive); both runs must leave the
    same codes and scales in every page, bit for bit.

    Zero queries make every weight exactly 1: both paths then compute the mean of the value rows
    and may differ only in the last place of the bf16 output, while a row read at the wrong time
    would move the mean by its change over the length. With random queries each path rounds its
    weights to bf16 against its own running maxima, an error of at most 2^-9 of the spread of the
    value rows around the output each (bounded by 2 max |v|), so the paths may differ by
    2^-7 max |v| plus two units in the last place."""
    rng = np.random.default_rng(33)
    M, BS = 60, 16
    prompt = rng.choice(np.array([0, 16, 32, 5, 47, 100, 260], np.int32), M)
    prompt[7] = 3000
    out = np.clip(np.exp(rng.normal(np.log(12), 0.9, M)), 1, 60).astype(np.int32)
    ref = S.simulate(prompt, out, out, BS, BS * int(((prompt + out + 15) // 16).max()),
                     int(((prompt + out + 15) // 16).max()), "lpt")
    steps = ref.makespan
    hist, cache = {}, {}
    vmax = 2.0   # synthetic prompt values lie in (-2, 2) for both caches
    for two in (False, True):
        eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, lpt=True,
                       kv_fp8=kv == "e4m3", seed=9, two_launch=two, history_steps=steps)
        if queries == "zero":
            eng.q.zero_()
        vmax = max(vmax, float(eng.v_new.float().abs().max()))
        assert eng.run() == steps
        torch.cuda.synchronize()
        hist[two] = eng.history.float().cpu()
        cache[two] = [t.cpu().view(torch.uint8) if t.dtype != torch.float32 else t.cpu().view(torch.int32)
                      for t in ((eng.k_pages, eng.v_pages, eng.k_scales, eng.v_scales) if kv == "e4m3"
                                else (eng.k_pages, eng.v_pages))]
        eng.close()
    for x, y, name in zip(cache[False], cache[True], ("k pages", "v pages", "k scales", "v scales")):
        assert torch.equal(x, y), f"{name} differ between the launch modes"
    a, b = hist[False], hist[True]
    assert torch.isfinite(a).all() and torch.isfinite(b).all()
    mag = torch.maximum(a.abs(), b.abs()).clamp_min(2.0 ** -126)
    ulp = torch.exp2(torch.floor(torch.log2(mag)) - 7)   # bf16 spacing at the larger magnitude
    bound = ulp + 1e-5 if queries == "zero" else 2 * ulp + 2.0 ** -7 * vmax
    err = (a - b).abs()
    bad = err > bound
    assert not bad.any(), (f"{int(bad.sum())} elements differ, first at step "
                           f"{int(bad.nonzero()[0, 0])}, max |diff| {float(err.max()):.3g}")
    print(f"one-launch vs two-launch: max |diff| {float(err.max()):.3g} over {steps} steps", flush=True)


def test_engine_clears_empty_rows_after_caller_writes_out():
    """The one-launch step clears an empty slot's output rows once, not every step. A caller that
    writes `out` between run calls (here: NaN everywhere) must still find zero rows for the empty
    slots, and the oracle's rows for the others, after the next call."""
    prompt = np.array([40, 7, 300, 0, 90, 16], np.int32)
    out = np.array([3, 60, 9, 25, 1, 40], np.int32)
    BS, Hq, Hkv, D = 8, 8, 2, 128          # more slots than samples: some slots are always empty
    eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, lpt=True,
                   seed=6)
    ref = S.simulate(prompt, out, out, BS, eng.num_pages, eng.max_blocks, "lpt", checkpoints=range(0, 10000))
    done = 0
    for c in (0, 4, 12, 30, ref.makespan - 1):
        done += eng.run(c + 1 - done)
        torch.cuda.synchronize()
        lens = eng.seq_lens.cpu().numpy()
        table = eng.block_table.cpu().numpy()
        assert lens.tolist() == ref.checkpoints[c][0], f"step {c}: lengths"
        want = oracle.decode_attn(_host_u16(eng.q), _host_u16(eng.k_pages), _host_u16(eng.v_pages), table, lens,
                                  eng.scale)
        got = eng.out.float().cpu()
        for b in range(BS):
            if lens[b] == 0:
                assert torch.all(got[b] == 0), f"step {c}: empty slot {b} not cleared"
        parity.assert_parity(eng.out, want, f"attention at step {c}")
        eng.out.fill_(float("nan"))      # the caller's write between calls
    eng.close()


@pytest.mark.parametrize("kv", ["bf16", "e4m3"])
@pytest.mark.parametrize("case", range(8))
def test_engine_launch_modes_agree_on_random_shapes(kv, case):
    """Seeded head shapes, slot counts and prompt mixes (whole pages, 0-token prompts, long
    prompts that give units of several workgroups): both launch modes must leave the same cache,
    bit for bit (E4M3 codes and scales included), the same lengths and block table, and per-step
    outputs within the bound derived above (zero queries: the last bf16 place); the last step's
    output also matches the oracle."""
    rng = np.random.default_rng(530 + case)
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    D = int(rng.choice([64, 128]))
    BS = int(rng.integers(2, 24))
    M = int(rng.integers(BS, 3 * BS + 1))
    prompt = rng.choice(np.array([0, 1, 15, 16, 17, 31, 64, 200, 777, 2100], np.int32), M)
    out = np.clip(np.exp(rng.normal(np.log(10), 1.0, M)), 1, 80).astype(np.int32)
    need = int(((prompt + out + 15) // 16).max())
    steps = S.simulate(prompt, out, out, BS, BS * need, need, "lpt").makespan
    print(f"case {case}: Hkv {Hkv} G {G} D {D} BS {BS} M {M} steps {steps}", flush=True)
    hist, state = {}, {}
    for two in (False, True):
        eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=G * Hkv, num_kv_heads=Hkv, head_dim=D,
                       lpt=True, kv_fp8=kv == "e4m3", seed=case, two_launch=two, history_steps=steps)
        eng.q.zero_()
        assert eng.run() == steps
        torch.cuda.synchronize()
        hist[two] = eng.history.float().cpu()
        fp8 = kv == "e4m3"
        kp = eng.k_pages.cpu().numpy() if fp8 else _host_u16(eng.k_pages)
        vp = eng.v_pages.cpu().numpy() if fp8 else _host_u16(eng.v_pages)
        ks = eng.k_scales.cpu().numpy() if fp8 else None
        vs = eng.v_scales.cpu().numpy() if fp8 else None
        lens = eng.seq_lens.cpu().numpy()
        table = eng.block_table.cpu().numpy()
        state[two] = (kp, vp, ks, vs, lens, table)
        if not two:
            kw = dict(k_scales=ks, v_scales=vs) if fp8 else {}
            want = oracle.decode_attn(_host_u16(eng.q), kp, vp, table, lens, eng.scale, **kw)
            parity.assert_parity(eng.out, want, f"case {case}: last step")
        eng.close()
    a, b = state[False], state[True]
    for x, y, name in zip(a, b, ("k pages", "v pages", "k scales", "v scales", "lengths", "block table")):
        if x is not None:
            assert np.array_equal(x.view(np.uint8) if x.dtype != np.int32 else x,
                                  y.view(np.uint8) if y.dtype != np.int32 else y), f"{name} differ"
    h1, h2 = hist[False], hist[True]
    mag = torch.maximum(h1.abs(), h2.abs()).clamp_min(2.0 ** -126)
    ulp = torch.exp2(torch.floor(torch.log2(mag)) - 7)
    err = (h1 - h2).abs()
    assert torch.isfinite(h1).all() and torch.isfinite(h2).all()
    assert not (err > ulp + 1e-5).any(), f"max |diff| {float(err.max()):.3g}"


@pytest.mark.parametrize("kv", ["e4m3", "bf16"])
def test_engine_rows_that_change_every_step(kv):
    """Row sets of growing magnitude (x1, x4, x16, x64, x256, in turn): with an E4M3 cache every
    append after a smaller set raises its page's scale and re-encodes rows that the same step's
    attention reads (any page holding generated rows of two sets has been re-encoded). The
    one-launch step appends a unit's row only after the unit's reads, so both launch modes must
    leave the same codes and scales, bit for bit, and the same per-step outputs (zero queries: to
    the last bf16 place); the last step also matches the oracle on the device cache. With a bf16
    cache every generated token of the samples that finish in the last step holds its step's set."""
    rng = np.random.default_rng(91)
    M, BS, Hq, Hkv, D, R = 20, 6, 8, 2, 128, 5
    prompt = rng.choice(np.array([0, 3, 16, 21, 40, 77], np.int32), M)
    out = np.clip(np.exp(rng.normal(np.log(30), 0.8, M)), 2, 100).astype(np.int32)
    need = int(((prompt + out + 15) // 16).max())
    ref = S.simulate(prompt, out, out, BS, BS * need, need, "lpt")
    steps = ref.makespan
    assert int(out.max()) >= 17   # some page holds generated rows of several sets
    fp8 = kv == "e4m3"
    hist, cache = {}, {}
    for two in (False, True):
        eng = E.Engine(prompt, out, out, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, lpt=True,
                       kv_fp8=fp8, seed=5, two_launch=two, history_steps=steps, row_sets=R)
        scale = (4.0 ** torch.arange(R, device=DEV, dtype=torch.float32)).view(R, 1, 1, 1)
        eng.k_new.copy_((eng.k_new.float() * scale).to(torch.bfloat16))
        eng.v_new.copy_((eng.v_new.float() * scale).to(torch.bfloat16))
        eng.q.zero_()
        assert eng.run() == steps
        torch.cuda.synchronize()
        hist[two] = eng.history.float().cpu()
        kp = eng.k_pages.cpu().numpy() if fp8 else _host_u16(eng.k_pages)
        vp = eng.v_pages.cpu().numpy() if fp8 else _host_u16(eng.v_pages)
        ks = eng.k_scales.cpu().numpy() if fp8 else None
        vs = eng.v_scales.cpu().numpy() if fp8 else None
        lens, table = eng.seq_lens.cpu().numpy(), eng.block_table.cpu().numpy()
        cache[two] = (kp, vp, ks, vs, lens, table)
        if not fp8 and not two:   # token t of sample i, made in step admit + (t - p), holds that step's set
            kn = _host_u16(eng.k_new)
            for i in range(M):
                b = ref.slot[i]
                if ref.finish_step[i] != steps - 1:
                    continue   # finished earlier: its pages may have been handed out again
                for t in range(int(prompt[i]), int(prompt[i] + out[i])):
                    step = ref.admit_step[i] + (t - int(prompt[i]))
                    assert np.array_equal(kp[table[b, t // 16], :, t % 16, :], kn[step % R, b]), (i, t)
        if not two:
            kw = dict(k_scales=ks, v_scales=vs) if fp8 else {}
            want = oracle.decode_attn(_host_u16(eng.q), kp, vp, table, lens, eng.scale, **kw)
            if fp8:
                vdq = torch.from_numpy(vp).view(torch.float8_e4m3fn).double().numpy() * vs[:, :, None, None]
            else:
                vdq = torch.from_numpy(vp.view(np.int16)).view(torch.bfloat16).double().numpy()
            parity.assert_parity(eng.out, want, "last step",
                                 value_scale=parity.value_rms_rows(vdq, table, lens, Hq))
        eng.close()
    for x, y, name in zip(cache[False], cache[True], ("k pages", "v pages", "k scales", "v scales", "lengths",
                                                      "block table")):
        if x is not None:
            assert np.array_equal(x.view(np.uint8) if x.dtype != np.int32 else x,
                                  y.view(np.uint8) if y.dtype != np.int32 else y), f"{name} differ"
    a, b = hist[False], hist[True]
    assert torch.isfinite(a).all() and torch.isfinite(b).all()
    mag = torch.maximum(a.abs(), b.abs()).clamp_min(2.0 ** -126)
    ulp = torch.exp2(torch.floor(torch.log2(mag)) - 7)
    err = (a - b).abs()
    assert not (err > ulp + 1e-5 * mag.clamp_min(1.0)).any(), f"max |diff| {float(err.max()):.3g}"
