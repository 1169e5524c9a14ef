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


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "e4m3"])
@pytest.mark.parametrize("lpt", [True, False], ids=["lpt", "fifo"])
def test_engine_matches_oracle(lpt, fp8):
    prompt, out, est = _case(11 if lpt else 12, M=30)
    BS, Hq, Hkv, D = 6, 8, 2, 128
    eng = E.Engine(prompt, out, est, batch_slots=BS, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
                   kv_fp8=fp8, lpt=lpt, seed=3)
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
