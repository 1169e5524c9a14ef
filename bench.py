"""Benchmark: one decode step of paged GQA decode attention on one MI355X.

A step is one ``sl_decode_attn`` call over the whole synthetic batch (the
split-KV kernel, which partitions the work itself, and the log-sum-exp
merge), with every input
already resident in HBM. Prints one JSON line:

  value      algorithmic bytes per step / wall time per step (GB/s), where the
             algorithmic bytes are the K/V page bytes of every live token
             (2 * D * bytes-per-element per token and KV head; FP8 adds the two
             4-byte scales per page and KV head), q and out (2 * Hq * D * 2 per
             sequence) and one 4-byte block-table entry per page;
  roofline   the split-KV kernel alone: the same algorithmic bytes over its
             average duration from HIP events recorded around it on the launch
             stream; HBM-bound, peak 8 TB/s; ``traffic`` comes from the
             committed rocprofv3 counter summary for this workload when it was
             taken on the current kernel source, else null;
  cpu_baseline  the fp64 CPU oracle timed on the host cores on a bounded
             sample of the same batch (the sequences and the byte count are
             named in ``sample``); its outputs are also compared with the GPU's;
             ``single_thread`` times it on one core over a 32-sequence subset;
  configs    the other long-tail decode steps measured the same way in the
             same run (straggler-only, 72B-like, E4M3 cache): step time, GB/s,
             % of peak, steps/s, the split kernel's roofline and an oracle
             baseline on a seeded subset of 32 sequences (always the longest
             and the shortest) timed on all cores and on one.

Single GPU only: ``--gpus`` above 1 exits with an explanation.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
PEAK_HBM_GBS = 8000.0
METRIC = "decode-attn achieved HBM GB/s (% of MI355X peak) + decode steps/s, long-tail batch"
KERNEL_SOURCES = ["paper_2504_15930_amd/csrc/decode_split.hip", "paper_2504_15930_amd/csrc/decode_unit.h",
                  "paper_2504_15930_amd/csrc/sl_internal.h"]
# Decode steps measured besides the headline one, with the share of peak HBM bandwidth each
# one's step is to reach (None: reported only) and the layer count of the model whose heads it
# has (Qwen2.5-7B: 28 layers, Qwen2.5-72B: 80), for attention-only steps/s of a whole model.
OTHER_CONFIGS = ["straggler", "qwen72b_longtail", "fp8_qwen7b_longtail"]
TARGET_PCT = {"qwen7b_longtail": 75.0, "qwen72b_longtail": 75.0, "straggler": 60.0, "fp8_qwen7b_longtail": None}
MODEL_LAYERS = {"qwen7b_longtail": 28, "fp8_qwen7b_longtail": 28, "qwen72b_longtail": 80, "straggler": 80}
# bf16 weights a whole model's decode step reads once (every decode step touches all parameters,
# Section 2.2): Qwen2.5-7B holds about 7.6 B parameters, Qwen2.5-72B about 72.7 B.
MODEL_WEIGHT_BYTES = {"qwen7b_longtail": 15.2e9, "fp8_qwen7b_longtail": 15.2e9, "qwen72b_longtail": 145.4e9,
                      "straggler": 145.4e9}


def algorithmic_bytes(seq_lens: np.ndarray, num_q_heads: int, num_kv_heads: int, head_dim: int,
                      kv_bytes: int, page_size: int = 16) -> int:
    L = np.maximum(seq_lens.astype(np.int64), 0)
    pages = -(-L // page_size)
    kv = int(L.sum()) * num_kv_heads * 2 * head_dim * kv_bytes
    scales = int(pages.sum()) * num_kv_heads * 2 * 4 if kv_bytes == 1 else 0
    qo = len(L) * 2 * num_q_heads * head_dim * 2
    table = int(pages.sum()) * 4
    return kv + scales + qo + table


def prefix_unique_bytes(seq_lens: np.ndarray, num_groups: int, shared_pages: int, num_q_heads: int,
                        num_kv_heads: int, head_dim: int, kv_bytes: int, page_size: int = 16) -> int:
    """Algorithmic bytes of prefix-shared attention when every sequence belongs to one of ``num_groups``
    groups sharing ``shared_pages`` full pages: each shared page (its K and V rows, its table entry and,
    for E4M3, its two scales) once per group, every own token and own page once, q and out."""
    L = np.maximum(seq_lens.astype(np.int64), 0)
    own_tokens = int((L - page_size * shared_pages).sum())
    own_pages = int((-(-L // page_size) - shared_pages).sum())
    pages = num_groups * shared_pages + own_pages
    kv = (num_groups * shared_pages * page_size + own_tokens) * num_kv_heads * 2 * head_dim * kv_bytes
    scales = pages * num_kv_heads * 2 * 4 if kv_bytes == 1 else 0
    return kv + len(L) * 2 * num_q_heads * head_dim * 2 + pages * 4 + scales


def append_bytes(seq_lens: np.ndarray, num_kv_heads: int, head_dim: int, kv_bytes: int) -> int:
    """Algorithmic bytes of one KV append: the new K and V rows (bf16) read, their cached form
    written, the per-(page, head) scales read and written (E4M3), and one length and one
    block-table entry per appending sequence. Re-encoded earlier rows are not counted."""
    n = int((seq_lens >= 1).sum())
    rows = n * num_kv_heads * 2 * head_dim * (2 + kv_bytes)
    scales = n * num_kv_heads * 2 * 8 if kv_bytes == 1 else 0
    return rows + scales + n * 8


def generation(w, fp8: bool, seed: int, dev) -> dict:
    """A whole generation on the decode engine: 512 samples with long-tailed output lengths
    (lognormal, median 1024, sigma 1, capped at 8192; prompts of 256-768 tokens) on 128 batch
    slots with the workload's head shape. The admission estimate is the true length times a
    lognormal error (sigma 0.3). Runs LPT and FIFO admission; every step is KV append + decode
    attention for one layer, timed with events around the whole run. The engine runs steps with
    little attention work in one launch; the same two runs with every step as split kernel +
    merge are reported beside them."""
    import torch

    from paper_2504_15930_amd import engine as E

    rng = np.random.default_rng(seed)
    M, BS = 512, 128
    prompt = rng.integers(256, 769, M).astype(np.int32)
    out = np.clip(np.exp(rng.normal(np.log(1024), 1.0, M)), 16, 8192).astype(np.int32)
    est = np.maximum(1, out * np.exp(rng.normal(0.0, 0.3, M))).astype(np.int32)
    res = {"samples": M, "batch_slots": BS, "output_tokens": int(out.sum()), "max_output": int(out.max()),
           "what": "KV append + decode attention per step, one layer", "kv_dtype": "e4m3" if fp8 else "bf16"}
    arms = [("lpt", True, False), ("fifo", False, False), ("lpt_two_launch", True, True),
            ("fifo_two_launch", False, True)]
    for name, lpt, two in arms:
        print(f"[bench] generation ({name})", file=sys.stderr, flush=True)
        eng = E.Engine(prompt, out, est, batch_slots=BS, num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads,
                       head_dim=w.head_dim, kv_fp8=fp8, lpt=lpt, seed=seed, device=dev, two_launch=two)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        steps = eng.run()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        active = eng.schedule()[4]
        res[name] = {"steps": steps, "ms": round(ms, 2), "us_per_step": round(1e3 * ms / steps, 2),
                     "output_tokens_per_s": round(out.sum() / (ms * 1e-3), 1),
                     "steps_under_quarter_busy": int((active < BS // 4).sum())}
        eng.close()
        del eng
        torch.cuda.empty_cache()
    res["lpt_speedup_over_fifo"] = round(res["fifo"]["ms"] / res["lpt"]["ms"], 3)
    return res


def ptl_at(batch: int, prof_b, prof_s) -> float:
    """PTL(batch) from a measured profile: linear between profiled batch sizes, the first value
    below them, the last segment continued beyond them (as the dispatching code reads it)."""
    xs, ys = list(prof_b), list(prof_s)
    if batch <= xs[0] or len(xs) == 1:
        return ys[0]
    for k in range(1, len(xs)):
        if batch <= xs[k]:
            return ys[k - 1] + (ys[k] - ys[k - 1]) * (batch - xs[k - 1]) / (xs[k] - xs[k - 1])
    return ys[-1] + (ys[-1] - ys[-2]) * (batch - xs[-1]) / (xs[-1] - xs[-2])


DISPATCH_REGIMES = [(1024, 128), (1024, 32), (4096, 128), (4096, 32)]   # (prompts, most decoded at once)


def dispatch_experiment(w, seed: int, dev, stream_gbs: float | None = None) -> dict:
    """Skewness-aware dispatching (Algorithm 2 with Equation 2) fed by PTL(BS) measured here,
    against random dispatching, with the generation stage of every plan run on the decode engine.

    PTL(BS): one decode step (KV append + attention, this workload's heads) over BS sequences of
    2048 cached tokens, for BS = 1 .. 256. A batch of prompts (256-768 tokens) has true output
    lengths lognormal (median 1024, sigma 1, capped at 8192); the estimates the dispatcher sees are
    the truth times a lognormal error (sigma 0.3), standing in for the output-length ranker; the
    length distribution D is a separate draw. N = 8 instances, alpha = 0.2. Three arms per regime:
    random dispatch, skewness-aware dispatch on the noisy estimates, and skewness-aware dispatch on
    the true lengths (the known-lengths setting). Every instance of every plan runs its prompts on
    the engine (LPT admission by the arm's lengths, at most ``max_batch`` at once), and the stage
    time of a plan is its slowest instance. Beside each measured stage: Equation 2's estimate for
    the plan, and Sum over steps of PTL(sequences active in that step) along the slowest instance's
    actual schedule. The regimes: 1024 prompts with 128 per instance at once (a random instance
    holds 128 prompts: one round), and with 32 (four rounds), the case Equation 2's ceil(M / BS)
    and the paper's scheduling-order discussion are about; 4096 prompts with 128 at once (a random
    instance holds 512 prompts: four rounds); and 4096 prompts with 32 at once (sixteen rounds, so
    that an instance's steps are set by its total output rather than by its longest sample).

    With ``stream_gbs`` (this GPU's measured streaming rate) every plan also gets a modelled
    whole-model stage: per instance, its measured one-layer time times the model's layer count,
    plus its step count times the time to stream the model's bf16 weights once at that rate (the
    per-step floor that a whole model's decode step has and attention alone lacks); the stage is
    the slowest instance."""
    import torch

    from paper_2504_15930_amd import dispatch as Dsp
    from paper_2504_15930_amd import engine as E
    from paper_2504_15930_amd import inputs, sl

    Hq, Hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
    prof_b = [1, 2, 4, 8, 16, 32, 64, 128, 256]
    prof_s = []
    for bs in prof_b:
        b = inputs.make_paged_batch([2048] * bs, Hq, Hkv, D, seed=seed + 1, device=dev, poison=False)
        kn = torch.randn((bs, Hkv, D), device=dev).to(torch.bfloat16)
        out = torch.empty_like(b.q)
        for it in range(35):
            if it == 5:
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
            sl.kv_append(kn, kn, b.block_table, b.seq_lens, b.k_pages, b.v_pages, num_q_heads=Hq)
            sl.run_batch(b, out=out)
        e1.record()
        torch.cuda.synchronize()
        prof_s.append(e0.elapsed_time(e1) / 30 * 1e-3)
        del b
        torch.cuda.empty_cache()
    N, alpha = 8, 0.2
    res = {"ptl_profile": {"batch": prof_b, "us": [round(x * 1e6, 2) for x in prof_s],
                           "what": "KV append + decode attention, 2048 cached tokens per sequence"},
           "instances": N, "alpha": alpha, "estimate_error_sigma": 0.3, "regimes": []}
    layers = MODEL_LAYERS.get(w.name)
    weight_ms = None
    if stream_gbs and layers and w.name in MODEL_WEIGHT_BYTES:
        weight_ms = MODEL_WEIGHT_BYTES[w.name] / (stream_gbs * 1e9) * 1e3
        res["whole_model"] = {"layers": layers, "weight_bytes": MODEL_WEIGHT_BYTES[w.name],
                              "stream_GBps": round(stream_gbs, 1), "weight_ms_per_step": round(weight_ms, 4),
                              "what": "per instance: layers x its measured one-layer time + its steps x the "
                                      "time to stream the weights once; stage = slowest instance"}

    for P, maxb in DISPATCH_REGIMES:
        rng = np.random.default_rng(seed)
        true = np.clip(np.exp(rng.normal(np.log(1024), 1.0, P)), 16, 8192).astype(np.int32)
        est = np.maximum(1, true * np.exp(rng.normal(0.0, 0.3, P))).astype(np.int32)
        prompt = rng.integers(256, 769, P).astype(np.int32)
        dist = np.clip(np.exp(rng.normal(np.log(1024), 1.0, 1024)), 16, 8192).astype(np.int32)

        def run_plan(inst, order_len):
            """Every instance of a plan on the engine; its slowest instance is the stage time."""
            per, sched, steps = [], [], []
            for k in range(N):
                idx = np.nonzero(inst == k)[0]
                if len(idx) == 0:
                    per.append(0.0)
                    sched.append(0.0)
                    steps.append(0)
                    continue
                eng = E.Engine(prompt[idx], true[idx], order_len[idx], batch_slots=min(len(idx), maxb),
                               num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, lpt=True, seed=seed, device=dev)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                eng.run()
                e1.record()
                torch.cuda.synchronize()
                n_steps, active = eng.schedule()[3:5]
                per.append(round(e0.elapsed_time(e1), 2))
                sched.append(round(1e3 * sum(ptl_at(int(a), prof_b, prof_s) for a in active), 2))
                steps.append(int(n_steps))
                eng.close()
                del eng
                torch.cuda.empty_cache()
            k = int(np.argmax(per))
            r = {"stage_ms": per[k], "instance_ms": per, "instance_steps": steps, "slowest_instance": k,
                 "slowest_prompts": int((inst == k).sum()), "slowest_longest_output": int(true[inst == k].max()),
                 "schedule_ptl_estimate_ms": sched[k]}
            if weight_ms is not None:
                r["whole_model_stage_ms"] = round(max(layers * t + n * weight_ms for t, n in zip(per, steps)), 1)
            return r

        reg = {"prompts": P, "max_batch": maxb}
        print(f"[bench] dispatch {P} prompts, {maxb} at once: random", file=sys.stderr, flush=True)
        perm = np.random.default_rng(seed + 1).permutation(P)
        rinst = np.empty(P, np.int32)
        rinst[perm] = np.arange(P) % N
        reg["random"] = run_plan(rinst, est)
        for arm, lengths in (("skew_est", est), ("skew_true", true)):
            done = {}
            for combine in ("sum", "max"):
                print(f"[bench] dispatch {P} prompts, {maxb} at once: {arm} ({combine})", file=sys.stderr, flush=True)
                nl, nr, lat, inst = Dsp.plan(lengths, alpha, dist, N, prof_b, prof_s, maxb, combine)
                if (nl, nr) not in done:
                    done[(nl, nr)] = run_plan(inst, lengths)
                r = dict(done[(nl, nr)])
                r.update(long_tail_instances=nl, regular_instances=nr, eq2_estimate_ms=round(lat * 1e3, 2),
                         speedup_over_random=round(reg["random"]["stage_ms"] / max(r["stage_ms"], 1e-9), 3))
                if weight_ms is not None:
                    r["whole_model_speedup_over_random"] = round(
                        reg["random"]["whole_model_stage_ms"] / max(r["whole_model_stage_ms"], 1e-9), 3)
                reg[f"{arm}_{combine}"] = r
        res["regimes"].append(reg)
    return res


def prefix_subgroups(samples: int, group: int) -> int:
    """Sub-groups a group of ``samples`` members is read as: one shared unit holds at most
    min(16, 64 / G) members (64 query rows of G heads each)."""
    return -(-samples // min(16, 64 // group))


def prefix_experiment(w, seed: int, dev, steps: int, warmup: int, prompts: int = 32, samples: int = 8) -> dict:
    """Prefix sharing on a GRPO-like batch with this workload's heads and cache type: ``prompts``
    x ``samples``, 1024-token prompts (64 shared pages per group), generated lengths lognormal
    (median 512, sigma 1, capped at 4096). Plain decode attention reads every sample's copy of the
    prompt pages; the prefix path reads them once per sub-group (a group larger than one shared
    unit holds is read as several). ``unique_bytes`` counts what the prefix path has to read
    (shared pages and their scales once per sub-group); ``ideal_bytes`` once per group."""
    import torch

    from paper_2504_15930_amd import inputs, sl

    prompt_len = 1024
    b, starts, shared = inputs.make_grpo_batch(prompts, samples, prompt_len, seed=seed + 11, device=dev,
                                               num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads,
                                               head_dim=w.head_dim, kv_dtype=w.kv_dtype)
    torch.cuda.synchronize()
    L = b.seq_lens.cpu().numpy().astype(np.int64)
    Hq, Hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
    kvb = 1 if w.kv_dtype == "e4m3" else 2
    plain_bytes = algorithmic_bytes(L, Hq, Hkv, D, kvb)
    subs = prefix_subgroups(samples, Hq // Hkv)
    unique_bytes = prefix_unique_bytes(L, prompts * subs, prompt_len // 16, Hq, Hkv, D, kvb)
    ideal_bytes = prefix_unique_bytes(L, prompts, prompt_len // 16, Hq, Hkv, D, kvb)
    out = torch.empty_like(b.q)

    def plain():
        sl.run_batch(b, out=out)

    def prefixed():
        if kvb == 1:
            sl.decode_attn_prefix_fp8(b.q, b.k_pages, b.v_pages, b.k_scales, b.v_scales, b.block_table,
                                      b.seq_lens, b.scale, starts, shared, out=out)
        else:
            sl.decode_attn_prefix(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale, starts,
                                  shared, out=out)

    res = {}
    for name, fn in (("plain", plain), ("prefix", prefixed)):
        for _ in range(warmup):
            fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / steps
    return {
        "what": "decode attention with prefix sharing vs plain, GRPO-like batch",
        "config": {"kv_dtype": w.kv_dtype, "prompts": prompts, "samples": samples, "prompt_len": prompt_len,
                   "gen_median": 512,
                   "gen_sigma": 1.0, "gen_cap": 4096, "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D,
                   "total_tokens": int(L.sum()), "max_seq_len": int(L.max())},
        "plain_ms": round(res["plain"], 5),
        "prefix_ms": round(res["prefix"], 5),
        "speedup": round(res["plain"] / res["prefix"], 3),
        "subgroups_per_group": subs,
        "plain_bytes": plain_bytes,
        "unique_bytes": unique_bytes,
        "ideal_bytes": ideal_bytes,
        "plain_GBps": round(plain_bytes / (res["plain"] * 1e-3) / 1e9, 2),
        "prefix_unique_GBps": round(unique_bytes / (res["prefix"] * 1e-3) / 1e9, 2),
        "prefix_effective_GBps": round(plain_bytes / (res["prefix"] * 1e-3) / 1e9, 2),
    }


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_counter_summary(workload: str) -> dict | None:
    """key = value lines of profiles/decode_split_<workload>_counters.txt, if present."""
    path = os.path.join(ROOT, "profiles", f"decode_split_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    out = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                out[k.strip()] = v.strip()
    return out


def traffic_bytes(workload: str) -> float | None:
    c = read_counter_summary(workload)
    if not c or c.get("kernel_source_sha") != kernel_source_hash():
        return None
    try:
        fetch = float(c["fetch_kib_per_dispatch"]) * float(c["fetch_scale"])
        write = float(c["write_kib_per_dispatch"]) * float(c["write_scale"])
    except (KeyError, ValueError):
        return None
    return (fetch + write) * 1024.0


def compact_rows(batch, rows):
    """Host copies of the inputs the oracle needs for sequences ``rows`` of a device batch: only
    the pages they reference, compacted on the device and renumbered in their block-table rows,
    so every cached token stays where the definition reads it."""
    import torch

    L = batch.seq_lens.cpu().numpy()
    bt = batch.block_table[list(rows)].cpu().numpy()
    lens = L[list(rows)]
    nb = -(-np.maximum(lens, 0) // 16)
    used = np.unique(np.concatenate([bt[i, :nb[i]] for i in range(len(rows))]))
    remap = np.zeros(int(used.max()) + 1, dtype=np.int32)
    remap[used] = np.arange(len(used), dtype=np.int32)
    new_bt = np.zeros_like(bt)
    for i in range(len(rows)):
        new_bt[i, :nb[i]] = remap[bt[i, :nb[i]]]
    idx = torch.as_tensor(used.astype(np.int64), device=batch.k_pages.device)

    def bits(t):
        t = t.cpu().contiguous()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    args = dict(q=bits(batch.q[list(rows)]), k_pages=bits(batch.k_pages.index_select(0, idx)),
                v_pages=bits(batch.v_pages.index_select(0, idx)), block_table=new_bt, seq_lens=lens,
                scale=batch.scale)
    if batch.kv_dtype == "e4m3":
        args["k_scales"] = batch.k_scales.index_select(0, idx).cpu().numpy()
        args["v_scales"] = batch.v_scales.index_select(0, idx).cpu().numpy()
    return args


def parity_vs_gpu(out_gpu, rows, ref) -> dict:
    g = out_gpu[list(rows)].float().cpu().double().numpy()
    err = float(np.abs(g - ref).max())
    rel = float((np.sqrt(((g - ref) ** 2).sum(-1)) / np.maximum(np.sqrt((ref ** 2).sum(-1)), 1e-30)).max())
    return dict(max_abs_err=err, max_row_rel_l2=rel)


def subset_rows(seq_lens: np.ndarray, n: int = 32, seed: int = 123) -> list[int]:
    """n sequences of a batch (all of them if it has fewer): the longest and the shortest, the
    rest a seeded random choice."""
    L = np.asarray(seq_lens)
    if len(L) <= n:
        return list(range(len(L)))
    pick = {int(np.argmax(L)), int(np.argmin(L))}
    for i in np.random.default_rng(seed).permutation(len(L)):
        if len(pick) >= n:
            break
        pick.add(int(i))
    return sorted(pick)


def oracle_timed(args, threads: int, passes: int = 1):
    import oracle

    t0 = time.perf_counter()
    for _ in range(passes):
        ref = oracle.decode_attn(args["q"], args["k_pages"], args["v_pages"], args["block_table"],
                                 args["seq_lens"], args["scale"], k_scales=args.get("k_scales"),
                                 v_scales=args.get("v_scales"), threads=threads)
    return ref, time.perf_counter() - t0


def all_cores() -> int:
    """Threads the oracle uses by default on this host (OpenMP's default, i.e. the cores this
    process may run on unless OMP_NUM_THREADS says otherwise)."""
    import oracle

    return oracle.max_threads(0)


def oracle_subset_baseline(batch, out_gpu, n: int = 32) -> dict:
    """The oracle on a seeded subset of ``n`` sequences (always the longest and the shortest),
    timed once on all cores and once on one core, in GB/s of the subset's algorithmic bytes."""
    L = batch.seq_lens.cpu().numpy()
    rows = subset_rows(L, n)
    args = compact_rows(batch, rows)
    Hq, D = batch.q.shape[1], batch.q.shape[2]
    Hkv = batch.k_pages.shape[1]
    kvb = 1 if batch.kv_dtype == "e4m3" else 2
    nbytes = algorithmic_bytes(L[rows], Hq, Hkv, D, kvb)
    cores = all_cores()
    ref, dt = oracle_timed(args, cores)
    ref1, dt1 = oracle_timed(args, 1)
    sample = (f"{len(rows)} of {len(L)} sequences incl. the longest and the shortest ({int(L[rows].sum())} "
              f"tokens, {nbytes / 1e6:.1f} MB algorithmic), seeded choice, 1 pass")
    return dict(value=round(nbytes / dt / 1e9, 4), unit="GB/s", cores=cores, kind="oracle", seconds=round(dt, 3),
                sample=sample, parity_vs_gpu=parity_vs_gpu(out_gpu, rows, ref),
                single_thread=dict(value=round(nbytes / dt1 / 1e9, 4), unit="GB/s", cores=1, seconds=round(dt1, 3),
                                   sample=sample, same_result_as_all_cores=bool(np.array_equal(ref, ref1))))


def cpu_baseline(batch, out_gpu, target_s: float) -> dict:
    """Time the oracle on all cores on a growing seeded sample of sequences until ~target_s of CPU
    work; when the whole batch takes less than half of that, time repeated passes over it instead.
    ``single_thread``: the 32-sequence subset of ``oracle_subset_baseline`` on one core."""
    L = batch.seq_lens.cpu().numpy()
    order = list(np.random.default_rng(123).permutation(len(L)))
    Hq, D = batch.q.shape[1], batch.q.shape[2]
    Hkv = batch.k_pages.shape[1]
    kvb = 1 if batch.kv_dtype == "e4m3" else 2
    cores = all_cores()

    n = 1
    rows = order[:n]
    args = compact_rows(batch, rows)
    ref, dt = oracle_timed(args, cores)
    while dt < target_s / 4 and n < len(L):
        rate = max(dt, 1e-3) / max(1, int(L[rows].sum()))
        want_tokens = target_s / rate
        cum = np.cumsum(L[order])
        n = int(min(len(L), max(n + 1, np.searchsorted(cum, want_tokens) + 1)))
        rows = order[:n]
        args = compact_rows(batch, rows)
        ref, dt = oracle_timed(args, cores)
    passes = 1
    if n == len(L) and dt < target_s / 2:   # the whole batch is quick: repeat it
        passes = max(2, int(round(target_s / max(dt, 1e-3))))
        ref, dt = oracle_timed(args, cores, passes)
    nbytes = algorithmic_bytes(L[rows], Hq, Hkv, D, kvb) * passes
    sub = oracle_subset_baseline(batch, out_gpu)
    return dict(value=round(nbytes / dt / 1e9, 4), unit="GB/s", cores=cores,
                kind="oracle", seconds=round(dt, 3),
                sample=f"{len(rows)} of {len(L)} sequences ({int(L[rows].sum())} tokens, "
                       f"{nbytes / passes / 1e6:.1f} MB algorithmic), seeded choice, {passes} pass(es)",
                parity_vs_gpu=parity_vs_gpu(out_gpu, rows, ref),
                single_thread=sub["single_thread"])


def measure_attention(workload: str, batch, out, steps: int, warmup: int, workers: int) -> dict:
    """Time ``steps`` whole decode-attention calls on ``batch`` (events around exactly those calls,
    after ``warmup`` untimed ones), then the split-KV kernel alone over ``steps`` more calls (HIP
    events the library records around it on its launch stream)."""
    import torch

    from paper_2504_15930_amd import inputs, sl

    w = inputs.WORKLOADS[workload]
    L = batch.seq_lens.cpu().numpy()
    kvb = 1 if batch.kv_dtype == "e4m3" else 2
    nbytes = algorithmic_bytes(L, w.num_q_heads, w.num_kv_heads, w.head_dim, kvb)
    print(f"[bench] {workload}: warmup {warmup}", file=sys.stderr, flush=True)
    for _ in range(warmup):
        sl.run_batch(batch, out=out, num_workers=workers)
    torch.cuda.synchronize()

    # Pass A: exactly `steps` whole calls, bracketed by events on the stream and
    # nothing else inside the timed region.
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    print(f"[bench] {workload}: timing {steps} steps", file=sys.stderr, flush=True)
    wall0 = time.perf_counter()
    t_all0.record()
    for _ in range(steps):
        sl.run_batch(batch, out=out, num_workers=workers)
    t_all1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0

    # Pass B: the same calls again, each with HIP events that the library
    # records around the split-KV kernel on its launch stream. The extra event
    # records lengthen the step slightly, so this pass only supplies the
    # kernel's duration.
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for e in starts + stops:
        e.record()                          # creates the underlying hipEvent
    t_b0 = torch.cuda.Event(enable_timing=True)
    t_b1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    print(f"[bench] {workload}: timing {steps} split-KV kernels", file=sys.stderr, flush=True)
    t_b0.record()
    for i in range(steps):
        sl.run_batch(batch, out=out, num_workers=workers, timing=(starts[i].cuda_event, stops[i].cuda_event))
    t_b1.record()
    torch.cuda.synchronize()

    step_ms = t_all0.elapsed_time(t_all1) / steps
    kern_ms = [a.elapsed_time(b) for a, b in zip(starts, stops)]
    kern_avg = float(np.mean(kern_ms))
    gbs = nbytes / (step_ms * 1e-3) / 1e9
    achieved = nbytes / (kern_avg * 1e-3) / 1e9
    nw = sl.num_workers(sl.make_desc(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, 16,
                                     batch.block_table.shape[1], batch.k_pages.shape[0], workers), fp8=kvb == 1)
    traffic = traffic_bytes(workload)
    target = TARGET_PCT.get(workload)
    return {
        "ms_per_step": round(step_ms, 5),
        "wall_ms_per_step": round(wall * 1e3 / steps, 5),
        "GBps": round(gbs, 2),
        "pct_of_peak": round(100 * gbs / PEAK_HBM_GBS, 2),
        "steps_per_s": round(1e3 / step_ms, 2),
        "model_layers": MODEL_LAYERS.get(workload),
        "model_steps_per_s": round(1e3 / step_ms / MODEL_LAYERS[workload], 2) if workload in MODEL_LAYERS else None,
        "target_pct_of_peak": target,
        "meets_target": None if target is None else bool(100 * gbs / PEAK_HBM_GBS >= target),
        "config": {
            "workload": workload, "batch": w.batch, "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "page_size": 16,
            "kv_dtype": batch.kv_dtype, "total_tokens": int(L.sum()), "max_seq_len": int(L.max()),
            "algorithmic_bytes": nbytes, "workers": nw,
        },
        "roofline": {
            "kernel": "split_kv_kernel",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "traffic_over_algorithmic": None if traffic is None else round(traffic / nbytes, 4),
            # the HBM bytes the counters saw per launch over this run's kernel time
            "traffic_GBps": None if traffic is None else round(traffic / (kern_avg * 1e-3) / 1e9, 2),
            "kernel_ms": round(kern_avg, 5),
            "ms_per_step_with_kernel_events": round(t_b0.elapsed_time(t_b1) / steps, 5),
            "kernel_ms_p10_p90": [round(float(np.percentile(kern_ms, 10)), 5),
                                  round(float(np.percentile(kern_ms, 90)), 5)],
            "algorithmic_bytes_per_launch": nbytes,
            "kernel_source_sha": kernel_source_hash(),
        },
    }


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen7b_longtail")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--workers", type=int, default=0, help="split-KV workers (0: library default)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline (0 disables every oracle timing)")
    ap.add_argument("--configs", default=",".join(OTHER_CONFIGS),
                    help="comma-separated workloads measured besides --workload ('' for none)")
    ap.add_argument("--generation", type=int, default=1,
                    help="also run a whole long-tail generation (decode engine, LPT vs FIFO admission); 0 skips it")
    ap.add_argument("--dispatch", type=int, default=1,
                    help="also run skewness-aware against random dispatching on the decode engine; 0 skips it")
    ap.add_argument("--prefix", type=int, default=1,
                    help="also time prefix-shared against plain decode attention on a GRPO-like batch; 0 skips it")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="instead of the benchmark, run `steps` plain device-to-device copies of "
                         "BYTES bytes (the reference kernel for scaling HBM counters)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the decode-attention path here runs on a single "
              "MI355X and has no multi-GPU mode; run it with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    from paper_2504_15930_amd import inputs, sl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        n = args.copy_calibration
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "steps": args.steps,
                          "GBps_read_plus_write": round(2 * n / dt / 1e9, 1)}), flush=True)
        return 0
    w = inputs.WORKLOADS[args.workload]
    print(f"[bench] generating {args.workload} (seed {args.seed})", file=sys.stderr, flush=True)
    batch = inputs.make_batch(args.workload, seed=args.seed, device=dev)
    torch.cuda.synchronize()
    L = batch.seq_lens.cpu().numpy()
    kvb = 1 if batch.kv_dtype == "e4m3" else 2
    out = torch.empty_like(batch.q)
    head = measure_attention(args.workload, batch, out, args.steps, args.warmup, args.workers)
    nbytes = head["config"]["algorithmic_bytes"]
    result = {
        "metric": METRIC,
        "value": head["GBps"],
        "unit": "GB/s",
        "pct_of_peak": head["pct_of_peak"],
        "steps_per_s": head["steps_per_s"],
        "model_steps_per_s": head["model_steps_per_s"],
        "target_pct_of_peak": head["target_pct_of_peak"],
        "meets_target": head["meets_target"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "wall_ms_per_step": head["wall_ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "e4m3" if kvb == 1 else "bf16",
        "accumulate": "f32",
        "data": "synthetic",
        "config": dict(head["config"], seed=args.seed),
        "roofline": head["roofline"],
    }
    # KV append (the step before attention) and the whole decode step (append +
    # attention). The new rows overwrite each sequence's newest slot, so
    # repeating the step leaves the sequence lengths and the bytes unchanged.
    print(f"[bench] kv append + decode step, {args.steps} steps", file=sys.stderr, flush=True)
    gen = torch.Generator(device=dev).manual_seed(args.seed + 7)
    B, Hq, D = batch.q.shape
    Hkv = batch.k_pages.shape[1]
    k_new = torch.randn((B, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
    v_new = torch.randn((B, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
    fp8_kw = dict(k_scales=batch.k_scales, v_scales=batch.v_scales) if kvb == 1 else {}

    def append(timing=None):
        sl.kv_append(k_new, v_new, batch.block_table, batch.seq_lens, batch.k_pages, batch.v_pages,
                     num_q_heads=Hq, timing=timing, **fp8_kw)

    for _ in range(args.warmup):
        append()
        sl.run_batch(batch, out=out, num_workers=args.workers)
    torch.cuda.synchronize()
    d0 = torch.cuda.Event(enable_timing=True)
    d1 = torch.cuda.Event(enable_timing=True)
    d0.record()
    for _ in range(args.steps):
        append()
        sl.run_batch(batch, out=out, num_workers=args.workers)
    d1.record()
    torch.cuda.synchronize()
    decode_ms = d0.elapsed_time(d1) / args.steps
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for e in starts + stops:
        e.record()
    for i in range(args.steps):
        append(timing=(starts[i].cuda_event, stops[i].cuda_event))
    torch.cuda.synchronize()
    app_ms = float(np.mean([s.elapsed_time(e) for s, e in zip(starts, stops)]))
    app_bytes = append_bytes(L, Hkv, D, kvb)
    result["kv_append"] = {
        "kernel": "append_kernel", "bound": "latency", "kernel_ms": round(app_ms, 5),
        "algorithmic_bytes_per_launch": app_bytes,
        "achieved": round(app_bytes / (app_ms * 1e-3) / 1e9, 2), "unit": "GB/s",
        "frac_of_hbm_peak": round(app_bytes / (app_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 5),
    }
    result["decode_step"] = {
        "what": "kv append + decode attention, one layer", "ms_per_step": round(decode_ms, 5),
        "steps_per_s": round(1e3 / decode_ms, 2),
        "GBps": round((nbytes + app_bytes) / (decode_ms * 1e-3) / 1e9, 2),
    }
    if args.cpu_seconds > 0:
        # The appends above rewrote each sequence's newest slot: run the step once more so the
        # output the oracle is compared with belongs to the cache as it now stands.
        sl.run_batch(batch, out=out, num_workers=args.workers)
        torch.cuda.synchronize()
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(batch, out, args.cpu_seconds)
    else:
        result["cpu_baseline"] = None

    # The other decode steps, one batch resident at a time.
    configs = [c for c in args.configs.split(",") if c and c != args.workload]
    if configs:
        del batch, out, k_new, v_new
        torch.cuda.empty_cache()
        result["configs"] = {}
        for name in configs:
            print(f"[bench] generating {name} (seed {args.seed})", file=sys.stderr, flush=True)
            cb = inputs.make_batch(name, seed=args.seed, device=dev)
            cout = torch.empty_like(cb.q)
            torch.cuda.synchronize()
            r = measure_attention(name, cb, cout, args.steps, args.warmup, args.workers)
            if args.cpu_seconds > 0:
                print(f"[bench] {name}: cpu baseline (oracle, subset)", file=sys.stderr, flush=True)
                r["cpu_baseline"] = oracle_subset_baseline(cb, cout)
            result["configs"][name] = r
            del cb, cout
            torch.cuda.empty_cache()

    if args.prefix:
        print("[bench] prefix sharing", file=sys.stderr, flush=True)
        result["prefix"] = prefix_experiment(w, args.seed, dev, args.steps, args.warmup)
        print("[bench] prefix sharing, 16 samples per prompt", file=sys.stderr, flush=True)
        result["prefix_16"] = prefix_experiment(w, args.seed, dev, args.steps, args.warmup, prompts=16, samples=16)
    if args.generation:
        result["generation"] = generation(w, kvb == 1, args.seed, dev)
    if args.dispatch:
        result["dispatch"] = dispatch_experiment(w, args.seed, dev, stream_gbs=result["roofline"]["achieved"])
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
