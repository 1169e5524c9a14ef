"""Seeded synthetic decode batches (shared by the GPU path's tests and by the oracle).

This module only *draws inputs*; it holds none of the attention arithmetic.
Both sides of every parity check receive the very same tensors from here.

Workloads follow the shape of StreamRL's generation stage: a decode batch of
hundreds of in-flight samples whose output lengths are long-tailed (Section 2.4,
"skewness bubbles"; Section 7 setup, "Dataset": maximum output 20K, very
long-tail), with Qwen2.5-7B / -72B head counts (Table "LLM specifications",
Section 7 setup, "Models"). The paper's own prompts and responses are not used;
lognormal generated lengths stand in for its long-tail output-length
distribution.

Recipe (every workload):
  1. ``rng = numpy.random.default_rng(seed)`` draws the lengths first, then the
     physical page assignment (a permutation of the pool, cut into one run per
     sequence).
  2. q, K, V are ``torch.randn`` (fp32, standard normal) rounded to bf16, from
     ``torch.Generator`` objects seeded with seed+1, seed+2, seed+3 on the
     device the tensors are made on.
  3. Pool slots that hold no live token (slots past the end of a sequence's last
     page, pages no sequence references) are filled with NaN, and padding
     entries of the block table point at an all-NaN "poison" page, so any read
     outside the live tokens shows up in the result.
  4. FP8 workloads quantise the bf16 K/V per (page, KV head): scale =
     max|x| / 448 over the live slots (1 when that is 0), codes = round-to-
     nearest-even of x / scale saturated to +-448 (OCP E4M3); non-live slots get
     the NaN code 0x7F.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

PAGE_SIZE = 16
E4M3_MAX = 448.0
E4M3_NAN = 0x7F


@dataclass(frozen=True)
class Workload:
    """A named decode-step shape: batch, heads, head_dim and a length law."""

    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    lengths: str                 # "uniform" (lo, hi inclusive) or "lognormal"
    params: tuple                # uniform: (lo, hi); lognormal: (prompt, median, sigma, cap)
    kv_dtype: str = "bf16"       # "bf16" or "e4m3"
    fixed_pool: int = 0          # >0: pool of this many pages, table = perm(pool).reshape(B, -1)
    description: str = ""
    page_size: int = PAGE_SIZE


WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("tiny", 8, 4, 2, 64, "uniform", (1, 256), fixed_pool=160,
                 description="single decode step, batch 8, 4 q / 2 kv heads, D=64, "
                             "lengths uniform in [1,256], 160-page pool"),
        Workload("qwen7b_longtail", 256, 28, 4, 128, "lognormal", (512, 2048, 1.0, 16384),
                 description="7B-like decode step: batch 256, 28 q / 4 kv heads, D=128, "
                             "512 prompt + lognormal(median 2048, sigma 1.0) capped 16384"),
        Workload("straggler", 16, 64, 8, 128, "uniform", (8192, 32768),
                 description="straggler tail: batch 16, 64 q / 8 kv heads, D=128, "
                             "lengths uniform in [8192,32768]"),
        Workload("qwen72b_longtail", 512, 64, 8, 128, "lognormal", (1024, 4096, 1.2, 32768),
                 description="72B-like decode step: batch 512, 64 q / 8 kv heads, D=128, "
                             "1024 prompt + lognormal(median 4096, sigma 1.2) capped 32768"),
        Workload("fp8_qwen7b_longtail", 512, 28, 4, 128, "lognormal", (512, 2048, 1.0, 32768),
                 kv_dtype="e4m3",
                 description="FP8 KV cache: batch 512, 28 q / 4 kv heads, D=128, e4m3 K/V with "
                             "per-(page, kv head) fp32 scales, 512 prompt + lognormal(2048, 1.0) "
                             "capped 32768"),
    ]
}


def draw_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    """Sequence lengths of workload ``w`` (int64 [B]) drawn from ``rng``."""
    if w.lengths == "uniform":
        lo, hi = w.params
        return rng.integers(lo, hi + 1, w.batch).astype(np.int64)
    if w.lengths == "lognormal":
        prompt, median, sigma, cap = w.params
        x = rng.lognormal(math.log(median), sigma, w.batch)
        return prompt + np.clip(np.floor(x), 1, cap).astype(np.int64)
    raise ValueError(f"unknown length law {w.lengths!r}")


@dataclass
class Batch:
    """One decode step's inputs, on one device."""

    q: torch.Tensor                 # bf16 [B, Hq, D]
    k_pages: torch.Tensor           # bf16 or uint8 [N, Hkv, P, D]
    v_pages: torch.Tensor
    block_table: torch.Tensor       # int32 [B, max_blocks]
    seq_lens: torch.Tensor          # int32 [B]
    scale: float                    # fp32 value of 1/sqrt(D)
    k_scales: torch.Tensor | None = None   # float32 [N, Hkv] (e4m3 only)
    v_scales: torch.Tensor | None = None
    poison_page: int = -1           # id of the all-NaN page (-1: none)
    meta: dict = field(default_factory=dict)

    @property
    def kv_dtype(self) -> str:
        return "bf16" if self.k_pages.dtype == torch.bfloat16 else "e4m3"

    def host_arrays(self) -> dict:
        """numpy views for the oracle: bf16 as uint16 bit patterns, e4m3 as uint8."""
        def bits(t):
            t = t.detach().cpu().contiguous()
            if t.dtype == torch.bfloat16:
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
        d = dict(q=bits(self.q), k_pages=bits(self.k_pages), v_pages=bits(self.v_pages),
                 block_table=self.block_table.cpu().numpy(), seq_lens=self.seq_lens.cpu().numpy(),
                 scale=self.scale)
        if self.k_scales is not None:
            d["k_scales"] = self.k_scales.cpu().numpy()
            d["v_scales"] = self.v_scales.cpu().numpy()
        return d


def _randn_bf16(shape, seed: int, device, chunk_rows: int = 1 << 14) -> torch.Tensor:
    """Standard-normal fp32 draws rounded to bf16, generated in chunks along dim 0."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    rows = shape[0]
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        out[r0:r1] = torch.randn((r1 - r0, *shape[1:]), generator=gen, device=device,
                                 dtype=torch.float32).to(torch.bfloat16)
    return out


def _live_slots(block_table: np.ndarray, lengths: np.ndarray, num_pages: int, P: int) -> np.ndarray:
    """bool [num_pages, P]: slot holds a token some sequence attends to."""
    live = np.zeros((num_pages, P), dtype=bool)
    for b, L in enumerate(lengths):
        L = int(L)
        if L <= 0:
            continue
        nb = -(-L // P)
        pages = block_table[b, :nb]
        live[pages[:-1]] = True
        last = L - (nb - 1) * P
        live[pages[-1], :last] = True
    return live


def make_paged_batch(lengths, num_q_heads: int, num_kv_heads: int, head_dim: int, *,
                     seed: int = 0, device="cpu", kv_dtype: str = "bf16",
                     block_table: np.ndarray | None = None, num_pages: int | None = None,
                     rng: np.random.Generator | None = None, page_size: int = PAGE_SIZE,
                     poison: bool = True, meta: dict | None = None) -> Batch:
    """A decode batch with the given lengths.

    When ``block_table`` is None the pool holds exactly the pages the sequences
    need plus one poison page; a random permutation of the pool (drawn from
    ``rng``, default ``default_rng(seed)``) is cut into one run per sequence and
    padding entries point at the poison page. A caller-supplied table (e.g.
    with aliasing rows) must come with ``num_pages``.
    """
    P = page_size
    lengths = np.asarray(lengths, dtype=np.int64)
    B = lengths.shape[0]
    if rng is None:
        rng = np.random.default_rng(seed)
    npg = -(-lengths // P)
    poison_page = -1
    if block_table is None:
        total = int(npg.sum())
        perm = rng.permutation(total).astype(np.int32)
        max_blocks = max(1, int(npg.max()) if B else 1)
        poison_page = total
        block_table = np.full((B, max_blocks), poison_page, dtype=np.int32)
        cum = np.concatenate([[0], np.cumsum(npg)])
        for b in range(B):
            block_table[b, :npg[b]] = perm[cum[b]:cum[b + 1]]
        num_pages = total + 1
    else:
        block_table = np.ascontiguousarray(block_table, dtype=np.int32)
        if num_pages is None:
            raise ValueError("num_pages is required with an explicit block_table")
    dev = torch.device(device)
    D, Hkv = head_dim, num_kv_heads
    q = _randn_bf16((B, num_q_heads, D), seed + 1, dev)
    k = _randn_bf16((num_pages, Hkv, P, D), seed + 2, dev)
    v = _randn_bf16((num_pages, Hkv, P, D), seed + 3, dev)
    live_np = _live_slots(block_table, lengths, num_pages, P)
    live = torch.from_numpy(live_np).to(dev)[:, None, :, None]
    if poison:
        nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=dev)
        k = torch.where(live, k, nan)
        v = torch.where(live, v, nan)
    batch = Batch(q=q, k_pages=k, v_pages=v,
                  block_table=torch.from_numpy(block_table).to(dev),
                  seq_lens=torch.from_numpy(lengths.astype(np.int32)).to(dev),
                  scale=float(np.float32(1.0 / math.sqrt(D))), poison_page=poison_page,
                  meta=dict(meta or {}, seed=seed))
    if kv_dtype == "e4m3":
        batch.k_pages, batch.k_scales = quantize_e4m3(k, live)
        batch.v_pages, batch.v_scales = quantize_e4m3(v, live)
    elif kv_dtype != "bf16":
        raise ValueError(f"unknown kv dtype {kv_dtype!r}")
    return batch


def quantize_e4m3(x: torch.Tensor, live: torch.Tensor, chunk: int = 1 << 13):
    """Per-(page, head) E4M3 codes (uint8) and fp32 scales of a bf16 page pool.

    ``live`` is a bool mask broadcastable to ``x`` ([N, 1, P, 1]); dead slots get
    the NaN code and do not contribute to the scale.
    """
    N, H, P, D = x.shape
    codes = torch.empty((N, H, P, D), dtype=torch.uint8, device=x.device)
    scales = torch.empty((N, H), dtype=torch.float32, device=x.device)
    for n0 in range(0, N, chunk):
        n1 = min(N, n0 + chunk)
        xs = x[n0:n1].float()
        lv = live[n0:n1]
        amax = torch.where(lv, xs.abs(), torch.zeros((), device=x.device)).amax(dim=(2, 3))
        sc = torch.where(amax > 0, amax / E4M3_MAX, torch.ones((), device=x.device))
        y = (xs / sc[:, :, None, None]).clamp(-E4M3_MAX, E4M3_MAX)
        c = y.to(torch.float8_e4m3fn).view(torch.uint8)
        c = torch.where(lv, c, torch.full((), E4M3_NAN, dtype=torch.uint8, device=x.device))
        codes[n0:n1] = c
        scales[n0:n1] = sc
    return codes, scales


def make_grpo_batch(num_prompts: int, samples: int, prompt_len: int, *, seed: int = 0, device="cpu",
                    num_q_heads: int = 28, num_kv_heads: int = 4, head_dim: int = 128,
                    gen_median: float = 512.0, gen_sigma: float = 1.0, gen_cap: int = 4096,
                    poison: bool = True, kv_dtype: str = "bf16"):
    """A GRPO-like decode batch: ``samples`` consecutive sequences per prompt share the prompt's
    floor(prompt_len / 16) full pages (same page ids, hence the same tokens) and continue on
    pages of their own; each has generated floor(X) tokens, ln X ~ N(ln gen_median, gen_sigma^2),
    clipped to [0, gen_cap]. ``kv_dtype`` "e4m3" stores the pages as E4M3 codes with
    per-(page, KV head) scales. Returns (batch, group_start [num_prompts + 1], shared_pages
    [num_prompts]) with the two int32 tensors on ``device``."""
    rng = np.random.default_rng(seed)
    B = num_prompts * samples
    gen = np.clip(np.floor(np.exp(rng.normal(np.log(gen_median), gen_sigma, B))), 0, gen_cap).astype(np.int64)
    lengths = prompt_len + gen
    sp = prompt_len // PAGE_SIZE
    own = -(-lengths // PAGE_SIZE) - sp
    total = num_prompts * sp + int(own.sum())
    perm = rng.permutation(total).astype(np.int32)
    poison_page = total
    max_blocks = max(1, int((-(-lengths // PAGE_SIZE)).max()))
    table = np.full((B, max_blocks), poison_page, dtype=np.int32)
    pos = 0
    for k in range(num_prompts):
        common = perm[pos:pos + sp]
        pos += sp
        for b in range(k * samples, (k + 1) * samples):
            table[b, :sp] = common
            table[b, sp:sp + own[b]] = perm[pos:pos + own[b]]
            pos += own[b]
    batch = make_paged_batch(lengths, num_q_heads, num_kv_heads, head_dim, seed=seed, device=device,
                             kv_dtype=kv_dtype, block_table=table, num_pages=total + 1, rng=rng, poison=poison,
                             meta=dict(workload="grpo", prompts=num_prompts, samples=samples, prompt_len=prompt_len))
    batch.poison_page = poison_page
    dev = torch.device(device)
    starts = torch.arange(0, B + 1, samples, dtype=torch.int32, device=dev)
    shared = torch.full((num_prompts,), sp, dtype=torch.int32, device=dev)
    return batch, starts, shared


def make_batch(name: str, seed: int = 0, device="cpu", poison: bool = True) -> Batch:
    """The named workload's decode step, drawn with ``seed``."""
    w = WORKLOADS[name]
    rng = np.random.default_rng(seed)
    lengths = draw_lengths(w, rng)
    meta = dict(workload=w.name, description=w.description)
    if w.fixed_pool:
        table = rng.permutation(w.fixed_pool).astype(np.int32).reshape(w.batch, -1)
        return make_paged_batch(lengths, w.num_q_heads, w.num_kv_heads, w.head_dim, seed=seed,
                                device=device, kv_dtype=w.kv_dtype, block_table=table,
                                num_pages=w.fixed_pool, rng=rng, page_size=w.page_size,
                                poison=poison, meta=meta)
    return make_paged_batch(lengths, w.num_q_heads, w.num_kv_heads, w.head_dim, seed=seed,
                            device=device, kv_dtype=w.kv_dtype, rng=rng,
                            page_size=w.page_size, poison=poison, meta=meta)
