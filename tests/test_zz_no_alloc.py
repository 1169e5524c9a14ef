"""sl_decode_attn_noalloc (the entry point that allocates nothing) against sl_decode_attn and the
oracle, through the C ABI: two calls in a row on the library's fixed scratch array, the second on
a smaller batch, then the 7B-like long-tail batch at full size with the default worker count, and
replays of a call captured in a HIP graph."""
import numpy as np
import pytest
import torch

from paper_2504_15930_amd import inputs, sl
from parity import assert_parity, oracle_full, oracle_rows, sample_rows

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")]
DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)


def _bits(t):
    return t.detach().cpu().view(torch.int16)


def _lognormal_lengths(B, seed, median, cap):
    rng = np.random.default_rng(seed)
    return np.clip(np.exp(rng.normal(np.log(median), 1.0, B)), 1, cap).astype(np.int64)


@pytest.mark.parametrize("workers", [0, 7])
def test_two_calls_second_smaller(workers):
    first = inputs.make_paged_batch(_lognormal_lengths(48, 1, 600, 4000), 28, 4, 128, seed=3, device=DEV)
    L2 = _lognormal_lengths(9, 2, 100, 700)
    L2[0] = 1   # a single-token context and an empty sequence in the second call
    L2[1] = 0
    second = inputs.make_paged_batch(L2, 28, 4, 128, seed=4, device=DEV)
    for name, b in (("first", first), ("second (smaller)", second)):
        _say("noalloc", name, "workers", workers, "batch", b.q.shape[0])
        want = sl.decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale,
                              num_workers=workers)
        got = sl.decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale,
                                     num_workers=workers)
        torch.cuda.synchronize()
        assert torch.equal(_bits(got), _bits(want)), f"{name}: differs from sl_decode_attn"
        assert_parity(got, oracle_full(b), f"noalloc {name} workers={workers}")


def test_full_size_7b_like():
    b = inputs.make_batch("qwen7b_longtail", seed=0, device=DEV)
    _say("noalloc qwen7b_longtail, default workers")
    want = sl.run_batch(b)
    got = sl.decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
    torch.cuda.synchronize()
    assert torch.equal(_bits(got), _bits(want))
    rows = sample_rows(b.seq_lens, 8, seed=5)
    assert_parity(got[rows], oracle_rows(b, rows), "noalloc qwen7b_longtail")


def test_scratch_limit_rejected_before_launch():
    b = inputs.make_paged_batch([5, 9], 32, 2, 128, seed=6, device=DEV)
    out = torch.full_like(b.q, 7.0)
    with pytest.raises(sl.SlError) as e:
        sl.decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale, out=out,
                               num_workers=65536)
    assert e.value.status == -7
    torch.cuda.synchronize()
    assert bool((out.float() == 7.0).all()), "a rejected call enqueued work"


def test_replays_of_a_captured_call():
    """The use the entry point exists for: one call captured in a HIP graph (through torch's graph
    capture, after one eager call that looks up the scratch address), replayed five times with eager
    work between the replays (the queries rewritten, an unrelated call on a workspace); every replay
    equals sl_decode_attn on the same inputs, bit for bit."""
    rng = np.random.default_rng(5)
    lens = np.clip(np.exp(rng.normal(np.log(500), 1.0, 40)), 1, 3000).astype(np.int64)
    b = inputs.make_paged_batch(lens, 28, 4, 128, seed=6, device=DEV, poison=False)
    other = inputs.make_paged_batch(rng.integers(1, 900, 12), 16, 2, 64, seed=7, device=DEV, poison=False)
    out = torch.empty_like(b.q)
    sl.decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale, out=out)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sl.decode_attn_noalloc(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale, out=out)
    gen = torch.Generator(device=DEV).manual_seed(8)
    for r in range(5):
        print("graph replay", r, flush=True)
        b.q.copy_(torch.randn(b.q.shape, generator=gen, device=DEV).to(torch.bfloat16))
        sl.run_batch(other)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = sl.decode_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.seq_lens, b.scale)
        torch.cuda.synchronize()
        assert torch.equal(_bits(out), _bits(want)), f"replay {r} differs"
