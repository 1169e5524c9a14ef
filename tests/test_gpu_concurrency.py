"""Two host threads calling the library at the same time, each on its own stream.

Each thread runs decode attention on its own batch (one bf16 cache, one E4M3)
on a torch stream of its own, so the binding gives each stream its own cached
workspace and the library's per-device information is read from both threads
at once. Every output must equal, bit for bit, the same call made alone
beforehand: the kernels' results depend only on their inputs.
"""
import threading

import numpy as np
import pytest
import torch

from paper_2504_15930_amd import inputs, sl

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")]
DEV = "cuda:0"
CALLS = 25


def test_two_threads_on_two_streams_match_calls_made_alone():
    rng = np.random.default_rng(71)
    batches = [
        inputs.make_paged_batch(rng.integers(1, 3000, 64), 28, 4, 128, seed=72, device=DEV, kv_dtype="bf16",
                                poison=False),
        inputs.make_paged_batch(rng.integers(1, 5000, 48), 28, 4, 128, seed=73, device=DEV, kv_dtype="e4m3",
                                poison=False),
    ]
    want = [sl.run_batch(b).clone() for b in batches]
    torch.cuda.synchronize()
    outs = [[torch.empty_like(b.q) for _ in range(CALLS)] for b in batches]
    streams = [torch.cuda.Stream(device=DEV) for _ in batches]
    errors = []
    start = threading.Barrier(len(batches))

    def work(i):
        try:
            with torch.cuda.stream(streams[i]):
                start.wait()
                for k in range(CALLS):
                    sl.run_batch(batches[i], out=outs[i][k])
            streams[i].synchronize()
        except Exception as e:   # handed to the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(batches))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i, b in enumerate(batches):
        ref = want[i].view(torch.int16)
        for k in range(CALLS):
            assert torch.equal(outs[i][k].view(torch.int16), ref), f"{b.kv_dtype} call {k} differs"
