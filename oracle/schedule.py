"""Reference for the multi-step decode loop's scheduling (continuous batching with
longest-processing-time-first admission) and its KV page bookkeeping.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this module. Plain Python, no
numerics: every result is an integer and is compared exactly.

What it computes (StreamRL Section 5.3, "Scheduling Order"). An instance holds
more samples than its batch size BS, so samples run in several rounds. The
batch is BS parallel slots; each decode step every occupied slot generates
one token of its sample; a sample needing ``o`` output tokens occupies its slot
for ``o`` consecutive steps (continuous batching, Section 6, releases it as
soon as it finishes). Samples enter in descending order of their estimated
output length (LPT, a 4/3-approximation of the minimum makespan, Graham
1969), and whenever a sample finishes the next sample in that order takes the
freed slot. ``order="fifo"`` admits in index order instead.

Readings where the paper is silent:
  * ties in the estimated length keep index order;
  * freed slots are refilled before the next step, lowest slot first;
  * sample i brings a prompt of p_i tokens whose KV pages exist on admission;
    during the step in which it generates its k-th token (k = 1..o_i) its
    sequence length is p_i + k (the new token included), so the new token's
    position is p_i + k - 1;
  * KV pages (16 tokens) come from one LIFO free stack that initially pops
    0, 1, 2, ...; a sample takes ceil(p_i / 16) pages on admission (block
    order) and one more page in every step whose new token starts a page; a
    finished sample's pages are pushed back last block first, so they are
    popped again in block order.
"""
from __future__ import annotations

from dataclasses import dataclass, field

PAGE = 16


@dataclass
class Schedule:
    makespan: int                                  # decode steps until every sample is done
    slot: list[int]                                # per sample
    admit_step: list[int]                          # first step the sample generates in
    finish_step: list[int]                         # last step the sample generates in
    checkpoints: dict = field(default_factory=dict)  # step -> (seq_lens, block_table rows)


def admission_order(est_len, order: str = "lpt") -> list[int]:
    """Sample indices in admission order: LPT = descending estimate, ties by index."""
    idx = list(range(len(est_len)))
    if order == "lpt":
        return sorted(idx, key=lambda i: (-int(est_len[i]), i))
    if order == "fifo":
        return idx
    raise ValueError(order)


def simulate(prompt_len, output_len, est_len, batch_slots: int, num_pages: int, max_blocks: int,
             order: str = "lpt", checkpoints=()) -> Schedule:
    """Run the loop to completion. ``checkpoints`` names steps whose per-slot sequence
    lengths and block tables (as the device would hold them during that step) are kept."""
    M = len(output_len)
    assert len(prompt_len) == M and len(est_len) == M
    assert all(int(o) >= 1 for o in output_len) and all(int(p) >= 0 for p in prompt_len)
    queue = admission_order(est_len, order)
    head = 0
    free = list(range(num_pages - 1, -1, -1))      # pop() -> 0, 1, 2, ...
    occupant = [-1] * batch_slots                  # sample in each slot
    made = [0] * batch_slots                       # tokens generated so far by that sample
    pages = [[] for _ in range(batch_slots)]       # pages held, block order
    table = [[-1] * max_blocks for _ in range(batch_slots)]
    slot = [-1] * M
    admit = [-1] * M
    finish = [-1] * M
    kept = {}
    want = set(checkpoints)
    step = 0
    while True:
        for b in range(batch_slots):               # refill free slots, lowest first
            if occupant[b] < 0 and head < M:
                i = queue[head]
                head += 1
                occupant[b], made[b] = i, 0
                slot[i], admit[i] = b, step
                n = -(-int(prompt_len[i]) // PAGE)
                assert n <= max_blocks
                pages[b] = [free.pop() for _ in range(n)]
                for blk, pg in enumerate(pages[b]):
                    table[b][blk] = pg
        if all(o < 0 for o in occupant):
            break
        lens = [0] * batch_slots
        for b in range(batch_slots):
            i = occupant[b]
            if i < 0:
                continue
            t = int(prompt_len[i]) + made[b]       # position of this step's token
            if t % PAGE == 0:
                assert t // PAGE == len(pages[b]) < max_blocks
                pg = free.pop()
                pages[b].append(pg)
                table[b][t // PAGE] = pg
            lens[b] = t + 1
        if step in want:
            kept[step] = (list(lens), [list(r) for r in table])
        for b in range(batch_slots):               # the step runs; then bookkeeping
            i = occupant[b]
            if i < 0:
                continue
            made[b] += 1
            if made[b] == int(output_len[i]):
                finish[i] = step
                for pg in reversed(pages[b]):
                    free.append(pg)
                pages[b] = []
                occupant[b] = -1
        step += 1
    return Schedule(makespan=step, slot=slot, admit_step=admit, finish_step=finish, checkpoints=kept)


def makespan_of_list_schedule(sizes, machines: int, order) -> int:
    """Greedy list scheduling of jobs ``sizes`` taken in ``order`` on identical machines:
    each job goes to the machine that becomes free first (lowest index on ties)."""
    loads = [0] * machines
    for j in order:
        m = min(range(machines), key=lambda k: (loads[k], k))
        loads[m] += int(sizes[j])
    return max(loads) if loads else 0
