"""Planted mistakes in the scheduling oracle (oracle/schedule.py) must trip a pin.

Each case copies the module, plants one plausible mistake (admission order,
tie-break, refill order, timing of admission, page accounting) and runs every
pin of test_schedule_oracle against the copy.
"""
import importlib.util
import os
import sys

import pytest

import test_schedule_oracle as pins
from oracle import schedule as S

MUTANTS = [
    ("lpt_ascending", "key=lambda i: (-int(est_len[i]), i)", "key=lambda i: (int(est_len[i]), i)"),
    ("ties_reversed", "key=lambda i: (-int(est_len[i]), i)", "key=lambda i: (-int(est_len[i]), -i)"),
    ("order_by_true_length", "queue = admission_order(est_len, order)", "queue = admission_order(output_len, order)"),
    ("refill_highest_slot_first", "for b in range(batch_slots):               # refill",
     "for b in reversed(range(batch_slots)):     # refill"),
    ("pages_returned_in_block_order", "for pg in reversed(pages[b]):", "for pg in pages[b]:"),
    ("finish_one_step_late", "if made[b] == int(output_len[i]):", "if made[b] == int(output_len[i]) + 1:"),
    ("length_excludes_new_token", "lens[b] = t + 1", "lens[b] = t"),
    ("new_page_off_by_one", "if t % PAGE == 0:", "if t % PAGE == 1:"),
]


def _load_mutant(tmp_path, name, old, new):
    src = open(S.__file__).read()
    assert old in src, f"mutation target not found: {old!r}"
    path = os.path.join(tmp_path, f"schedule_{name}.py")
    with open(path, "w") as f:
        f.write(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location(f"schedule_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod          # dataclasses look their module up there
    try:
        spec.loader.exec_module(mod)
    finally:
        sys.modules.pop(spec.name, None)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    mod = _load_mutant(str(tmp_path), name, old, new)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, IndexError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} survived every pin"
