"""Planted mistakes in the oracle must trip at least one pin.

Each case copies one oracle source (``oracle/oracle.c`` for decode attention,
``oracle/append.c`` for the KV append), plants one plausible mistake (a dropped
term, a wrong index, a transposed layout, a wrong constant), builds the copy
with the other sources on the CPU and runs every pin of ``oracle_pins`` against
it in a child process, so that a mutant which crashes also counts as caught.
The real oracle is never modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle import build as oracle_build

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)

# (name, original text, replacement, which occurrence (0-based)[, source file])
MUTANTS = [
    ("head_map_modulo", "int g = h / G;", "int g = h % Hkv;", 0),
    ("block_table_transposed", "block_table[(size_t)b * max_blocks + t / P]",
     "block_table[(size_t)(t / P) * max_blocks + b]", 0),
    ("slot_off_by_one", "int slot = t % P;", "int slot = (t + 1) % P;", 0),
    ("slot_off_by_one_pass2", "int slot = t % P;", "int slot = (t + 1) % P;", 1),
    ("scale_dropped", "s[t] = scale * dot;", "s[t] = dot;", 0),
    ("no_max_subtraction", "double w = exp(s[t] - m);", "double w = exp(s[t]);", 0),
    ("min_not_max", "if (s[t] > m)", "if (s[t] < m)", 0),
    ("max_starts_at_zero", "m = s[0];", "m = 0.0;", 0),
    ("not_normalised", "out_row[d] /= z;", "out_row[d] /= 1.0;", 0),
    ("sum_counts_tokens", "z += w;", "z += 1.0;", 0),
    ("layout_head_slot_swapped", "size_t idx = (((size_t)page * Hkv + g) * P + slot) * D + d;",
     "size_t idx = (((size_t)page * P + slot) * Hkv + g) * D + d;", 0),
    ("query_row_of_kv_head", "q + ((size_t)b * Hq + h) * D", "q + ((size_t)b * Hq + g) * D", 0),
    ("last_token_dropped", "for (t = 0; t < L; ++t) {", "for (t = 0; t < L - 1; ++t) {", 1),
    ("e4m3_bias", "mag = ldexp(1.0 + (double)m / 8.0, e - 7);",
     "mag = ldexp(1.0 + (double)m / 8.0, e - 8);", 0),
    ("e4m3_subnormal_exponent", "mag = ldexp((double)m / 8.0, 1 - 7);",
     "mag = ldexp((double)m / 8.0, -7);", 0),
    ("e4m3_positive_nan_missed", "if (e == 0xF && m == 0x7)", "if (e == 0xF && m == 0x7 && sign)", 0),
    ("key_uses_value_scales", "kv_value(kv_kind, k_pages, k_scales,",
     "kv_value(kv_kind, k_pages, v_scales,", 0),
    ("scale_ignores_head", "scales[(size_t)page * Hkv + g]", "scales[(size_t)page * Hkv]", 0),
    ("bf16_shift", "uint32_t u = (uint32_t)bits << 16;", "uint32_t u = (uint32_t)bits << 15;", 0),
    # KV append / E4M3 quantise-on-write
    ("append_after_new_token", "const int t = L - 1;", "const int t = L;", 0, "append.c"),
    ("append_head_stride", "const size_t tile = ((size_t)page * Hkv + g) * P * D;",
     "const size_t tile = ((size_t)page * Hkv) * P * D;", 0, "append.c"),
    ("append_scale_never_grows", "if (a <= reach) {", "if (1) {", 0, "append.c"),
    ("append_no_reencode", "for (int j = 0; j < slot; ++j)", "for (int j = 0; j < 0; ++j)", 0, "append.c"),
    ("append_reencode_keeps_old_scale", "*c = sl_oracle_e4m3_encode(v / s);",
     "*c = sl_oracle_e4m3_encode(v / s_old);", 0, "append.c"),
    ("append_fresh_page_keeps_scale", "if (slot == 0) {", "if (0) {", 0, "append.c"),
    ("append_amax_signed", "const float v = fabsf(bf16_to_float(x[d]));", "const float v = bf16_to_float(x[d]);",
     0, "append.c"),
    ("append_kv_scales_swapped", "&k_scales[(size_t)page * Hkv + g]);", "&v_scales[(size_t)page * Hkv + g]);",
     0, "append.c"),
    ("encode_truncates", "double k = nearbyint((m - 1.0) * 8.0);", "double k = floor((m - 1.0) * 8.0);", 0,
     "append.c"),
    ("encode_no_saturation", "if (a >= 448.0)", "if (a >= 1e300)", 0, "append.c"),
    ("encode_subnormal_step", "nearbyint(a / ldexp(1.0, -9))", "nearbyint(a / ldexp(1.0, -10))", 0, "append.c"),
    ("encode_nan_as_zero", "return 0x7F;", "return 0x00;", 0, "append.c"),
]

CHILD = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle_pins
failed = []
for pin in oracle_pins.ALL_PINS:
    try:
        pin({lib!r})
    except (AssertionError, ValueError) as e:
        failed.append(pin.__name__)
print("FAILED:", ",".join(failed))
sys.exit(1 if failed else 0)
"""


def _mutate(src: str, old: str, new: str, occurrence: int) -> str:
    start = -1
    for _ in range(occurrence + 1):
        start = src.find(old, start + 1)
        assert start >= 0, f"mutation target not found: {old!r} #{occurrence}"
    return src[:start] + new + src[start + len(old):]


def _run_mutant(tmpdir, name, old, new, occ, fname="oracle.c"):
    sources = []
    for src_path in oracle_build.SOURCES:
        if os.path.basename(src_path) == fname:
            with open(src_path) as f:
                src = f.read()
            path = os.path.join(tmpdir, f"{name}_{fname}")
            with open(path, "w") as f:
                f.write(_mutate(src, old, new, occ))
            sources.append(path)
        else:
            sources.append(src_path)
    assert len(sources) == len(oracle_build.SOURCES) and any(tmpdir in s for s in sources), fname
    lib = oracle_build.build(sources, os.path.join(tmpdir, f"lib{name}.so"), extra=["-w"])
    env = dict(os.environ, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-c", CHILD.format(root=ROOT, tests=TESTS, lib=lib)],
                       capture_output=True, text=True, timeout=300, env=env)
    return name, r.returncode, (r.stdout + r.stderr)[-400:]


def test_every_mutant_is_caught(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    survivors = [(n, out) for n, rc, out in results if rc == 0]
    assert not survivors, f"mutants not caught by any pin: {survivors}"


def test_unmutated_copy_passes(tmp_path):
    name, rc, out = _run_mutant(str(tmp_path), "identity", "int g = h / G;", "int g = h / G;", 0)
    assert rc == 0, out
