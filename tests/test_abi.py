"""The C ABI on the host: the library loads, exports what include/sl.h declares,
and rejects bad arguments before touching the GPU (no compute calls here)."""
import ctypes
import glob
import os
import re

import pytest
import torch

from paper_2504_15930_amd import sl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    names = set()
    for header in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(header).read(), flags=re.S)
        names |= set(re.findall(r"\b(sl_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sl.LIBRARY):
        from paper_2504_15930_amd import build
        build.build()
    return sl.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(sl.EXPORTS) | set(sl.ENGINE_EXPORTS) | set(sl.DISPATCH_EXPORTS), names
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in sl.STATUS_NAMES:
        assert len(sl.status_string(code)) > 5
    assert sl.status_string(12345) == "unknown status"


def _desc(**kw):
    args = dict(batch=4, num_q_heads=8, num_kv_heads=2, head_dim=128, page_size=16, max_blocks=8,
                num_pages=64, num_workers=32)
    args.update(kw)
    return sl.make_desc(**args)


FAKE = 0x10000  # a 16-byte aligned address that is never dereferenced by these calls


def _call(lib, d, q=FAKE, k=FAKE, v=FAKE, bt=FAKE, lens=FAKE, out=FAKE):
    return lib.sl_decode_attn(ctypes.byref(d) if d is not None else None, q, k, v, bt, lens,
                              0.125, out)


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=7, num_kv_heads=2), -2),
    (dict(batch=-1), -2),
    (dict(num_pages=0), -2),
    (dict(max_blocks=0), -2),
    (dict(num_workers=-3), -2),
    (dict(head_dim=96), -3),
    (dict(page_size=32), -3),
    (dict(num_q_heads=34, num_kv_heads=2), -3),
    (dict(batch=9000), -3),
    (dict(batch=8192, max_blocks=1 << 17, num_kv_heads=8, num_q_heads=8), -3),
    (dict(batch=4096, max_blocks=1 << 13, num_kv_heads=8, num_q_heads=8), -3),
    (dict(num_pages=1 << 29, num_kv_heads=8, num_q_heads=8), -3),
    (dict(num_workers=65537), -3),
])
def test_desc_validation(lib, kw, status):
    d = _desc(**kw)
    assert _call(lib, d) == status
    n = ctypes.c_size_t(0)
    assert lib.sl_decode_attn_workspace_size(ctypes.byref(d), ctypes.byref(n)) == status


def test_null_and_alignment(lib):
    assert _call(lib, None) == -1
    d = _desc()
    assert _call(lib, d, q=None) == -1
    assert _call(lib, d, out=None) == -1
    assert _call(lib, d, q=FAKE + 8) == -6
    assert _call(lib, d, k=FAKE + 2) == -6
    assert _call(lib, d, bt=FAKE + 2) == -6
    assert _call(lib, d, bt=FAKE + 4) == -4          # 4-byte aligned is enough; no workspace
    st = lib.sl_decode_attn_fp8(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                0.125, FAKE)
    assert st == -1


def test_batch_zero_is_a_noop(lib):
    d = _desc(batch=0)
    assert _call(lib, d, q=None, k=None, v=None, bt=None, lens=None, out=None) == 0


def test_workspace_size_and_check(lib):
    d = _desc(batch=4, num_workers=32, num_q_heads=8, num_kv_heads=2, head_dim=128)
    n = sl.workspace_size(d)
    align = lambda x: (x + 255) // 256 * 256
    G = 4
    # cum_pages [B + 1], part_ml [2 NW][G][2], part_acc [2 NW][G][D] (the split kernel derives its
    # tiles from the lengths and the block table, so there is no tile list)
    assert n == (align(4 * 5) + align(4 * 2 * 32 * G * 2) + align(4 * 2 * 32 * G * 128))
    assert sl.num_workers(d) == 32
    d.workspace = None
    assert _call(lib, d) == -4
    d.workspace, d.workspace_bytes = 0x100000, n - 1
    assert _call(lib, d) == -4
    d.workspace, d.workspace_bytes = 0x100000 + 16, n + 64
    assert _call(lib, d) == -4                        # not 256-byte aligned


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-device error path")
def test_default_workers_without_device(lib):
    d = _desc(num_workers=0)
    n = ctypes.c_size_t(0)
    assert lib.sl_decode_attn_workspace_size(ctypes.byref(d), ctypes.byref(n)) == -5


def test_binding_rejects_cpu_tensors(lib):
    q = torch.zeros(2, 4, 64, dtype=torch.bfloat16)
    k = torch.zeros(3, 2, 16, 64, dtype=torch.bfloat16)
    bt = torch.zeros(2, 1, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU"):
        sl.decode_attn(q, k, k, bt, torch.ones(2, dtype=torch.int32), 0.125)


def _append(lib, d, fp8=False, kn=FAKE, vn=FAKE, bt=FAKE, lens=FAKE, kp=FAKE, vp=FAKE, ks=FAKE, vs=FAKE):
    ref = ctypes.byref(d) if d is not None else None
    if fp8:
        return lib.sl_kv_append_fp8(ref, kn, vn, bt, lens, kp, vp, ks, vs)
    return lib.sl_kv_append(ref, kn, vn, bt, lens, kp, vp)


@pytest.mark.parametrize("fp8", [False, True])
def test_append_rejects_bad_arguments(lib, fp8):
    """KV append validates before touching the GPU: nulls, shapes, alignment; batch 0 is a no-op."""
    assert _append(lib, None, fp8) == -1
    d = _desc()
    assert _append(lib, d, fp8, kn=None) == -1
    assert _append(lib, d, fp8, vp=None) == -1
    assert _append(lib, d, fp8, kn=FAKE + 2) == -6
    assert _append(lib, d, fp8, kp=FAKE + 4) == -6
    assert _append(lib, d, fp8, lens=FAKE + 1) == -6
    if fp8:
        assert _append(lib, d, fp8, ks=None) == -1
        assert _append(lib, d, fp8, vs=FAKE + 2) == -6
    assert _append(lib, _desc(head_dim=96), fp8) == -3
    assert _append(lib, _desc(page_size=8), fp8) == -3
    assert _append(lib, _desc(num_kv_heads=3), fp8) == -2
    assert _append(lib, _desc(batch=0), fp8, kn=None, vn=None, bt=None, lens=None, kp=None, vp=None,
                   ks=None, vs=None) == 0


def test_engine_rejects_bad_arguments(lib):
    """The engine validates its configuration before allocating anything."""
    from paper_2504_15930_amd import engine as E
    E._lib()
    handle = ctypes.c_void_p()
    lens = (ctypes.c_int32 * 2)(10, 20)
    outs = (ctypes.c_int32 * 2)(5, 6)
    cfg = E.Config(2, 1, 0, 0, 0.125, ctypes.addressof(lens), ctypes.addressof(outs), ctypes.addressof(outs))
    bufs = E.Buffers(_desc(batch=2, max_blocks=4, num_pages=8), *([FAKE] * 10))
    assert lib.sl_engine_create(None, ctypes.byref(bufs), ctypes.byref(handle)) == -1
    assert lib.sl_engine_create(ctypes.byref(cfg), ctypes.byref(bufs), None) == -1
    assert lib.sl_engine_create(ctypes.byref(cfg), ctypes.byref(bufs), ctypes.byref(handle)) == -4  # no workspace
    bad = E.Buffers(_desc(batch=2, head_dim=96), *([FAKE] * 10))
    assert lib.sl_engine_create(ctypes.byref(cfg), ctypes.byref(bad), ctypes.byref(handle)) == -3
    # with a (never touched) workspace: the launch mode, the output history and its alignment
    d = _desc(batch=2, max_blocks=4, num_pages=8)
    d.workspace, d.workspace_bytes = FAKE, 1 << 30
    mode = E.Config(2, 1, 0, 0, 0.125, ctypes.addressof(lens), ctypes.addressof(outs), ctypes.addressof(outs), 2)
    assert lib.sl_engine_create(ctypes.byref(mode), ctypes.byref(E.Buffers(d, *([FAKE] * 10))),
                                ctypes.byref(handle)) == -2
    for hist, steps, status in [(None, 3, -1), (FAKE, -1, -2), (FAKE + 8, 1, -6)]:
        b = E.Buffers(d, *([FAKE] * 10), hist, steps)
        assert lib.sl_engine_create(ctypes.byref(cfg), ctypes.byref(b), ctypes.byref(handle)) == status
    b = E.Buffers(d, *([FAKE] * 10), None, 0, -1)   # a negative number of row sets
    assert lib.sl_engine_create(ctypes.byref(cfg), ctypes.byref(b), ctypes.byref(handle)) == -2
    n = ctypes.c_int32(0)
    assert lib.sl_engine_run(None, 1, ctypes.byref(n)) == -1
    assert lib.sl_engine_destroy(None) == 0


def _prefix(lib, d, fp8=False, q=FAKE, kp=FAKE, vp=FAKE, ks=FAKE, vs=FAKE, bt=FAKE, lens=FAKE, gs=FAKE, sp=FAKE,
            ng=2, out=FAKE):
    ref = ctypes.byref(d) if d is not None else None
    if fp8:
        return lib.sl_decode_attn_prefix_fp8(ref, q, kp, vp, ks, vs, bt, lens, gs, sp, ng, 0.125, out)
    return lib.sl_decode_attn_prefix(ref, q, kp, vp, bt, lens, gs, sp, ng, 0.125, out)


@pytest.mark.parametrize("fp8", [False, True])
def test_prefix_rejects_bad_arguments(lib, fp8):
    """Prefix-shared attention validates before touching the GPU: nulls (the group arrays only when
    there are groups, the scales only for E4M3), alignment, the group count, the batch limit and the
    workspace; batch 0 is a no-op."""
    d = _desc()
    assert _prefix(lib, None, fp8) == -1
    assert _prefix(lib, d, fp8, q=None) == -1
    assert _prefix(lib, d, fp8, gs=None) == -1
    assert _prefix(lib, d, fp8, sp=None) == -1
    assert _prefix(lib, d, fp8, q=FAKE + 8) == -6
    assert _prefix(lib, d, fp8, kp=FAKE + 2) == -6
    assert _prefix(lib, d, fp8, gs=FAKE + 2) == -6
    assert _prefix(lib, d, fp8, ng=-1) == -2
    assert _prefix(lib, d, fp8, ng=5) == -2                  # more groups than sequences
    assert _prefix(lib, _desc(batch=4097), fp8, ng=0) == -3
    assert _prefix(lib, d, fp8, gs=None, sp=None, ng=0) == -4   # no groups: the arrays are not needed
    assert _prefix(lib, d, fp8) == -4                        # valid arguments, no workspace
    if fp8:
        assert _prefix(lib, d, fp8, ks=None) == -1
        assert _prefix(lib, d, fp8, vs=FAKE + 2) == -6
    else:
        assert _prefix(lib, d, fp8, ks=None, vs=None) == -4  # the bf16 call takes no scales
    assert _prefix(lib, _desc(batch=0), fp8, q=None, kp=None, vp=None, ks=None, vs=None, bt=None, lens=None,
                   gs=None, sp=None, ng=0, out=None) == 0
    n0, n1 = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.sl_decode_attn_prefix_workspace_size(ctypes.byref(d), 2, ctypes.byref(n0)) == 0
    assert lib.sl_decode_attn_prefix_workspace_size(ctypes.byref(d), 4, ctypes.byref(n1)) == 0
    assert n1.value >= n0.value > 0
    assert lib.sl_decode_attn_prefix_workspace_size(ctypes.byref(d), 5, ctypes.byref(n0)) == -2


def test_missing_library_fails_loudly():
    """Without the built library every entry point is unreachable: loading raises, there is no fallback."""
    import subprocess
    import sys
    code = ("from paper_2504_15930_amd import sl\n"
            "try:\n    sl.load('/nonexistent/libsl.so')\n"
            "except ImportError as e:\n    print('ImportError', e)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "ImportError /nonexistent/libsl.so is missing" in r.stdout


def test_noalloc_host_checks(lib):
    # Errors found on the host, before the fixed scratch array is looked up (no GPU needed).
    assert lib.sl_decode_attn_noalloc(None, FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE) == -1
    d = _desc(num_q_heads=7, num_kv_heads=2)
    assert lib.sl_decode_attn_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE) == -2
    # 65536 workers x 16 query heads x (128 + 2) floats x 2 slots: far beyond the fixed array
    d = _desc(num_q_heads=32, num_kv_heads=2, num_workers=65536)
    assert lib.sl_decode_attn_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE) == -7
    assert "fixed array" in sl.status_string(-7)
    d = _desc(batch=0)
    assert lib.sl_decode_attn_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE) == 0
