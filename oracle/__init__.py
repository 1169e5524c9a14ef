"""CPU oracle for paged decode attention (fp64).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package. The GPU library
never uses it.

The arithmetic lives in ``oracle.c`` (plain C, double precision, two-pass
softmax); this module only marshals numpy arrays into it. Every function
follows the definition written at the top of ``oracle.c``.

Parity status: pinned. The ``-m "not gpu"`` tests check it against
``torch.nn.functional.scaled_dot_product_attention`` in float64 on dense
tensors scattered into pages by the test, against closed forms (one cached
token, identical keys, constant values, a dominant token), against
invariants (page order, aliasing block tables, head permutation inside a
group) and against ``torch.float8_e4m3fn`` for all 256 FP8 codes; mutated
copies of ``oracle.c`` are shown to fail those checks.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_LIBS: dict[str, ctypes.CDLL] = {}


def load(path: str | None = None) -> ctypes.CDLL:
    """Load (building first if absent) the oracle library at ``path``; by default the one named
    by the environment variable SL_ORACLE_LIBRARY (a build with the host sanitizers, say), else
    the standard build."""
    path = path or os.environ.get("SL_ORACLE_LIBRARY") or _build.LIBRARY
    lib = _LIBS.get(path)
    if lib is not None:
        return lib
    if path == _build.LIBRARY and not os.path.exists(path):
        _build.build()
    lib = ctypes.CDLL(path)
    lib.sl_oracle_bf16_to_double.restype = ctypes.c_double
    lib.sl_oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
    lib.sl_oracle_e4m3_to_double.restype = ctypes.c_double
    lib.sl_oracle_e4m3_to_double.argtypes = [ctypes.c_uint8]
    lib.sl_oracle_max_threads.restype = ctypes.c_int
    lib.sl_oracle_max_threads.argtypes = [ctypes.c_int]
    p = ctypes.c_void_p
    i = ctypes.c_int
    lib.sl_oracle_decode_attn.restype = ctypes.c_int
    lib.sl_oracle_decode_attn.argtypes = [i, i, i, i, i, i, i, i, p, p, p, p, p, p, p,
                                          ctypes.c_float, p, i, p, i]
    lib.sl_oracle_e4m3_encode.restype = ctypes.c_uint8
    lib.sl_oracle_e4m3_encode.argtypes = [ctypes.c_float]
    lib.sl_oracle_kv_append.restype = ctypes.c_int
    lib.sl_oracle_kv_append.argtypes = [i, i, i, i, i, i, i, p, p, p, p, p, p, p, p]
    _LIBS[path] = lib
    return lib


def _arr(a, dtype) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    return a


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def decode_attn(q, k_pages, v_pages, block_table, seq_lens, scale, *,
                k_scales=None, v_scales=None, rows=None, threads: int = 0,
                lib: str | None = None) -> np.ndarray:
    """Decode attention in fp64.

    q            uint16 [B, Hq, D]          bf16 bit patterns
    k_pages      uint16 [N, Hkv, P, D]      bf16 bits, or uint8 (FP8 E4M3 codes)
    v_pages      same dtype and shape as k_pages
    block_table  int32  [B, max_blocks]     page id of each logical page
    seq_lens     int32  [B]                 cached tokens per sequence
    scale        float                      widened from its fp32 value
    k_scales, v_scales  float32 [N, Hkv]    required for FP8 pages
    rows         int32 [R] or None          sequences to compute (None: all)

    Returns float64 [R, Hq, D] (R = B when rows is None).
    """
    q = _arr(q, np.uint16)
    kv_kind = 0 if np.asarray(k_pages).dtype == np.uint16 else 1
    kdt = np.uint16 if kv_kind == 0 else np.uint8
    k_pages = _arr(k_pages, kdt)
    v_pages = _arr(v_pages, kdt)
    block_table = _arr(block_table, np.int32)
    seq_lens = _arr(seq_lens, np.int32)
    if kv_kind == 1:
        k_scales = _arr(k_scales, np.float32)
        v_scales = _arr(v_scales, np.float32)
    B, Hq, D = q.shape
    N, Hkv, P, D2 = k_pages.shape
    if D2 != D or v_pages.shape != k_pages.shape:
        raise ValueError("q / k_pages / v_pages shapes disagree")
    if block_table.ndim != 2 or block_table.shape[0] != B or seq_lens.shape != (B,):
        raise ValueError("block_table / seq_lens shapes disagree with q")
    if kv_kind == 1 and (k_scales.shape != (N, Hkv) or v_scales.shape != (N, Hkv)):
        raise ValueError("scales must have shape [num_pages, Hkv]")
    if rows is None:
        rows_arr, nrows = None, B
    else:
        rows_arr = _arr(np.asarray(rows, dtype=np.int32), np.int32)
        nrows = rows_arr.shape[0]
    out = np.zeros((nrows, Hq, D), dtype=np.float64)
    rc = load(lib).sl_oracle_decode_attn(
        kv_kind, B, Hq, Hkv, D, P, block_table.shape[1], N, _ptr(q), _ptr(k_pages),
        _ptr(v_pages), _ptr(k_scales), _ptr(v_scales), _ptr(block_table), _ptr(seq_lens),
        float(np.float32(scale)), _ptr(rows_arr), nrows, _ptr(out), int(threads))
    if rc != 0:
        raise ValueError("oracle rejected its arguments (bad length, page id or shape)")
    return out


def e4m3_to_double(code: int, lib: str | None = None) -> float:
    """Value of one OCP FP8 E4M3 code."""
    return load(lib).sl_oracle_e4m3_to_double(code)


def bf16_to_double(bits: int, lib: str | None = None) -> float:
    """Value of one bf16 bit pattern."""
    return load(lib).sl_oracle_bf16_to_double(bits)


def max_threads(threads: int = 0, lib: str | None = None) -> int:
    """Threads the oracle's parallel loop uses for ``threads`` (0: default)."""
    return load(lib).sl_oracle_max_threads(threads)


def e4m3_encode(values, lib=None) -> np.ndarray:
    """OCP E4M3 codes (uint8) of float32 ``values``: nearest, ties to even, saturating, NaN -> 0x7F."""
    lib = lib if isinstance(lib, ctypes.CDLL) else load(lib)
    v = np.asarray(values, dtype=np.float32).ravel()
    return np.array([lib.sl_oracle_e4m3_encode(ctypes.c_float(float(x))) for x in v],
                    dtype=np.uint8).reshape(np.shape(values))


def kv_append(k_new, v_new, block_table, seq_lens, k_pages, v_pages, *, k_scales=None,
              v_scales=None, lib=None):
    """Append the step's new rows (see ``append.c``); returns updated copies.

    ``k_new``/``v_new``: bf16 bits (uint16) [B, Hkv, D]. ``k_pages``/``v_pages``:
    uint16 (bf16) or uint8 (E4M3 codes) [N, Hkv, P, D]; E4M3 needs fp32
    ``k_scales``/``v_scales`` [N, Hkv]. Returns ``(k_pages, v_pages)`` or, for
    E4M3, ``(k_pages, v_pages, k_scales, v_scales)``.
    """
    lib = lib if isinstance(lib, ctypes.CDLL) else load(lib)
    kn = _arr(k_new, np.uint16)
    vn = _arr(v_new, np.uint16)
    bt = _arr(block_table, np.int32)
    sl = _arr(seq_lens, np.int32)
    kp = np.array(k_pages, copy=True, order="C")
    vp = np.array(v_pages, copy=True, order="C")
    fp8 = kp.dtype == np.uint8
    if kp.dtype not in (np.uint8, np.uint16) or vp.dtype != kp.dtype:
        raise TypeError("pages must be uint16 (bf16 bits) or uint8 (E4M3 codes)")
    N, Hkv, P, D = kp.shape
    B = kn.shape[0]
    if kn.shape != (B, Hkv, D) or vn.shape != (B, Hkv, D) or bt.shape[0] != B or sl.shape != (B,):
        raise ValueError("shape mismatch")
    ks = vs = None
    if fp8:
        ks = np.array(k_scales, dtype=np.float32, copy=True, order="C")
        vs = np.array(v_scales, dtype=np.float32, copy=True, order="C")
        if ks.shape != (N, Hkv) or vs.shape != (N, Hkv):
            raise ValueError("scales must be [N, Hkv]")
    ptr = lambda a: None if a is None else a.ctypes.data
    rc = lib.sl_oracle_kv_append(1 if fp8 else 0, B, Hkv, D, P, bt.shape[1], N, ptr(kn), ptr(vn),
                                 ptr(bt), ptr(sl), ptr(kp), ptr(vp), ptr(ks), ptr(vs))
    if rc != 0:
        raise ValueError("oracle kv_append rejected its arguments")
    return (kp, vp, ks, vs) if fp8 else (kp, vp)
