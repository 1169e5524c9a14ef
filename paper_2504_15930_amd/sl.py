"""ctypes binding of ``libsl`` (``include/sl.h``): argument marshalling only.

Every step of the decode path (KV append and attention) runs in the HIP kernels of
``libsl.so``; torch supplies device memory, the current stream and (for
profiling) events. There is no fallback: without the built library or
without a GPU tensor every entry point raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# SL_LIBRARY may name another build of the same sources (the host-sanitized one of the tests).
LIBRARY = os.environ.get("SL_LIBRARY") or os.path.join(HERE, "libsl.so")

SL_OK = 0
STATUS_NAMES = {0: "SL_OK", -1: "SL_ERR_NULL", -2: "SL_ERR_SHAPE", -3: "SL_ERR_UNSUPPORTED",
                -4: "SL_ERR_WORKSPACE", -5: "SL_ERR_HIP", -6: "SL_ERR_ALIGNMENT", -7: "SL_ERR_SCRATCH_LIMIT"}
EXPORTS = ["sl_decode_attn_workspace_size", "sl_decode_attn_num_workers", "sl_decode_attn",
           "sl_decode_attn_fp8", "sl_kv_append", "sl_kv_append_fp8", "sl_decode_attn_prefix",
           "sl_decode_attn_prefix_fp8", "sl_decode_attn_prefix_workspace_size", "sl_decode_attn_noalloc",
           "sl_status_string"]
# include/sl_engine.h (typed in engine.py)
ENGINE_EXPORTS = ["sl_engine_create", "sl_engine_run", "sl_engine_schedule", "sl_engine_destroy"]
# include/sl_dispatch.h (typed in dispatch.py)
DISPATCH_EXPORTS = ["sl_generation_latency", "sl_dispatch_plan"]


class SlError(RuntimeError):
    """A libsl call returned an error status."""

    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({status_string(status)})")


class Desc(ctypes.Structure):
    """Mirror of ``sl_attn_desc``."""

    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("num_workers", ctypes.c_int32),
        ("stream", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("timing_start", ctypes.c_void_p),
        ("timing_stop", ctypes.c_void_p),
    ]


_lib: ctypes.CDLL | None = None


def load(path: str = LIBRARY) -> ctypes.CDLL:
    """Load libsl (once). The HIP runtime torch already loaded is reused."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2504_15930_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    D = ctypes.POINTER(Desc)
    lib.sl_decode_attn_workspace_size.argtypes = [D, ctypes.POINTER(ctypes.c_size_t)]
    lib.sl_decode_attn_num_workers.argtypes = [D, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
    lib.sl_decode_attn.argtypes = [D, P, P, P, P, P, ctypes.c_float, P]
    lib.sl_decode_attn_fp8.argtypes = [D, P, P, P, P, P, P, P, ctypes.c_float, P]
    lib.sl_kv_append.argtypes = [D, P, P, P, P, P, P]
    lib.sl_decode_attn_prefix.argtypes = [D, P, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_float, P]
    lib.sl_decode_attn_prefix_fp8.argtypes = [D, P, P, P, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_float, P]
    lib.sl_decode_attn_prefix_workspace_size.argtypes = [D, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.sl_kv_append_fp8.argtypes = [D, P, P, P, P, P, P, P, P]
    lib.sl_decode_attn_noalloc.argtypes = [D, P, P, P, P, P, ctypes.c_float, P]
    lib.sl_status_string.argtypes = [ctypes.c_int32]
    lib.sl_status_string.restype = ctypes.c_char_p
    for name in EXPORTS[:-1]:
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().sl_status_string(status).decode()


def make_desc(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_blocks, num_pages,
              num_workers=0, stream=None, workspace=None, workspace_bytes=0,
              timing=None) -> Desc:
    d = Desc()
    d.batch, d.num_q_heads, d.num_kv_heads, d.head_dim = batch, num_q_heads, num_kv_heads, head_dim
    d.page_size, d.max_blocks_per_seq, d.num_pages = page_size, max_blocks, num_pages
    d.num_workers = num_workers
    d.stream = stream
    d.workspace = workspace
    d.workspace_bytes = workspace_bytes
    if timing is not None:
        d.timing_start, d.timing_stop = timing
    return d


def _check(status: int, where: str):
    if status != SL_OK:
        raise SlError(status, where)


def workspace_size(desc: Desc) -> int:
    n = ctypes.c_size_t(0)
    _check(load().sl_decode_attn_workspace_size(ctypes.byref(desc), ctypes.byref(n)),
           "sl_decode_attn_workspace_size")
    return n.value


def num_workers(desc: Desc, fp8: bool = False) -> int:
    n = ctypes.c_int32(0)
    _check(load().sl_decode_attn_num_workers(ctypes.byref(desc), int(fp8), ctypes.byref(n)),
           "sl_decode_attn_num_workers")
    return n.value


_workspaces: dict[tuple[int, int], torch.Tensor] = {}


def _workspace(device: torch.device, nbytes: int) -> torch.Tensor:
    """A cached scratch buffer of at least ``nbytes`` (256-byte aligned by torch) per (device,
    current stream). Calls on one stream run one after the other, so they may share a buffer;
    calls on two streams could overlap, so each stream gets its own. The buffer is allocated
    while its stream is current, so when it is replaced by a larger one torch's allocator hands
    its memory out again only in that stream's order, after the kernels that used it."""
    idx = device.index if device.index is not None else torch.cuda.current_device()
    key = (idx, torch.cuda.current_stream(device).cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def _need(t: torch.Tensor, name: str, dtype, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU (libsl has no CPU path)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _run(fp8, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, out,
         num_workers_, workspace, timing):
    kv_dtype = torch.uint8 if fp8 else torch.bfloat16
    _need(q, "q", torch.bfloat16, 3)
    _need(k_pages, "k_pages", kv_dtype, 4)
    _need(v_pages, "v_pages", kv_dtype, 4)
    _need(block_table, "block_table", torch.int32, 2)
    _need(seq_lens, "seq_lens", torch.int32, 1)
    if fp8:
        _need(k_scales, "k_scales", torch.float32, 2)
        _need(v_scales, "v_scales", torch.float32, 2)
    B, Hq, D = q.shape
    N, Hkv, P, D2 = k_pages.shape
    if D2 != D or tuple(v_pages.shape) != tuple(k_pages.shape):
        raise ValueError("q, k_pages and v_pages disagree on shape")
    if block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_table / seq_lens rows must equal the batch")
    if fp8 and (tuple(k_scales.shape) != (N, Hkv) or tuple(v_scales.shape) != (N, Hkv)):
        raise ValueError("scales must have shape [num_pages, num_kv_heads]")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 3)
        if out.shape != q.shape:
            raise ValueError("out must have the shape of q")
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        desc = make_desc(B, Hq, Hkv, D, P, block_table.shape[1], N, num_workers_, stream)
        if B == 0:
            return out
        need = workspace_size(desc)
        ws = workspace if workspace is not None else _workspace(q.device, need)
        desc.workspace = ws.data_ptr()
        desc.workspace_bytes = ws.numel() * ws.element_size()
        if timing is not None:
            desc.timing_start, desc.timing_stop = timing
        lib = load()
        if fp8:
            st = lib.sl_decode_attn_fp8(ctypes.byref(desc), q.data_ptr(), k_pages.data_ptr(),
                                        v_pages.data_ptr(), k_scales.data_ptr(), v_scales.data_ptr(),
                                        block_table.data_ptr(), seq_lens.data_ptr(), float(scale),
                                        out.data_ptr())
            _check(st, "sl_decode_attn_fp8")
        else:
            st = lib.sl_decode_attn(ctypes.byref(desc), q.data_ptr(), k_pages.data_ptr(),
                                    v_pages.data_ptr(), block_table.data_ptr(), seq_lens.data_ptr(),
                                    float(scale), out.data_ptr())
            _check(st, "sl_decode_attn")
    return out


def decode_attn(q, k_pages, v_pages, block_table, seq_lens, scale, *, out=None, num_workers=0,
                workspace=None, timing=None) -> torch.Tensor:
    """``sl_decode_attn`` on torch tensors (bf16 KV cache); returns ``out`` [B, Hq, D] bf16.

    ``timing`` optionally holds two raw hipEvent handles recorded around the
    split-KV kernel. The call is asynchronous on the current stream.
    """
    return _run(False, q, k_pages, v_pages, None, None, block_table, seq_lens, scale, out,
                num_workers, workspace, timing)


def decode_attn_noalloc(q, k_pages, v_pages, block_table, seq_lens, scale, *, out=None,
                        num_workers=0) -> torch.Tensor:
    """``sl_decode_attn_noalloc``: ``sl_decode_attn`` with the library's fixed scratch array instead
    of a workspace (the call allocates nothing). Calls on one GPU must not overlap in time."""
    _need(q, "q", torch.bfloat16, 3)
    _need(k_pages, "k_pages", torch.bfloat16, 4)
    _need(v_pages, "v_pages", torch.bfloat16, 4)
    _need(block_table, "block_table", torch.int32, 2)
    _need(seq_lens, "seq_lens", torch.int32, 1)
    B, Hq, D = q.shape
    N, Hkv, P, D2 = k_pages.shape
    if D2 != D or tuple(v_pages.shape) != tuple(k_pages.shape):
        raise ValueError("q, k_pages and v_pages disagree on shape")
    if block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_table / seq_lens rows must equal the batch")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 3)
        if out.shape != q.shape:
            raise ValueError("out must have the shape of q")
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        desc = make_desc(B, Hq, Hkv, D, P, block_table.shape[1], N, num_workers, stream)
        _check(load().sl_decode_attn_noalloc(ctypes.byref(desc), q.data_ptr(), k_pages.data_ptr(),
                                             v_pages.data_ptr(), block_table.data_ptr(), seq_lens.data_ptr(),
                                             float(scale), out.data_ptr()),
               "sl_decode_attn_noalloc")
    return out


def decode_attn_fp8(q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, *,
                    out=None, num_workers=0, workspace=None, timing=None) -> torch.Tensor:
    """``sl_decode_attn_fp8``: K/V pages are uint8 E4M3 codes with fp32 [N, Hkv] scales."""
    return _run(True, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, out,
                num_workers, workspace, timing)


def run_batch(batch, **kw) -> torch.Tensor:
    """Decode attention on an ``inputs.Batch`` (dispatches on its KV dtype)."""
    if batch.kv_dtype == "e4m3":
        return decode_attn_fp8(batch.q, batch.k_pages, batch.v_pages, batch.k_scales,
                               batch.v_scales, batch.block_table, batch.seq_lens, batch.scale, **kw)
    return decode_attn(batch.q, batch.k_pages, batch.v_pages, batch.block_table, batch.seq_lens,
                       batch.scale, **kw)


def kv_append(k_new, v_new, block_table, seq_lens, k_pages, v_pages, *, k_scales=None,
              v_scales=None, num_q_heads=None, timing=None):
    """``sl_kv_append`` / ``sl_kv_append_fp8`` on torch tensors, in place.

    ``k_new``/``v_new``: bf16 [B, Hkv, D] rows of the step's new token;
    ``seq_lens`` already counts it. A uint8 page pool selects the E4M3 path,
    which needs fp32 ``k_scales``/``v_scales`` [N, Hkv] (updated in place).
    Asynchronous on the current stream.
    """
    fp8 = k_pages.dtype == torch.uint8
    kv_dtype = torch.uint8 if fp8 else torch.bfloat16
    _need(k_new, "k_new", torch.bfloat16, 3)
    _need(v_new, "v_new", torch.bfloat16, 3)
    _need(k_pages, "k_pages", kv_dtype, 4)
    _need(v_pages, "v_pages", kv_dtype, 4)
    _need(block_table, "block_table", torch.int32, 2)
    _need(seq_lens, "seq_lens", torch.int32, 1)
    if fp8:
        _need(k_scales, "k_scales", torch.float32, 2)
        _need(v_scales, "v_scales", torch.float32, 2)
    B, Hkv, D = k_new.shape
    N, Hkv2, P, D2 = k_pages.shape
    if (Hkv2, D2) != (Hkv, D) or tuple(v_new.shape) != (B, Hkv, D) or v_pages.shape != k_pages.shape:
        raise ValueError("k_new / v_new / pages disagree on shape")
    if block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("block_table / seq_lens rows must equal the batch")
    if fp8 and (tuple(k_scales.shape) != (N, Hkv) or tuple(v_scales.shape) != (N, Hkv)):
        raise ValueError("scales must have shape [num_pages, num_kv_heads]")
    with torch.cuda.device(k_new.device):
        stream = torch.cuda.current_stream(k_new.device).cuda_stream
        desc = make_desc(B, num_q_heads or Hkv, Hkv, D, P, block_table.shape[1], N, 0, stream)
        if timing is not None:
            desc.timing_start, desc.timing_stop = timing
        lib = load()
        if fp8:
            st = lib.sl_kv_append_fp8(ctypes.byref(desc), k_new.data_ptr(), v_new.data_ptr(),
                                      block_table.data_ptr(), seq_lens.data_ptr(), k_pages.data_ptr(),
                                      v_pages.data_ptr(), k_scales.data_ptr(), v_scales.data_ptr())
            _check(st, "sl_kv_append_fp8")
        else:
            st = lib.sl_kv_append(ctypes.byref(desc), k_new.data_ptr(), v_new.data_ptr(),
                                  block_table.data_ptr(), seq_lens.data_ptr(), k_pages.data_ptr(),
                                  v_pages.data_ptr())
            _check(st, "sl_kv_append")


def _run_prefix(fp8, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, group_start,
                shared_pages, out, num_workers, workspace, timing):
    kv_dtype = torch.uint8 if fp8 else torch.bfloat16
    _need(q, "q", torch.bfloat16, 3)
    _need(k_pages, "k_pages", kv_dtype, 4)
    _need(v_pages, "v_pages", kv_dtype, 4)
    _need(block_table, "block_table", torch.int32, 2)
    _need(seq_lens, "seq_lens", torch.int32, 1)
    _need(group_start, "group_start", torch.int32, 1)
    _need(shared_pages, "shared_pages", torch.int32, 1)
    if fp8:
        _need(k_scales, "k_scales", torch.float32, 2)
        _need(v_scales, "v_scales", torch.float32, 2)
    ng = shared_pages.shape[0]
    if group_start.shape[0] != ng + 1:
        raise ValueError("group_start must have num_groups + 1 entries")
    B, Hq, D = q.shape
    N, Hkv, P, D2 = k_pages.shape
    if D2 != D or v_pages.shape != k_pages.shape or block_table.shape[0] != B or seq_lens.shape[0] != B:
        raise ValueError("shape mismatch")
    if fp8 and (tuple(k_scales.shape) != (N, Hkv) or tuple(v_scales.shape) != (N, Hkv)):
        raise ValueError("scales must have shape [num_pages, num_kv_heads]")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", torch.bfloat16, 3)
        if out.shape != q.shape:
            raise ValueError("out must have the shape of q")
    lib = load()
    with torch.cuda.device(q.device):
        stream = torch.cuda.current_stream(q.device).cuda_stream
        desc = make_desc(B, Hq, Hkv, D, P, block_table.shape[1], N, num_workers, stream)
        if B == 0:
            return out
        need = ctypes.c_size_t(0)
        _check(lib.sl_decode_attn_prefix_workspace_size(ctypes.byref(desc), ng, ctypes.byref(need)),
               "sl_decode_attn_prefix_workspace_size")
        ws = workspace if workspace is not None else _workspace(q.device, need.value)
        desc.workspace = ws.data_ptr()
        desc.workspace_bytes = ws.numel() * ws.element_size()
        if timing is not None:
            desc.timing_start, desc.timing_stop = timing
        if fp8:
            _check(lib.sl_decode_attn_prefix_fp8(ctypes.byref(desc), q.data_ptr(), k_pages.data_ptr(),
                                                 v_pages.data_ptr(), k_scales.data_ptr(), v_scales.data_ptr(),
                                                 block_table.data_ptr(), seq_lens.data_ptr(),
                                                 group_start.data_ptr(), shared_pages.data_ptr(), ng,
                                                 float(scale), out.data_ptr()),
                   "sl_decode_attn_prefix_fp8")
        else:
            _check(lib.sl_decode_attn_prefix(ctypes.byref(desc), q.data_ptr(), k_pages.data_ptr(),
                                             v_pages.data_ptr(), block_table.data_ptr(), seq_lens.data_ptr(),
                                             group_start.data_ptr(), shared_pages.data_ptr(), ng, float(scale),
                                             out.data_ptr()),
                   "sl_decode_attn_prefix")
    return out


def decode_attn_prefix(q, k_pages, v_pages, block_table, seq_lens, scale, group_start, shared_pages, *,
                       out=None, num_workers=0, workspace=None, timing=None) -> torch.Tensor:
    """``sl_decode_attn_prefix``: decode attention reading each group's shared pages once.

    ``group_start`` (int32 [G+1]) and ``shared_pages`` (int32 [G]) are device tensors;
    consecutive sequences of a group share their first ``shared_pages[k]`` pages.
    """
    return _run_prefix(False, q, k_pages, v_pages, None, None, block_table, seq_lens, scale, group_start,
                       shared_pages, out, num_workers, workspace, timing)


def decode_attn_prefix_fp8(q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, group_start,
                           shared_pages, *, out=None, num_workers=0, workspace=None, timing=None) -> torch.Tensor:
    """``sl_decode_attn_prefix_fp8``: prefix sharing over uint8 E4M3 pages with fp32 [N, Hkv] scales."""
    return _run_prefix(True, q, k_pages, v_pages, k_scales, v_scales, block_table, seq_lens, scale, group_start,
                       shared_pages, out, num_workers, workspace, timing)
