"""ctypes binding of the decode engine (``include/sl_engine.h``): argument marshalling only.

The engine runs a whole generation (continuous batching with LPT admission)
by driving ``libsl``'s KV append and decode-attention kernels step by step;
its schedule and page bookkeeping live in C++, every step's work in HIP
kernels. Device buffers are torch tensors owned by the ``Engine`` object.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import sl


class Config(ctypes.Structure):
    _fields_ = [
        ("num_samples", ctypes.c_int32),
        ("admission", ctypes.c_int32),
        ("kv_fp8", ctypes.c_int32),
        ("fill_seed", ctypes.c_uint32),
        ("attn_scale", ctypes.c_float),
        ("prompt_len", ctypes.c_void_p),
        ("output_len", ctypes.c_void_p),
        ("est_len", ctypes.c_void_p),
        ("launch_mode", ctypes.c_int32),
    ]


class Buffers(ctypes.Structure):
    _fields_ = [
        ("desc", sl.Desc),
        ("q", ctypes.c_void_p),
        ("k_new", ctypes.c_void_p),
        ("v_new", ctypes.c_void_p),
        ("k_pages", ctypes.c_void_p),
        ("v_pages", ctypes.c_void_p),
        ("k_scales", ctypes.c_void_p),
        ("v_scales", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("seq_lens", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("out_history", ctypes.c_void_p),
        ("history_steps", ctypes.c_int32),
        ("row_sets", ctypes.c_int32),
    ]


def _lib():
    lib = sl.load()
    if not getattr(lib, "_engine_typed", False):
        P = ctypes.c_void_p
        lib.sl_engine_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Buffers), ctypes.POINTER(P)]
        lib.sl_engine_run.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
        lib.sl_engine_schedule.argtypes = [P, P, P, P, ctypes.POINTER(ctypes.c_int32), P, ctypes.c_int32]
        lib.sl_engine_destroy.argtypes = [P]
        for name in ("sl_engine_create", "sl_engine_run", "sl_engine_schedule", "sl_engine_destroy"):
            getattr(lib, name).restype = ctypes.c_int
        lib._engine_typed = True
    return lib


class Engine:
    """One generation run: ``M`` samples on ``batch_slots`` slots of one GPU.

    Allocates (with torch) the page pool, block table, lengths, query and
    new-row buffers, output and workspace; ``q``/``k_new``/``v_new`` hold
    seeded random rows used in every step (with ``row_sets`` > 1, ``k_new`` and
    ``v_new`` hold that many sets [R][BS][Hkv][D] and step s appends set
    s % R). ``two_launch`` makes every step run the split kernel and the
    merge; ``history_steps`` > 0 keeps the outputs of the first that many
    steps in ``history``.
    """

    def __init__(self, prompt_len, output_len, est_len=None, *, batch_slots: int, num_q_heads: int,
                 num_kv_heads: int, head_dim: int, kv_fp8: bool = False, lpt: bool = True,
                 num_pages: int | None = None, max_blocks: int | None = None, seed: int = 0,
                 num_workers: int = 0, two_launch: bool = False, history_steps: int = 0, row_sets: int = 1,
                 device="cuda:0"):
        self.prompt_len = np.ascontiguousarray(prompt_len, dtype=np.int32)
        self.output_len = np.ascontiguousarray(output_len, dtype=np.int32)
        self.est_len = np.ascontiguousarray(self.output_len if est_len is None else est_len, dtype=np.int32)
        M = len(self.output_len)
        need = int(((self.prompt_len.astype(np.int64) + self.output_len + 15) // 16).max())
        self.max_blocks = max_blocks or need
        self.num_pages = num_pages or batch_slots * self.max_blocks
        self.BS, self.Hq, self.Hkv, self.D = batch_slots, num_q_heads, num_kv_heads, head_dim
        self.fp8 = kv_fp8
        dev = torch.device(device)
        g = torch.Generator(device=dev).manual_seed(seed)
        kv_dtype = torch.uint8 if kv_fp8 else torch.bfloat16
        pool = (self.num_pages, num_kv_heads, 16, head_dim)
        self.k_pages = torch.zeros(pool, dtype=kv_dtype, device=dev)
        self.v_pages = torch.zeros(pool, dtype=kv_dtype, device=dev)
        self.k_scales = torch.ones((self.num_pages, num_kv_heads), dtype=torch.float32, device=dev) if kv_fp8 else None
        self.v_scales = torch.ones((self.num_pages, num_kv_heads), dtype=torch.float32, device=dev) if kv_fp8 else None
        self.block_table = torch.zeros((batch_slots, self.max_blocks), dtype=torch.int32, device=dev)
        self.seq_lens = torch.zeros(batch_slots, dtype=torch.int32, device=dev)
        self.q = torch.randn((batch_slots, num_q_heads, head_dim), generator=g, device=dev).to(torch.bfloat16)
        rows = ((row_sets,) if row_sets > 1 else ()) + (batch_slots, num_kv_heads, head_dim)
        self.k_new = torch.randn(rows, generator=g, device=dev).to(torch.bfloat16)
        self.v_new = torch.randn(rows, generator=g, device=dev).to(torch.bfloat16)
        self.out = torch.zeros((batch_slots, num_q_heads, head_dim), dtype=torch.bfloat16, device=dev)
        self.history = (torch.zeros((history_steps, batch_slots, num_q_heads, head_dim), dtype=torch.bfloat16,
                                    device=dev) if history_steps > 0 else None)
        self.scale = float(np.float32(1.0 / np.sqrt(head_dim)))
        self.stream = torch.cuda.current_stream(dev)
        desc = sl.make_desc(batch_slots, num_q_heads, num_kv_heads, head_dim, 16, self.max_blocks,
                            self.num_pages, num_workers, self.stream.cuda_stream)
        self.workspace = torch.empty(max(sl.workspace_size(desc), 256), dtype=torch.uint8, device=dev)
        desc.workspace = self.workspace.data_ptr()
        desc.workspace_bytes = self.workspace.numel()
        ptr = lambda t: None if t is None else t.data_ptr()
        self._bufs = Buffers(desc, ptr(self.q), ptr(self.k_new), ptr(self.v_new), ptr(self.k_pages),
                             ptr(self.v_pages), ptr(self.k_scales), ptr(self.v_scales), ptr(self.block_table),
                             ptr(self.seq_lens), ptr(self.out), ptr(self.history), int(history_steps),
                             int(row_sets))
        self._cfg = Config(M, 1 if lpt else 0, 1 if kv_fp8 else 0, seed & 0xFFFFFFFF, self.scale,
                           self.prompt_len.ctypes.data, self.output_len.ctypes.data, self.est_len.ctypes.data,
                           1 if two_launch else 0)
        torch.cuda.synchronize(dev)
        handle = ctypes.c_void_p()
        sl._check(_lib().sl_engine_create(ctypes.byref(self._cfg), ctypes.byref(self._bufs), ctypes.byref(handle)),
                  "sl_engine_create")
        self._h = handle
        self.M = M

    def run(self, max_steps: int = 1 << 30) -> int:
        """Enqueue up to ``max_steps`` decode steps; returns how many were enqueued."""
        n = ctypes.c_int32(0)
        sl._check(_lib().sl_engine_run(self._h, int(max_steps), ctypes.byref(n)), "sl_engine_run")
        return n.value

    def schedule(self):
        """(slot, admit_step, finish_step, steps, active-per-step) as numpy arrays / int."""
        slot = np.full(self.M, -1, np.int32)
        adm = np.full(self.M, -1, np.int32)
        fin = np.full(self.M, -1, np.int32)
        steps = ctypes.c_int32(0)
        _lib().sl_engine_schedule(self._h, None, None, None, ctypes.byref(steps), None, 0)
        act = np.zeros(max(steps.value, 1), np.int32)
        sl._check(_lib().sl_engine_schedule(self._h, slot.ctypes.data, adm.ctypes.data, fin.ctypes.data,
                                            ctypes.byref(steps), act.ctypes.data, len(act)), "sl_engine_schedule")
        return slot, adm, fin, steps.value, act[:steps.value]

    def close(self):
        if getattr(self, "_h", None):
            sl._check(_lib().sl_engine_destroy(self._h), "sl_engine_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
