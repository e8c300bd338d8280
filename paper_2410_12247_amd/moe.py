"""Thin Python binding of libmoe.so (include/moe.h): argument marshalling only.

Every step of the MoE FFN runs in the HIP library; these wrappers turn torch
tensors into device pointers and the current torch stream into a hipStream_t,
and raise ``MoEError`` on a non-zero status.  The library must be built
(``python -m paper_2410_12247_amd.build``); if it is missing, loading fails
loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmoe.so")

GEMM_AUTO, GEMM_GROUP, GEMM_DENSE = 0, 1, 2
CHUNK_EXPERTS, CHUNK_TOKENS = 0, 1
FLAG_TIMING, FLAG_TIMING_GEMM, FLAG_EXACT_ORDER, FLAG_SERIAL = 1, 2, 4, 8

# the entry points include/moe.h declares
EXPORTS = ("moe_workspace_bytes", "moe_workspace_guards", "moe_route", "moe_permute", "moe_gather", "moe_ffn_group",
           "moe_ffn_dense", "moe_combine", "moe_ffn_forward", "moe_ffn_forward_noalloc",
           "moe_last_timing",
           "moe_gemm_plan", "moe_pipeline_plan", "moe_choose_pipeline_n", "moe_status_string",
           "moe_last_error")


class MoEError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_int64), ("hidden", ctypes.c_int32),
                ("inter", ctypes.c_int32), ("experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("local_begin", ctypes.c_int32),
                ("local_count", ctypes.c_int32), ("renormalize", ctypes.c_int32),
                ("shared_inter", ctypes.c_int32)]


class Opts(ctypes.Structure):
    _fields_ = [("gemm_mode", ctypes.c_int32), ("dense_min_rows", ctypes.c_int32),
                ("pipeline_n", ctypes.c_int32), ("gemm_cu_budget", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("chunk_mode", ctypes.c_int32),
                ("dense_tile_rows", ctypes.c_int32), ("side_cus", ctypes.c_int32),
                ("group_tile_rows", ctypes.c_int32)]


class Timing(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("route_ms", "permute_ms", "gather_ms", "gateup_ms",
                                             "down_ms", "shared_ms", "combine_ms", "total_ms")] + \
               [(n, ctypes.c_int32) for n in ("gateup_launches", "down_launches",
                                             "dense_stages", "group_stages", "pipeline_n",
                                             "calls")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class PipelineEval(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("t_comm_us", "t_comp_us", "t_comm_n_us",
                                              "t_comp_n_us", "eps0", "eps1", "overlap_frac",
                                              "gain_us")] + \
               [("enabled", ctypes.c_int32), ("pipeline_n", ctypes.c_int32)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


_lib = None


def lib():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run python -m paper_2410_12247_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    D, O = ctypes.POINTER(Dims), ctypes.POINTER(Opts)
    L.moe_workspace_bytes.argtypes = [D, O]
    L.moe_workspace_bytes.restype = SZ
    L.moe_workspace_guards.argtypes = [D, O, ctypes.POINTER(ctypes.c_int64), ctypes.c_int32]
    L.moe_workspace_guards.restype = ctypes.c_int32
    L.moe_route.argtypes = [D, P, P, P, P, P, P]
    L.moe_permute.argtypes = [D, P, P, P, P, P, P, P, P, SZ, P]
    L.moe_gather.argtypes = [D, I32, I32, P, P, P, P, P]
    L.moe_ffn_group.argtypes = [D, I32, I32, P, P, P, P, P, P, P, I32, P]
    L.moe_ffn_dense.argtypes = [I64, I32, I32, P, P, P, P, P, P, P]
    L.moe_combine.argtypes = [D, I32, I32, P, P, P, P, P, I32, P]
    L.moe_ffn_forward.argtypes = [D, O, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
    L.moe_ffn_forward_noalloc.argtypes = [D, O, P, P, P, P, P, P, P, P, P, P, P, P, P, P]
    L.moe_last_timing.argtypes = [ctypes.POINTER(Timing)]
    L.moe_pipeline_plan.argtypes = [D, O, P, I32, ctypes.POINTER(PipelineEval)]
    L.moe_gemm_plan.argtypes = [D, O, I32, P, ctypes.POINTER(I32), P,
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    L.moe_choose_pipeline_n.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double, I32,
                                        ctypes.POINTER(I32), ctypes.POINTER(ctypes.c_double)]
    L.moe_status_string.argtypes = [I32]
    L.moe_status_string.restype = ctypes.c_char_p
    L.moe_last_error.restype = ctypes.c_char_p
    for name in ("moe_route", "moe_permute", "moe_gather", "moe_ffn_group", "moe_ffn_dense",
                 "moe_combine", "moe_ffn_forward", "moe_ffn_forward_noalloc", "moe_last_timing",
                 "moe_choose_pipeline_n", "moe_gemm_plan", "moe_pipeline_plan"):
        getattr(L, name).restype = I32
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        L = lib()
        raise MoEError(status, f"{L.moe_status_string(status).decode()}: "
                               f"{L.moe_last_error().decode()}")


def dims(tokens, hidden, inter, experts, top_k, local_begin=0, local_count=None,
         renormalize=True, shared_inter=0) -> Dims:
    return Dims(int(tokens), int(hidden), int(inter), int(experts), int(top_k),
                int(local_begin), int(experts if local_count is None else local_count),
                int(bool(renormalize)), int(shared_inter))


def opts(gemm_mode=GEMM_AUTO, dense_min_rows=0, pipeline_n=1, gemm_cu_budget=0,
         timing=False, chunk_mode=CHUNK_EXPERTS, exact_order=False, serial=False,
         dense_tile_rows=0, side_cus=0, group_tile_rows=0) -> Opts:
    """timing: False, True (every phase) or "gemm" (the GEMM launches only).
    exact_order: no K split of the grouped GEMM's last round (the same bits
    for every pipeline number, stage kind, CU budget and GEMM kind).
    serial: every stage on the caller's stream, nothing overlapped."""
    o = Opts()
    o.gemm_mode, o.dense_min_rows, o.pipeline_n = gemm_mode, dense_min_rows, pipeline_n
    o.gemm_cu_budget = gemm_cu_budget
    o.flags = FLAG_TIMING_GEMM if timing == "gemm" else (FLAG_TIMING if timing else 0)
    if exact_order:
        o.flags |= FLAG_EXACT_ORDER
    if serial:
        o.flags |= FLAG_SERIAL
    o.chunk_mode = chunk_mode
    o.dense_tile_rows = dense_tile_rows
    o.side_cus = side_cus
    o.group_tile_rows = group_tile_rows
    return o


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("tensors passed to libmoe must be contiguous device tensors")
    return ctypes.c_void_p(t.data_ptr())


def _s(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def workspace_bytes(d: Dims, o: Optional[Opts] = None) -> int:
    return lib().moe_workspace_bytes(ctypes.byref(d), ctypes.byref(o) if o is not None else None)


WS_GUARD_BYTES = 256  # MOE_WS_GUARD_BYTES


def workspace_guards(d: Dims, o: Optional[Opts] = None) -> list:
    """Byte offsets of the workspace's guard gaps (WS_GUARD_BYTES each)."""
    ob = ctypes.byref(o) if o is not None else None
    n = lib().moe_workspace_guards(ctypes.byref(d), ob, None, 0)
    if n < 0:
        raise MoEError(1, "moe_workspace_guards: invalid dims or options")
    buf = (ctypes.c_int64 * max(n, 1))()
    lib().moe_workspace_guards(ctypes.byref(d), ob, buf, n)
    return list(buf[:n])


def route(d, x, w_router, bias, topk_ids, topk_w, stream=None):
    _check(lib().moe_route(ctypes.byref(d), _p(x), _p(w_router), _p(bias), _p(topk_ids),
                           _p(topk_w), _s(stream)))


def permute(d, topk_ids, x, counts, offsets, sorted_slot, slot_row, x_perm, ws, stream=None):
    _check(lib().moe_permute(ctypes.byref(d), _p(topk_ids), _p(x), _p(counts), _p(offsets),
                             _p(sorted_slot), _p(slot_row), _p(x_perm), _p(ws),
                             ws.numel() * ws.element_size(), _s(stream)))


def gather(d, e_first, e_count, offsets, sorted_slot, x, x_perm, stream=None):
    _check(lib().moe_gather(ctypes.byref(d), e_first, e_count, _p(offsets), _p(sorted_slot),
                            _p(x), _p(x_perm), _s(stream)))


def ffn_group(d, e_first, e_count, offsets, x_perm, w_gate, w_up, w_down, act, y_perm,
              cu_budget=0, stream=None):
    _check(lib().moe_ffn_group(ctypes.byref(d), e_first, e_count, _p(offsets), _p(x_perm),
                               _p(w_gate), _p(w_up), _p(w_down), _p(act), _p(y_perm),
                               cu_budget, _s(stream)))


def ffn_dense(rows, hidden, inter, x, w_gate, w_up, w_down, act, y, stream=None):
    _check(lib().moe_ffn_dense(int(rows), hidden, inter, _p(x), _p(w_gate), _p(w_up),
                               _p(w_down), _p(act), _p(y), _s(stream)))


def combine(d, e_first, e_count, y_perm, topk_ids, slot_row, topk_w, y, accumulate,
            stream=None):
    _check(lib().moe_combine(ctypes.byref(d), e_first, e_count, _p(y_perm), _p(topk_ids),
                             _p(slot_row), _p(topk_w), _p(y), int(accumulate), _s(stream)))


def forward(d, o, x, w_router, bias, w_gate, w_up, w_down, shared_gate, shared_up, shared_down,
            y, topk_ids, topk_w, counts, ws, stream=None):
    _check(lib().moe_ffn_forward(ctypes.byref(d), ctypes.byref(o) if o is not None else None,
                                 _p(x), _p(w_router), _p(bias), _p(w_gate), _p(w_up),
                                 _p(w_down), _p(shared_gate), _p(shared_up), _p(shared_down),
                                 _p(y), _p(topk_ids), _p(topk_w), _p(counts), _p(ws),
                                 ws.numel() * ws.element_size(), _s(stream)))


def forward_noalloc(d, o, x, w_router, bias, w_gate, w_up, w_down, shared_gate, shared_up,
                    shared_down, y, topk_ids, topk_w, counts, stream=None):
    """moe_ffn_forward_noalloc: the forward with the library's static scratch
    buffer instead of a workspace (no allocation in the call)."""
    _check(lib().moe_ffn_forward_noalloc(
        ctypes.byref(d), ctypes.byref(o) if o is not None else None, _p(x), _p(w_router),
        _p(bias), _p(w_gate), _p(w_up), _p(w_down), _p(shared_gate), _p(shared_up),
        _p(shared_down), _p(y), _p(topk_ids), _p(topk_w), _p(counts), _s(stream)))


def choose_pipeline_n(c_ms: float, k_ms: float, b_ms: float, local_count: int):
    """(PN, gain in ms) from the paper's pipeline overhead model."""
    pn = ctypes.c_int32()
    gain = ctypes.c_double()
    _check(lib().moe_choose_pipeline_n(float(c_ms), float(k_ms), float(b_ms), int(local_count),
                                       ctypes.byref(pn), ctypes.byref(gain)))
    return pn.value, gain.value


def last_timing() -> dict:
    t = Timing()
    _check(lib().moe_last_timing(ctypes.byref(t)))
    return t.as_dict()


def pipeline_plan(d: Dims, o: Optional[Opts], rows, pipeline_n: int) -> dict:
    """The paper's pipeline terms for PN = pipeline_n (0: the library's
    choice) from host row counts per local expert."""
    import numpy as np
    r = np.ascontiguousarray(rows, dtype=np.int32)
    ev = PipelineEval()
    _check(lib().moe_pipeline_plan(ctypes.byref(d), ctypes.byref(o) if o is not None else None,
                                   r.ctypes.data_as(ctypes.c_void_p), int(pipeline_n),
                                   ctypes.byref(ev)))
    return ev.as_dict()


def gemm_plan(d: Dims, o: Optional[Opts], rows):
    """AUTO's plan for one stage with host row counts `rows`: (dense, tile
    rows per expert, predicted group us, predicted dense us)."""
    import numpy as np
    r = np.ascontiguousarray(rows, dtype=np.int32)
    tiles = np.zeros(len(r), np.int32)
    dense = ctypes.c_int32()
    gus, dus = ctypes.c_double(), ctypes.c_double()
    _check(lib().moe_gemm_plan(ctypes.byref(d), ctypes.byref(o) if o is not None else None,
                               len(r), r.ctypes.data_as(ctypes.c_void_p), ctypes.byref(dense),
                               tiles.ctypes.data_as(ctypes.c_void_p), ctypes.byref(gus),
                               ctypes.byref(dus)))
    return bool(dense.value), tiles.tolist(), gus.value, dus.value


class MoEBuffers:
    """Device tensors of one workload plus the workspace, for callers that
    want the whole forward with one call (tests, benchmark, smoke)."""

    def __init__(self, d: Dims, o: Optional[Opts], device="cuda"):
        T, k, H = d.tokens, d.top_k, d.hidden
        self.d, self.o = d, o
        self.y = torch.empty((T, H), dtype=torch.float32, device=device)
        self.topk_ids = torch.empty((T, k), dtype=torch.int32, device=device)
        self.topk_w = torch.empty((T, k), dtype=torch.float32, device=device)
        self.counts = torch.empty((d.local_count,), dtype=torch.int32, device=device)
        nbytes = workspace_bytes(d, o if o is not None else opts())
        self.ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=device)

    def run(self, x, w_router, bias, w_gate, w_up, w_down, shared_gate=None, shared_up=None,
            shared_down=None, stream=None):
        forward(self.d, self.o, x, w_router, bias, w_gate, w_up, w_down, shared_gate,
                shared_up, shared_down, self.y, self.topk_ids, self.topk_w, self.counts,
                self.ws, stream)
        return self.y
