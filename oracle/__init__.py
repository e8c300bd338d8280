"""ctypes loader for the CPU oracle of the routed MoE FFN (oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this package; the product path never does.  It
shares nothing with the HIP library.  Arrays in: bf16 as raw uint16 bit
patterns, fp32 as float32, indices as int32; everything C-contiguous.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "oracle.c")
LIB = os.path.join(_HERE, "liboracle.so")
# -ffp-contract=off: no fused multiply-add except where the source asks for
# one (the router's fmaf); no fast-math, so every sum keeps source order.
CFLAGS = ["-O2", "-mfma", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared"]

_lib = None


def build() -> str:
    tmp = LIB + ".tmp"
    subprocess.check_call(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"])
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build()
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    i64, i32 = ctypes.c_int64, ctypes.c_int
    lib.oracle_router_logits.argtypes = [P, P, P, i64, i32, i32, P]
    lib.oracle_topk.argtypes = [P, i64, i32, i32, i32, P, P]
    lib.oracle_dispatch.argtypes = [P, i64, i32, i32, i32, P, P, P, P]
    lib.oracle_dispatch.restype = i64
    lib.oracle_expert_row.argtypes = [P, P, P, P, i32, i32, i32, P]
    lib.oracle_expert_rows.argtypes = [P, P, P, P, P, P, i32, i32, i32, i32, P]
    lib.oracle_expert_row_list.argtypes = [P, P, P, i64, P, P, P, i32, i32, P]
    lib.oracle_moe_tokens.argtypes = [P, P, P, P, i64, i32, i32, i32, i32, i32,
                                      P, P, P, i32, i32, P, P, P, P]
    lib.oracle_combine.argtypes = [P, P, P, P, i64, i32, i32, P]
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def router_logits(x_bits, w_router, bias=None):
    """Router logits z [T,E] fp32 (sequential fp32 fma over h, then + bias)."""
    x_bits = _c(x_bits, np.uint16)
    w_router = _c(w_router, np.float32)
    T, H = x_bits.shape
    E = w_router.shape[0]
    assert w_router.shape == (E, H)
    if bias is not None:
        bias = _c(bias, np.float32)
        assert bias.shape == (E,)
    z = np.empty((T, E), np.float32)
    _load().oracle_router_logits(_p(x_bits), _p(w_router), _p(bias), T, H, E, _p(z))
    return z


def topk(z, k, renorm):
    """Top-k ids [T,k] int32 ordered (logit desc, index asc) and fp32 weights."""
    z = _c(z, np.float32)
    T, E = z.shape
    ids = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float32)
    _load().oracle_topk(_p(z), T, E, k, int(bool(renorm)), _p(ids), _p(w))
    return ids, w


def dispatch(ids, e0, EL):
    """Stable expert-sorted dispatch: counts, offsets, sorted_slot, slot_row."""
    ids = _c(ids, np.int32)
    T, k = ids.shape
    counts = np.empty(EL, np.int32)
    offsets = np.empty(EL + 1, np.int32)
    sorted_slot = np.empty(T * k, np.int32)
    slot_row = np.empty(T * k, np.int32)
    R = _load().oracle_dispatch(_p(ids), T, k, e0, EL, _p(counts), _p(offsets),
                                _p(sorted_slot), _p(slot_row))
    return counts, offsets, sorted_slot[:R].copy(), slot_row


def expert_row(x_row_bits, w_gate, w_up, w_down, el):
    """FFN of one row through local expert el -> fp32 [H]."""
    x_row_bits = _c(x_row_bits, np.uint16)
    w_gate, w_up, w_down = (_c(a, np.uint16) for a in (w_gate, w_up, w_down))
    EL, I, H = w_gate.shape
    y = np.empty(H, np.float32)
    _load().oracle_expert_row(_p(x_row_bits), _p(w_gate), _p(w_up), _p(w_down), H, I, el, _p(y))
    return y


def expert_row_list(x_bits, tokens, experts, w_gate, w_up, w_down):
    """FFN rows for (token, local expert) pairs -> fp32 [n, H]."""
    x_bits = _c(x_bits, np.uint16)
    tok = _c(tokens, np.int64)
    el = _c(experts, np.int32)
    assert tok.shape == el.shape
    w_gate, w_up, w_down = (_c(a, np.uint16) for a in (w_gate, w_up, w_down))
    EL, I, H = w_gate.shape
    y = np.empty((len(tok), H), np.float32)
    _load().oracle_expert_row_list(_p(x_bits), _p(tok), _p(el), len(tok), _p(w_gate),
                                   _p(w_up), _p(w_down), H, I, _p(y))
    return y


def expert_rows(x_bits, sorted_slot, offsets, w_gate, w_up, w_down, k):
    """All dispatched rows y_perm [R,H] fp32."""
    x_bits = _c(x_bits, np.uint16)
    sorted_slot = _c(sorted_slot, np.int32)
    offsets = _c(offsets, np.int32)
    w_gate, w_up, w_down = (_c(a, np.uint16) for a in (w_gate, w_up, w_down))
    EL, I, H = w_gate.shape
    R = int(offsets[-1])
    y = np.empty((R, H), np.float32)
    _load().oracle_expert_rows(_p(x_bits), _p(sorted_slot), _p(offsets), _p(w_gate),
                               _p(w_up), _p(w_down), H, I, k, EL, _p(y))
    return y


def moe_tokens(x_bits, ids, w, tokens, w_gate, w_up, w_down, e0,
               n_shared=0, shared_gate=None, shared_up=None, shared_down=None):
    """MoE FFN output rows for the listed tokens -> fp32 [len(tokens), H]."""
    x_bits = _c(x_bits, np.uint16)
    ids = _c(ids, np.int32)
    w = _c(w, np.float32)
    tok = _c(tokens, np.int64)
    w_gate, w_up, w_down = (_c(a, np.uint16) for a in (w_gate, w_up, w_down))
    EL, I, H = w_gate.shape
    k = ids.shape[1]
    Is = 0
    if n_shared:
        shared_gate, shared_up, shared_down = (
            _c(a, np.uint16) for a in (shared_gate, shared_up, shared_down))
        Is = shared_gate.shape[0] // n_shared
    y = np.empty((len(tok), H), np.float32)
    _load().oracle_moe_tokens(_p(x_bits), _p(ids), _p(w), _p(tok), len(tok), H, I, k,
                              e0, EL, _p(w_gate), _p(w_up), _p(w_down), n_shared, Is,
                              _p(shared_gate), _p(shared_up), _p(shared_down), _p(y))
    return y


def combine(y_perm, slot_row, w, y_init=None):
    """y [T,H] = sum_j w[t,j] * y_perm[slot_row[t,j]] (+ y_init)."""
    y_perm = _c(y_perm, np.float32)
    slot_row = _c(slot_row, np.int32)
    w = _c(w, np.float32)
    T, k = w.shape
    H = y_perm.shape[1] if y_perm.ndim == 2 and y_perm.shape[0] else (
        y_init.shape[1] if y_init is not None else 0)
    if y_init is not None:
        y_init = _c(y_init, np.float32)
    y = np.empty((T, H), np.float32)
    _load().oracle_combine(_p(y_perm), _p(slot_row.reshape(-1)), _p(w), _p(y_init), T, H, k, _p(y))
    return y


def route(x_bits, w_router, bias, k, renorm):
    z = router_logits(x_bits, w_router, bias)
    ids, w = topk(z, k, renorm)
    return z, ids, w
