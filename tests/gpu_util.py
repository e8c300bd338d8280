"""Helpers for the GPU parity tests: upload synthetic inputs, run the C-ABI
entry points, compare with the oracle."""
from __future__ import annotations

import numpy as np
import torch

from paper_2410_12247_amd import moe, synth

# FFN output tolerance against the fp32 oracle fed the same bf16 inputs
MAX_ABS = 2e-2
REL_FRO = 5e-3


def dev():
    return torch.device("cuda:0")


def bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev()).view(torch.bfloat16)


def f32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())


def i32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev())


def bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


class Dev:
    """A workload's tensors on the GPU."""

    def __init__(self, inp: synth.MoEInputs):
        s = inp.shape
        self.inp, self.s = inp, s
        self.x = bf16(inp.x)
        self.w_router = f32(inp.w_router)
        self.bias = f32(inp.bias) if inp.bias is not None else None
        self.w_gate = bf16(inp.w_gate)
        self.w_up = bf16(inp.w_up)
        self.w_down = bf16(inp.w_down)
        self.sg = bf16(inp.shared_gate) if s.n_shared else None
        self.su = bf16(inp.shared_up) if s.n_shared else None
        self.sd = bf16(inp.shared_down) if s.n_shared else None
        self.d = moe.dims(s.T, s.H, s.I, s.E, s.k, s.e0, s.EL, s.renorm, s.shared_inter)

    def forward(self, o=None):
        buf = moe.MoEBuffers(self.d, o if o is not None else moe.opts(), dev())
        buf.run(self.x, self.w_router, self.bias, self.w_gate, self.w_up, self.w_down,
                self.sg, self.su, self.sd)
        torch.cuda.synchronize()
        return buf


def assert_close(got: np.ndarray, ref: np.ndarray, what: str,
                 max_abs: float = MAX_ABS, rel_fro: float = REL_FRO):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = float(np.abs(got - ref).max()) if got.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref)) / nref if nref > 0 else float(np.linalg.norm(got))
    assert err <= max_abs and rel <= rel_fro, \
        f"{what}: max-abs {err:.3g} (<= {max_abs}), rel-frobenius {rel:.3g} (<= {rel_fro})"
    return err, rel
