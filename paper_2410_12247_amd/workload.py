"""Device copies of a synthetic workload (torch tensors on the GPU) and the
one-call forward over them.  Marshalling only: uploads the arrays that
``synth`` draws and calls the C-ABI."""
from __future__ import annotations

import numpy as np
import torch

from . import moe, synth


def device() -> torch.device:
    return torch.device("cuda", torch.cuda.current_device())


def bf16(a: np.ndarray, dev=None) -> torch.Tensor:
    """bf16 bit patterns (uint16) -> torch.bfloat16 on the GPU."""
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
    return t.to(dev or device()).view(torch.bfloat16)


def f32(a: np.ndarray, dev=None) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev or device())


def i32(a: np.ndarray, dev=None) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev or device())


def bits(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 -> bf16 bit patterns (uint16) on the host."""
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


class DeviceInputs:
    """A workload's tensors on the GPU plus its moe_dims."""

    def __init__(self, inp: synth.MoEInputs, dev=None):
        s = inp.shape
        dev = dev or device()
        self.inp, self.s = inp, s
        self.x = bf16(inp.x, dev)
        self.w_router = f32(inp.w_router, dev)
        self.bias = f32(inp.bias, dev) if inp.bias is not None else None
        self.w_gate = bf16(inp.w_gate, dev)
        self.w_up = bf16(inp.w_up, dev)
        self.w_down = bf16(inp.w_down, dev)
        self.sg = bf16(inp.shared_gate, dev) if s.n_shared else None
        self.su = bf16(inp.shared_up, dev) if s.n_shared else None
        self.sd = bf16(inp.shared_down, dev) if s.n_shared else None
        self.d = moe.dims(s.T, s.H, s.I, s.E, s.k, s.e0, s.EL, s.renorm, s.shared_inter)
        self.dev = dev

    def buffers(self, o=None) -> moe.MoEBuffers:
        return moe.MoEBuffers(self.d, o if o is not None else moe.opts(), self.dev)

    def run(self, buf: moe.MoEBuffers, stream=None):
        return buf.run(self.x, self.w_router, self.bias, self.w_gate, self.w_up, self.w_down,
                       self.sg, self.su, self.sd, stream)

    def forward(self, o=None) -> moe.MoEBuffers:
        buf = self.buffers(o)
        self.run(buf)
        torch.cuda.synchronize()
        return buf
