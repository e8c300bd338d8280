"""Helpers for the GPU parity tests: device uploads come from the package's
workload module; this file adds the tolerance check."""
from __future__ import annotations

import numpy as np
import torch

from paper_2410_12247_amd.workload import DeviceInputs as Dev  # noqa: F401
from paper_2410_12247_amd.workload import bf16, bits, f32, i32  # noqa: F401

# FFN output tolerance against the fp32 oracle fed the same bf16 inputs
MAX_ABS = 2e-2
REL_FRO = 5e-3


def dev():
    return torch.device("cuda:0")


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


# workspace canary: the byte the guard gaps are filled with before a call
CANARY = 0xA5


def canary_fill(ws: torch.Tensor):
    ws.fill_(CANARY)


def assert_guards(ws: torch.Tensor, guards, what: str):
    """Every guard gap of the workspace still holds the canary."""
    from paper_2410_12247_amd import moe
    torch.cuda.synchronize()
    for off in guards:
        gap = ws[off:off + moe.WS_GUARD_BYTES]
        assert gap.numel() == moe.WS_GUARD_BYTES, f"{what}: guard at {off} past the workspace"
        bad = int((gap != CANARY).sum())
        assert bad == 0, f"{what}: {bad} bytes of the guard gap at offset {off} written"
