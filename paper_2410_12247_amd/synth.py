"""Seeded synthetic inputs shaped like the paper's MoE workloads.

This module is the only code the tests, the benchmark, the GPU path's
callers and the CPU oracle have in common.  It holds no arithmetic of the
method: it draws Gaussian tensors, rounds them to bf16 and builds the fixed
router bias used for the skewed load sweep.

Workloads (the paper measures trained Mixtral 8x7B, DBRX and DeepSeekV2;
trained weights and real router statistics are absent here, so Gaussian
tensors of the same shapes stand in for them):

* ``tiny``    : 512 tokens, hidden 256, 8 experts, SwiGLU width 512, top-2,
                renormalised weights.
* ``mixtral`` : Mixtral-8x7B-shaped tensor-parallel shard, 16384 tokens,
                hidden 4096, 8 experts, width 3584 (14336/4), top-2, renorm.
* ``dbrx``    : DBRX-shaped TP shard, 8192 tokens, hidden 6144, 16 experts,
                width 1344 (10752/8), top-4, renorm.
* ``dsv2``    : DeepSeekV2-shaped expert-parallel share, 16384 tokens routed
                over 160 experts, top-6 softmax over all 160 (no renorm);
                the 20 local experts [0, 20) of hidden 5120, width 1536 are
                computed, plus 2 shared experts of width 1536 on every token.
* ``mixtral_ep`` : Mixtral 8x7B as the paper deploys it with expert
                parallelism over 4 GPUs: one GPU's 2 local experts [0, 2) of
                full width 14336 (hidden 4096, top-2 of 8, renorm) over 16384
                routed tokens (about 8192 rows: the TP shard's GEMM flops).
* ``dbrx_ep`` : DBRX over 8 GPUs: 2 local experts [0, 2) of width 10752
                (hidden 6144, top-4 of 16, renorm) over 8192 routed tokens
                (about 4096 rows: the TP shard's GEMM flops).
* decode      : any shape at T = 1 .. 64 tokens (``with_tokens``; x is the
                first draw, so the weights of such a draw differ from the
                full-T draw's).
* ``zipf``    : the dsv2 local-expert shape without shared experts, at
                T in {64, 256, 1024, 4096, 16384, 65536}, with a router bias
                that gives a Zipf(1.2) popularity over the 160 experts.

Recipe: numpy ``Generator(PCG64)`` seeded with ``[2410, cfg_index]`` (for
``zipf`` the weights use ``[2410, 4]`` and x uses ``[2410, 4, T]``); draw
order x, router, gate, up, down, shared gate, shared up, shared down; each a
``standard_normal(float32)`` times sigma (1 for x, 0.02 for every weight);
bf16 values come from round-to-nearest-even of those fp32 draws.  The router
matrix stays fp32.  Expert weight stacks hold only the local experts:
gate and up ``[EL, I, H]``, down ``[EL, H, I]``; shared weights are the
concatenation of the shared experts: gate and up ``[n_shared*Is, H]``, down
``[H, n_shared*Is]``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

ZIPF_TOKENS = (64, 256, 1024, 4096, 16384, 65536)


@dataclasses.dataclass(frozen=True)
class MoEShape:
    name: str
    index: int          # seed component
    T: int              # tokens
    H: int              # hidden
    I: int              # routed expert SwiGLU width
    E: int              # router width (experts in the whole model)
    EL: int             # local experts computed here: [e0, e0 + EL)
    k: int              # top-k
    renorm: bool        # softmax over the k selected (True) or over all E
    e0: int = 0
    n_shared: int = 0   # shared experts applied to every token
    Is: int = 0         # width of each shared expert
    zipf_bias: bool = False

    @property
    def shared_inter(self) -> int:
        return self.n_shared * self.Is

    def with_tokens(self, T: int) -> "MoEShape":
        return dataclasses.replace(self, T=T)


SHAPES = {
    "tiny": MoEShape("tiny", 0, 512, 256, 512, 8, 8, 2, True),
    "mixtral": MoEShape("mixtral", 1, 16384, 4096, 3584, 8, 8, 2, True),
    "dbrx": MoEShape("dbrx", 2, 8192, 6144, 1344, 16, 16, 4, True),
    "dsv2": MoEShape("dsv2", 3, 16384, 5120, 1536, 160, 20, 6, False,
                     n_shared=2, Is=1536),
    "zipf": MoEShape("zipf", 4, 16384, 5120, 1536, 160, 20, 6, False,
                     zipf_bias=True),
    "mixtral_ep": MoEShape("mixtral_ep", 5, 16384, 4096, 14336, 8, 2, 2, True),
    "dbrx_ep": MoEShape("dbrx_ep", 6, 8192, 6144, 10752, 16, 2, 4, True),
}


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even) and return the uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def zipf_bias(E: int = 160, EL: int = 20, H: int = 5120, alpha: float = 1.2,
              sigma_w: float = 0.02) -> np.ndarray:
    """Router bias giving a Zipf(alpha) top-1 popularity over E experts.

    Logits of a N(0,1) token through an N(0, sigma_w) router are close to
    N(0, sz^2) with sz = sigma_w*sqrt(H); a Gumbel of matched variance has
    scale beta = sz*sqrt(6)/pi, under which a bias of -alpha*beta*ln(rank)
    makes the argmax pick rank r with probability proportional to r^-alpha.
    Ranks interleave the local experts [0, EL) across the popularity range:
    rank(e) = (E/EL)*(e mod EL) + floor(e/EL) + 1.
    """
    per = E // EL
    e = np.arange(E)
    rank = per * (e % EL) + e // EL + 1
    sz = sigma_w * math.sqrt(H)
    beta = sz * math.sqrt(6.0) / math.pi
    return (-alpha * beta * np.log(rank)).astype(np.float32)


@dataclasses.dataclass
class MoEInputs:
    shape: MoEShape
    x: np.ndarray             # [T,H] uint16 (bf16 bits)
    w_router: np.ndarray      # [E,H] float32
    bias: Optional[np.ndarray]  # [E] float32 or None
    w_gate: np.ndarray        # [EL,I,H] uint16
    w_up: np.ndarray          # [EL,I,H] uint16
    w_down: np.ndarray        # [EL,H,I] uint16
    shared_gate: Optional[np.ndarray] = None  # [n_shared*Is, H] uint16
    shared_up: Optional[np.ndarray] = None
    shared_down: Optional[np.ndarray] = None  # [H, n_shared*Is] uint16


def _normal_bf16(rng, shape, sigma):
    return bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma))


def make_inputs(shape: MoEShape, seed: Optional[tuple] = None,
                x_seed: Optional[tuple] = None, router_only: bool = False) -> MoEInputs:
    """Draw one workload.  ``seed`` overrides ``(2410, shape.index)``;
    ``x_seed`` (used by the zipf sweep) draws x from its own stream.
    ``router_only`` stops after the router matrix (x and the router are the
    first draws, so they are the same values either way)."""
    s = shape
    rng = np.random.Generator(np.random.PCG64(list(seed or (2410, s.index))))
    if x_seed is None and s.zipf_bias:
        x_seed = (2410, s.index, s.T)
    if x_seed is not None:
        x = _normal_bf16(np.random.Generator(np.random.PCG64(list(x_seed))), (s.T, s.H), 1.0)
    else:
        x = _normal_bf16(rng, (s.T, s.H), 1.0)
    w_router = rng.standard_normal((s.E, s.H), dtype=np.float32) * np.float32(0.02)
    bias = zipf_bias(s.E, s.EL, s.H) if s.zipf_bias else None
    if router_only:
        return MoEInputs(s, x, w_router, bias, None, None, None)
    w_gate = _normal_bf16(rng, (s.EL, s.I, s.H), 0.02)
    w_up = _normal_bf16(rng, (s.EL, s.I, s.H), 0.02)
    w_down = _normal_bf16(rng, (s.EL, s.H, s.I), 0.02)
    sg = su = sd = None
    if s.n_shared:
        sg = _normal_bf16(rng, (s.n_shared * s.Is, s.H), 0.02)
        su = _normal_bf16(rng, (s.n_shared * s.Is, s.H), 0.02)
        # down weights of shared expert j occupy columns [j*Is, (j+1)*Is)
        sd = np.concatenate([_normal_bf16(rng, (s.H, s.Is), 0.02)
                             for _ in range(s.n_shared)], axis=1)
    return MoEInputs(s, x, w_router, bias, w_gate, w_up, w_down, sg, su, sd)


def custom_shape(name="custom", index=100, **kw) -> MoEShape:
    """Shape for parity cases that are not one of the named workloads."""
    return MoEShape(name=name, index=index, **kw)
