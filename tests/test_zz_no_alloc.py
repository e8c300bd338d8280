"""moe_ffn_forward_noalloc (the forward for callers that cannot allocate:
its scratch is the library's static device buffer) against moe_ffn_forward
on the same inputs and options, through the C-ABI: two calls in a row, the
second on a smaller input, each with the same ids, weights and counts bit
for bit, the same y bits, and y within the FFN tolerance of the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_12247_amd import moe, synth

from gpu_util import Dev, assert_close

pytestmark = pytest.mark.gpu

C = synth.custom_shape
# the first call fills most of the buffer; the second, smaller one adds
# shared experts (all steps on the caller's stream) and a local window
FIRST = synth.SHAPES["tiny"]
SECOND = C(name="noalloc2", index=219, T=200, H=256, I=128, E=160, EL=20, e0=20, k=6,
           renorm=False, n_shared=2, Is=128)


def _noalloc(g, o):
    s = g.s
    dev = g.x.device
    y = torch.full((s.T, s.H), float("nan"), dtype=torch.float32, device=dev)
    ids = torch.full((s.T, s.k), -1, dtype=torch.int32, device=dev)
    w = torch.full((s.T, s.k), float("nan"), dtype=torch.float32, device=dev)
    counts = torch.full((s.EL,), -1, dtype=torch.int32, device=dev)
    moe.forward_noalloc(g.d, o, g.x, g.w_router, g.bias, g.w_gate, g.w_up, g.w_down, g.sg,
                        g.su, g.sd, y, ids, w, counts)
    torch.cuda.synchronize()
    return y, ids, w, counts


@pytest.mark.parametrize("o", [moe.opts(), moe.opts(exact_order=True)],
                         ids=["default", "exact_order"])
def test_noalloc_matches_forward_twice(o):
    for shp in (FIRST, SECOND):
        print(f"noalloc: {shp.name} T={shp.T}", flush=True)
        inp = synth.make_inputs(shp)
        g = Dev(inp)
        # (the entry point's own layout runs one stream: no second K-split
        # scratch for the shared FFN, so it is smaller than workspace_bytes)
        y, ids, w, counts = _noalloc(g, o)
        ref = g.forward(o)
        assert torch.equal(ids, ref.topk_ids)
        assert torch.equal(w, ref.topk_w)
        assert torch.equal(counts, ref.counts)
        assert torch.equal(y, ref.y), "noalloc y differs from moe_ffn_forward"
        _, oids, ow = oracle.route(inp.x, inp.w_router, inp.bias, shp.k, shp.renorm)
        assert np.array_equal(ids.cpu().numpy(), oids)
        yo = oracle.moe_tokens(inp.x, oids, ow, np.arange(shp.T), inp.w_gate, inp.w_up,
                               inp.w_down, shp.e0, shp.n_shared, inp.shared_gate,
                               inp.shared_up, inp.shared_down)
        assert_close(y.cpu().numpy(), yo, f"noalloc {shp.name}")
