"""GPU parity of every step of the routed MoE FFN against the CPU oracle, at
sizes the oracle finishes in seconds that still span several GEMM tiles and
ragged tails.  All calls go through the C-ABI (libmoe.so)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2410_12247_amd import moe, synth

from gpu_util import Dev, assert_close, assert_guards, bf16, bits, canary_fill, dev, f32, i32

pytestmark = pytest.mark.gpu

C = synth.custom_shape
CASES = {
    # the tiny workload in full
    "tiny": synth.SHAPES["tiny"],
    # ragged: H = 5*64, I = 3*64 (partial gate/up and down tiles), T not a
    # multiple of any tile
    "ragged8": C(name="ragged8", index=201, T=1000, H=320, I=192, E=8, EL=8, k=2, renorm=True),
    # a local window [3, 8) of 16 experts, top-4
    "window": C(name="window", index=202, T=777, H=512, I=384, E=16, EL=5, e0=3, k=4,
                renorm=True),
    # DeepSeekV2-like: 20 of 160 local, top-6 without renorm, shared experts
    "fine": C(name="fine", index=203, T=333, H=256, I=128, E=160, EL=20, k=6, renorm=False,
              n_shared=2, Is=128),
    # k == E
    "k_eq_E": C(name="k_eq_E", index=204, T=64, H=128, I=64, E=6, EL=6, k=6, renorm=False),
    # a single token
    "one": C(name="one", index=205, T=1, H=256, I=256, E=8, EL=8, k=2, renorm=True),
    # few experts with many rows each: several grouped token tiles per expert
    # plus a ragged last one
    "tall4": C(name="tall4", index=209, T=1500, H=192, I=320, E=4, EL=4, k=2, renorm=True),
    # many buckets and chunks: 160 local experts of 256 (the dispatch scan
    # over more than one wave of buckets), top-8, 24000 slots (24 histogram
    # chunks: the scan's sixteen-chunk unrolled loop plus a remainder)
    "wide": C(name="wide", index=218, T=3000, H=128, I=64, E=256, EL=160, e0=50, k=8,
              renorm=True),
}
# Shapes whose grouped GEMMs leave a partial last round on a 256-workgroup
# grid with K long enough to be cut (pieces of at least 32 K stages of 32):
# split2 cuts both GEMMs in 2 (K = 2048), split3 the down GEMM in 3
# (K = 3072, ragged experts in a local window), split4 and split8 the
# gate/up GEMM in 4 and 8 (K = 4096 and 8192, few rows per expert);
# split_shared runs the shared FFN (width 2048) as one grouped expert of all
# T rows, whose down GEMM (one tile, K = 2048) is cut in 2.
SPLIT_CASES = {
    "split2": C(name="split2", index=210, T=300, H=2048, I=2048, E=8, EL=8, k=2, renorm=True),
    "split3": C(name="split3", index=212, T=250, H=320, I=3072, E=16, EL=6, e0=5, k=4,
                renorm=False),
    "split4": C(name="split4", index=211, T=64, H=4096, I=512, E=8, EL=8, k=2, renorm=True),
    "split8": C(name="split8", index=213, T=32, H=8192, I=256, E=8, EL=8, k=2, renorm=True),
    "split_shared": C(name="split_shared", index=215, T=300, H=256, I=128, E=8, EL=8, k=2,
                      renorm=True, n_shared=1, Is=2048),
    # one partial round of more than half the grid in tiles of 192 or more
    # token rows at most half full (stream-K: the round's K stages spread
    # evenly over 256 workgroups, a piece ending one tile and starting the
    # next): the gate/up GEMM's 132 tiles (11 per expert, 192-row tiles,
    # K = 2048) with the down GEMM's 96 cut in 2; then the down GEMM's 144
    # tiles (256-row tiles, K = 512) with 24 gate/up tiles cut in 8
    "streamk_gu": C(name="streamk_gu", index=220, T=192, H=2048, I=1408, E=12, EL=12, k=4,
                    renorm=True),
    "streamk_dn": C(name="streamk_dn", index=221, T=256, H=6144, I=512, E=6, EL=6, k=2,
                    renorm=True),
}
CASES.update(SPLIT_CASES)
# the grouped tile heights the stream-K cases are built for (the library's
# own choice for experts of a few dozen rows is the 128-row tile, which
# never takes the stream-K tail)
SPLIT_TILE_ROWS = {"streamk_gu": 192, "streamk_dn": 256}

_cache = {}


def case(name):
    if name not in _cache:
        inp = synth.make_inputs(CASES[name])
        _, ids, w = oracle.route(inp.x, inp.w_router, inp.bias, inp.shape.k, inp.shape.renorm)
        _cache[name] = (inp, ids, w)
    return _cache[name]


def oracle_y(inp, ids, w, tokens):
    s = inp.shape
    return oracle.moe_tokens(inp.x, ids, w, tokens, inp.w_gate, inp.w_up, inp.w_down, s.e0,
                             s.n_shared, inp.shared_gate, inp.shared_up, inp.shared_down)


def weights_match(got, ref):
    # fp64 softmax rounded once on both sides; allow one fp32 ulp
    return np.all(np.abs(got.astype(np.float64) - ref) <= 2.0 ** -23 * np.abs(ref) + 1e-30)


@pytest.mark.parametrize("name", list(CASES))
def test_route(name):
    inp, ids, w = case(name)
    g = Dev(inp)
    s = inp.shape
    gids = torch.empty((s.T, s.k), dtype=torch.int32, device=dev())
    gw = torch.empty((s.T, s.k), dtype=torch.float32, device=dev())
    moe.route(g.d, g.x, g.w_router, g.bias, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)


@pytest.mark.parametrize("T,E", [(4000, 160), (8192, 160), (12001, 130), (16384, 160),
                                 (20000, 150)])
def test_route_many_experts_token_tiles(T, E):
    """The register-tiled router for 129-160 experts takes 1, 2 or 4 tokens
    per thread by batch size (below 8192, below 16384, from 16384): every band,
    ragged T and E not a multiple of the 32 expert groups, against the oracle
    bit for bit."""
    shp = C(name=f"tiles{T}_{E}", index=216, T=T, H=128, I=64, E=E, EL=4, k=6, renorm=False)
    inp = synth.make_inputs(shp, router_only=True)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, shp.k, shp.renorm)
    d = moe.dims(T, shp.H, shp.I, E, shp.k, 0, shp.EL, False)
    gids = torch.empty((T, shp.k), dtype=torch.int32, device=dev())
    gw = torch.empty((T, shp.k), dtype=torch.float32, device=dev())
    moe.route(d, bf16(inp.x), f32(inp.w_router), None, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)


@pytest.mark.parametrize("T,E,k", [(777, 256, 8), (2500, 256, 8), (1500, 200, 7)])
def test_maximum_experts_and_top_k(T, E, k):
    """The supported maximum, 256 experts with top-8 (and a ragged 200 with
    top-7): the router alone (16 experts per thread) and the whole forward
    (the lane router in blocks of 16 experts up to 4096 tokens, the
    combine of eight slots)
    against the oracle."""
    shp = C(name=f"max{T}_{E}", index=217, T=T, H=192, I=128, E=E, EL=32, e0=E - 40, k=k,
            renorm=True)
    inp = synth.make_inputs(shp)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, k, True)
    g = Dev(inp)
    gids = torch.empty((T, k), dtype=torch.int32, device=dev())
    gw = torch.empty((T, k), dtype=torch.float32, device=dev())
    moe.route(g.d, g.x, g.w_router, g.bias, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)
    buf = g.forward()
    assert np.array_equal(buf.topk_ids.cpu().numpy(), ids)
    counts, *_ = oracle.dispatch(ids, shp.e0, shp.EL)
    assert np.array_equal(buf.counts.cpu().numpy(), counts)
    assert_close(buf.y.cpu().numpy(), oracle_y(inp, ids, w, np.arange(T)), f"E={E} k={k}")


@pytest.mark.parametrize("T,E,H,k,renorm,use_bias", [
    (1, 1, 64, 1, True, False),         # one token, one expert, one stage
    (100, 3, 128, 2, False, True),      # E <= 4: two waves of 2 experts, two stages
    (60000, 4, 64, 2, True, False),     # E <= 4, a large batch
    (1000, 5, 448, 2, True, True),      # 7 stages: not a multiple of the 6-slot ring
    (16383, 8, 384, 2, True, False),    # four waves of 2 experts (Mixtral's form)
    (30001, 7, 128, 3, False, True),    # E <= 8, a large batch, ragged last block
    (8193, 16, 768, 4, True, False),    # 2 per lane in two sets of 32 tokens (DBRX's form)
    (14000, 11, 192, 4, False, True),   # E <= 16 past ~13650 tokens: 4 per lane
    (33, 16, 6144, 4, True, True),      # DBRX's width, one partial workgroup
])
def test_route_lane_shapes(T, E, H, k, renorm, use_bias):
    """The lane-per-token router (E <= 16) in each of its shapes, picked by
    expert count and batch size, with ragged token blocks, 1 to 96 stages
    and the bias, against the oracle bit for bit."""
    rng = np.random.default_rng(1000 + E + T)
    xb = synth.bf16_bits(rng.standard_normal((T, H), dtype=np.float32))
    wr = rng.standard_normal((E, H), dtype=np.float32) * np.float32(0.02)
    bias = (rng.standard_normal(E, dtype=np.float32) * np.float32(0.1)) if use_bias else None
    _, ids, w = oracle.route(xb, wr, bias, k, renorm)
    d = moe.dims(T, H, 64, E, k, renormalize=renorm)
    gids = torch.empty((T, k), dtype=torch.int32, device=dev())
    gw = torch.empty((T, k), dtype=torch.float32, device=dev())
    moe.route(d, bf16(xb), f32(wr), f32(bias) if use_bias else None, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)


@pytest.mark.parametrize("T,E,H,k,renorm,use_bias", [
    (1, 8, 4096, 2, True, False),       # decode, Mixtral's router
    (1, 1, 64, 1, True, True),          # one expert, one block
    (33, 16, 6144, 4, True, True),      # DBRX's width, 16 lanes
    (511, 5, 192, 2, False, True),      # three blocks (odd: the pair loop's tail)
    (512, 8, 64, 2, True, False),       # the last batch size on the chain kernel
    (513, 8, 64, 2, True, False),       # the first on the lane kernel
    (32, 16, 8192, 3, False, False),    # the widest 16-expert row in 64 KB of LDS
    (2, 8, 12288, 2, True, True),       # the widest 8-expert row
])
def test_route_chain_shapes(T, E, H, k, renorm, use_bias):
    """The chain-per-lane router for few tokens (one wave per token, a lane
    per expert, x widened into LDS, router rows through an LDS ring): 1 to
    192 blocks of 64 h, odd block counts, the batch-size boundary with the
    lane kernel, the widest rows that fit, with the bias, against the
    oracle bit for bit."""
    rng = np.random.default_rng(2000 + E + T + H)
    xb = synth.bf16_bits(rng.standard_normal((T, H), dtype=np.float32))
    wr = rng.standard_normal((E, H), dtype=np.float32) * np.float32(0.02)
    bias = (rng.standard_normal(E, dtype=np.float32) * np.float32(0.1)) if use_bias else None
    _, ids, w = oracle.route(xb, wr, bias, k, renorm)
    d = moe.dims(T, H, 64, E, k, renormalize=renorm)
    gids = torch.empty((T, k), dtype=torch.int32, device=dev())
    gw = torch.empty((T, k), dtype=torch.float32, device=dev())
    moe.route(d, bf16(xb), f32(wr), f32(bias) if use_bias else None, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)


@pytest.mark.parametrize("name,kw", [
    ("tiny", {}),
    ("fine", {}),                                          # shared experts, no renorm
    ("ragged8", dict(gemm_mode=moe.GEMM_DENSE)),           # dense launches, host counts
    ("split4", {}),                                        # K-split partials and fixup
    ("window", dict(pipeline_n=5, exact_order=True)),      # one expert per stage
    ("tall4", dict(pipeline_n=2, chunk_mode=moe.CHUNK_TOKENS, timing=True)),
])
def test_workspace_guards_untouched(name, kw):
    """Canary-filled guard gaps around every workspace region hold the
    canary after two forwards under each option set (no kernel writes past
    its region), and the forward still routes as the oracle does."""
    inp, ids, _ = case(name)
    g = Dev(inp)
    o = moe.opts(**kw)
    guards = moe.workspace_guards(g.d, o)
    assert len(guards) >= 15
    buf = g.buffers(o)
    canary_fill(buf.ws)
    g.run(buf)
    g.run(buf)
    assert_guards(buf.ws, guards, name)
    assert np.array_equal(buf.topk_ids.cpu().numpy(), ids)


# Decode-sized shapes whose grouped down GEMM takes the skinny tile (at most
# 64 rows per expert, at least two 64-column tiles per compute unit of a
# 256-CU device): tile rows 16, 32 and 64, K shorter than the LDS ring,
# more tiles per compute unit than fit its LDS at once, a local window
# whose later pipeline stages start at expert e_first > 0.
@pytest.mark.parametrize("T,E,EL,e0,k,H,I,shared", [
    (5, 64, 64, 0, 8, 1024, 256, 0),      # 16-row tiles
    (64, 8, 8, 0, 2, 4096, 256, 0),       # 32-row tiles
    (64, 4, 4, 0, 2, 8192, 128, 0),       # 64-row tiles; 4 K stages
    (64, 2, 2, 0, 2, 16384, 64, 0),       # every expert exactly 64 rows
    (64, 4, 4, 0, 2, 16384, 128, 0),      # 64-row tiles, 4 per CU (2 resident at once)
    (48, 32, 16, 8, 8, 4096, 128, 0),     # a local window; PN = 2 stays skinny
    (40, 160, 160, 0, 6, 512, 256, 512),  # many experts, most empty; shared FFN
])
def test_skinny_down_gemm(T, E, EL, e0, k, H, I, shared):
    """The skinny down tile: output within the tolerance of the oracle, and
    in exact order the same bits as per-expert dense launches of the general
    tile, for any pipeline number and through moe_ffn_group."""
    shp = C(name=f"skinny{T}_{E}", index=219, T=T, H=H, I=I, E=E, EL=EL, e0=e0, k=k,
            renorm=True, n_shared=1 if shared else 0, Is=shared)
    inp = synth.make_inputs(shp)
    _, ids, w = oracle.route(inp.x, inp.w_router, inp.bias, k, True)
    g = Dev(inp)
    buf = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True))
    assert np.array_equal(buf.topk_ids.cpu().numpy(), ids)
    y = buf.y.clone()
    assert_close(y.cpu().numpy(), oracle_y(inp, ids, w, np.arange(T)), f"skinny T={T} E={E}")
    dense = g.forward(moe.opts(gemm_mode=moe.GEMM_DENSE, exact_order=True)).y
    assert torch.equal(y, dense), "skinny grouped and dense forwards differ"
    # default options: the gate/up GEMM may cut its last round along K
    assert_close(g.forward(moe.opts()).y.cpu().numpy(), y.cpu().numpy(), "default options",
                 2e-3, 1e-4)
    # pipelined stages: every stage after the first starts at expert e_first > 0
    for pn in [p for p in (2, 4) if EL % p == 0]:
        yp = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, pipeline_n=pn, exact_order=True)).y
        assert torch.equal(yp, y), f"PN={pn} differs"
    if 2 * EL <= 256:  # token-range stages take PN * EL dispatch buckets
        yt = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, pipeline_n=2, exact_order=True,
                                chunk_mode=moe.CHUNK_TOKENS)).y
        assert torch.equal(yt, y), "token-range stages differ"
    # moe_ffn_group over gathered rows against per-expert dense launches
    counts, offsets, sorted_slot, _ = oracle.dispatch(ids, e0, EL)
    R = int(offsets[-1])
    assert R > 0
    xp = bf16(inp.x[sorted_slot // k])
    act = torch.empty((R, I), dtype=torch.bfloat16, device=dev())
    yg = torch.full((R, H), float("nan"), dtype=torch.float32, device=dev())
    moe.ffn_group(g.d, 0, EL, i32(offsets), xp, g.w_gate, g.w_up, g.w_down, act, yg)
    yd = torch.full_like(yg, float("nan"))
    act_d = torch.empty_like(act)
    for e in range(EL):
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        if r1 > r0:
            moe.ffn_dense(r1 - r0, H, I, xp[r0:r1], g.w_gate[e], g.w_up[e], g.w_down[e],
                          act_d[r0:r1], yd[r0:r1])
    torch.cuda.synchronize()
    assert torch.equal(yg, yd), "moe_ffn_group and moe_ffn_dense bits differ"


def test_route_ties_and_signed_zero():
    """Exact ties in the logits (duplicated router rows, zero rows) must go to
    the lower expert index, -0 and +0 being equal."""
    rng = np.random.default_rng(9)
    T, H, E, k = 300, 64, 12, 4
    xb = synth.bf16_bits(rng.standard_normal((T, H), dtype=np.float32))
    wr = rng.standard_normal((E, H), dtype=np.float32) * np.float32(0.1)
    wr[5] = wr[2]
    wr[9] = wr[2]
    wr[7] = 0.0
    wr[3] = 0.0
    xb[:20] = synth.bf16_bits(np.zeros((20, H), np.float32))  # all logits +0
    xb[20:40] = synth.bf16_bits(-np.zeros((20, H), np.float32))
    _, ids, w = oracle.route(xb, wr, None, k, True)
    d = moe.dims(T, H, 64, E, k)
    gids = torch.empty((T, k), dtype=torch.int32, device=dev())
    gw = torch.empty((T, k), dtype=torch.float32, device=dev())
    moe.route(d, bf16(xb), f32(wr), None, gids, gw)
    torch.cuda.synchronize()
    assert np.array_equal(gids.cpu().numpy(), ids)
    assert weights_match(gw.cpu().numpy(), w)


@pytest.mark.parametrize("name", list(CASES))
def test_permute_and_gather(name):
    inp, ids, _ = case(name)
    s = inp.shape
    g = Dev(inp)
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, s.e0, s.EL)
    rcap = s.T * min(s.k, s.EL)
    gc = torch.empty(s.EL, dtype=torch.int32, device=dev())
    go = torch.empty(s.EL + 1, dtype=torch.int32, device=dev())
    gss = torch.full((rcap,), -7, dtype=torch.int32, device=dev())
    gsr = torch.empty(s.T * s.k, dtype=torch.int32, device=dev())
    gxp = torch.empty((rcap, s.H), dtype=torch.bfloat16, device=dev())
    ws = torch.empty(moe.workspace_bytes(g.d), dtype=torch.uint8, device=dev())
    moe.permute(g.d, i32(ids), g.x, gc, go, gss, gsr, gxp, ws)
    torch.cuda.synchronize()
    R = int(offsets[-1])
    assert np.array_equal(gc.cpu().numpy(), counts)
    assert np.array_equal(go.cpu().numpy(), offsets)
    assert np.array_equal(gss.cpu().numpy()[:R], sorted_slot)
    assert np.array_equal(gsr.cpu().numpy(), slot_row)
    assert np.array_equal(bits(gxp[:R]), inp.x[sorted_slot // s.k])


@pytest.mark.parametrize("name", ["tiny", "ragged8", "window", "fine"])
def test_ffn_group_and_dense_rows(name):
    """GroupGemm over all local experts and DenseGemm per expert: every
    dispatched row against the oracle's expert FFN, and the two GEMM kinds
    bit-identical."""
    inp, ids, _ = case(name)
    s = inp.shape
    g = Dev(inp)
    counts, offsets, sorted_slot, _ = oracle.dispatch(ids, s.e0, s.EL)
    R = int(offsets[-1])
    xp = inp.x[sorted_slot // s.k]
    gxp = bf16(xp) if R else torch.empty((0, s.H), dtype=torch.bfloat16, device=dev())
    act = torch.empty((max(R, 1), s.I), dtype=torch.bfloat16, device=dev())
    yg = torch.full((max(R, 1), s.H), float("nan"), dtype=torch.float32, device=dev())
    moe.ffn_group(g.d, 0, s.EL, i32(offsets), gxp if R else act, g.w_gate, g.w_up,
                  g.w_down, act, yg)
    yd = torch.full((max(R, 1), s.H), float("nan"), dtype=torch.float32, device=dev())
    act_d = torch.empty_like(act)
    for e in range(s.EL):
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        if r1 > r0:
            moe.ffn_dense(r1 - r0, s.H, s.I, gxp[r0:r1], g.w_gate[e], g.w_up[e], g.w_down[e],
                          act_d[r0:r1], yd[r0:r1])
    torch.cuda.synchronize()
    experts = np.repeat(np.arange(s.EL), counts)
    ref = oracle.expert_row_list(inp.x, sorted_slot // s.k, experts, inp.w_gate, inp.w_up,
                                 inp.w_down)
    got_g = yg.cpu().numpy()[:R]
    assert_close(got_g, ref, f"{name} group rows")
    assert np.array_equal(got_g, yd.cpu().numpy()[:R]), "GroupGemm and DenseGemm bits differ"


@pytest.mark.parametrize("name", ["ragged8", "fine"])
def test_combine(name):
    inp, ids, w = case(name)
    s = inp.shape
    g = Dev(inp)
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, s.e0, s.EL)
    R = int(offsets[-1])
    rng = np.random.default_rng(3)
    yp = rng.standard_normal((max(R, 1), s.H)).astype(np.float32)
    init = rng.standard_normal((s.T, s.H)).astype(np.float32)
    ref0 = oracle.combine(yp, slot_row.reshape(s.T, s.k), w)
    ref1 = oracle.combine(yp, slot_row.reshape(s.T, s.k), w, init)
    y = torch.full((s.T, s.H), float("nan"), dtype=torch.float32, device=dev())
    moe.combine(g.d, 0, s.EL, f32(yp), i32(ids), i32(slot_row), f32(w), y, 0)
    torch.cuda.synchronize()
    assert_close(y.cpu().numpy(), ref0, "combine", max_abs=1e-5, rel_fro=1e-6)
    # accumulate over stages in order: same bits as one call
    y1 = f32(init)
    moe.combine(g.d, 0, s.EL, f32(yp), i32(ids), i32(slot_row), f32(w), y1, 1)
    y2 = f32(init)
    half = s.EL // 2
    moe.combine(g.d, 0, half, f32(yp), i32(ids), i32(slot_row), f32(w), y2, 1)
    moe.combine(g.d, half, s.EL - half, f32(yp), i32(ids), i32(slot_row), f32(w), y2, 1)
    torch.cuda.synchronize()
    assert_close(y1.cpu().numpy(), ref1, "combine+init", max_abs=1e-5, rel_fro=1e-6)
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("name", list(CASES))
def test_forward(name):
    inp, ids, w = case(name)
    s = inp.shape
    buf = Dev(inp).forward()
    counts, *_ = oracle.dispatch(ids, s.e0, s.EL)
    assert np.array_equal(buf.topk_ids.cpu().numpy(), ids)
    assert weights_match(buf.topk_w.cpu().numpy(), w)
    assert np.array_equal(buf.counts.cpu().numpy(), counts)
    ref = oracle_y(inp, ids, w, np.arange(s.T))
    assert_close(buf.y.cpu().numpy(), ref, f"{name} forward")


@pytest.mark.parametrize("name", ["ragged8", "fine"])
def test_forward_invariant_to_pipeline_and_gemm_kind(name):
    """With MOE_FLAG_EXACT_ORDER, PN, the GEMM kind, the CU budget, serial
    stages and a repeated call all give the same bits."""
    inp, _, _ = case(name)
    g = Dev(inp)
    EL = inp.shape.EL
    base = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True)).y.clone()
    for pn in [p for p in (1, 2, 4, 5) if EL % p == 0]:
        for mode in (moe.GEMM_GROUP, moe.GEMM_DENSE, moe.GEMM_AUTO):
            y = g.forward(moe.opts(gemm_mode=mode, pipeline_n=pn, exact_order=True)).y
            assert torch.equal(y, base), f"PN={pn} mode={mode} differs"
        y = g.forward(moe.opts(pipeline_n=pn, exact_order=True, serial=True)).y
        assert torch.equal(y, base), f"serial PN={pn} differs"
    y = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, gemm_cu_budget=40, exact_order=True)).y
    assert torch.equal(y, base), "CU budget changes the bits"


@pytest.mark.parametrize("name", ["ragged8", "fine"])
def test_side_cus_and_library_pipeline_number(name):
    """CU-masked side streams (the gather and combine streams on side_cus
    CUs, the GEMM stream and its grid on the rest) and the library's own
    choice of PN (pipeline_n = 0, after the row counts): same bits as the
    unmasked forward in exact order, and the chosen PN is the one
    moe_pipeline_plan gives for those counts."""
    inp, ids, w = case(name)
    g = Dev(inp)
    s = inp.shape
    base = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True)).y.clone()
    for side in (8, 32, 64):
        for pn in [p for p in (1, 2, 4) if s.EL % p == 0]:
            y = g.forward(moe.opts(pipeline_n=pn, side_cus=side, exact_order=True)).y
            assert torch.equal(y, base), f"side_cus={side} PN={pn} changes the bits"
    buf = g.forward(moe.opts(pipeline_n=0, timing=True, exact_order=True))
    assert torch.equal(buf.y, base)
    chosen = moe.last_timing()["pipeline_n"]
    counts = buf.counts.cpu().numpy()
    plan = moe.pipeline_plan(g.d, moe.opts(pipeline_n=0, exact_order=True), counts, 0)
    assert chosen == plan["pipeline_n"]
    ref = oracle_y(inp, ids, w, np.arange(s.T))
    y = g.forward(moe.opts(pipeline_n=0, side_cus=32)).y
    assert_close(y.cpu().numpy(), ref, f"{name} PN auto, side CUs")


@pytest.mark.parametrize("name", ["ragged8", "fine"])
def test_forward_timing_modes(name):
    """Timing every phase or only the GEMMs leaves the result unchanged; the
    GEMM-only mode reports GEMM time and zero for the other phases, on one
    stream (PN = 1) and across streams (PN > 1, shared experts)."""
    inp, _, _ = case(name)
    g = Dev(inp)
    for pn in (1, 2):
        base = g.forward(moe.opts(pipeline_n=pn)).y.clone()
        y = g.forward(moe.opts(pipeline_n=pn, timing=True)).y
        t_all = moe.last_timing()
        assert torch.equal(y, base)
        y = g.forward(moe.opts(pipeline_n=pn, timing="gemm")).y
        t_gemm = moe.last_timing()
        assert torch.equal(y, base)
        assert t_all["route_ms"] > 0 and t_all["combine_ms"] > 0 and t_all["total_ms"] > 0
        assert t_gemm["route_ms"] == 0 and t_gemm["combine_ms"] == 0 and t_gemm["total_ms"] == 0
        assert t_gemm["gateup_ms"] > 0 and t_gemm["down_ms"] > 0
        assert t_gemm["gateup_launches"] == t_all["gateup_launches"] >= 1
        if inp.shape.n_shared:
            assert t_gemm["shared_ms"] > 0
        # timed calls add up until read: three calls, one read
        for _ in range(3):
            y = g.forward(moe.opts(pipeline_n=pn, timing="gemm")).y
        t3 = moe.last_timing()
        assert t3["calls"] == 3 and t_gemm["calls"] == 1
        assert t3["gateup_launches"] == 3 * t_gemm["gateup_launches"]
        assert t3["group_stages"] == 3 * t_gemm["group_stages"]
        assert torch.equal(y, base)


@pytest.mark.parametrize("name", ["tall4", "ragged8", "window"])
def test_dense_tile_heights(name):
    """DenseGemm and GroupGemm launches with every tile height (128, 192,
    256, 320 token rows, forced, and the one the launch-cost model picks):
    the same bits as GroupGemm's own choice in exact order, and within the
    oracle bar with the K split."""
    inp, ids, w = case(name)
    g = Dev(inp)
    s = inp.shape
    base = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True)).y.clone()
    ref = oracle_y(inp, ids, w, np.arange(s.T))
    for bm in (0, 128, 192, 256, 320):
        for pn in (1, s.EL):
            y = g.forward(moe.opts(gemm_mode=moe.GEMM_DENSE, dense_tile_rows=bm, pipeline_n=pn,
                                   exact_order=True)).y
            assert torch.equal(y, base), f"dense tile {bm} PN={pn} changes the bits"
        y = g.forward(moe.opts(gemm_mode=moe.GEMM_DENSE, dense_tile_rows=bm)).y
        assert_close(y.cpu().numpy(), ref, f"{name} dense tile {bm} with K split")
        y = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, group_tile_rows=bm,
                               exact_order=True)).y
        assert torch.equal(y, base), f"group tile {bm} changes the bits"
        y = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, group_tile_rows=bm)).y
        assert_close(y.cpu().numpy(), ref, f"{name} group tile {bm} with K split")
    # AUTO with one expert per stage may take either kind: same bits again
    y = g.forward(moe.opts(pipeline_n=s.EL, exact_order=True)).y
    assert torch.equal(y, base)


@pytest.mark.parametrize("name", ["ragged8", "fine", "one"])
def test_forward_token_range_stages(name):
    """Token-range stages (each stage all experts over a token range, weights
    re-read per stage) give the same bits and counts as expert-group stages,
    for PN that need not divide EL and PN above T."""
    inp, ids, _ = case(name)
    g = Dev(inp)
    s = inp.shape
    ref = g.forward(moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True))
    base, counts = ref.y.clone(), ref.counts.clone()
    for pn in (1, 2, 3, 7):
        if pn * s.EL > 256:
            continue
        for mode in (moe.GEMM_GROUP, moe.GEMM_DENSE, moe.GEMM_AUTO):
            buf = g.forward(moe.opts(gemm_mode=mode, pipeline_n=pn, chunk_mode=moe.CHUNK_TOKENS,
                                     exact_order=True))
            assert torch.equal(buf.y, base), f"token stages PN={pn} mode={mode} differ"
            assert torch.equal(buf.counts, counts)


@pytest.mark.parametrize("name", list(SPLIT_CASES))
def test_forward_k_split(name):
    """The K split of the grouped GEMM's last round: the result meets the
    oracle bar, is the same bits on every call, and differs from the
    one-pass (exact-order) result only by accumulation order; with pipeline
    stages and a CU budget (other tile counts and splits) it meets the bar
    too."""
    inp, ids, w = case(name)
    g = Dev(inp)
    s = inp.shape
    ref = oracle_y(inp, ids, w, np.arange(s.T))
    bm = SPLIT_TILE_ROWS.get(name, 0)
    y = g.forward(moe.opts(group_tile_rows=bm)).y.clone()
    assert_close(y.cpu().numpy(), ref, f"{name} split")
    for _ in range(2):
        assert torch.equal(g.forward(moe.opts(group_tile_rows=bm)).y, y), \
            "split result not deterministic"
    ye = g.forward(moe.opts(exact_order=True, group_tile_rows=bm)).y.clone()
    assert_close(ye.cpu().numpy(), ref, f"{name} exact order")
    # where the fp32 down GEMM is cut, the pieces' sums differ from one pass
    # in the last bits somewhere (the evidence that the split ran; a cut
    # gate/up shows only through rare bf16 rounding flips of act)
    if name in ("split2", "split3", "split_shared", "streamk_gu", "streamk_dn"):
        assert not torch.equal(y, ye), "no tile was split"
    assert_close(y.cpu().numpy(), ye.cpu().numpy().astype(np.float64), f"{name} split vs exact",
                 max_abs=2e-3, rel_fro=1e-4)
    for o in (moe.opts(pipeline_n=2, group_tile_rows=bm), moe.opts(gemm_cu_budget=48),
              moe.opts(gemm_cu_budget=96, group_tile_rows=bm)):
        yo = g.forward(o).y
        assert_close(yo.cpu().numpy(), ref, f"{name} PN={o.pipeline_n} budget={o.gemm_cu_budget}")


def exact_sum_inputs(inp):
    """Integer-valued operands whose GEMM sums are exact in fp32 in any
    order: x is 1 on its first 64 features (the rest in {-1, 0, 1}, so the
    routing still varies), every gate row sums 32 of those ones (g = 32, and
    silu(32) = 32 in fp32: e^-32 vanishes beside 1), every up row has at most
    4 entries of +-1 among them (u in [-4, 4], act = 32 u exact in bf16),
    and the down weights are in {-1, 0, 1}.  Any cut of K then gives the
    one-pass bits."""
    s = inp.shape
    rng = np.random.default_rng(s.index)
    one = synth.bf16_bits(np.ones(1, np.float32))[0]

    def ints(shape, lo=-1, hi=1):
        return synth.bf16_bits(rng.integers(lo, hi + 1, size=shape).astype(np.float32))

    x = ints((s.T, s.H))
    x[:, :64] = one
    inp.x = x

    def gate_up(rows):
        g = np.zeros((rows, s.H), np.uint16)
        g[:, :32] = one
        u = np.zeros((rows, s.H), np.float32)
        for r in range(rows):
            u[r, rng.choice(64, size=4, replace=False)] = rng.choice([-1.0, 1.0], size=4)
        return g, synth.bf16_bits(u)

    wg, wu = zip(*(gate_up(s.I) for _ in range(s.EL)))
    inp.w_gate, inp.w_up = np.stack(wg), np.stack(wu)
    inp.w_down = ints((s.EL, s.H, s.I))
    if s.n_shared:
        inp.shared_gate, inp.shared_up = gate_up(s.n_shared * s.Is)
        inp.shared_down = ints((s.H, s.n_shared * s.Is))
    return inp


@pytest.mark.parametrize("name", list(SPLIT_CASES))
def test_k_split_exact_sums(name):
    """Every K split (equal pieces, stream-K, under pipeline stages and CU
    budgets) on operands whose sums are exact in any order: the same bits as
    one pass over K, so each piece covers exactly its stages and the fixup
    adds exactly the tile's pieces."""
    inp = exact_sum_inputs(synth.make_inputs(CASES[name]))
    g = Dev(inp)
    ye = g.forward(moe.opts(exact_order=True)).y.clone()
    assert torch.isfinite(ye).all()
    bm = SPLIT_TILE_ROWS.get(name, 0)
    for o in (moe.opts(group_tile_rows=bm), moe.opts(), moe.opts(pipeline_n=2, group_tile_rows=bm),
              moe.opts(gemm_cu_budget=48, group_tile_rows=bm), moe.opts(gemm_cu_budget=96)):
        y = g.forward(o).y
        assert torch.equal(y, ye), f"{name} PN={o.pipeline_n} budget={o.gemm_cu_budget}"


@pytest.mark.parametrize("T,E,bias", [(1, 17, False), (37, 40, True), (32, 160, True),
                                       (1024, 17, False),
                                       (1024, 160, True), (1025, 160, False), (64, 32, True),
                                       (33, 256, False), (500, 96, True), (4096, 40, True),
                                       (4097, 40, False)])
def test_forward_routing_many_experts(T, E, bias):
    """Routing inside the forward for E > 16: at a few tokens (tokens x
    expert blocks of 16 up to 512) from the chain-per-lane router, else up
    to 4096 tokens from the lane-per-token router, both in blocks of 16
    experts (a ragged last block when 16 does not divide E; 33 tokens leave
    a ragged token block), through the workspace, and a separate selection;
    above that from the register-tiled router.  Ids, weights, counts and y match the oracle;
    duplicated router rows make exact ties, which go to the lower expert
    index."""
    shp = C(name=f"many{T}_{E}", index=214, T=T, H=192, I=64, E=E, EL=4, e0=E - 4, k=6,
            renorm=False)
    inp = synth.make_inputs(shp)
    if bias:
        inp.bias = np.random.default_rng(E).standard_normal(E).astype(np.float32)
    inp.w_router[E - 1] = inp.w_router[3]
    inp.w_router[9] = inp.w_router[3]
    inp.w_router[E - 2] = inp.w_router[E - 3]
    _, ids, w = oracle.route(inp.x, inp.w_router, inp.bias, shp.k, shp.renorm)
    buf = Dev(inp).forward()
    assert np.array_equal(buf.topk_ids.cpu().numpy(), ids)
    assert weights_match(buf.topk_w.cpu().numpy(), w)
    counts, *_ = oracle.dispatch(ids, shp.e0, shp.EL)
    assert np.array_equal(buf.counts.cpu().numpy(), counts)
    assert_close(buf.y.cpu().numpy(), oracle_y(inp, ids, w, np.arange(T)), f"T={T} E={E}")


def test_forward_token_stages_hot_expert_and_empty_stages():
    """All rows on one expert, PN larger than the token count leaves empty
    stages; shared experts make every stage accumulate."""
    shp = C(name="hot_tok", index=208, T=5, H=128, I=64, E=8, EL=8, k=1, renorm=True,
            n_shared=1, Is=64)
    inp = synth.make_inputs(shp)
    inp.bias = np.zeros(8, np.float32)
    inp.bias[2] = 1e4
    _, ids, w = oracle.route(inp.x, inp.w_router, inp.bias, 1, True)
    g = Dev(inp)
    for pn in (4, 8, 16):
        buf = g.forward(moe.opts(pipeline_n=pn, chunk_mode=moe.CHUNK_TOKENS))
        assert np.array_equal(buf.counts.cpu().numpy(), [0, 0, 5, 0, 0, 0, 0, 0])
        assert_close(buf.y.cpu().numpy(), oracle_y(inp, ids, w, np.arange(5)), f"PN={pn}")


def test_forward_all_tokens_to_one_expert():
    shp = C(name="hot", index=206, T=700, H=256, I=128, E=8, EL=8, k=1, renorm=True)
    inp = synth.make_inputs(shp)
    inp.bias = np.zeros(8, np.float32)
    inp.bias[5] = 1e4
    _, ids, w = oracle.route(inp.x, inp.w_router, inp.bias, 1, True)
    assert np.all(ids == 5)
    for mode in (moe.GEMM_GROUP, moe.GEMM_DENSE):
        buf = Dev(inp).forward(moe.opts(gemm_mode=mode, pipeline_n=4))
        assert np.array_equal(buf.counts.cpu().numpy(), [0, 0, 0, 0, 0, 700, 0, 0])
        assert_close(buf.y.cpu().numpy(), oracle_y(inp, ids, w, np.arange(700)), "hot expert")


def test_forward_no_local_rows():
    """Every token routes outside the local window: y is exactly zero."""
    shp = C(name="away", index=207, T=100, H=128, I=64, E=8, EL=2, e0=0, k=1, renorm=True)
    inp = synth.make_inputs(shp)
    inp.bias = np.zeros(8, np.float32)
    inp.bias[6] = 1e4
    buf = Dev(inp).forward(moe.opts(gemm_mode=moe.GEMM_AUTO, pipeline_n=2))
    assert np.all(buf.counts.cpu().numpy() == 0)
    assert torch.count_nonzero(buf.y).item() == 0


def test_zero_tokens_is_a_noop():
    shp = synth.SHAPES["tiny"]
    d = moe.dims(0, shp.H, shp.I, shp.E, shp.k)
    y = torch.full((1, shp.H), 3.0, device=dev())
    ws = torch.empty(16, dtype=torch.uint8, device=dev())
    dummy = torch.empty(1, dtype=torch.bfloat16, device=dev())
    moe.forward(d, moe.opts(), dummy, f32(np.zeros(1)), None, dummy, dummy, dummy, None, None,
                None, y, None, None, None, ws)
    torch.cuda.synchronize()
    assert torch.all(y == 3.0)


def test_forward_from_two_host_threads():
    """Two host threads calling moe_ffn_forward on one device at once, each on
    its own torch stream and buffers, with options that use the library's
    side streams, events and pinned counts (shared experts, PN = 2, DenseGemm
    needing host row counts): every result has the bits of the same call made
    alone."""
    import threading

    names = ("fine", "ragged8")
    opts = {"fine": moe.opts(pipeline_n=2, exact_order=True),
            "ragged8": moe.opts(gemm_mode=moe.GEMM_DENSE, pipeline_n=4, exact_order=True)}
    devs = {n: Dev(case(n)[0]) for n in names}
    ref = {n: devs[n].forward(opts[n]).y.clone() for n in names}
    errors = []

    def worker(n):
        try:
            g = devs[n]
            s = torch.cuda.Stream()
            buf = g.buffers(opts[n])
            with torch.cuda.stream(s):
                for _ in range(20):
                    g.run(buf, stream=s)
                    s.synchronize()
                    if not torch.equal(buf.y, ref[n]):
                        errors.append(f"{n}: bits differ")
                        return
        except Exception as e:  # reported below
            errors.append(f"{n}: {e!r}")

    threads = [threading.Thread(target=worker, args=(n,)) for n in names]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a forward thread did not finish"
    assert not errors, errors
