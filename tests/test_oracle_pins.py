"""Pins of the CPU oracle against facts fixed outside the oracle itself.

Each test checks one oracle function against something it cannot agree with
by construction: exact integer arithmetic, brute-force enumeration, library
routines (numpy / torch / scipy in fp64), closed forms, the paper's Fig. 7a
routing example, and the expected-activated-experts formula of Sec. 3.2.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from paper_2410_12247_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dyadic_bits(rng, shape, lim=8, scale=2.0 ** -4):
    ints = rng.integers(-lim, lim + 1, size=shape)
    return synth.bf16_bits(ints.astype(np.float32) * np.float32(scale)), ints


# ---------------------------------------------------------------- router ---

def test_router_logits_exact_on_dyadic_inputs():
    """x, Wr, bias on a 2^-4 grid: every product and partial sum is exact in
    fp32, so z must equal the integer dot product exactly."""
    rng = np.random.default_rng(1)
    T, H, E = 37, 200, 11
    xb, xi = _dyadic_bits(rng, (T, H))
    wi = rng.integers(-8, 9, size=(E, H))
    wr = wi.astype(np.float32) / np.float32(16)
    bi = rng.integers(-50, 51, size=E)
    bias = bi.astype(np.float32) / np.float32(256)
    z = oracle.router_logits(xb, wr, bias)
    exact = (xi.astype(np.int64) @ wi.T.astype(np.int64) + bi[None, :]) / 256.0
    assert np.array_equal(z.astype(np.float64), exact)
    z0 = oracle.router_logits(xb, wr, None)
    assert np.array_equal(z0.astype(np.float64), (xi @ wi.T) / 256.0)


def test_router_logits_close_to_fp64_dot_on_gaussian_inputs():
    """Generic values: within the standard fp32 summation bound of the fp64
    library dot product (catches a dropped term or a transposed operand)."""
    rng = np.random.default_rng(2)
    T, H, E = 16, 1024, 24
    xb = synth.bf16_bits(rng.standard_normal((T, H), dtype=np.float32))
    wr = rng.standard_normal((E, H), dtype=np.float32) * np.float32(0.02)
    z = oracle.router_logits(xb, wr).astype(np.float64)
    x = synth.bf16_to_f32(xb).astype(np.float64)
    ref = x @ wr.astype(np.float64).T
    bound = H * 2.0 ** -24 * (np.abs(x) @ np.abs(wr.astype(np.float64)).T)
    assert np.all(np.abs(z - ref) <= bound)


def test_router_accumulates_in_ascending_h_order():
    """Reading of the unstated order: one fp32 accumulator, h ascending.
    With x = [2^24, 1, -2^24] and unit weights the ascending chain gives 0
    (2^24 + 1 rounds to 2^24); descending order would give 1."""
    xb = synth.bf16_bits(np.array([[2.0 ** 24, 1.0, -(2.0 ** 24)]], np.float32))
    wr = np.ones((1, 3), np.float32)
    assert oracle.router_logits(xb, wr)[0, 0] == 0.0
    xb_rev = synth.bf16_bits(np.array([[-(2.0 ** 24), 1.0, 2.0 ** 24]], np.float32))
    assert oracle.router_logits(xb_rev, wr)[0, 0] == 1.0


def test_router_uses_fused_multiply_add():
    """acc = -round(a*b) then acc = fma(a, b, acc) leaves the exact rounding
    error of a*b, which a separate multiply and add would lose."""
    a = np.float32(1.0 + 2.0 ** -7)            # exactly representable in bf16
    b = np.float32(1.0 + 2.0 ** -20 + 2.0 ** -22)
    p = np.float32(a * b)                       # fp32-rounded product
    exact_err = float(a) * float(b) - float(p)
    assert exact_err != 0.0
    xb = synth.bf16_bits(np.array([[1.0, a]], np.float32))
    wr = np.array([[-p, b]], np.float32)
    z = oracle.router_logits(xb, wr)[0, 0]
    assert float(z) == np.float32(exact_err)


# ----------------------------------------------------------------- top-k ---

def _brute_topk(z, k):
    return [sorted(range(len(zt)), key=lambda e: (-float(zt[e]), e))[:k] for zt in z]


@pytest.mark.parametrize("E,k", [(6, 2), (8, 2), (16, 4), (160, 6), (5, 5)])
def test_topk_matches_brute_force_with_ties(E, k):
    rng = np.random.default_rng(E * 10 + k)
    T = 300
    # few distinct values -> many exact ties; include both signed zeros
    vals = np.array([-1.5, -0.0, 0.0, 0.25, 0.25, 1.0, 2.0], np.float32)
    z = vals[rng.integers(0, len(vals), size=(T, E))]
    ids, _ = oracle.topk(z, k, renorm=True)
    assert ids.tolist() == _brute_topk(z, k)


def test_topk_signed_zero_tie_goes_to_lower_index():
    z = np.array([[-0.0, 0.0, -1.0], [0.0, -0.0, -1.0]], np.float32)
    ids, _ = oracle.topk(z, 1, renorm=True)
    assert ids[:, 0].tolist() == [0, 0]


def test_renorm_weights_closed_forms():
    rng = np.random.default_rng(3)
    T, E = 500, 8
    z = (rng.standard_normal((T, E)) * 2.0).astype(np.float32)
    # k = 1 with renormalisation: the single weight is exactly 1
    _, w1 = oracle.topk(z, 1, renorm=True)
    assert np.all(w1 == 1.0)
    # k = 2: two-way softmax is the logistic of the logit difference
    ids, w2 = oracle.topk(z, 2, renorm=True)
    z0 = z[np.arange(T), ids[:, 0]].astype(np.float64)
    z1 = z[np.arange(T), ids[:, 1]].astype(np.float64)
    assert np.all(w2[:, 0] == scipy.special.expit(z0 - z1).astype(np.float32))
    assert np.all(w2[:, 1] == scipy.special.expit(z1 - z0).astype(np.float32))
    # any k: weights sum to 1 up to fp32 rounding of each term
    _, w4 = oracle.topk(z, 4, renorm=True)
    assert np.all(np.abs(w4.astype(np.float64).sum(1) - 1.0) <= 4 * 2.0 ** -24)


def test_full_softmax_weights_match_library_softmax():
    rng = np.random.default_rng(4)
    T, E, k = 200, 160, 6
    z = (rng.standard_normal((T, E)) * 1.4).astype(np.float32)
    ids, w = oracle.topk(z, k, renorm=False)
    sm = scipy.special.softmax(z.astype(np.float64), axis=1)
    ref = np.take_along_axis(sm, ids.astype(np.int64), axis=1).astype(np.float32)
    assert np.allclose(w, ref, rtol=2.0 ** -22, atol=0)
    assert np.all(w.astype(np.float64).sum(1) < 1.0)
    # E == k without renormalisation is the full softmax, in rank order
    ids5, w5 = oracle.topk(z[:, :5], 5, renorm=False)
    sm5 = scipy.special.softmax(z[:, :5].astype(np.float64), axis=1)
    assert np.allclose(w5, np.take_along_axis(sm5, ids5.astype(np.int64), 1), rtol=2.0 ** -22)


# -------------------------------------------------------------- dispatch ---

def test_fig7a_routing_example():
    d = json.load(open(os.path.join(GOLDEN, "fig7a_routing.json")))
    E, k = d["E"], d["k"]
    zl = np.array(d["logits"], np.float32)
    xb = synth.bf16_bits(zl)
    z = oracle.router_logits(xb, np.eye(E, dtype=np.float32))
    assert np.array_equal(z, zl)
    ids, _ = oracle.topk(z, k, renorm=True)
    counts, offsets, sorted_slot, _ = oracle.dispatch(ids, 0, E)
    for e_str, toks in d["expert_tokens_from_paper"].items():
        e = int(e_str)
        rows = sorted_slot[offsets[e]:offsets[e + 1]]
        assert (rows // k).tolist() == toks


@pytest.mark.parametrize("E,EL,e0,k,T", [(8, 8, 0, 2, 1000), (160, 20, 0, 6, 700),
                                         (160, 20, 40, 6, 333), (16, 16, 0, 4, 1),
                                         (4, 1, 3, 2, 50)])
def test_dispatch_invariants(E, EL, e0, k, T):
    rng = np.random.default_rng(T + E)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, e0, EL)
    loc = ids.reshape(-1) - e0
    is_loc = (loc >= 0) & (loc < EL)
    # counts are the histogram of local ids; offsets its exclusive prefix
    assert counts.tolist() == np.bincount(loc[is_loc], minlength=EL).tolist()
    assert offsets.tolist() == [0] + np.cumsum(counts).tolist()
    R = int(offsets[-1])
    assert len(sorted_slot) == R == int(is_loc.sum())
    # bijection between local slots and rows
    assert np.all(slot_row[sorted_slot] == np.arange(R))
    assert np.all(slot_row[~is_loc] == -1)
    assert np.array_equal(np.sort(sorted_slot), np.flatnonzero(is_loc))
    # stable order: expert ascending, then slot (= token) ascending
    slots = np.flatnonzero(is_loc)
    ref = slots[np.lexsort((slots, loc[is_loc]))]
    assert np.array_equal(sorted_slot, ref)


def test_expected_activated_experts_formula():
    """Sec. 3.2: with m tokens each choosing k of E experts uniformly, the
    expected number of experts with at least one token is
    (1 - (1 - k/E)^m) * E.  Checked by Monte Carlo through oracle.dispatch."""
    rng = np.random.default_rng(5)
    E, k = 64, 6
    for m in (1, 4, 16, 64):
        trials = 400
        act = []
        for _ in range(trials):
            ids = np.stack([rng.permutation(E)[:k] for _ in range(m)]).astype(np.int32)
            counts, *_ = oracle.dispatch(ids, 0, E)
            act.append(int((counts > 0).sum()))
        act = np.array(act, np.float64)
        expect = (1 - (1 - k / E) ** m) * E
        assert abs(act.mean() - expect) <= 4 * act.std() / math.sqrt(trials) + 1e-9


# ------------------------------------------------------------------- FFN ---

def _f64(bits):
    return synth.bf16_to_f32(bits).astype(np.float64)


def _swiglu_torch(x, wg, wu, wd):
    """Textbook SwiGLU FFN with torch fp64 library ops: Wd (silu(Wg x) * Wu x)."""
    x, wg, wu, wd = (torch.from_numpy(a) for a in (x, wg, wu, wd))
    a = torch.nn.functional.silu(x @ wg.T) * (x @ wu.T)
    return (a @ wd.T).numpy()


def _small_case(T, H, I, E, EL, k, renorm, seed, e0=0, n_shared=0, Is=0):
    shp = synth.custom_shape(T=T, H=H, I=I, E=E, EL=EL, k=k, renorm=renorm, e0=e0,
                             n_shared=n_shared, Is=Is, index=seed)
    return synth.make_inputs(shp)


def test_single_expert_top1_is_dense_swiglu():
    inp = _small_case(T=9, H=64, I=96, E=1, EL=1, k=1, renorm=True, seed=11)
    z, ids, w = oracle.route(inp.x, inp.w_router, None, 1, True)
    assert np.all(ids == 0) and np.all(w == 1.0)
    y = oracle.moe_tokens(inp.x, ids, w, np.arange(9), inp.w_gate, inp.w_up, inp.w_down, 0)
    ref = _swiglu_torch(_f64(inp.x), _f64(inp.w_gate[0]), _f64(inp.w_up[0]), _f64(inp.w_down[0]))
    assert np.array_equal(y, ref.astype(np.float32)) or np.allclose(y, ref, rtol=1e-6, atol=1e-7)
    # the dispatched-row path agrees with the per-token path
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, 0, 1)
    yp = oracle.expert_rows(inp.x, sorted_slot, offsets, inp.w_gate, inp.w_up, inp.w_down, 1)
    assert np.allclose(yp, ref, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("renorm,e0,EL", [(True, 0, 8), (False, 2, 3)])
def test_moe_matches_dense_masked_brute_force(renorm, e0, EL):
    """Every expert applied to every token with torch fp64, then masked by the
    routing and weighted: independent of the dispatch order and combine."""
    E, k, T, H, I = 8, 3, 21, 64, 80
    inp = _small_case(T=T, H=H, I=I, E=E, EL=EL, k=k, renorm=renorm, seed=12, e0=e0)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, k, renorm)
    y = oracle.moe_tokens(inp.x, ids, w, np.arange(T), inp.w_gate, inp.w_up, inp.w_down, e0)
    x = _f64(inp.x)
    ref = np.zeros((T, H))
    for el in range(EL):
        ye = _swiglu_torch(x, _f64(inp.w_gate[el]), _f64(inp.w_up[el]), _f64(inp.w_down[el]))
        ye = ye.astype(np.float32).astype(np.float64)    # expert rows are fp32 values
        sel = (ids == e0 + el)
        coef = (w.astype(np.float64) * sel).sum(1)
        ref += coef[:, None] * ye
    assert np.allclose(y, ref, rtol=1e-6, atol=1e-7)
    # combine from dispatched rows agrees with the per-token path
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, e0, EL)
    yp = oracle.expert_rows(inp.x, sorted_slot, offsets, inp.w_gate, inp.w_up, inp.w_down, k)
    yc = oracle.combine(yp, slot_row.reshape(T, k), w)
    assert np.allclose(yc, y, rtol=1e-6, atol=1e-7)


def test_identical_experts_with_renorm_give_the_single_ffn():
    E, k, T, H, I = 6, 2, 15, 64, 64
    inp = _small_case(T=T, H=H, I=I, E=E, EL=E, k=k, renorm=True, seed=13)
    wg = np.repeat(inp.w_gate[:1], E, 0)
    wu = np.repeat(inp.w_up[:1], E, 0)
    wd = np.repeat(inp.w_down[:1], E, 0)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, k, True)
    y = oracle.moe_tokens(inp.x, ids, w, np.arange(T), wg, wu, wd, 0)
    ref = _swiglu_torch(_f64(inp.x), _f64(wg[0]), _f64(wu[0]), _f64(wd[0]))
    assert np.allclose(y, ref, rtol=1e-5, atol=1e-6)


def test_down_weight_scaling_is_linear():
    E, k, T, H, I = 4, 2, 10, 64, 64
    inp = _small_case(T=T, H=H, I=I, E=E, EL=E, k=k, renorm=True, seed=14)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, k, True)
    y1 = oracle.moe_tokens(inp.x, ids, w, np.arange(T), inp.w_gate, inp.w_up, inp.w_down, 0)
    wd2 = synth.bf16_bits(synth.bf16_to_f32(inp.w_down) * np.float32(2.0))
    y2 = oracle.moe_tokens(inp.x, ids, w, np.arange(T), inp.w_gate, inp.w_up, wd2, 0)
    assert np.array_equal(y2, y1 * np.float32(2.0))


def test_two_shared_experts_equal_one_concatenated_expert():
    T, H, Is = 7, 64, 48
    inp = _small_case(T=T, H=H, I=32, E=4, EL=1, k=1, renorm=False, seed=15, e0=3,
                      n_shared=2, Is=Is)
    ids = np.zeros((T, 1), np.int32)          # expert 0 is not local: shared only
    w = np.ones((T, 1), np.float32)
    y = oracle.moe_tokens(inp.x, ids, w, np.arange(T), inp.w_gate, inp.w_up, inp.w_down, 3,
                          2, inp.shared_gate, inp.shared_up, inp.shared_down)
    ref = _swiglu_torch(_f64(inp.x), _f64(inp.shared_gate), _f64(inp.shared_up),
                        _f64(inp.shared_down))
    assert np.allclose(y, ref, rtol=1e-6, atol=1e-7)


def test_token_permutation_permutes_outputs():
    E, k, T, H, I = 8, 2, 12, 64, 64
    inp = _small_case(T=T, H=H, I=I, E=E, EL=E, k=k, renorm=True, seed=16)
    _, ids, w = oracle.route(inp.x, inp.w_router, None, k, True)
    y = oracle.moe_tokens(inp.x, ids, w, np.arange(T), inp.w_gate, inp.w_up, inp.w_down, 0)
    perm = np.random.default_rng(0).permutation(T)
    xp = inp.x[perm]
    _, idsp, wp = oracle.route(xp, inp.w_router, None, k, True)
    yp = oracle.moe_tokens(xp, idsp, wp, np.arange(T), inp.w_gate, inp.w_up, inp.w_down, 0)
    assert np.array_equal(yp, y[perm])


def test_zipf_bias_skews_popularity():
    """The sweep's bias makes expert popularity fall with rank (checked on the
    oracle's routing of a sample of the workload)."""
    shp = synth.SHAPES["zipf"].with_tokens(1024)
    inp = synth.make_inputs(shp, router_only=True)
    _, ids, _ = oracle.route(inp.x, inp.w_router, inp.bias, 1, False)
    cnt = np.bincount(ids[:, 0], minlength=160)
    per = 8
    rank = per * (np.arange(160) % 20) + np.arange(160) // 20 + 1
    top = cnt[np.argsort(rank)]
    assert top[:8].sum() > 10 * max(1, top[-80:].sum() // 10)


# ----------------------------------------------- row list and combine init ---

def test_expert_row_list_matches_library_swiglu_per_pair():
    """oracle.expert_row_list on an arbitrary list of (token, local expert)
    pairs (repeats, every expert, tokens out of order) against the SwiGLU of
    that token through that expert with torch fp64 library ops, rounded to
    fp32 once.  A wrong token index, a wrong expert stack or a transposed
    down matrix changes whole rows."""
    E, T, H, I = 5, 17, 64, 96
    inp = _small_case(T=T, H=H, I=I, E=E, EL=E, k=2, renorm=True, seed=17)
    rng = np.random.default_rng(17)
    tok = np.concatenate([rng.integers(0, T, size=30), [T - 1, 0, 0]]).astype(np.int64)
    el = np.concatenate([rng.integers(0, E, size=30), [E - 1, 0, E - 1]]).astype(np.int32)
    y = oracle.expert_row_list(inp.x, tok, el, inp.w_gate, inp.w_up, inp.w_down)
    x = _f64(inp.x)
    for n in range(len(tok)):
        e = int(el[n])
        ref = _swiglu_torch(x[tok[n]:tok[n] + 1], _f64(inp.w_gate[e]), _f64(inp.w_up[e]),
                            _f64(inp.w_down[e]))[0]
        assert np.allclose(y[n], ref, rtol=1e-6, atol=1e-7), (n, int(tok[n]), e)
    # the list path and the dispatched-row path give the same bits for the
    # same (token, expert) rows
    _, ids, _ = oracle.route(inp.x, inp.w_router, None, 2, True)
    counts, offsets, sorted_slot, _ = oracle.dispatch(ids, 0, E)
    yp = oracle.expert_rows(inp.x, sorted_slot, offsets, inp.w_gate, inp.w_up, inp.w_down, 2)
    yl = oracle.expert_row_list(inp.x, sorted_slot // 2, np.repeat(np.arange(E), counts),
                                inp.w_gate, inp.w_up, inp.w_down)
    assert np.array_equal(yl, yp)


def test_combine_with_initial_value_is_a_sparse_matrix_product():
    """oracle.combine(y_perm, slot_row, w, y_init): y = y_init + A y_perm,
    where A [T, R] holds w[t, j] at column slot_row[t, j] (no entry for a
    non-local slot), computed here as one torch fp64 matrix product.  Also
    the special cases that leave y_init untouched (zero weights, zero rows)."""
    E, EL, e0, k, T, H = 8, 5, 2, 3, 40, 24
    rng = np.random.default_rng(18)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts, offsets, sorted_slot, slot_row = oracle.dispatch(ids, e0, EL)
    R = int(offsets[-1])
    assert 0 < R < T * k  # some slots are not local
    y_perm = rng.standard_normal((R, H)).astype(np.float32)
    w = rng.random((T, k)).astype(np.float32)
    y_init = rng.standard_normal((T, H)).astype(np.float32)
    sr = slot_row.reshape(T, k)
    y = oracle.combine(y_perm, sr, w, y_init)
    A = np.zeros((T, R))
    for t in range(T):
        for j in range(k):
            if sr[t, j] >= 0:
                A[t, sr[t, j]] += float(w[t, j])
    ref = (torch.from_numpy(y_init.astype(np.float64)) +
           torch.from_numpy(A) @ torch.from_numpy(y_perm.astype(np.float64))).numpy()
    assert np.allclose(y, ref, rtol=2.0 ** -23, atol=1e-30)
    # with an initial value the result differs from the plain combine by it
    y0 = oracle.combine(y_perm, sr, w)
    assert np.allclose(y.astype(np.float64) - y0, y_init, rtol=1e-6, atol=1e-6)
    # nothing to add: y_init comes back bit for bit
    assert np.array_equal(oracle.combine(y_perm, sr, np.zeros_like(w), y_init), y_init)
    assert np.array_equal(oracle.combine(np.zeros_like(y_perm), sr, w, y_init), y_init)
    # no local slot at all: y_init again, and zeros without it
    none = np.full_like(sr, -1)
    assert np.array_equal(oracle.combine(y_perm, none, w, y_init), y_init)
    assert np.all(oracle.combine(y_perm, none, w) == 0.0)
