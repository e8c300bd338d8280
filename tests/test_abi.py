"""CPU checks of the C-ABI library: it loads, exports what include/moe.h
declares, sizes workspaces on the host, and rejects bad arguments before any
GPU work (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2410_12247_amd import moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    L = moe.lib()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), f"libmoe.so does not export {n}"
    assert set(names) == set(moe.EXPORTS)


def test_status_strings():
    L = moe.lib()
    assert L.moe_status_string(0) == b"ok"
    assert L.moe_status_string(3) == b"workspace too small"


def test_workspace_bytes_host_only():
    d = moe.dims(16384, 4096, 3584, 8, 2)
    fw = moe.workspace_bytes(d, moe.opts())
    pm = moe.workspace_bytes(d)
    assert 0 < pm < fw
    R = 16384 * 2
    # forward workspace holds act (bf16) and y_perm (fp32) rows
    assert fw >= R * (3584 * 2 + 4096 * 4)
    assert moe.workspace_bytes(moe.dims(16, 100, 64, 8, 2), moe.opts()) == 0  # H % 64


BAD = [
    (dict(tokens=-1), 1),
    (dict(hidden=100), 1),
    (dict(inter=0), 1),
    (dict(experts=300), 2),
    (dict(top_k=9), 2),
    (dict(top_k=0), 1),
    (dict(top_k=5, experts=4), 1),
    (dict(local_begin=6, local_count=4), 1),
    (dict(local_count=0), 1),
    (dict(renormalize=2), 1),
    (dict(shared_inter=96), 1),
    (dict(tokens=1 << 29, top_k=8), 1),
]


@pytest.mark.parametrize("change,status", BAD)
def test_invalid_dims_rejected_before_any_gpu_work(change, status):
    base = dict(tokens=64, hidden=256, inter=128, experts=8, top_k=2, local_begin=0,
                local_count=8, renormalize=1, shared_inter=0)
    base.update(change)
    d = moe.Dims(**base)
    fake = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    L = moe.lib()
    st = L.moe_route(ctypes.byref(d), fake, fake, None, fake, fake, None)
    assert st == status, L.moe_last_error()
    assert L.moe_last_error()
    st = L.moe_ffn_forward(ctypes.byref(d), None, fake, fake, None, fake, fake, fake, None,
                           None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == status


def test_invalid_options_and_buffers_rejected():
    L = moe.lib()
    d = moe.dims(64, 256, 128, 8, 2)
    fake = ctypes.c_void_p(16)
    for o in (moe.opts(pipeline_n=3), moe.opts(pipeline_n=-1), moe.opts(gemm_mode=7),
              moe.opts(gemm_cu_budget=-1), moe.opts(side_cus=-1),
              moe.opts(group_tile_rows=64), moe.opts(group_tile_rows=-128),
              moe.opts(dense_tile_rows=100),
              moe.opts(pipeline_n=0, chunk_mode=moe.CHUNK_TOKENS)):
        st = L.moe_ffn_forward(ctypes.byref(d), ctypes.byref(o), fake, fake, None, fake, fake,
                               fake, None, None, None, fake, None, None, None, fake, 1 << 40,
                               None)
        assert st == 1, L.moe_last_error()
    # token-range stages: PN need not divide EL, PN * EL must fit 256 buckets
    tok = moe.CHUNK_TOKENS
    assert L.moe_workspace_bytes(ctypes.byref(d), ctypes.byref(moe.opts(pipeline_n=3,
                                                                        chunk_mode=tok))) > 0
    assert L.moe_workspace_bytes(ctypes.byref(d), ctypes.byref(moe.opts(pipeline_n=3))) == 0
    assert L.moe_workspace_bytes(ctypes.byref(d), ctypes.byref(moe.opts(chunk_mode=2))) == 0
    assert L.moe_workspace_bytes(ctypes.byref(d), ctypes.byref(moe.opts(pipeline_n=33,
                                                                        chunk_mode=tok))) == 0
    o = moe.opts(pipeline_n=33, chunk_mode=tok)  # 33 * 8 buckets > 256
    st = L.moe_ffn_forward(ctypes.byref(d), ctypes.byref(o), fake, fake, None, fake, fake, fake,
                           None, None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == 2, L.moe_last_error()
    o = moe.opts(chunk_mode=2)
    st = L.moe_ffn_forward(ctypes.byref(d), ctypes.byref(o), fake, fake, None, fake, fake, fake,
                           None, None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == 1
    o = moe.opts()
    o.flags = 16  # unknown flag
    st = L.moe_ffn_forward(ctypes.byref(d), ctypes.byref(o), fake, fake, None, fake, fake, fake,
                           None, None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == 1
    assert moe.opts(timing="gemm").flags == 2 and moe.opts(timing=True).flags == 1
    assert moe.opts(exact_order=True).flags == 4
    assert moe.opts(timing="gemm", exact_order=True).flags == 6
    o = moe.opts(side_cus=250)  # at most 248 CUs for the side streams
    st = L.moe_ffn_forward(ctypes.byref(d), ctypes.byref(o), fake, fake, None, fake, fake, fake,
                           None, None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == 1
    # workspace too small
    st = L.moe_ffn_forward(ctypes.byref(d), None, fake, fake, None, fake, fake, fake, None,
                           None, None, fake, None, None, None, fake, 10, None)
    assert st == 3
    # NULL required tensors
    st = L.moe_route(ctypes.byref(d), None, fake, None, fake, fake, None)
    assert st == 1
    # shared experts declared but not given
    ds = moe.dims(64, 256, 128, 8, 2, shared_inter=128)
    st = L.moe_ffn_forward(ctypes.byref(ds), None, fake, fake, None, fake, fake, fake, None,
                           None, None, fake, None, None, None, fake, 1 << 40, None)
    assert st == 1
    # expert ranges
    assert L.moe_gather(ctypes.byref(d), 6, 3, fake, fake, fake, fake, None) == 1
    assert L.moe_combine(ctypes.byref(d), 0, 9, fake, fake, fake, fake, fake, 0, None) == 1
    assert L.moe_combine(ctypes.byref(d), 0, 8, fake, fake, fake, fake, fake, 2, None) == 1
    assert L.moe_ffn_group(ctypes.byref(d), -1, 2, fake, fake, fake, fake, fake, fake, fake, 0,
                           None) == 1
    assert L.moe_ffn_dense(10, 100, 64, fake, fake, fake, fake, fake, fake, None) == 1
    assert L.moe_last_timing(None) == 1


def test_zero_token_calls_are_noops_on_the_host():
    L = moe.lib()
    d = moe.dims(0, 256, 128, 8, 2)
    assert L.moe_route(ctypes.byref(d), None, None, None, None, None, None) == 0
    assert L.moe_permute(ctypes.byref(d), None, None, None, None, None, None, None, None, 0,
                         None) == 0
    assert L.moe_ffn_dense(0, 256, 128, None, None, None, None, None, None, None) == 0


def test_pipeline_n_chooser_model():
    """moe_choose_pipeline_n against the properties of the paper's pipeline
    model (Sec. 5.2): gain C(1 - 1/N) - (kN + b), best near sqrt(C/k),
    bounded by C - b - 2 sqrt(kC), only divisors of the local expert count,
    no pipeline unless it gains."""
    ch = moe.choose_pipeline_n
    # sqrt(C/k) = 4 divides 20: the closed form, with the bound reached
    pn, g = ch(16.0, 1.0, 0.0, 20)
    assert pn == 4 and g == pytest.approx(16 - 2 * (16 * 1.0) ** 0.5)
    # sqrt(9) = 3 does not divide 20: the better neighbour among 2, 4, 5
    # (gains 2.5, 2.75, 2.2)
    pn, g = ch(9.0, 1.0, 0.0, 20)
    assert pn == 4 and g == pytest.approx(2.75)
    # no per-stage overhead: the more stages, the better
    assert ch(5.0, 0.0, 0.0, 20)[0] == 20
    assert ch(5.0, 0.0, 0.0, 7)[0] == 7
    # a fixed overhead above every gain keeps one stage
    assert ch(16.0, 1.0, 10.0, 20) == (1, 0.0)
    # nothing to hide, one expert, or a prime count with a steep overhead
    assert ch(0.0, 0.1, 0.0, 8) == (1, 0.0)
    assert ch(16.0, 0.1, 0.0, 1) == (1, 0.0)
    assert ch(1.0, 1.0, 0.0, 7) == (1, 0.0)
    # the gain never exceeds the paper's bound and is the best divisor's
    for C, k, b, EL in [(3.0, 0.05, 0.1, 20), (0.14, 0.1, 0.0, 8), (2.0, 0.3, -0.2, 16),
                        (40.0, 0.01, 1.0, 160)]:
        pn, g = ch(C, k, b, EL)
        assert EL % pn == 0
        if pn > 1:
            assert g <= C - b - 2 * (k * C) ** 0.5 + 1e-12
        gains = {n: C - b - (C / n + k * n) for n in range(2, EL + 1) if EL % n == 0}
        assert g == pytest.approx(max([0.0] + list(gains.values())))
    # invalid arguments
    for args in [(float("nan"), 1.0, 0.0, 8), (-1.0, 1.0, 0.0, 8), (1.0, -1.0, 0.0, 8),
                 (1.0, 1.0, float("inf"), 8), (1.0, 1.0, 0.0, 0), (1.0, 1.0, 0.0, 257)]:
        with pytest.raises(moe.MoEError) as e:
            ch(*args)
        assert e.value.status == 1


def test_workspace_holds_only_what_the_options_use():
    """Gathered rows only when the GEMM cannot read token rows straight from x
    (T * H * 2 bytes reach 2^32), K-split partials only when a GEMM may cut
    tiles."""
    d = moe.dims(16384, 4096, 3584, 8, 2)
    R = 16384 * 2
    auto = moe.workspace_bytes(d, moe.opts())
    group = moe.workspace_bytes(d, moe.opts(gemm_mode=moe.GEMM_GROUP))
    exact = moe.workspace_bytes(d, moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=True))
    assert auto == group
    assert group - exact >= 256 * 256 * 320 * 4              # 256 partial tiles of fp32
    assert exact >= R * (3584 * 2 + 4096 * 4)                # act + y_perm
    assert exact < R * (3584 * 2 + 4096 * 4) + R * 4096      # no x_perm [R][H] bf16
    big = moe.dims(600000, 4096, 64, 8, 1)                   # 4.9 GB of x
    nb = moe.workspace_bytes(big, moe.opts(exact_order=True))
    assert nb >= 600000 * 4096 * (2 + 4)                     # x_perm + y_perm


def test_noalloc_forward_rejects_on_the_host():
    """moe_ffn_forward_noalloc refuses, before touching the GPU, what it
    cannot do without allocating: options that need row counts on the host,
    timing, and workloads whose workspace exceeds its 256 MiB buffer."""
    L = moe.lib()
    fake = ctypes.c_void_p(16)  # never dereferenced: validation fails first

    def call(d, o):
        return L.moe_ffn_forward_noalloc(ctypes.byref(d), ctypes.byref(o) if o else None, fake,
                                         fake, None, fake, fake, fake, None, None, None, fake,
                                         None, None, None, None)

    small = moe.dims(64, 256, 128, 8, 2)
    for o in (moe.opts(pipeline_n=2), moe.opts(gemm_mode=moe.GEMM_DENSE),
              moe.opts(dense_min_rows=16), moe.opts(timing=True), moe.opts(timing="gemm")):
        assert call(small, o) == 2, L.moe_last_error()
    assert call(small, moe.opts(pipeline_n=3)) == 1          # invalid as in moe_ffn_forward
    big = moe.dims(16384, 4096, 3584, 8, 2)                   # the Mixtral-shaped shard
    assert moe.workspace_bytes(big, moe.opts()) > 256 << 20
    assert call(big, moe.opts()) == 2
    assert b"256" in L.moe_last_error() or b"268435456" in L.moe_last_error()
    assert L.moe_ffn_forward_noalloc(ctypes.byref(small), None, None, fake, None, fake, fake,
                                     fake, None, None, None, fake, None, None, None, None) == 1
    zero = moe.dims(0, 256, 128, 8, 2)
    assert call(zero, moe.opts()) == 0


def test_workspace_guards_layout():
    """Guard gaps (moe_workspace_guards): one after every region, in order,
    inside the workspace, the last one ending it; regions never overlap a
    gap; invalid dims are refused."""
    L = moe.lib()
    G = moe.WS_GUARD_BYTES
    for d, o in [(moe.dims(16384, 4096, 3584, 8, 2), moe.opts()),
                 (moe.dims(16384, 5120, 1536, 160, 6, 0, 20, False, 3072), moe.opts()),
                 (moe.dims(300, 256, 128, 8, 2), moe.opts(exact_order=True)),
                 (moe.dims(1500, 192, 320, 4, 2), moe.opts(pipeline_n=2,
                                                           chunk_mode=moe.CHUNK_TOKENS)),
                 (moe.dims(777, 512, 384, 16, 4, 3, 5), None)]:
        guards = moe.workspace_guards(d, o)
        total = moe.workspace_bytes(d, o)
        assert len(guards) >= (3 if o is None else 15)
        assert guards[0] > 0
        assert all(b >= a + G for a, b in zip(guards, guards[1:]))
        assert guards[-1] + G == total
        assert all(g % 256 == 0 for g in guards)
    # capacity smaller than the count: the first offsets, and the full count
    d = moe.dims(16384, 4096, 3584, 8, 2)
    buf = (ctypes.c_int64 * 2)()
    n = L.moe_workspace_guards(ctypes.byref(d), None, buf, 2)
    assert n == 3 and list(buf) == moe.workspace_guards(d)[:2]
    with pytest.raises(moe.MoEError):
        moe.workspace_guards(moe.dims(16, 100, 64, 8, 2))  # hidden not a multiple of 64
    assert L.moe_workspace_guards(ctypes.byref(d), None, None, 4) == -1


def test_gemm_plan_model():
    """AUTO's GroupGemm / DenseGemm plan for one stage (moe_gemm_plan, host
    only): forced modes, per-expert tile heights among the built ones, an
    empty expert, the fixed threshold, and the model's choices on the shapes
    whose measurements set it."""
    L = moe.lib()
    d = moe.dims(16384, 5120, 1536, 160, 6, 0, 20, False)
    plan = moe.gemm_plan
    # one expert of 4096 rows, DeepSeekV2 expert shape: 320-row tiles leave
    # 156 of 256 workgroups busy for gate/up; a dense launch picks its height
    dense, tiles, gus, dus = plan(d, moe.opts(), [4096])
    assert tiles[0] in (128, 192, 256, 320)
    assert dense == (dus < gus)
    # forced kinds
    assert plan(d, moe.opts(gemm_mode=moe.GEMM_GROUP), [4096])[0] is False
    # a grouped launch's tile height: never taller than the smallest that
    # holds its largest expert (320 above 256 rows); among those, the one
    # the model prices lowest when that is at least 5% below the holding
    # height's price.  One expert: the dense pick is the model's cheapest
    # height, so the grouped price lies within 5% above it
    grouped = moe.opts(gemm_mode=moe.GEMM_GROUP)
    assert plan(d, grouped, [1, 0])[1] == [128, 128]
    assert plan(d, grouped, [128, 3])[1] == [128, 128]
    for rows, hold in (([129], 192), ([200, 7], 256), ([100, 257], 320), ([40] * 20, 128),
                       ([300] * 20, 320), ([4096], 320), ([8192], 320), ([3200], 320)):
        for exact in (False, True):
            o = moe.opts(gemm_mode=moe.GEMM_GROUP, exact_order=exact)
            _, tiles, gus, dus = plan(d, o, rows)
            assert len(set(tiles)) == 1 and tiles[0] in (128, 192, 256, 320)
            assert tiles[0] <= hold
            if len(rows) == 1:
                assert dus <= gus * (1 + 1e-9) and gus <= dus / 0.95 * (1 + 1e-9)
    # a few rows per expert: the 128-row tile (every height holds them in
    # one tile, and it streams the weights fastest); 300 rows each: one
    # 320-row tile per expert against three of 128
    assert plan(d, grouped, [100, 257])[1] == [128, 128]
    assert plan(d, grouped, [300] * 20)[1] == [320] * 20
    # a forced grouped height
    for bm in (128, 192, 256, 320):
        o = moe.opts(gemm_mode=moe.GEMM_GROUP, group_tile_rows=bm)
        assert plan(d, o, [40, 0, 700])[1] == [bm] * 3
    dense, tiles, _, _ = plan(d, moe.opts(gemm_mode=moe.GEMM_DENSE), [4096, 0, 17])
    assert dense and tiles[1] == 0 and tiles[0] > 0 and tiles[2] > 0
    dense, tiles, _, _ = plan(d, moe.opts(gemm_mode=moe.GEMM_DENSE, dense_tile_rows=192),
                              [4096, 5])
    assert tiles == [192, 192]
    # many experts per stage: always one grouped launch under AUTO
    assert plan(d, moe.opts(), [600] * 20)[0] is False
    # the fixed threshold of Sec. 3.2: dense iff every expert reaches m
    assert plan(d, moe.opts(dense_min_rows=1000), [1200, 3000])[0] is True
    assert plan(d, moe.opts(dense_min_rows=1000), [999, 3000])[0] is False
    # predicted times grow with the load
    g1, d1 = plan(d, moe.opts(), [1024])[2:]
    g2, d2 = plan(d, moe.opts(), [8192])[2:]
    assert 0 < g1 < g2 and 0 < d1 < d2
    # invalid arguments
    with pytest.raises(moe.MoEError):
        plan(d, moe.opts(), [-1])
    with pytest.raises(moe.MoEError):
        plan(d, moe.opts(dense_tile_rows=100), [10])
    r = (ctypes.c_int32 * 1)(5)
    out = ctypes.c_int32()
    assert L.moe_gemm_plan(ctypes.byref(d), None, 0, r, ctypes.byref(out), None, None,
                           None) == 1
    assert L.moe_gemm_plan(ctypes.byref(d), None, 1, None, ctypes.byref(out), None, None,
                           None) == 1


def test_pipeline_enable_condition():
    """moe_pipeline_plan evaluates the paper's enable condition (Sec. 5.2
    item 4: N S(m/N) / S(m) <= 1 + eps0 and N G(m/N, E/N) / G(m, E) <=
    1 + eps1, eps0 = 0.32 and eps1 = 0.03 as in its DeepSeekV2 test) and
    gain L(N) - R(N) (item 5); pipeline_n = 0 picks the enabled divisor
    with the largest positive gain.  Checked against the definitions on
    the terms the call reports."""
    plan = moe.pipeline_plan
    d = moe.dims(16384, 5120, 1536, 160, 6, 0, 20, False)
    rows = [600 + 37 * e for e in range(20)]
    one = plan(d, moe.opts(), rows, 1)
    assert one["eps0"] == 0 and one["eps1"] == 0 and one["gain_us"] == 0 and one["enabled"]
    assert one["t_comm_us"] == one["t_comm_n_us"] and one["t_comp_us"] == one["t_comp_n_us"]
    for n in (2, 4, 5, 10, 20):
        ev = plan(d, moe.opts(), rows, n)
        assert ev["pipeline_n"] == n
        assert ev["t_comm_us"] == one["t_comm_us"] and ev["t_comp_us"] == one["t_comp_us"]
        assert ev["eps0"] == pytest.approx(ev["t_comm_n_us"] / ev["t_comm_us"] - 1)
        assert ev["eps1"] == pytest.approx(ev["t_comp_n_us"] / ev["t_comp_us"] - 1)
        C = min(ev["t_comm_us"], ev["t_comp_us"])
        R = (ev["t_comp_n_us"] - ev["t_comp_us"]) + (ev["t_comm_n_us"] - ev["t_comm_us"])
        assert ev["overlap_frac"] == 0.0   # the full grid leaves no CU to the combine
        assert C * (n - 1) / n * ev["overlap_frac"] - R - ev["gain_us"] == \
            pytest.approx(20.0 * (n - 1))
        # a CU budget of 192 of 256 leaves a quarter of the CUs to the side streams
        eb = plan(d, moe.opts(gemm_cu_budget=192), rows, n)
        assert eb["overlap_frac"] == 0.25
        Cb = min(eb["t_comm_us"], eb["t_comp_us"])
        Rb = (eb["t_comp_n_us"] - eb["t_comp_us"]) + (eb["t_comm_n_us"] - eb["t_comm_us"])
        assert Cb * (n - 1) / n * 0.25 - Rb - eb["gain_us"] == pytest.approx(20.0 * (n - 1))
        assert plan(d, moe.opts(side_cus=64), rows, n)["overlap_frac"] == 0.25
        assert ev["enabled"] == int(ev["eps0"] <= 0.32 and ev["eps1"] <= 0.03)
        # cutting never makes the stages' work smaller than the whole
        assert ev["eps0"] > 0 and ev["eps1"] > -1e-9
    # the library's choice: the best enabled divisor whose gain is at least
    # 5% of the unsplit GEMM time, else 1
    best = plan(d, moe.opts(), rows, 0)
    cands = [plan(d, moe.opts(), rows, n) for n in (2, 4, 5, 10, 20)]
    ok = [c for c in cands if c["enabled"] and c["gain_us"] > 0 and
          c["gain_us"] >= 0.05 * c["t_comp_us"]]
    assert best["pipeline_n"] == (max(ok, key=lambda c: c["gain_us"])["pipeline_n"] if ok else 1)
    # one GPU: each stage's combine re-reads and re-writes all of y, so the
    # stand-in communication does not split (eps0 far above 0.32) and no PN
    # is enabled on the Mixtral- or DeepSeekV2-shaped loads
    mix = moe.dims(16384, 4096, 3584, 8, 2)
    assert plan(mix, moe.opts(), [4096] * 8, 2)["eps0"] > 0.32
    assert plan(mix, moe.opts(), [4096] * 8, 0)["pipeline_n"] == 1
    assert plan(d, moe.opts(), rows, 0)["pipeline_n"] == 1
    # PN must divide the local experts; expert stages only
    with pytest.raises(moe.MoEError):
        plan(d, moe.opts(), rows, 3)
    with pytest.raises(moe.MoEError):
        plan(d, moe.opts(chunk_mode=moe.CHUNK_TOKENS, pipeline_n=2), rows, 2)
    with pytest.raises(moe.MoEError):
        plan(d, moe.opts(), [-1] + rows[1:], 2)


def test_binding_structs_match_the_header():
    """The ctypes mirrors of moe_opts, moe_timing and moe_pipeline_eval have
    the header's sizes and field order (a mismatch would shift every field
    after it), and convert to dicts."""
    assert ctypes.sizeof(moe.Opts) == 9 * 4
    assert ctypes.sizeof(moe.Timing) == 8 * 4 + 6 * 4
    assert ctypes.sizeof(moe.PipelineEval) == 8 * 8 + 2 * 4
    assert [f for f, _ in moe.Opts._fields_][-3:] == ["dense_tile_rows", "side_cus",
                                                      "group_tile_rows"]
    assert moe.Timing().as_dict()["pipeline_n"] == 0
    assert set(moe.PipelineEval().as_dict()) >= {"eps0", "eps1", "gain_us", "enabled"}
