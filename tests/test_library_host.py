"""CPU tests of the library: it loads, exports every declared symbol, and its
host-side algorithms (grouping, deployment, tables, look-ahead) agree with the
oracle; argument validation fails cleanly without touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as wl
from oracle import placement, similarity, tables
from paper_2607_17154_amd import ordermoe as om

from ._pipeline import build_case, library_tables

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "ordermoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ordermoe_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 12
    L = om.lib()
    for n in names:
        assert hasattr(L, n), n
        assert n in om.EXPORTS, n


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4"])
def test_grouping_matches_oracle(name):
    cfg = wl.LAYER_CONFIGS[name]
    cfg = cfg.with_(T_cal=min(cfg.T_cal, 4096))
    W = wl.router(cfg)
    m = similarity.build(wl.calibration(cfg), W, cfg.k, cfg.theta, cfg.alpha_f)
    sim32 = m["sim"].astype(np.float32)
    g_or, c_or = similarity.group_experts(sim32.astype(np.float64), m["counts"], np.float32(cfg.theta))
    _, _, I_or = similarity.importance(sim32.astype(np.float64), m["counts"], g_or, cfg.alpha_f)
    g, c, I = om.ordermoe_group_experts(sim32, m["counts"], cfg.theta, cfg.alpha_f)
    assert list(g) == list(g_or) and c == c_or
    np.testing.assert_array_equal(I, I_or)
    assert len(c) == cfg.clusters


GOLDEN = os.path.join(ROOT, "tests", "golden")


@pytest.mark.parametrize("case", sorted(f for f in os.listdir(GOLDEN) if f.startswith("placement_")))
def test_place_matches_hand_traces(case):
    import json
    g = json.load(open(os.path.join(GOLDEN, case)))
    x, used = om.ordermoe_place([np.array(v) for v in g["group_of"]],
                                [np.array(v, float) for v in g["importance"]],
                                [np.array(v, float) for v in g["p"]], g["C"], g["pi"],
                                g["lambda1"], int(g["redundancy"]))
    for l, want in enumerate(g["servers_of_expert"]):
        got = [sorted(int(m) for m in np.nonzero(x[l][:, j])[0]) for j in range(len(want))]
        assert got == want
    np.testing.assert_allclose(used, g["used"])


def test_place_matches_oracle_random():
    rng = np.random.default_rng(11)
    for trial in range(25):
        N = int(rng.integers(1, 4))
        M = int(rng.integers(2, 7))
        E = [int(rng.integers(3, 14)) for _ in range(N)]
        group_of = [rng.integers(0, 4, size=e).astype(np.int32) for e in E]
        imp = [rng.random(e) for e in E]
        p = [rng.integers(1, 3, size=e).astype(float) for e in E]
        need = sum(v.sum() for v in p)
        C = rng.integers(2, 8, size=M).astype(float)
        while C.sum() < need * 1.2:
            C[int(rng.integers(0, M))] += 2
        pi = rng.random(M)
        red = int(rng.integers(0, 3))
        x_or, b_or = placement.place(group_of, imp, p, C, pi, 0.5, red)
        x_lib, b_lib = om.ordermoe_place(group_of, imp, p, C, pi, 0.5, red)
        for l in range(N):
            np.testing.assert_array_equal(x_lib[l], x_or[l])
        np.testing.assert_array_equal(b_lib, b_or)


def test_place_random_matches_oracle():
    rng = np.random.default_rng(12)
    for trial in range(25):
        N, M = int(rng.integers(1, 4)), int(rng.integers(2, 9))
        p = [rng.integers(1, 4, size=int(rng.integers(3, 20))).astype(float) for _ in range(N)]
        need = sum(v.sum() for v in p)
        C = rng.integers(2, 9, size=M).astype(float)
        while C.sum() < need * float(rng.uniform(1.0, 2.5)):
            C[int(rng.integers(0, M))] += 1
        seed = int(rng.integers(0, 2 ** 63)) * 2 + 1
        red = int(rng.integers(0, 2))
        x_or, b_or = placement.place_random(p, C, seed, bool(red))
        x_lib, b_lib = om.ordermoe_place_random(p, C, seed, red)
        for l in range(N):
            np.testing.assert_array_equal(x_lib[l], x_or[l])
        np.testing.assert_array_equal(b_lib, b_or)


def test_place_random_rejects_bad_input():
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_place_random([np.ones(3)], [1.0, 1.0], 0)
    assert ei.value.code == om.ECAPACITY
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_place_random([np.array([1.0, 0.0])], [4.0, 4.0], 0)
    assert ei.value.code == om.EINVAL
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_place([np.array([0, 1])], [np.ones(2)], [np.ones(2)], [4.0, 4.0], [0.5, 0.5],
                          0.5, 3)
    assert ei.value.code == om.EINVAL


def test_place_capacity_error():
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_place([np.array([0, 1, 2])], [np.ones(3)], [np.ones(3)], [1.0, 1.0], [0.5, 0.5])
    assert ei.value.code == om.ECAPACITY


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4"])
def test_tables_match_oracle(name):
    case = build_case(wl.LAYER_CONFIGS[name].with_(T_cal=2048), T=8)
    tabs = library_tables(case)
    np.testing.assert_array_equal(tabs["S"], case.S)       # bit-exact fp32
    cfg = case.cfg
    for r in range(cfg.E):
        subs = tables.substitutes(case.sim32, case.model["group_of"], cfg.theta, r)
        subs = sorted(subs, key=lambda kq: (kq[1], kq[0]))
        n = int(tabs["t1_n"][r])
        assert n == len(subs)
        assert [int(v) for v in tabs["t1_k"][r, :n]] == [k for k, _ in subs]
        assert [np.float32(v) for v in tabs["t1_q"][r, :n]] == [q for _, q in subs]
        mask = sum(1 << m for m in range(cfg.M) if case.x_dep[m, r])
        assert int(tabs["srvmask"][r]) == mask


def test_tables_reject_undeployed_expert():
    case = build_case(wl.C1.with_(T_cal=512), T=4)
    x = case.x_dep.copy()
    x[:, 3] = 0
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_build_tables(case.sim32, case.model["group_of"], 0.7, x, case.net.B,
                                 case.net.tau, case.net.F, case.z_bits, case.c, case.dref, 0.5)
    assert ei.value.code == om.EINVAL and "eq 2" in str(ei.value)
    with pytest.raises(om.OrderMoEError):
        om.ordermoe_build_tables(case.sim32, case.model["group_of"], 0.7, case.x_dep, case.net.B,
                                 case.net.tau, case.net.F, case.z_bits, case.c, case.dref, 0.5,
                                 gmax=0)


def _lookahead_inputs(rng, N, M, E):
    x = (rng.random((N, M, E)) < 0.4).astype(np.uint8)
    for l in range(N):
        for j in range(E):
            if not x[l, :, j].any():
                x[l, int(rng.integers(0, M)), j] = 1
    sims = []
    for l in range(N):
        s = rng.uniform(0.5, 1.0, size=(E, E)).astype(np.float32)
        s = np.triu(s, 1) + np.triu(s, 1).T + np.eye(E, dtype=np.float32)
        sims.append(s)
    groups = [rng.integers(0, 2, size=E).astype(np.int32) for _ in range(N)]
    top1 = [rng.integers(0, E, size=60) for _ in range(N)]
    P = tables.transitions(top1, [E] * N)
    B = rng.uniform(1e9, 1e10, size=(M, M))
    tau = rng.uniform(2e-4, 2e-2, size=(M, M))
    F = rng.uniform(2e13, 1.1e14, size=M)
    c = [np.full(E, 6.0 * 64 * 128) for _ in range(N)]
    theta = np.float32([tables.theta_layer(l + 1, N) for l in range(N)])
    z = np.full(N, 8.0 * 64 * 2)
    dref = np.array([tables.d_ref(c[l], F) for l in range(N)])
    return x, sims, groups, P, B, tau, F, c, theta, z, dref


@pytest.mark.parametrize("H,pin", [(1, 1), (2, 1), (3, 1), (3, 0)])
def test_lookahead_matches_oracle(H, pin):
    rng = np.random.default_rng(H * 10 + pin)
    N, M, E = 4, 3, 6
    x, sims, groups, P, B, tau, F, c, theta, z, dref = _lookahead_inputs(rng, N, M, E)
    Qbar = 0.25
    phi_or = tables.lookahead(H, P, list(x), sims, groups, list(theta), list(z), B, tau, c, F,
                              list(dref), 0.5, 0.5, Qbar, pin_local_exact=pin)
    phi_lib = om.ordermoe_build_lookahead(H, np.stack(P), x, np.stack(sims), np.stack(groups),
                                          theta, z, np.stack(c), dref, B, tau, F, 0.5, 0.5, Qbar,
                                          pin, 1)
    for l in range(N):
        np.testing.assert_allclose(phi_lib[l], phi_or[l], rtol=1e-12, atol=0)
    if H == 1:
        assert np.all(phi_lib == 0)


def test_device_entry_points_validate_before_launch():
    # invalid arguments are rejected on the host; nothing touches a GPU here
    lay = om.Layer(dtype=om.BF16, d=100, E=8, k=2, M=2, gmax=1)
    out = om.RouteOut()
    rc = om.lib().ordermoe_route_select(ctypes.byref(lay), None, 0, None, None, ctypes.byref(out),
                                        None, 0, None)
    assert rc == om.EINVAL and "multiple of 64" in om.last_error()
    lay.d = 128
    lay.k = 9
    rc = om.lib().ordermoe_route_select(ctypes.byref(lay), None, 0, None, None, ctypes.byref(out),
                                        None, 0, None)
    assert rc == om.EINVAL
    lay.dtype = 7
    rc = om.lib().ordermoe_route_select(ctypes.byref(lay), None, 0, None, None, ctypes.byref(out),
                                        None, 0, None)
    assert rc == om.EDTYPE
    ex = om.Experts(dtype=om.BF16, d=4096, f=100, E=8, n_local=1, n_shared=0)
    assert om.lib().ordermoe_forward_workspace_size(ctypes.byref(ex), 16, 2) == 0
    rc = om.lib().ordermoe_local_moe_forward(ctypes.byref(ex), None, 0, 2, None, None, None, None,
                                             0, None, None, None, 0, None)
    assert rc == om.EINVAL and "f must be" in om.last_error()
    rc = om.lib().ordermoe_build_similarity(None, 10, 64, None, 300, om.BF16, 2, 0.7, 0.5, *([None] * 9),
                                            None, 0, None)
    assert rc == om.EINVAL
    assert om.lib().ordermoe_pack_gate_up(om.BF16, 1, 10, 64, None, None, None, None) == om.EINVAL
    # bf16 packing blocks 256 rows by 64 K: the shapes must divide (checked before any pointer)
    assert om.lib().ordermoe_pack_gate_up(om.BF16, 1, 96, 64, None, None, None, None) == om.EINVAL
    assert om.lib().ordermoe_pack_down(om.BF16, 1, 100, 128, None, None, None) == om.EINVAL
    assert om.lib().ordermoe_pack_down(om.BF16, 1, 256, 96, None, None, None) == om.EINVAL
    assert om.lib().ordermoe_pack_down(om.BF16, 1, 256, 128, None, None, None) == om.EINVAL   # null pointers
    assert om.lib().ordermoe_pack_down(om.F32, 0, 100, 8, None, None, None) == om.OK           # nothing to do
    # the device builds of eq 41-42: sizes, pointers and workspace checked before any launch
    L = om.lib()
    assert L.ordermoe_estimate_transitions_device(4, 300, 10, None, None, None, 0, None) == om.EINVAL
    assert L.ordermoe_estimate_transitions_device(4, 8, 10, None, None, None, 0, None) == om.EINVAL
    assert L.ordermoe_estimate_transitions_device(1, 8, 10, None, None, None, 0, None) == om.OK   # nothing to do
    need = L.ordermoe_transitions_device_workspace_size(4, 8)
    assert need == 3 * 8 * 8 * 4
    rc = L.ordermoe_estimate_transitions_device(4, 8, 10, ctypes.c_void_p(16), ctypes.c_void_p(16),
                                                ctypes.c_void_p(16), need - 1, None)
    assert rc == om.EWORKSPACE
    assert L.ordermoe_lookahead_device_workspace_size(4, 8, 33) == 0
    args = [None] * 11 + [0.5, 0.5, 1.0, 1, 1]
    assert L.ordermoe_build_lookahead_device(4, 8, 2, 0, *args, None, None, 0, None) == om.EINVAL    # H < 1
    assert L.ordermoe_build_lookahead_device(4, 8, 2, 2, *args[:15], 3, None, None, 0, None) == om.EINVAL
    rc = L.ordermoe_build_lookahead_device(4, 8, 2, 3, *args, ctypes.c_void_p(16), ctypes.c_void_p(16),
                                           1 << 20, None)
    assert rc == om.EINVAL and "null pointer" in om.last_error()          # H > 1 needs every input


@pytest.mark.parametrize("E", [129, 200, 256])
def test_similarity_build_rejects_more_than_128_experts(E):
    """The device build of eq 3-5 covers E <= 128 (its tile holds 128 experts);
    routing accepts up to 256.  Between the two the build returns EINVAL with a
    message naming the limit, before any pointer is looked at or anything is
    launched (all pointers here are null)."""
    rc = om.lib().ordermoe_build_similarity(None, 1024, 4096, None, E, om.BF16, 2, 0.7, 0.5,
                                            *([None] * 9), None, 0, None)
    assert rc == om.EINVAL
    assert "[1, 128]" in om.last_error()


def test_workspace_sizes_are_monotone():
    a = om.ordermoe_route_workspace_size(100, 2, 4)
    b = om.ordermoe_route_workspace_size(10000, 2, 4)
    assert 0 < a < b
    ex = om.Experts(dtype=om.BF16, d=4096, f=14336, E=8, n_local=2, n_shared=0)
    ids = np.array([0, 4], np.int32)
    ex.local_experts = ids.ctypes.data_as(ctypes.c_void_p)
    ex.w_gate_up = 16
    ex.w_down = 16
    s1 = om.lib().ordermoe_forward_workspace_size(ctypes.byref(ex), 100, 2)
    s2 = om.lib().ordermoe_forward_workspace_size(ctypes.byref(ex), 1000, 2)
    assert 0 < s1 < s2


def test_forward_rejects_operands_past_31_bit_offsets():
    """The GEMMs address operands with 32-bit byte offsets: T*d*esz, 2*f*d*esz,
    2*n_shared*f*d*esz and T*n_shared*f*esz must stay below 2^31 (no launch)."""
    ids = np.array([0, 4], np.int32)

    def experts(d, f, n_shared=0):
        ex = om.Experts(dtype=om.BF16, d=d, f=f, E=8, n_local=2, n_shared=n_shared)
        ex.local_experts = ids.ctypes.data_as(ctypes.c_void_p)
        ex.w_gate_up = ex.w_down = 16
        if n_shared:
            ex.w_shared_gate_up = ex.w_shared_down = 16
        return ex

    L = om.lib()
    ex = experts(4096, 1024)
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), (1 << 18) - 1, 2) > 0   # T*d*2 < 2^31
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 1 << 18, 2) == 0        # T*d*2 = 2^31
    p = ctypes.c_void_p(16)
    rc = L.ordermoe_local_moe_forward(ctypes.byref(ex), p, 1 << 18, 2, p, p, p, p, 0, p, p, p, 1 << 40, None)
    assert rc == om.EINVAL and "2^31" in om.last_error()
    # one expert's activation rows (at most T of them): T f 2 bytes
    ex = experts(256, 14336)
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 74898, 2) > 0
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 74899, 2) == 0
    # one expert's packed gate/up weights: 2 f d 2 bytes
    ex = experts(32768, 16384)                                 # 2^31 bytes exactly
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 16, 2) == 0
    ex = experts(32768, 16384 - 128)
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 16, 2) > 0
    # the shared experts side by side, and their activation rows
    ex = experts(4096, 14336, n_shared=16)                     # 2 * 16 * f * d * 2 > 2^31
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 16, 2) == 0
    ex = experts(256, 16384, n_shared=4)                       # 2 n f d 2 = 2^26; T n f 2 >= 2^31 at T = 2^14
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), (1 << 14) - 1, 2) > 0
    assert L.ordermoe_forward_workspace_size(ctypes.byref(ex), 1 << 14, 2) == 0


def test_noalloc_route_select_rejects_batches_beyond_its_scratch():
    """The allocation-free routing call checks the batch's workspace against its
    fixed scratch on the host and returns ORDERMOE_EWORKSPACE before any launch."""
    L = om.lib()
    T, k, M = 400000, 8, 32
    assert L.ordermoe_route_workspace_size(T, k, M) > om.NOALLOC_SCRATCH_BYTES
    assert L.ordermoe_route_workspace_size(65536, k, M) <= om.NOALLOC_SCRATCH_BYTES
    lay = om.Layer(dtype=om.BF16, d=512, E=64, k=k, M=M, gmax=3)
    for n in ("w_router", "t1_k", "t1_q", "t1_n", "srvmask", "S"):
        setattr(lay, n, 256)
    out = om.RouteOut()
    for n, _ in om.RouteOut._fields_:
        setattr(out, n, 256)
    p = ctypes.c_void_p(256)
    rc = L.ordermoe_route_select_noalloc(ctypes.byref(lay), p, T, p, p, ctypes.byref(out), None)
    assert rc == om.EWORKSPACE and "scratch" in om.last_error()
    # argument checks come first, as in ordermoe_route_select
    lay.k = 9
    assert L.ordermoe_route_select_noalloc(ctypes.byref(lay), p, T, p, p, ctypes.byref(out), None) == om.EINVAL


def test_weight_adaptation_oracle_pins():
    """eq 45: a step of kappa (Q_bar - T_bar) on omega_Q, projected onto [0, 1],
    with omega_T = 1 - omega_Q."""
    from oracle import tables
    # budget utilisation above the normalised delay: more weight on quality
    wq, wt = tables.adapt_weights(0.5, 0.1, 0.8, 1.0)
    assert wq == pytest.approx(0.52, rel=1e-15) and wt == pytest.approx(0.48, rel=1e-15)
    # the other way round: more weight on delay
    wq, _ = tables.adapt_weights(0.5, 0.1, 1.0, 0.2)
    assert wq == pytest.approx(0.42, rel=1e-15)
    # fixed point when both objectives are equally far behind
    assert tables.adapt_weights(0.3, 0.7, 0.6, 0.6) == (0.3, 0.7)
    # projection at both ends; kappa = 0 never moves
    assert tables.adapt_weights(0.95, 1.0, 0.0, 1.0) == (1.0, 0.0)
    assert tables.adapt_weights(0.05, 1.0, 1.0, 0.0) == (0.0, 1.0)
    assert tables.adapt_weights(0.25, 0.0, 3.0, 0.0) == (0.25, 0.75)


def test_library_weight_adaptation_matches_the_oracle():
    from oracle import tables
    from paper_2607_17154_amd import ordermoe as om
    rng = np.random.default_rng(11)
    for _ in range(200):
        wq, kappa, tb, qb = rng.random(), rng.random() * 2, rng.random() * 2, rng.random() * 2
        assert om.ordermoe_adapt_weights(wq, kappa, tb, qb) == tables.adapt_weights(wq, kappa, tb, qb)
    for bad in ((-0.1, 0.1, 0.5, 0.5), (1.1, 0.1, 0.5, 0.5), (0.5, -1.0, 0.5, 0.5),
                (0.5, 0.1, float("nan"), 0.5), (0.5, 0.1, 0.5, -0.1)):
        with pytest.raises(om.OrderMoEError):
            om.ordermoe_adapt_weights(*bad)
