"""GPU parity of the HIP library against the CPU oracle, through the C ABI.

Bar (stated by the method's evaluation contract): expert indices, execution
decisions, budgets, locations and dispatch lists bit-exact on every token
whose router logit margin is at least 1e-4 on both sides (the others are
flagged, counted and excluded); layer outputs within max relative error 2e-2
(bf16) / 1e-4 (fp32) per token, tokens without local rows exactly zero."""
import numpy as np
import pytest

import workloads as wl
from oracle import layer as olayer

from ._pipeline import (DeviceLayer, build_case, gemm_plan, host, library_tables, oracle_decisions,
                        oracle_output)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

TOL = {"bf16": 2e-2, "f32": 1e-4}

# the library's maximum sizes: 256 experts (16 clusters of 16, so every expert
# has the full 15 substitutes), top-8, 32 servers, server 0 holding 64 experts
# (capacities summing to exactly one copy of every expert), a shared expert.
# Router rows spread by sigma 0.5 at logit scale 4/sqrt(d), so that near-ties
# among a cluster's 16 members (margin < 1e-4) stay rare
CMAX = wl.LayerConfig(name="max_T600_d512_E256_f256_top8_M32", dtype="bf16", seed=9, T=600, d=512, E=256,
                      f=256, k=8, n_shared=1, clusters=16, cluster_size=16, sigma=0.5,
                      centre_std=4 * 512 ** -0.5, M=32, m0=0, capacity=(64.0,) + (6.0,) * 30 + (12.0,),
                      loc_mode="uniform", Qbar=0.25, theta=0.7, T_cal=4096)

# reduced shapes that span several tiles with ragged tails; full shapes below
SMALL = {
    "C1": wl.C1,
    "C2s": wl.C2.with_(T=1000, T_cal=4096),
    "C3s": wl.C3.with_(T=1500, T_cal=4096),
    "C4s": wl.C4.with_(T=1700, T_cal=4096),
    # the Local Substitute Only baseline: substitutes only on the token's server
    "C3s_local_sub": wl.C3.with_(T=1500, T_cal=4096, allow_sub=2),
    # 12 and 16 servers (the server-count sweep), tokens starting on every server
    "C4s_M12": wl.C4.with_(T=1700, T_cal=4096, M=12, capacity=(8.0,) * 12, loc_mode="uniform"),
    "C4s_M16": wl.C4.with_(T=1700, T_cal=4096, M=16, capacity=(8.0,) * 16, loc_mode="uniform"),
    "Cmax": CMAX,
    # the leftover-tile split along K (pieces of at least 16 K tiles), with one
    # shared expert so that the down projection's shared tiles have the routed K
    # and split too: the down projection in 2 pieces with no whole round (128
    # tiles), and the gate/up projection in 2 pieces after a whole round (312)
    "C3split": wl.C3.with_(T=600, d=2048, f=2048, n_shared=1, T_cal=4096),
    "C4split": wl.C4.with_(T=1200, d=2048, f=3072, n_shared=1, T_cal=4096),
    # four shared experts: the down projection's shared K is four times the
    # routed K, so its shared tiles are cut into two K halves
    "C3sh": wl.C3.with_(T=600, d=1024, f=512, n_shared=4, T_cal=4096),
    # 16-token routing blocks with their token rows staged in LDS (at most one
    # block per CU, d % 512 == 0), the last block holding 9 tokens
    "C2xl": wl.C2.with_(T=3001, d=2048, f=1024, T_cal=4096),
    # the same path at its bounds: 16 experts, d = 4096, 16 rows of 8 KB per block
    "C2xl16": wl.C2.with_(T=4001, f=512, E=16, clusters=8, cluster_size=2, capacity=(8.0,) * 4,
                          T_cal=4096),
    # a batch large enough for 256-row down tiles (the host's row bound fills
    # the grid eight times over), over two whole rounds and a partial one
    "C4tall": wl.C4.with_(T=4700, d=4096, f=256, T_cal=4096),
}
# shapes whose GEMM plan splits leftover tiles along K (checked on the GPU's rows)
SPLIT = {"C3split": {"gate_up": 0, "down": 2}, "C4split": {"gate_up": 2, "down": 1},
         "C2": {"gate_up": 2}, "C2x": {"gate_up": 3}}
# shapes whose down projection cuts its shared tiles into two K halves
SHARED_HALVES = {"C3sh", "C3"}
# shapes whose down projection takes 256-row tiles (large batches)
TALL_DOWN = {"C4", "C4tall"}
# decode-sized batches (at most 128 tokens): the thin-GEMM path of the forward
DECODE = {
    "C2d": wl.C2.with_(T=64, T_cal=4096),
    "C3d": wl.C3.with_(T=128, T_cal=4096),
    "C4d": wl.C4.with_(T=97, T_cal=4096),
    "C4d_M16": wl.C4.with_(T=97, T_cal=4096, M=16, capacity=(8.0,) * 16, loc_mode="uniform"),
    "Cmax_d": CMAX.with_(T=97),
}
FULL = {"C2": wl.C2.with_(T_cal=4096), "C3": wl.C3.with_(T_cal=4096), "C4": wl.C4.with_(T_cal=4096),
        # large batches with a ragged last block of the 32-token routing kernels:
        # at most 16 experts, and 17..64 experts (router rows staged in LDS)
        "C2x": wl.C2.with_(T=8192 + 33, T_cal=4096), "C3x": wl.C3.with_(T=8192 + 17, T_cal=4096)}

_cache = {}


def _case(name, cfg, **kw):
    key = (name, tuple(sorted(kw.items())))
    if key not in _cache:
        case = build_case(cfg, **kw)
        tabs = library_tables(case)
        _cache[key] = (case, tabs)
    return _cache[key]


def _flags(dec, out):
    return (dec["margin"] < 1e-4) | (host(out["margin"]) < 1e-4)


def _check_decisions(case, dec, out, max_flagged=0.01):
    cfg = case.cfg
    T, k = dec["idx"].shape
    fl = _flags(dec, out)
    ok = ~fl
    print("[%s] T=%d flagged=%d" % (cfg.name, T, int(fl.sum())), flush=True)
    assert fl.sum() <= max(2, max_flagged * T)
    g = {n: host(out[n]) for n in ("idx", "exec_k", "exec_m", "cls", "qhat_out", "loc_out", "flag")}
    np.testing.assert_array_equal(g["idx"][ok], dec["idx"][ok])
    np.testing.assert_array_equal(g["exec_k"][ok], dec["exec_k"][ok])
    np.testing.assert_array_equal(g["exec_m"][ok], dec["exec_m"][ok])
    np.testing.assert_array_equal(g["cls"][ok], dec["cls"][ok])
    np.testing.assert_array_equal(g["qhat_out"][ok], dec["qhat_out"][ok])
    np.testing.assert_array_equal(g["loc_out"][ok], dec["loc_out"][ok])
    np.testing.assert_array_equal(g["flag"].astype(bool), host(out["margin"]) < 1e-4)
    # gates: fp32 softmax of fp32 logits against fp64
    np.testing.assert_allclose(host(out["w"])[ok], dec["w"][ok], rtol=2e-4, atol=2e-6)
    # dispatch list: equal to the oracle's rule applied to the GPU's own decisions
    # (every token), and to the oracle's list once flagged tokens are dropped
    lst_gpu = host(out["dispatch"])
    cnt_gpu = host(out["dst_count"])
    counters = host(out["counters"])
    n_remote = int(counters[6])
    lst_self, cnt_self, tr_self = olayer.dispatch(g["exec_m"], case.loc, cfg.M)
    np.testing.assert_array_equal(lst_gpu[:n_remote], lst_self)
    np.testing.assert_array_equal(cnt_gpu, cnt_self)
    assert int(counters[5]) == tr_self
    lst_or, _, _ = olayer.dispatch(dec["exec_m"], case.loc, cfg.M)
    keep = lambda L: L[ok[L // k]]
    np.testing.assert_array_equal(keep(lst_gpu[:n_remote]), keep(lst_or))
    np.testing.assert_array_equal(counters[:4], olayer.class_counts(g["cls"]))
    assert int(counters[4]) == int(g["flag"].sum())
    assert int(counters[7]) == 0
    return ok


def _check_output(case, dec, y_gpu, tokens, ok, tol):
    want = oracle_output(case, dec, tokens)
    got = host(y_gpu)[tokens]
    worst = 0.0
    for i, t in enumerate(tokens):
        if not ok[t]:
            continue
        ref = np.max(np.abs(want[i]))
        if ref == 0.0:
            assert np.all(got[i] == 0.0), t
            continue
        err = np.max(np.abs(got[i] - want[i])) / ref
        worst = max(worst, err)
    print("[%s] output max rel err %.3g over %d tokens" % (case.cfg.name, worst, len(tokens)), flush=True)
    assert worst <= tol


def _check_split(name, case, rows):
    """The shapes meant to exercise the split along K do split (host mirror of
    the launch plan, from the GPU's own row counts)."""
    if name not in SPLIT and name not in SHARED_HALVES and name not in TALL_DOWN:
        return
    plan = gemm_plan(case.cfg, rows, len(case.local))
    print("[%s] GEMM plan (tiles, grid, rounds, left, split, shared halves, tile rows): %s"
          % (case.cfg.name, plan), flush=True)
    assert plan["down"][6] == (256 if name in TALL_DOWN else 192), plan["down"]
    for gemm, want in SPLIT.get(name, {}).items():
        assert plan[gemm][4] == want, (gemm, plan[gemm])
    assert plan["down"][5] == int(name in SHARED_HALVES), plan["down"]
    assert plan["gate_up"][5] == 0, plan["gate_up"]


@pytest.mark.parametrize("name", list(SMALL))
def test_layer_parity_small(name):
    case, tabs = _case(name, SMALL[name])
    dl = DeviceLayer(case, tabs)
    x, loc, qh = dl.inputs()
    T = case.X.shape[0]
    out = dl.route(x, loc, qh, T)
    y, ro = dl.forward(x, loc, out, T)
    torch.cuda.synchronize()
    dec = oracle_decisions(case)
    ok = _check_decisions(case, dec, out)
    # row offsets: the GPU's own local rows, recounted from its decisions
    rows = host(ro)
    assert rows[0] == 0 and np.all(np.diff(rows) >= 0)
    _check_split(name, case, rows)
    _check_output(case, dec, y, np.arange(T), ok, TOL[case.cfg.dtype])


@pytest.mark.parametrize("name", list(DECODE))
def test_layer_parity_decode_batch(name):
    case, tabs = _case(name, DECODE[name])
    dl = DeviceLayer(case, tabs)
    x, loc, qh = dl.inputs()
    T = case.X.shape[0]
    out = dl.route(x, loc, qh, T)
    y, ro = dl.forward(x, loc, out, T)
    torch.cuda.synchronize()
    dec = oracle_decisions(case)
    ok = _check_decisions(case, dec, out)
    _check_output(case, dec, y, np.arange(T), ok, TOL[case.cfg.dtype])


@pytest.mark.parametrize("name", list(FULL))
def test_layer_parity_full_shape(name):
    """The full-size layers in the launch configuration the benchmark times:
    decisions and every unflagged token's output against the oracle."""
    case, tabs = _case(name, FULL[name])
    dl = DeviceLayer(case, tabs)
    x, loc, qh = dl.inputs()
    T = case.X.shape[0]
    out = dl.route(x, loc, qh, T)
    y, ro = dl.forward(x, loc, out, T)
    torch.cuda.synchronize()
    dec = oracle_decisions(case)
    ok = _check_decisions(case, dec, out)
    _check_split(name, case, host(ro))
    _check_output(case, dec, y, np.arange(T), ok, TOL[case.cfg.dtype])


@pytest.mark.parametrize("Qbar", wl.C4_QBAR_SWEEP)
def test_quality_budget_sweep(Qbar):
    cfg = wl.C4.with_(T=2048, T_cal=4096, Qbar=Qbar)
    case, tabs = _case("C4q%g" % Qbar, cfg, qhat_scale=0.0)
    dl = DeviceLayer(case, tabs, with_experts=False)
    x, loc, qh = dl.inputs()
    out = dl.route(x, loc, qh, case.X.shape[0])
    torch.cuda.synchronize()
    dec = oracle_decisions(case)
    _check_decisions(case, dec, out)
    assert np.all(host(out["qhat_out"]) <= np.float32(Qbar))       # Property 2
    if Qbar == 0.0:
        assert not np.any(host(out["cls"]) & 1)


def test_partly_spent_budget_and_remote_sources():
    cfg = wl.C3.with_(T=3000, T_cal=4096, Qbar=0.03)
    case, tabs = _case("C3spent", cfg, qhat_scale=0.03)
    dl = DeviceLayer(case, tabs, with_experts=False)
    x, loc, qh = dl.inputs()
    out = dl.route(x, loc, qh, case.X.shape[0])
    torch.cuda.synchronize()
    _check_decisions(case, oracle_decisions(case), out)


def test_no_substitution_sum_over_servers_is_exact_moe():
    # Qbar = 0: every slot runs its target; the outputs of all servers add up
    # to the plain top-k MoE layer
    cfg = wl.C3.with_(T=700, T_cal=4096, Qbar=0.0)
    case, tabs = _case("C3exact", cfg)
    dec = oracle_decisions(case)
    assert np.array_equal(dec["exec_k"], dec["idx"])
    total = None
    for m in range(cfg.M):
        local = [int(j) for j in np.nonzero(case.x_dep[m])[0]]
        c_m = build_case(cfg.with_(m0=m), T=700)
        dl = DeviceLayer(c_m, library_tables(c_m), with_experts=True)
        x, loc, qh = dl.inputs()
        out = dl.route(x, loc, qh, 700)
        y, _ = dl.forward(x, loc, out, 700)
        torch.cuda.synchronize()
        assert c_m.local == local
        total = host(y).astype(np.float64) if total is None else total + host(y)
    want = sum(olayer.server_output(case.X, dec["w"], dec["exec_k"], dec["exec_m"], case.loc, m,
                                    case.expert, case.shared(), np.arange(700)) for m in range(cfg.M))
    fl = dec["margin"] < 1e-4
    err = np.max(np.abs(total - want)[~fl], axis=1) / np.max(np.abs(want[~fl]), axis=1)
    print("exact-MoE max rel err %.3g" % err.max(), flush=True)
    assert err.max() <= TOL["bf16"]


def test_all_local_means_no_remote():
    cfg = wl.C2.with_(T=512, T_cal=4096)
    case, _ = _case("C2local", cfg)
    case.x_dep = case.x_dep.copy()
    case.x_dep[cfg.m0, :] = 1
    case.local = list(range(cfg.E))
    tabs = library_tables(case)
    dl = DeviceLayer(case, tabs, with_experts=False)
    x, loc, qh = dl.inputs()
    out = dl.route(x, loc, qh, 512)
    torch.cuda.synchronize()
    assert np.all(host(out["cls"]) == 0)
    c = host(out["counters"])
    assert c[2] == 0 and c[3] == 0 and c[5] == 0 and c[6] == 0
    assert np.all(host(out["dst_count"]) == 0)


@pytest.mark.parametrize("variant", ["pin0", "renorm0"])
def test_selection_variants(variant):
    kw = {"pin0": dict(pin_local_exact=0), "renorm0": dict(renorm=0)}[variant]
    cfg = wl.C3.with_(T=1200, T_cal=4096, **kw)
    case, tabs = _case("C3" + variant, cfg)
    dl = DeviceLayer(case, tabs, with_experts=False)
    x, loc, qh = dl.inputs()
    out = dl.route(x, loc, qh, 1200)
    torch.cuda.synchronize()
    _check_decisions(case, oracle_decisions(case), out)


def test_negative_and_signed_zero_costs_order_as_floats():
    """eq 43's argmin over J = S + (omega_Q / Qbar) Q when the static costs are
    shifted below zero (and some entries are -0): the device's packed key
    orders J as the float comparison of the oracle does."""
    cfg = wl.C3.with_(T=1200, T_cal=4096)
    case, tabs = _case("C3s_costs", cfg)
    import copy
    case = copy.copy(case)
    shift = np.float32(np.median(case.S))
    S = (case.S - shift).astype(np.float32)
    S[S == 0] = np.float32(-0.0)
    S[0, 1, :3] = np.float32(-0.0)
    assert (S < 0).mean() > 0.3
    case.S = S
    tabs = dict(tabs, S=S.copy())
    dl = DeviceLayer(case, tabs, with_experts=False)
    x, loc, qh = dl.inputs()
    out = dl.route(x, loc, qh, cfg.T)
    torch.cuda.synchronize()
    _check_decisions(case, oracle_decisions(case), out)


def test_empty_and_single_token_batches():
    case, tabs = _case("C1", wl.C1)
    dl = DeviceLayer(case, tabs)
    for T in (0, 1, 17):
        x, loc, qh = dl.inputs(case.X[:T], case.loc[:T], case.qhat[:T])
        if T == 0:
            x = torch.empty((0, case.cfg.d), device="cuda")
        out = dl.route(x, loc, qh, T)
        y, ro = dl.forward(x, loc, out, T)
        torch.cuda.synchronize()
        c = host(out["counters"])
        assert c[:4].sum() == T * case.cfg.k and c[7] == 0
        if T == 0:
            assert np.all(host(ro) == 0) and np.all(c == 0)
        else:
            dec = oracle_decisions(case)
            sl = slice(0, T)
            np.testing.assert_array_equal(host(out["exec_k"]), dec["exec_k"][sl])


def test_invalid_locations_are_counted_not_routed():
    case, tabs = _case("C1", wl.C1)
    dl = DeviceLayer(case, tabs, with_experts=False)
    loc = case.loc.copy()
    loc[5] = 7
    loc[9] = 255
    x, loc_d, qh = dl.inputs(loc=loc)
    out = dl.route(x, loc_d, qh, case.X.shape[0])
    torch.cuda.synchronize()
    c = host(out["counters"])
    assert c[7] == 2
    ek = host(out["exec_k"])
    assert np.all(ek[[5, 9]] == -1) and np.all(host(out["cls"])[[5, 9]] == 255)
    assert c[:4].sum() == (case.X.shape[0] - 2) * case.cfg.k


@pytest.mark.parametrize("name", ["C3s", "C3d", "C3split", "C3sh", "C2", "C4"])
def test_runs_are_bitwise_deterministic(name):
    """Two runs give the same bits; C3split, C3sh and the full C2 layer split
    GEMM tiles along K, whose pieces are summed in K order by whichever
    workgroup arrives last; the full C4 layer runs 256-row down tiles."""
    case, tabs = _case(name, {**SMALL, **DECODE, **FULL}[name])
    dl = DeviceLayer(case, tabs)
    x, loc, qh = dl.inputs()
    T = case.X.shape[0]
    res = []
    for _ in range(2):
        out = dl.route(x, loc, qh, T)
        y, _ = dl.forward(x, loc, out, T)
        torch.cuda.synchronize()
        n_remote = int(host(out["counters"])[6])
        res.append((host(out["exec_k"]), host(out["dispatch"])[:n_remote], host(y),
                    host(out["counters"])))
    for a, b in zip(res[0], res[1]):
        np.testing.assert_array_equal(a, b)


def test_graph_replay_matches_eager():
    """route/select and the local forward captured in a HIP graph: every
    replay, with eager work and synchronisation between them, equals the eager
    result bit for bit (decode-sized and prefill-sized batches)."""
    for name in ("C3d", "C2s"):
        case, tabs = _case(name, {**SMALL, **DECODE}[name])
        dl = DeviceLayer(case, tabs)
        x, loc, qh = dl.inputs()
        T = case.X.shape[0]
        cfg = case.cfg
        from paper_2607_17154_amd import ordermoe as om
        out = om.alloc_route_out(T, cfg.k, cfg.M, "cuda")
        ws_r = torch.empty(max(om.ordermoe_route_workspace_size(T, cfg.k, cfg.M), 1), dtype=torch.uint8,
                           device="cuda")
        y = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
        ro = torch.empty(dl.experts.n_local + 2, dtype=torch.int32, device="cuda")
        ws_f = torch.empty(max(om.ordermoe_forward_workspace_size(dl.experts, T, cfg.k), 1),
                           dtype=torch.uint8, device="cuda")

        def step():
            om.ordermoe_route_select(dl.layer, x, T, loc, qh, out, ws_r)
            om.ordermoe_local_moe_forward(dl.experts, x, T, cfg.k, out["w"], out["exec_k"], out["exec_m"],
                                          loc, cfg.m0, y, ro, ws_f)

        step()
        torch.cuda.synchronize()
        want = [host(out[n]) for n in ("exec_k", "exec_m", "counters")] + [host(y)]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for rep in range(3):
            y.zero_()
            out["exec_k"].fill_(-7)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            got = [host(out[n]) for n in ("exec_k", "exec_m", "counters")] + [host(y)]
            for a_, b_ in zip(got, want):
                np.testing.assert_array_equal(a_, b_)
        del g
