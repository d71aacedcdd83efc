"""Decode stream through the 32-layer stack on the GPU, through the C ABI.

Each layer's route/select reads the locations and accumulated losses the
previous layer wrote on the device (Algorithm 2's loop over layers), with the
layer's threshold (eq 6) and look-ahead tables (eq 41-42, H = 3).  The oracle
runs the same chain from its own outputs.  A token whose router margin falls
below 1e-4 on either side at some layer is flagged there and its decisions at
that layer are not compared; the oracle then takes the GPU's recorded location
and accumulated loss for it, so every token enters every layer in the same
state on both sides and every unflagged (token, layer) pair is compared (the
count is asserted).  Property 2
(the accumulated loss never exceeds the budget) is checked on every token at
every layer.  The local expert FFN of server 0 is checked at the first and
the last layer against the oracle's output."""
import numpy as np
import pytest

import workloads as wl
from oracle import layer as olayer

from ._pipeline import host, stream_library_tables, stream_oracle_layer, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_17154_amd import ordermoe as om  # noqa: E402

FORWARD_LAYERS = (0, 31)


def _gpu_chain(sc, keep_layers=()):
    """Run the route/select chain of the stack on the GPU; every layer's outputs
    (host) and the device inputs of the layers in keep_layers."""
    cfg = sc.cfg
    theta32, phi, tabs = stream_library_tables(sc)
    T = cfg.T
    loc = torch.zeros(T, dtype=torch.uint8, device="cuda")
    qh = torch.zeros(T, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(om.ordermoe_route_workspace_size(T, cfg.k, cfg.M), 1), dtype=torch.uint8,
                     device="cuda")
    gmax = 15
    layers, keep = [], {}
    for l in range(cfg.N):
        wr = to_device(sc.W_r[l], cfg.dtype)
        tdev = {n: torch.from_numpy(np.ascontiguousarray(v)).cuda() for n, v in tabs[l].items()
                if n != "srvmask"}
        tdev["srvmask"] = torch.from_numpy(tabs[l]["srvmask"].view(np.int32)).cuda()
        L = om.make_layer(om.BF16, cfg.d, cfg.E, cfg.k, cfg.M, gmax, wr, tdev, cfg.Qbar, cfg.omega_Q,
                          cfg.pin_local_exact, cfg.allow_sub, cfg.renorm)
        x = to_device(sc.X[l], cfg.dtype)
        out = om.alloc_route_out(T, cfg.k, cfg.M, "cuda")
        om.ordermoe_route_select(L, x, T, loc, qh, out, ws)
        torch.cuda.synchronize()
        rec = {n: host(v) for n, v in out.items()}
        rec["loc_in"] = host(loc)
        layers.append(rec)
        if l in keep_layers:
            keep[l] = (x, loc.clone(), out)
        loc, qh = out["loc_out"], out["qhat_out"]   # carried to the next layer on the device
    return dict(layers=layers, keep=keep)


def _oracle_chain(sc, gpu_layers):
    """The oracle's own chain: per layer its decisions, the locations it started
    from, and the tokens not flagged (on either side) at that layer.  After a
    layer, a flagged token's location and accumulated loss are re-synced to the
    values the GPU recorded for it (its decision may legitimately differ)."""
    cfg = sc.cfg
    loc = np.zeros(cfg.T, np.uint8)
    qh = np.zeros(cfg.T, np.float32)
    res = []
    for l in range(cfg.N):
        dec = stream_oracle_layer(sc, l, loc, qh)
        g = gpu_layers[l]
        flag = (dec["margin"] < 1e-4) | (g["margin"] < 1e-4)
        res.append(dict(dec=dec, loc_in=loc, qhat_in=qh, live=~flag, flag=flag))
        loc = np.where(flag, g["loc_out"], dec["loc_out"]).astype(np.uint8)
        qh = np.where(flag, g["qhat_out"], dec["qhat_out"]).astype(np.float32)
    return res


def _compare_chain(sc, gpu_layers, oracle_chain):
    """Decisions bit-exact on live tokens at every layer, the GPU's inputs are
    its previous outputs, Property 2, counters and dispatch lists; returns the
    first layer at which substitution has stopped."""
    cfg = sc.cfg
    T, k = cfg.T, cfg.k
    exhausted_layer = None
    compared = flagged = 0
    for l in range(cfg.N):
        g = gpu_layers[l]
        dec, loc, live, flag = (oracle_chain[l][n] for n in ("dec", "loc_in", "live", "flag"))
        if l > 0:
            np.testing.assert_array_equal(g["loc_in"], gpu_layers[l - 1]["loc_out"])
            # both sides start the layer in the same state, every token
            np.testing.assert_array_equal(oracle_chain[l]["qhat_in"], gpu_layers[l - 1]["qhat_out"])
        np.testing.assert_array_equal(g["loc_in"], loc, err_msg="H %d layer %d loc_in" % (cfg.H, l))
        ok = live
        compared += int(ok.sum())
        flagged += int(flag.sum())
        for n in ("idx", "exec_k", "exec_m", "cls", "qhat_out", "loc_out"):
            np.testing.assert_array_equal(g[n][ok], dec[n][ok], err_msg="H %d layer %d %s" % (cfg.H, l, n))
        # Property 2 on every token, flagged or not
        assert np.all(g["qhat_out"] <= np.float32(cfg.Qbar)), l
        # class counters and the dispatch list of the GPU's own decisions
        c = g["counters"]
        np.testing.assert_array_equal(c[:4], olayer.class_counts(g["cls"]))
        lst, cnt, tr = olayer.dispatch(g["exec_m"], g["loc_in"], cfg.M)
        n_remote = int(c[6])
        np.testing.assert_array_equal(g["dispatch"][:n_remote], lst)
        np.testing.assert_array_equal(g["dst_count"], cnt)
        assert int(c[5]) == tr and int(c[7]) == 0
        lst_o, _, _ = olayer.dispatch(dec["exec_m"], loc, cfg.M)
        sel = lambda a: a[ok[a // k]]
        np.testing.assert_array_equal(sel(g["dispatch"][:n_remote]), sel(lst_o))
        subs = int(c[1] + c[3])
        if exhausted_layer is None and l > 0 and subs < 0.02 * T * k:
            exhausted_layer = l
        print("H %d layer %2d: LE/LS/RE/RS %s  flagged %d  compared %d  max Qhat %.4f" % (
            cfg.H, l, list(c[:4]), int(flag.sum()), int(ok.sum()), float(g["qhat_out"].max())), flush=True)
    print("H %d: %d of %d (token, layer) pairs compared, %d flagged; substitution stops at layer %s"
          % (cfg.H, compared, T * cfg.N, flagged, exhausted_layer), flush=True)
    assert compared == T * cfg.N - flagged
    assert flagged <= 0.02 * T * cfg.N
    return exhausted_layer


@pytest.fixture(scope="module")
def chain(stream_case):
    return _gpu_chain(stream_case, FORWARD_LAYERS)


@pytest.fixture(scope="module")
def oracle_chain(stream_case, chain):
    return _oracle_chain(stream_case, chain["layers"])


def test_chain_decisions_match_the_oracle(stream_case, chain, oracle_chain):
    exhausted_layer = _compare_chain(stream_case, chain["layers"], oracle_chain)
    # the budget binds mid-stream: substitutions give way to exact execution
    assert exhausted_layer is not None and 4 <= exhausted_layer < stream_case.cfg.N - 4


def test_delay_simulator_follows_the_device_trajectory(stream_case, chain):
    """The library's delay simulator (eq 13-17, eq 22) over the device's
    decisions: its trajectory equals the locations the kernels carried from
    layer to layer, its remote-slot and transfer counts equal the kernels'
    counters, and its delays equal the oracle's evaluation of the same
    decisions bit for bit."""
    from oracle import delay as odelay
    sc, cfg = stream_case, stream_case.cfg
    g = chain["layers"]
    em = np.stack([r["exec_m"].reshape(cfg.T, cfg.k) for r in g])
    ek = np.stack([r["exec_k"].reshape(cfg.T, cfg.k) for r in g])
    z = [sc.z_bits] * cfg.N
    c = [sc.c] * cfg.N
    sim = om.ordermoe_simulate_delay(g[0]["loc_in"], em, ek, c, z, sc.net.B, sc.net.tau, sc.net.F)
    for l in range(cfg.N):
        np.testing.assert_array_equal(sim["loc"][l], g[l]["loc_in"])
    cnt = np.sum([r["counters"] for r in g], axis=0)
    assert sim["remote_slots"] == int(cnt[om.CNT_REMOTE_SLOTS])
    assert sim["transfers"] == int(cnt[om.CNT_TRANSFERS])
    assert sim["slots"] == int(cnt[:4].sum())
    want = odelay.simulate(g[0]["loc_in"], em, ek, c, z, sc.net.B, sc.net.tau, sc.net.F)
    np.testing.assert_array_equal(sim["delay"], want["delay"])
    np.testing.assert_array_equal(sim["work"], want["work"])


@pytest.mark.parametrize("H,allow_sub", [(1, 1), (5, 1), (3, 2)])
def test_chain_decisions_match_the_oracle_at_other_horizons(stream_case, H, allow_sub):
    """The look-ahead sweep of Fig. 7: the myopic rule (H = 1) and the deepest
    horizon swept (H = 5) run the same chain comparison, and so does the Local
    Substitute Only mode (allow_sub = 2)."""
    from ._pipeline import with_horizon
    sc = with_horizon(stream_case, H, allow_sub=allow_sub)
    g = _gpu_chain(sc)
    _compare_chain(sc, g["layers"], _oracle_chain(sc, g["layers"]))


@pytest.fixture(scope="module")
def stream_case_ratio1():
    """The 32-layer stack at memory ratio 1.0 (one copy of every expert): the
    look-ahead (eq 42-43) changes decisions here."""
    from ._pipeline import build_stream
    return build_stream(wl.C5_STREAM.with_(memory_ratio=1.0))


def test_lookahead_decides_at_memory_ratio_one(stream_case_ratio1):
    """At H = 3 and H = 1 the chains both match the oracle slot for slot, and
    the look-ahead term moves at least one slot to another (server, expert)
    than the myopic rule picks (eq 43 with Phi != 0)."""
    from ._pipeline import with_horizon
    runs = {}
    for H in (1, 3):
        sc = stream_case_ratio1 if H == stream_case_ratio1.cfg.H else with_horizon(stream_case_ratio1, H)
        g = _gpu_chain(sc)
        _compare_chain(sc, g["layers"], _oracle_chain(sc, g["layers"]))
        runs[H] = g["layers"]
    differ = sum(int(np.sum((a["exec_m"] != b["exec_m"]) | (a["exec_k"] != b["exec_k"])))
                 for a, b in zip(runs[1], runs[3]))
    print("memory ratio 1.0: %d slots decided differently at H = 3 than at H = 1" % differ, flush=True)
    assert differ > 0


@pytest.mark.parametrize("layer", FORWARD_LAYERS)
def test_local_forward_of_a_stream_layer(stream_case, chain, oracle_chain, layer):
    sc, cfg = stream_case, stream_case.cfg
    x, loc, out = chain["keep"][layer]
    oc = oracle_chain[layer]
    local = sc.local[layer]
    cache = {}

    def expert(j):
        if j not in cache:
            cache[j] = wl.stream_expert(cfg, layer, j)
        return cache[j]

    n = len(local)
    wg = torch.empty((n, cfg.f, cfg.d), dtype=torch.bfloat16, device="cuda")
    wu = torch.empty_like(wg)
    wd = torch.empty((n, cfg.d, cfg.f), dtype=torch.bfloat16, device="cuda")
    for i, j in enumerate(local):
        a, b, c = expert(j)
        wg[i], wu[i], wd[i] = to_device(a, "bf16"), to_device(b, "bf16"), to_device(c, "bf16")
    wgu = torch.empty((n, 2 * cfg.f, cfg.d), dtype=torch.bfloat16, device="cuda")
    om.ordermoe_pack_gate_up(wg, wu, wgu)
    wdp = torch.empty_like(wd)
    om.ordermoe_pack_down(wd, wdp)
    del wg, wu, wd
    ex = om.make_experts(om.BF16, cfg.d, cfg.f, cfg.E, local, wgu, wdp)
    T = cfg.T
    y = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
    ro = torch.empty(n + 2, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(om.ordermoe_forward_workspace_size(ex, T, cfg.k), 1), dtype=torch.uint8,
                     device="cuda")
    om.ordermoe_local_moe_forward(ex, x, T, cfg.k, out["w"], out["exec_k"], out["exec_m"], loc,
                                  cfg.m0, y, ro, ws)
    torch.cuda.synchronize()
    rows = host(ro)
    print("layer %d: %d local rows over %d experts" % (layer, int(rows[-1]), int(np.sum(np.diff(rows[:-1]) > 0))),
          flush=True)
    # the oracle's output from its own decisions, on the tokens whose decisions
    # agree (not flagged up to this layer)
    dec = oc["dec"]
    tokens = np.nonzero(oc["live"])[0]
    want = olayer.server_output(sc.X[layer], dec["w"], dec["exec_k"], dec["exec_m"], oc["loc_in"],
                                cfg.m0, expert, [], tokens)
    got = host(y)[tokens]
    worst = 0.0
    for t in range(len(tokens)):
        ref = np.max(np.abs(want[t]))
        if ref == 0.0:
            assert np.all(got[t] == 0.0), t
            continue
        worst = max(worst, float(np.max(np.abs(got[t] - want[t])) / ref))
    print("layer %d output max rel err %.3g over %d tokens" % (layer, worst, len(tokens)), flush=True)
    assert worst <= 2e-2
