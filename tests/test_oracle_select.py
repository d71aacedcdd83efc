"""Pins of the oracle's runtime selection (eq 36-44) and dispatch, CPU only."""
from fractions import Fraction

import numpy as np
import pytest

import workloads as wl
from oracle import layer, route, similarity, tables


def _f32_round(fr: Fraction) -> np.float32:
    """Correctly rounded fp32 value of an exact rational (ties to even)."""
    f = np.float32(float(fr))
    best = None
    for c in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        err = abs(Fraction(float(c)) - fr)
        key = (err, int(np.float32(c).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return np.float32(best[1])


def _brute_select_token(r_list, s, qhat, x, sim, group_of, theta, S, Qbar, omega_Q, pin, allow):
    """Enumerate every (m, k) of the grid, keep those in A (eq 40) and take the
    argmin of eq 43 with exact arithmetic rounded once to fp32."""
    M, E = x.shape
    cq = np.float32(np.float32(omega_Q) / np.float32(Qbar)) if Qbar > 0 else np.float32(0)
    out = []
    for r in r_list:
        if pin and x[s, r]:
            out.append((r, s, 0, np.float32(0)))
            continue
        best = None
        for m in range(M):
            for kk in range(E):
                if not x[m, kk]:
                    continue
                if kk == r:
                    q = np.float32(0)
                else:
                    if not (allow and Qbar > 0):
                        continue
                    if allow == 2 and m != s:      # local substitutes only
                        continue
                    in_v = group_of[kk] == group_of[r] and np.float32(sim[r, kk]) >= np.float32(theta)
                    if not in_v:
                        continue
                    q = np.float32((np.float32(1) - np.float32(sim[r, kk])) * np.float32(0.5))
                    if not (np.float32(qhat + q) <= np.float32(Qbar)):
                        continue
                J = _f32_round(Fraction(float(cq)) * Fraction(float(q)) + Fraction(float(S[s, m, kk])))
                key = (float(J), float(q), kk != r, kk, m != s, m)
                if best is None or key < best[0]:
                    best = (key, kk, m, q)
        _, kk, m, q = best
        c = (2 if m != s else 0) | (1 if kk != r else 0)
        out.append((kk, m, c, q))
        qhat = np.float32(qhat + q)
    return out, qhat


def _random_layer(rng, T):
    E = int(rng.integers(2, 7))
    M = int(rng.integers(1, 4))
    k = int(rng.integers(1, min(3, E) + 1))
    group_of = rng.integers(0, 2, size=E).astype(np.int32)
    sim = rng.choice(np.float32([0.3, 0.6, 0.8, 0.9, 0.95]), size=(E, E)).astype(np.float32)
    sim = np.triu(sim, 1) + np.triu(sim, 1).T + np.eye(E, dtype=np.float32)
    x = (rng.random((M, E)) < 0.5).astype(np.uint8)
    for j in range(E):
        if x[:, j].sum() == 0:
            x[int(rng.integers(0, M)), j] = 1
    S = rng.choice(np.float32([0.5, 0.5, 0.75, 2.0, 40.0]), size=(M, M, E)).astype(np.float32)
    idx = np.array([rng.permutation(E)[:k] for _ in range(T)], dtype=np.int32)
    loc = rng.integers(0, M, size=T).astype(np.uint8)
    Qbar = float(rng.choice([0.0, 0.05, 0.1, 0.3]))
    qhat = (rng.random(T) * Qbar).astype(np.float32)
    theta = float(rng.choice([0.5, 0.85]))
    return dict(E=E, M=M, k=k, group_of=group_of, sim=sim, x=x, S=S, idx=idx, loc=loc,
                Qbar=Qbar, qhat=qhat, theta=theta)


@pytest.mark.parametrize("pin", [0, 1])
def test_select_matches_exhaustive_enumeration(pin):
    rng = np.random.default_rng(10 + pin)
    for trial in range(40):
        L = _random_layer(rng, 60)
        allow = int(rng.integers(0, 3))
        o = layer.select(L["idx"], L["x"], L["sim"], L["group_of"], L["theta"], L["S"],
                         L["Qbar"], 0.5, L["loc"], L["qhat"], pin, allow)
        for t in range(60):
            want, qh = _brute_select_token(list(L["idx"][t]), int(L["loc"][t]), L["qhat"][t],
                                           L["x"], L["sim"], L["group_of"], L["theta"], L["S"],
                                           L["Qbar"], 0.5, pin, allow)
            got = [(int(o["exec_k"][t, s]), int(o["exec_m"][t, s]), int(o["cls"][t, s]))
                   for s in range(L["k"])]
            assert got == [(a, b, c) for (a, b, c, _) in want], (trial, t)
            assert o["qhat_out"][t] == qh
            assert o["loc_out"][t] == want[0][1]


def _c1_pipeline(Qbar=None, allow_sub=1, all_local=False, T=None):
    cfg = wl.C1 if Qbar is None else wl.C1.with_(Qbar=Qbar)
    W = wl.router(cfg)
    model = similarity.build(wl.calibration(cfg), W, cfg.k, cfg.theta)
    x, _ = __import__("oracle").placement.place([model["group_of"]], [model["I"]],
                                                 [np.ones(cfg.E)], np.array(cfg.capacity),
                                                 np.full(cfg.M, 1.0 / cfg.M))
    x = x[0]
    if all_local:
        x = x.copy()
        x[cfg.m0, :] = 1
    net = wl.network(cfg)
    c = np.full(cfg.E, 6.0 * cfg.d * cfg.f)
    dref = tables.d_ref(c, net.F)
    S = tables.static_cost(cfg.M, cfg.E, cfg.d * cfg.bytes_per_el * 8.0, net.B, net.tau, c,
                           net.F, dref, cfg.omega_T)
    X = wl.tokens(cfg, T)
    idx, w, mg, _ = route.route(X, W, cfg.k)
    loc = wl.token_locations(cfg, len(X))
    qh = wl.accumulated_loss(cfg, len(X))
    sim32 = model["sim"].astype(np.float32)
    o = layer.select(idx, x, sim32, model["group_of"], cfg.theta, S, cfg.Qbar, cfg.omega_Q,
                     loc, qh, cfg.pin_local_exact, allow_sub)
    return cfg, model, x, idx, o, loc, qh, sim32


def test_property1_feasibility_and_local_sub_in_group():
    cfg, model, x, idx, o, loc, qh, sim32 = _c1_pipeline()
    T, k = idx.shape
    for t in range(T):
        for s in range(k):
            r, kk, m = idx[t, s], o["exec_k"][t, s], o["exec_m"][t, s]
            assert x[m, kk] == 1                                       # c.6
            if kk != r:                                                # c.7
                assert model["group_of"][kk] == model["group_of"][r]
                assert sim32[r, kk] >= np.float32(cfg.theta)
            if o["cls"][t, s] == 1:
                assert m == loc[t] and x[loc[t], kk] == 1
    counts = layer.class_counts(o["cls"])
    assert counts.sum() == T * k
    # the C1 deployment holds {0,2,4,6} on server 0: every target of the
    # other half is substituted locally by its group partner
    assert counts[0] > 0 and counts[1] > 0 and counts[2] == 0 and counts[3] == 0


def test_property2_budget_invariant():
    rng = np.random.default_rng(7)
    for trial in range(30):
        L = _random_layer(rng, 80)
        o = layer.select(L["idx"], L["x"], L["sim"], L["group_of"], L["theta"], L["S"],
                         L["Qbar"], 0.5, L["loc"], L["qhat"], 0, 1)
        assert np.all(o["qhat_out"] <= np.float32(L["Qbar"]))


def test_all_local_gives_no_remote_and_empty_dispatch():
    cfg, model, x, idx, o, loc, qh, _ = _c1_pipeline(all_local=True)
    assert np.all(o["cls"] == 0)
    lst, cnt, transfers = layer.dispatch(o["exec_m"], loc, cfg.M)
    assert len(lst) == 0 and transfers == 0 and cnt.sum() == 0


@pytest.mark.parametrize("Qbar,allow", [(0.0, 1), (0.25, 0)])
def test_no_substitution_means_exact(Qbar, allow):
    cfg, model, x, idx, o, loc, qh, _ = _c1_pipeline(Qbar=Qbar, allow_sub=allow)
    assert np.array_equal(o["exec_k"], idx)
    assert np.all(o["qhat_out"] == 0)


def test_dispatch_hand_example():
    exec_m = np.array([[1, 0], [2, 2], [0, 1]], dtype=np.uint8)
    loc = np.array([0, 0, 1], dtype=np.uint8)
    lst, cnt, transfers = layer.dispatch(exec_m, loc, 3)
    # remote slots: (t0,s0)->1, (t1,s0)->2, (t1,s1)->2, (t2,s0)->0
    assert list(lst) == [2 * 2 + 0, 0 * 2 + 0, 1 * 2 + 0, 1 * 2 + 1]
    assert list(cnt) == [1, 1, 2]
    assert transfers == 3
