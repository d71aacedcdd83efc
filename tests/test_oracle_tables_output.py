"""Pins of the oracle's tables (eq 6, 37-38, 41-42) and layer output, CPU only."""
import numpy as np
import pytest

import workloads as wl
from oracle import layer, placement, route, similarity, tables


def test_theta_endpoints():
    N = 32
    th = [tables.theta_layer(l, N, 0.5, 0.9) for l in range(1, N + 1)]
    assert th[0] == pytest.approx(0.9) and th[-1] == pytest.approx(0.5)
    assert all(a > b for a, b in zip(th, th[1:]))
    assert tables.theta_layer(1, 1, 0.5, 0.9) == pytest.approx(0.7)


def test_static_cost_closed_form():
    B = np.array([[1.0, 4.0], [4.0, 1.0]])
    tau = np.array([[0.0, 0.5], [0.5, 0.0]])
    F = np.array([2.0, 4.0])
    c = np.array([8.0, 8.0, 8.0])
    S = tables.static_cost(2, 3, 2.0, B, tau, c, F, dref=2.0, omega_T=0.5)
    # local: 0.5 * (8/F_m) / 2 ; remote adds 0.5 * (2/4 + 0.5) / 2
    assert S[0, 0, 1] == np.float32(1.0) and S[1, 1, 2] == np.float32(0.5)
    assert S[0, 1, 0] == np.float32(0.5 + 0.25) and S[1, 0, 0] == np.float32(1.0 + 0.25)


def _phi_tiny(H, pin=1):
    x2 = np.array([[1, 0], [0, 1]], dtype=np.uint8)
    P1 = np.array([[0.25, 0.75], [1.0, 0.0]])
    I2 = np.eye(2, dtype=np.float32)
    return tables.lookahead(H, [P1], [np.ones((2, 2), np.uint8), x2], [I2, I2],
                            [np.array([0, 1]), np.array([0, 1])], [0.7, 0.7], [1.0, 1.0],
                            np.ones((2, 2)), np.array([[0.0, 1.0], [1.0, 0.0]]),
                            [np.ones(2), np.ones(2)], np.array([1.0, 2.0]), [1.0, 1.0],
                            omega_T=1.0, omega_Q=0.0, Qbar=0.0, pin_local_exact=pin)


def test_lookahead_hand_example():
    # 2 layers, 2 servers; layer-2 expert 0 lives on server 0, expert 1 on
    # server 1; compute delay 1 on server 0, 0.5 on server 1; a move costs 2.
    # From server 0: next target 0 costs 1 (stay), target 1 costs 2 + 0.5.
    # From server 1: next target 0 costs 2 + 1, target 1 costs 0.5.
    phi = _phi_tiny(H=2)
    want = np.array([[0.25 * 1 + 0.75 * 2.5, 1.0 * 1],
                     [0.25 * 3 + 0.75 * 0.5, 1.0 * 3]])
    np.testing.assert_allclose(phi[0], want, rtol=1e-15)
    assert np.all(phi[1] == 0)


def test_lookahead_h1_is_zero():
    for p in _phi_tiny(H=1):
        assert np.all(p == 0)


def test_lookahead_all_local_closed_form():
    # every expert on every server and the pin rule: each future layer costs
    # the local compute delay, so Phi^{(h)}_l(m,k) = sum of the next
    # min(h, N-1-l) layers' omega_T c / (F_m d_ref) for observed rows.
    rng = np.random.default_rng(3)
    N, M, E, H = 5, 3, 4, 3
    x = [np.ones((M, E), np.uint8) for _ in range(N)]
    top1 = [rng.integers(0, E - 1, size=400) for _ in range(N)]  # expert E-1 never top-1
    P = tables.transitions(top1, [E] * N)
    F = np.array([1.0, 2.0, 5.0])
    c = [np.full(E, 3.0 + l) for l in range(N)]
    dref = [1.5] * N
    sims = [np.eye(E, dtype=np.float32)] * N
    g = [np.arange(E)] * N
    phi = tables.lookahead(H, P, x, sims, g, [0.7] * N, [1.0] * N, np.ones((M, M)),
                           np.ones((M, M)), c, F, dref, 0.5, 0.5, 0.25)
    for l in range(N):
        for m in range(M):
            for kk in range(E):
                if l == N - 1 or kk == E - 1:
                    assert phi[l][m, kk] == 0
                    continue
                want = sum(0.5 * c[l + j][0] / (F[m] * dref[l + j])
                           for j in range(1, min(H - 1, N - 1 - l) + 1))
                assert phi[l][m, kk] == pytest.approx(want, rel=1e-12)


def _textbook_moe(X, W, k, experts, shared):
    """Per-token dense top-k SwiGLU MoE with explicit vector operations."""
    T, d = X.shape
    y = np.zeros((T, d))
    for t in range(T):
        xt = X[t].astype(np.float64)
        lg = W.astype(np.float64) @ xt
        order = sorted(range(len(lg)), key=lambda e: (-lg[e], e))[:k]
        ex = np.exp(lg[order] - lg.max())
        gw = ex / ex.sum()
        for wgt, e in zip(gw, order):
            Wg, Wu, Wd = experts[e]
            h = Wg.astype(np.float64) @ xt
            u = Wu.astype(np.float64) @ xt
            y[t] += wgt * (Wd.astype(np.float64) @ (h / (1 + np.exp(-h)) * u))
        for Wg, Wu, Wd in shared:
            h = Wg.astype(np.float64) @ xt
            u = Wu.astype(np.float64) @ xt
            y[t] += Wd.astype(np.float64) @ (h / (1 + np.exp(-h)) * u)
    return y


@pytest.mark.parametrize("Qbar,allow", [(0.0, 1), (0.25, 0)])
def test_sum_over_servers_is_exact_moe_without_substitution(Qbar, allow):
    cfg = wl.C3.with_(T=40, d=32, f=24, E=10, clusters=2, cluster_size=5, n_shared=2,
                      M=3, capacity=(4.0, 4.0, 4.0), T_cal=512, Qbar=Qbar, k=3,
                      centre_std=32 ** -0.5)
    W = wl.router(cfg)
    model = similarity.build(wl.calibration(cfg), W, cfg.k, cfg.theta)
    x, _ = placement.place([model["group_of"]], [model["I"]], [np.ones(cfg.E)],
                           np.array(cfg.capacity), np.full(cfg.M, 1 / cfg.M))
    x = x[0]
    net = wl.network(cfg)
    c = np.full(cfg.E, 6.0 * cfg.d * cfg.f)
    S = tables.static_cost(cfg.M, cfg.E, 8.0 * cfg.d * 2, net.B, net.tau, c, net.F,
                           tables.d_ref(c, net.F), cfg.omega_T)
    X = wl.tokens(cfg)
    idx, w, _, _ = route.route(X, W, cfg.k)
    loc = wl.token_locations(cfg)
    o = layer.select(idx, x, model["sim"].astype(np.float32), model["group_of"], cfg.theta, S,
                     cfg.Qbar, cfg.omega_Q, loc, wl.accumulated_loss(cfg), 1, allow)
    experts = {e: wl.expert(cfg, e) for e in range(cfg.E)}
    shared = [wl.shared_expert(cfg, i) for i in range(cfg.n_shared)]
    total = sum(layer.server_output(X, w, o["exec_k"], o["exec_m"], loc, m,
                                    lambda e: experts[e], shared) for m in range(cfg.M))
    want = _textbook_moe(X, W, cfg.k, experts, shared)
    np.testing.assert_allclose(total, want, rtol=1e-10, atol=1e-13)
    # some slots really were remote, so the sum crosses servers
    assert np.any(o["cls"] >= 2)


def test_transitions_hand_example_and_dref():
    top1 = [np.array([0, 0, 0, 1, 2]), np.array([1, 1, 0, 1, 1])]
    P = tables.transitions(top1, [3, 2])
    np.testing.assert_allclose(P[0], [[1 / 3, 2 / 3], [0.0, 1.0], [0.0, 1.0]])
    assert len(P) == 1
    assert tables.d_ref(np.array([2.0, 4.0]), np.array([1.0, 3.0])) == pytest.approx(1.5)
