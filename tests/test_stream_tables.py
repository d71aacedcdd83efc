"""The offline model of the 32-layer decode stack (128 experts, top-8, 8
servers, memory ratio 2.0, H = 3): the oracle's construction against what the
paper fixes, and the library's host tables (eq 6, 41, 42, 7, 37-38) against
the oracle's, bit for bit."""
import numpy as np
import pytest

import workloads as wl
from oracle import tables


def test_thresholds_follow_eq6(stream_case):
    sc = stream_case
    th = np.array(sc.theta)
    # eq 6: theta_1 = theta_max, theta_N = theta_min, linear in between
    assert th[0] == 0.9 and th[-1] == 0.5
    np.testing.assert_allclose(np.diff(th), -(0.4 / 31), rtol=1e-12)


def test_planted_clusters_are_recovered_at_every_threshold(stream_case):
    # 32 planted clusters of 4 experts; the greedy cover returns them for every theta_l
    cls = wl.stream_clusters(wl.C5_STREAM)
    for l, m in enumerate(stream_case.models):
        g, cl = m["group_of"], cls[l]
        assert len(set(g.tolist())) == 32
        for c in range(32):
            assert len(set(g[cl == c].tolist())) == 1


def test_deployment_constraints(stream_case):
    sc, cfg = stream_case, stream_case.cfg
    used = np.zeros(cfg.M)
    for l in range(cfg.N):
        x = sc.x_dep[l]
        assert np.all(x.sum(axis=0) >= 1)            # c.1: every expert deployed
        used += x.sum(axis=1)
        # the replicas complete group coverage: each server covers all 32 groups
        g = sc.models[l]["group_of"]
        for m in range(cfg.M):
            assert len(set(g[x[m] == 1].tolist())) == 32
    assert np.all(used <= np.array(cfg.capacity))    # c.2: memory per server
    assert used.sum() == cfg.memory_ratio * cfg.N * cfg.E


def test_transitions_are_distributions_with_cluster_persistence(stream_case):
    sc = stream_case
    cls = wl.stream_clusters(wl.C5_STREAM)
    for l, P in enumerate(sc.P):
        # P_l maps layer-l experts to layer-(l+1) experts: same planted cluster index
        same = cls[l][:, None] == cls[l + 1][None, :]
        s = P.sum(axis=1)
        assert np.all((np.abs(s - 1) < 1e-12) | (s == 0))
        assert np.all(P >= 0)
        # the AR chains keep a token's top-1 expert in its cluster far above the
        # 4/128 a memoryless stream would give
        rows = s > 0
        assert (P[rows] * same[rows]).sum() / rows.sum() > 0.15


def test_lookahead_is_zero_at_the_last_layer_and_bounded(stream_case):
    sc = stream_case
    assert np.all(sc.phi[-1] == 0)
    # Phi_l^(H-1) sums H-1 future per-step costs of at most the worst candidate
    assert np.all(sc.phi[0] >= 0)


def test_library_tables_match_the_oracle_bit_for_bit(stream_case):
    from tests._pipeline import stream_library_tables
    sc = stream_case
    theta32, phi, tabs = stream_library_tables(sc)
    for l in range(sc.cfg.N):
        assert np.float32(sc.theta[l]) == theta32[l]
        np.testing.assert_array_equal(phi[l], sc.phi[l])
        np.testing.assert_array_equal(tabs[l]["S"].view(np.uint32), sc.S[l].view(np.uint32))
        # substitutes (eq 7) with their loss (eq 18), in (Q, k) order
        for r in range(sc.cfg.E):
            want = sorted(((float(q), k) for k, q in
                           tables.substitutes(sc.sim32[l], sc.models[l]["group_of"], sc.theta[l], r)))
            n = int(tabs[l]["t1_n"][r])
            got = [(float(tabs[l]["t1_q"][r, i]), int(tabs[l]["t1_k"][r, i])) for i in range(n)]
            assert got == want
        srv = np.zeros(sc.cfg.E, np.uint32)
        for m in range(sc.cfg.M):
            srv |= (sc.x_dep[l][m].astype(np.uint32) << np.uint32(m))
        np.testing.assert_array_equal(tabs[l]["srvmask"], srv)


def test_library_transition_estimate_matches_the_oracle():
    from paper_2607_17154_amd import ordermoe as om
    rng = np.random.default_rng(5)
    top1 = rng.integers(0, 12, size=(4, 500)).astype(np.int32)
    top1[1, :50] = 3                      # a row with many observations
    top1[:, 7] = 11
    P = om.ordermoe_estimate_transitions(top1, 12)
    want = tables.transitions([top1[l] for l in range(4)], [12] * 4)
    for l in range(3):
        np.testing.assert_array_equal(P[l], want[l])
    # rows of experts never seen as top-1 are zero
    top1b = np.zeros((2, 10), np.int32)
    Pb = om.ordermoe_estimate_transitions(top1b, 3)
    np.testing.assert_array_equal(Pb[0], [[1, 0, 0], [0, 0, 0], [0, 0, 0]])


def test_library_theta_layer():
    from paper_2607_17154_amd import ordermoe as om
    for N in (1, 2, 5, 32):
        for l in range(1, N + 1):
            assert om.ordermoe_theta_layer(l, N, 0.5, 0.9) == np.float32(tables.theta_layer(l, N, 0.5, 0.9))


@pytest.mark.parametrize("H", [1, 2, 5])
def test_library_lookahead_matches_the_oracle_at_every_horizon(stream_case, H):
    """The look-ahead sweep of Fig. 7 (H = 1 .. 5): the library's Phi (eq 42) and
    cost tables equal the oracle's bit for bit at each depth; H = 1 is the
    myopic rule (Phi = 0)."""
    from tests._pipeline import stream_library_tables, with_horizon
    sc = with_horizon(stream_case, H)
    _, phi, tabs = stream_library_tables(sc)
    for l in range(sc.cfg.N):
        np.testing.assert_array_equal(phi[l], sc.phi[l])
        np.testing.assert_array_equal(tabs[l]["S"].view(np.uint32), sc.S[l].view(np.uint32))
    if H == 1:
        assert all(np.all(p == 0) for p in phi)
    else:
        assert any(np.any(p > 0) for p in phi)


def test_library_lookahead_matches_the_oracle_with_local_substitutes_only(stream_case):
    """The Local Substitute Only mode (allow_sub = 2): the future candidate sets
    keep substitutes on the source server only; library and oracle agree bit
    for bit."""
    from tests._pipeline import stream_library_tables, with_horizon
    sc = with_horizon(stream_case, 3, allow_sub=2)
    _, phi, tabs = stream_library_tables(sc)
    for l in range(sc.cfg.N):
        np.testing.assert_array_equal(phi[l], sc.phi[l])
        np.testing.assert_array_equal(tabs[l]["S"].view(np.uint32), sc.S[l].view(np.uint32))
    # fewer future candidates can only raise each minimum
    ref = with_horizon(stream_case, 3)
    for l in range(sc.cfg.N):
        assert np.all(phi[l] >= ref.phi[l])
