"""Pins of the oracle's router, similarity model and grouping (CPU only).

Each check is against something other than the oracle itself: a brute-force
loop, a closed form, a hand-traced example or a statistical limit."""
import math

import numpy as np
import pytest

import workloads as wl
from oracle import route, similarity


def _brute_topk(row, k):
    # repeated arg-max with ties to the lower index (textbook selection)
    left = list(range(len(row)))
    out = []
    for _ in range(k):
        best = left[0]
        for j in left[1:]:
            if row[j] > row[best]:
                best = j
        out.append(best)
        left.remove(best)
    return out


def test_topk_matches_selection_with_ties():
    rng = np.random.default_rng(5)
    L = rng.integers(-3, 4, size=(200, 9)).astype(np.float64)  # many exact ties
    for k in (1, 2, 4, 9):
        idx, srt = route.topk(L, k)
        for t in range(L.shape[0]):
            assert list(idx[t]) == _brute_topk(L[t], k)


def test_margin_hand_example():
    L = np.array([[3.0, 1.0, 2.5, 2.4, -1.0]])
    idx, srt = route.topk(L, 2)        # top-3 sorted: 3.0, 2.5, 2.4
    assert list(idx[0]) == [0, 2]
    assert route.margin(srt)[0] == pytest.approx(0.1)
    idx, srt = route.topk(L, 5)        # k = E: gaps among all five
    assert route.margin(srt)[0] == pytest.approx(0.1)


def test_gate_is_softmax():
    rng = np.random.default_rng(1)
    L = rng.standard_normal((50, 8))
    idx, _ = route.topk(L, 3)
    p = np.exp(L) / np.exp(L).sum(axis=1, keepdims=True)
    w0 = route.gate(L, idx, renorm=0)
    w1 = route.gate(L, idx, renorm=1)
    for t in range(50):
        sel = p[t, idx[t]]
        np.testing.assert_allclose(w0[t], sel, rtol=1e-12)
        np.testing.assert_allclose(w1[t], sel / sel.sum(), rtol=1e-12)


def test_cosine_brute_force_and_zero_row():
    rng = np.random.default_rng(2)
    H = rng.standard_normal((5, 11))
    H[3] = 0.0
    S = similarity.cosine_similarity(H)
    for i in range(5):
        for j in range(5):
            if i == j:
                assert S[i, j] == 1.0
            elif i == 3 or j == 3:
                assert S[i, j] == 0.0
            else:
                num = sum(H[i, t] * H[j, t] for t in range(11))
                den = math.sqrt(sum(v * v for v in H[i])) * math.sqrt(sum(v * v for v in H[j]))
                assert S[i, j] == pytest.approx(num / den, abs=1e-14)
    assert np.array_equal(S, S.T)


def test_cosine_limit_for_gaussian_calibration():
    # For X ~ N(0, I), E[H_i . H_j] / T = w_i . w_j, so Sim -> cos(w_i, w_j)
    # with fluctuations of order 1/sqrt(T).
    rng = np.random.default_rng(3)
    d, E, T = 32, 6, 200000
    W = rng.standard_normal((E, d))
    X = rng.standard_normal((T, d))
    S = similarity.cosine_similarity(similarity.logit_matrix(X, W))
    nw = np.linalg.norm(W, axis=1)
    C = (W @ W.T) / np.outer(nw, nw)
    assert np.max(np.abs(S - C)) < 6.0 / math.sqrt(T)


def test_counts_sum_and_frequency():
    rng = np.random.default_rng(4)
    H = rng.standard_normal((7, 300))
    n = similarity.activation_counts(H, 3)
    assert n.sum() == 300 * 3
    f, rho, I = similarity.importance(np.eye(7), n, np.arange(7), 0.5)
    assert f.sum() == pytest.approx(1.0)
    # singleton groups: rho = Sim(j, j) = 1
    np.testing.assert_allclose(rho, 1.0)
    np.testing.assert_allclose(I, 0.5 * f + 0.5)


def test_grouping_hand_example():
    # 4 experts; activation order 2, 0, 3, 1 (counts), theta 0.6.
    # 2 -> first centre (group 0). 0: Sim(0,2)=0.2 < 0.6 -> centre (group 1).
    # 3: Sim(3,2)=0.7, Sim(3,0)=0.65 -> group of 2 (group 0).
    # 1: Sim(1,2)=0.6, Sim(1,0)=0.6 -> not below theta; tie -> earlier centre 2.
    S = np.array([[1.0, 0.6, 0.2, 0.65],
                  [0.6, 1.0, 0.6, 0.1],
                  [0.2, 0.6, 1.0, 0.7],
                  [0.65, 0.1, 0.7, 1.0]])
    counts = np.array([30, 5, 40, 10])
    g, centres = similarity.group_experts(S, counts, 0.6)
    assert centres == [2, 0]
    assert list(g) == [1, 0, 0, 0]
    # strictness of eq 24: at theta = 0.7 expert 3 (Sim 0.7 to centre 2) joins
    g, centres = similarity.group_experts(S, counts, 0.7)
    assert centres[:2] == [2, 0] and g[3] == 0
    # rho (eq 27): mean over the group including the expert itself
    f, rho, I = similarity.importance(S, counts, np.array([1, 0, 0, 0]), 0.5)
    assert rho[2] == pytest.approx((0.6 + 1.0 + 0.7) / 3)
    assert rho[0] == pytest.approx(1.0)


@pytest.mark.parametrize("theta", [0.5, 0.7, 0.9])
def test_planted_clusters_recovered(theta):
    cfg = wl.C1
    W = wl.router(cfg)
    Xc = wl.calibration(cfg)
    m = similarity.build(Xc, W, cfg.k, theta)
    assert len(m["centres"]) == cfg.clusters
    planted = np.arange(cfg.E) // cfg.cluster_size
    for a in range(cfg.E):
        for b in range(cfg.E):
            assert (m["group_of"][a] == m["group_of"][b]) == (planted[a] == planted[b])


def test_bf16_rounding_of_generator():
    a = np.array([1.0, 1.00390625, 1.005859375, -2.0009765625, 3.0e-3], dtype=np.float32)
    r = wl.round_to_bf16(a)
    # bf16 keeps 8 significant bits: the spacing just above 1 is 2^-7
    assert r[0] == 1.0
    assert r[1] == 1.0          # 1 + 2^-8 is a tie -> even (1.0)
    assert r[2] == np.float32(1.0078125)  # 1 + 1.5 * 2^-8 rounds up
    assert r[3] == -2.0
    assert abs(r[4] - 3.0e-3) <= 3.0e-3 * 2 ** -8


def test_counts_brute_force():
    rng = np.random.default_rng(8)
    H = rng.integers(-2, 3, size=(6, 90)).astype(np.float64)   # ties present
    n = similarity.activation_counts(H, 2)
    want = np.zeros(6, dtype=np.int64)
    for t in range(90):
        for e in _brute_topk(H[:, t], 2):
            want[e] += 1
    assert np.array_equal(n, want)
