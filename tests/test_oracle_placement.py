"""Pins of the oracle's deployment (Algorithm 1, eq 29-35), CPU only."""
import json
import os

import numpy as np
import pytest

from oracle import placement

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


@pytest.mark.parametrize("case", ["placement_4groups_2servers.json",
                                  "placement_4groups_4servers.json",
                                  "placement_waiting_list.json",
                                  "placement_redundancy.json",
                                  "placement_popularity.json"])
def test_hand_traced_placements(case):
    g = _load(case)
    group_of = [np.array(v) for v in g["group_of"]]
    imp = [np.array(v, dtype=float) for v in g["importance"]]
    p = [np.array(v, dtype=float) for v in g["p"]]
    x, b = placement.place(group_of, imp, p, np.array(g["C"], dtype=float),
                           np.array(g["pi"], dtype=float), g["lambda1"], g["redundancy"])
    for l, want in enumerate(g["servers_of_expert"]):
        got = [sorted(int(m) for m in np.nonzero(x[l][:, j])[0]) for j in range(len(want))]
        assert got == want, (case, l)
    np.testing.assert_allclose(b, g["used"])


def test_constraints_c1_c3_random():
    rng = np.random.default_rng(0)
    for trial in range(30):
        N = int(rng.integers(1, 4))
        M = int(rng.integers(2, 6))
        E = [int(rng.integers(3, 12)) for _ in range(N)]
        group_of = [rng.integers(0, 4, size=e) for e in E]
        imp = [rng.random(e) for e in E]
        p = [np.ones(e) for e in E]   # unit memory: no fragmentation
        need = int(sum(pl.sum() for pl in p))
        C = rng.integers(1, need + 1, size=M).astype(float)
        while C.sum() < need:
            C[int(rng.integers(0, M))] += 1.0
        x, b = placement.place(group_of, imp, p, C, np.full(M, 1.0 / M), 0.5, True)
        for l in range(N):
            assert np.all(x[l].sum(axis=0) >= 1)               # c.2
            assert set(np.unique(x[l])) <= {0, 1}              # c.3
        used = np.zeros(M)
        for l in range(N):
            used += (x[l] * p[l][None, :]).sum(axis=1)
        np.testing.assert_allclose(used, b)
        assert np.all(b <= C + 1e-9)                           # c.1


def test_capacity_error():
    with pytest.raises(placement.CapacityError):
        placement.place([np.array([0, 0, 1])], [np.ones(3)], [np.ones(3)],
                        np.array([1.0, 1.0]), np.array([0.5, 0.5]))


def test_redundancy_stops_when_all_groups_covered():
    # 2 groups of 2 on 2 servers with room for 4 each: after the mandatory
    # part every server covers both groups, so no replica has positive benefit.
    x, b = placement.place([np.array([0, 0, 1, 1])], [np.ones(4)], [np.ones(4)],
                           np.array([4.0, 4.0]), np.array([0.5, 0.5]), 0.5, True)
    assert x[0].sum() == 4


def test_popularity_equals_eq33_when_every_group_is_one_expert():
    # with singleton groups y(m, l, g(j)) = x(m, l, j) = 0 for every candidate,
    # so the group-coverage factor of eq 33 is 1 and both rules coincide
    rng = np.random.default_rng(3)
    for trial in range(10):
        M, E = int(rng.integers(2, 6)), int(rng.integers(4, 12))
        w = [rng.random(E), rng.random(E)]
        p = [np.ones(E), np.ones(E)]
        C = np.full(M, float(int(2 * E * 1.6 / M) + 1))
        pi = rng.random(M)
        singles = [np.arange(E), np.arange(E)]
        xa, ba = placement.place(singles, w, p, C, pi, 0.5, True)
        xb, bb = placement.place(singles, w, p, C, pi, 0.5, 2)
        for l in range(2):
            np.testing.assert_array_equal(xa[l], xb[l])
        np.testing.assert_array_equal(ba, bb)


def test_popularity_fills_memory_with_the_most_popular_missing_experts():
    # one layer, equal pi, unit memory: each server's replicas are the most
    # popular experts it lacks, and every server ends full
    rng = np.random.default_rng(4)
    E, M = 16, 4
    w = rng.random(E)
    g = rng.integers(0, 4, size=E)
    C = np.full(M, 6.0)
    x0, _ = placement.place([g], [w], [np.ones(E)], C, np.full(M, 0.25), 0.5, False)
    x, b = placement.place([g], [w], [np.ones(E)], C, np.full(M, 0.25), 0.5, 2)
    np.testing.assert_array_equal(b, C)
    for m in range(M):
        added = np.nonzero(x[0][m] & ~x0[0][m])[0]
        missing = np.nonzero(x0[0][m] == 0)[0]
        top = missing[np.argsort(-w[missing], kind="stable")][:len(added)]
        assert sorted(added.tolist()) == sorted(top.tolist())


def test_splitmix64_published_outputs():
    # the first outputs of SplitMix64 for seeds 0 and 1234567, as published
    # with the generator's reference implementation
    r = placement.SplitMix64(0)
    assert [r.next() for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                           0x06C45D188009454F]
    r = placement.SplitMix64(1234567)
    assert [r.next() for _ in range(3)] == [6457827717110365317, 3203168211198807973,
                                           9817491932198370423]


def test_random_deployment_constraints_and_determinism():
    rng = np.random.default_rng(6)
    for trial in range(20):
        N, M = int(rng.integers(1, 4)), int(rng.integers(2, 7))
        p = [rng.integers(1, 3, size=int(rng.integers(3, 12))).astype(float) for _ in range(N)]
        need = sum(v.sum() for v in p)
        C = np.full(M, float(np.ceil(need * 1.5 / M)) + 2)
        for red in (False, True):
            x, b = placement.place_random(p, C, seed=trial, redundancy=red)
            used = np.zeros(M)
            for l in range(N):
                assert np.all(x[l].sum(axis=0) >= 1)           # c.2
                assert set(np.unique(x[l])) <= {0, 1}          # c.3
                used += (x[l] * p[l][None, :]).sum(axis=1)
            np.testing.assert_array_equal(used, b)
            assert np.all(b <= C)                              # c.1 (room to spare)
            if red:
                # nothing more fits: every missing (l, m, j) is larger than m's free memory
                for l in range(N):
                    for m in range(M):
                        for j in np.nonzero(x[l][m] == 0)[0]:
                            assert b[m] + p[l][j] > C[m]
            x2, b2 = placement.place_random(p, C, seed=trial, redundancy=red)
            for l in range(N):
                np.testing.assert_array_equal(x[l], x2[l])


def test_random_deployment_spreads_uniformly():
    # no memory pressure: the mandatory server of each expert is uniform over
    # the M servers (chi-square over 4000 experts, 3 degrees of freedom; the
    # 99.99% quantile is 21.1)
    M, E = 4, 4000
    x, _ = placement.place_random([np.ones(E)], np.full(M, float(E)), seed=99, redundancy=False)
    counts = x[0].sum(axis=1)
    chi2 = float(((counts - E / M) ** 2 / (E / M)).sum())
    assert chi2 < 21.1
    # and the first server drawn is feasible[next() % M] with next() the first output
    r = placement.SplitMix64(99)
    assert x[0][r.next() % M, 0] == 1


def test_random_deployment_capacity_error():
    with pytest.raises(placement.CapacityError):
        placement.place_random([np.ones(3)], np.array([1.0, 1.0]), seed=0)
