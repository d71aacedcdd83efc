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
                                  "placement_redundancy.json"])
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
