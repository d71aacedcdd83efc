"""Pins of the delay / workload / traffic oracle (eq 13-17, eq 22) and the
library's simulator against it, CPU only."""
import numpy as np
import pytest

from oracle import delay

# two servers: link 0-1 of 2 Gbit/s and 5 ms, compute 10 and 40 TFLOP/s
B2 = np.array([[1e10, 2e9], [2e9, 1e10]])
TAU2 = np.array([[0.0, 5e-3], [5e-3, 0.0]])
F2 = np.array([10e12, 40e12])


def test_hand_traced_trajectory():
    # one token from server 0, two layers, top-1: layer 0 on server 1 (eq 13
    # transfer from the access server), layer 1 on server 1 again (eq 14: no
    # transfer), then 1 expert of each layer's 2 with c = (2e9, 4e9) FLOP
    z = [8e6, 8e6]
    c = [np.array([2e9, 4e9]), np.array([2e9, 4e9])]
    em = np.array([[[1]], [[1]]], np.uint8)
    ek = np.array([[[1]], [[0]]], np.int32)
    r = delay.simulate(np.array([0]), em, ek, c, z, B2, TAU2, F2)
    want = (8e6 / 2e9 + 5e-3) + 4e9 / 40e12 + 2e9 / 40e12      # 4 ms + 5 ms + 0.1 ms + 0.05 ms
    assert r["delay"][0] == pytest.approx(want, rel=1e-15)
    assert r["delay"][0] == pytest.approx(9.15e-3, rel=1e-12)
    assert r["loc"].tolist() == [[0], [1]]
    assert r["transfers"] == 1 and r["remote_slots"] == 1 and r["slots"] == 2
    assert r["traffic_bytes"] == 1e6
    np.testing.assert_array_equal(r["work"], [0.0, 6e9])


def test_top2_slots_pay_their_own_transfer_and_share_one_message():
    # top-2 at one layer: both slots on the remote server 1 -> two eq-14 delays
    # (each slot is one decision) but one transfer of the representation
    c = [np.array([1e9, 1e9, 1e9])]
    em = np.array([[[1, 1]]], np.uint8)
    ek = np.array([[[0, 2]]], np.int32)
    r = delay.simulate(np.array([0]), em, ek, c, [1.6e6], B2, TAU2, F2)
    assert r["delay"][0] == pytest.approx(2 * (1.6e6 / 2e9 + 5e-3) + 2 * 1e9 / 40e12, rel=1e-15)
    assert r["transfers"] == 1 and r["remote_slots"] == 2 and r["traffic_bytes"] == 2e5


def test_all_local_is_pure_compute():
    rng = np.random.default_rng(0)
    N, T, k, M = 4, 9, 3, 5
    E = [6, 7, 5, 6]
    c = [rng.uniform(1e9, 5e9, e) for e in E]
    F = rng.uniform(20e12, 110e12, M)
    loc0 = rng.integers(0, M, T).astype(np.uint8)
    em = np.repeat(loc0[None, :, None], N, axis=0).repeat(k, axis=2)
    ek = np.stack([rng.integers(0, E[l], (T, k)) for l in range(N)]).astype(np.int32)
    Bm = rng.uniform(1e9, 1e10, (M, M))
    r = delay.simulate(loc0, em, ek, c, [1e6] * N, Bm, np.full((M, M), 1e-3), F)
    want = np.array([sum(c[l][ek[l, t, j]] / F[loc0[t]] for l in range(N) for j in range(k)) for t in range(T)])
    np.testing.assert_allclose(r["delay"], want, rtol=1e-13)
    assert r["transfers"] == 0 and r["remote_slots"] == 0 and r["traffic_bytes"] == 0
    # eq 22: every server's workload is the FLOP of the slots it ran; the total is every slot's FLOP
    assert r["work"].sum() == pytest.approx(sum(c[l][ek[l]].sum() for l in range(N)), rel=1e-13)


def test_token_follows_slot_zero_and_invalid_locations_stay():
    c = [np.ones(2) * 1e9] * 3
    em = np.array([[[1, 0], [2, 2]], [[0, 0], [2, 2]], [[2, 1], [2, 2]]], np.uint8)
    ek = np.zeros((3, 2, 2), np.int32)
    B3 = np.full((3, 3), 1e9)
    r = delay.simulate(np.array([0, 7]), em, ek, c, [1e6] * 3, B3, np.zeros((3, 3)), np.ones(3) * 1e12)
    # token 0: 0 -> 1 (slot 0 of layer 0) -> 0 -> 2; token 1 is not on a server: nothing runs
    assert r["loc"][:, 0].tolist() == [0, 1, 0] and r["loc"][:, 1].tolist() == [7, 7, 7]
    assert r["delay"][1] == 0.0 and r["slots"] == 6
    # layer 0: slot 0 remote (1); layer 1 from server 1: both slots remote on 0; layer 2 from 0: 2 and 1
    assert r["remote_slots"] == 1 + 2 + 2 and r["transfers"] == 1 + 1 + 2


def test_library_simulator_matches_the_oracle_bit_for_bit():
    from paper_2607_17154_amd import ordermoe as om
    rng = np.random.default_rng(7)
    for trial in range(12):
        N, T, k, M = int(rng.integers(1, 6)), int(rng.integers(0, 40)), int(rng.integers(1, 9)), int(rng.integers(1, 9))
        E = [int(rng.integers(1, 20)) for _ in range(N)]
        c = [rng.uniform(1e8, 1e10, e) for e in E]
        Bm = rng.uniform(1e9, 1e10, (M, M))
        tau = rng.uniform(2e-4, 2e-2, (M, M))
        F = rng.uniform(20e12, 110e12, M)
        z = rng.uniform(1e4, 1e6, N)
        loc0 = rng.integers(0, M + 2, T).astype(np.uint8)          # some tokens off the servers
        em = rng.integers(0, M, (N, T, k)).astype(np.uint8)
        em[rng.random((N, T, k)) < 0.05] = 255
        ek = np.stack([rng.integers(0, E[l], (T, k)) for l in range(N)]).astype(np.int32).reshape(N, T, k)
        want = delay.simulate(loc0, em, ek, c, z, Bm, tau, F)
        got = om.ordermoe_simulate_delay(loc0, em, ek, c, z, Bm, tau, F)
        np.testing.assert_array_equal(got["delay"], want["delay"])
        np.testing.assert_array_equal(got["work"], want["work"])
        np.testing.assert_array_equal(got["loc"].astype(np.int64), want["loc"])
        for n in ("transfers", "traffic_bytes", "remote_slots", "slots"):
            assert got[n] == want[n], n


def test_library_simulator_rejects_bad_input():
    from paper_2607_17154_amd import ordermoe as om
    c = [np.ones(2)]
    em = np.zeros((1, 1, 1), np.uint8)
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_simulate_delay([0], em, np.array([[[2]]], np.int32), c, [1.0], B2, TAU2, F2)
    assert ei.value.code == om.EINVAL
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_simulate_delay([0], em, np.zeros((1, 1, 1), np.int32), c, [1.0], B2, TAU2, [0.0, 1.0])
    assert ei.value.code == om.EINVAL
