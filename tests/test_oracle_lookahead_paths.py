"""Pins of the oracle's look-ahead cost-to-go (Section V-C, eq 41-43), CPU only.

Three checks that do not reuse the oracle's recursion:

* hand-traced two-layer stacks whose next-layer minimum is a budget-free
  substitute (so the quality term omega_Q * Q / Qbar of eq 38 decides the
  value), or where dropping the pin on the local exact expert lets a remote
  exact copy win;
* a literal expansion of eq 42 on tiny random stacks (E <= 6, M <= 3, N <= 4,
  H <= 3): every future target path k -> k' -> k'' ... is expanded with its
  transition probabilities, the candidate sets are built here from eq 7, the
  deployment and the selection mode, and no partial result is cached;
* the reading of Property 3 (part 2): Phi^(h)(m, k) equals the expected cost
  actually paid over the next h layers when, along every future target
  sequence weighted by its probability, each layer picks the candidate that
  minimises its per-step cost plus the remaining look-ahead -- evaluated by
  walking the explicit sequences and adding the per-step costs of eq 37-38.
"""
import itertools

import numpy as np
import pytest

from oracle import tables


# ------------------------------------------------------------ eq 37-38 and eq 7, written out here
def _q(sim32, r, k):
    """eq 18 with phi = identity, in fp32: Q(r, k) = (1 - Sim(r, k)) / 2; 0 for the target itself."""
    if k == r:
        return 0.0
    return float((np.float32(1.0) - np.float32(sim32[r, k])) * np.float32(0.5))


def _g(inst, l, s, m, k, r):
    """Per-step cost of executing target r of layer l by expert k on server m,
    the token coming from server s: omega_T * d / d_ref + omega_Q * Q / Qbar."""
    move = 0.0 if s == m else inst["z"][l] / inst["B"][s][m] + inst["tau"][s][m]
    d = move + inst["c"][l][k] / inst["F"][m]
    v = inst["omega_T"] * d / inst["dref"][l]
    Qbar = float(np.float32(inst["Qbar"]))
    if Qbar > 0:
        v += inst["omega_Q"] * _q(inst["sim"][l], r, k) / Qbar
    return v


def _cands(inst, l, s, r):
    """Budget-free candidate set of target r at layer l for a token on server s."""
    memo = inst.setdefault("_cands", {})
    if (l, s, r) not in memo:
        memo[(l, s, r)] = _cand_list(inst, l, s, r)
    return memo[(l, s, r)]


def _cand_list(inst, l, s, r):
    x = inst["x"][l]
    M = x.shape[0]
    if inst["pin"] and x[s][r]:
        return [(s, r)]
    out = [(m, r) for m in range(M) if x[m][r]]
    if inst["allow_sub"] and float(np.float32(inst["Qbar"])) > 0:
        sim, grp, th = inst["sim"][l], inst["group"][l], np.float32(inst["theta"][l])
        for k in range(x.shape[1]):
            if k == r or grp[k] != grp[r] or not np.float32(sim[r, k]) >= th:
                continue
            for m in range(M):
                if x[m][k] and (inst["allow_sub"] != 2 or m == s):
                    out.append((m, k))
    return out


def _phi_paths(inst, l, m, k, h):
    """eq 42 expanded literally: sum over next targets of P times the minimum
    over that target's candidates of (per-step cost + the same expansion one
    layer further with one step less).  No caching."""
    N = len(inst["x"])
    if h == 0 or l + 1 >= N:
        return 0.0
    P = inst["P"][l]
    tot = 0.0
    for r1 in range(P.shape[1]):
        p = P[k, r1]
        best = None
        for (m1, k1) in _cands(inst, l + 1, m, r1):
            v = _g(inst, l + 1, m, m1, k1, r1) + _phi_paths(inst, l + 1, m1, k1, h - 1)
            best = v if best is None or v < best else best
        tot += p * (0.0 if best is None else best)
    return tot


def _oracle_phi(inst, H):
    return tables.lookahead(H, inst["P"], inst["x"], inst["sim"], inst["group"], inst["theta"], inst["z"],
                            inst["B"], inst["tau"], inst["c"], inst["F"], inst["dref"], inst["omega_T"],
                            inst["omega_Q"], inst["Qbar"], pin_local_exact=inst["pin"],
                            allow_sub=inst["allow_sub"])


# ------------------------------------------------------------ hand-traced stacks
def _two_layer(F, move, x2, P, sim, Qbar, pin=1, allow_sub=1, omega_Q=1.0):
    """Two layers, two servers, two experts per layer in one similarity group;
    z / B is half of a move and tau the other half; c = 1; d_ref = 1; omega_T = 1."""
    M = 2
    x1 = np.ones((M, 2), np.uint8)
    S = np.array([[1.0, sim], [sim, 1.0]], np.float32)
    return dict(x=[x1, np.array(x2, np.uint8)], P=[np.array(P, float)], sim=[S, S],
                group=[np.zeros(2, int), np.zeros(2, int)], theta=[0.7, 0.7], z=[1.0, 1.0],
                B=np.array([[1.0, 2.0 / move], [2.0 / move, 1.0]]),
                tau=np.array([[0.0, move / 2], [move / 2, 0.0]]),
                c=[np.ones(2), np.ones(2)], F=np.array(F, float), dref=[1.0, 1.0],
                omega_T=1.0, omega_Q=omega_Q, Qbar=Qbar, pin=pin, allow_sub=allow_sub)


# Layer-2 expert 0 lives on server 1 only, expert 1 on server 0 only; both
# servers compute an expert in 1; a move costs 2; Sim(0, 1) = 0.75, so a
# substitute costs Q = 0.125.  Next-layer targets: from expert 0 half and
# half, from expert 1 a quarter to expert 0.
HAND_P = [[0.5, 0.5], [0.25, 0.75]]
HAND_X2 = [[0, 1], [1, 0]]


@pytest.mark.parametrize("Qbar,allow_sub,V_sub", [
    # Qbar = 0.5: the substitute costs 1 + 0.125 / 0.5 = 1.25 < 3, the remote exact
    (0.5, 1, 1.25),
    # Local Substitute Only: the substitute sits on the token's server, same value
    (0.5, 2, 1.25),
    # Qbar = 1/32: the substitute costs 1 + 4 = 5 > 3, so the remote exact wins
    (1.0 / 32, 1, 3.0),
    # no substitution: only the remote exact copy
    (0.5, 0, 3.0),
    # Qbar = 0: the quality term and the substitutes are off
    (0.0, 1, 3.0),
])
def test_hand_traced_substitute_is_the_future_minimum(Qbar, allow_sub, V_sub):
    inst = _two_layer([1.0, 1.0], 2.0, HAND_X2, HAND_P, 0.75, Qbar, allow_sub=allow_sub)
    # V[s][r']: next-layer cost of target r' from server s.  The target held by
    # the token's own server is pinned (cost 1); the other one is V_sub.
    V = [[V_sub, 1.0], [1.0, V_sub]]
    want = np.array([[HAND_P[k][0] * V[m][0] + HAND_P[k][1] * V[m][1] for k in range(2)] for m in range(2)])
    phi = _oracle_phi(inst, H=2)
    np.testing.assert_allclose(phi[0], want, rtol=1e-15, atol=0)
    assert np.all(phi[1] == 0)
    # spelled out for the default case
    if Qbar == 0.5 and allow_sub == 1:
        np.testing.assert_allclose(phi[0], [[1.125, 1.0625], [1.125, 1.1875]], rtol=1e-15)


@pytest.mark.parametrize("pin,want0", [(1, 1.0), (0, 0.75)])
def test_hand_traced_pin_rule(pin, want0):
    # no substitution; layer-2 expert 0 on both servers, expert 1 on server 0;
    # server 0 computes in 1, server 1 in 0.25; a move costs 0.5; every token
    # targets expert 0 next.  From server 0 the pinned local copy costs 1, the
    # copy on server 1 costs 0.5 + 0.25 = 0.75; from server 1 the local copy
    # (0.25) is cheapest either way.
    inst = _two_layer([1.0, 4.0], 0.5, [[1, 1], [1, 0]], [[1.0, 0.0], [1.0, 0.0]], 0.75, 0.5,
                      pin=pin, allow_sub=0)
    phi = _oracle_phi(inst, H=2)
    np.testing.assert_allclose(phi[0], [[want0, want0], [0.25, 0.25]], rtol=1e-15)


def test_hand_traced_three_layers_carry_the_chosen_server():
    # three layers of the first hand stack; layer 3 equals layer 2.  At H = 3 the
    # layer-2 step from server s, target r', adds the layer-3 look-ahead of the
    # pair it chose: Phi_1(m', k') is the H = 2 value of the two-layer stack.
    inst = _two_layer([1.0, 1.0], 2.0, HAND_X2, HAND_P, 0.75, 0.5)
    for key in ("x", "sim", "group", "theta", "z", "c", "dref"):
        inst[key] = inst[key] + [inst[key][-1]]
    inst["P"] = inst["P"] + [inst["P"][0]]
    inst["x"][1] = inst["x"][2] = np.array(HAND_X2, np.uint8)
    phi1 = np.array([[1.125, 1.0625], [1.125, 1.1875]])     # Phi_1^(1)(m, k), as above
    # from server s, target r': candidates (pinned local exact, or remote exact /
    # substitute on s) with their per-step cost, then + Phi_1^(1) of the pair
    def V(s, r):
        if HAND_X2[s][r]:
            return 1.0 + phi1[s, r]
        exact = 3.0 + phi1[1 - s, r]
        sub = 1.25 + phi1[s, 1 - r]
        return min(exact, sub)
    want = np.array([[sum(HAND_P[k][r] * V(m, r) for r in range(2)) for k in range(2)] for m in range(2)])
    phi = _oracle_phi(inst, H=3)
    np.testing.assert_allclose(phi[0], want, rtol=1e-15)
    np.testing.assert_allclose(phi[1], phi1, rtol=1e-15)
    assert np.all(phi[2] == 0)
    # the substitute, not the remote exact copy, is the minimum from server 0 for target 0
    assert 1.25 + phi1[0, 1] < 3.0 + phi1[1, 0]


# ------------------------------------------------------------ tiny random stacks
def _random_stack(rng, N, M, E, Qbar, pin, allow_sub):
    x = []
    for _ in range(N):
        xl = (rng.random((M, E)) < 0.45).astype(np.uint8)
        for j in range(E):                                    # every expert somewhere (eq 2)
            if not xl[:, j].any():
                xl[rng.integers(M), j] = 1
        x.append(xl)
    group = [rng.integers(0, 2, size=E) for _ in range(N)]
    sim = []
    for l in range(N):
        S = rng.uniform(0.5, 1.0, size=(E, E)).astype(np.float32)
        S = np.minimum(S, S.T)
        np.fill_diagonal(S, 1.0)
        S[0, 1] = S[1, 0] = np.float32(0.7)                   # on the threshold: feasible (eq 7 inclusive)
        sim.append(S)
    P = []
    for _ in range(N - 1):
        p = rng.random((E, E)) * (rng.random((E, E)) < 0.6)
        p[rng.integers(E)] = 0.0                              # an unseen row: zero
        tot = p.sum(axis=1, keepdims=True)
        P.append(np.divide(p, tot, out=np.zeros_like(p), where=tot > 0))
    B = rng.uniform(1.0, 4.0, size=(M, M))
    B = (B + B.T) / 2
    tau = rng.uniform(0.0, 1.0, size=(M, M))
    tau = (tau + tau.T) / 2
    np.fill_diagonal(tau, 0.0)
    return dict(x=x, P=P, sim=sim, group=group, theta=[0.7] * N, z=list(rng.uniform(0.5, 2.0, size=N)),
                B=B, tau=tau, c=[rng.uniform(0.5, 2.0, size=E) for _ in range(N)],
                F=rng.uniform(0.5, 2.0, size=M), dref=list(rng.uniform(0.5, 1.5, size=N)),
                omega_T=0.5, omega_Q=0.5, Qbar=Qbar, pin=pin, allow_sub=allow_sub)


COMBOS = [(pin, sub, Qbar) for pin in (0, 1) for sub in (0, 1, 2) for Qbar in (0.0, 0.3)]


@pytest.mark.parametrize("pin,allow_sub,Qbar", COMBOS)
def test_oracle_equals_the_literal_path_expansion(pin, allow_sub, Qbar):
    rng = np.random.default_rng(100 * pin + 10 * allow_sub + int(Qbar * 10))
    for trial in range(4):
        N, M, E = int(rng.integers(2, 5)), int(rng.integers(2, 4)), int(rng.integers(3, 7))
        inst = _random_stack(rng, N, M, E, Qbar, pin, allow_sub)
        for H in (1, 2, 3):
            phi = _oracle_phi(inst, H)
            for l in range(N):
                want = np.array([[_phi_paths(inst, l, m, k, H - 1) for k in range(E)] for m in range(M)])
                np.testing.assert_allclose(phi[l], want, rtol=1e-12, atol=0,
                                           err_msg="trial %d H %d layer %d" % (trial, H, l))
            if H > 1 and N > 1:
                assert np.any(phi[0] > 0)


def _walk(inst, l, m, k, h, phis, prefix):
    """Follow one explicit prefix of future targets from (m, k) at layer l: at
    each layer the token takes the candidate minimising its per-step cost plus
    the oracle's look-ahead of the remaining depth (first in the candidate
    order on ties).  Returns the prefix's probability and the per-step cost
    paid at its last layer."""
    prob, s, kk, cost = 1.0, m, k, 0.0
    for j, r in enumerate(prefix):
        prob *= inst["P"][l + j][kk, r]
        if prob == 0.0:
            return 0.0, 0.0
        rest = h - 1 - j                                    # look-ahead depth left after this step
        best, arg = None, None
        for (m1, k1) in _cands(inst, l + 1 + j, s, r):
            v = _g(inst, l + 1 + j, s, m1, k1, r) + (phis[rest][l + 1 + j][m1, k1] if rest > 0 else 0.0)
            if best is None or v < best:
                best, arg = v, (m1, k1)
        cost = _g(inst, l + 1 + j, s, arg[0], arg[1], r)
        s, kk = arg
    return prob, cost


def _realized_cost(inst, l, m, k, h, phis):
    """Expected per-step cost paid over the next h layers after executing k on
    server m at layer l: every explicit prefix of future targets (k', then k'',
    ...) of length 1..h, weighted by its probability, adds the per-step cost
    paid at its last layer."""
    N = len(inst["x"])
    total = 0.0
    for j in range(min(h, N - 1 - l)):
        for prefix in itertools.product(*[range(inst["P"][l + i].shape[1]) for i in range(j + 1)]):
            prob, cost = _walk(inst, l, m, k, h, phis, prefix)
            total += prob * cost
    return total


@pytest.mark.parametrize("pin,allow_sub", [(1, 1), (0, 1), (1, 2), (0, 0)])
def test_phi_is_the_expected_cost_of_the_trajectory_it_induces(pin, allow_sub):
    rng = np.random.default_rng(7 + 3 * pin + allow_sub)
    for trial in range(3):
        N, M, E = 4, int(rng.integers(2, 4)), int(rng.integers(3, 6))
        inst = _random_stack(rng, N, M, E, 0.3, pin, allow_sub)
        # Phi^(h) for every depth h = 0..2 (oracle horizon H = h + 1)
        phis = {h: _oracle_phi(inst, h + 1) for h in range(3)}
        for h in (1, 2):
            for l in range(N - 1):
                for m in range(M):
                    for k in range(E):
                        want = _realized_cost(inst, l, m, k, h, phis)
                        assert phis[h][l][m, k] == pytest.approx(want, rel=1e-12, abs=1e-15), \
                            (trial, h, l, m, k)


def test_substitute_sets_follow_eq7():
    """R_{l,r}: same group, not r itself, Sim >= theta (inclusive, fp32), with
    Q = fp32((1 - Sim) / 2), listed in increasing expert index."""
    S = np.array([[1.0, 0.7, 0.9, 0.95, 0.69999],
                  [0.7, 1.0, 0.8, 0.8, 0.8],
                  [0.9, 0.8, 1.0, 0.8, 0.8],
                  [0.95, 0.8, 0.8, 1.0, 0.8],
                  [0.69999, 0.8, 0.8, 0.8, 1.0]], np.float32)
    group = np.array([0, 0, 0, 1, 0])
    subs = tables.substitutes(S, group, 0.7, 0)
    assert [k for k, _ in subs] == [1, 2]                   # 3: other group; 4: below theta
    assert subs[0][1] == np.float32((np.float32(1.0) - np.float32(0.7)) * np.float32(0.5))
    assert float(subs[1][1]) == 0.050000011920928955          # fp32 of (1 - 0.9f) / 2: 0.100000024 / 2
    assert tables.substitutes(S, group, 0.7, 3) == []        # alone in its group
    assert [k for k, _ in tables.substitutes(S, group, 0.8, 1)] == [2, 4]
