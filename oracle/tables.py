"""Oracle: per-layer decision tables of the online selection.  TEST INFRASTRUCTURE ONLY.

  * theta_l = theta_min + (theta_max - theta_min) (N - l) / (N - 1), l = 1..N
    (eq 6); a single layer (N = 1) takes the midpoint (reading: eq 6 divides by
    zero there);
  * feasible substitutes R_{l,r} = same-group experts k != r with
    Sim(r, k) >= theta_l (eq 7), compared in fp32;
  * substitution loss Q(r, k) = fp32((1 - Sim(r, k)) / 2) (eq 18, phi = identity);
  * per-step delay d(m, k | s) = 1[s != m] (z / B_{s,m} + tau_{s,m}) + c_k / F_m
    (eq 37) and the static part of the per-step cost (eq 38) plus the
    look-ahead cost-to-go, S[s][m][k] = omega_T d(m,k|s) / d_ref + Phi[m][k],
    evaluated in fp64 and rounded once to fp32.  The quality term of eq 38,
    omega_Q Q / Qbar, depends on the token and is added at run time;
  * d_ref = mean_k c_k / mean_m F_m (reading: the per-step delay of local exact
    execution on an average server);
  * look-ahead (eq 41-42), reading: transition probabilities P_l(k -> k')
    estimated from top-1 transitions between consecutive layers on calibration
    tokens, rows with no observation are all zero; the future candidate sets
    drop the budget test (the future budget is unknown) and keep the pin rule;
    Phi^{(0)} = 0 and the last layer's Phi = 0; the runtime uses Phi^{(H-1)};
  * weight adaptation (eq 45): omega_Q += kappa (Q_bar - T_bar), projected onto
    [0, 1], omega_T = 1 - omega_Q.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np


def theta_layer(l: int, N: int, theta_min: float = 0.5, theta_max: float = 0.9) -> float:
    """eq (6), 1-based layer index."""
    if N == 1:
        return 0.5 * (theta_min + theta_max)
    return theta_min + (theta_max - theta_min) * (N - l) / (N - 1)


def substitutes(sim32: np.ndarray, group_of: np.ndarray, theta: float, r: int):
    """R_{l,r} as a list of (k, Q(r,k)) in increasing expert index (eq 7, 18)."""
    E = sim32.shape[0]
    th = np.float32(theta)
    out = []
    for kk in range(E):
        if kk == r or group_of[kk] != group_of[r]:
            continue
        s = np.float32(sim32[r, kk])
        if s >= th:
            q = (np.float32(1.0) - s) * np.float32(0.5)
            out.append((kk, np.float32(q)))
    return out


def d_ref(c: np.ndarray, F: np.ndarray) -> float:
    return float(np.mean(c)) / float(np.mean(F))


def step_delay(s: int, m: int, kk: int, z: float, B: np.ndarray, tau: np.ndarray,
               c: np.ndarray, F: np.ndarray) -> float:
    """eq (37)."""
    trans = (z / B[s, m] + tau[s, m]) if s != m else 0.0
    return trans + c[kk] / F[m]


def static_cost(M: int, E: int, z: float, B, tau, c, F, dref: float, omega_T: float,
                phi: Optional[np.ndarray] = None) -> np.ndarray:
    """S [M][M][E] float32: omega_T d(m,k|s)/d_ref + Phi[m][k], rounded once."""
    S = np.zeros((M, M, E), dtype=np.float32)
    for s in range(M):
        for m in range(M):
            for kk in range(E):
                v = omega_T * step_delay(s, m, kk, z, B, tau, c, F) / dref
                if phi is not None:
                    v = v + float(phi[m, kk])
                S[s, m, kk] = np.float32(v)
    return S


def transitions(top1: Sequence[np.ndarray], E: Sequence[int]) -> List[np.ndarray]:
    """P_l [E_l, E_{l+1}] from per-layer top-1 experts of the same calibration
    tokens (eq 41); the last layer gets no matrix."""
    P = []
    for l in range(len(top1) - 1):
        n = np.zeros((E[l], E[l + 1]))
        for a, b in zip(top1[l], top1[l + 1]):
            n[int(a), int(b)] += 1
        tot = n.sum(axis=1, keepdims=True)
        P.append(np.divide(n, tot, out=np.zeros_like(n), where=tot > 0))
    return P


def lookahead(H: int, P: Sequence[np.ndarray], x: Sequence[np.ndarray],
              sim32: Sequence[np.ndarray], group_of: Sequence[np.ndarray],
              theta: Sequence[float], z: Sequence[float], B, tau,
              c: Sequence[np.ndarray], F, dref: Sequence[float],
              omega_T: float, omega_Q: float, Qbar: float,
              pin_local_exact: int = 1, allow_sub: int = 1) -> List[np.ndarray]:
    """Phi_l^{(H-1)} [M, E_l] for every layer l (eq 42), fp64.

    Phi_l^{(h)}(m, k) = sum_{k'} P_l(k -> k') * min over the budget-free
    candidates (m', k'') of target k' at layer l+1 of
    [ g_{l+1}(m', k'' | s = m) + Phi_{l+1}^{(h-1)}(m', k'') ]."""
    N = len(x)
    M = x[0].shape[0]
    Qbar = float(np.float32(Qbar))   # the runtime budget is an fp32 quantity

    def g_next(l1, s, m1, k1, r1):
        q = 0.0
        if k1 != r1:
            q = float((np.float32(1.0) - np.float32(sim32[l1][r1, k1])) * np.float32(0.5))
        val = omega_T * step_delay(s, m1, k1, z[l1], B, tau, c[l1], F) / dref[l1]
        if Qbar > 0:
            val += omega_Q * q / Qbar
        return val

    subs_memo = {}

    def candidates(l1, s, r1):
        if pin_local_exact and x[l1][s, r1]:
            return [(s, r1)]
        ks = [r1]
        if allow_sub and Qbar > 0:
            if (l1, r1) not in subs_memo:
                subs_memo[(l1, r1)] = [kk for kk, _ in substitutes(sim32[l1], group_of[l1], theta[l1], r1)]
            ks += subs_memo[(l1, r1)]
        # allow_sub = 2: substitutes only on the source server (exact targets anywhere)
        return [(m1, k1) for k1 in ks for m1 in range(M) if x[l1][m1, k1]
                and not (allow_sub == 2 and k1 != r1 and m1 != s)]

    memo = {}

    def phi(l, h):
        key = (l, h)
        if key in memo:
            return memo[key]
        E_l = x[l].shape[1]
        out = np.zeros((M, E_l))
        if h > 0 and l + 1 < N:
            nxt = phi(l + 1, h - 1)
            E1 = x[l + 1].shape[1]
            # V[m, k'] = best next-layer cost from source m for next target k'
            V = np.zeros((M, E1))
            for m in range(M):
                for r1 in range(E1):
                    best = None
                    for (m1, k1) in candidates(l + 1, m, r1):
                        v = g_next(l + 1, m, m1, k1, r1) + nxt[m1, k1]
                        if best is None or v < best:
                            best = v
                    V[m, r1] = 0.0 if best is None else best
            # out[m, k] = sum over r1 of P[k, r1] V[m, r1], added in increasing r1
            # (elementwise over (m, k), so every entry is the plain sequential sum)
            for r1 in range(E1):
                out += V[:, r1][:, None] * P[l][:, r1][None, :]
        memo[key] = out
        return out

    return [phi(l, H - 1) for l in range(N)]


def adapt_weights(omega_Q: float, kappa: float, T_bar: float, Q_bar: float):
    """Section V-D, eq 45: omega_Q moves by kappa (Q_bar - T_bar), projected
    onto [0, 1]; omega_T = 1 - omega_Q.  Returns (omega_Q, omega_T)."""
    w = omega_Q + kappa * (Q_bar - T_bar)
    w = min(1.0, max(0.0, w))
    return w, 1.0 - w
