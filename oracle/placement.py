"""Oracle: importance-aware expert deployment (Algorithm 1, second and third
parts; Section IV-B and IV-C).  TEST INFRASTRUCTURE ONLY.

Mandatory placement, per layer:
  * experts in non-increasing memory demand p (ties: lower index);
  * memory-feasible servers F = {m : b_m + p <= C_m} (eq 29);
  * Score(m) = lambda1 * b_m / C_m + lambda2 * eta_m, eta_m = number of the
    expert's group already on m in this layer (eq 30); the expert goes to the
    feasible server of least score (eq 31), ties to the lower server index;
  * an expert with F empty waits; after the layer the waiting experts go to
    the server with the largest remaining memory C_m - b_m (ties: lower index).
  b_m (used memory) accumulates over all layers.

Redundant placement, over all layers (eq 32-35), greedy:
  * y_{m,l,g} = 1 when server m already holds an expert of group g of layer l;
  * benefit B(m,l,j) = pi_m I_j (1 - y_{m,l,g(j)}) / p_j (eq 33) for candidates
    with x = 0 that fit the remaining memory;
  * repeatedly deploy the candidate of largest positive benefit (ties: lower
    (l, m, j)), update y and b, until none is left.
Reading of eq 32: the sum runs over the experts k of group g(j) in layer l.

Baselines of Section VI-A (readings; the paper names them without giving
their procedure):
  * Popularity-based Replication (`redundancy=2`): the redundant part above
    with benefit pi_m w_j / p_j, i.e. without the group-coverage factor;
    the caller passes activation frequencies as w.
  * Random Deployment (`place_random`): each expert once, layer by layer in
    index order, on a server drawn uniformly from the memory-feasible ones
    (none feasible: the most remaining memory, ties to the lower index);
    then every (l, m, j) without a copy, in a Fisher-Yates-shuffled order,
    is placed if it fits.  Draws come from SplitMix64 (Steele, Lea and
    Flood, OOPSLA 2014), a uniform integer below n being next() % n.
fp64 throughout.  The benefit of every candidate is evaluated elementwise with
numpy (same operations and order per candidate as the formula above); the
layers are padded to a common expert count with zero-importance entries,
which never have a positive benefit.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np


class CapacityError(ValueError):
    pass


def place(group_of: Sequence[np.ndarray], importance: Sequence[np.ndarray],
          p: Sequence[np.ndarray], C: np.ndarray, pi: np.ndarray,
          lambda1: float = 0.5, redundancy=True):
    """Returns (x: list over layers of [M, E_l] uint8, b [M] used memory).
    redundancy: False/0 none, True/1 eq 33, 2 popularity (no (1 - y) factor)."""
    N = len(group_of)
    M = len(C)
    lambda2 = 1.0 - lambda1
    tot_p = sum(float(np.sum(pl)) for pl in p)
    if tot_p > float(np.sum(C)):
        raise CapacityError("total expert memory exceeds the servers' capacity")
    b = np.zeros(M)
    x: List[np.ndarray] = [np.zeros((M, len(g)), dtype=np.uint8) for g in group_of]

    for l in range(N):
        g = group_of[l]
        E = len(g)
        order = sorted(range(E), key=lambda j: (-float(p[l][j]), j))
        waiting = []
        for j in order:
            best_m, best_score = -1, None
            same_group = np.asarray(g) == g[j]
            for m in range(M):
                if not (b[m] + p[l][j] <= C[m]):
                    continue
                eta = int(np.sum(x[l][m, same_group]))
                score = lambda1 * b[m] / C[m] + lambda2 * eta
                if best_score is None or score < best_score:
                    best_m, best_score = m, score
            if best_m < 0:
                waiting.append(j)
            else:
                x[l][best_m, j] = 1
                b[best_m] += p[l][j]
        for j in waiting:
            best_m = max(range(M), key=lambda m: (C[m] - b[m], -m))
            x[l][best_m, j] = 1
            b[best_m] += p[l][j]

    if redundancy:
        Emax = max(len(gl) for gl in group_of)
        G = np.zeros((N, Emax), dtype=np.int64)          # group ids (padding: own group)
        I = np.zeros((N, Emax))                          # importance (padding: 0)
        P = np.ones((N, Emax))                           # memory demand (padding: 1)
        X = np.ones((N, M, Emax), dtype=np.uint8)        # deployment (padding: held)
        for l in range(N):
            E = len(group_of[l])
            G[l, :E] = np.asarray(group_of[l])
            G[l, E:] = G[l, :E].max(initial=-1) + 1 + np.arange(Emax - E)
            I[l, :E] = importance[l]
            P[l, :E] = p[l]
            X[l, :, :E] = x[l]
        pim = np.asarray(pi, dtype=np.float64)
        same = G[:, :, None] == G[:, None, :]                          # [l, j, k]
        # y[l, m, j] = 1 when server m holds some expert of j's group in layer l
        y = np.zeros((N, M, Emax), dtype=np.int64)
        for l in range(N):
            for m in range(M):
                for kk in np.nonzero(X[l, m])[0]:
                    y[l, m, same[l, kk]] = 1
        while True:
            if redundancy == 2:
                Bnf = pim[None, :, None] * I[:, None, :] / P[:, None, :] * np.ones_like(y)
            else:
                Bnf = pim[None, :, None] * I[:, None, :] * (1 - y) / P[:, None, :]
            fits = (b[None, :, None] + P[:, None, :]) <= np.asarray(C)[None, :, None]
            cand = (X == 0) & fits & (Bnf > 0)
            if not cand.any():
                break
            Bm = np.where(cand, Bnf, -np.inf)
            flat = int(np.argmax(Bm))           # first maximum: lowest (l, m, j)
            l, m, j = np.unravel_index(flat, Bm.shape)
            X[l, m, j] = 1
            y[l, m, same[l, j]] = 1
            x[l][m, j] = 1
            b[m] += p[l][j]
    return x, b


MASK64 = (1 << 64) - 1


class SplitMix64:
    """SplitMix64 from its published definition: add the golden-ratio
    increment 0x9E3779B97F4A7C15 to the state, then mix the state with
    xor-shift 30 / multiply 0xBF58476D1CE4E5B9 / xor-shift 27 / multiply
    0x94D049BB133111EB / xor-shift 31, all modulo 2^64."""

    def __init__(self, seed: int):
        self.state = seed & MASK64

    def next(self) -> int:
        self.state = (self.state + 0x9E3779B97F4A7C15) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)

    def below(self, n: int) -> int:
        return self.next() % n


def place_random(p: Sequence[np.ndarray], C: np.ndarray, seed: int, redundancy: bool = True):
    """Random Deployment baseline (Section VI-A; reading in the module
    header).  Returns (x: list over layers of [M, E_l] uint8, b [M])."""
    N = len(p)
    M = len(C)
    if sum(float(np.sum(pl)) for pl in p) > float(np.sum(C)):
        raise CapacityError("total expert memory exceeds the servers' capacity")
    rng = SplitMix64(seed)
    b = np.zeros(M)
    x: List[np.ndarray] = [np.zeros((M, len(pl)), dtype=np.uint8) for pl in p]
    for l in range(N):
        for j in range(len(p[l])):
            feasible = [m for m in range(M) if b[m] + p[l][j] <= C[m]]
            if feasible:
                m = feasible[rng.below(len(feasible))]
            else:
                m = max(range(M), key=lambda q: (C[q] - b[q], -q))
            x[l][m, j] = 1
            b[m] += p[l][j]
    if redundancy:
        cand = [(l, m, j) for l in range(N) for m in range(M) for j in range(len(p[l]))
                if x[l][m, j] == 0]
        for i in range(len(cand) - 1, 0, -1):        # Fisher-Yates, from the end
            r = rng.below(i + 1)
            cand[i], cand[r] = cand[r], cand[i]
        for (l, m, j) in cand:
            if b[m] + p[l][j] <= C[m]:
                x[l][m, j] = 1
                b[m] += p[l][j]
    return x, b
