"""Oracle: expert similarity model and layer-aware grouping.  TEST INFRASTRUCTURE ONLY.

Section III-B and IV-A of the paper, Algorithm 1 steps for one layer:
  * routing-logit matrix H = W_r X_cal^T (eq 3), one row per expert;
  * Sim(i, j) = cosine of rows i and j of H (eq 4); a row of zero norm has
    Sim 0 to every other expert and 1 to itself (reading: eq 4 is undefined there);
  * activation counts n_j = number of (calibration token, top-k slot) pairs
    routed to j, with the same top-k rule as the router; f_j = n_j / sum n (eq 5);
  * greedy representative cover (eq 24-26): experts visited in decreasing
    activation frequency (ties: lower index); an expert becomes a new dominant
    expert when its largest similarity to the existing dominant experts is
    below theta (strict), otherwise it joins the most similar dominant expert
    (ties: the one made dominant first), using the dominant experts that exist
    at that moment;
  * representativeness rho_j = mean of Sim(j, k) over j's group, j included
    (eq 27); importance I_j = alpha_f f_j + alpha_r rho_j (eq 28).
fp64 throughout.
"""
from __future__ import annotations

import numpy as np

from .route import topk


def logit_matrix(X_cal: np.ndarray, W_r: np.ndarray) -> np.ndarray:
    """H [E, T_cal] in fp64 (eq 3)."""
    return np.asarray(W_r, dtype=np.float64) @ np.asarray(X_cal, dtype=np.float64).T


def cosine_similarity(H: np.ndarray) -> np.ndarray:
    """Sim [E, E] (eq 4)."""
    G = H @ H.T
    nrm = np.sqrt(np.diag(G))
    E = H.shape[0]
    S = np.zeros((E, E))
    for i in range(E):
        for j in range(E):
            if nrm[i] > 0 and nrm[j] > 0:
                S[i, j] = G[i, j] / (nrm[i] * nrm[j])
        S[i, i] = 1.0
    return S


def activation_counts(H: np.ndarray, k: int) -> np.ndarray:
    """n_j [E] int64: top-k slot counts over the calibration tokens."""
    idx, _ = topk(H.T, k)
    return np.bincount(idx.ravel(), minlength=H.shape[0]).astype(np.int64)


def group_experts(sim: np.ndarray, counts: np.ndarray, theta: float):
    """Greedy representative cover (eq 24-26).

    Returns (group_of [E] -> group index, centres) where group g is the g-th
    dominant expert created and centres[g] is that expert."""
    E = sim.shape[0]
    order = sorted(range(E), key=lambda j: (-int(counts[j]), j))
    centres = []
    group_of = np.full(E, -1, dtype=np.int32)
    for j in order:
        if not centres:
            best_c, best_s = None, -np.inf
        else:
            best_c, best_s = centres[0], sim[j, centres[0]]
            for c in centres[1:]:
                if sim[j, c] > best_s:
                    best_c, best_s = c, sim[j, c]
        if best_c is None or best_s < theta:
            centres.append(j)
            group_of[j] = len(centres) - 1
        else:
            group_of[j] = centres.index(best_c)
    return group_of, centres


def importance(sim: np.ndarray, counts: np.ndarray, group_of: np.ndarray, alpha_f: float):
    """(f [E], rho [E], I [E]) of eq 5, 27, 28."""
    E = sim.shape[0]
    tot = float(np.sum(counts))
    f = np.array([counts[j] / tot if tot > 0 else 0.0 for j in range(E)])
    rho = np.zeros(E)
    for j in range(E):
        members = [kk for kk in range(E) if group_of[kk] == group_of[j]]
        rho[j] = sum(sim[j, kk] for kk in members) / len(members)
    I = alpha_f * f + (1.0 - alpha_f) * rho
    return f, rho, I


def build(X_cal, W_r, k: int, theta: float, alpha_f: float = 0.5):
    """The whole per-layer offline model: dict with H-derived Sim, counts,
    groups, centres, f, rho and I."""
    H = logit_matrix(X_cal, W_r)
    sim = cosine_similarity(H)
    counts = activation_counts(H, k)
    group_of, centres = group_experts(sim, counts, theta)
    f, rho, I = importance(sim, counts, group_of, alpha_f)
    return dict(sim=sim, counts=counts, group_of=group_of, centres=centres, f=f, rho=rho, I=I)
