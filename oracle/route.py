"""Oracle: router logits, gate and top-k of one MoE layer.  TEST INFRASTRUCTURE ONLY.

The router is replicated on every server and runs where the token resides
(Section III-C); its logits for one token are the runtime form of eq (3):
l_e = sum_i x_i W_r[e, i].  The paper does not describe the gate itself, so
the readings are: top-k by logit with ties to the lower expert index; the gate
weight of a selected expert is the softmax probability renormalised over the
top-k (renorm = 1) or over all experts (renorm = 0); the "logit margin" of a
token is the smallest gap between adjacent sorted logits among its top-(k+1)
(top-k when k = E).  Everything is computed in fp64 from the exact input values.
"""
from __future__ import annotations

import numpy as np

MARGIN_FLAG = 1e-4


def router_logits(X: np.ndarray, W_r: np.ndarray) -> np.ndarray:
    """[T, E] fp64 logits, eq (3) per token."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(W_r, dtype=np.float64).T


def topk(logits: np.ndarray, k: int):
    """Top-k expert indices [T, k] in rank order (descending logit, ties to the
    lower index) and the sorted logits [T, min(k+1, E)]."""
    order = np.argsort(-logits, axis=1, kind="stable")
    kk = min(k + 1, logits.shape[1])
    srt = np.take_along_axis(logits, order[:, :kk], axis=1)
    return order[:, :k].astype(np.int32), srt


def margin(sorted_logits: np.ndarray) -> np.ndarray:
    """Smallest adjacent gap among the sorted top logits, per token."""
    if sorted_logits.shape[1] < 2:
        return np.full(sorted_logits.shape[0], np.inf)
    return np.min(sorted_logits[:, :-1] - sorted_logits[:, 1:], axis=1)


def gate(logits: np.ndarray, idx: np.ndarray, renorm: int = 1) -> np.ndarray:
    """Gate weights [T, k] of the selected experts (fp64)."""
    mx = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - mx)
    sel = np.take_along_axis(p, idx.astype(np.int64), axis=1)
    den = sel.sum(axis=1, keepdims=True) if renorm else p.sum(axis=1, keepdims=True)
    return sel / den


def route(X: np.ndarray, W_r: np.ndarray, k: int, renorm: int = 1):
    """Returns (idx [T,k] int32, w [T,k] fp64, margin [T] fp64, logits [T,E] fp64)."""
    L = router_logits(X, W_r)
    idx, srt = topk(L, k)
    return idx, gate(L, idx, renorm), margin(srt), L
