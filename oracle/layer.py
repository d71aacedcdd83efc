"""Oracle: selection, dispatch list and one server's MoE-layer output.
TEST INFRASTRUCTURE ONLY.

  * select(): Algorithm 2's per-token decision for one layer (eq 36-44), in
    the plain-C routine oracle/select.c;
  * dispatch(): every slot whose execution server differs from the token's
    location needs the token representation (z_l bytes) sent there (eq 13-14);
    the list is ordered by (destination, token, slot) and the number of
    distinct (token, destination) pairs counts the transfers;
  * server_output(): the output that server m0 produces for each token:
    y[q] = sum over slots s executed on m0 of w_s * FFN_{k*_s}(x_q), plus, for
    tokens residing on m0, the sum of the always-local shared experts (weight
    1); FFN(x) = W_down (silu(W_gate x) * (W_up x)), silu(a) = a / (1 + e^-a).
    The sum is taken slot by slot in fp64 (no merging of repeated experts).
"""
from __future__ import annotations

import ctypes
from typing import Callable, Dict, Optional, Sequence

import numpy as np

from ._clib import lib

CLS_NAMES = ("local_exact", "local_sub", "remote_exact", "remote_sub")


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def select(idx: np.ndarray, x: np.ndarray, sim32: np.ndarray, group_of: np.ndarray,
           theta: float, S: np.ndarray, Qbar: float, omega_Q: float,
           loc_in: np.ndarray, qhat_in: np.ndarray, pin_local_exact: int = 1,
           allow_sub: int = 1) -> Dict[str, np.ndarray]:
    T, k = idx.shape
    M, E = x.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    x = np.ascontiguousarray(x, dtype=np.uint8)
    sim32 = np.ascontiguousarray(sim32, dtype=np.float32)
    group_of = np.ascontiguousarray(group_of, dtype=np.int32)
    S = np.ascontiguousarray(S, dtype=np.float32)
    loc_in = np.ascontiguousarray(loc_in, dtype=np.uint8)
    qhat_in = np.ascontiguousarray(qhat_in, dtype=np.float32)
    out = dict(exec_k=np.empty((T, k), np.int32), exec_m=np.empty((T, k), np.uint8),
               cls=np.empty((T, k), np.uint8), qhat_out=np.empty(T, np.float32),
               loc_out=np.empty(T, np.uint8))
    rc = lib().orc_select(T, k, E, M, _p(idx), _p(x), _p(sim32), _p(group_of),
                          ctypes.c_float(theta), _p(S), ctypes.c_float(Qbar),
                          ctypes.c_float(omega_Q), pin_local_exact, allow_sub,
                          _p(loc_in), _p(qhat_in), _p(out["exec_k"]), _p(out["exec_m"]),
                          _p(out["cls"]), _p(out["qhat_out"]), _p(out["loc_out"]))
    if rc != 0:
        raise ValueError("oracle selection failed (rc=%d): a target expert is deployed nowhere" % rc)
    return out


def dispatch(exec_m: np.ndarray, loc_in: np.ndarray, M: int):
    """Remote slots ordered by (destination, token, slot) as q*k+s codes, the
    per-destination counts and the number of distinct (token, destination)."""
    T, k = exec_m.shape
    entries = []
    pairs = set()
    for q in range(T):
        for s in range(k):
            m = int(exec_m[q, s])
            if m != int(loc_in[q]):
                entries.append((m, q, s))
                pairs.add((q, m))
    entries.sort()
    lst = np.array([q * k + s for (_, q, s) in entries], dtype=np.int32)
    cnt = np.zeros(M, dtype=np.int32)
    for (m, _, _) in entries:
        cnt[m] += 1
    return lst, cnt, len(pairs)


def class_counts(cls: np.ndarray) -> np.ndarray:
    return np.array([int(np.sum(cls == c)) for c in range(4)], dtype=np.int64)


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def ffn(xrows: np.ndarray, Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray) -> np.ndarray:
    """SwiGLU expert FFN applied to rows [R, d] in fp64 (torch Linear layouts)."""
    xr = np.asarray(xrows, dtype=np.float64)
    h = xr @ np.asarray(Wg, dtype=np.float64).T
    u = xr @ np.asarray(Wu, dtype=np.float64).T
    return (silu(h) * u) @ np.asarray(Wd, dtype=np.float64).T


def server_output(X: np.ndarray, w: np.ndarray, exec_k: np.ndarray, exec_m: np.ndarray,
                  loc_in: np.ndarray, server: int, expert_weights: Callable[[int], tuple],
                  shared_weights: Sequence[tuple] = (), tokens: Optional[np.ndarray] = None
                  ) -> np.ndarray:
    """y [len(tokens), d] fp64 for the given tokens (all tokens by default).

    expert_weights(j) returns (W_gate, W_up, W_down) of routed expert j."""
    T, k = exec_k.shape
    tok = np.arange(T) if tokens is None else np.asarray(tokens)
    d = X.shape[1]
    y = np.zeros((len(tok), d))
    for e in sorted({int(exec_k[q, s]) for q in tok for s in range(k) if exec_m[q, s] == server}):
        Wg, Wu, Wd = expert_weights(e)
        for s in range(k):
            sel = [i for i, q in enumerate(tok) if exec_m[q, s] == server and exec_k[q, s] == e]
            if not sel:
                continue
            rows = tok[sel]
            y[sel] += np.asarray(w[rows, s], dtype=np.float64)[:, None] * ffn(X[rows], Wg, Wu, Wd)
    res = [i for i, q in enumerate(tok) if int(loc_in[q]) == server]
    if res:
        for (Wg, Wu, Wd) in shared_weights:
            y[res] += ffn(X[tok[res]], Wg, Wu, Wd)
    return y
