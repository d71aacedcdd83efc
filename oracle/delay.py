"""Oracle: delay, server workload and traffic of realized decisions
(Section III-C/D, eq 13-17; Section III-F, eq 22).  TEST INFRASTRUCTURE ONLY.

The paper's model has one execution server per token and layer.  Readings for
top-k, where every slot is one decision:
  * every executed slot pays eq 15's compute c_k / F_m on its server m and,
    when m differs from the token's location s before the layer, the transfer
    of eq 13 (first layer, s = the access server) or eq 14 (later layers),
    z_l / B_{s,m} + tau_{s,m};
  * after layer l the token resides on slot 0's execution server; the return
    path is not modelled;
  * a token whose location is not a server (>= M) executes nothing at that
    layer and keeps its location, and so does a slot whose server is >= M;
  * traffic: the token representation travels once to every distinct remote
    server of a layer, z_l / 8 bytes each;
  * eq 22 workload of server m: the sum of c_k over the slots it executes.
Per-user delays (eq 17) are sums of per-token delays over the user's tokens.

fp64 throughout, plain loops in the order token, layer, slot (delays) and
layer, token, slot (workload and counts).
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np


def simulate(loc0: np.ndarray, exec_m: np.ndarray, exec_k: np.ndarray, c: Sequence[np.ndarray],
             z_bits: Sequence[float], B: np.ndarray, tau: np.ndarray, F: np.ndarray) -> Dict:
    """loc0 [T] access servers; exec_m, exec_k [N][T][k] decisions per layer;
    c[l] [E_l] FLOP per expert; z_bits [N]; B, tau [M][M]; F [M].
    Returns delay [T] (s), work [M] (FLOP), loc [N][T] (location before each
    layer), transfers, traffic_bytes, remote_slots, slots."""
    N, T, k = exec_m.shape
    M = len(F)
    loc = np.zeros((N, T), dtype=np.int64)
    s = [int(v) for v in loc0]
    for l in range(N):
        for t in range(T):
            loc[l, t] = s[t]
            if s[t] < M and exec_m[l, t, 0] < M:
                s[t] = int(exec_m[l, t, 0])
    delay = np.zeros(T)
    for t in range(T):
        d = 0.0
        for l in range(N):
            src = int(loc[l, t])
            if src >= M:
                continue
            for j in range(k):
                m = int(exec_m[l, t, j])
                if m >= M:
                    continue
                if m != src:
                    d += float(z_bits[l]) / float(B[src, m]) + float(tau[src, m])    # eq 13 / 14
                d += float(c[l][int(exec_k[l, t, j])]) / float(F[m])               # eq 15
        delay[t] = d                                                               # eq 16-17
    work = np.zeros(M)
    transfers = remote = slots = 0
    traffic = 0.0
    for l in range(N):
        for t in range(T):
            src = int(loc[l, t])
            if src >= M:
                continue
            dests = set()
            for j in range(k):
                m = int(exec_m[l, t, j])
                if m >= M:
                    continue
                slots += 1
                work[m] += float(c[l][int(exec_k[l, t, j])])                        # eq 22
                if m != src:
                    remote += 1
                    dests.add(m)
            transfers += len(dests)
            traffic += len(dests) * (float(z_bits[l]) / 8.0)
    return dict(delay=delay, work=work, loc=loc, transfers=transfers, traffic_bytes=traffic,
                remote_slots=remote, slots=slots)
