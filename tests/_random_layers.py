"""Seeded random layer configurations over the C ABI's parameter space, for
the GPU parity sweep (tests/test_gpu_random_layers.py).  Holds no arithmetic
of the method: it only draws LayerConfig fields."""
import math

import numpy as np

import workloads as wl

N_RANDOM = 30


def random_layer(i: int) -> wl.LayerConfig:
    rng = np.random.default_rng(7919 * (i + 1))
    pick = lambda xs: xs[int(rng.integers(0, len(xs)))]
    f32 = i % 6 == 5
    if f32:
        d, f = pick([128, 192, 256, 512]), pick([96, 160, 256, 512])
    else:
        d, f = pick([256, 512, 768, 1024]), pick([128, 256, 384, 640])
    if i == 0:
        clusters, size = 1, 1                                  # one expert
    elif i == 1:
        clusters, size = 16, 16                                # 256 experts
    else:
        clusters, size = int(rng.integers(1, 17)), int(rng.integers(1, 9))
    E = clusters * size
    k = int(rng.integers(1, min(E, 8) + 1))
    M = 1 if i == 2 else (32 if i == 1 else int(rng.integers(1, 33)))
    M = max(M, math.ceil(E / 64))                              # at most 64 experts per server
    cap = min(64, math.ceil(E / M) + int(rng.integers(0, 3)))
    return wl.LayerConfig(
        name="random%02d_%s_d%d_E%d_f%d_top%d_M%d" % (i, "f32" if f32 else "bf16", d, E, f, k, M),
        dtype="f32" if f32 else "bf16", seed=500 + i,
        T=pick([1, 7, 64, 128, 129, 333, 1000, 2049]), d=d, E=E, f=f, k=k,
        n_shared=int(rng.integers(0, 2 if f32 else 5)),
        clusters=clusters, cluster_size=size, sigma=pick([0.1, 0.3, 0.5]),
        centre_std=pick([1.0, 4.0]) * d ** -0.5, M=M, m0=int(rng.integers(0, M)),
        capacity=tuple(float(cap) for _ in range(M)), loc_mode=pick(["zero", "uniform"]),
        Qbar=pick([0.0, 0.1, 0.25, 1.0]), theta=pick([0.5, 0.7, 0.9]), T_cal=2048,
        renorm=int(rng.integers(0, 2)), pin_local_exact=int(rng.integers(0, 2)),
        allow_sub=int(rng.integers(0, 3)))


def qhat_scale(i: int) -> float:
    return 0.2 if i % 3 == 1 else 0.0
