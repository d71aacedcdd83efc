"""Seeded synthetic workloads for one OrderMoE MoE layer.

This module holds only random draws, the rounding of those draws to the run's
storage type, and the constants that describe each workload.  None of the
method's arithmetic lives here: the HIP library (through its binding) and the
CPU oracle both receive these arrays as plain inputs, and neither imports the
other.

Sizes and value distributions follow the five layer shapes the method is
evaluated on (Section VI-A: Switch/Qwen/Mixtral-class MoE layers, H = 3,
theta in [0.5, 0.9], memory ratio 2.0) and the testbed ranges of Section VI-A
for the synthetic network tables (bandwidth 1-10 Gbit/s, latency 0.2-20 ms,
compute 20-110 TFLOP/s).  Trained weights and the paper's datasets are not
used; every tensor is drawn here.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Optional, Tuple

import numpy as np

# sub-stream identifiers: each tensor has its own SeedSequence so that drawing
# one expert's weights never depends on having drawn another's.
_S_CENTRES, _S_NOISE, _S_X, _S_XCAL, _S_WG, _S_WU, _S_WD = 1, 2, 3, 4, 5, 6, 7
_S_SHARED, _S_LOC, _S_NET, _S_QHAT = 8, 9, 1000, 11
_S_PERM = 12


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even).

    Returns float32 values that are exactly representable in bfloat16.
    Inputs are finite draws from normal distributions (no NaN handling)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    r = (u + bias) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of bfloat16-exact float32 values (the bf16 encoding)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_to_bf16(a) if dtype == "bf16" else a


@dataclass(frozen=True)
class LayerConfig:
    """One MoE layer as seen by one simulated edge server."""

    name: str
    dtype: str            # storage/compute type of activations and weights: "f32" | "bf16"
    seed: int
    T: int                # routed tokens in the batch
    d: int                # hidden size
    E: int                # routed experts in the layer
    f: int                # FFN width of one routed expert (SwiGLU)
    k: int                # top-k
    n_shared: int         # always-local shared experts, FFN width f each
    clusters: int         # planted router clusters
    cluster_size: int     # experts per planted cluster
    sigma: float          # per-expert router noise, relative to centre_std
    centre_std: float     # absolute std of the router cluster centres
    M: int                # simulated servers
    m0: int               # the server this GPU plays
    capacity: Tuple[float, ...]  # C_m in expert units (every expert costs p = 1)
    loc_mode: str         # "zero": every token starts on server 0; "uniform": U{0..M-1}
    Qbar: float           # per-token quality budget (eq 39)
    theta: float          # similarity threshold of this layer (eq 6)
    T_cal: int            # calibration tokens for the similarity model (eq 3)
    omega_T: float = 0.5  # eq 23 weights; omega_T + omega_Q = 1
    omega_Q: float = 0.5
    alpha_f: float = 0.5  # eq 28 weights; alpha_f + alpha_r = 1
    lambda1: float = 0.5  # eq 30 weights; lambda1 + lambda2 = 1
    renorm: int = 1       # renormalise the gate over the top-k
    pin_local_exact: int = 1
    allow_sub: int = 1

    @property
    def bytes_per_el(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "LayerConfig":
        return replace(self, **kw)


def _cap(M: int, per: float) -> Tuple[float, ...]:
    return tuple(float(per) for _ in range(M))


# Tiny correctness layer, fp32: 4 planted groups of 2 experts, 2 servers.
C1 = LayerConfig(name="tiny_fp32_T256_d512_E8_f1024_top2", dtype="f32", seed=0,
                 T=256, d=512, E=8, f=1024, k=2, n_shared=0,
                 clusters=4, cluster_size=2, sigma=0.1, centre_std=1.0,
                 M=2, m0=0, capacity=_cap(2, 4), loc_mode="zero",
                 Qbar=0.25, theta=0.7, T_cal=2048)

# Mixtral-8x7B-shaped layer: 4 servers holding 2 experts each.
C2 = LayerConfig(name="mixtral_T4096_d4096_E8_f14336_top2", dtype="bf16", seed=1,
                 T=4096, d=4096, E=8, f=14336, k=2, n_shared=0,
                 clusters=4, cluster_size=2, sigma=0.1, centre_std=4096 ** -0.5,
                 M=4, m0=0, capacity=_cap(4, 2), loc_mode="zero",
                 Qbar=0.25, theta=0.7, T_cal=8192)

# Qwen-MoE-A2.7B-shaped fine-grained layer with 4 shared experts.
C3 = LayerConfig(name="qwenmoe_T8192_d2048_E60s4_f1408_top4", dtype="bf16", seed=2,
                 T=8192, d=2048, E=60, f=1408, k=4, n_shared=4,
                 clusters=12, cluster_size=5, sigma=0.15, centre_std=2048 ** -0.5,
                 M=4, m0=0, capacity=_cap(4, 15), loc_mode="uniform",
                 Qbar=0.25, theta=0.7, T_cal=8192)

# DeepSeek-MoE-shaped layer with 2 shared experts, 8 servers.
C4 = LayerConfig(name="deepseek_T16384_d2048_E64s2_f1408_top6", dtype="bf16", seed=3,
                 T=16384, d=2048, E=64, f=1408, k=6, n_shared=2,
                 clusters=16, cluster_size=4, sigma=0.2, centre_std=2048 ** -0.5,
                 M=8, m0=0, capacity=_cap(8, 8), loc_mode="zero",
                 Qbar=0.25, theta=0.7, T_cal=8192)

# Quality-budget sweep points of the DeepSeek-shaped layer.
C4_QBAR_SWEEP = (0.0, 0.03, 0.06, 0.12, 0.25)

LAYER_CONFIGS = {"C1": C1, "C2": C2, "C3": C3, "C4": C4}


@dataclass(frozen=True)
class BuildConfig:
    """Similarity-model build of one 128-expert layer (eq 3-5, 24-28)."""

    name: str = "simbuild_Tcal65536_d4096_E128_top8"
    dtype: str = "bf16"
    seed: int = 4
    T_cal: int = 65536
    d: int = 4096
    E: int = 128
    k: int = 8
    clusters: int = 32
    cluster_size: int = 4
    sigma: float = 0.15
    centre_std: float = 4096 ** -0.5
    theta: float = 0.7
    alpha_f: float = 0.5


C5_BUILD = BuildConfig()


@dataclass(frozen=True)
class StreamConfig:
    """A decode stream through an N-layer stack of 128-expert top-8 MoE layers
    (Section V: tokens carry their location and accumulated loss from layer to
    layer; Section VI-A: H = 3, theta_l from 0.9 down to 0.5, memory ratio 2.0).

    The token states entering consecutive layers, and the router cluster
    centres of consecutive layers, are first-order autoregressive chains with
    correlation rho_x and rho_c, standing in for a trained model's residual
    stream: a token's top-1 expert then tends to stay in the same cluster from
    one layer to the next, which is what the transition estimate (eq 41) and
    the look-ahead (eq 42) feed on.  The same chains give the calibration
    tokens of every layer."""

    name: str = "decode_N32_T64_d4096_E128_f1536_top8"
    dtype: str = "bf16"
    seed: int = 4
    N: int = 32            # layers
    T: int = 64            # tokens of the decode batch
    d: int = 4096
    E: int = 128
    f: int = 1536
    k: int = 8
    n_shared: int = 0
    clusters: int = 32
    cluster_size: int = 4
    sigma: float = 0.15
    centre_std: float = 4096 ** -0.5
    M: int = 8
    m0: int = 0
    memory_ratio: float = 2.0   # total server memory / one copy of every expert
    loc_mode: str = "zero"      # every token starts on server 0 at the first layer
    Qbar: float = 1.0
    H: int = 3
    theta_min: float = 0.5
    theta_max: float = 0.9
    T_cal: int = 2048
    rho_x: float = 0.8
    rho_c: float = 0.8
    omega_T: float = 0.5
    omega_Q: float = 0.5
    alpha_f: float = 0.5
    lambda1: float = 0.5
    renorm: int = 1
    pin_local_exact: int = 1
    allow_sub: int = 1

    @property
    def bytes_per_el(self) -> int:
        return 2

    @property
    def capacity(self) -> Tuple[float, ...]:
        """C_m in expert units: memory_ratio copies of the N*E experts over M servers."""
        return _cap(self.M, self.memory_ratio * self.N * self.E / self.M)

    def with_(self, **kw) -> "StreamConfig":
        return replace(self, **kw)


C5_STREAM = StreamConfig()


# ---------------------------------------------------------------- generators
def router(cfg) -> np.ndarray:
    """W_r [E, d]: row j = centre[j // cluster_size] + sigma * centre_std * N(0, 1)."""
    c = _rng(cfg.seed, _S_CENTRES).standard_normal((cfg.clusters, cfg.d), dtype=np.float32)
    n = _rng(cfg.seed, _S_NOISE).standard_normal((cfg.E, cfg.d), dtype=np.float32)
    cl = np.arange(cfg.E) // cfg.cluster_size
    w = cfg.centre_std * (c[cl] + np.float32(cfg.sigma) * n)
    return _store(w, cfg.dtype)


def tokens(cfg, T: Optional[int] = None) -> np.ndarray:
    """X [T, d] ~ N(0, 1): the token representations entering the layer."""
    T = cfg.T if T is None else T
    return _store(_rng(cfg.seed, _S_X).standard_normal((T, cfg.d), dtype=np.float32), cfg.dtype)


def calibration(cfg, T_cal: Optional[int] = None) -> np.ndarray:
    """X_cal [T_cal, d] ~ N(0, 1): calibration tokens for the similarity model."""
    T_cal = cfg.T_cal if T_cal is None else T_cal
    return _store(_rng(cfg.seed, _S_XCAL).standard_normal((T_cal, cfg.d), dtype=np.float32),
                  cfg.dtype)


def expert(cfg: LayerConfig, j: int):
    """Weights of routed expert j in torch Linear layout ([out, in]), N(0, 0.02^2):
    W_gate [f, d], W_up [f, d], W_down [d, f]."""
    s = np.float32(0.02)
    g = _rng(cfg.seed, _S_WG, j).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    u = _rng(cfg.seed, _S_WU, j).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    dn = _rng(cfg.seed, _S_WD, j).standard_normal((cfg.d, cfg.f), dtype=np.float32) * s
    return _store(g, cfg.dtype), _store(u, cfg.dtype), _store(dn, cfg.dtype)


def shared_expert(cfg: LayerConfig, i: int):
    """Weights of shared expert i, same layout and distribution as a routed expert."""
    s = np.float32(0.02)
    g = _rng(cfg.seed, _S_SHARED, 3 * i + 0).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    u = _rng(cfg.seed, _S_SHARED, 3 * i + 1).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    dn = _rng(cfg.seed, _S_SHARED, 3 * i + 2).standard_normal((cfg.d, cfg.f), dtype=np.float32) * s
    return _store(g, cfg.dtype), _store(u, cfg.dtype), _store(dn, cfg.dtype)


def _ar_chain(rng: np.random.Generator, steps: int, shape, rho: float):
    """Yield z_0, ..., z_{steps-1}: z_0 ~ N(0,1), z_l = rho z_{l-1} + sqrt(1-rho^2) N(0,1)."""
    a, b = np.float32(rho), np.float32(np.sqrt(1.0 - rho * rho))
    z = rng.standard_normal(shape, dtype=np.float32)
    yield z
    for _ in range(1, steps):
        z = a * z + b * rng.standard_normal(shape, dtype=np.float32)
        yield z


def stream_clusters(cfg: StreamConfig) -> np.ndarray:
    """Planted cluster of every expert of every layer [N][E]: cluster_size
    experts per cluster, the members drawn by a seeded permutation per layer
    (expert numbers carry no similarity, as in a trained model)."""
    out = np.empty((cfg.N, cfg.E), dtype=np.int64)
    for l in range(cfg.N):
        perm = _rng(cfg.seed, _S_PERM, l).permutation(cfg.E)
        out[l, perm] = np.arange(cfg.E) // cfg.cluster_size
    return out


def stream_routers(cfg: StreamConfig):
    """W_r of every layer [N][E][d]: row j = centre_l[cluster_l(j)] +
    sigma * N(0,1), times centre_std; the centres follow an AR(1) chain over the
    layers, so cluster c of one layer resembles cluster c of the next."""
    cent = _ar_chain(_rng(cfg.seed, _S_CENTRES), cfg.N, (cfg.clusters, cfg.d), cfg.rho_c)
    noise = _rng(cfg.seed, _S_NOISE)
    cls = stream_clusters(cfg)
    out = np.empty((cfg.N, cfg.E, cfg.d), dtype=np.float32)
    for l, c in enumerate(cent):
        n = noise.standard_normal((cfg.E, cfg.d), dtype=np.float32)
        out[l] = _store(cfg.centre_std * (c[cls[l]] + np.float32(cfg.sigma) * n), cfg.dtype)
    return out


def stream_tokens(cfg: StreamConfig, T: Optional[int] = None) -> np.ndarray:
    """X_l [N][T][d]: the states of the decode batch entering each layer
    (an AR(1) chain per token), rounded to the storage type."""
    T = cfg.T if T is None else T
    out = np.empty((cfg.N, T, cfg.d), dtype=np.float32)
    for l, z in enumerate(_ar_chain(_rng(cfg.seed, _S_X), cfg.N, (T, cfg.d), cfg.rho_x)):
        out[l] = _store(z, cfg.dtype)
    return out


def stream_calibration(cfg: StreamConfig, T_cal: Optional[int] = None):
    """Yield X_cal_l [T_cal][d] for l = 0..N-1: calibration tokens followed
    through the stack (the same AR(1) recipe as the decode batch)."""
    T_cal = cfg.T_cal if T_cal is None else T_cal
    for z in _ar_chain(_rng(cfg.seed, _S_XCAL), cfg.N, (T_cal, cfg.d), cfg.rho_x):
        yield _store(z, cfg.dtype)


def stream_expert(cfg: StreamConfig, l: int, j: int):
    """Weights of expert j of layer l (0-based), torch Linear layout, N(0, 0.02^2)."""
    s = np.float32(0.02)
    g = _rng(cfg.seed, _S_WG, l, j).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    u = _rng(cfg.seed, _S_WU, l, j).standard_normal((cfg.f, cfg.d), dtype=np.float32) * s
    dn = _rng(cfg.seed, _S_WD, l, j).standard_normal((cfg.d, cfg.f), dtype=np.float32) * s
    return _store(g, cfg.dtype), _store(u, cfg.dtype), _store(dn, cfg.dtype)


def token_locations(cfg: LayerConfig, T: Optional[int] = None) -> np.ndarray:
    """loc_in [T] uint8: the server each token resides on before the layer (eq 36)."""
    T = cfg.T if T is None else T
    if cfg.loc_mode == "zero":
        return np.zeros(T, dtype=np.uint8)
    return _rng(cfg.seed, _S_LOC).integers(0, cfg.M, size=T).astype(np.uint8)


def accumulated_loss(cfg: LayerConfig, T: Optional[int] = None, scale: float = 0.0) -> np.ndarray:
    """Qhat_in [T] float32: accumulated substitution loss entering the layer.

    scale = 0 gives the first-layer value (all zeros); scale > 0 draws
    U[0, scale) per token to exercise a partly spent budget."""
    T = cfg.T if T is None else T
    if scale == 0.0:
        return np.zeros(T, dtype=np.float32)
    return (_rng(cfg.seed, _S_QHAT).random(T, dtype=np.float32) * np.float32(scale)).astype(np.float32)


@dataclass(frozen=True)
class Network:
    B: np.ndarray    # [M, M] bandwidth, bit/s (symmetric)
    tau: np.ndarray  # [M, M] propagation + queuing delay, s (symmetric, zero diagonal)
    F: np.ndarray    # [M] compute capability, FLOP/s


def network(cfg, M: Optional[int] = None) -> Network:
    """Synthetic edge network in the testbed's ranges (Section VI-A)."""
    M = cfg.M if M is None else M
    g = _rng(cfg.seed + _S_NET)
    B = np.zeros((M, M))
    tau = np.zeros((M, M))
    for a in range(M):
        for b in range(a + 1, M):
            B[a, b] = B[b, a] = g.uniform(1e9, 10e9)
            tau[a, b] = tau[b, a] = g.uniform(0.2e-3, 20e-3)
    for a in range(M):
        B[a, a] = 10e9
    F = g.uniform(20e12, 110e12, size=M)
    return Network(B=B, tau=tau, F=F)


def small_layer(cfg: LayerConfig, **kw) -> LayerConfig:
    """A reduced copy of a layer shape for tests (sizes the oracle finishes quickly)."""
    return cfg.with_(**kw)
