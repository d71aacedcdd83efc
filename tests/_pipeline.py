"""Test harness: one MoE layer instance built for both the oracle and the HIP
library from the same seeded inputs.

The offline model (similarity, groups, deployment) is the oracle's; the
library builds its own decision tables from it with ordermoe_build_tables, and
the tests check those tables against the oracle's.  Everything device-side
goes through the library's C ABI.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

import workloads as wl
from oracle import layer as olayer
from oracle import placement, route, similarity, tables


@dataclass
class Case:
    cfg: wl.LayerConfig
    W_r: np.ndarray
    X: np.ndarray
    loc: np.ndarray
    qhat: np.ndarray
    model: Dict
    sim32: np.ndarray
    x_dep: np.ndarray
    net: wl.Network
    c: np.ndarray
    dref: float
    z_bits: float
    S: np.ndarray
    local: List[int]
    _experts: Dict[int, tuple] = field(default_factory=dict)
    _shared: Optional[List[tuple]] = None

    def expert(self, j: int):
        if j not in self._experts:
            self._experts[j] = wl.expert(self.cfg, j)
        return self._experts[j]

    def shared(self) -> List[tuple]:
        if self._shared is None:
            self._shared = [wl.shared_expert(self.cfg, i) for i in range(self.cfg.n_shared)]
        return self._shared


def build_case(cfg: wl.LayerConfig, T: Optional[int] = None, qhat_scale: float = 0.0) -> Case:
    W = wl.router(cfg)
    model = similarity.build(wl.calibration(cfg), W, cfg.k, cfg.theta, cfg.alpha_f)
    x_dep, _ = placement.place([model["group_of"]], [model["I"]], [np.ones(cfg.E)],
                               np.array(cfg.capacity), np.full(cfg.M, 1.0 / cfg.M), cfg.lambda1)
    x_dep = x_dep[0]
    net = wl.network(cfg)
    c = np.full(cfg.E, 6.0 * cfg.d * cfg.f)
    dref = tables.d_ref(c, net.F)
    z_bits = 8.0 * cfg.d * cfg.bytes_per_el
    S = tables.static_cost(cfg.M, cfg.E, z_bits, net.B, net.tau, c, net.F, dref, cfg.omega_T)
    T = cfg.T if T is None else T
    local = [int(j) for j in np.nonzero(x_dep[cfg.m0])[0]]
    return Case(cfg=cfg, W_r=W, X=wl.tokens(cfg, T), loc=wl.token_locations(cfg, T),
                qhat=wl.accumulated_loss(cfg, T, qhat_scale), model=model,
                sim32=model["sim"].astype(np.float32), x_dep=x_dep, net=net, c=c, dref=dref,
                z_bits=z_bits, S=S, local=local)


def oracle_decisions(case: Case, Qbar: Optional[float] = None):
    cfg = case.cfg
    Qbar = cfg.Qbar if Qbar is None else Qbar
    idx, w, margin, _ = route.route(case.X, case.W_r, cfg.k, cfg.renorm)
    sel = olayer.select(idx, case.x_dep, case.sim32, case.model["group_of"], cfg.theta, case.S,
                        Qbar, cfg.omega_Q, case.loc, case.qhat, cfg.pin_local_exact, cfg.allow_sub)
    sel.update(idx=idx, w=w, margin=margin)
    return sel


def oracle_output(case: Case, dec: Dict, tokens: np.ndarray) -> np.ndarray:
    return olayer.server_output(case.X, dec["w"], dec["exec_k"], dec["exec_m"], case.loc,
                                case.cfg.m0, case.expert, case.shared(), tokens)


# ------------------------------------------------------------------ device side
def library_tables(case: Case, gmax: int = 15):
    from paper_2607_17154_amd import ordermoe as om
    cfg = case.cfg
    return om.ordermoe_build_tables(case.sim32, case.model["group_of"], cfg.theta, case.x_dep,
                                    case.net.B, case.net.tau, case.net.F, case.z_bits, case.c,
                                    case.dref, cfg.omega_T, None, gmax)


def to_device(a: np.ndarray, dtype: str, device="cuda"):
    """Upload a float32 host array holding values of the run dtype."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.to(device)


class DeviceLayer:
    """Device buffers and ABI structs of one layer on server m0."""

    def __init__(self, case: Case, tabs: Dict, Qbar: Optional[float] = None, gmax: int = 15,
                 with_experts: bool = True):
        import torch
        from paper_2607_17154_amd import ordermoe as om
        cfg = case.cfg
        self.case, self.cfg = case, cfg
        self.code = om.BF16 if cfg.dtype == "bf16" else om.F32
        dev = "cuda"
        self.w_router = to_device(case.W_r, cfg.dtype)
        self.tabs_dev = {n: torch.from_numpy(np.ascontiguousarray(v)).to(dev)
                         for n, v in tabs.items() if n != "srvmask"}
        self.tabs_dev["srvmask"] = torch.from_numpy(tabs["srvmask"].view(np.int32)).to(dev)
        self.Qbar = cfg.Qbar if Qbar is None else Qbar
        self.layer = om.make_layer(self.code, cfg.d, cfg.E, cfg.k, cfg.M, gmax, self.w_router,
                                   self.tabs_dev, self.Qbar, cfg.omega_Q, cfg.pin_local_exact,
                                   cfg.allow_sub, cfg.renorm)
        self.experts = None
        if with_experts:
            self._upload_experts()

    def _upload_experts(self):
        import torch
        from paper_2607_17154_amd import ordermoe as om
        cfg, case = self.cfg, self.case
        tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        n = len(case.local)
        g = torch.empty((max(n, 1), cfg.f, cfg.d), dtype=tdt, device="cuda")
        u = torch.empty_like(g)
        dn = torch.empty((max(n, 1), cfg.d, cfg.f), dtype=tdt, device="cuda")
        for i, j in enumerate(case.local):
            Wg, Wu, Wd = case.expert(j)
            g[i] = to_device(Wg, cfg.dtype)
            u[i] = to_device(Wu, cfg.dtype)
            dn[i] = to_device(Wd, cfg.dtype)
        self.w_gu = torch.empty((max(n, 1), 2 * cfg.f, cfg.d), dtype=tdt, device="cuda")
        om.ordermoe_pack_gate_up(g, u, self.w_gu)
        self.w_dn = torch.empty_like(dn)
        om.ordermoe_pack_down(dn, self.w_dn)
        self.w_sh_gu = self.w_sh_dn = None
        if cfg.n_shared:
            sh = case.shared()
            sg = torch.cat([to_device(s[0], cfg.dtype) for s in sh], 0).unsqueeze(0).contiguous()
            su = torch.cat([to_device(s[1], cfg.dtype) for s in sh], 0).unsqueeze(0).contiguous()
            self.w_sh_gu = torch.empty((1, 2 * cfg.n_shared * cfg.f, cfg.d), dtype=tdt, device="cuda")
            om.ordermoe_pack_gate_up(sg, su, self.w_sh_gu)
            sd = torch.cat([to_device(s[2], cfg.dtype) for s in sh], 1).unsqueeze(0).contiguous()
            self.w_sh_dn = torch.empty_like(sd)
            om.ordermoe_pack_down(sd, self.w_sh_dn)
        torch.cuda.synchronize()
        del g, u, dn
        self.experts = om.make_experts(self.code, cfg.d, cfg.f, cfg.E, case.local, self.w_gu,
                                       self.w_dn, cfg.n_shared, self.w_sh_gu, self.w_sh_dn)

    def inputs(self, X=None, loc=None, qhat=None):
        import torch
        case = self.case
        X = case.X if X is None else X
        loc = case.loc if loc is None else loc
        qhat = case.qhat if qhat is None else qhat
        return (to_device(X, self.cfg.dtype), torch.from_numpy(np.ascontiguousarray(loc)).cuda(),
                torch.from_numpy(np.ascontiguousarray(qhat, dtype=np.float32)).cuda())

    def route(self, x, loc, qhat, T: int):
        import torch
        from paper_2607_17154_amd import ordermoe as om
        out = om.alloc_route_out(T, self.cfg.k, self.cfg.M, "cuda")
        ws = torch.empty(max(om.ordermoe_route_workspace_size(T, self.cfg.k, self.cfg.M), 1),
                         dtype=torch.uint8, device="cuda")
        om.ordermoe_route_select(self.layer, x, T, loc, qhat, out, ws)
        return out

    def forward(self, x, loc, out, T: int, server: Optional[int] = None):
        import torch
        from paper_2607_17154_amd import ordermoe as om
        server = self.cfg.m0 if server is None else server
        tdt = torch.bfloat16 if self.cfg.dtype == "bf16" else torch.float32
        y = torch.empty((T, self.cfg.d), dtype=tdt, device="cuda")
        ro = torch.empty(self.experts.n_local + 2, dtype=torch.int32, device="cuda")
        ws = torch.empty(max(om.ordermoe_forward_workspace_size(self.experts, T, self.cfg.k), 1),
                         dtype=torch.uint8, device="cuda")
        om.ordermoe_local_moe_forward(self.experts, x, T, self.cfg.k, out["w"], out["exec_k"],
                                      out["exec_m"], loc, server, y, ro, ws)
        return y, ro


def host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


# ------------------------------------------------------------------ decode stream
@dataclass
class StreamCase:
    """The offline model of an N-layer stack, built by the oracle: per layer the
    router, similarity model and threshold, the joint deployment, transition
    probabilities, look-ahead cost-to-go and static cost tables."""
    cfg: wl.StreamConfig
    W_r: np.ndarray            # [N, E, d]
    X: np.ndarray              # [N, T, d] states of the decode batch entering each layer
    theta: List[float]         # eq 6, fp64
    models: List[Dict]
    sim32: List[np.ndarray]
    x_dep: List[np.ndarray]    # [N] of [M, E]
    P: List[np.ndarray]        # [N-1] of [E, E]
    net: wl.Network
    c: np.ndarray              # [E] compute per expert (same for every layer)
    dref: float
    z_bits: float
    phi: List[np.ndarray]      # [N] of [M, E]
    S: List[np.ndarray]        # [N] of [M, M, E] fp32
    local: List[List[int]]     # experts of server m0 per layer


def build_stream(cfg: wl.StreamConfig) -> StreamCase:
    W = wl.stream_routers(cfg)
    theta = [tables.theta_layer(l + 1, cfg.N, cfg.theta_min, cfg.theta_max) for l in range(cfg.N)]
    models, top1 = [], []
    for l, Xc in enumerate(wl.stream_calibration(cfg)):
        models.append(similarity.build(Xc, W[l], cfg.k, theta[l], cfg.alpha_f))
        idx, _, _, _ = route.route(Xc, W[l], 1, cfg.renorm)
        top1.append(idx[:, 0])
    groups = [m["group_of"] for m in models]
    x_dep, _ = placement.place(groups, [m["I"] for m in models], [np.ones(cfg.E)] * cfg.N,
                               np.array(cfg.capacity), np.full(cfg.M, 1.0 / cfg.M), cfg.lambda1)
    P = tables.transitions(top1, [cfg.E] * cfg.N)
    net = wl.network(cfg)
    c = np.full(cfg.E, 6.0 * cfg.d * cfg.f)
    dref = tables.d_ref(c, net.F)
    z_bits = 8.0 * cfg.d * cfg.bytes_per_el
    sim32 = [m["sim"].astype(np.float32) for m in models]
    phi = tables.lookahead(cfg.H, P, x_dep, sim32, groups, theta, [z_bits] * cfg.N, net.B, net.tau,
                           [c] * cfg.N, net.F, [dref] * cfg.N, cfg.omega_T, cfg.omega_Q, cfg.Qbar,
                           cfg.pin_local_exact, cfg.allow_sub)
    S = [tables.static_cost(cfg.M, cfg.E, z_bits, net.B, net.tau, c, net.F, dref, cfg.omega_T, phi[l])
         for l in range(cfg.N)]
    local = [[int(j) for j in np.nonzero(x_dep[l][cfg.m0])[0]] for l in range(cfg.N)]
    return StreamCase(cfg=cfg, W_r=W, X=wl.stream_tokens(cfg), theta=theta, models=models,
                      sim32=sim32, x_dep=x_dep, P=P, net=net, c=c, dref=dref, z_bits=z_bits,
                      phi=phi, S=S, local=local)


def stream_oracle_layer(sc: StreamCase, l: int, loc: np.ndarray, qhat: np.ndarray):
    """Routing and selection of layer l for the decode batch (the per-layer step
    of Algorithm 2), from the tokens' locations and accumulated losses."""
    cfg = sc.cfg
    idx, w, margin, _ = route.route(sc.X[l], sc.W_r[l], cfg.k, cfg.renorm)
    sel = olayer.select(idx, sc.x_dep[l], sc.sim32[l], sc.models[l]["group_of"], sc.theta[l], sc.S[l],
                        cfg.Qbar, cfg.omega_Q, loc, qhat, cfg.pin_local_exact, cfg.allow_sub)
    sel.update(idx=idx, w=w, margin=margin)
    return sel


def stream_library_tables(sc: StreamCase, gmax: int = 15):
    """The library's look-ahead (eq 41-42) and per-layer tables, from the
    oracle's offline model."""
    from paper_2607_17154_amd import ordermoe as om
    cfg = sc.cfg
    N = cfg.N
    theta32 = np.array([om.ordermoe_theta_layer(l + 1, N, cfg.theta_min, cfg.theta_max)
                        for l in range(N)], np.float32)
    phi = om.ordermoe_build_lookahead(cfg.H, np.stack(sc.P), np.stack(sc.x_dep), np.stack(sc.sim32),
                                      np.stack([m["group_of"] for m in sc.models]), theta32,
                                      np.full(N, sc.z_bits), np.tile(sc.c, (N, 1)), np.full(N, sc.dref),
                                      sc.net.B, sc.net.tau, sc.net.F, cfg.omega_T, cfg.omega_Q, cfg.Qbar,
                                      cfg.pin_local_exact, cfg.allow_sub)
    tabs = [om.ordermoe_build_tables(sc.sim32[l], sc.models[l]["group_of"], float(theta32[l]),
                                     sc.x_dep[l], sc.net.B, sc.net.tau, sc.net.F, sc.z_bits, sc.c,
                                     sc.dref, cfg.omega_T, phi[l], gmax) for l in range(N)]
    return theta32, phi, tabs


def with_horizon(sc: StreamCase, H: int, allow_sub: Optional[int] = None) -> StreamCase:
    """The same stack with the look-ahead depth H (eq 42), and optionally
    another substitution mode: the oracle's Phi and cost tables recomputed,
    everything else shared."""
    import dataclasses
    cfg = dataclasses.replace(sc.cfg, H=H, allow_sub=sc.cfg.allow_sub if allow_sub is None else allow_sub)
    groups = [m["group_of"] for m in sc.models]
    phi = tables.lookahead(H, sc.P, sc.x_dep, sc.sim32, groups, sc.theta, [sc.z_bits] * cfg.N, sc.net.B,
                           sc.net.tau, [sc.c] * cfg.N, sc.net.F, [sc.dref] * cfg.N, cfg.omega_T, cfg.omega_Q,
                           cfg.Qbar, cfg.pin_local_exact, cfg.allow_sub)
    S = [tables.static_cost(cfg.M, cfg.E, sc.z_bits, sc.net.B, sc.net.tau, sc.c, sc.net.F, sc.dref,
                            cfg.omega_T, phi[l]) for l in range(cfg.N)]
    return dataclasses.replace(sc, cfg=cfg, phi=phi, S=S)


# ------------------------------------------------------------ GEMM work plan (host mirror)
# The bf16 grouped GEMMs of the local forward (batches above 128 tokens) run
# 256 x 256 gate/up tiles and 192 x 256 down tiles over a persistent grid of at
# most 256 workgroups (one per CU on MI355X, at most four per tile); the tiles
# left after whole rounds are cut along K into up to 4 pieces of at least 16 K
# tiles of 64 when at least two workgroups per tile are free and every group
# has the same K.  Tests use this
# mirror to know which of their shapes exercise the split.
def gemm_plan(cfg, rows, n_local: int, cus: int = 256):
    """rows: the forward's row_offsets output [n_local + 2].  Returns
    {"gate_up": (tiles, grid, rounds, left, split, shared_halves, tile_rows), "down": (...)};
    shared_halves is 1 when the shared tiles are cut into two K halves."""
    R = np.diff(np.asarray(rows, dtype=np.int64))       # rows per group, shared last
    has_sh = cfg.n_shared > 0
    T, k, d, f, ns = cfg.T, cfg.k, cfg.d, cfg.f, cfg.n_shared
    rr = T * min(k, n_local)
    rs = T if has_sh else 0

    def grid_of(ub):
        g = min(cus, 4 * ub)
        g = (g + 7) & ~7
        return min(max(g, 8), 256)

    def plan(bm, bn, Nr, Ns, Kr, Ks, ub):
        tiles = sum(-(-int(R[g]) // bm) * (Nr // bn) for g in range(n_local))
        if has_sh:
            tiles += -(-int(R[n_local]) // bm) * (Ns // bn)
        grid = grid_of(ub)
        nsh = -(-int(R[n_local]) // bm) * (Ns // bn) if has_sh else 0
        halves = int(nsh > 0 and Ks >= 2 * Kr and Ks % 256 == 0 and 2 * nsh <= grid)
        items = tiles + nsh * halves
        rounds = items // grid
        left = items - rounds * grid
        split = min(grid // left, 4, Kr // 128, Kr // 64 // 16) if left else 0
        if has_sh and Ks != Kr:
            split = 1
        return tiles, grid, rounds, left, split, halves, bm

    ub_gu = (-(-rr // 256) + n_local) * (2 * f // 256) + ((-(-rs // 256) + 1) * (2 * ns * f // 256) if has_sh else 0)
    # down tiles of 256 rows when even those would fill the grid eight times over
    bm_dn = 256 if (-(-(rr + rs) // 256) + n_local + int(has_sh)) * (d // 256) >= 8 * 256 else 192
    ub_dn = (-(-(rr + rs) // bm_dn) + n_local + int(has_sh)) * (d // 256)
    return {"gate_up": plan(256, 256, 2 * f, 2 * ns * f, d, d, ub_gu),
            "down": plan(bm_dn, 256, d, d, f, ns * f, ub_dn)}
