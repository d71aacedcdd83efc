"""Benchmark: one OrderMoE MoE layer on one MI355X.

A step is the whole layer path of one server over one batch: routing and
server-expert selection with the dispatch list (ordermoe_route_select), then
the local grouped SwiGLU FFN with the weighted combine
(ordermoe_local_moe_forward).  Workload: the Mixtral-8x7B-shaped layer --
4096 tokens of hidden 4096, 8 experts of FFN 14336, top-2, 4 simulated
servers holding 2 experts each -- bf16, synthetic seeded inputs, inputs
resident in HBM before the timed region.  The timed steps run as a serving
loop runs consecutive batches: step i on HIP stream i mod S (--streams, 2 by
default) with its own outputs and workspaces, so two batches are in flight and
one batch's small kernels and GEMM tiles fill the CUs that the other's GEMM
tails leave idle; the line also reports the one-stream step time (one batch
at a time, the step's latency), and the run fails if any stream's outputs
differ from the one-stream outputs.

Prints one compact JSON line (rank 0).  Besides tokens/s it reports the
roofline of the dominant kernel (the grouped gate/up GEMM) from its average
launch time measured with HIP events on the launch stream, and the CPU oracle
timed on a bounded sample of the same workload.  The other legs (the Qwen- and
DeepSeek-shaped layers, the similarity build, the sweeps, the decode stream)
go to a JSON file (--out, by default gpurun_out/bench_full.json); the line
carries one figure of each.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemm_gate_up_mixtral_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_17154_amd", "csrc", "moe_forward.hip")


def source_sha256(path: str) -> str:
    import hashlib
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def _measured_traffic():
    """HBM bytes per launch of the gate/up GEMM from the committed rocprofv3
    counter summary, if it was taken on the current kernel source."""
    try:
        lines = open(TRAFFIC_PROFILE).read().splitlines()
    except OSError:
        return None
    vals = {}
    for ln in lines:
        if ln.startswith("- ") and ":" in ln:
            k, v = ln[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("kernel source sha256") != source_sha256(GEMM_SOURCE):
        return None
    try:
        return int(vals["HBM bytes per launch (scaled)"])
    except (KeyError, ValueError):
        return None


def _calibrate_copy(torch, gib: int = 1):
    """A plain device copy of known size, for scaling the HBM byte counters."""
    n = gib * (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))


def _upload(cfg, torch, a):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch.bfloat16) if cfg.dtype == "bf16" else t).to("cuda")


def _layer_model(cfg, torch, om):
    """The layer's offline model through the library: similarity build on the
    GPU, deployment (Algorithm 1) and decision tables on the host."""
    import workloads as wl
    dev = "cuda"
    up = lambda a: _upload(cfg, torch, a)
    W = wl.router(cfg)
    Xc = wl.calibration(cfg)
    ws = torch.empty(om.ordermoe_similarity_workspace_size(Xc.shape[0], cfg.d, cfg.E),
                     dtype=torch.uint8, device=dev)
    model = om.ordermoe_build_similarity(up(Xc), up(W), cfg.k, cfg.theta, cfg.alpha_f, ws)
    del ws
    x_dep, _ = om.ordermoe_place([model["group_of"]], [model["importance"]], [np.ones(cfg.E)],
                                 np.array(cfg.capacity), np.full(cfg.M, 1.0 / cfg.M), cfg.lambda1, 1)
    x_dep = x_dep[0]
    net = wl.network(cfg)
    c = np.full(cfg.E, 6.0 * cfg.d * cfg.f)
    dref = float(np.mean(c)) / float(np.mean(net.F))
    z_bits = 8.0 * cfg.d * cfg.bytes_per_el
    tabs = om.ordermoe_build_tables(model["sim"], model["group_of"], cfg.theta, x_dep, net.B,
                                    net.tau, net.F, z_bits, c, dref, cfg.omega_T)
    tabs_dev = {n: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for n, v in tabs.items()
                if n != "srvmask"}
    tabs_dev["srvmask"] = torch.from_numpy(tabs["srvmask"].view(np.int32)).to(dev)
    w_router = up(W)
    code = om.BF16 if cfg.dtype == "bf16" else om.F32
    return dict(W=W, Xc=Xc, model=model, x_dep=x_dep, net=net, c=c, dref=dref, z_bits=z_bits,
                tabs_dev=tabs_dev, w_router=w_router, code=code)


def _setup(cfg, torch, om):
    """Library-side layer: similarity build on the GPU, deployment and tables
    on the host, expert weights of this server packed on the device."""
    import workloads as wl
    dev = "cuda"
    up = lambda a: _upload(cfg, torch, a)
    lm = _layer_model(cfg, torch, om)
    W, model, x_dep, net, c, dref, z_bits = (lm[n] for n in ("W", "model", "x_dep", "net", "c", "dref", "z_bits"))
    tabs_dev, w_router, code = lm["tabs_dev"], lm["w_router"], lm["code"]
    layer = om.make_layer(code, cfg.d, cfg.E, cfg.k, cfg.M, 15, w_router, tabs_dev, cfg.Qbar,
                          cfg.omega_Q, cfg.pin_local_exact, cfg.allow_sub, cfg.renorm)
    local = [int(j) for j in np.nonzero(x_dep[cfg.m0])[0]]
    n = len(local)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    w_gu = torch.empty((n, 2 * cfg.f, cfg.d), dtype=tdt, device=dev)
    w_dn = torch.empty((n, cfg.d, cfg.f), dtype=tdt, device=dev)
    for i, j in enumerate(local):
        g, u, dn = wl.expert(cfg, j)
        gd, ud = up(g), up(u)
        om.ordermoe_pack_gate_up(gd.unsqueeze(0), ud.unsqueeze(0), w_gu[i:i + 1])
        om.ordermoe_pack_down(up(dn).unsqueeze(0), w_dn[i:i + 1])
        del gd, ud
    w_sh_gu = w_sh_dn = None
    if cfg.n_shared:
        sh = [wl.shared_expert(cfg, i) for i in range(cfg.n_shared)]
        sg = torch.cat([up(a[0]) for a in sh], 0).unsqueeze(0).contiguous()
        su = torch.cat([up(a[1]) for a in sh], 0).unsqueeze(0).contiguous()
        w_sh_gu = torch.empty((1, 2 * cfg.n_shared * cfg.f, cfg.d), dtype=tdt, device=dev)
        om.ordermoe_pack_gate_up(sg, su, w_sh_gu)
        sd = torch.cat([up(a[2]) for a in sh], 1).unsqueeze(0).contiguous()
        w_sh_dn = torch.empty_like(sd)
        om.ordermoe_pack_down(sd, w_sh_dn)
        del sg, su, sd
    experts = om.make_experts(code, cfg.d, cfg.f, cfg.E, local, w_gu, w_dn, cfg.n_shared, w_sh_gu, w_sh_dn)
    X = wl.tokens(cfg)
    st = dict(layer=layer, experts=experts, keep=(w_router, tabs_dev, w_gu, w_dn, w_sh_gu, w_sh_dn), local=local,
              x=up(X), loc=torch.from_numpy(wl.token_locations(cfg)).to(dev),
              qhat=torch.from_numpy(wl.accumulated_loss(cfg)).to(dev), X=X, W=W, model=model,
              x_dep=x_dep, net=net, c=c, dref=dref, z_bits=z_bits)
    st["out"] = om.alloc_route_out(cfg.T, cfg.k, cfg.M, dev)
    st["out_struct"] = om.route_out_struct(st["out"])
    st["ws_r"] = torch.empty(om.ordermoe_route_workspace_size(cfg.T, cfg.k, cfg.M), dtype=torch.uint8,
                             device=dev)
    st["ws_f"] = torch.empty(om.ordermoe_forward_workspace_size(experts, cfg.T, cfg.k),
                             dtype=torch.uint8, device=dev)
    st["y"] = torch.empty((cfg.T, cfg.d), dtype=tdt, device=dev)
    st["ro"] = torch.empty(n + 2, dtype=torch.int32, device=dev)
    return st


def _step(cfg, st, om, stream=None):
    o = st["out"]
    om.ordermoe_route_select(st["layer"], st["x"], cfg.T, st["loc"], st["qhat"], o, st["ws_r"],
                             out_struct=st["out_struct"], stream=stream)
    om.ordermoe_local_moe_forward(st["experts"], st["x"], cfg.T, cfg.k, o["w"], o["exec_k"],
                                  o["exec_m"], st["loc"], cfg.m0, st["y"], st["ro"], st["ws_f"],
                                  stream=stream)


def _batch_sets(cfg, st, torch, om, n):
    """n independent sets of per-batch buffers (route outputs, workspaces,
    layer output) over the same weights and tables; set 0 is st itself."""
    sets = [st]
    for _ in range(n - 1):
        s = dict(st)
        s["out"] = om.alloc_route_out(cfg.T, cfg.k, cfg.M, "cuda")
        s["out_struct"] = om.route_out_struct(s["out"])
        for key in ("ws_r", "ws_f", "y", "ro"):
            s[key] = torch.empty_like(st[key])
        sets.append(s)
    return sets


def _timed_steps(cfg, sets, streams, steps, torch, om):
    """Runs `steps` layer steps, step i on stream i mod S with buffer set
    i mod S, so that S consecutive batches are in flight (each batch's kernels
    stay in order on its stream; batches share no buffer).  Returns the
    milliseconds from a start event on the current stream, which every stream
    waits for, to an end event after the current stream has waited for all of
    them."""
    cur = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(cur)
    for s in streams:
        s.wait_event(e0)
    for i in range(steps):
        j = i % len(streams)
        _step(cfg, sets[j], om, stream=streams[j])
    for s in streams:
        ev = torch.cuda.Event()
        ev.record(s)
        cur.wait_event(ev)
    e1.record(cur)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


_STREAMS = []


def _streams(torch, n):
    """The same n streams for every leg: HIP spreads streams over a few
    hardware queues in creation order, and two streams that land on one queue
    run one after the other, so the process creates its streams once."""
    while len(_STREAMS) < n:
        _STREAMS.append(torch.cuda.Stream())
    return _STREAMS[:n]


def _pipelined(cfg, st, torch, om, n_streams, steps, warmup):
    """Step time with n_streams batches in flight, and the check that every
    set's outputs equal the single-stream outputs bit for bit."""
    names = ("exec_k", "exec_m", "w", "counters")
    ref = dict(y=st["y"].clone(), ro=st["ro"].clone(), **{n: st["out"][n].clone() for n in names})
    sets = _batch_sets(cfg, st, torch, om, n_streams)
    streams = _streams(torch, n_streams)
    # two untimed passes: the first concurrent use of new streams costs several
    # milliseconds once (queue set-up), which would otherwise land in the timed steps
    for _ in range(2):
        _timed_steps(cfg, sets, streams, max(warmup, 2 * n_streams), torch, om)
    ms = _timed_steps(cfg, sets, streams, steps, torch, om)
    equal = all(torch.equal(s["y"], ref["y"]) and torch.equal(s["ro"], ref["ro"]) and
                all(torch.equal(s["out"][n], ref[n]) for n in names) for s in sets)
    del sets[1:]
    return ms, equal


def _cpu_baseline(cfg, st, target_s: float):
    """The oracle as it stands on a bounded token sample of the same layer."""
    import workloads as wl
    from oracle import layer as olayer
    from oracle import route, similarity, tables
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    # the oracle's own offline model (not timed: built once per layer)
    model = similarity.build(wl.calibration(cfg, 4096), st["W"], cfg.k, cfg.theta, cfg.alpha_f)
    S = tables.static_cost(cfg.M, cfg.E, st["z_bits"], st["net"].B, st["net"].tau, st["c"],
                           st["net"].F, st["dref"], cfg.omega_T)
    experts = {}

    def ew(j):
        if j not in experts:
            experts[j] = wl.expert(cfg, j)
        return experts[j]

    loc = wl.token_locations(cfg)
    qh = wl.accumulated_loss(cfg)

    split = [0.0, 0.0]                 # decisions, outputs: seconds over the timed passes

    def run(n):
        X = st["X"][:n]
        t0 = time.perf_counter()
        idx, w, mg, _ = route.route(X, st["W"], cfg.k, cfg.renorm)
        sel = olayer.select(idx, st["x_dep"], model["sim"].astype(np.float32), model["group_of"],
                            cfg.theta, S, cfg.Qbar, cfg.omega_Q, loc[:n], qh[:n],
                            cfg.pin_local_exact, cfg.allow_sub)
        olayer.dispatch(sel["exec_m"], loc[:n], cfg.M)
        t1 = time.perf_counter()
        olayer.server_output(X, w, sel["exec_k"], sel["exec_m"], loc[:n], cfg.m0, ew, (),
                             np.arange(n))
        t2 = time.perf_counter()
        split[0] += t1 - t0
        split[1] += t2 - t1
        return t2 - t0

    for j in st["local"]:
        ew(j)
    n = 16
    dt = run(n)
    while dt < target_s / 4 and n < cfg.T:
        n = min(cfg.T, int(n * max(2.0, target_s / max(dt, 1e-3) * 0.8)))
        split[:] = [0.0, 0.0]
        dt = run(n)
    reps = 1
    if dt < target_s / 2:
        # the whole batch is quick: repeat it to a bounded sample of about target_s seconds
        reps = max(1, int(target_s / max(dt, 1e-3)))
        split[:] = [0.0, 0.0]
        dt = sum(run(n) for _ in range(reps))
    dec_s, out_s = split
    res = {"value": reps * n / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
           "sample": "%d pass(es) over the first %d of the %d tokens (route fp64, selection, "
                     "dispatch, fp64 FFN of server %d); %.1f s" % (reps, n, cfg.T, cfg.m0, dt),
           "decisions_tokens_per_s": reps * n / dec_s, "outputs_tokens_per_s": reps * n / out_s}
    # the same path on one host thread, on a smaller sample of about a quarter of target_s
    try:
        from threadpoolctl import threadpool_limits
        n1 = int(max(16, min(cfg.T, target_s / 4 / max(dt / (reps * n) * cores, 1e-9))))
        split[:] = [0.0, 0.0]
        with threadpool_limits(limits=1):
            d1 = run(n1)
        res["one_core"] = {"value": n1 / d1, "decisions_tokens_per_s": n1 / split[0],
                           "outputs_tokens_per_s": n1 / split[1],
                           "sample": "the first %d tokens, %.1f s" % (n1, d1)}
    except ImportError:  # pragma: no cover
        pass
    return res


def _simbuild(torch, om, reps: int = 5):
    """Similarity-model build of a 128-expert layer over 65536 calibration tokens of
    hidden 4096 (eq 3-5): average device time of its two kernels, HBM fraction."""
    import workloads as wl
    cfg = wl.C5_BUILD
    up = lambda a: torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).to("cuda")
    xc, w = up(wl.calibration(cfg)), up(wl.router(cfg))
    ws = torch.empty(om.ordermoe_similarity_workspace_size(cfg.T_cal, cfg.d, cfg.E),
                     dtype=torch.uint8, device="cuda")
    om.ordermoe_build_similarity(xc, w, cfg.k, cfg.theta, cfg.alpha_f, ws)   # warm-up
    om.ordermoe_timing_read(reset=True)
    om.ordermoe_timing_enable(True)
    for _ in range(reps):
        res = om.ordermoe_build_similarity(xc, w, cfg.k, cfg.theta, cfg.alpha_f, ws)
    om.ordermoe_timing_enable(False)
    kt = om.ordermoe_timing_read(reset=True)
    us = sum(v[0] / v[1] for k, v in kt.items() if k.startswith("sim_")) * 1e3
    nbytes = cfg.T_cal * cfg.d * 2 + cfg.E * cfg.d * 2
    return {"workload": cfg.name, "groups": len(res["centres"]), "device_us": us,
            "kernels_avg_us": {k: v[0] / v[1] * 1e3 for k, v in kt.items()},
            "hbm_bytes": nbytes, "achieved_GBs": nbytes / us / 1e3,
            "hbm_frac": nbytes / us / 1e3 / PEAK_HBM_GBS}


def _other_layers(torch, om, steps: int = 30, warmup: int = 5, n_streams: int = 2):
    """The Qwen-MoE-shaped (8192 tokens, 60 experts + 4 shared, top-4) and
    DeepSeek-MoE-shaped (16384 tokens, 64 experts + 2 shared, top-6) layers of
    server 0: step time, the FFN GEMMs' MFMA rates and routing's HBM rate."""
    import workloads as wl
    res = {}
    for key, cfg in (("C3", wl.C3), ("C4", wl.C4)):
        st = _setup(cfg, torch, om)
        for _ in range(warmup):
            _step(cfg, st, om)
        torch.cuda.synchronize()
        ms_one = _timed_steps(cfg, [st], [torch.cuda.current_stream()], steps, torch, om) / steps
        ms, equal = ms_one * steps, True
        if n_streams > 1:
            ms, equal = _pipelined(cfg, st, torch, om, n_streams, steps, warmup)
            if not equal:
                raise RuntimeError("%s: outputs differ between streams" % key)
        ms /= steps
        om.ordermoe_timing_read(reset=True)
        om.ordermoe_timing_enable(True)
        for _ in range(steps):
            _step(cfg, st, om)
        torch.cuda.synchronize()
        om.ordermoe_timing_enable(False)
        kt = om.ordermoe_timing_read(reset=True)
        avg = {n: v[0] / v[1] * 1e3 for n, v in kt.items()}
        ro = st["ro"].cpu().numpy()
        n_loc = len(st["local"])
        r_routed = int(ro[n_loc])
        r_shared = int(ro[-1]) - r_routed
        fl_gu = 2.0 * cfg.d * 2 * cfg.f * r_routed + 2.0 * cfg.d * 2 * cfg.n_shared * cfg.f * r_shared
        fl_dn = fl_gu / 2
        gu_us = sum(v for n, v in avg.items() if n.startswith("gemm_gate_up"))
        rt_bytes = cfg.T * cfg.d * 2 + cfg.E * cfg.d * 2 + cfg.T * cfg.k * 14 + cfg.T * 11
        rt_us = avg.get("route_select", float("nan"))
        res[key] = {"workload": cfg.name, "streams": n_streams, "ms_per_step": ms,
                    "tokens_per_s": cfg.T / (ms / 1e3), "ms_per_step_one_stream": ms_one,
                    "local_rows_routed": r_routed, "local_rows_shared": r_shared,
                    "gemm_gate_up_TFLOPs": fl_gu / gu_us / 1e6,
                    "gemm_gate_up_frac": fl_gu / gu_us / 1e6 / PEAK_BF16_TFLOPS,
                    "gemm_down_TFLOPs": fl_dn / avg["gemm_down"] / 1e6,
                    "gemm_down_frac": fl_dn / avg["gemm_down"] / 1e6 / PEAK_BF16_TFLOPS,
                    "route_select_us": rt_us, "route_hbm_frac": rt_bytes / rt_us / 1e3 / PEAK_HBM_GBS,
                    "kernels_avg_us": dict(sorted(avg.items()))}
        del st
        torch.cuda.empty_cache()
    return res


def _quality_sweep(torch, om):
    """Quality-budget sweep of the DeepSeek-MoE-shaped layer (16384 tokens,
    64 experts + 2 shared, top-6, 8 servers): for each budget Qbar, routing
    and selection, then the local FFN of every simulated server; the servers'
    outputs add up to the system output.  Reports the share of slots executed
    on another server and the relative deviation (Frobenius) of the system
    output from the zero-budget one, which is the exact top-k MoE output.
    Expert weights are drawn on the device, N(0, 0.02^2) in bf16."""
    import workloads as wl
    cfg = wl.C4
    dev = "cuda"
    lm = _layer_model(cfg, torch, om)
    x_dep, code = lm["x_dep"], lm["code"]
    E, d, f, M, T, k, nsh = cfg.E, cfg.d, cfg.f, cfg.M, cfg.T, cfg.k, cfg.n_shared
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    bf = torch.bfloat16
    g = torch.randn((E, f, d), generator=gen, device=dev, dtype=bf) * 0.02
    u = torch.randn((E, f, d), generator=gen, device=dev, dtype=bf) * 0.02
    w_gu_all = torch.empty((E, 2 * f, d), dtype=bf, device=dev)
    om.ordermoe_pack_gate_up(g, u, w_gu_all)
    del g, u
    dn = torch.randn((E, d, f), generator=gen, device=dev, dtype=bf) * 0.02
    w_dn_all = torch.empty_like(dn)
    om.ordermoe_pack_down(dn, w_dn_all)
    del dn
    sg = torch.randn((1, nsh * f, d), generator=gen, device=dev, dtype=bf) * 0.02
    su = torch.randn((1, nsh * f, d), generator=gen, device=dev, dtype=bf) * 0.02
    w_sh_gu = torch.empty((1, 2 * nsh * f, d), dtype=bf, device=dev)
    om.ordermoe_pack_gate_up(sg, su, w_sh_gu)
    del sg, su
    sd = torch.randn((1, d, nsh * f), generator=gen, device=dev, dtype=bf) * 0.02
    w_sh_dn = torch.empty_like(sd)
    om.ordermoe_pack_down(sd, w_sh_dn)
    del sd
    servers = []
    for m in range(M):
        local = [int(j) for j in np.nonzero(x_dep[m])[0]]
        sel = torch.tensor(local, dtype=torch.long, device=dev)
        w_gu, w_dn = w_gu_all[sel].contiguous(), w_dn_all[sel].contiguous()
        ex = om.make_experts(code, d, f, E, local, w_gu, w_dn, nsh, w_sh_gu, w_sh_dn)
        servers.append((ex, (w_gu, w_dn), torch.empty(len(local) + 2, dtype=torch.int32, device=dev)))
    x = _upload(cfg, torch, wl.tokens(cfg))
    loc = torch.from_numpy(wl.token_locations(cfg)).to(dev)
    qh = torch.zeros(T, dtype=torch.float32, device=dev)
    out = om.alloc_route_out(T, k, M, dev)
    ws_r = torch.empty(om.ordermoe_route_workspace_size(T, k, M), dtype=torch.uint8, device=dev)
    ws_f = torch.empty(max(om.ordermoe_forward_workspace_size(sv[0], T, k) for sv in servers),
                       dtype=torch.uint8, device=dev)
    y = torch.empty((T, d), dtype=bf, device=dev)
    ysum = torch.empty((T, d), dtype=torch.float32, device=dev)
    points, y0 = [], None
    for qbar in wl.C4_QBAR_SWEEP:
        layer = om.make_layer(code, d, E, k, M, 15, lm["w_router"], lm["tabs_dev"], qbar, cfg.omega_Q,
                              cfg.pin_local_exact, cfg.allow_sub, cfg.renorm)
        om.ordermoe_route_select(layer, x, T, loc, qh, out, ws_r)
        ysum.zero_()
        for m, (ex, _, ro) in enumerate(servers):
            om.ordermoe_local_moe_forward(ex, x, T, k, out["w"], out["exec_k"], out["exec_m"], loc, m, y,
                                          ro, ws_f)
            ysum += y.float()
        cnt = out["counters"].cpu().numpy()
        if y0 is None:
            y0 = ysum.clone()          # the sweep starts at Qbar = 0: exact top-k MoE
        rel = float(torch.linalg.norm(ysum - y0) / torch.linalg.norm(y0))
        points.append({"Qbar": qbar, "remote_ratio": float(cnt[6]) / (T * k),
                       "classes_LE_LS_RE_RS": [int(v) for v in cnt[:4]],
                       "flagged_tokens": int(cnt[4]), "rel_deviation": rel})
    return {"workload": cfg.name, "servers": M, "points": points,
            "weights": "device draws, N(0, 0.02^2) bf16; routers, tokens and deployment as the layer"}


def _stream_base(torch, om, cfg):
    """The stack's similarity models through the library: per layer the
    similarity build on the GPU (with the top-1 of each calibration token),
    then the transition estimate (eq 41) on the host.  None of it depends on
    the servers or their memory."""
    import workloads as wl
    dev = "cuda"
    up = lambda a: torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).to(dev)
    N, E, k = cfg.N, cfg.E, cfg.k
    W = wl.stream_routers(cfg)
    theta = [om.ordermoe_theta_layer(l + 1, N, cfg.theta_min, cfg.theta_max) for l in range(N)]
    ws = torch.empty(om.ordermoe_similarity_workspace_size(cfg.T_cal, cfg.d, E), dtype=torch.uint8,
                     device=dev)
    top1 = torch.empty((N, cfg.T_cal), dtype=torch.int32, device=dev)
    w_router, models = [], []
    for l, Xc in enumerate(wl.stream_calibration(cfg)):
        w_router.append(up(W[l]))
        models.append(om.ordermoe_build_similarity(up(Xc), w_router[l], k, theta[l], cfg.alpha_f, ws,
                                                   top1=top1[l]))
    del ws
    P = om.ordermoe_estimate_transitions(top1.cpu().numpy(), E)
    return dict(theta=theta, w_router=w_router, models=models, P=P,
                X=[up(x) for x in wl.stream_tokens(cfg)])


# deployments of the variant study: Algorithm 1 and its ablations, and the two
# deployment baselines of Section VI-A
DEPLOYMENTS = ("ordermoe", "no_redundancy", "no_dispersion", "popularity", "random")


def _stream_deploy(om, cfg, base, mode="ordermoe", net=None):
    """A deployment of the stack on cfg.M servers of cfg.capacity (Algorithm 1
    unless `mode` names a variant) with the network and per-step costs of
    eq 37-38."""
    import workloads as wl
    N, E, M = cfg.N, cfg.E, cfg.M
    ones, C = [np.ones(E)] * N, np.array(cfg.capacity)
    if mode == "random":
        x_dep, _ = om.ordermoe_place_random(ones, C, cfg.seed, 1)
    else:
        groups = [m["group_of"] for m in base["models"]]
        if mode == "popularity":      # replicas by activation frequency (counts over the calibration set)
            w = [m["counts"] / max(1, int(np.sum(m["counts"]))) for m in base["models"]]
        else:
            w = [m["importance"] for m in base["models"]]
        lam = 1.0 if mode == "no_dispersion" else cfg.lambda1
        red = {"no_redundancy": 0, "popularity": 2}.get(mode, 1)
        x_dep, _ = om.ordermoe_place(groups, w, ones, C, np.full(M, 1.0 / M), lam, red)
    net = wl.network(cfg) if net is None else net
    c = np.full(E, 6.0 * cfg.d * cfg.f)
    dref = float(np.mean(c)) / float(np.mean(net.F))
    z_bits = 8.0 * cfg.d * cfg.bytes_per_el
    return dict(base, x_dep=x_dep, net=net, c=c, dref=dref, z_bits=z_bits, deployment=mode)


def _stream_model(torch, om, cfg):
    """The stack's offline model: similarity models, transitions and the joint
    deployment (Algorithm 1)."""
    return _stream_deploy(om, cfg, _stream_base(torch, om, cfg))


def _group_coverage(cfg, sm):
    """Local group coverage: over layers and servers, the share of the layer's
    similarity groups with at least one member on the server (the y of eq 32,
    averaged)."""
    cov = []
    for l, md in enumerate(sm["models"]):
        g = np.asarray(md["group_of"])
        ng = len(set(g.tolist()))
        for m in range(cfg.M):
            cov.append(len(set(g[sm["x_dep"][l][m] == 1].tolist())) / ng)
    return float(np.mean(cov))


def _stream_lookahead(om, cfg, sm, H, omega_T, omega_Q, allow_sub=None):
    """Phi_l^(H-1) of every layer (eq 42) by the library."""
    N = cfg.N
    return om.ordermoe_build_lookahead(H, sm["P"], np.stack(sm["x_dep"]), np.stack([m["sim"] for m in sm["models"]]),
                                      np.stack([m["group_of"] for m in sm["models"]]),
                                      np.array(sm["theta"], np.float32), np.full(N, sm["z_bits"]),
                                      np.tile(sm["c"], (N, 1)), np.full(N, sm["dref"]), sm["net"].B,
                                      sm["net"].tau, sm["net"].F, omega_T, omega_Q, cfg.Qbar,
                                      cfg.pin_local_exact, cfg.allow_sub if allow_sub is None else allow_sub)


def _device_lookahead_inputs(torch, cfg, sm):
    """The look-ahead inputs of the stack as device tensors (for the device build)."""
    N = cfg.N
    d = lambda a, t: torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=t))).cuda()
    return dict(P=d(sm["P"], np.float64), x=d(np.stack(sm["x_dep"]), np.uint8),
                sim=d(np.stack([m["sim"] for m in sm["models"]]), np.float32),
                group_of=d(np.stack([m["group_of"] for m in sm["models"]]), np.int32),
                theta=d(np.array(sm["theta"], np.float32), np.float32), z_bits=d(np.full(N, sm["z_bits"]), np.float64),
                c=d(np.tile(sm["c"], (N, 1)), np.float64), d_ref=d(np.full(N, sm["dref"]), np.float64),
                B=d(sm["net"].B, np.float64), tau=d(sm["net"].tau, np.float64), F=d(sm["net"].F, np.float64))


def _device_lookahead(torch, om, cfg, inputs, H, omega_T, omega_Q, reps=5):
    """Phi^(H-1) built on the device (eq 41-42): the result and the average time
    of one build (HIP events around `reps` builds)."""
    phi = om.ordermoe_build_lookahead_device(H, omega_T=omega_T, omega_Q=omega_Q, Qbar=cfg.Qbar,
                                             pin_local_exact=cfg.pin_local_exact, allow_sub=cfg.allow_sub, **inputs)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        om.ordermoe_build_lookahead_device(H, omega_T=omega_T, omega_Q=omega_Q, Qbar=cfg.Qbar,
                                           pin_local_exact=cfg.pin_local_exact, allow_sub=cfg.allow_sub,
                                           phi=phi, **inputs)
    e1.record()
    torch.cuda.synchronize()
    return phi.cpu().numpy(), e0.elapsed_time(e1) / reps * 1e3


def _stream_layers(torch, om, cfg, sm, phi, omega_T, omega_Q, allow_sub=None):
    """Per layer: the decision tables (eq 7, 18, 37-38 with Phi) on the device
    and the layer struct."""
    out = []
    for l in range(cfg.N):
        md = sm["models"][l]
        tabs = om.ordermoe_build_tables(md["sim"], md["group_of"], sm["theta"][l], sm["x_dep"][l], sm["net"].B,
                                        sm["net"].tau, sm["net"].F, sm["z_bits"], sm["c"], sm["dref"], omega_T,
                                        phi[l])
        tdev = {n: torch.from_numpy(np.ascontiguousarray(v)).to("cuda") for n, v in tabs.items()
                if n != "srvmask"}
        tdev["srvmask"] = torch.from_numpy(tabs["srvmask"].view(np.int32)).to("cuda")
        L = om.make_layer(om.BF16, cfg.d, cfg.E, cfg.k, cfg.M, 15, sm["w_router"][l], tdev, cfg.Qbar, omega_Q,
                          cfg.pin_local_exact, cfg.allow_sub if allow_sub is None else allow_sub, cfg.renorm)
        out.append((L, tdev))
    return out


def _route_chain(torch, om, cfg, sm, layers, qh0=None):
    """The route/select chain through the stack for the decode batch (the
    location and accumulated loss carried on the device); per layer the host
    copies of the decisions and counters."""
    T, k, M = cfg.T, cfg.k, cfg.M
    loc = torch.zeros(T, dtype=torch.uint8, device="cuda")
    qh = torch.zeros(T, dtype=torch.float32, device="cuda") if qh0 is None else qh0
    ws = torch.empty(om.ordermoe_route_workspace_size(T, k, M), dtype=torch.uint8, device="cuda")
    recs = []
    for l, (L, _) in enumerate(layers):
        out = om.alloc_route_out(T, k, M, "cuda")
        om.ordermoe_route_select(L, sm["X"][l], T, loc, qh, out, ws)
        recs.append((loc, out))
        loc, qh = out["loc_out"], out["qhat_out"]
    torch.cuda.synchronize()
    return [dict(loc_in=li.cpu().numpy(), exec_m=o["exec_m"].cpu().numpy(), exec_k=o["exec_k"].cpu().numpy(),
                 counters=o["counters"].cpu().numpy(), qhat_out=o["qhat_out"].cpu().numpy()) for li, o in recs]


def _simulate(cfg, sm, recs):
    """The library's delay simulator (eq 13-17, eq 22) over the realized
    decisions of the chain: per token the delay of its executed slots along
    its trajectory (seconds), per server the FLOP it executed, and the
    transfer and slot counts."""
    from paper_2607_17154_amd import ordermoe as om
    em = np.stack([r["exec_m"].reshape(cfg.T, cfg.k) for r in recs])
    ek = np.stack([r["exec_k"].reshape(cfg.T, cfg.k) for r in recs])
    net = sm["net"]
    return om.ordermoe_simulate_delay(recs[0]["loc_in"], em, ek, [sm["c"]] * cfg.N, [sm["z_bits"]] * cfg.N,
                                      net.B, net.tau, net.F)


def _token_delays(cfg, sm, recs):
    return _simulate(cfg, sm, recs)["delay"]


def _trajectory_metrics(cfg, sm, recs):
    """Along the realized trajectories (the simulator): the mean modeled delay
    per token, cross-server transfers (distinct token-destination pairs per
    layer) and their traffic per 1000 tokens, the server workload imbalance
    (max over mean of eq 22), slot classes, the budget used at the end."""
    T = cfg.T
    sim = _simulate(cfg, sm, recs)
    cls = np.zeros(4, np.int64)
    for r in recs:
        cls += r["counters"][:4].astype(np.int64)
    slots = cls.sum()
    work = sim["work"]
    return {"delay_ms_per_token": float(sim["delay"].mean() * 1e3),
            "transfers_per_token_layer": sim["transfers"] / (T * cfg.N),
            "traffic_MB_per_1000_tokens": sim["traffic_bytes"] / T * 1000 / 1e6,
            "workload_max_over_mean": float(work.max() / work.mean()),
            "remote_ratio": float(cls[2] + cls[3]) / slots, "classes_LE_LS_RE_RS": [int(v) for v in cls],
            "budget_used": float(np.mean(recs[-1]["qhat_out"]) / cfg.Qbar)}


def _horizon_sweep(torch, om):
    """Look-ahead depth sweep (Fig. 7 of the paper) on the 32-layer decode stack,
    at memory ratios 2.0 and 1.0: for H = 1 .. 5 the library builds Phi^(H-1)
    (eq 42) on the host, then the
    route/select chain runs through the 32 layers for the 64-token batch.
    Reports the modeled delay and cross-server transfers of the realized
    trajectories, slot classes, budget used, and the time of the Phi build on
    the host and on the device (the device build checked equal to the host's;
    the per-token decision cost on the GPU does not depend on H: Phi is a
    table lookup)."""
    import workloads as wl
    points = []
    # memory ratio 2.0 (the paper's default: every server then holds a member of
    # every group) and 1.0 (each server holds half of the groups)
    for ratio in (2.0, 1.0):
        cfg = wl.C5_STREAM.with_(memory_ratio=ratio)
        sm = _stream_model(torch, om, cfg)
        dev_in = _device_lookahead_inputs(torch, cfg, sm)
        for H in (1, 2, 3, 4, 5):
            t0 = time.perf_counter()
            phi = _stream_lookahead(om, cfg, sm, H, cfg.omega_T, cfg.omega_Q)
            t_phi = time.perf_counter() - t0
            phi_d, us_d = _device_lookahead(torch, om, cfg, dev_in, H, cfg.omega_T, cfg.omega_Q)
            layers = _stream_layers(torch, om, cfg, sm, phi, cfg.omega_T, cfg.omega_Q)
            met = _trajectory_metrics(cfg, sm, _route_chain(torch, om, cfg, sm, layers))
            met.update(memory_ratio=ratio, H=H, phi_build_ms=t_phi * 1e3, phi_build_device_us=us_d,
                       phi_device_equals_host=bool(np.array_equal(phi_d, np.stack(phi))))
            points.append(met)
        del sm
    return {"workload": wl.C5_STREAM.name, "points": points}


def _run_variant(torch, om, cfg, sm, H, allow_sub):
    phi = _stream_lookahead(om, cfg, sm, H, cfg.omega_T, cfg.omega_Q, allow_sub=allow_sub)
    layers = _stream_layers(torch, om, cfg, sm, phi, cfg.omega_T, cfg.omega_Q, allow_sub=allow_sub)
    met = _trajectory_metrics(cfg, sm, _route_chain(torch, om, cfg, sm, layers))
    cls = met["classes_LE_LS_RE_RS"]
    met.update(local_ratio=(cls[0] + cls[1]) / max(1, sum(cls)), group_coverage=_group_coverage(cfg, sm),
               H=H, allow_sub=allow_sub, deployment=sm["deployment"])
    return met


def _variants(torch, om):
    """The paper's in-method variants and deployment baselines (Section VI-A,
    Fig. 4, 5, 9, 10, 12a) on the 32-layer decode stack, every one through the
    same route/select kernel and host tables: per variant the modeled delay
    along the realized trajectories (eq 37), cross-server transfers, slot
    classes, budget used and local group coverage.
      * variants, at the stack's per-token budget and at one that lasts the
        stack: full OrderMoE (H = 3); without look-ahead (H = 1); without
        redundancy; without same-group dispersion (lambda2 = 0); Similarity
        Deployment without Substitute (exact only); Local Substitute Only;
        Popularity-based Replication; Random Deployment;
      * memory ratio 1.0 .. 3.0, Algorithm 1 against popularity replication
        (Fig. 9: local group coverage and delay);
      * 4 .. 16 servers at memory ratio 2.0, OrderMoE against exact-only
        execution on the same deployment (Fig. 12a); servers 0..M-1 are the
        leading rows of one 16-server network, so adding servers keeps the
        others' links and speeds."""
    import workloads as wl
    cfg = wl.C5_STREAM
    base = _stream_base(torch, om, cfg)
    H = cfg.H
    out = {"workload": cfg.name, "H": H}
    runs = [("ordermoe", "ordermoe", H, 1), ("without_lookahead", "ordermoe", 1, 1),
            ("without_redundancy", "no_redundancy", H, 1), ("without_dispersion", "no_dispersion", H, 1),
            ("without_substitute", "ordermoe", H, 0), ("local_substitute_only", "ordermoe", H, 2),
            ("popularity_replication", "popularity", H, 1), ("random_deployment", "random", H, 1)]
    deps, rows = {}, []
    # the stack's budget (Q-bar = 1.0: used up near layer 16) and one that lasts the stack
    for qbar in (cfg.Qbar, 2.5):
        cq = cfg.with_(Qbar=qbar)
        for name, dep, h, sub in runs:
            if dep not in deps:
                deps[dep] = _stream_deploy(om, cfg, base, dep)
            met = _run_variant(torch, om, cq, deps[dep], h, sub)
            met.update(variant=name, Qbar=qbar)
            rows.append(met)
    out["variants"] = rows
    out["copies_per_expert_layer0"] = {n: np.bincount(d["x_dep"][0].sum(axis=0)).tolist() for n, d in deps.items()}
    del deps
    mem = []
    for ratio in (1.0, 1.5, 2.0, 2.5, 3.0):
        c = cfg.with_(memory_ratio=ratio)
        for dep in ("ordermoe", "popularity"):
            met = _run_variant(torch, om, c, _stream_deploy(om, c, base, dep), H, 1)
            met["memory_ratio"] = ratio
            mem.append(met)
    out["memory_ratio_sweep"] = mem
    net16 = wl.network(cfg, M=16)
    srv = []
    for M in (4, 8, 12, 16):
        c = cfg.with_(M=M)
        net = wl.Network(B=net16.B[:M, :M].copy(), tau=net16.tau[:M, :M].copy(), F=net16.F[:M].copy())
        sm = _stream_deploy(om, c, base, "ordermoe", net=net)
        for sub in (1, 0):
            met = _run_variant(torch, om, c, sm, H, sub)
            met["servers"] = M
            srv.append(met)
    out["server_sweep"] = srv
    return out


def _property3(torch, om, T: int = 1024, H: int = 3):
    """Statistical check of Property 3 (the look-ahead selection is no worse
    than the myopic one in expectation when the calibration transitions match
    the runtime routing): the 32-layer stack at memory ratio 1.0 (each server
    holds half of the groups, so the choice between servers matters), T
    independent decode tokens drawn by the same generator as the calibration
    tokens, each run through the chain with H = 1 and with H; the per-token
    modeled delays (eq 13-17 along the realized trajectories) are compared
    in pairs."""
    import workloads as wl
    cfg = wl.C5_STREAM.with_(memory_ratio=1.0, T=T)
    sm = _stream_deploy(om, cfg, _stream_base(torch, om, cfg))
    dl = {}
    for h in (1, H):
        phi = _stream_lookahead(om, cfg, sm, h, cfg.omega_T, cfg.omega_Q)
        recs = _route_chain(torch, om, cfg, sm, _stream_layers(torch, om, cfg, sm, phi, cfg.omega_T, cfg.omega_Q))
        dl[h] = _simulate(cfg, sm, recs)["delay"]
    diff = (dl[H] - dl[1]) * 1e3
    se = float(diff.std(ddof=1) / np.sqrt(T))
    return {"workload": cfg.name, "memory_ratio": 1.0, "tokens": T, "H": H,
            "delay_ms_per_token_H1": float(dl[1].mean() * 1e3), "delay_ms_per_token_H": float(dl[H].mean() * 1e3),
            "paired_diff_ms_mean": float(diff.mean()), "paired_diff_ms_stderr": se,
            "paired_diff_ms_ci95": [float(diff.mean() - 1.96 * se), float(diff.mean() + 1.96 * se)],
            "tokens_better": int((diff < 0).sum()), "tokens_worse": int((diff > 0).sum()),
            "tokens_equal": int((diff == 0).sum())}


def _weight_adaptation(torch, om, windows: int = 14, kappa: float = 0.1):
    """Weight adaptation (eq 45) as a host control loop on the 32-layer decode
    stack (H = 3): each observation window is one decode step of the 64-token
    batch through the stack.  After a window, T_bar = mean over tokens of the
    modeled delay over the delay of pure exact execution on the same
    deployment (the exact-only chain, allow_sub = 0), Q_bar = mean accumulated
    loss over the per-token budget (eq 23's normalisation); the library's
    eq-45 update gives the next (omega_Q, omega_T), with which Phi and the cost
    tables are rebuilt."""
    import workloads as wl
    cfg = wl.C5_STREAM
    sm = _stream_model(torch, om, cfg)
    phi_x = _stream_lookahead(om, cfg, sm, cfg.H, cfg.omega_T, cfg.omega_Q, allow_sub=0)
    t_ref = _token_delays(cfg, sm, _route_chain(torch, om, cfg, sm, _stream_layers(
        torch, om, cfg, sm, phi_x, cfg.omega_T, cfg.omega_Q, allow_sub=0)))
    wq, wt = cfg.omega_Q, cfg.omega_T
    trace = []
    for w in range(windows):
        phi = _stream_lookahead(om, cfg, sm, cfg.H, wt, wq)
        recs = _route_chain(torch, om, cfg, sm, _stream_layers(torch, om, cfg, sm, phi, wt, wq))
        t_bar = float(np.mean(_token_delays(cfg, sm, recs) / t_ref))
        q_bar = float(np.mean(recs[-1]["qhat_out"]) / cfg.Qbar)
        met = _trajectory_metrics(cfg, sm, recs)
        trace.append({"window": w, "omega_Q": wq, "omega_T": wt, "T_bar": t_bar, "Q_bar": q_bar,
                      "remote_ratio": met["remote_ratio"], "classes_LE_LS_RE_RS": met["classes_LE_LS_RE_RS"]})
        wq, wt = om.ordermoe_adapt_weights(wq, kappa, t_bar, q_bar)
    return {"workload": cfg.name, "kappa": kappa, "H": cfg.H,
            "exact_delay_ms_per_token": float(np.mean(t_ref) * 1e3), "windows": trace}


def _decode_stream(torch, om, steps: int = 10, warmup: int = 2):
    """Decode stream through a 32-layer stack of 128-expert top-8 layers (64
    tokens, hidden 4096, FFN 1536, 8 servers, memory ratio 2.0, H = 3), server
    0's share: per layer route/select with the location and accumulated loss
    carried on the device from the previous layer, then the local expert FFN.
    The offline model is built by the library (similarity on the device,
    transitions, deployment, look-ahead and tables on the host).  Expert
    weights of server 0 (32 per layer, 38.7 GB in all) are drawn on the device,
    N(0, 0.02^2) in bf16, and stay resident.  The 32-layer step is timed as a
    HIP graph replay (also with eager launches); reports time per layer and the
    HBM fraction of the weights the layer has to stream."""
    import workloads as wl
    cfg = wl.C5_STREAM
    dev = "cuda"
    up = lambda a: torch.from_numpy(wl.bf16_bits(a).view(np.int16)).view(torch.bfloat16).to(dev)
    N, E, M, T, k = cfg.N, cfg.E, cfg.M, cfg.T, cfg.k
    sm = _stream_model(torch, om, cfg)
    theta, w_router, models, x_dep, net, c, dref, z_bits = (
        sm[n] for n in ("theta", "w_router", "models", "x_dep", "net", "c", "dref", "z_bits"))
    phi = _stream_lookahead(om, cfg, sm, cfg.H, cfg.omega_T, cfg.omega_Q)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed)
    layers = []
    tab_layers = _stream_layers(torch, om, cfg, sm, phi, cfg.omega_T, cfg.omega_Q)
    for l in range(N):
        L, tdev = tab_layers[l]
        local = [int(j) for j in np.nonzero(x_dep[l][cfg.m0])[0]]
        n = len(local)
        g = torch.randn((n, cfg.f, cfg.d), generator=gen, device=dev, dtype=torch.bfloat16) * 0.02
        u = torch.randn((n, cfg.f, cfg.d), generator=gen, device=dev, dtype=torch.bfloat16) * 0.02
        w_gu = torch.empty((n, 2 * cfg.f, cfg.d), dtype=torch.bfloat16, device=dev)
        om.ordermoe_pack_gate_up(g, u, w_gu)
        del g, u
        dn = torch.randn((n, cfg.d, cfg.f), generator=gen, device=dev, dtype=torch.bfloat16) * 0.02
        w_dn = torch.empty_like(dn)
        om.ordermoe_pack_down(dn, w_dn)
        del dn
        ex = om.make_experts(om.BF16, cfg.d, cfg.f, E, local, w_gu, w_dn)
        out = om.alloc_route_out(T, k, M, dev)
        layers.append(dict(L=L, keep=(tdev, w_gu, w_dn), ex=ex, out=out, os=om.route_out_struct(out),
                           ro=torch.empty(n + 2, dtype=torch.int32, device=dev), n_local=n))
    xs = sm["X"]
    ws_r = torch.empty(om.ordermoe_route_workspace_size(T, k, M), dtype=torch.uint8, device=dev)
    ws_f = torch.empty(max(max(om.ordermoe_forward_workspace_size(Ld["ex"], T, k) for Ld in layers), 1),
                       dtype=torch.uint8, device=dev)
    y = torch.empty((T, cfg.d), dtype=torch.bfloat16, device=dev)
    loc0 = torch.zeros(T, dtype=torch.uint8, device=dev)
    q0 = torch.zeros(T, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    def step():
        loc, qh = loc0, q0
        for l in range(N):
            Ld = layers[l]
            o = Ld["out"]
            om.ordermoe_route_select(Ld["L"], xs[l], T, loc, qh, o, ws_r, out_struct=Ld["os"])
            om.ordermoe_local_moe_forward(Ld["ex"], xs[l], T, k, o["w"], o["exec_k"], o["exec_m"], loc,
                                          cfg.m0, y, Ld["ro"], ws_f)
            loc, qh = o["loc_out"], o["qhat_out"]

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    # the same step captured once in a HIP graph and replayed (no launch gaps)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    graph.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1)
    del graph
    # per-kernel averages from a separate pass (the events add a little time per launch)
    om.ordermoe_timing_read(reset=True)
    om.ordermoe_timing_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    om.ordermoe_timing_enable(False)
    kt = om.ordermoe_timing_read(reset=True)
    expert_bytes = 3 * cfg.f * cfg.d * 2
    active, rows, cls = [], [], np.zeros(4, np.int64)
    for Ld in layers:
        ro = Ld["ro"].cpu().numpy()
        active.append(int(np.sum(np.diff(ro[:Ld["n_local"] + 1]) > 0)))
        rows.append(int(ro[-1]))
        cls += Ld["out"]["counters"].cpu().numpy()[:4].astype(np.int64)
    w_bytes = expert_bytes * float(np.sum(active))
    other = N * (E * cfg.d * 2 + 2 * T * cfg.d * 2)        # routers, x in, y out
    us_layer = ms_graph / steps / N * 1e3
    us_layer_eager = ms / steps / N * 1e3
    gemm_us = sum(kt[n][0] / kt[n][1] for n in ("gemm_gate_up", "gemm_down")
                  if n in kt) * 1e3
    return {"workload": cfg.name, "layers": N, "tokens": T, "server": cfg.m0,
            "us_per_layer": us_layer, "us_per_layer_eager_launches": us_layer_eager,
            "ms_per_token_step": ms_graph / steps,
            "local_rows_per_layer": float(np.mean(rows)),
            "active_local_experts_per_layer": float(np.mean(active)),
            "classes_LE_LS_RE_RS": [int(v) for v in cls],
            "weight_bytes_per_layer": w_bytes / N,
            "hbm_frac_layer": (w_bytes + other) / (ms_graph / steps / 1e3) / 1e9 / PEAK_HBM_GBS,
            "hbm_frac_ffn_gemms": (w_bytes / N) / (gemm_us * 1e-6) / 1e9 / PEAK_HBM_GBS,
            "kernels_avg_us": {n: v[0] / v[1] * 1e3 for n, v in sorted(kt.items())}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--streams", type=int, default=2,
                    help="consecutive batches in flight, one HIP stream each (1: one batch at a time)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-simbuild", action="store_true",
                    help="skip the similarity-build measurement (65536 x 4096 calibration tokens)")
    ap.add_argument("--no-other-layers", action="store_true",
                    help="skip the Qwen-MoE- and DeepSeek-MoE-shaped layer measurements")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the quality-budget sweep of the DeepSeek-MoE-shaped layer")
    ap.add_argument("--no-horizon", action="store_true",
                    help="skip the look-ahead depth sweep H = 1..5 of the decode stack")
    ap.add_argument("--no-adapt", action="store_true",
                    help="skip the eq-45 weight-adaptation loop on the decode stack")
    ap.add_argument("--no-property3", action="store_true",
                    help="skip the paired look-ahead / myopic check of Property 3 on 1024 decode tokens")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the variant / baseline / memory-ratio / server-count study of the decode stack")
    ap.add_argument("--no-stream", action="store_true",
                    help="skip the 32-layer decode-stream measurement")
    ap.add_argument("--only", choices=("layer", "simbuild", "stream", "sweep", "horizon", "adapt",
                                       "variants", "property3"),
                    help="run one leg alone (for profiling): the layer step without the other "
                         "legs, or only the similarity build / decode stream (prints that leg's "
                         "JSON object)")
    ap.add_argument("--config", choices=("C2", "C3", "C4"), default="C2",
                    help="with --only layer: the layer to step (C2 Mixtral-shaped, the headline; C3 "
                         "Qwen-MoE-shaped; C4 DeepSeek-MoE-shaped), for profiling")
    ap.add_argument("--out", default=os.path.join(ROOT, "gpurun_out", "bench_full.json"),
                    help="file that receives every leg's results (stdout gets one compact line)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 1 GiB device copy (to scale rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.streams < 1:
        ap.error("--streams must be at least 1")
    if args.gpus != 1:
        print("bench.py measures one GPU: the layer runs one simulated server's experts on one "
              "MI355X; other servers are placement masks, so --gpus %d is not supported"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        _calibrate_copy(torch)
        return

    import workloads as wl
    from paper_2607_17154_amd import ordermoe as om
    if not os.path.exists(om.LIB_PATH):
        from paper_2607_17154_amd import build as _b
        _b.build()
    cfg = wl.C2
    if args.config != "C2":
        if args.only != "layer":
            print("--config applies to --only layer", file=sys.stderr)
            sys.exit(2)
        cfg = getattr(wl, args.config)
    torch.cuda.set_device(0)
    if args.only == "simbuild":
        print(json.dumps(_simbuild(torch, om)))
        return
    if args.only == "stream":
        print(json.dumps(_decode_stream(torch, om, steps=args.steps, warmup=args.warmup)))
        return
    if args.only == "sweep":
        print(json.dumps(_quality_sweep(torch, om)))
        return
    if args.only == "horizon":
        print(json.dumps(_horizon_sweep(torch, om)))
        return
    if args.only == "adapt":
        print(json.dumps(_weight_adaptation(torch, om)))
        return
    if args.only == "variants":
        print(json.dumps(_variants(torch, om)))
        return
    if args.only == "property3":
        print(json.dumps(_property3(torch, om)))
        return
    if args.only == "layer":
        args.no_simbuild = args.no_stream = args.no_cpu_baseline = args.no_other_layers = True
        args.no_sweep = args.no_horizon = args.no_adapt = args.no_variants = args.no_property3 = True
    print("bench: setting up %s" % cfg.name, file=sys.stderr, flush=True)
    st = _setup(cfg, torch, om)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        _step(cfg, st, om)
    torch.cuda.synchronize()
    # one batch at a time on one stream (no per-kernel events): the latency of a step
    ms_one = _timed_steps(cfg, [st], [torch.cuda.current_stream()], args.steps, torch, om)
    print("bench: %d steps on one stream in %.3f ms" % (args.steps, ms_one), file=sys.stderr, flush=True)
    # the timed steps, as a serving loop runs them: consecutive batches
    # alternate over --streams streams, so one batch's routing and row kernels
    # and the next batch's GEMM fill the CUs that the other batch's GEMM tails
    # leave idle
    ms, streams_equal = ms_one, True
    if args.streams > 1:
        ms, streams_equal = _pipelined(cfg, st, torch, om, args.streams, args.steps, args.warmup)
        if not streams_equal:
            print("bench: outputs differ between streams", file=sys.stderr, flush=True)
            sys.exit(1)
    print("bench: %d steps over %d stream(s) in %.3f ms" % (args.steps, args.streams, ms), file=sys.stderr,
          flush=True)
    # the same number of steps again with the library's HIP events around every
    # kernel launch (on the launch stream), for the per-kernel durations; the
    # events themselves add time between the kernels, so this pass is not the
    # step time
    om.ordermoe_timing_read(reset=True)
    om.ordermoe_timing_enable(True)
    e2, e3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e2.record()
    for _ in range(args.steps):
        _step(cfg, st, om)
    e3.record()
    torch.cuda.synchronize()
    om.ordermoe_timing_enable(False)
    ms_events = e2.elapsed_time(e3)
    kt = om.ordermoe_timing_read(reset=True)
    print("bench: %d steps with per-kernel events in %.3f ms" % (args.steps, ms_events), file=sys.stderr,
          flush=True)

    rows = st["ro"].cpu().numpy()
    R = int(rows[-1])
    counters = st["out"]["counters"].cpu().numpy()
    # the gate/up GEMM is one launch per step: whole rounds of 256 x 256 tiles,
    # then the remaining tiles split along K over all workgroups
    gu_avg_s = kt["gemm_gate_up"][0] / kt["gemm_gate_up"][1] / 1e3
    # gate and up projections: 2 d 2f per routed row, 2 d 2 n_shared f per row of the shared group
    r_routed = int(rows[len(st["local"])])
    gu_flops = 2.0 * cfg.d * 2 * cfg.f * (r_routed + max(cfg.n_shared, 1) * (R - r_routed))
    achieved = gu_flops / gu_avg_s / 1e12
    ms_step = ms / args.steps
    metric = "MoE-layer tokens/s on 1 MI355X (route+substitute+grouped FFN); % MFMA peak"
    roofline = {"bound": "mfma", "kernel": "gemm_gate_up", "achieved": achieved,
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                "traffic": _measured_traffic() if cfg is wl.C2 else None, "flop_per_launch": gu_flops,
                "avg_launch_us": gu_avg_s * 1e6}
    why = ("the Mixtral-8x7B-shaped layer: the paper's headline model (its latency, traffic and "
           "throughput results are on Mixtral-8x7B); the DeepSeek-shaped layer carries more FLOPs "
           "but is not a model the paper evaluates") if cfg is wl.C2 else "a profiling run of another layer"
    config = {"workload": cfg.name, "why": why, "streams": args.streams,
              "tokens": cfg.T, "hidden": cfg.d, "experts": cfg.E, "ffn": cfg.f, "top_k": cfg.k,
              "servers": cfg.M, "server": cfg.m0, "local_experts": st["local"], "local_rows": R,
              "classes_LE_LS_RE_RS": [int(v) for v in counters[:4]],
              "flagged_tokens": int(counters[4]), "remote_transfers": int(counters[5])}
    res = {
        "metric": metric,
        "value": cfg.T * args.steps / (ms / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; random-init expert and router weights of the layer shape)",
        "config": config,
        "roofline": roofline,
        "kernels_avg_us": {k: v[0] / v[1] * 1e3 for k, v in sorted(kt.items())},
        "ms_per_step_one_stream": ms_one / args.steps,
        "ms_per_step_with_kernel_events": ms_events / args.steps,
        "mfma_frac_ffn": (1.5 * gu_flops) / (ms_step / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
    }
    if not args.no_simbuild:
        print("bench: similarity build", file=sys.stderr, flush=True)
        res["similarity_build"] = _simbuild(torch, om)
    if not args.no_other_layers:
        print("bench: C3 and C4 layers", file=sys.stderr, flush=True)
        res["other_layers"] = _other_layers(torch, om, n_streams=args.streams)
    if not args.no_sweep:
        print("bench: quality-budget sweep", file=sys.stderr, flush=True)
        res["quality_sweep"] = _quality_sweep(torch, om)
        torch.cuda.empty_cache()
    if not args.no_horizon:
        print("bench: look-ahead depth sweep", file=sys.stderr, flush=True)
        res["horizon_sweep"] = _horizon_sweep(torch, om)
        torch.cuda.empty_cache()
    if not args.no_adapt:
        print("bench: weight adaptation", file=sys.stderr, flush=True)
        res["weight_adaptation"] = _weight_adaptation(torch, om)
        torch.cuda.empty_cache()
    if not args.no_property3:
        print("bench: Property 3 check", file=sys.stderr, flush=True)
        res["property3"] = _property3(torch, om)
        torch.cuda.empty_cache()
    if not args.no_variants:
        print("bench: variants and baselines", file=sys.stderr, flush=True)
        res["variants"] = _variants(torch, om)
        torch.cuda.empty_cache()
    if not args.no_stream:
        print("bench: decode stream", file=sys.stderr, flush=True)
        del st["experts"], st["keep"]
        torch.cuda.empty_cache()
        res["decode_stream"] = _decode_stream(torch, om)
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        res["cpu_baseline"] = _cpu_baseline(cfg, st, args.cpu_seconds)
    # every leg goes to the results file; stdout gets one compact line
    out_path = args.out
    os.makedirs(os.path.dirname(os.path.abspath(out_path)), exist_ok=True)
    with open(out_path, "w") as fh:
        json.dump(res, fh, indent=1)
    print("bench: all legs written to %s" % out_path, file=sys.stderr, flush=True)
    print(json.dumps(_compact(res, out_path)))


def _compact(res: dict, out_path: str) -> dict:
    """The headline line: the metric on the Mixtral-shaped layer, the gate/up
    GEMM's roofline, the CPU oracle, and one figure per other leg."""
    line = {k: res[k] for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                                "higher_is_better", "scaling", "vs_baseline", "dtype", "data")}
    cfgd = res["config"]
    line["config"] = {k: cfgd[k] for k in ("workload", "why", "streams", "local_rows", "classes_LE_LS_RE_RS",
                                           "flagged_tokens")}
    line["ms_per_step_one_stream"] = round(res["ms_per_step_one_stream"], 4)
    rf = res["roofline"]
    line["roofline"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in rf.items()}
    ka = res["kernels_avg_us"]
    line["kernels_avg_us"] = {k: round(v, 1) for k, v in ka.items()}
    if "cpu_baseline" in res:
        cb = res["cpu_baseline"]
        line["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
        line["cpu_baseline"]["os_cpu_count"] = os.cpu_count()
        line["cpu_baseline"]["OMP_NUM_THREADS"] = os.environ.get("OMP_NUM_THREADS")
    other = {}
    for key, v in res.get("other_layers", {}).items():
        other[key] = {"ms_per_step": round(v["ms_per_step"], 4), "tokens_per_s": round(v["tokens_per_s"]),
                      "ms_per_step_one_stream": round(v["ms_per_step_one_stream"], 4),
                      "gate_up_frac": round(v["gemm_gate_up_frac"], 3),
                      "down_frac": round(v["gemm_down_frac"], 3),
                      "route_hbm_frac": round(v["route_hbm_frac"], 3)}
    if "similarity_build" in res:
        sb = res["similarity_build"]
        other["C5_build"] = {"device_us": round(sb["device_us"], 1), "hbm_frac": round(sb["hbm_frac"], 3)}
    if "decode_stream" in res:
        ds = res["decode_stream"]
        other["C5_stream"] = {"us_per_layer": round(ds["us_per_layer"], 1),
                              "hbm_frac_ffn_gemms": round(ds["hbm_frac_ffn_gemms"], 3)}
    if other:
        line["other"] = other
    line["details"] = os.path.relpath(out_path, ROOT) if out_path.startswith(ROOT) else out_path
    return line


if __name__ == "__main__":
    main()
