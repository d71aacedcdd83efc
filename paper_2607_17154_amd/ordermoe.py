"""ctypes binding of libordermoe.so (include/ordermoe.h).

Argument marshalling only: every function here takes torch tensors (device
buffers) or numpy arrays (host buffers), checks their dtype/size, and passes
their addresses to the C entry point of the same name.  All computation runs
in the library's HIP kernels and host C++; there is no Python or PyTorch
fallback.  Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libordermoe.so")

OK, EINVAL, EDTYPE, ECAPACITY, EHIP, EWORKSPACE = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
MAX_SERVERS, MAX_EXPERTS, MAX_TOPK, MAX_SUBS, MAX_LOCAL = 32, 256, 8, 15, 64
NOALLOC_SCRATCH_BYTES = 8 << 20
MARGIN_FLAG = 1.0e-4
CNT_LOCAL_EXACT, CNT_LOCAL_SUB, CNT_REMOTE_EXACT, CNT_REMOTE_SUB = 0, 1, 2, 3
CNT_FLAGGED, CNT_TRANSFERS, CNT_REMOTE_SLOTS, CNT_INVALID, NUM_COUNTERS = 4, 5, 6, 7, 8

# every symbol include/ordermoe.h declares
EXPORTS = ("ordermoe_last_error", "ordermoe_similarity_workspace_size", "ordermoe_build_similarity",
           "ordermoe_group_experts", "ordermoe_place", "ordermoe_build_tables",
           "ordermoe_build_lookahead", "ordermoe_route_workspace_size", "ordermoe_route_select",
           "ordermoe_forward_workspace_size", "ordermoe_local_moe_forward",
           "ordermoe_pack_gate_up", "ordermoe_pack_down", "ordermoe_timing_enable", "ordermoe_timing_read",
           "ordermoe_estimate_transitions", "ordermoe_theta_layer", "ordermoe_adapt_weights",
           "ordermoe_place_random", "ordermoe_simulate_delay", "ordermoe_lookahead_device_workspace_size",
           "ordermoe_build_lookahead_device", "ordermoe_transitions_device_workspace_size",
           "ordermoe_estimate_transitions_device", "ordermoe_route_select_noalloc")
TIMING_NAME = 64


class OrderMoEError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("ordermoe error %d: %s" % (code, msg))
        self.code = code


_P = ctypes.c_void_p
_I32, _I64, _F32, _F64, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_size_t


class Layer(ctypes.Structure):
    _fields_ = [("dtype", _I32), ("d", _I32), ("E", _I32), ("k", _I32), ("M", _I32), ("gmax", _I32),
                ("pin_local_exact", _I32), ("allow_sub", _I32), ("renorm", _I32),
                ("Qbar", _F32), ("omega_Q", _F32),
                ("w_router", _P), ("t1_k", _P), ("t1_q", _P), ("t1_n", _P), ("srvmask", _P), ("S", _P)]


class RouteOut(ctypes.Structure):
    _fields_ = [(n, _P) for n in ("idx", "w", "margin", "flag", "exec_k", "exec_m", "cls", "qhat_out",
                                  "loc_out", "dispatch", "dst_count", "counters")]


class Experts(ctypes.Structure):
    _fields_ = [("dtype", _I32), ("d", _I32), ("f", _I32), ("E", _I32), ("n_local", _I32),
                ("n_shared", _I32), ("local_experts", _P), ("w_gate_up", _P), ("w_down", _P),
                ("w_shared_gate_up", _P), ("w_shared_down", _P)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libordermoe.so is not built (expected at %s); build it with "
                          "`python -m paper_2607_17154_amd.build`" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    L.ordermoe_last_error.restype = ctypes.c_char_p
    L.ordermoe_last_error.argtypes = []
    L.ordermoe_similarity_workspace_size.restype = _SZ
    L.ordermoe_similarity_workspace_size.argtypes = [_I64, _I32, _I32]
    L.ordermoe_build_similarity.restype = ctypes.c_int
    L.ordermoe_build_similarity.argtypes = [_P, _I64, _I32, _P, _I32, _I32, _I32, _F32, _F64,
                                            _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
    L.ordermoe_estimate_transitions.restype = ctypes.c_int
    L.ordermoe_estimate_transitions.argtypes = [_I32, _I32, _I64, _P, _P]
    L.ordermoe_theta_layer.restype = ctypes.c_int
    L.ordermoe_theta_layer.argtypes = [_I32, _I32, _F64, _F64, _P]
    L.ordermoe_adapt_weights.restype = ctypes.c_int
    L.ordermoe_adapt_weights.argtypes = [_F64, _F64, _F64, _F64, _P, _P]
    L.ordermoe_group_experts.restype = ctypes.c_int
    L.ordermoe_group_experts.argtypes = [_I32, _P, _P, _F32, _F64, _P, _P, _P, _P]
    L.ordermoe_place.restype = ctypes.c_int
    L.ordermoe_place.argtypes = [_I32, _P, _I32, _P, _P, _P, _P, _P, _F64, _I32, _P, _P]
    L.ordermoe_place_random.restype = ctypes.c_int
    L.ordermoe_place_random.argtypes = [_I32, _P, _I32, _P, _P, ctypes.c_uint64, _I32, _P, _P]
    L.ordermoe_lookahead_device_workspace_size.restype = _SZ
    L.ordermoe_lookahead_device_workspace_size.argtypes = [_I32, _I32, _I32]
    L.ordermoe_build_lookahead_device.restype = ctypes.c_int
    L.ordermoe_build_lookahead_device.argtypes = [_I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                                  _P, _F64, _F64, _F32, _I32, _I32, _P, _P, _SZ, _P]
    L.ordermoe_transitions_device_workspace_size.restype = _SZ
    L.ordermoe_transitions_device_workspace_size.argtypes = [_I32, _I32]
    L.ordermoe_estimate_transitions_device.restype = ctypes.c_int
    L.ordermoe_estimate_transitions_device.argtypes = [_I32, _I32, _I64, _P, _P, _P, _SZ, _P]
    L.ordermoe_simulate_delay.restype = ctypes.c_int
    L.ordermoe_simulate_delay.argtypes = [_I32, _I64, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                          _P, _P]
    L.ordermoe_build_tables.restype = ctypes.c_int
    L.ordermoe_build_tables.argtypes = [_I32, _I32, _P, _P, _F32, _P, _P, _P, _P, _F64, _P, _F64,
                                        _F64, _P, _I32, _P, _P, _P, _P, _P]
    L.ordermoe_build_lookahead.restype = ctypes.c_int
    L.ordermoe_build_lookahead.argtypes = [_I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P,
                                           _P, _P, _P, _F64, _F64, _F32, _I32, _I32, _P]
    L.ordermoe_route_workspace_size.restype = _SZ
    L.ordermoe_route_workspace_size.argtypes = [_I64, _I32, _I32]
    L.ordermoe_route_select.restype = ctypes.c_int
    L.ordermoe_route_select.argtypes = [ctypes.POINTER(Layer), _P, _I64, _P, _P,
                                        ctypes.POINTER(RouteOut), _P, _SZ, _P]
    L.ordermoe_route_select_noalloc.restype = ctypes.c_int
    L.ordermoe_route_select_noalloc.argtypes = [ctypes.POINTER(Layer), _P, _I64, _P, _P,
                                                ctypes.POINTER(RouteOut), _P]
    L.ordermoe_forward_workspace_size.restype = _SZ
    L.ordermoe_forward_workspace_size.argtypes = [ctypes.POINTER(Experts), _I64, _I32]
    L.ordermoe_local_moe_forward.restype = ctypes.c_int
    L.ordermoe_local_moe_forward.argtypes = [ctypes.POINTER(Experts), _P, _I64, _I32, _P, _P, _P,
                                             _P, _I32, _P, _P, _P, _SZ, _P]
    L.ordermoe_pack_gate_up.restype = ctypes.c_int
    L.ordermoe_pack_gate_up.argtypes = [_I32, _I32, _I32, _I32, _P, _P, _P, _P]
    L.ordermoe_pack_down.restype = ctypes.c_int
    L.ordermoe_pack_down.argtypes = [_I32, _I32, _I32, _I32, _P, _P, _P]
    L.ordermoe_timing_enable.restype = ctypes.c_int
    L.ordermoe_timing_enable.argtypes = [_I32]
    L.ordermoe_timing_read.restype = ctypes.c_int
    L.ordermoe_timing_read.argtypes = [_I32, _P, _P, _P, _P, _I32]
    _lib = L
    return L


def last_error() -> str:
    return lib().ordermoe_last_error().decode()


def _check(rc: int):
    if rc != OK:
        raise OrderMoEError(rc, last_error())


# ---------------------------------------------------------------- helpers
def _host(a: Optional[np.ndarray], dtype, n: Optional[int] = None):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(a, dtype=dtype)
    if n is not None and arr.size != n:
        raise ValueError("host array has %d elements, expected %d" % (arr.size, n))
    return arr, arr.ctypes.data_as(_P)


def _dev(t, dtype=None, n: Optional[int] = None) -> int:
    """Address of a contiguous device tensor (0 for None)."""
    if t is None:
        return 0
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError("expected %s, got %s" % (dtype, t.dtype))
    if n is not None and t.numel() != n:
        raise ValueError("device tensor has %d elements, expected %d" % (t.numel(), n))
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def _torch_dtype(code: int):
    import torch
    return torch.bfloat16 if code == BF16 else torch.float32


# ---------------------------------------------------------------- entry points
def ordermoe_similarity_workspace_size(T_cal: int, d: int, E: int) -> int:
    return int(lib().ordermoe_similarity_workspace_size(T_cal, d, E))


def ordermoe_build_similarity(x_cal, w_router, topk: int, theta: float, alpha_f: float,
                              workspace, stream=None, top1=None) -> Dict[str, np.ndarray]:
    """Sim and counts on the device, grouping on the host (eq 3-5, 24-28).
    top1: optional int32 device tensor [T_cal] that receives each calibration
    token's top-1 expert."""
    import torch
    T_cal, d = x_cal.shape
    E = w_router.shape[0]
    code = BF16 if x_cal.dtype == torch.bfloat16 else F32
    sim_dev = torch.empty((E, E), dtype=torch.float32, device=x_cal.device)
    cnt_dev = torch.empty(E, dtype=torch.int64, device=x_cal.device)
    top1_p = _dev(top1, torch.int32, T_cal)
    sim_h = np.empty((E, E), np.float32)
    cnt_h = np.empty(E, np.int64)
    g = np.empty(E, np.int32)
    c = np.empty(E, np.int32)
    ng = np.zeros(1, np.int32)
    imp = np.empty(E, np.float64)
    _check(lib().ordermoe_build_similarity(
        _dev(x_cal, _torch_dtype(code)), T_cal, d, _dev(w_router, _torch_dtype(code), E * d), E, code,
        topk, theta, alpha_f, _dev(sim_dev), _dev(cnt_dev), top1_p, sim_h.ctypes.data_as(_P),
        cnt_h.ctypes.data_as(_P), g.ctypes.data_as(_P), c.ctypes.data_as(_P),
        ng.ctypes.data_as(_P), imp.ctypes.data_as(_P), _dev(workspace), workspace.numel(),
        _stream(stream)))
    K = int(ng[0])
    return dict(sim=sim_h, counts=cnt_h, group_of=g, centres=[int(v) for v in c[:K]],
                importance=imp, sim_dev=sim_dev, counts_dev=cnt_dev)


def ordermoe_estimate_transitions(top1: np.ndarray, E: int) -> np.ndarray:
    """P [N-1][E][E] from the top-1 experts [N][T_cal] of the same calibration
    tokens at consecutive layers (eq 41)."""
    t = np.ascontiguousarray(top1, dtype=np.int32)
    N, T_cal = t.shape
    P = np.zeros((max(N - 1, 0), E, E), dtype=np.float64)
    _check(lib().ordermoe_estimate_transitions(N, E, T_cal, t.ctypes.data_as(_P),
                                               P.ctypes.data_as(_P)))
    return P


def ordermoe_theta_layer(l: int, N: int, theta_min: float, theta_max: float) -> float:
    """theta_l of eq 6 (1-based l), as the float32 value the tables use."""
    out = np.zeros(1, np.float32)
    _check(lib().ordermoe_theta_layer(l, N, theta_min, theta_max, out.ctypes.data_as(_P)))
    return float(out[0])


def ordermoe_adapt_weights(omega_Q: float, kappa: float, T_bar: float, Q_bar: float):
    """(omega_Q, omega_T) after one eq-45 update."""
    wq = np.zeros(1, np.float64)
    wt = np.zeros(1, np.float64)
    _check(lib().ordermoe_adapt_weights(omega_Q, kappa, T_bar, Q_bar, wq.ctypes.data_as(_P),
                                        wt.ctypes.data_as(_P)))
    return float(wq[0]), float(wt[0])


def ordermoe_group_experts(sim: np.ndarray, counts: np.ndarray, theta: float, alpha_f: float):
    E = sim.shape[0]
    s, sp = _host(sim, np.float32, E * E)
    n, npt = _host(counts, np.int64, E)
    g = np.empty(E, np.int32)
    c = np.empty(E, np.int32)
    ng = np.zeros(1, np.int32)
    imp = np.empty(E, np.float64)
    _check(lib().ordermoe_group_experts(E, sp, npt, theta, alpha_f, g.ctypes.data_as(_P),
                                        c.ctypes.data_as(_P), ng.ctypes.data_as(_P),
                                        imp.ctypes.data_as(_P)))
    return g, [int(v) for v in c[:int(ng[0])]], imp


def ordermoe_place(group_of: Sequence[np.ndarray], importance: Sequence[np.ndarray],
                   p: Sequence[np.ndarray], C, pi, lambda1: float = 0.5, redundancy: int = 1):
    """Returns (list of [M, E_l] uint8 deployments, used memory [M])."""
    N = len(group_of)
    E_l = np.array([len(g) for g in group_of], dtype=np.int32)
    M = len(C)
    g, gp = _host(np.concatenate([np.asarray(v) for v in group_of]), np.int32)
    im, ip = _host(np.concatenate([np.asarray(v) for v in importance]), np.float64)
    pp, ppp = _host(np.concatenate([np.asarray(v) for v in p]), np.float64)
    Cc, Cp = _host(C, np.float64, M)
    pic, pip = _host(pi, np.float64, M)
    x = np.zeros(int(M * E_l.sum()), np.uint8)
    used = np.zeros(M, np.float64)
    _check(lib().ordermoe_place(N, E_l.ctypes.data_as(_P), M, gp, ip, ppp, Cp, pip, lambda1,
                                redundancy, x.ctypes.data_as(_P), used.ctypes.data_as(_P)))
    out, off = [], 0
    for e in E_l:
        out.append(x[off:off + M * e].reshape(M, e).copy())
        off += M * e
    return out, used


def ordermoe_place_random(p: Sequence[np.ndarray], C, seed: int, redundancy: int = 1):
    """Random Deployment: returns (list of [M, E_l] uint8 deployments, used memory [M])."""
    N = len(p)
    E_l = np.array([len(v) for v in p], dtype=np.int32)
    M = len(C)
    pp, ppp = _host(np.concatenate([np.asarray(v) for v in p]), np.float64)
    Cc, Cp = _host(C, np.float64, M)
    x = np.zeros(int(M * E_l.sum()), np.uint8)
    used = np.zeros(M, np.float64)
    _check(lib().ordermoe_place_random(N, E_l.ctypes.data_as(_P), M, ppp, Cp,
                                       int(seed) & 0xFFFFFFFFFFFFFFFF, redundancy,
                                       x.ctypes.data_as(_P), used.ctypes.data_as(_P)))
    out, off = [], 0
    for e in E_l:
        out.append(x[off:off + M * e].reshape(M, e).copy())
        off += M * e
    return out, used


def ordermoe_simulate_delay(loc0, exec_m, exec_k, c: Sequence[np.ndarray], z_bits, B, tau, F):
    """Delay per token (s), workload per server (FLOP), the location entering
    each layer [N][T] and the counts: dict(delay, work, loc, transfers,
    traffic_bytes, remote_slots, slots).  exec_m, exec_k: [N][T][k] host arrays."""
    em = np.ascontiguousarray(exec_m, dtype=np.uint8)
    N, T, k = em.shape
    ek = np.ascontiguousarray(exec_k, dtype=np.int32).reshape(N, T, k)
    M = len(F)
    E_l = np.array([len(v) for v in c], dtype=np.int32)
    l0, l0p = _host(loc0, np.uint8, T)
    cc, cp = _host(np.concatenate([np.asarray(v, dtype=np.float64) for v in c]), np.float64)
    zz, zp = _host(z_bits, np.float64, N)
    Bb, Bp = _host(B, np.float64, M * M)
    tt, tp = _host(tau, np.float64, M * M)
    FF, Fp = _host(F, np.float64, M)
    delay = np.zeros(T, np.float64)
    work = np.zeros(M, np.float64)
    stats = np.zeros(4, np.float64)
    loc = np.zeros((N, T), np.uint8)
    _check(lib().ordermoe_simulate_delay(N, T, k, M, E_l.ctypes.data_as(_P), l0p, em.ctypes.data_as(_P),
                                         ek.ctypes.data_as(_P), cp, zp, Bp, tp, Fp, delay.ctypes.data_as(_P),
                                         work.ctypes.data_as(_P), stats.ctypes.data_as(_P),
                                         loc.ctypes.data_as(_P)))
    return dict(delay=delay, work=work, loc=loc, transfers=int(stats[0]), traffic_bytes=float(stats[1]),
                remote_slots=int(stats[2]), slots=int(stats[3]))


def ordermoe_build_tables(sim: np.ndarray, group_of: np.ndarray, theta: float, x: np.ndarray,
                          B: np.ndarray, tau: np.ndarray, F: np.ndarray, z_bits: float,
                          c: np.ndarray, d_ref: float, omega_T: float,
                          phi: Optional[np.ndarray] = None, gmax: int = MAX_SUBS):
    """Host tables: dict(t1_k [E,gmax] i32, t1_q [E,gmax] f32, t1_n [E] i32,
    srvmask [E] u32, S [M,M,E] f32)."""
    M, E = x.shape
    s, sp = _host(sim, np.float32, E * E)
    g, gp = _host(group_of, np.int32, E)
    xx, xp = _host(x, np.uint8, M * E)
    Bb, Bp = _host(B, np.float64, M * M)
    tt, tp = _host(tau, np.float64, M * M)
    FF, Fp = _host(F, np.float64, M)
    cc, cp = _host(c, np.float64, E)
    ph, php = _host(phi, np.float64, M * E)
    out = dict(t1_k=np.empty((E, gmax), np.int32), t1_q=np.empty((E, gmax), np.float32),
               t1_n=np.empty(E, np.int32), srvmask=np.empty(E, np.uint32),
               S=np.empty((M, M, E), np.float32))
    _check(lib().ordermoe_build_tables(E, M, sp, gp, theta, xp, Bp, tp, Fp, z_bits, cp, d_ref,
                                       omega_T, php, gmax, *(out[n].ctypes.data_as(_P) for n in
                                                             ("t1_k", "t1_q", "t1_n", "srvmask", "S"))))
    return out


def ordermoe_build_lookahead(H: int, P: np.ndarray, x: np.ndarray, sim: np.ndarray,
                             group_of: np.ndarray, theta: np.ndarray, z_bits: np.ndarray,
                             c: np.ndarray, d_ref: np.ndarray, B: np.ndarray, tau: np.ndarray,
                             F: np.ndarray, omega_T: float, omega_Q: float, Qbar: float,
                             pin_local_exact: int = 1, allow_sub: int = 1) -> np.ndarray:
    """Phi [N, M, E] (eq 41-42).  P: [N-1, E, E]; x: [N, M, E]; sim: [N, E, E]."""
    N, M, E = x.shape
    arrs = [_host(P, np.float64, (N - 1) * E * E) if N > 1 else (None, None),
            _host(x, np.uint8, N * M * E), _host(sim, np.float32, N * E * E),
            _host(group_of, np.int32, N * E), _host(theta, np.float32, N),
            _host(z_bits, np.float64, N), _host(c, np.float64, N * E), _host(d_ref, np.float64, N),
            _host(B, np.float64, M * M), _host(tau, np.float64, M * M), _host(F, np.float64, M)]
    phi = np.empty((N, M, E), np.float64)
    _check(lib().ordermoe_build_lookahead(N, E, M, H, *(p for _, p in arrs), omega_T, omega_Q, Qbar,
                                          pin_local_exact, allow_sub, phi.ctypes.data_as(_P)))
    return phi


def ordermoe_build_lookahead_device(H: int, P, x, sim, group_of, theta, z_bits, c, d_ref, B, tau, F,
                                    omega_T: float, omega_Q: float, Qbar: float, pin_local_exact: int = 1,
                                    allow_sub: int = 1, phi=None, ws=None, stream=None):
    """Phi [N, M, E] float64 on the device (eq 41-42), equal to
    ordermoe_build_lookahead's.  Every argument array is a contiguous device
    tensor: P float64 [N-1, E, E] (None when N = 1), x uint8 [N, M, E], sim
    float32 [N, E, E], group_of int32 [N, E], theta float32 [N], z_bits, d_ref
    float64 [N], c float64 [N, E], B, tau float64 [M, M], F float64 [M]."""
    import torch
    N, M, E = x.shape
    if phi is None:
        phi = torch.empty((N, M, E), dtype=torch.float64, device=x.device)
    need = int(lib().ordermoe_lookahead_device_workspace_size(N, E, M))
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    f64 = torch.float64
    args = [_dev(P, f64, (N - 1) * E * E) if N > 1 else 0, _dev(x, torch.uint8, N * M * E),
            _dev(sim, torch.float32, N * E * E), _dev(group_of, torch.int32, N * E), _dev(theta, torch.float32, N),
            _dev(z_bits, f64, N), _dev(c, f64, N * E), _dev(d_ref, f64, N), _dev(B, f64, M * M),
            _dev(tau, f64, M * M), _dev(F, f64, M)]
    _check(lib().ordermoe_build_lookahead_device(N, E, M, H, *args, omega_T, omega_Q, Qbar, pin_local_exact,
                                                 allow_sub, _dev(phi, f64, N * M * E), _dev(ws), ws.numel(),
                                                 _stream(stream)))
    return phi


def ordermoe_estimate_transitions_device(top1, E: int, P=None, ws=None, stream=None):
    """P [N-1, E, E] float64 on the device (eq 41) from the device top-1
    experts top1 int32 [N, T_cal]; equal to ordermoe_estimate_transitions'."""
    import torch
    N, T_cal = top1.shape
    if P is None:
        P = torch.empty((max(N - 1, 0), E, E), dtype=torch.float64, device=top1.device)
    need = int(lib().ordermoe_transitions_device_workspace_size(N, E))
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=top1.device)
    _check(lib().ordermoe_estimate_transitions_device(N, E, T_cal, _dev(top1, torch.int32, N * T_cal),
                                                      _dev(P, torch.float64, (N - 1) * E * E) if N > 1 else 0,
                                                      _dev(ws), ws.numel(), _stream(stream)))
    return P


def ordermoe_route_workspace_size(T: int, k: int, M: int) -> int:
    return int(lib().ordermoe_route_workspace_size(T, k, M))


def make_layer(dtype: int, d: int, E: int, k: int, M: int, gmax: int, w_router, tables_dev: Dict,
               Qbar: float, omega_Q: float, pin_local_exact: int = 1, allow_sub: int = 1,
               renorm: int = 1) -> Layer:
    """ordermoe_layer from device tensors (tables_dev: t1_k, t1_q, t1_n, srvmask, S)."""
    import torch
    return Layer(dtype=dtype, d=d, E=E, k=k, M=M, gmax=gmax, pin_local_exact=pin_local_exact,
                 allow_sub=allow_sub, renorm=renorm, Qbar=Qbar, omega_Q=omega_Q,
                 w_router=_dev(w_router, _torch_dtype(dtype), E * d),
                 t1_k=_dev(tables_dev["t1_k"], torch.int32, E * gmax),
                 t1_q=_dev(tables_dev["t1_q"], torch.float32, E * gmax),
                 t1_n=_dev(tables_dev["t1_n"], torch.int32, E),
                 srvmask=_dev(tables_dev["srvmask"], torch.int32, E),
                 S=_dev(tables_dev["S"], torch.float32, M * M * E))


def alloc_route_out(T: int, k: int, M: int, device) -> Dict:
    import torch
    kw = dict(device=device)
    return dict(idx=torch.empty((T, k), dtype=torch.int32, **kw),
                w=torch.empty((T, k), dtype=torch.float32, **kw),
                margin=torch.empty(T, dtype=torch.float32, **kw),
                flag=torch.empty(T, dtype=torch.uint8, **kw),
                exec_k=torch.empty((T, k), dtype=torch.int32, **kw),
                exec_m=torch.empty((T, k), dtype=torch.uint8, **kw),
                cls=torch.empty((T, k), dtype=torch.uint8, **kw),
                qhat_out=torch.empty(T, dtype=torch.float32, **kw),
                loc_out=torch.empty(T, dtype=torch.uint8, **kw),
                dispatch=torch.empty(max(T * k, 1), dtype=torch.int32, **kw),
                dst_count=torch.empty(M, dtype=torch.int32, **kw),
                counters=torch.empty(NUM_COUNTERS, dtype=torch.int64, **kw))


def route_out_struct(o: Dict) -> RouteOut:
    return RouteOut(**{n: o[n].data_ptr() for n, _ in RouteOut._fields_})


def ordermoe_route_select(layer: Layer, x, T: int, loc_in, qhat_in, out: Dict, workspace,
                          stream=None, out_struct: Optional[RouteOut] = None):
    import torch
    if T > 0:
        _dev(x, _torch_dtype(layer.dtype), T * layer.d)
        _dev(loc_in, torch.uint8, T)
        _dev(qhat_in, torch.float32, T)
    s = out_struct if out_struct is not None else route_out_struct(out)
    _check(lib().ordermoe_route_select(ctypes.byref(layer), x.data_ptr() if T > 0 else 0, T,
                                       loc_in.data_ptr() if T > 0 else 0,
                                       qhat_in.data_ptr() if T > 0 else 0, ctypes.byref(s),
                                       _dev(workspace), workspace.numel(), _stream(stream)))


def ordermoe_route_select_noalloc(layer: Layer, x, T: int, loc_in, qhat_in, out: Dict, stream=None,
                                  out_struct: Optional[RouteOut] = None):
    """ordermoe_route_select with the library's fixed per-GPU scratch instead
    of a caller workspace (allocates nothing)."""
    import torch
    if T > 0:
        _dev(x, _torch_dtype(layer.dtype), T * layer.d)
        _dev(loc_in, torch.uint8, T)
        _dev(qhat_in, torch.float32, T)
    s = out_struct if out_struct is not None else route_out_struct(out)
    _check(lib().ordermoe_route_select_noalloc(ctypes.byref(layer), x.data_ptr() if T > 0 else 0, T,
                                               loc_in.data_ptr() if T > 0 else 0,
                                               qhat_in.data_ptr() if T > 0 else 0, ctypes.byref(s),
                                               _stream(stream)))


def make_experts(dtype: int, d: int, f: int, E: int, local_experts: Sequence[int], w_gate_up,
                 w_down, n_shared: int = 0, w_shared_gate_up=None, w_shared_down=None):
    """ordermoe_experts from device tensors; keeps the host id array alive."""
    ids = np.ascontiguousarray(np.asarray(local_experts, dtype=np.int32))
    s = Experts(dtype=dtype, d=d, f=f, E=E, n_local=len(ids), n_shared=n_shared,
                local_experts=ids.ctypes.data_as(_P) if len(ids) else None,
                w_gate_up=_dev(w_gate_up), w_down=_dev(w_down),
                w_shared_gate_up=_dev(w_shared_gate_up), w_shared_down=_dev(w_shared_down))
    s._ids = ids
    return s


def ordermoe_forward_workspace_size(experts: Experts, T: int, k: int) -> int:
    return int(lib().ordermoe_forward_workspace_size(ctypes.byref(experts), T, k))


def ordermoe_local_moe_forward(experts: Experts, x, T: int, k: int, w, exec_k, exec_m, loc_in,
                               server: int, y, row_offsets, workspace, stream=None):
    import torch
    if T > 0:
        _dev(x, _torch_dtype(experts.dtype), T * experts.d)
        _dev(y, _torch_dtype(experts.dtype), T * experts.d)
        _dev(w, torch.float32, T * k)
        _dev(exec_k, torch.int32, T * k)
        _dev(exec_m, torch.uint8, T * k)
        _dev(loc_in, torch.uint8, T)
    _dev(row_offsets, torch.int32, experts.n_local + 2)
    ptr = (lambda t: t.data_ptr() if T > 0 else 0)
    _check(lib().ordermoe_local_moe_forward(ctypes.byref(experts), ptr(x), T, k, ptr(w), ptr(exec_k),
                                            ptr(exec_m), ptr(loc_in), server, ptr(y),
                                            row_offsets.data_ptr(), _dev(workspace),
                                            workspace.numel(), _stream(stream)))


def ordermoe_pack_gate_up(w_gate, w_up, out, stream=None):
    """w_gate, w_up: [n, f, d] device tensors; out: [n, 2f, d]."""
    import torch
    n, f, d = w_gate.shape
    code = BF16 if w_gate.dtype == torch.bfloat16 else F32
    _check(lib().ordermoe_pack_gate_up(code, n, f, d, _dev(w_gate), _dev(w_up, w_gate.dtype, n * f * d),
                                       _dev(out, w_gate.dtype, 2 * n * f * d), _stream(stream)))


def ordermoe_pack_down(w_down, out, stream=None):
    """w_down: [n, d, f] device tensor; out: [n, d, f] (packed layout)."""
    import torch
    n, d, f = w_down.shape
    code = BF16 if w_down.dtype == torch.bfloat16 else F32
    _check(lib().ordermoe_pack_down(code, n, d, f, _dev(w_down), _dev(out, w_down.dtype, n * d * f),
                                    _stream(stream)))


def ordermoe_timing_enable(on: bool = True):
    _check(lib().ordermoe_timing_enable(1 if on else 0))


def ordermoe_timing_read(reset: bool = True) -> Dict[str, tuple]:
    """{kernel name: (total ms, launches)} since the last reset."""
    cap = 64
    names = ctypes.create_string_buffer(cap * TIMING_NAME)
    ms = np.zeros(cap, np.float64)
    n = np.zeros(cap, np.int64)
    cnt = np.zeros(1, np.int32)
    _check(lib().ordermoe_timing_read(cap, names, ms.ctypes.data_as(_P), n.ctypes.data_as(_P),
                                      cnt.ctypes.data_as(_P), 1 if reset else 0))
    out = {}
    for i in range(min(int(cnt[0]), cap)):
        nm = names.raw[i * TIMING_NAME:(i + 1) * TIMING_NAME].split(b"\0", 1)[0].decode()
        out[nm] = (float(ms[i]), int(n[i]))
    return out
