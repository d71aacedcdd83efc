"""Transition statistics (eq 41) and the look-ahead cost-to-go (eq 42) built on
the device, through the C ABI: against the oracle's transitions and Phi
(exact / within 1e-12 relative), and against the host library's bit for bit."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_17154_amd import ordermoe as om  # noqa: E402

from ._pipeline import stream_library_tables, with_horizon  # noqa: E402


def _dev(a, dtype=None):
    return torch.from_numpy(np.ascontiguousarray(a if dtype is None else a.astype(dtype))).cuda()


@pytest.mark.parametrize("N,E,T", [(5, 12, 3000), (32, 128, 2048), (3, 7, 0), (1, 8, 100)])
def test_device_transitions_equal_the_host_estimate(N, E, T):
    rng = np.random.default_rng(N * 1000 + E)
    top1 = rng.integers(0, E, size=(N, T)).astype(np.int32)
    if T > 50:
        top1[:, :50] = rng.integers(0, 3, size=(N, 50))      # a few heavy rows
        top1[1 % N, 7] = E - 1
    got = om.ordermoe_estimate_transitions_device(_dev(top1), E)
    torch.cuda.synchronize()
    if N == 1:
        assert got.numel() == 0
        return
    want = om.ordermoe_estimate_transitions(top1, E)
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    # the oracle's estimate (eq 41): counts over the same tokens, row-normalised
    from oracle import tables
    P_or = tables.transitions([top1[l] for l in range(N)], [E] * N)
    for l in range(N - 1):
        np.testing.assert_allclose(got.cpu().numpy()[l], P_or[l], rtol=1e-15, atol=0, err_msg="layer %d" % l)


def _device_phi(sc, H, allow_sub, pin):
    cfg = sc.cfg
    N, E, M = cfg.N, cfg.E, cfg.M
    theta32 = np.array([om.ordermoe_theta_layer(l + 1, N, cfg.theta_min, cfg.theta_max) for l in range(N)],
                       np.float32)
    args = dict(P=_dev(np.stack(sc.P), np.float64), x=_dev(np.stack(sc.x_dep), np.uint8),
                sim=_dev(np.stack(sc.sim32), np.float32),
                group_of=_dev(np.stack([m["group_of"] for m in sc.models]), np.int32),
                theta=_dev(theta32), z_bits=_dev(np.full(N, sc.z_bits)), c=_dev(np.tile(sc.c, (N, 1)), np.float64),
                d_ref=_dev(np.full(N, sc.dref)), B=_dev(sc.net.B, np.float64), tau=_dev(sc.net.tau, np.float64),
                F=_dev(sc.net.F, np.float64))
    phi = om.ordermoe_build_lookahead_device(H, omega_T=cfg.omega_T, omega_Q=cfg.omega_Q, Qbar=cfg.Qbar,
                                             pin_local_exact=pin, allow_sub=allow_sub, **args)
    torch.cuda.synchronize()
    return phi.cpu().numpy()


@pytest.mark.parametrize("H,allow_sub,pin", [(1, 1, 1), (2, 1, 1), (3, 1, 1), (5, 1, 1), (3, 0, 1), (3, 2, 1),
                                             (3, 1, 0)])
def test_device_lookahead_equals_the_host_tables(stream_case, H, allow_sub, pin):
    """The 32-layer stack (128 experts, 8 servers): Phi^(H-1) of every layer."""
    import dataclasses
    from oracle import tables
    sc = with_horizon(stream_case, H, allow_sub=allow_sub)
    sc = dataclasses.replace(sc, cfg=dataclasses.replace(sc.cfg, pin_local_exact=pin))
    cfg = sc.cfg
    _, phi_host, _ = stream_library_tables(sc)
    got = _device_phi(sc, H, allow_sub, pin)
    # the oracle's Phi^(H-1) of the same stack and mode
    phi_or = tables.lookahead(H, sc.P, sc.x_dep, sc.sim32, [m["group_of"] for m in sc.models], sc.theta,
                              [sc.z_bits] * cfg.N, sc.net.B, sc.net.tau, [sc.c] * cfg.N, sc.net.F,
                              [sc.dref] * cfg.N, cfg.omega_T, cfg.omega_Q, cfg.Qbar, pin, allow_sub)
    for l in range(sc.cfg.N):
        np.testing.assert_allclose(got[l], phi_or[l], rtol=1e-12, atol=0, err_msg="oracle, layer %d" % l)
        np.testing.assert_array_equal(got[l], phi_host[l], err_msg="layer %d" % l)
    if H == 1:
        assert np.all(got == 0)
    else:
        assert np.all(got[-1] == 0) and np.any(got > 0)


def test_device_lookahead_rejects_a_short_workspace(stream_case):
    sc = stream_case
    N, M, E = sc.cfg.N, sc.cfg.M, sc.cfg.E
    need = om.lib().ordermoe_lookahead_device_workspace_size(N, E, M)
    assert need == 2 * N * M * E * 8
    ws = torch.empty(need - 8, dtype=torch.uint8, device="cuda")
    x = torch.zeros((N, M, E), dtype=torch.uint8, device="cuda")
    with pytest.raises(om.OrderMoEError) as ei:
        om.ordermoe_build_lookahead_device(1, None, x, None, None, None, None, None, None, None, None, None,
                                           0.5, 0.5, 1.0, ws=ws)
    assert ei.value.code == om.EWORKSPACE
