"""Batches in flight together on two HIP streams, through the C ABI.

Routing and the local forward of two different batches are queued on two
streams, interleaved several times over, with separate outputs and
workspaces but shared weights, tables and router.  Each batch's outputs must
equal, bit for bit, those of the same batch run alone on the default stream
(the library keeps no device state between calls, and the split-K counters and
partial tiles live in each call's workspace)."""
import numpy as np
import pytest

import workloads as wl

from ._pipeline import DeviceLayer, build_case, host, library_tables

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_17154_amd import ordermoe as om  # noqa: E402

ROUTE = ("idx", "w", "exec_k", "exec_m", "cls", "qhat_out", "loc_out", "dst_count", "counters")


class _Batch:
    def __init__(self, dl, x, loc, qh, T):
        cfg = dl.cfg
        self.dl, self.x, self.loc, self.qh, self.T = dl, x, loc, qh, T
        self.out = om.alloc_route_out(T, cfg.k, cfg.M, "cuda")
        self.ws_r = torch.empty(om.ordermoe_route_workspace_size(T, cfg.k, cfg.M), dtype=torch.uint8,
                                device="cuda")
        self.ws_f = torch.empty(om.ordermoe_forward_workspace_size(dl.experts, T, cfg.k), dtype=torch.uint8,
                                device="cuda")
        self.y = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
        self.ro = torch.empty(dl.experts.n_local + 2, dtype=torch.int32, device="cuda")

    def run(self, stream):
        dl, cfg, o = self.dl, self.dl.cfg, self.out
        om.ordermoe_route_select(dl.layer, self.x, self.T, self.loc, self.qh, o, self.ws_r, stream=stream)
        om.ordermoe_local_moe_forward(dl.experts, self.x, self.T, cfg.k, o["w"], o["exec_k"], o["exec_m"],
                                      self.loc, cfg.m0, self.y, self.ro, self.ws_f, stream=stream)

    def snapshot(self):
        torch.cuda.synchronize()
        snap = {n: host(self.out[n]).copy() for n in ROUTE}
        n_remote = int(snap["counters"][om.CNT_REMOTE_SLOTS])
        snap["dispatch"] = host(self.out["dispatch"])[:n_remote].copy()
        snap["y"] = host(self.y).copy()
        snap["ro"] = host(self.ro).copy()
        return snap


# a layer whose GEMMs split tiles along K (shared group included), and the
# Mixtral-shaped layer at a reduced batch
@pytest.mark.parametrize("cfg,T1,T2", [
    (wl.C3.with_(T=600, d=1024, f=512, n_shared=1, T_cal=4096), 600, 451),
    (wl.C2.with_(T=700, d=1024, f=1024, T_cal=4096), 700, 333),
])
def test_two_streams_equal_one_batch_at_a_time(cfg, T1, T2):
    print("concurrent: %s d=%d f=%d T=%d,%d" % (cfg.name, cfg.d, cfg.f, T1, T2), flush=True)
    case = build_case(cfg)
    dl = DeviceLayer(case, library_tables(case))
    x, loc, qh = dl.inputs()
    rng = np.random.default_rng(7)
    perm = torch.from_numpy(rng.permutation(cfg.T)[:T2].astype(np.int64)).cuda()
    b1 = _Batch(dl, x[:T1].contiguous(), loc[:T1].contiguous(), qh[:T1].contiguous(), T1)
    b2 = _Batch(dl, x[perm].contiguous(), loc[perm].contiguous(), qh[perm].contiguous(), T2)
    cur = torch.cuda.current_stream()
    b1.run(cur)
    want1 = b1.snapshot()
    b2.run(cur)
    want2 = b2.snapshot()
    assert not np.array_equal(want1["ro"], want2["ro"])      # the batches differ
    for b in (b1, b2):
        b.y.zero_()
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(4):
        b1.run(s1)
        b2.run(s2)
    got1, got2 = b1.snapshot(), b2.snapshot()
    for want, got, tag in ((want1, got1, "batch 1"), (want2, got2, "batch 2")):
        for n in want:
            np.testing.assert_array_equal(got[n], want[n], err_msg="%s %s" % (tag, n))
