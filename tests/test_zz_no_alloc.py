"""ordermoe_route_select_noalloc against ordermoe_route_select, through the C ABI.

The allocation-free variant takes its workspace from the library's fixed
per-GPU scratch; its outputs must equal those of the workspace variant bit for
bit.  Two calls in a row on one GPU, the second with a smaller batch (the
scratch keeps the first call's contents), for prefill-sized batches (32-token
blocks; 16-token blocks with their token rows in LDS) and a decode-sized one
(whose router is split over K into partial logits held in the scratch)."""
import numpy as np
import pytest

import workloads as wl

from ._pipeline import DeviceLayer, build_case, host, library_tables

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_17154_amd import ordermoe as om  # noqa: E402

OUTS = ("idx", "w", "margin", "flag", "exec_k", "exec_m", "cls", "qhat_out", "loc_out", "dst_count", "counters")


def _compare(dl, x, loc, qh, T):
    cfg = dl.cfg
    print("no-alloc: %s T=%d" % (cfg.name, T), flush=True)
    want = dl.route(x, loc, qh, T)
    got = om.alloc_route_out(T, cfg.k, cfg.M, "cuda")
    for v in got.values():
        v.fill_(-3) if v.dtype != torch.uint8 else v.fill_(77)
    om.ordermoe_route_select_noalloc(dl.layer, x, T, loc, qh, got)
    torch.cuda.synchronize()
    for n in OUTS:
        np.testing.assert_array_equal(host(got[n]), host(want[n]), err_msg=n)
    n_remote = int(host(want["counters"])[om.CNT_REMOTE_SLOTS])
    np.testing.assert_array_equal(host(got["dispatch"])[:n_remote], host(want["dispatch"])[:n_remote])
    return n_remote


@pytest.mark.parametrize("cfg,T1,T2", [
    (wl.C4.with_(T=3000, T_cal=4096), 3000, 1100),
    # 16-token blocks with their token rows staged in LDS (both batches)
    (wl.C2.with_(T=2049, T_cal=4096), 2049, 1100),
    (wl.C2.with_(T=97, T_cal=4096), 97, 40),
])
def test_noalloc_route_select_equals_the_workspace_variant(cfg, T1, T2):
    case = build_case(cfg)
    dl = DeviceLayer(case, library_tables(case), with_experts=False)
    x, loc, qh = dl.inputs()
    assert om.lib().ordermoe_route_workspace_size(T1, cfg.k, cfg.M) <= om.NOALLOC_SCRATCH_BYTES
    r1 = _compare(dl, x, loc, qh, T1)
    # a smaller batch second: the scratch still holds the first call's data
    r2 = _compare(dl, x[:T2].contiguous(), loc[:T2].contiguous(), qh[:T2].contiguous(), T2)
    assert r1 > 0 and r2 > 0           # remote slots: the dispatch list is exercised
