"""GPU parity of the similarity-model build (eq 3-5, 24-28) against the oracle."""
import numpy as np
import pytest

import workloads as wl
from oracle import route, similarity

from ._pipeline import host, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

CASES = {
    "C1": wl.C1,
    "C2": wl.C2.with_(T_cal=8192),
    "C4": wl.C4.with_(T_cal=8192),
    "C5s": wl.C5_BUILD.__class__(T_cal=16384 + 77),
    "C5": wl.C5_BUILD,
}


@pytest.mark.parametrize("name", list(CASES))
def test_similarity_build_parity(name):
    from paper_2607_17154_amd import ordermoe as om
    cfg = CASES[name]
    W = wl.router(cfg)
    Xc = wl.calibration(cfg)
    print("[%s] T_cal=%d d=%d E=%d" % (name, Xc.shape[0], cfg.d, cfg.E), flush=True)
    ws = torch.empty(om.ordermoe_similarity_workspace_size(Xc.shape[0], cfg.d, cfg.E),
                     dtype=torch.uint8, device="cuda")
    got = om.ordermoe_build_similarity(to_device(Xc, cfg.dtype), to_device(W, cfg.dtype), cfg.k,
                                       cfg.theta, cfg.alpha_f, ws)
    want = similarity.build(Xc, W, cfg.k, cfg.theta, cfg.alpha_f)
    d_sim = np.max(np.abs(got["sim"] - want["sim"]))
    print("[%s] max |dSim| = %.3g" % (name, d_sim), flush=True)
    assert d_sim <= 1e-4
    np.testing.assert_array_equal(got["sim"], host(got["sim_dev"]))
    assert np.all(np.diag(got["sim"]) == 1.0)
    np.testing.assert_allclose(got["sim"], got["sim"].T, atol=1e-6)
    # counts may differ only through calibration tokens within a rounding
    # distance of a top-k tie
    H = similarity.logit_matrix(Xc, W)
    _, srt = route.topk(H.T, cfg.k)
    near = int(np.sum(route.margin(srt) < 1e-4))
    dn = np.abs(got["counts"] - want["counts"])
    print("[%s] count diff max %d (near-tie tokens %d)" % (name, dn.max(), near), flush=True)
    assert dn.sum() <= 2 * near
    assert got["counts"].sum() == Xc.shape[0] * cfg.k
    assert list(got["group_of"]) == list(want["group_of"])
    assert got["centres"] == list(want["centres"])
    np.testing.assert_allclose(got["importance"], want["I"], atol=1e-4)
    assert len(got["centres"]) == cfg.clusters
