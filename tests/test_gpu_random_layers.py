"""Seeded random layers across the C ABI's parameter space, on the GPU.

Thirty layers drawn by tests/_random_layers.py: 1 to 256 experts, 1 to 32
servers, top-1 to top-8, 0 to 4 shared experts, bf16 and fp32, batches of 1
token to 2049 (decode-sized thin GEMMs, ragged tiles, split K), fresh and
partly spent budgets, both token-location modes, and every selection mode
(pin 0/1, allow_sub 0/1/2, renorm 0/1).  For each: the routing decisions and
dispatch list bit-exact with the oracle (eq 3, 36-44) on unflagged tokens and
every token's layer output within the bar (bf16 2e-2, fp32 1e-4 relative),
exactly as the fixed-shape parity tests check them.  Random logits put more
tokens within 1e-4 of a tie than the planted workloads do, so up to 3% of
the tokens may be flagged (they are counted and left out of the comparison)."""
import numpy as np
import pytest

from ._pipeline import DeviceLayer, host
from ._random_layers import N_RANDOM, qhat_scale, random_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from .test_gpu_parity import TOL, _case, _check_decisions, _check_output  # noqa: E402
from ._pipeline import oracle_decisions  # noqa: E402


@pytest.mark.parametrize("i", range(N_RANDOM))
def test_random_layer_parity(i):
    cfg = random_layer(i)
    print("random layer %d: %s T=%d n_shared=%d m0=%d loc=%s Qbar=%g pin=%d allow_sub=%d renorm=%d" % (
        i, cfg.name, cfg.T, cfg.n_shared, cfg.m0, cfg.loc_mode, cfg.Qbar, cfg.pin_local_exact, cfg.allow_sub,
        cfg.renorm), flush=True)
    case, tabs = _case("random%d" % i, cfg, qhat_scale=qhat_scale(i))
    dl = DeviceLayer(case, tabs)
    x, loc, qh = dl.inputs()
    T = case.X.shape[0]
    out = dl.route(x, loc, qh, T)
    y, ro = dl.forward(x, loc, out, T)
    torch.cuda.synchronize()
    dec = oracle_decisions(case)
    ok = _check_decisions(case, dec, out, max_flagged=0.03)
    rows = host(ro)
    assert rows[0] == 0 and np.all(np.diff(rows) >= 0)
    _check_output(case, dec, y, np.arange(T), ok, TOL[cfg.dtype])
