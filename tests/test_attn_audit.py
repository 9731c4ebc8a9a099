"""Host logic of the attention / Ulysses recovery audit (App. B) against the oracle's model
functions: the recovery gap (Eq. 2), pressure (Eq. 3), the backlog recurrence (Eq. 5) and the
tile-aligned recovery threshold."""
import math

import pytest

from oracle import xstage_model as om
from paper_2607_23264_amd import attn_a2a as aa
from paper_2607_23264_amd import xstage as X


def _model(t0a=0.8, t0b=5e-8, R=56000.0, Q=16.0e6, K=512):
    return X.xs_model(t0a, t0b, R, Q, K, 0)


@pytest.mark.parametrize("M,qloop", [(8192, 289.0), (16384, 570.0), (32768, 1175.0), (4096, 60.0)])
def test_audit_matches_the_model_definitions(M, qloop):
    m = _model()
    K = 512
    tiles = 8 * M // 128
    cell = {"grid": K, "tiles": tiles, "qloop_us_median": qloop, "sigma_us_per_kv_tile": qloop / (M // 64)}
    a = aa.audit(m, cell)
    V = K * 128 * 128 * 2
    T0 = 0.8 + 5e-8 * V
    assert a["V_bytes"] == V
    assert a["G_star_us"] == pytest.approx(float(om.recovery_gap(V, 56000.0, T0)), rel=1e-12)
    _, rho = om.pressure(V, T0, qloop, 56000.0)
    assert a["rho"] == pytest.approx(float(rho), rel=1e-12)
    assert a["delta_b_bytes"] == pytest.approx(float(om.delta_b(V, T0, qloop, 56000.0)), rel=1e-9, abs=1e-6)
    n = math.ceil(tiles / K)
    assert a["output_boundaries_per_producer"] == n
    q = om.backlog_recurrence([V] * n, [T0] * n, [qloop] * n, 56000.0)
    assert a["E_res_bound_us"] == pytest.approx(max(0.0, (q[n - 1] + V) / 56000.0 - T0), rel=1e-9)
    sigma = qloop / (M // 64)
    assert a["M_ub_star"] == om.fa_recovery_threshold(64, a["G_star_us"], sigma)
    assert a["guard_ok"] == (float(om.b_iso(V, T0, 56000.0)) <= 16.0e6 + 1e-6)


def test_summary_fits_the_coupled_slope():
    m = _model()
    cells = []
    for M, cc in ((8192, 100.0), (16384, 400.0), (32768, 1000.0)):
        c = {"sink": "host", "M": M, "grid": 512, "tiles": 8 * M // 128, "qloop_us_median": 300.0,
             "sigma_us_per_kv_tile": 2.0, "E_res_us": 5.0, "speedup_vs_serial": 1.2, "coupled_residual_us": cc}
        c["audit"] = aa.audit(m, c)
        cells.append(c)
    s = aa.summarize(cells)["host"]
    # boundaries 1, 2, 4 -> residuals 100, 400, 1000: slope 300 per boundary exactly
    assert s["coupled_slope_us_per_boundary"] == pytest.approx(300.0)
    assert s["model_drain_us_per_boundary"] == pytest.approx(512 * 32768 / 56000.0)
