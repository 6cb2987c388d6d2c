"""GPU parity of the geometry probe (kia_geometry_probe) against the fp64
oracle on exact-score (dyadic) inputs, so that the extrema, levels and
buckets are the same on both sides. Counts and the quantile's order
statistics are exact; the sums carry fp32 rounding: span, width and norms
within 1e-5 relative, the entropy, top-bucket mass and TV within 2e-4
absolute (sums of up to 11k terms), the effective bucket count within
1e-4 relative. Shapes cover every head size, causal and not, ragged tails,
and rows long enough for the second and the ninth order statistic of the
0.1% quantile."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402
import test_gpu_parity as P  # noqa: E402

CASES = [(1, 2, 100, 64, 4, 1, 1.5), (1, 1, 77, 16, 1, 0, 2.0), (2, 1, 300, 128, 16, 1, 2.5),
         (1, 1, 2100, 32, 4, 1, 2.0), (1, 1, 9000, 16, 4, 1, 2.0), (1, 1, 12000, 16, 4, 1, 2.0)]


def gpu_probe(q, k, K, calib, tau, recon, causal):
    B, H, T, d = q.shape
    qg, kg = q.cuda(), k.cuda()
    _, st = kia.forward(qg, kg, torch.zeros_like(qg), K, calib, tau, recon, "weight", False,
                        causal)
    out = torch.full((B, H, T, 10), float("nan"), device="cuda")
    kia.kia_geometry_probe(qg, kg, st, out, K, calib, tau, recon, causal)
    torch.cuda.synchronize()
    return out.cpu().double().numpy()


@pytest.mark.parametrize("calib", ("minmax", "fwm"))
@pytest.mark.parametrize("recon", ("lerp", "nearest"))
def test_geometry_probe_matches_oracle(oracle_mod, calib, recon):
    G = oracle_mod.GEO
    for i, (B, H, T, d, K, causal, sc) in enumerate(CASES):
        tag = f"geometry {calib}/{recon} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, _, _ = make_inputs(B, H, T, d, seed=700 + i, qk_scale=sc, dyadic=True)
        g = gpu_probe(q, k, K, calib, 6.0, recon, causal)
        r = oracle_mod.geometry(q.double().numpy(), k.double().numpy(), K, calib, 6.0, recon,
                                causal)
        assert np.isfinite(g).all(), tag
        rel = lambda x, y: np.max(np.abs(x - y) / np.maximum(np.abs(y), 1e-30))
        for f in ("span", "h", "qnorm", "knorm"):
            assert rel(g[..., G[f]], r[..., G[f]]) <= 1e-5, (tag, f)
        zq = G["zq001"]
        assert np.max(np.abs(g[..., zq] - r[..., zq])) <= 1e-6 * (1 + np.max(np.abs(r[..., zq])))
        assert np.max(np.abs(g[..., G["frac_z_lt_m6"]] - r[..., G["frac_z_lt_m6"]])) <= 1e-6, tag
        for f in ("entropy", "top_mass", "tv"):
            err = np.max(np.abs(g[..., G[f]] - r[..., G[f]]))
            assert err <= 2e-4, (tag, f, err)
        assert rel(g[..., G["eff_buckets"]], r[..., G["eff_buckets"]]) <= 1e-4, tag


def test_geometry_probe_rejects_other_operators():
    q, k, _, _ = make_inputs(1, 1, 64, 16, seed=1)
    qg, kg = q.cuda(), k.cuda()
    _, st = kia.forward(qg, kg, qg, 4, "fwm", 8.0, "lerp", "weight", False, True)
    out = torch.zeros((1, 1, 64, 10), device="cuda")
    for calib, recon in (("resolved", "lerp"), ("fwm", "softmax")):
        with pytest.raises(kia.KiaError):
            kia.kia_geometry_probe(qg, kg, st, out, 4, calib, 8.0, recon, True)
