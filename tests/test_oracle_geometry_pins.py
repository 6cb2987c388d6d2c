"""Pins of the oracle's geometry-probe statistics (Sec. 2 and the appendix
paragraph on the geometry probe) against independent references: numpy's
quantile and norms, scipy's entropy, brute-force counts, and closed forms
for degenerate rows, two-key rows, grid-point rows and FWM rows with a tail.
CPU only."""
import math

import numpy as np
import pytest
from scipy.stats import entropy as scipy_entropy

G = None


@pytest.fixture(scope="module")
def geo(oracle_mod):
    global G
    G = oracle_mod.GEO
    return oracle_mod.geometry


def fp32_scores(q, k):
    d = q.shape[-1]
    sc = np.float32(1.0 / math.sqrt(d))
    dot = (q.astype(np.float64) @ np.swapaxes(k.astype(np.float64), -1, -2)).astype(np.float32)
    return (dot * sc).astype(np.float32).astype(np.float64)


@pytest.mark.parametrize("calib", ("minmax", "fwm"))
@pytest.mark.parametrize("recon", ("lerp", "nearest"))
@pytest.mark.parametrize("causal", (1, 0))
def test_statistics_against_independent_references(oracle_mod, geo, calib, recon, causal):
    """Quantile (numpy, linear), entropy (scipy), norms (numpy), fraction
    below -6 (count), span and native width, and the bounds of TV, top mass
    and effective buckets, on random rows of several lengths."""
    rng = np.random.default_rng(41)
    for T, d, K, sig in ((37, 16, 4, 2.0), (300, 64, 16, 3.0), (1100, 32, 4, 2.5)):
        q = rng.normal(size=(1, 2, T, d)) * sig
        k = rng.normal(size=(1, 2, T, d))
        out = geo(q, k, K, calib, 6.0, recon, causal)
        S = fp32_scores(q, k)
        for h in range(2):
            for i in range(0, T, 1 if T < 500 else 7):
                n = i + 1 if causal else T
                s = S[0, h, i, :n]
                z = s - s.max()
                o = out[0, h, i]
                assert o[G["span"]] == s.max() - s.min()
                hw = (s.max() - s.min()) / K if calib == "minmax" else 6.0 / K
                assert abs(o[G["h"]] - hw) <= 1e-15 * max(1.0, hw)
                assert abs(o[G["zq001"]] - np.quantile(z, 0.001)) <= 1e-12 * (1 + abs(z.min()))
                p = np.exp(z) / np.exp(z).sum()
                assert abs(o[G["entropy"]] - scipy_entropy(p)) <= 1e-12
                assert o[G["frac_z_lt_m6"]] == np.count_nonzero(z < -6) / n
                assert abs(o[G["qnorm"]] - np.linalg.norm(q[0, h, i])) <= 1e-12 * np.linalg.norm(q[0, h, i])
                assert abs(o[G["knorm"]] - np.linalg.norm(k[0, h, i])) <= 1e-12 * np.linalg.norm(k[0, h, i])
                assert 0.0 <= o[G["tv"]] <= 1.0
                assert 0.0 <= o[G["top_mass"]] <= 1.0 + 1e-15
                assert 1.0 - 1e-12 <= o[G["eff_buckets"]] <= min(n, K + 2) + 1e-9


def given(S):
    """q, k with q.k / sqrt(d) = S exactly (d = 16 or 64, k = sqrt(d) I)."""
    T = S.shape[0]
    d = 16 if T <= 16 else 64
    q = np.zeros((1, 1, T, d))
    q[0, 0, :, :T] = S
    k = np.zeros((1, 1, T, d))
    k[0, 0, :, :T] = np.eye(T) * math.sqrt(d)
    return q, k


def test_degenerate_rows(geo):
    """Equal scores: MinMax is degenerate (uniform P, App. A) and so is the
    softmax: TV = 0, entropy = log n, one bucket, nothing below -6."""
    S = np.full((10, 10), 0.75)
    q, k = given(S)
    for calib in ("minmax", "fwm"):
        for recon in ("lerp", "nearest"):
            o = geo(q, k, 4, calib, 6.0, recon, causal=False)[0, 0]
            assert np.all(np.abs(o[:, G["tv"]]) <= 1e-15)
            assert np.allclose(o[:, G["entropy"]], math.log(10), rtol=0, atol=1e-14)
            assert np.allclose(o[:, G["eff_buckets"]], 1.0, rtol=0, atol=1e-14)
            assert np.all(o[:, G["frac_z_lt_m6"]] == 0) and np.all(o[:, G["span"]] == 0)


def test_two_key_rows_closed_form(geo):
    """Row with keys at M and m under MinMax: the argmax sits on the top level
    (l = K, r = K-1), the argmin on level 0 (r = 0 for K > 1), both on grid
    points, so P^native is the two-element softmax (TV = 0), the top-bucket
    mass is 1/(1 + e^{m-M}), and the effective bucket count is
    exp of the binary entropy."""
    for K in (2, 4, 16):
        for gap in (0.5, 3.0, 9.0):
            S = np.array([[1.0, 1.0 - gap], [1.0 - gap, 1.0]])
            q, k = given(S)
            for recon in ("lerp", "nearest"):
                o = geo(q, k, K, "minmax", 6.0, recon, causal=False)[0, 0, 0]
                p = 1.0 / (1.0 + math.exp(-gap))
                assert abs(o[G["tv"]]) <= 1e-15
                assert abs(o[G["top_mass"]] - p) <= 1e-15
                hb = -(p * math.log(p) + (1 - p) * math.log(1 - p))
                assert abs(o[G["eff_buckets"]] - math.exp(hb)) <= 1e-13


def test_grid_point_rows_have_no_distortion(geo):
    """Scores on MinMax grid points: w^L = w^N = e^z (Sec. 3), so P^native
    is the softmax and TV = 0 for LERP and Nearest; each key's bucket is its
    grid point, so the effective bucket count is exp H of the softmax."""
    K = 4
    S = np.zeros((12, 12))
    for i in range(12):
        S[i] = -2.0 + 0.5 * (np.arange(12) % (K + 1))   # m = -2, M = 0, h = 0.5
    q, k = given(S)
    for recon in ("lerp", "nearest"):
        o = geo(q, k, K, "minmax", 6.0, recon, causal=False)[0, 0]
        assert np.all(np.abs(o[:, G["tv"]]) <= 1e-15)
    o = geo(q, k, K, "minmax", 6.0, "nearest", causal=False)[0, 0, 0]
    z = S[0] - S[0].max()
    p = np.exp(z) / np.exp(z).sum()
    qb = np.array([p[np.arange(12) % (K + 1) == b].sum() for b in range(K + 1)])
    assert abs(o[G["eff_buckets"]] - math.exp(scipy_entropy(qb))) <= 1e-13


def test_fwm_tail_row_closed_form(geo):
    """FWM with window keys on grid points and the rest below -tau: inside
    the window P^native = e^z / W_window, outside 0, so TV equals the
    softmax mass of the tail, and the tail is its own bucket."""
    tau, K = 6.0, 4
    win = np.array([0.0, -1.5, -3.0, -4.5, -6.0])       # grid points, h = 1.5
    tailz = np.array([-6.5, -9.0, -13.0])
    row = np.concatenate([win, tailz])
    S = np.tile(row, (8, 1))
    q, k = given(S)
    e = np.exp(row)
    tmass = e[len(win):].sum() / e.sum()
    for recon in ("lerp", "nearest"):
        o = geo(q, k, K, "fwm", tau, recon, causal=False)[0, 0, 0]
        assert abs(o[G["tv"]] - tmass) <= 1e-15
        assert abs(o[G["frac_z_lt_m6"]] - 3 / 8) <= 1e-15
    o = geo(q, k, K, "fwm", tau, "nearest", causal=False)[0, 0, 0]
    qb = np.concatenate([e[: len(win)], [e[len(win):].sum()]]) / e.sum()
    assert abs(o[G["eff_buckets"]] - math.exp(scipy_entropy(qb))) <= 1e-13
    assert abs(o[G["top_mass"]] - e[0] / e.sum()) <= 1e-15
