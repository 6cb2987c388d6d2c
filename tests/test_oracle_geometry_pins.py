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


def test_off_grid_rows_closed_form(geo):
    """Rows with keys off the grid, where the Nearest forward P^N differs
    from P^L (geometry probe paragraph: TV is taken against the operator's
    own forward probabilities). Worked by hand:

    MinMax, K = 2, z = (0, -1/4, -5/4, -2): m - M = -2, h = 1, levels
    b = (-2, -1, 0); u = (2, 7/4, 3/4, 0), so r = (1, 1, 0, 0),
    t = (1, 3/4, 3/4, 0), l = (2, 2, 1, 0); w^N = (1, 1, e^-1, e^-2) and
    w^L = (1, 1/4 e^-1 + 3/4, 1/4 e^-2 + 3/4 e^-1, e^-2).

    FWM, tau = 4, K = 2, z = (0, -1/2, -5/2, -7/2, -5): h = 2, levels
    b = (-4, -2, 0); u = (2, 7/4, 3/4, 1/4), the last key in the tail, so
    l = (2, 2, 1, 0), r = (1, 1, 0, 0); w^N = (1, 1, e^-2, e^-4, 0) and
    w^L = (1, 1/4 e^-2 + 3/4, 1/4 e^-4 + 3/4 e^-2, 3/4 e^-4 + 1/4 e^-2, 0).

    Top bucket: level K (Nearest) or interval K-1 (LERP) holds the first two
    keys in both rows; buckets are levels resp. intervals, the FWM tail one
    more bucket."""
    e = math.exp
    cases = [
        ("minmax", 6.0, [0.0, -0.25, -1.25, -2.0],
         [1.0, 1.0, e(-1), e(-2)],
         [1.0, 0.25 * e(-1) + 0.75, 0.25 * e(-2) + 0.75 * e(-1), e(-2)],
         {"nearest": [[0, 1], [2], [3]], "lerp": [[0, 1], [2, 3]]}),
        ("fwm", 4.0, [0.0, -0.5, -2.5, -3.5, -5.0],
         [1.0, 1.0, e(-2), e(-4), 0.0],
         [1.0, 0.25 * e(-2) + 0.75, 0.25 * e(-4) + 0.75 * e(-2), 0.75 * e(-4) + 0.25 * e(-2), 0.0],
         {"nearest": [[0, 1], [2], [3], [4]], "lerp": [[0, 1], [2, 3], [4]]}),
    ]
    for calib, tau, z, wN, wL, buckets in cases:
        z = np.array(z)
        S = np.tile(z, (z.size, 1))
        q, k = given(S)
        pe = np.exp(z) / np.exp(z).sum()
        for recon in ("nearest", "lerp"):
            w = np.array(wN if recon == "nearest" else wL)
            p = w / w.sum()
            o = geo(q, k, 2, calib, tau, recon, causal=False)[0, 0, 0]
            assert abs(o[G["tv"]] - 0.5 * np.abs(p - pe).sum()) <= 1e-15, (calib, recon)
            assert abs(o[G["top_mass"]] - pe[:2].sum()) <= 1e-15, (calib, recon)
            qb = np.array([pe[ix].sum() for ix in buckets[recon]])
            assert abs(o[G["eff_buckets"]] - math.exp(scipy_entropy(qb))) <= 1e-13, (calib, recon)
        # the two reconstructions' forward probabilities differ here, so the
        # TV of one is not the TV of the other
        pN, pL = np.array(wN) / sum(wN), np.array(wL) / sum(wL)
        assert abs(np.abs(pN - pe).sum() - np.abs(pL - pe).sum()) > 1e-3
