"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is a closed form,
an exact-rational brute force, a finite difference, an identity the paper
states, or a bound the paper prints (tests/golden/paper_bounds.json). A
plausible slip in the oracle (a dropped calibration term, a sign, an index
off by one, the wrong normalization point of a surrogate) fails at least one
of them. CPU only.
"""
import json
import math
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
with open(os.path.join(HERE, "golden", "paper_bounds.json")) as fh:
    BOUNDS = json.load(fh)

# "resolved": the tail-policy diagnostic (FWM step and origin, grid continued
# below -tau with negative indices, no zero tail)
CALIBS = ("minmax", "fwm", "resolved")
SURROGATES = (("lerp", "weight"), ("nearest", "weight"), ("nearest", "prob"))


def softmax(x):
    e = np.exp(np.asarray(x, dtype=np.float64) - np.max(x))
    return e / e.sum()


def rand_row(rng, n, sigma=1.0):
    """Random scores, rounded to fp32: the operator acts on fp32 scores
    (App. A), where K (s - m) and (s - M) + tau are exact in fp64."""
    return rng.normal(0.0, sigma, size=n).astype(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Forward pins
# --------------------------------------------------------------------------

@pytest.mark.parametrize("calib", CALIBS)
@pytest.mark.parametrize("recon", ("lerp", "nearest"))
def test_rows_sum_to_one(oracle_mod, calib, recon):
    """Normalization P = w / sum w (App. A): rows sum to 1, P >= 0."""
    rng = np.random.default_rng(11)
    for K in (1, 2, 3, 4, 7, 16, 64):
        for n in (1, 2, 3, 17, 64):
            for sigma in (1.0, 5.0):
                out = oracle_mod.row(rand_row(rng, n, sigma), K=K, calib=calib,
                                     tau=8.0, recon=recon)
                assert abs(out["P"].sum() - 1.0) <= 1e-14
                assert (out["P"] >= 0).all()


@pytest.mark.parametrize("K", (1, 2, 4, 5, 16, 64))
def test_grid_endpoints_are_exact(oracle_mod, K):
    """The argmax key sits on b_K = 0 (w = 1); under MinMax the argmin key on
    b_0 = m - M (w = e^{m-M}), for LERP and Nearest alike (Sec. 3 grid,
    App. A index clip)."""
    rng = np.random.default_rng(K)
    for _ in range(20):
        s = rand_row(rng, 9, 2.0)
        for recon in ("lerp", "nearest"):
            out = oracle_mod.row(s, K=K, calib="minmax", recon=recon)
            a, b = int(out["amax"]), int(out["amin"])
            assert out["wL"][a] == 1.0 and out["wN"][a] == 1.0
            e = math.exp(s[b] - s[a])
            assert out["wL"][b] == e and out["wN"][b] == e
            fw = oracle_mod.row(s, K=K, calib="fwm", tau=8.0, recon=recon)
            assert fw["wL"][a] == 1.0 and fw["wN"][a] == 1.0


@pytest.mark.parametrize("K", (1, 2, 4, 16, 64))
@pytest.mark.parametrize("recon,ste", SURROGATES)
def test_two_key_row_is_two_element_softmax(oracle_mod, K, recon, ste):
    """A two-key MinMax row is exactly the two-element softmax, forward and
    full backward (App. B, derivative of the full hard map: a two-key row is
    the two-element softmax; verified there to 1e-16)."""
    rng = np.random.default_rng(100 + K)
    tol = 4 * BOUNDS["two_key_softmax_identity"]["value"]
    for _ in range(50):
        s = rand_row(rng, 2, 3.0)
        g = rng.normal(size=2)
        out = oracle_mod.row(s, g, K=K, calib="minmax", recon=recon, ste=ste)
        P = softmax(s)
        assert np.max(np.abs(out["P"] - P)) <= tol
        ref = P * (g - np.dot(P, g))     # softmax backward
        assert np.max(np.abs(out["dS"] - ref)) <= tol * (1 + np.max(np.abs(ref))) * 4


def test_minmax_scores_on_grid_points_give_softmax(oracle_mod):
    """Scores on grid points: w^L = w^N = e^z, so LERP = Nearest = softmax
    (Sec. 3 reconstruction; App. A LERP and Nearest)."""
    rng = np.random.default_rng(3)
    for K in (2, 4, 8, 16):
        m, M = -3.0, -3.0 + K * 0.75          # h = 0.75 exactly
        for _ in range(10):
            ks = rng.integers(0, K + 1, size=12)
            ks[0], ks[1] = 0, K
            s = m + ks * 0.75
            for recon in ("lerp", "nearest"):
                out = oracle_mod.row(s, K=K, calib="minmax", recon=recon)
                assert np.max(np.abs(out["P"] - softmax(s))) <= 1e-15


def test_fwm_scores_on_grid_points_give_windowed_softmax(oracle_mod):
    """FWM: grid b_r = -tau + r tau/K anchored at the max, zero weight for
    z < -tau (Sec. 3, App. A FWM); on grid points it is softmax over the
    window keys."""
    rng = np.random.default_rng(4)
    for K, tau in ((4, 8.0), (16, 8.0), (4, 6.0), (8, 6.0)):
        h = tau / K
        M = 1.25
        for _ in range(10):
            ks = rng.integers(0, K + 1, size=10)
            ks[0] = K
            s = M - tau + ks * h
            s = np.concatenate([s, [M - tau - 0.5, M - tau - 3.0]])  # tail keys
            inwin = np.arange(s.size) < 10
            for recon in ("lerp", "nearest"):
                out = oracle_mod.row(s, K=K, calib="fwm", tau=tau, recon=recon)
                ref = np.zeros(s.size)
                ref[inwin] = softmax(s[inwin])
                assert np.max(np.abs(out["P"] - ref)) <= 1e-15
                assert (out["tail"][~inwin] == 1).all()


def chord_excess(h):
    """max over t in [0,1] of (1 - t + t e^h) e^{-t h} - 1 (convexity of exp)."""
    if h == 0:
        return 0.0
    ts = np.linspace(0, 1, 20001)
    return float(np.max((1 - ts + ts * np.exp(h)) * np.exp(-ts * h)) - 1)


@pytest.mark.parametrize("calib", CALIBS)
def test_reconstruction_bounds(oracle_mod, calib):
    """LERP is a chord of the convex exponential: e^z <= w^L <= e^z(1+eps_h).
    Nearest rounds by at most h/2 in z: e^{-h/2} <= w^N / e^z <= e^{h/2}
    (Sec. 3 reconstruction)."""
    rng = np.random.default_rng(5)
    for K in (1, 2, 4, 16):
        for _ in range(20):
            s = rand_row(rng, 30, 2.5)
            out = oracle_mod.row(s, K=K, calib=calib, tau=8.0)
            h = out["h"]
            z = s - s.max()
            keep = out["tail"] == 0
            ez = np.exp(z[keep])
            wl, wn = out["wL"][keep], out["wN"][keep]
            eps = chord_excess(h)
            assert (wl >= ez * (1 - 1e-14)).all()
            assert (wl <= ez * (1 + eps) * (1 + 1e-9)).all()
            assert (wn / ez >= math.exp(-h / 2) * (1 - 1e-14)).all()
            assert (wn / ez <= math.exp(h / 2) * (1 + 1e-14)).all()


@pytest.mark.parametrize("calib", CALIBS)
def test_lerp_converges_to_softmax_at_rate_K_minus_2(oracle_mod, calib):
    """At fixed span the LERP chord error is O(h^2) = O(1/K^2), so P^L ->
    softmax with the error dropping ~4x per doubling of K (Sec. 3; K trend
    observed in Sec. 5)."""
    rng = np.random.default_rng(6)
    s = rand_row(rng, 200, 1.0)
    tau = 20.0  # FWM window wider than the span: no tail
    errs = []
    for K in (8, 16, 32, 64, 128):
        out = oracle_mod.row(s, K=K, calib=calib, tau=tau, recon="lerp")
        errs.append(np.max(np.abs(out["P"] - softmax(s))))
    ratios = [errs[i] / errs[i + 1] for i in range(len(errs) - 1)]
    assert all(3.0 <= q <= 5.0 for q in ratios), (errs, ratios)


def test_resolved_window_is_fwm_and_tail_is_kept(oracle_mod):
    """The resolved grid (tail-policy appendix) keeps FWM's step tau/K and
    origin -tau: keys inside the window get FWM's interval, level and
    unnormalized weights exactly (the appendix: in-window weights
    bit-identical to FWM's); keys below -tau are not zeroed but continue on
    the grid, w^N = e^{-tau + l tau/K} with negative l."""
    rng = np.random.default_rng(31)
    for K in (1, 2, 4, 16):
        for tau in (3.0, 6.0, 8.0):
            for _ in range(10):
                s = rand_row(rng, 40, 4.0)
                for recon in ("lerp", "nearest"):
                    fw = oracle_mod.row(s, K=K, calib="fwm", tau=tau, recon=recon)
                    rs = oracle_mod.row(s, K=K, calib="resolved", tau=tau, recon=recon)
                    win = fw["tail"] == 0
                    for key in ("r", "l", "wL", "wN"):
                        assert np.array_equal(rs[key][win], fw[key][win]), key
                    assert (rs["tail"] == 0).all()
                    z = s - s.max()
                    below = ~win
                    assert (rs["l"][below] <= 0).all() and (rs["wN"][below] > 0).all()
                    grid = np.exp(-tau + rs["l"][below] * tau / K)
                    assert np.allclose(rs["wN"][below], grid, rtol=1e-14, atol=0)
                    assert (np.abs(np.log(rs["wN"][below]) - z[below]) <= tau / K / 2 + 1e-12).all()


def test_resolved_lerp_converges_to_softmax_with_tails(oracle_mod):
    """With every key on the grid, LERP over the resolved grid is within the
    chord bound of the full softmax on every key, tail keys included:
    e^z <= w^L <= e^z (1 + eps_h) gives |P^L / P^E - 1| <= eps_h with
    eps_h ~ h^2/8, h = tau/K, so P^L -> softmax at O(1/K^2) even when the
    row span exceeds tau; FWM stays off by the truncated tail mass."""
    rng = np.random.default_rng(32)
    s = rand_row(rng, 200, 4.0)
    tau = 4.0   # span ~ 25 >> tau: heavy tail
    pe = softmax(s)
    errs = []
    for K in (8, 16, 32, 64, 128):
        eps = chord_excess(tau / K)
        p = oracle_mod.row(s, K=K, calib="resolved", tau=tau, recon="lerp")["P"]
        rel = np.max(np.abs(p / pe - 1))
        assert rel <= eps * (1 + 1e-9), (K, rel, eps)
        errs.append(np.max(np.abs(p - pe)))
        pf = oracle_mod.row(s, K=K, calib="fwm", tau=tau, recon="lerp")["P"]
        assert np.max(np.abs(pf / pe - 1)) == 1.0  # zeroed tail keys
    assert errs[-1] < errs[0] / 100, errs


def _exact_indices(s, K, calib, tau):
    """r, l, tail by exact rational arithmetic on the given fp64 scores:
    l = argmin_k |z - b_k| with ties to the larger k (midpoint rounds up),
    r = largest k <= K-1 with b_k <= z (floor, clipped)."""
    S = [Fr(float(x)) for x in s]
    M, m = max(S), min(S)
    zlo = (m - M) if calib == "minmax" else -Fr(float(tau))
    # grid levels k = k0..K; the resolved grid continues below b_0 (k < 0)
    k0 = 0
    if calib == "resolved":
        k0 = min(0, math.floor(float((m - M - zlo) * K / (-zlo))) - 2)
    ks = range(k0, K + 1)
    b = {k: (1 - Fr(k, K)) * zlo for k in ks}
    rs, ls, tails = [], [], []
    for x in S:
        z = x - M
        if calib == "fwm" and z < zlo:
            rs.append(0); ls.append(0); tails.append(1)
            continue
        tails.append(0)
        if calib == "minmax" and M == m:
            rs.append(0); ls.append(0)
            continue
        r = max(k for k in ks if k <= K - 1 and b[k] <= z)
        dist = {k: abs(z - b[k]) for k in ks}
        best = min(dist.values())
        l = max(k for k in ks if dist[k] == best)
        rs.append(r); ls.append(l)
    return np.array(rs), np.array(ls), np.array(tails)


@pytest.mark.parametrize("calib", CALIBS)
def test_indices_match_exact_brute_force(oracle_mod, calib):
    """Interval r and nearest level l of every key equal the exact-rational
    brute force of App. A (floor with clip; nearest grid centre, midpoint up),
    including scores exactly on grid points and midpoints and one fp32 ulp
    away from them; FWM tail exactly at z = -tau stays in the window."""
    rng = np.random.default_rng(7)
    tau = 8.0
    rows = []
    for K in (1, 2, 3, 4, 5, 16):
        for _ in range(10):
            rows.append((K, rand_row(rng, 25, 2.0)))
        # crafted dyadic rows: h = 1/2 exactly, scores on grid points,
        # midpoints, and fp32 ulps either side of both
        # (grid placed so that no score is within 26 binades of zero: the
        # domain where one fp64 rounding equals the exact-real decision)
        if calib == "minmax":
            m = -1.375
            base = m + np.arange(0, 2 * K + 1) * 0.25
            M = m + 0.5 * K
        else:
            h = tau / K
            M = 0.8125
            lo = -4 * K if calib == "resolved" else 0  # below the window: negative r
            base = M - tau + np.arange(lo, 2 * K + 1) * (h / 2)
        base = base.astype(np.float32).astype(np.float64)   # fp32 scores
        up = np.nextafter(base.astype(np.float32), np.float32(np.inf)).astype(np.float64)
        dn = np.nextafter(base.astype(np.float32), np.float32(-np.inf)).astype(np.float64)
        s = np.concatenate([base, up, dn, [M]])
        s = s[(s <= M) & ((s >= base.min()) if calib == "minmax" else (s > -1e9))]
        if calib == "fwm":
            cut = np.float32(M - tau)
            s = np.concatenate([s, [M - tau, float(np.nextafter(cut, np.float32(-np.inf))),
                                    float(np.nextafter(cut, np.float32(np.inf))), M - tau - 1]])
        s = s[np.abs(s) > 1e-6]  # keep every score within 26 binades of the row scale
        rows.append((K, s))
    for K, s in rows:
        out = oracle_mod.row(s, K=K, calib=calib, tau=tau, recon="nearest")
        r, l, tail = _exact_indices(s, K, calib, tau)
        assert (out["tail"] == tail).all()
        assert (out["r"] == r).all(), (K, s)
        assert (out["l"] == l).all(), (K, s)


# --------------------------------------------------------------------------
# Backward pins
# --------------------------------------------------------------------------

def fd_grad(f, x, eps):
    g = np.zeros_like(x)
    for i in range(x.size):
        xp, xm = x.copy(), x.copy()
        xp[i] += eps
        xm[i] -= eps
        g[i] = (f(xp) - f(xm)) / (2 * eps)
    return g


def safe_row(rng, n, K, calib, tau, sigma=1.0, margin=2e-3):
    """A row whose keys sit at least ``margin`` (in u) from every interval
    boundary, midpoint and the FWM cut, with unique extrema."""
    while True:
        s = rand_row(rng, n, sigma)
        srt = np.sort(s)
        if np.min(np.diff(srt)) < 1e-3:
            continue
        M, m = s.max(), s.min()
        if calib == "minmax":
            u = K * (s - m) / (M - m)
            inner = (u > 1e-9) & (u < K - 1e-9)
        else:
            u = K * (s - M + tau) / tau
            inner = (u < K - 1e-9)
        frac = np.abs(2 * u - np.round(2 * u))
        if np.all(frac[inner] > 2 * margin):
            return s


@pytest.mark.parametrize("calib", CALIBS)
def test_lerp_full_gradient_matches_finite_differences(oracle_mod, calib):
    """LERP with the full calibration gradient is the exact Jacobian
    (Eq. full with Eq. calgrad; App. B, and its verification against autograd
    to < 1e-9). Central FD of L(s) = sum_j g_j P_j(s)."""
    rng = np.random.default_rng(8)
    tau = 6.0
    for K in (1, 2, 4, 16):
        for _ in range(8):
            s = safe_row(rng, 12, K, calib, tau, sigma=1.5)
            g = rng.normal(size=s.size)
            out = oracle_mod.row(s, g, K=K, calib=calib, tau=tau, recon="lerp")
            f = lambda x: float(np.dot(g, oracle_mod.row(x, K=K, calib=calib, tau=tau, recon="lerp")["P"]))
            fd = fd_grad(f, s, 1e-6)
            err = np.max(np.abs(fd - out["dS"])) / np.max(np.abs(fd))
            assert err < 1e-7, err


def lerp_weight_jacobian(oracle_mod, s, K, calib, tau, eps=1e-6):
    """J[j, i] = d w^L_j / d s_i by central differences of the oracle's w^L."""
    n = s.size
    J = np.zeros((n, n))
    for i in range(n):
        xp, xm = s.copy(), s.copy()
        xp[i] += eps
        xm[i] -= eps
        J[:, i] = (oracle_mod.row(xp, K=K, calib=calib, tau=tau)["wL"] -
                   oracle_mod.row(xm, K=K, calib=calib, tau=tau)["wL"]) / (2 * eps)
    return J


@pytest.mark.parametrize("calib", CALIBS)
@pytest.mark.parametrize("ste", ("weight", "prob"))
def test_ste_gradients_are_lerp_derivatives_at_their_point(oracle_mod, calib, ste):
    """Weight-STE: dS = J_{w^L}^T gamma^W, gamma^W = (g - <g>_{P^N}) / W^N
    (Eq. wste); Prob-STE: gamma^P = (g - <g>_{P^L}) / W^L (Eq. pste); both
    carry the LERP reconstruction derivatives incl. calibration (App. B)."""
    rng = np.random.default_rng(9)
    tau = 8.0
    for K in (2, 4, 16):
        for _ in range(6):
            s = safe_row(rng, 10, K, calib, tau, sigma=2.0)
            g = rng.normal(size=s.size)
            out = oracle_mod.row(s, g, K=K, calib=calib, tau=tau, recon="nearest", ste=ste)
            J = lerp_weight_jacobian(oracle_mod, s, K, calib, tau)
            if ste == "weight":
                PN = out["P"]          # forward P is the hard P^N
                gam = (g - np.dot(PN, g)) / out["WN"]
            else:
                PL = out["wL"] / out["WL"]
                gam = (g - np.dot(PL, g)) / out["WL"]
            ref = J.T @ gam
            err = np.max(np.abs(ref - out["dS"])) / np.max(np.abs(ref))
            assert err < 1e-7, err


@pytest.mark.parametrize("calib", CALIBS)
def test_surrogate_identities(oracle_mod, calib):
    """Prob-STE's backward is the Jacobian of normalize(w^L(s)), i.e. the
    LERP operator's dS; LERP makes the placement irrelevant; on grid points
    (w^N = w^L) Weight-STE equals Prob-STE (Sec. 3 / App. B)."""
    rng = np.random.default_rng(10)
    for K in (1, 4, 16):
        for _ in range(20):
            s = rand_row(rng, 15, 2.0)
            g = rng.normal(size=15)
            for detach in (False, True):
                lerp = oracle_mod.row(s, g, K=K, calib=calib, recon="lerp", detach=detach)
                lerp_p = oracle_mod.row(s, g, K=K, calib=calib, recon="lerp", ste="prob", detach=detach)
                prob = oracle_mod.row(s, g, K=K, calib=calib, recon="nearest", ste="prob", detach=detach)
                assert np.array_equal(lerp["dS"], lerp_p["dS"])
                assert np.array_equal(lerp["P"], lerp_p["P"])
                assert np.max(np.abs(prob["dS"] - lerp["dS"])) <= 1e-15 * (1 + np.max(np.abs(lerp["dS"])))
    K, m = 4, -2.0
    s = m + np.array([0, 1, 1, 2, 3, 4, 4, 0]) * 0.5
    g = rng.normal(size=s.size)
    w = oracle_mod.row(s, g, K=K, calib="minmax", recon="nearest", ste="weight")
    p = oracle_mod.row(s, g, K=K, calib="minmax", recon="nearest", ste="prob")
    assert np.max(np.abs(w["dS"] - p["dS"])) <= 1e-15


@pytest.mark.parametrize("calib", CALIBS)
@pytest.mark.parametrize("recon,ste", SURROGATES)
def test_zero_sum_full_and_violation_detach(oracle_mod, calib, recon, ste):
    """Full calibration gradient: Delta + dw/dM + dw/dm = 0 per key, so each
    row's dS sums to 0 (Sec. 3 zero-sum identity; FWM with dw/dM = -Delta).
    Detach keeps gamma Delta only and violates it (App. B detach; diagnostic
    A2 residuals)."""
    rng = np.random.default_rng(12)
    rho_detach = []
    for K in (1, 4, 16):
        for _ in range(30):
            s = rand_row(rng, 40, 2.5)
            g = rng.normal(size=40)
            full = oracle_mod.row(s, g, K=K, calib=calib, recon=recon, ste=ste)
            assert abs(full["dS"].sum()) <= 1e-13 * np.abs(full["dS"]).sum()
            det = oracle_mod.row(s, g, K=K, calib=calib, recon=recon, ste=ste, detach=True)
            rho_detach.append(abs(det["dS"].sum()) / np.abs(det["dS"]).sum())
    assert np.median(rho_detach) > 1e-3


@pytest.mark.parametrize("calib", CALIBS)
def test_calibration_terms_land_on_extrema_only(oracle_mod, calib):
    """g_full = g_self + g_M + g_m: full minus detach is nonzero only on the
    argmax (and MinMax argmin) keys, where it equals sum_j gamma_j dw_j/dM
    (resp. dm); cm = -(S_self + cM) and FWM cM = -S_self (App. B)."""
    rng = np.random.default_rng(13)
    for K in (2, 4, 16):
        for _ in range(20):
            s = rand_row(rng, 20, 2.0)
            g = rng.normal(size=20)
            full = oracle_mod.row(s, g, K=K, calib=calib, recon="nearest", ste="weight")
            det = oracle_mod.row(s, g, K=K, calib=calib, recon="nearest", ste="weight", detach=True)
            diff = full["dS"] - det["dS"]
            a, b = int(full["amax"]), int(full["amin"])
            mask = np.zeros(20, bool)
            mask[a] = True
            assert abs(diff[a] - full["cM"]) <= 1e-14
            if calib == "minmax":
                mask[b] = True
                assert abs(diff[b] - full["cm"]) <= 1e-14
                assert abs(full["cm"] + full["sself"] + full["cM"]) <= 1e-13
            else:
                assert abs(full["cM"] + full["sself"]) <= 1e-13
            assert np.all(diff[~mask] == 0.0)


def test_ties_split_evenly_and_stay_finite(oracle_mod):
    """Tied maxima/minima share the extremum gradient evenly (amax/amin
    convention, edge-case table); zero-sum still holds."""
    for calib in CALIBS:
        for K in (1, 4):
            s = np.array([1.0, 3.0, -2.0, 3.0, 0.5, -2.0, -2.0])
            g = np.array([0.2, 0.7, -0.1, 0.7, 0.4, -0.1, -0.1])
            out = oracle_mod.row(s, g, K=K, calib=calib, recon="nearest", ste="prob")
            assert out["nmax"] == 2 and out["amax"] == 1
            assert out["nmin"] == 3 and out["amin"] == 2
            assert out["dS"][1] == out["dS"][3]
            if calib == "minmax":
                assert out["dS"][2] == out["dS"][5] == out["dS"][6]
            assert abs(out["dS"].sum()) <= 1e-14
            assert np.isfinite(out["dS"]).all()


@pytest.mark.parametrize("calib", CALIBS)
@pytest.mark.parametrize("recon,ste", SURROGATES)
def test_p1_projection_is_a_zero_sum_shift_of_detach(oracle_mod, calib, recon, ste):
    """P1 (App. B, Detach): the projected detached row sums to zero, and it
    differs from plain detach by the same amount on every valid key (a
    per-row shift), while detach itself is not zero-sum."""
    rng = np.random.default_rng(21)
    for K in (1, 4, 16):
        for _ in range(20):
            n = int(rng.integers(2, 60))
            s = rand_row(rng, n, 2.5)
            g = rng.normal(size=n)
            det = oracle_mod.row(s, g, K=K, calib=calib, recon=recon, ste=ste, detach="detach")
            p1 = oracle_mod.row(s, g, K=K, calib=calib, recon=recon, ste=ste, detach="p1")
            scale = np.abs(det["dS"]).sum() + 1e-300
            assert abs(p1["dS"].sum()) <= 1e-13 * scale
            shift = p1["dS"] - det["dS"]
            assert np.ptp(shift) <= 1e-14 * scale
            assert np.allclose(shift, -det["dS"].sum() / n, rtol=1e-12, atol=1e-15 * scale)


@pytest.mark.parametrize("calib", CALIBS)
@pytest.mark.parametrize("recon,ste", SURROGATES)
def test_single_channel_modes(oracle_mod, calib, recon, ste):
    """max_only / min_only (appendix on the detached-gradient record: the
    single-channel ablation and the local decomposition): each adds to
    detach only on its own extremum's keys, ties split evenly, and the two
    channels add up to the full gradient; FWM has no minimum channel, so
    max_only is full and min_only is detach."""
    rng = np.random.default_rng(22)
    for K in (1, 4, 16):
        for trial in range(20):
            n = int(rng.integers(3, 50))
            s = rand_row(rng, n, 2.0)
            if trial % 4 == 0:  # exact ties of the max and of the min
                s[int(rng.integers(n))] = s.max()
                s[int(rng.integers(n))] = s.min()
            g = rng.normal(size=n)
            kw = dict(K=K, calib=calib, recon=recon, ste=ste)
            full = oracle_mod.row(s, g, detach="full", **kw)["dS"]
            det = oracle_mod.row(s, g, detach="detach", **kw)["dS"]
            mx = oracle_mod.row(s, g, detach="max_only", **kw)["dS"]
            mn = oracle_mod.row(s, g, detach="min_only", **kw)["dS"]
            gM, gm = mx - det, mn - det
            assert np.all(gM[s != s.max()] == 0.0)
            assert np.all(gm[s != s.min()] == 0.0)
            scale = np.abs(full).sum()
            # the same share on every tied key (up to the rounding of mx - det)
            assert np.ptp(gM[s == s.max()]) <= 1e-15 * scale
            assert np.ptp(gm[s == s.min()]) <= 1e-15 * scale
            assert np.allclose(det + gM + gm, full, rtol=0, atol=1e-14 * scale)
            if calib != "minmax":  # FWM and resolved: no minimum channel
                assert np.array_equal(mx, full) and np.array_equal(mn, det)


@pytest.mark.parametrize("calib", CALIBS)
def test_modes_at_attention_level(oracle_mod, calib):
    """Through the attention oracle: dV does not depend on the gradient mode
    (the value path has no calibration term), and under P1, as under the
    full gradient, every row of dS sums to zero, so the key gradients of a
    slice sum to zero, column by column."""
    rng = np.random.default_rng(23)
    B, H, T, d = 1, 2, 24, 16
    q, k, v, dO = (rng.normal(size=(B, H, T, d)) for _ in range(4))
    q = np.round(q * 8) / 8
    k = np.round(k * 8) / 8
    out = {}
    for mode in ("full", "detach", "max_only", "min_only", "p1"):
        out[mode] = oracle_mod.attn_bwd(q, k, v, dO, K=4, calib=calib, tau=8.0,
                                        recon="lerp", ste="weight", detach=mode,
                                        want_dS=True)
    dv_full = out["full"][2]
    for mode in out:  # (the oracle's threads add dV partials in any order)
        assert np.abs(out[mode][2] - dv_full).max() <= 1e-13 * np.abs(dv_full).max(), mode
    for mode in ("full", "p1"):
        dk, dS = out[mode][1], out[mode][4]
        assert np.abs(dS.sum(axis=-1)).max() <= 1e-12 * np.abs(dS).max()
        assert np.abs(dk.sum(axis=2)).max() <= 1e-11 * np.abs(dk).max()
    assert np.abs(out["detach"][4].sum(axis=-1)).max() > 1e-6


def test_degenerate_and_edge_rows(oracle_mod):
    """Edge-case table of App. A: degenerate MinMax rows (single key, equal
    scores, span <= 1e-12) give w = 1, uniform P and zero gradient; a span of
    1e-6 takes the regular branch and stays finite; FWM has no degenerate
    branch (single key / equal scores: all at the top grid value)."""
    eps = BOUNDS["degenerate_eps"]["value"]
    for recon, ste in SURROGATES:
        for detach in (False, True):
            kw = dict(recon=recon, ste=ste, detach=detach)
            one = oracle_mod.row([0.3], [1.0], K=4, calib="minmax", **kw)
            assert one["degen"] == 1 and one["P"][0] == 1.0 and one["dS"][0] == 0.0
            eq = oracle_mod.row([2.0] * 5, [1, 2, 3, 4, 5], K=4, calib="minmax", **kw)
            assert eq["degen"] == 1 and np.all(eq["P"] == 0.2) and np.all(eq["dS"] == 0.0)
            tiny = oracle_mod.row([1.0, 1.0 + eps / 2], [1.0, -1.0], K=4, calib="minmax", **kw)
            assert tiny["degen"] == 1
            small = oracle_mod.row([0.0, 1e-6, 5e-7], [1.0, -1.0, 0.5], K=4, calib="minmax", **kw)
            assert small["degen"] == 0
            assert np.isfinite(small["dS"]).all() and abs(small["P"].sum() - 1) < 1e-15
            f1 = oracle_mod.row([0.3], [1.0], K=4, calib="fwm", tau=8.0, **kw)
            assert f1["degen"] == 0 and f1["P"][0] == 1.0 and f1["dS"][0] == 0.0
            fe = oracle_mod.row([2.0] * 4, [1, 2, 3, 4], K=4, calib="fwm", tau=8.0, **kw)
            assert np.all(fe["P"] == 0.25) and np.isfinite(fe["dS"]).all()
            assert abs(fe["dS"].sum()) <= 1e-14


def test_hard_map_jacobian_and_negative_control(oracle_mod):
    """Eq. (hardjac): with indices fixed, d w^N_j / d s_i =
    c_j w^N_j (1[i=argmin] - 1[i=argmax]), c_j = 1 - l_j/K, checked by FD of
    the oracle's hard weights; the FWM hard map has zero Jacobian. The
    Weight-STE backward is NOT this derivative (App. B)."""
    rng = np.random.default_rng(14)
    K = 4
    for _ in range(10):
        s = safe_row(rng, 8, K, "minmax", 8.0, sigma=2.0)
        g = rng.normal(size=8)
        out = oracle_mod.row(s, g, K=K, calib="minmax", recon="nearest", ste="weight")
        n = s.size
        J = np.zeros((n, n))
        for i in range(n):
            xp, xm = s.copy(), s.copy()
            xp[i] += 1e-7
            xm[i] -= 1e-7
            J[:, i] = (oracle_mod.row(xp, K=K)["wN"] - oracle_mod.row(xm, K=K)["wN"]) / 2e-7
        a, b = int(out["amax"]), int(out["amin"])
        c = 1.0 - out["l"] / K
        ref = np.zeros((n, n))
        ref[:, b] += c * out["wN"]
        ref[:, a] -= c * out["wN"]
        assert np.max(np.abs(J - ref)) < 1e-6
        gam = (g - np.dot(out["P"], g)) / out["WN"]
        hard = J.T @ gam
        assert np.max(np.abs(hard - out["dS"])) > 1e-3 * np.max(np.abs(out["dS"]))
        fw = safe_row(rng, 8, K, "fwm", 8.0, sigma=2.0)
        Jf = np.zeros((n, n))
        for i in range(n):
            xp, xm = fw.copy(), fw.copy()
            xp[i] += 1e-7
            xm[i] -= 1e-7
            Jf[:, i] = (oracle_mod.row(xp, K=K, calib="fwm")["wN"] -
                        oracle_mod.row(xm, K=K, calib="fwm")["wN"])
        assert np.all(Jf == 0.0)


@pytest.mark.parametrize("calib", CALIBS)
def test_shift_invariance(oracle_mod, calib):
    """F(s + c 1) = F(s) (Sec. 3; diagnostic A1): with dyadic scores and a
    dyadic shift every step is exact, so P and dS are bitwise unchanged."""
    rng = np.random.default_rng(15)
    for K in (3, 4, 16):
        s = rng.integers(-64, 64, size=30) / 16.0
        g = rng.normal(size=30)
        for recon, ste in SURROGATES:
            a = oracle_mod.row(s, g, K=K, calib=calib, recon=recon, ste=ste)
            b = oracle_mod.row(s + 5.5, g, K=K, calib=calib, recon=recon, ste=ste)
            assert np.array_equal(a["P"], b["P"]) and np.array_equal(a["dS"], b["dS"])


# --------------------------------------------------------------------------
# Attention-level pins
# --------------------------------------------------------------------------

def safe_attn_inputs(rng, T, d, K, calib, tau, scale_qk=1.0):
    while True:
        q = rng.normal(size=(1, 1, T, d)) * scale_qk
        k = rng.normal(size=(1, 1, T, d)) * scale_qk
        s = (q[0, 0] @ k[0, 0].T) / math.sqrt(d)
        ok = True
        for i in range(1, T):
            row = s[i, : i + 1]
            if np.min(np.diff(np.sort(row))) < 1e-3:
                ok = False
                break
            M, m = row.max(), row.min()
            u = K * (row - m) / (M - m) if calib == "minmax" else K * (row - M + tau) / tau
            inner = (u > (-np.inf if calib == "resolved" else 1e-9)) & (u < K - 1e-9)
            if np.any(np.abs(2 * u - np.round(2 * u))[inner] < 4e-3):
                ok = False
                break
        if ok:
            return q, k


@pytest.mark.parametrize("calib", CALIBS)
def test_attention_gradients_match_finite_differences(oracle_mod, calib):
    """dQ, dK, dV of L = sum(dO * O) for LERP with the full gradient equal
    central differences (App. B value path dL/dV = P^T dO and the chain rule
    through S = Q K^T / sqrt(d); verification paragraph)."""
    rng = np.random.default_rng(16)
    T, d, K, tau = 6, 4, 4, 6.0
    q, k = safe_attn_inputs(rng, T, d, K, calib, tau)
    v = rng.normal(size=q.shape)
    dO = rng.normal(size=q.shape)
    kw = dict(K=K, calib=calib, tau=tau, recon="lerp", round_scores=False)
    dq, dk, dv, _, _ = oracle_mod.attn_bwd(q, k, v, dO, ste="weight", detach=False, **kw)

    def L(q_, k_, v_):
        o = oracle_mod.attn_fwd(q_, k_, v_, **kw)[0]
        return float(np.sum(o * dO))

    for name, x, ref in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        def f(flat):
            xx = flat.reshape(x.shape)
            args = {"q": q, "k": k, "v": v}
            args[name] = xx
            return L(args["q"], args["k"], args["v"])
        fd = fd_grad(f, x.ravel().copy(), 1e-6).reshape(x.shape)
        err = np.max(np.abs(fd - ref)) / np.max(np.abs(ref))
        assert err < 1e-7, (name, err)


def test_attention_nearest_value_gradient_is_hard_P(oracle_mod):
    """The value path uses the forward (hard) P: dL/dV = P^T dO (App. B);
    L is linear in V, so FD is exact up to rounding."""
    rng = np.random.default_rng(17)
    q = rng.normal(size=(1, 2, 7, 4))
    k = rng.normal(size=q.shape)
    v = rng.normal(size=q.shape)
    dO = rng.normal(size=q.shape)
    for calib in CALIBS:
        kw = dict(K=4, calib=calib, tau=8.0, recon="nearest")
        _, _, dv, _, _ = oracle_mod.attn_bwd(q, k, v, dO, ste="prob", detach=False, **kw)

        def f(flat):
            return float(np.sum(oracle_mod.attn_fwd(q, k, flat.reshape(v.shape), **kw)[0] * dO))
        fd = fd_grad(f, v.ravel().copy(), 1e-3).reshape(v.shape)
        assert np.max(np.abs(fd - dv)) < 1e-9


def test_attention_on_grid_is_causal_softmax_attention(oracle_mod):
    """With K = sqrt(d) I (T <= d) the scores are the entries of Q; placed on
    grid points, O equals causal softmax attention computed directly
    (Sec. 3 objects: S = QK^T/sqrt(d_h), P = w / W, O = P V; causal mask
    App. A)."""
    rng = np.random.default_rng(18)
    T = d = 16
    K = 4
    k = np.zeros((1, 1, T, d))
    k[0, 0] = np.eye(d) * math.sqrt(d)
    q = np.zeros((1, 1, T, d))
    for i in range(T):
        lv = rng.integers(0, K + 1, size=i + 1)
        lv[0] = 0
        lv[-1] = K
        q[0, 0, i, : i + 1] = -1.0 + lv * 0.5      # MinMax grid: h = 0.5
    v = rng.normal(size=(1, 1, T, d))
    for recon in ("lerp", "nearest"):
        o = oracle_mod.attn_fwd(q, k, v, K=K, calib="minmax", tau=8.0, recon=recon)[0]
        ref = np.zeros((T, d))
        for i in range(T):
            if i == 0:
                p = np.ones(1)
            else:
                p = softmax(q[0, 0, i, : i + 1])
            ref[i] = p @ v[0, 0, : i + 1]
        assert np.max(np.abs(o[0, 0] - ref)) < 1e-14


def test_dyadic_inputs_make_fp32_scores_exact(oracle_mod):
    """q, k in multiples of 1/8 with d in {16, 64}: q.k/sqrt(d) is exact in
    fp32, so the fp32-score oracle equals the fp64-score oracle bit for bit
    (the property the exact-score parity inputs rely on)."""
    rng = np.random.default_rng(19)
    for d in (16, 64):
        q = np.clip(np.round(rng.normal(size=(1, 2, 33, d)) * 8), -32, 32) / 8
        k = np.clip(np.round(rng.normal(size=(1, 2, 33, d)) * 8), -32, 32) / 8
        v = rng.normal(size=q.shape)
        a = oracle_mod.attn_fwd(q, k, v, K=4, calib="fwm", tau=8.0, recon="nearest",
                                round_scores=True, want_codes=True)
        b = oracle_mod.attn_fwd(q, k, v, K=4, calib="fwm", tau=8.0, recon="nearest",
                                round_scores=False, want_codes=True)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[3], b[3])
