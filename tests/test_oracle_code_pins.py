"""Pin of the oracle's index-code words (the per-pair codes of the forward,
compared bit for bit with the kernels' codes by the GPU parity tests):
decoded field by field, they must equal the exact-rational brute force of
App. A (interval r = floor with the clip, nearest level l with midpoints
rounding up, the FWM tail z < -tau), the degenerate MinMax branch of the
edge-case table (M - m <= 1e-12), the causal mask, and for the resolved
tail policy the two's-complement interval field (clamped at -8192). The
scores are placed exactly through k = sqrt(d) I, on grid points, midpoints,
one fp32 ulp either side of both, the FWM cut and far below it. CPU only."""
import math

import numpy as np
import pytest

from test_oracle_pins import _exact_indices

D = 64


def given(S):
    T = S.shape[0]
    q = np.zeros((1, 1, T, D))
    q[0, 0, :, :T] = S
    k = np.zeros((1, 1, T, D))
    k[0, 0, :, :T] = np.eye(T) * math.sqrt(D)
    return q, k


def boundary_values(K, calib, tau, rng):
    """fp32 scores on and around the decision boundaries of one row whose
    maximum is M (every value within 26 binades of the row scale)."""
    if calib == "minmax":
        m, M = -1.375, -1.375 + 0.5 * K
        base = m + np.arange(0, 2 * K + 1) * 0.25
    else:
        M, h = 0.8125, tau / K
        lo = -6 * K if calib == "resolved" else 0
        base = M - tau + np.arange(lo, 2 * K + 1) * (h / 2)
    base = base.astype(np.float32)
    up = np.nextafter(base, np.float32(np.inf))
    dn = np.nextafter(base, np.float32(-np.inf))
    s = np.concatenate([base, up, dn]).astype(np.float64)
    s = s[s <= M]
    if calib == "minmax":
        s = s[s >= base.min()]
    if calib == "fwm":
        cut = np.float32(M - tau)
        s = np.concatenate([s, [float(np.nextafter(cut, np.float32(-np.inf))), M - tau - 3.0]])
    s = s[np.abs(s) > 1e-6]
    return M, rng.permutation(s)


def rows_matrix(K, calib, tau, seed, T=64):
    """T x T fp32 score matrix: row i starts with its maximum, then
    boundary-placed values and random fp32 scores; a few rows are constant
    (MinMax degenerate)."""
    rng = np.random.default_rng(seed)
    M, vals = boundary_values(K, calib, tau, rng)
    S = np.empty((T, T))
    for i in range(T):
        pool = np.concatenate([vals, rng.uniform(M - (tau if calib != "minmax" else 0.5 * K),
                                                 M, size=T)]).astype(np.float32)
        row = rng.permutation(pool)[: T - 1].astype(np.float64)
        S[i] = np.concatenate([[M], row])
        S[i] = rng.permutation(S[i]) if i % 3 else S[i]
    S[5] = 0.75      # constant row: degenerate under MinMax
    S[9, :10] = -0.5  # causal prefix of row 9 constant
    return S


def decode(c, calib):
    c = c.astype(np.int64)
    if calib == "resolved":
        valid = (c >> 15) & 1
        up = (c >> 14) & 1
        r = c & 0x3FFF
        r = np.where(r >= 0x2000, r - 0x4000, r)
        return dict(valid=valid, r=r, l=r + up)
    return dict(valid=(c >> 14) & 1, degen=(c >> 15) & 1, tail=(c >> 13) & 1,
                r=c & 63, l=(c >> 6) & 127)


@pytest.mark.parametrize("calib", ("minmax", "fwm", "resolved"))
@pytest.mark.parametrize("causal", (1, 0))
@pytest.mark.parametrize("K", (1, 3, 4, 16))
def test_codes_decode_to_exact_decisions(oracle_mod, calib, causal, K):
    tau = 8.0
    S = rows_matrix(K, calib, tau, seed=100 * K + 10 * causal + len(calib))
    T = S.shape[0]
    q, k = given(S)
    v = np.zeros_like(q)
    _, info, _, codes = oracle_mod.attn_fwd(q, k, v, K, calib, tau, "nearest", causal=causal,
                                            want_codes=True)
    codes = codes[0, 0]
    for i in range(T):
        n = i + 1 if causal else T
        f = decode(codes[i], calib)
        assert np.all(codes[i, n:] == 0), (i, "keys past the causal limit carry no code")
        assert np.all(f["valid"][:n] == 1)
        s = S[i, :n]
        r, l, tail = _exact_indices(s, K, calib, tau)
        if calib == "minmax" and s.max() - s.min() <= 1e-12:
            assert np.all(codes[i, :n] == 0xC000), i   # valid | degenerate, r = l = 0
            assert info[0, 0, i, oracle_mod.RI["degen"]] == 1
            continue
        if calib == "resolved":
            assert np.array_equal(f["r"][:n], r) and np.array_equal(f["l"][:n], l), i
            continue
        assert np.all(f["degen"][:n] == 0)
        assert np.array_equal(f["tail"][:n], tail), i
        on = tail == 0
        assert np.all(codes[i, :n][~on] == 0x6000), i   # valid | tail, r = l = 0
        assert np.array_equal(f["r"][:n][on], r[on]), i
        assert np.array_equal(f["l"][:n][on], l[on]), i


def test_resolved_codes_clamp_far_intervals(oracle_mod):
    """The resolved interval field holds r down to -8192 exactly and clamps
    below; the level bit still says l = r + 1 (K = 64, tau = 1/2: a key 70
    nats below the maximum sits at u = -8896)."""
    K, tau = 64, 0.5
    zs = np.array([0.0, -0.25, -40.0, -63.5, -64.0, -64.0078125, -70.0, -70.00390625])
    S = np.tile(zs, (zs.size, 1))
    q, k = given(S)
    _, _, _, codes = oracle_mod.attn_fwd(q, k, np.zeros_like(q), K, "resolved", tau, "nearest",
                                         causal=False, want_codes=True)
    f = decode(codes[0, 0, 0], "resolved")
    r, l, _ = _exact_indices(zs, K, "resolved", tau)
    assert np.all(f["valid"] == 1)
    assert np.array_equal(f["r"], np.maximum(r, -8192))
    assert np.array_equal(f["l"] - f["r"], l - r)
    assert r.min() < -8192 and f["r"].min() == -8192
