"""Pins of the oracle's given-scores mode (App. A defines the operator on
rows of fp32 scores, so the scores a kernel computed can be handed to the
oracle as they are; q and k then enter only the products dQ = scale dS K
and dK = scale dS^T Q). CPU only.

1. Handed the fp32 scores that its own from-(q, k) path forms (computed
   here independently with numpy, exact for dyadic inputs), the given mode
   returns the same O, O^L, codes, row records and gradients bit for bit.
2. Scores placed on MinMax grid points, unrelated to q and k: every weight
   is e^z (Sec. 3), so O is the textbook softmax attention of those
   scores, dV = P^T dO with P = softmax, and dQ, dK are the products of the
   oracle's own dS with K and Q in the stated order.
"""
import math

import numpy as np
import pytest

from paper_2609_33591_amd.inputs import make_inputs


def fp32_scores(q, k):
    d = q.shape[-1]
    sc = np.float32(1.0 / math.sqrt(d))
    dot = (q.astype(np.float64) @ np.swapaxes(k.astype(np.float64), -1, -2)).astype(np.float32)
    return (dot * sc).astype(np.float32)


@pytest.mark.parametrize("calib,recon,ste", [("minmax", "lerp", "weight"),
                                             ("fwm", "nearest", "prob"),
                                             ("resolved", "nearest", "weight"),
                                             ("fwm", "bf16_exp", "weight")])
@pytest.mark.parametrize("causal", (1, 0))
def test_given_scores_equal_the_formed_ones(oracle_mod, calib, recon, ste, causal):
    q, k, v, dO = (x.double().numpy() for x in make_inputs(1, 2, 70, 32, seed=5, qk_scale=2.0,
                                                           dyadic=True))
    S = fp32_scores(q, k)
    a = dict(K=4, calib=calib, tau=8.0, recon=recon, causal=causal)
    o1, i1, ol1, c1 = oracle_mod.attn_fwd(q, k, v, want_ol=True, want_codes=True, **a)
    o2, i2, ol2, c2 = oracle_mod.attn_fwd(q, k, v, want_ol=True, want_codes=True, scores=S, **a)
    assert np.array_equal(o1, o2) and np.array_equal(ol1, ol2)
    assert np.array_equal(i1, i2) and np.array_equal(c1, c2)
    for detach in ("full", "detach", "p1"):
        g1 = oracle_mod.attn_bwd(q, k, v, dO, ste=ste, detach=detach, want_dS=True, **a)
        g2 = oracle_mod.attn_bwd(q, k, v, dO, ste=ste, detach=detach, want_dS=True, scores=S,
                                 **a)
        # dK, dV of a slice with fewer slices than threads are summed over
        # per-thread accumulators in arrival order (last-bit differences
        # from run to run); the rest is bitwise
        for name, x, y in zip(("dq", "dk", "dv", "info", "dS"), g1, g2):
            if name in ("dk", "dv"):
                assert np.max(np.abs(x - y)) <= 1e-14 * np.max(np.abs(x)), (detach, name)
            else:
                assert np.array_equal(x, y), (detach, name)


def test_grid_point_scores_give_softmax_attention(oracle_mod):
    """MinMax rows on grid points (K = 4, m = -2, M = 1, h = 3/4), scores
    unrelated to q and k, non-causal."""
    rng = np.random.default_rng(3)
    B, H, T, d, K = 1, 1, 24, 16, 4
    m, M = -2.0, 1.0
    lev = rng.integers(0, K + 1, size=(B, H, T, T))
    lev[..., 0] = 0
    lev[..., 1] = K                      # every row reaches m and M
    S = (m + lev * (M - m) / K).astype(np.float32)
    q, k, v, dO = (rng.normal(size=(B, H, T, d)) for _ in range(4))
    a = dict(K=K, calib="minmax", tau=8.0, causal=0, scores=S)
    for recon in ("lerp", "nearest"):
        o, info, _, _ = oracle_mod.attn_fwd(q, k, v, recon=recon, **a)
        dq, dk, dv, _, dS = oracle_mod.attn_bwd(q, k, v, dO, recon=recon, ste="weight",
                                               detach="full", want_dS=True, **a)
        z = S.astype(np.float64) - S.max(axis=-1, keepdims=True)
        P = np.exp(z) / np.exp(z).sum(axis=-1, keepdims=True)
        assert np.max(np.abs(o - P @ v)) <= 1e-13
        assert np.max(np.abs(dv - np.swapaxes(P, -1, -2) @ dO)) <= 1e-13
        sc = 1.0 / math.sqrt(d)
        assert np.max(np.abs(dq - sc * dS @ k)) <= 1e-12
        assert np.max(np.abs(dk - sc * np.swapaxes(dS, -1, -2) @ q)) <= 1e-12
        assert np.all(info[..., oracle_mod.RI["M"]] == M)
