"""Seeded synthetic inputs shared by the tests, the bench and the oracle
comparisons. This module holds no arithmetic of the method: it only draws
q, k, v, dO and describes the workloads.

The paper trains GPT-2-style models on FineWebEdu-3B / WikiText-103 with
fp32 attention; neither the corpora nor the checkpoints are used here.
Their attention shapes (124M: 12 heads, d_h = 64, T = 1024; a 1B-scale
shape; a long-context shape) are filled with i.i.d. N(0,1) draws instead,
in the order q, k, v, dO, from a CPU torch.Generator.
"""
from __future__ import annotations

import math

import torch

# name -> workload (shapes, operator variant, seed)
WORKLOADS = {
    "tiny": dict(B=1, H=1, T=64, d=16, K=4, calib="minmax", tau=8.0,
                 recon="lerp", ste="weight", detach=False, seed=0, qk_scale=1.0),
    "gpt2_124m": dict(B=8, H=12, T=1024, d=64, K=4, calib="fwm", tau=8.0,
                      recon="nearest", ste="prob", detach=False, seed=1, qk_scale=1.0),
    "scale_1b": dict(B=4, H=16, T=2048, d=128, K=16, calib="fwm", tau=8.0,
                     recon="nearest", ste="prob", detach=False, seed=20, qk_scale=1.0),
    "long_8k": dict(B=1, H=16, T=8192, d=128, K=4, calib="minmax", tau=8.0,
                    recon="lerp", ste="weight", detach=False, seed=21, qk_scale=2.0),
    # the paper's own call shapes: micro-batch 1 at T = 1024, d_h = 64, with
    # the 124M model's 12 heads and the 1B model's 24 heads (the operator of
    # the gpt2_124m workload)
    "paper_124m_mb1": dict(B=1, H=12, T=1024, d=64, K=4, calib="fwm", tau=8.0,
                           recon="nearest", ste="prob", detach=False, seed=30, qk_scale=1.0),
    "paper_1b_mb1": dict(B=1, H=24, T=1024, d=64, K=4, calib="fwm", tau=8.0,
                         recon="nearest", ste="prob", detach=False, seed=31, qk_scale=1.0),
}


def sweep_variants():
    """The variant sweep at the GPT-2-124M shape: {MinMax, FWM} x {LERP,
    Nearest} x {Weight, Prob} x K in {4, 16}, plus MinMax LERP with detached
    extrema at K in {4, 16}; seeds 2.. in this order."""
    out = []
    seed = 2
    for calib in ("minmax", "fwm"):
        for recon in ("lerp", "nearest"):
            for ste in ("weight", "prob"):
                for K in (4, 16):
                    out.append(dict(calib=calib, recon=recon, ste=ste, K=K,
                                    detach=False, seed=seed))
                    seed += 1
    for K in (4, 16):
        out.append(dict(calib="minmax", recon="lerp", ste="weight", K=K,
                        detach=True, seed=seed))
        seed += 1
    return out


def make_inputs(B, H, T, d, seed, qk_scale=1.0, dyadic=False):
    """q, k, v, dO as fp32 CPU tensors [B,H,T,d], N(0,1) in that order.

    dyadic=True rounds q and k to multiples of 1/8 in [-4, 4] (after the
    qk_scale), so that every q.k is exact in fp32 whatever the summation
    order, for d in {16, 32, 64, 128}: the exact-score parity inputs.
    """
    g = torch.Generator().manual_seed(int(seed))
    shape = (B, H, T, d)
    q = torch.randn(shape, generator=g, dtype=torch.float32) * qk_scale
    k = torch.randn(shape, generator=g, dtype=torch.float32) * qk_scale
    v = torch.randn(shape, generator=g, dtype=torch.float32)
    dO = torch.randn(shape, generator=g, dtype=torch.float32)
    if dyadic:
        q = torch.clamp(torch.round(q * 8), -32, 32) / 8
        k = torch.clamp(torch.round(k * 8), -32, 32) / 8
    return q, k, v, dO


def given_score_inputs(scores, d):
    """q, k [1,1,T,d] with k = sqrt(d) I (T <= d), so that for d in {16, 64}
    (power-of-two sqrt) the fp32 score of query i and key j is exactly
    scores[i, j]. Used to place scores on and around decision boundaries."""
    T = scores.shape[0]
    assert T <= d and d in (16, 64)
    q = torch.zeros(1, 1, T, d, dtype=torch.float32)
    q[0, 0, :, :T] = torch.as_tensor(scores, dtype=torch.float32)
    k = torch.zeros(1, 1, T, d, dtype=torch.float32)
    k[0, 0, :, :T] = torch.eye(T) * math.sqrt(d)
    return q, k
