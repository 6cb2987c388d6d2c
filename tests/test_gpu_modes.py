"""GPU parity of the backward's gradient modes beyond full/detach (max_only,
min_only, detach + P1 projection) and of the score-gradient decomposition
export (kia_debug_score_grad), against the fp64 oracle.

Bar as in test_gpu_parity: exact-score (dyadic) inputs, index codes and
extrema bit-exact, O within 1e-4, dQ/dK/dV within 1e-3 (fp32 inputs; 2e-2
for the bf16 variant). The decomposition: g_self (the detached dS) within
1e-4 of its largest magnitude per slice, and the channel row sums cM, cm
within 1e-4 of their largest magnitude.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402
import test_gpu_parity as P  # noqa: E402
import test_gpu_bf16 as P16  # noqa: E402

MODES = ("max_only", "min_only", "p1")
CASES = [(1, 1, 64, 16, 4, 1), (2, 1, 100, 64, 4, 1), (1, 2, 130, 32, 16, 1),
         (1, 1, 77, 64, 5, 0), (1, 1, 96, 128, 3, 1)]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("calib", ("minmax", "fwm"))
def test_modes_match_oracle(oracle_mod, mode, calib):
    for i, (B, H, T, d, K, causal) in enumerate(CASES):
        for recon, ste in (("lerp", "weight"), ("nearest", "prob"), ("nearest", "weight")):
            tag = f"{mode} {calib} {recon}/{ste} B{B} H{H} T{T} d{d} K{K} causal{causal}"
            P.flush("case " + tag)
            q, k, v, dO = make_inputs(B, H, T, d, seed=300 + i, qk_scale=1.5, dyadic=True)
            g = P.run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, mode, causal, codes=False)
            r = P.run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, mode, causal,
                             codes=False)
            P.compare(g, r, oracle_mod, calib, [(b, h) for b in range(B) for h in range(H)],
                      check_codes=False, tag=tag)


@pytest.mark.parametrize("mode", MODES)
def test_modes_bf16_match_oracle(oracle_mod, mode):
    for i, (B, H, T, d, K, causal) in enumerate(CASES):
        tag = f"bf16 {mode} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=320 + i, qk_scale=1.5, dyadic=True)
        (qb, kb, vb, db), (q, k, v, dO) = P16.bf16_inputs(q, k, v, dO)
        g = P16.run_gpu16(qb, kb, vb, db, K, "minmax", 8.0, "lerp", "weight", mode, causal,
                          codes=False)
        r = P.run_oracle(oracle_mod, q, k, v, dO, K, "minmax", 8.0, "lerp", "weight", mode,
                         causal, codes=False)
        P16.compare16(g, r, oracle_mod, "minmax", [(b, h) for b in range(B) for h in range(H)],
                      tag=tag)


def test_p1_full_size_gpt2_shape(oracle_mod):
    """P1 at the GPT-2-124M shape (LERP K=4 MinMax), one sampled slice."""
    P.full_size_check(oracle_mod, "gpt2_124m",
                      variant=dict(calib="minmax", recon="lerp", ste="weight", detach="p1"),
                      n_slices=1)


@pytest.mark.parametrize("calib", ("minmax", "fwm"))
@pytest.mark.parametrize("bf16", (False, True))
def test_score_grad_decomposition(oracle_mod, calib, bf16):
    """g_full = g_self + g_M + g_m: the exported detached dS and channel row
    sums against the oracle's detach-mode dS and its cM, cm."""
    B, H, T, d, K = 1, 2, 96, 64, 4
    q, k, v, dO = make_inputs(B, H, T, d, seed=340, qk_scale=1.5, dyadic=True)
    if bf16:
        (qg, kg, vg, dg), (q, k, v, dO) = P16.bf16_inputs(q, k, v, dO)
        qg, kg, vg, dg = (x.cuda() for x in (qg, kg, vg, dg))
    else:
        qg, kg, vg, dg = (x.cuda() for x in (q, k, v, dO))
    recon, ste = "lerp", "weight"
    o, st = kia.forward(qg, kg, vg, K, calib, 8.0, recon, ste, "full", True)
    kia.backward(qg, kg, vg, o, dg, st, K, calib, 8.0, recon, ste, "full", True)
    gs = torch.zeros((B, H, T, T), dtype=torch.float32, device="cuda")
    cM = torch.zeros((B, H, T), dtype=torch.float32, device="cuda")
    cm = torch.zeros_like(cM)
    kia.kia_debug_score_grad(st, gs, cM, cm, B, H, T, d, calib, recon, ste, True,
                             input_bf16=bf16)
    torch.cuda.synchronize()
    args = [x.double().numpy() for x in (q, k, v)]
    _, _, _, info, dS_det = oracle_mod.attn_bwd(*args, dO.double().numpy(), K=K, calib=calib,
                                               tau=8.0, recon=recon, ste=ste, detach="detach",
                                               want_dS=True)
    gs, cM, cm = (x.cpu().double().numpy() for x in (gs, cM, cm))
    tol = 2e-2 if bf16 else 1e-4
    RI = oracle_mod.RI
    for b in range(B):
        for h in range(H):
            ref = dS_det[b, h]
            assert np.abs(gs[b, h] - ref).max() <= tol * np.abs(ref).max(), (b, h)
            for x, key in ((cM, "cM"), (cm, "cm")):
                rx = info[b, h, :, RI[key]]  # (FWM: cM = -sum_j dS_j, cm = 0)
                den = max(np.abs(rx).max(), 1e-30)
                assert np.abs(x[b, h] - rx).max() <= tol * den, (b, h, key)
