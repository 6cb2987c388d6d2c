"""The deterministic backward (kia_set_deterministic) through the C ABI.

With the switch on, every reduction of the backward runs in a fixed order:
the key blocks' row sums are added up in key-block order, the calibration
terms of rows with unique extrema are gathered per key in row order, the
tied rows of a slice are taken by one wave, and no grid is split. So
repeated backward calls on the same forward must give bitwise equal dQ, dK
and dV, on shapes the default policy would split (small grids), on ragged
and non-causal shapes, and on given-score rows whose maxima (and minima)
are tied across several keys. The results still meet the parity bar
against the oracle (codes and extrema bit-exact, O 1e-4, dQ/dK/dV 1e-3;
bf16 inputs 2e-2), and differ from the default mode's only in fp32
summation order."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import WORKLOADS, make_inputs  # noqa: E402
import test_gpu_bf16 as B16  # noqa: E402
import test_gpu_parity as P  # noqa: E402

REPS = 3
# (calib, recon, ste, gradient mode)
VARIANTS = [("minmax", "lerp", "weight", "full"), ("fwm", "nearest", "prob", "full"),
            ("resolved", "nearest", "weight", "max_only"), ("minmax", "nearest", "prob", "min_only"),
            ("minmax", "lerp", "weight", "p1")]
# (B, H, T, d, K, causal): small grids (split by default), ragged tails,
# every head size, non-causal
SHAPES = [(1, 2, 300, 64, 4, 1), (1, 1, 257, 32, 16, 1), (2, 1, 130, 128, 3, 1),
          (1, 1, 77, 16, 5, 0)]


@pytest.fixture
def deterministic():
    kia.kia_set_deterministic(True)
    try:
        yield
    finally:
        kia.kia_set_deterministic(False)


def backward_reps(qg, kg, vg, dg, K, calib, tau, recon, ste, mode, causal):
    """One forward, then REPS backward calls on its statistics; host copies."""
    o, st = kia.forward(qg, kg, vg, K, calib, tau, recon, ste, mode, causal)
    reps = []
    for _ in range(REPS):
        g = kia.backward(qg, kg, vg, o, dg, st, K, calib, tau, recon, ste, mode, causal)
        torch.cuda.synchronize()
        reps.append([x.cpu() for x in g])
    return reps


def assert_bitwise(reps, tag):
    for rep in reps[1:]:
        for name, x, y in zip(("dq", "dk", "dv"), rep, reps[0]):
            assert torch.equal(x, y), (tag, name, float((x.float() - y.float()).abs().max()))


@pytest.mark.parametrize("variant", VARIANTS, ids=lambda v: "-".join(v))
def test_deterministic_backward_repeats_bitwise(oracle_mod, deterministic, variant):
    calib, recon, ste, mode = variant
    for i, (B, H, T, d, K, causal) in enumerate(SHAPES):
        tag = f"det {variant} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=900 + i, qk_scale=1.5, dyadic=True)
        reps = backward_reps(*(x.cuda() for x in (q, k, v, dO)), K, calib, 8.0, recon, ste,
                             mode, causal)
        assert_bitwise(reps, tag)
        # the parity bar, through the usual comparison (codes, extrema, O, grads)
        g = P.run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, mode, causal)
        for name, x in zip(("dq", "dk", "dv"), reps[0]):
            assert np.array_equal(g[name], x.double().numpy()), (tag, name)
        r = P.run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, mode, causal)
        P.compare(g, r, oracle_mod, calib, [(b, h) for b in range(B) for h in range(H)],
                  tag=tag)


@pytest.mark.parametrize("calib", ("minmax", "fwm"))
def test_deterministic_backward_with_tied_extrema(oracle_mod, deterministic, calib):
    """Given-score rows with exact ties of the maximum (and the minimum
    under MinMax), so that the tie path adds onto shared dK rows."""
    rng = np.random.default_rng(31)
    for d in (16, 64):
        T = d
        S = P.boundary_scores(rng, T, 4, calib, 8.0)
        q, k = P.given_score_inputs(S, d)
        v = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(d))
        dO = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(d + 1))
        for causal in (1, 0):
            tag = f"det ties {calib} d{d} causal{causal}"
            P.flush("case " + tag)
            reps = backward_reps(*(x.cuda() for x in (q, k, v, dO)), 4, calib, 8.0, "nearest",
                                 "prob", "full", causal)
            assert_bitwise(reps, tag)
            g = P.run_gpu(q, k, v, dO, 4, calib, 8.0, "nearest", "prob", "full", causal)
            assert np.any(g["nmax"][0, 0] > 1), "no tied maximum in the rows"
            r = P.run_oracle(oracle_mod, q, k, v, dO, 4, calib, 8.0, "nearest", "prob", "full",
                             causal)
            P.compare(g, r, oracle_mod, calib, [(0, 0)], tag=tag)


def test_deterministic_backward_bf16_inputs(oracle_mod, deterministic):
    for i, (B, H, T, d, K, causal) in enumerate(SHAPES):
        tag = f"det bf16 B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=950 + i, qk_scale=1.5, dyadic=True)
        (qb, kb, vb, db), (q, k, v, dO) = B16.bf16_inputs(q, k, v, dO)
        reps = backward_reps(*(x.cuda() for x in (qb, kb, vb, db)), K, "minmax", 8.0, "lerp",
                             "weight", "full", causal)
        assert_bitwise(reps, tag)
        r = P.run_oracle(oracle_mod, q, k, v, dO, K, "minmax", 8.0, "lerp", "weight", "full",
                         causal, codes=False)
        sl = [(b, h) for b in range(B) for h in range(H)]
        for name, x in zip(("dq", "dk", "dv"), reps[0]):
            assert P.rel_err(x.double().numpy(), r[name], sl) <= B16.B16_TOL, (tag, name)


def test_deterministic_backward_at_the_bench_shape(oracle_mod):
    """The GPT-2-124M bench workload (B8 H12 T1024 d64; FWM, Nearest,
    Prob-STE, K=4): two deterministic backward calls bitwise equal, within
    fp32 summation order of the default mode's, and every slice at the
    parity bar against the oracle on exact-score (dyadic) inputs."""
    w = WORKLOADS["gpt2_124m"]
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], "full", 1)
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], dyadic=True)
    qg, kg, vg, dg = (x.cuda() for x in (q, k, v, dO))
    P.flush("case det bench shape")
    default = backward_reps(qg, kg, vg, dg, *args)[0]
    kia.kia_set_deterministic(True)
    try:
        reps = backward_reps(qg, kg, vg, dg, *args)
    finally:
        kia.kia_set_deterministic(False)
    assert_bitwise(reps, "bench shape")
    for name, x, y in zip(("dq", "dk", "dv"), reps[0], default):
        den = float(y.abs().max())
        assert float((x - y).abs().max()) <= 1e-5 * den, name
    r = P.run_oracle(oracle_mod, q, k, v, dO, *args, codes=False)
    sl = [(b, h) for b in range(B) for h in range(H)]
    for name, x in zip(("dq", "dk", "dv"), reps[0]):
        assert P.rel_err(x.double().numpy(), r[name], sl) <= P.G_TOL, name


@pytest.mark.parametrize("recon", ("softmax", "bf16_exp", "fp8_exp"))
def test_deterministic_backward_exponential_weights(oracle_mod, recon):
    """The exponential weight functions keep the maximum on the gradient
    path (its channel lands on the argmax keys), so they take the gather
    too: repeated calls bitwise equal and, since the two modes share every
    kernel up to the reductions, within fp32 summation order (1e-5 of each
    tensor's largest value) of the default mode's gradients, which
    test_gpu_expw holds to the oracle. Softmax and FP8-exp also meet the
    1e-3 bar against the oracle here."""
    for i, (B, H, T, d, K, causal) in enumerate(SHAPES):
        tag = f"det {recon} B{B} H{H} T{T} d{d} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=970 + i, qk_scale=1.5, dyadic=True)
        args = ([x.cuda() for x in (q, k, v, dO)], (4, "fwm", 8.0, recon, "weight", "full", causal))
        default = backward_reps(*args[0], *args[1])[0]
        kia.kia_set_deterministic(True)
        try:
            reps = backward_reps(*args[0], *args[1])
        finally:
            kia.kia_set_deterministic(False)
        assert_bitwise(reps, tag)
        for name, x, y in zip(("dq", "dk", "dv"), reps[0], default):
            assert float((x - y).abs().max()) <= 1e-5 * float(y.abs().max()), (tag, name)
        if recon != "bf16_exp":
            r = P.run_oracle(oracle_mod, q, k, v, dO, 4, "fwm", 8.0, recon, "weight", "full",
                             causal, codes=False)
            sl = [(b, h) for b in range(B) for h in range(H)]
            for name, x in zip(("dq", "dk", "dv"), reps[0]):
                assert P.rel_err(x.double().numpy(), r[name], sl) <= P.G_TOL, (tag, name)
