"""Random parity sweep of the HIP path against the oracle (needs a GPU; not
collected by pytest).

    python tests/sweep_parity.py --seed 4 --fp32 1500 --bf16 600 --exp 800 \
        --bf16o 800 --forward-only 500

Each case draws an operator (calibration, reconstruction, surrogate,
gradient mode, K, tau), a shape (B, H, T from 1 to 1100 around tile edges,
every head size, causal or not), a grid policy and the deterministic switch,
on exact-score (dyadic) inputs, and checks it with the parity tests' own
comparisons:

* fp32: codes, stored decisions, extrema and ties bit-exact, W and O 1e-4,
  dQ/dK/dV 1e-3 (test_gpu_parity.compare);
* bf16 inputs: the same, O and gradients 2e-2 (test_gpu_bf16.compare16);
* exponential weight functions: test_gpu_expw.check (BF16-exp through its
  flip correction);
* bf16 inputs and outputs: O and gradients 2e-2;
* forward only: O of a KIA_GRAD_NONE forward bitwise that of the training
  forward (fp32, bf16 in, bf16 in and out).

A slice whose dQ/dK cancel below the rounding bound of their inputs
(test_gpu_parity.cancellation_floors; for bf16 with the operand rounding
2^-9) is held to its bar against that floor; such slices are counted and
printed.
Any other miss stops the sweep with the case.
"""
import argparse
import os
import random
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.dirname(HERE))

import torch  # noqa: E402

import oracle  # noqa: E402
import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402
import test_gpu_bf16 as B16  # noqa: E402
import test_gpu_expw as E  # noqa: E402
import test_gpu_parity as P  # noqa: E402

LENGTHS = [1, 2, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257, 300, 383, 400, 511, 640,
           1023, 1100]


def strict_then_floored(check, floors_of, tag):
    """Run check(floors=None); on a miss, run it again with the slices'
    cancellation floors. Returns True if the floors were needed."""
    try:
        check(None)
        return False
    except AssertionError as miss:
        check(floors_of())
        print(f"  cancellation floor: {tag}: {str(miss)[:160]}", flush=True)
        return True


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--seed", type=int, default=1)
    for leg in ("fp32", "bf16", "exp", "bf16o", "forward-only"):
        ap.add_argument("--" + leg, type=int, default=0, help=f"number of {leg} cases")
    a = ap.parse_args()
    legs = ([("fp32", a.fp32), ("bf16", a.bf16), ("exp", a.exp), ("bf16o", a.bf16o),
             ("forward-only", a.forward_only)])
    oracle.build(force=False)
    rng = random.Random(a.seed)
    t0, n, floored = time.time(), 0, 0
    for leg, count in legs:
        for _ in range(count):
            floored += run_case(rng, leg, n, a.seed)
            n += 1
    print(f"sweep ok: {n} cases ({', '.join(f'{c} {leg}' for leg, c in legs)}), "
          f"{floored} at the cancellation floor, {time.time() - t0:.1f} s", flush=True)


def run_case(rng, leg, n, seed):
    calib = rng.choice(["minmax", "fwm", "resolved"])
    recon = rng.choice(["lerp", "nearest"])
    ste = rng.choice(["weight", "prob"])
    mode = rng.choice(["full", "detach", "max_only", "min_only", "p1"])
    B, H = rng.choice([1, 2]), rng.choice([1, 2, 3])
    T = max(1, rng.choice(LENGTHS) + rng.choice([0, 0, 0, -1, 1, 7]))
    d = rng.choice([16, 32, 64, 128])
    K = rng.choice([1, 2, 3, 4, 5, 8, 16, 32, 64])
    tau = rng.choice([2.0, 4.0, 8.0, 12.0])
    sc = rng.choice([0.5, 1.0, 1.5, 2.5])
    causal = rng.choice([1, 1, 0])
    policy = rng.choice(["auto", "auto", "wide", "split"])
    det = rng.random() < 0.3
    if leg == "exp":
        recon = rng.choice(["softmax", "bf16_exp", "fp8_exp"])
        mode = rng.choice(["full", "detach", "max_only", "p1"])
        sc *= 2
    tag = (f"#{n} {leg} {calib} {recon} {ste} {mode} B{B} H{H} T{T} d{d} K{K} tau{tau} "
           f"scale{sc} causal{causal} {policy} det{int(det)}")
    P.flush("case " + tag)
    q, k, v, dO = make_inputs(B, H, T, d, seed=5000 + 1000 * seed + n, qk_scale=sc, dyadic=True)
    sl = [(b, h) for b in range(B) for h in range(H)]
    op = (K, calib, tau, recon, ste, mode, causal)
    kia.kia_set_grid_policy(policy)
    kia.kia_set_deterministic(det)
    try:
        if leg == "forward-only":
            for dt, out in ((torch.float32, None), (torch.bfloat16, None),
                            (torch.bfloat16, torch.bfloat16)):
                qg, kg, vg = (x.to(dt).cuda() for x in (q, k, v))
                o0, _ = kia.forward(qg, kg, vg, *op[:5], "full", causal, out_dtype=out)
                o1, _ = kia.forward(qg, kg, vg, *op[:5], "none", causal, out_dtype=out)
                assert torch.equal(o0, o1), tag
            return False
        if leg == "fp32":
            g = P.run_gpu(q, k, v, dO, *op)
            r = P.run_oracle(oracle, q, k, v, dO, *op)
            return strict_then_floored(
                lambda f: P.compare(g, r, oracle, calib, sl, tag=tag, floors=f),
                lambda: P.cancellation_floors(q, k, v, dO, sl), tag)
        if leg == "exp":
            g, r = E.run(oracle, q, k, v, dO, recon, mode, causal)
            return strict_then_floored(
                lambda f: E.check(g, r, oracle, sl, tag, floors=f),
                lambda: P.cancellation_floors(q, k, v, dO, sl), tag)
        (qb, kb, vb, db), (q, k, v, dO) = B16.bf16_inputs(q, k, v, dO)
        if leg == "bf16":
            g = B16.run_gpu16(qb, kb, vb, db, *op)
            r = P.run_oracle(oracle, q, k, v, dO, *op)
            return strict_then_floored(
                lambda f: B16.compare16(g, r, oracle, calib, sl, tag=tag, floors=f),
                lambda: P.cancellation_floors(q, k, v, dO, sl, B16.B16_TOL, 2.0 ** -9), tag)
        g = {x: y.double().numpy() for x, y in B16.run_bf16o(qb, kb, vb, db, *op).items()}
        r = P.run_oracle(oracle, q, k, v, dO, *op, codes=False)

        def check(f):
            f = f or {}
            errs = [P.rel_err(g[x], r[x], sl, f.get(x)) for x in ("o", "dq", "dk", "dv")]
            assert max(errs) <= B16.B16_TOL, (tag, errs)

        return strict_then_floored(
            check, lambda: P.cancellation_floors(q, k, v, dO, sl, B16.B16_TOL, 2.0 ** -9), tag)
    finally:
        kia.kia_set_grid_policy("auto")
        kia.kia_set_deterministic(False)


if __name__ == "__main__":
    main()
