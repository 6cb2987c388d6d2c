"""GPU parity of the bf16-input variant (kia_attn_fwd_bf16 / kia_attn_bwd_bf16)
against the fp64 oracle run on the same bf16-rounded inputs.

Bar: with dyadic q, k (multiples of 1/8 in [-4, 4], exact in bf16, so every
product and partial sum of a score is exact whatever the MFMA's order) the
scores equal the oracle's, and so must the index codes, extrema positions
and tie counts, bit for bit; W (an fp32 sum of fp32 weights) within 1e-4.
O, dQ, dK, dV within 2e-2 relative error (max |x - ref| / max |ref| per
slice): the second products round their computed operand (P, w^L, dS) to
bf16. For unrounded N(0,1) bf16 inputs the scores carry the fp32
accumulation error, so only the tolerances are checked.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import WORKLOADS, make_inputs  # noqa: E402
import test_gpu_parity as P  # noqa: E402

B16_TOL = 2e-2


def bf16_inputs(*xs):
    """The bf16 inputs and, as fp32, the exact values the oracle sees."""
    b = [x.to(torch.bfloat16) for x in xs]
    return b, [x.float() for x in b]


def run_gpu16(qb, kb, vb, db, K, calib, tau, recon, ste, detach, causal, codes=True,
              keep=None):
    B, H, T, d = qb.shape
    qg, kg, vg, dg = (x.cuda() for x in (qb, kb, vb, db))
    o, st = kia.forward(qg, kg, vg, K, calib, tau, recon, ste, detach, causal)
    stats = {f: kia.stats_field(st, B, H, T, d, f).clone() for f in P.STAT_KEYS}
    cd = cs = None
    if codes:
        cd = torch.zeros((B, H, T, T), dtype=torch.int16, device="cuda")
        kia.kia_debug_codes_bf16(qg, kg, st, cd, K, calib, tau, recon, causal)
        cs = P.stored_codes(st, B, H, T, d, K, calib, tau, recon, ste, causal)
    dq, dk, dv = kia.backward(qg, kg, vg, o, dg, st, K, calib, tau, recon, ste,
                              detach, causal)
    torch.cuda.synchronize()
    out = dict(o=o.cpu().double().numpy(), dq=dq.cpu().double().numpy(),
               dk=dk.cpu().double().numpy(), dv=dv.cpu().double().numpy())
    out.update({f: t.cpu().numpy() for f, t in stats.items()})
    pick = (lambda x: x) if keep is None else \
        (lambda x: x.reshape(-1, *x.shape[2:])[list(keep)].unsqueeze(0))
    if cd is not None:
        out["codes"] = pick(cd).cpu().numpy().view(np.uint16)
        out["codes_stored"] = pick(cs).cpu().numpy().view(np.uint16)
        after = P.stored_codes(st, B, H, T, d, K, calib, tau, recon, ste, causal)
        assert torch.equal(after, cs)
        assert torch.equal(cd, cs)
    return out


def compare16(g, r, oracle, calib, slices_bh, exact=True, tag="", floors=None):
    RI = oracle.RI
    for (b, h) in slices_bh:
        info = r["info"][b, h]
        w_err = np.max(np.abs(g["W"][b, h] - info[:, RI["W"]]) / info[:, RI["W"]])
        if exact:
            assert np.array_equal(g["M"][b, h].astype(np.float64), info[:, RI["M"]]), tag
            assert np.array_equal(g["amax"][b, h], info[:, RI["amax"]].astype(np.int32)), tag
            assert np.array_equal(g["nmax"][b, h], info[:, RI["nmax"]].astype(np.int32)), tag
            if calib == "minmax":
                assert np.array_equal(g["m"][b, h].astype(np.float64), info[:, RI["m"]]), tag
                assert np.array_equal(g["amin"][b, h], info[:, RI["amin"]].astype(np.int32)), tag
                assert np.array_equal(g["nmin"][b, h], info[:, RI["nmin"]].astype(np.int32)), tag
            assert w_err < P.O_TOL, (tag, w_err)
            if "codes" in g and r["codes"] is not None:
                for key in ("codes", "codes_stored"):
                    bad = np.argwhere(g[key][b, h] != r["codes"][b, h])
                    assert bad.size == 0, (tag, key, bad[:5])
        else:
            assert w_err < 1e-3, (tag, w_err)
    floors = floors or {}
    errs = [P.rel_err(g[x], r[x], slices_bh, floors.get(x)) for x in ("o", "dq", "dk", "dv")]
    assert max(errs) <= B16_TOL, (tag, errs)
    return errs


# (seed, B, H, T, d, K, tau, calib, recon, ste, mode), causal, qk_scale 1:
# two-key rows with a slice whose dQ cancels to ~5e-4 of its
# no-cancellation size (two such slices a random sweep of bf16 exact-score
# cases met)
ONE_HOT16 = [(10250, 2, 3, 2, 16, 16, 2.0, "fwm", "nearest", "weight", "max_only"),
             (10281, 2, 2, 2, 32, 1, 4.0, "fwm", "nearest", "prob", "full")]


@pytest.mark.parametrize("case", ONE_HOT16, ids=lambda c: f"seed{c[0]}")
def test_bf16_cancelling_slices_at_the_bf16_floor(oracle_mod, case):
    """The bf16 products round their computed operands (the forward's
    weights, so O and D = dO.O, and dS) to bf16, an error of up to 2^-9 of
    the operands. Where a slice's dQ or dK cancels below that rounding
    bound (test_gpu_parity.cancellation_floors with operand_eps 2^-9), its
    2e-2 bar is taken against the floor; the decisions, extrema, W, O and
    dV keep the usual bars, and the case must hold such a slice."""
    seed, B, H, T, d, K, tau, calib, recon, ste, mode = case
    P.flush(f"case bf16 one-hot seed{seed}")
    q, k, v, dO = make_inputs(B, H, T, d, seed=seed, qk_scale=1.0, dyadic=True)
    (qb, kb, vb, db), (q, k, v, dO) = bf16_inputs(q, k, v, dO)
    g = run_gpu16(qb, kb, vb, db, K, calib, tau, recon, ste, mode, 1)
    r = P.run_oracle(oracle_mod, q, k, v, dO, K, calib, tau, recon, ste, mode, 1)
    sl = [(b, h) for b in range(B) for h in range(H)]
    floors = P.cancellation_floors(q, k, v, dO, sl, tol=B16_TOL, operand_eps=2.0 ** -9)
    assert any(np.abs(r["dq"][b, h]).max() < floors["dq"][(b, h)] for (b, h) in sl)
    compare16(g, r, oracle_mod, calib, sl, tag=f"bf16 one-hot seed{seed}", floors=floors)


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_bf16_exact_score_parity_small(oracle_mod, variant):
    calib, recon, ste, detach = variant
    for i, (B, H, T, d, K, causal, sc) in enumerate(P.SHAPES):
        tag = f"bf16 {variant} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=200 + i, qk_scale=sc, dyadic=True)
        (qb, kb, vb, db), (q, k, v, dO) = bf16_inputs(q, k, v, dO)
        g = run_gpu16(qb, kb, vb, db, K, calib, 8.0, recon, ste, detach, causal)
        r = P.run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
        compare16(g, r, oracle_mod, calib, [(b, h) for b in range(B) for h in range(H)],
                  tag=tag)


def full_size16(oracle_mod, name, dyadic, n_slices=2, variant=None):
    w = dict(WORKLOADS[name])
    if variant:
        w.update(variant)
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], qk_scale=w["qk_scale"], dyadic=dyadic)
    (qb, kb, vb, db), (q, k, v, dO) = bf16_inputs(q, k, v, dO)
    args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"], 1)
    P.flush(f"case bf16 full {name} {variant} dyadic={dyadic}")
    sl = P.sample_slices(B, H, n_slices, w["seed"])
    idx = [b * H + h for (b, h) in sl]
    # unrounded inputs: the device still checks its recomputed codes
    # against its stored decisions on every slice; the oracle's codes are
    # compared on exact-score inputs
    g = run_gpu16(qb, kb, vb, db, *args, keep=idx)
    qs, ks, vs, ds = P.restrict(q, k, v, dO, sl)
    r = P.run_oracle(oracle_mod, qs, ks, vs, ds, *args, codes=dyadic)
    gs = {key: (val.reshape(-1, *val.shape[2:])[idx][None]
                if isinstance(val, np.ndarray) and not key.startswith("codes") else val)
          for key, val in g.items()}
    return compare16(gs, r, oracle_mod, w["calib"], [(0, i) for i in range(len(sl))],
                     exact=dyadic, tag=f"bf16 {name} {variant}")


def test_bf16_full_size_1b_exact_scores(oracle_mod):
    """1B-scale workload (B4 H16 T2048 d128, bf16 inputs; FWM, Nearest,
    Prob-STE, K=16), dyadic q, k: codes and extrema bit-exact."""
    full_size16(oracle_mod, "scale_1b", dyadic=True)


def test_bf16_full_size_1b_unrounded(oracle_mod):
    """The same workload with N(0,1) inputs rounded to bf16."""
    full_size16(oracle_mod, "scale_1b", dyadic=False)


@pytest.mark.parametrize("calib", ["minmax", "fwm", "resolved"])
def test_bf16_gpt2_shape(oracle_mod, calib):
    """GPT-2-124M shape with bf16 inputs, LERP and Nearest, one slice each."""
    for recon, ste in (("lerp", "weight"), ("nearest", "prob")):
        full_size16(oracle_mod, "gpt2_124m", dyadic=True, n_slices=1,
                    variant=dict(calib=calib, recon=recon, ste=ste))


def to_bf16_bits(x):
    """fp32 tensor -> bfloat16 (round to nearest even), as torch does."""
    return x.to(torch.bfloat16)


def run_bf16o(qb, kb, vb, db, K, calib, tau, recon, ste, detach, causal):
    """The bf16-output entry points (kia_attn_fwd_bf16o / kia_attn_bwd_bf16o)
    on the device; outputs as fp32 host arrays."""
    qg, kg, vg, dg = (x.cuda() for x in (qb, kb, vb, db))
    o, st = kia.forward(qg, kg, vg, K, calib, tau, recon, ste, detach, causal,
                        out_dtype=torch.bfloat16)
    dq, dk, dv = kia.backward(qg, kg, vg, o, dg, st, K, calib, tau, recon, ste, detach, causal)
    torch.cuda.synchronize()
    assert all(x.dtype == torch.bfloat16 for x in (o, dq, dk, dv))
    return {n: x.float().cpu() for n, x in zip(("o", "dq", "dk", "dv"), (o, dq, dk, dv))}


@pytest.mark.parametrize("variant", [("fwm", "nearest", "prob", False),
                                     ("minmax", "lerp", "weight", False),
                                     ("minmax", "nearest", "weight", True),
                                     ("resolved", "nearest", "prob", False),
                                     ("fwm", "lerp", "prob", "p1")],
                         ids=lambda v: "-".join(map(str, v)))
def test_bf16_output_variant(oracle_mod, variant):
    """bf16 o, dq, dk, dv on the parity shapes: within 2e-2 of the oracle.
    O is exactly the nearest-even rounding of the fp32-output path's O (the
    same kernels, one rounding at the store). So is dV when no grid is split
    (grid policy "wide"); under the default policy these small shapes split
    the main kernel's query ranges, whose parts add into dV atomically in an
    order that may vary, so dV is then within one bf16 rounding of the
    fp32-output value. dQ, dK are within one bf16 rounding of it for
    Prob-STE with Nearest (whose D comes from the fp32 O^L on both paths;
    elsewhere D takes the bf16 O)."""
    calib, recon, ste, detach = variant

    def one_rounding(x, f32):
        ulp = torch.maximum(f32.abs(), x.abs()) * 2.0 ** -7 + 1e-30
        return bool(torch.all((x - f32).abs() <= ulp))

    for i, (B, H, T, d, K, causal, sc) in enumerate(P.SHAPES):
        tag = f"bf16o {variant} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=300 + i, qk_scale=sc, dyadic=True)
        (qb, kb, vb, db), (q, k, v, dO) = bf16_inputs(q, k, v, dO)
        g = run_bf16o(qb, kb, vb, db, K, calib, 8.0, recon, ste, detach, causal)
        ref = run_gpu16(qb, kb, vb, db, K, calib, 8.0, recon, ste, detach, causal, codes=False)
        r = P.run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal,
                         codes=False)
        sl = [(b, h) for b in range(B) for h in range(H)]
        errs = [P.rel_err(g[x].double().numpy(), r[x], sl) for x in ("o", "dq", "dk", "dv")]
        assert max(errs) <= B16_TOL, (tag, errs)
        assert torch.equal(g["o"], to_bf16_bits(torch.from_numpy(ref["o"]).float()).float()), tag
        assert one_rounding(g["dv"], torch.from_numpy(ref["dv"]).float()), (tag, "dv")
        if recon == "nearest" and ste == "prob":
            for x in ("dq", "dk"):
                assert one_rounding(g[x], torch.from_numpy(ref[x]).float()), (tag, x)
        kia.kia_set_grid_policy("wide")
        try:
            gw = run_bf16o(qb, kb, vb, db, K, calib, 8.0, recon, ste, detach, causal)
            rw = run_gpu16(qb, kb, vb, db, K, calib, 8.0, recon, ste, detach, causal, codes=False)
        finally:
            kia.kia_set_grid_policy("auto")
        for x in ("o", "dv"):
            want = to_bf16_bits(torch.from_numpy(rw[x]).float())
            assert torch.equal(gw[x], want.float()), (tag, "wide", x)


@pytest.mark.parametrize("name", ("paper_124m_mb1", "paper_1b_mb1"))
def test_bf16_output_paper_call_shapes(oracle_mod, name):
    """The paper's micro-batch-1 call shapes (B1, T1024, d64, 12 or 24 heads;
    FWM, Nearest, Prob-STE, K=4) through the bf16-output entry points, every
    slice against the oracle at 2e-2."""
    w = WORKLOADS[name]
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], dyadic=True)
    (qb, kb, vb, db), (q, k, v, dO) = bf16_inputs(q, k, v, dO)
    args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"], 1)
    P.flush(f"case bf16o {name}")
    g = run_bf16o(qb, kb, vb, db, *args)
    r = P.run_oracle(oracle_mod, q, k, v, dO, *args, codes=False)
    sl = [(b, h) for b in range(B) for h in range(H)]
    errs = [P.rel_err(g[x].double().numpy(), r[x], sl) for x in ("o", "dq", "dk", "dv")]
    P.flush(f"  errors o dq dk dv: {errs}")
    assert max(errs) <= B16_TOL, (name, errs)
