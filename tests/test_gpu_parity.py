"""GPU parity of the HIP path (through the C-ABI) against the fp64 oracle.

Bar: index codes (interval r, nearest level l, FWM tail, degenerate rows),
argmax/argmin positions and tie counts bit-exact; O within 1e-4 and
dQ/dK/dV within 1e-3 relative error (max |x - ref| / max |ref| per (b,h)
slice, maximised over slices) for fp32 inputs.

Bit-exact index parity needs the kernel and the oracle to see the same fp32
scores; the score of a pair is a floating-point dot product whose rounding
depends on the summation order. Two input families make the scores exact:
dyadic q, k (multiples of 1/8, every q.k exact in fp32) and given scores
(k = sqrt(d) I). For unrounded N(0,1) inputs only what is unique is
compared bit for bit (rows whose keys all lie clear of every decision
boundary by the fp32 score error), the rest through invariants.
"""
import math
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import (WORKLOADS, given_score_inputs,  # noqa: E402
                                         make_inputs, sweep_variants)

O_TOL, G_TOL = 1e-4, 1e-3
STAT_KEYS = ("M", "m", "W", "WL", "amax", "amin", "nmax", "nmin")


def flush(msg):
    print(msg, flush=True)


def run_gpu(q, k, v, dO, K, calib, tau, recon, ste, detach, causal, codes=True,
            want_gself=False, keep=None):
    """Forward (plus index codes recomputed and decoded from the stored
    decisions) and backward on the device; returns host arrays. keep: the
    flattened (b,h) slice indices of the [B,H,T,T] arrays to bring back as
    [1, n, T, T] (all slices if None)."""
    B, H, T, d = q.shape
    qg, kg, vg, dg = (x.cuda() for x in (q, k, v, dO))
    o, st = kia.forward(qg, kg, vg, K, calib, tau, recon, ste, detach, causal)
    stats = {f: kia.stats_field(st, B, H, T, d, f).clone() for f in STAT_KEYS}
    cd = cs = None
    if codes:
        # the codes recomputed by the forward's device code, and the decoded
        # decisions the forward stored for the backward (stats field U)
        cd = torch.zeros((B, H, T, T), dtype=torch.int16, device="cuda")
        kia.kia_debug_codes(qg, kg, st, cd, K, calib, tau, recon, causal)
        cs = stored_codes(st, B, H, T, d, K, calib, tau, recon, ste, causal)
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
        # the backward reads U and leaves it as the forward wrote it; the
        # recomputed codes equal the stored decisions on every slice
        after = stored_codes(st, B, H, T, d, K, calib, tau, recon, ste, causal)
        assert torch.equal(after, cs)
        assert torch.equal(cd, cs)
        del cd, cs, after
    if want_gself:
        # the detached score gradient as the backward computed it (its dS
        # scratch holds it under every gradient mode)
        gs = torch.zeros((B, H, T, T), dtype=torch.float32, device="cuda")
        cM = torch.zeros((B, H, T), dtype=torch.float32, device="cuda")
        kia.kia_debug_score_grad(st, gs, cM, torch.zeros_like(cM), B, H, T, d, calib, recon,
                                 ste, causal)
        out["g_self"] = pick(gs).cpu().double().numpy()
    return out


def stored_codes(st, B, H, T, d, K, calib, tau, recon, ste, causal):
    cs = torch.zeros((B, H, T, T), dtype=torch.int16, device="cuda")
    kia.kia_debug_codes_stored(st, cs, B, H, T, d, K, calib, tau, recon, ste, causal)
    return cs


def run_oracle(oracle, q, k, v, dO, K, calib, tau, recon, ste, detach, causal,
               slices=None, codes=True):
    args = [x.double().numpy() for x in (q, k, v)]
    o, info, _, cd = oracle.attn_fwd(*args, K=K, calib=calib, tau=tau, recon=recon,
                                     causal=causal, want_codes=codes, slices=slices)
    dq, dk, dv, _, _ = oracle.attn_bwd(*args, dO.double().numpy(), K=K, calib=calib,
                                       tau=tau, recon=recon, ste=ste, detach=detach,
                                       causal=causal, slices=slices)
    return dict(o=o, dq=dq, dk=dk, dv=dv, info=info, codes=cd)


def oracle_grad(mode):
    """The gradient mode's name (False/True are full/detach)."""
    if isinstance(mode, str):
        return mode
    return {0: "full", 1: "detach", 2: "max_only", 3: "min_only", 4: "p1"}[int(mode)]


def oracle_scores(q, k):
    """fp32 scores fl32(fl32(q.k) fl32(1/sqrt(d))) in numpy from the fp64
    dot product (exact for the exact-score inputs), as fp64 [B,H,T,T]."""
    d = q.shape[-1]
    sc = np.float32(1.0 / math.sqrt(d))
    dot = (q.double().numpy() @ np.swapaxes(k.double().numpy(), -1, -2)).astype(np.float32)
    return (dot * sc).astype(np.float32).astype(np.float64)


def rel_err(x, ref, sl, floor=None):
    """max over (b,h) slices in sl of max|x - ref| / max|ref| (or / the
    slice's floor[(b, h)] where that is larger)."""
    worst = 0.0
    for (b, h) in sl:
        den = np.max(np.abs(ref[b, h]))
        if floor is not None:
            den = max(den, floor[(b, h)])
        num = np.max(np.abs(x[b, h] - ref[b, h]))
        worst = max(worst, num / den if den > 0 else num)
    return worst


def compare(g, r, oracle, calib, slices_bh, check_codes=True, tag="", floors=None):
    RI = oracle.RI
    for (b, h) in slices_bh:
        info = r["info"][b, h]
        assert np.array_equal(g["M"][b, h].astype(np.float64), info[:, RI["M"]]), tag
        assert np.array_equal(g["amax"][b, h], info[:, RI["amax"]].astype(np.int32)), tag
        assert np.array_equal(g["nmax"][b, h], info[:, RI["nmax"]].astype(np.int32)), tag
        if calib == "minmax":
            assert np.array_equal(g["m"][b, h].astype(np.float64), info[:, RI["m"]]), tag
            assert np.array_equal(g["amin"][b, h], info[:, RI["amin"]].astype(np.int32)), tag
            assert np.array_equal(g["nmin"][b, h], info[:, RI["nmin"]].astype(np.int32)), tag
        # W (fp32 sum of up to T weights) enters O as a divisor: O's bound
        w_err = np.max(np.abs(g["W"][b, h] - info[:, RI["W"]]) / info[:, RI["W"]])
        assert w_err < O_TOL, (tag, w_err)
        if check_codes:
            for key in ("codes", "codes_stored"):
                bad = np.argwhere(g[key][b, h] != r["codes"][b, h])
                assert bad.size == 0, (tag, key, bad[:5], g[key][b, h][tuple(bad[0])],
                                       r["codes"][b, h][tuple(bad[0])])
    eo = rel_err(g["o"], r["o"], slices_bh)
    floors = floors or {}
    eq = rel_err(g["dq"], r["dq"], slices_bh, floors.get("dq"))
    ek = rel_err(g["dk"], r["dk"], slices_bh, floors.get("dk"))
    ev = rel_err(g["dv"], r["dv"], slices_bh)
    assert eo <= O_TOL, (tag, "O", eo)
    assert eq <= G_TOL and ek <= G_TOL and ev <= G_TOL, (tag, eq, ek, ev)
    return eo, eq, ek, ev


VARIANTS = [(c, rc, s, dt) for c in ("minmax", "fwm", "resolved") for rc in ("lerp", "nearest")
            for s in ("weight", "prob") for dt in (False, True)]
# (B, H, T, d, K, causal, qk_scale): tiles, ragged tails, every head size
SHAPES = [(1, 1, 1, 16, 4, 1, 1.0), (1, 2, 33, 16, 1, 1, 1.0), (2, 1, 100, 64, 4, 1, 1.0),
          (1, 1, 257, 32, 16, 1, 2.5), (1, 2, 130, 128, 3, 1, 1.0), (1, 1, 77, 64, 5, 0, 2.0),
          (1, 1, 300, 64, 64, 1, 1.5)]


@pytest.mark.parametrize("variant", VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_exact_score_parity_small(oracle_mod, variant):
    calib, recon, ste, detach = variant
    for i, (B, H, T, d, K, causal, sc) in enumerate(SHAPES):
        tag = f"{variant} B{B} H{H} T{T} d{d} K{K} causal{causal}"
        flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=100 + i, qk_scale=sc, dyadic=True)
        g = run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
        r = run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
        compare(g, r, oracle_mod, calib, [(b, h) for b in range(B) for h in range(H)], tag=tag)


@pytest.mark.parametrize("policy", ("wide", "split"))
@pytest.mark.parametrize("variant", [("minmax", "lerp", "weight", False),
                                     ("fwm", "nearest", "prob", False),
                                     ("resolved", "nearest", "prob", True)],
                         ids=lambda v: "-".join(map(str, v)))
def test_exact_score_parity_grid_policies(oracle_mod, policy, variant):
    """The small shapes again with the launch shape forced: "wide" takes the
    forward's two row groups x two key halves and the unsplit backward, which
    the default policy keeps for grids that fill the chip; "split" takes four
    key quarters (d <= 64) and the split backward at every size."""
    calib, recon, ste, detach = variant
    kia.kia_set_grid_policy(policy)
    try:
        for i, (B, H, T, d, K, causal, sc) in enumerate(SHAPES):
            tag = f"{policy} {variant} B{B} H{H} T{T} d{d} K{K} causal{causal}"
            flush("case " + tag)
            q, k, v, dO = make_inputs(B, H, T, d, seed=100 + i, qk_scale=sc, dyadic=True)
            g = run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
            r = run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
            compare(g, r, oracle_mod, calib, [(b, h) for b in range(B) for h in range(H)],
                    tag=tag)
    finally:
        kia.kia_set_grid_policy("auto")


def boundary_scores(rng, T, K, calib, tau):
    """fp32 scores per row placed on grid points, midpoints, one ulp either
    side of them, on exact ties of the max/min and (FWM) on the cut."""
    S = np.zeros((T, T), dtype=np.float32)
    for i in range(T):
        M = np.float32(rng.integers(-8, 8) / 4)
        if calib == "minmax":
            span = np.float32(K * 0.25 * rng.integers(1, 5))
            m = np.float32(M - span)
            u = rng.integers(0, 2 * K + 1, size=T) / 2.0
            base = (m + u * (span / K)).astype(np.float32)
        else:
            # FWM: around the cut and above; resolved: far below the cut too
            lo = -8 * K if calib == "resolved" else -4
            u = rng.integers(lo, 2 * K + 1, size=T) / 2.0
            base = (M - tau + u * (tau / K)).astype(np.float32)
        jig = rng.integers(-1, 2, size=T)
        row = base.copy()
        row[jig == 1] = np.nextafter(base[jig == 1], np.float32(np.inf))
        row[jig == -1] = np.nextafter(base[jig == -1], np.float32(-np.inf))
        row = np.minimum(row, M)
        if calib == "minmax":
            row = np.maximum(row, m)
            row[rng.integers(0, T)] = m
        row[rng.integers(0, T)] = M
        row[rng.integers(0, T)] = M   # likely a tie of the maximum
        S[i] = row
    return S


@pytest.mark.parametrize("calib", ("minmax", "fwm", "resolved"))
@pytest.mark.parametrize("causal", (1, 0))
def test_given_scores_on_decision_boundaries(oracle_mod, calib, causal):
    rng = np.random.default_rng(7 if calib == "minmax" else 8)
    for d in (16, 64):
        T = d
        for K in (1, 4, 16):
            S = boundary_scores(rng, T, K, calib, 8.0)
            q, k = given_score_inputs(S, d)
            v = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(K))
            dO = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(K + 1))
            for recon, ste in (("lerp", "weight"), ("nearest", "weight"), ("nearest", "prob")):
                tag = f"given {calib} causal{causal} d{d} K{K} {recon}-{ste}"
                flush("case " + tag)
                g = run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, False, causal)
                r = run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste, False, causal)
                compare(g, r, oracle_mod, calib, [(0, 0)], tag=tag)


def edge_case_scores(T):
    """Rows of the App. A edge-case table as fp32 scores (row 0 of a causal
    call has a single valid key): constant rows (degenerate under MinMax, all
    keys on the top level under FWM), a span of 1e-6 (MinMax's regular
    branch with h = 2.5e-7 at K = 4), spans just below and above the
    degenerate threshold 1e-12 near zero, exact ties of the maximum and the
    minimum, two-valued rows, and FWM rows with every key but the maximum
    beyond the window or exactly on the cut."""
    S = np.zeros((T, T), dtype=np.float32)
    rng = np.random.default_rng(17)
    for i in range(T):
        kind = i % 9
        if kind == 0:
            row = np.full(T, np.float32(0.75))
        elif kind == 1:
            row = (np.float32(-0.5) + np.float32(1e-6) * rng.random(T)).astype(np.float32)
            row[rng.integers(0, T)] = np.float32(-0.5)
            row[rng.integers(0, T)] = np.float32(-0.5) + np.float32(1e-6)
        elif kind == 2:
            row = np.where(rng.random(T) < 0.5, 0.0, 1e-13).astype(np.float32)
        elif kind == 3:
            row = np.where(rng.random(T) < 0.5, 0.0, 3e-12).astype(np.float32)
        elif kind == 4:
            row = rng.choice(np.array([-1.0, 0.0, 2.0], dtype=np.float32), size=T)
        elif kind == 5:
            row = np.full(T, np.float32(-9.0))
            row[:: 3] = np.float32(0.0)
        elif kind == 6:
            row = np.full(T, np.float32(-8.0))        # on the FWM cut (tau = 8)
            row[rng.integers(0, T)] = np.float32(0.0)
        elif kind == 7:
            row = np.full(T, np.float32(-20.0))       # far in the FWM tail
            row[1::4] = np.float32(1.5)
        else:
            row = (rng.normal(size=T) * 3).astype(np.float32)
            row[rng.integers(0, T, size=3)] = row.max()
            row[rng.integers(0, T, size=3)] = row.min()
        S[i] = row
    return S


@pytest.mark.parametrize("calib", ("minmax", "fwm", "resolved"))
def test_given_scores_edge_case_rows(oracle_mod, calib):
    """The edge-case rows of App. A through the operator (codes, extrema and
    stored decisions bit-exact; O, dQ, dK, dV at the usual bar), causal and
    not, every surrogate, full and detached gradients."""
    for d in (16, 64):
        T = d
        S = edge_case_scores(T)
        q, k = given_score_inputs(S, d)
        v = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(d))
        dO = torch.randn(1, 1, T, d, generator=torch.Generator().manual_seed(d + 1))
        for causal in (1, 0):
            for K in (1, 4):
                for recon, ste in (("lerp", "weight"), ("nearest", "weight"), ("nearest", "prob")):
                    for detach in (False, True):
                        tag = f"edge {calib} causal{causal} d{d} K{K} {recon}-{ste} det{detach}"
                        flush("case " + tag)
                        g = run_gpu(q, k, v, dO, K, calib, 8.0, recon, ste, detach, causal)
                        r = run_oracle(oracle_mod, q, k, v, dO, K, calib, 8.0, recon, ste,
                                       detach, causal)
                        compare(g, r, oracle_mod, calib, [(0, 0)], tag=tag)


# ---------------------------------------------------------------------------
# Near one-hot slices: the score gradient cancels to below fp32's resolution
# ---------------------------------------------------------------------------
def cancellation_floors(q, k, v, dO, sl, tol=None, operand_eps=0.0):
    """Per slice, the max|ref| below which the relative bar `tol` (default
    G_TOL) is taken against a floor: the worst-case rounding of the
    gradient's inputs, as a fraction of the size dQ (dK) would have without
    cancellation, G max|k| (G max|q|) with G = d^-1/2 max_ij sum_k
    |dO_ik v_jk|. The two fp32 dot products behind g = dO.v and D each err
    by at most gamma_d = d 2^-24 of that scale (the standard bound for a
    dot product of length d); operand_eps adds the bf16 rounding of the
    products' computed operands (2^-9 for the bf16 variant). The floor is
    (2 gamma_d + operand_eps) / tol of the size, so that the bar there
    equals that rounding bound."""
    tol = G_TOL if tol is None else tol
    d = q.shape[-1]
    frac = (2 * d * 2.0 ** -24 + operand_eps) / tol
    floors = {"dq": {}, "dk": {}}
    for (b, h) in sl:
        qn, kn, vn, dn = (x[b, h].double().numpy() for x in (q, k, v, dO))
        G = (np.abs(dn) @ np.abs(vn).T).max() / math.sqrt(d)
        floors["dq"][(b, h)] = frac * G * np.abs(kn).max()
        floors["dk"][(b, h)] = frac * G * np.abs(qn).max()
    return floors


# (seed, B, H, T, d, K, tau, qk_scale, calib, recon, ste, mode), causal: rows
# of two keys whose scores lie so far apart that the row is one-hot up to
# ~1e-6, so the score gradient is a rounding-size fraction of dO v^T (the
# two such slices a random sweep of 3000 exact-score cases met)
ONE_HOT = [(7052, 1, 3, 2, 32, 3, 12.0, 2.5, "resolved", "nearest", "prob", "detach"),
           (7918, 2, 3, 2, 32, 16, 8.0, 2.5, "minmax", "nearest", "weight", "max_only")]


@pytest.mark.parametrize("case", ONE_HOT, ids=lambda c: f"seed{c[0]}")
def test_near_one_hot_slices_at_the_fp32_floor(oracle_mod, case):
    """Where a slice's dQ or dK has cancelled below the fp32 rounding bound
    of its inputs (cancellation_floors), its 1e-3 relative bar is taken
    against that floor. Every decision, the extrema, W, O and dV keep the
    usual bars, and the case must hold such a slice."""
    seed, B, H, T, d, K, tau, sc, calib, recon, ste, mode = case
    flush(f"case one-hot seed{seed}")
    q, k, v, dO = make_inputs(B, H, T, d, seed=seed, qk_scale=sc, dyadic=True)
    g = run_gpu(q, k, v, dO, K, calib, tau, recon, ste, mode, 1)
    r = run_oracle(oracle_mod, q, k, v, dO, K, calib, tau, recon, ste, mode, 1)
    sl = [(b, h) for b in range(B) for h in range(H)]
    floors = cancellation_floors(q, k, v, dO, sl)
    assert any(np.abs(r["dq"][b, h]).max() < floors["dq"][(b, h)] for (b, h) in sl)
    compare(g, r, oracle_mod, calib, sl, tag=f"one-hot seed{seed}", floors=floors)


def sample_slices(B, H, n, seed):
    rng = np.random.default_rng(seed)
    flat = rng.choice(B * H, size=min(n, B * H), replace=False)
    return sorted((int(f) // H, int(f) % H) for f in flat)


def restrict(q, k, v, dO, sl):
    """Inputs of the sampled (b,h) slices stacked as [1, n, T, d]."""
    idx = [b * q.shape[1] + h for (b, h) in sl]
    f = lambda x: x.reshape(-1, *x.shape[2:])[idx].unsqueeze(0)
    return f(q), f(k), f(v), f(dO)


def full_size_check(oracle_mod, name, variant=None, n_slices=2, dyadic=True):
    """The workload at its full size on the device; n_slices sampled (b,h)
    slices (all of them if n_slices >= B*H) against the oracle, codes and
    stored decisions included (the device compares its recomputed codes
    with its stored decisions on every slice)."""
    w = dict(WORKLOADS[name])
    if variant:
        w.update(variant)
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], qk_scale=w["qk_scale"], dyadic=dyadic)
    args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"], 1)
    sl = sample_slices(B, H, n_slices, w["seed"])
    idx = [b * H + h for (b, h) in sl]
    flush(f"case full {name} {variant} dyadic={dyadic} slices={len(sl)}")
    g = run_gpu(q, k, v, dO, *args, keep=idx)
    qs, ks, vs, ds = restrict(q, k, v, dO, sl)
    r = run_oracle(oracle_mod, qs, ks, vs, ds, *args)
    gs = {key: (val.reshape(-1, *val.shape[2:])[idx][None]
                if isinstance(val, np.ndarray) and not key.startswith("codes") else val)
          for key, val in g.items()}
    return compare(gs, r, oracle_mod, w["calib"], [(0, i) for i in range(len(sl))],
                   tag=f"{name} {variant}")


def test_full_size_gpt2_124m_exact_scores(oracle_mod):
    """Every one of the 96 (b,h) slices of the bench shape."""
    full_size_check(oracle_mod, "gpt2_124m", n_slices=96)


def test_full_size_tiny(oracle_mod):
    full_size_check(oracle_mod, "tiny", n_slices=1, dyadic=True)


@pytest.mark.parametrize("v", sweep_variants(), ids=lambda v: f"{v['calib']}-{v['recon']}-{v['ste']}-K{v['K']}{'-detach' if v['detach'] else ''}")
def test_variant_sweep_gpt2_shape(oracle_mod, v):
    full_size_check(oracle_mod, "gpt2_124m", variant=v, n_slices=1)


# ---------------------------------------------------------------------------
# Unrounded N(0,1) inputs (the bench's inputs): unique parts compared exactly
# ---------------------------------------------------------------------------

def fp32_scores_and_bound(q, k):
    """fp32 scores as the oracle forms them, and a bound on how far the
    kernel's fp32 MFMA score of the same pair can lie from it: one rounding
    per 2-term MFMA step of the running sum plus the two final roundings."""
    d = q.shape[-1]
    sc = np.float32(1.0 / math.sqrt(d))
    q64, k64 = q.double().numpy(), k.double().numpy()
    dot = q64 @ np.swapaxes(k64, -1, -2)
    s = (dot.astype(np.float32) * sc).astype(np.float32).astype(np.float64)
    A = np.abs(q64) @ np.abs(np.swapaxes(k64, -1, -2))
    eps = float(sc) * (d / 2 + 2) * 2.0 ** -24 * A + 2.0 ** -23 * np.abs(s)
    return s, eps


def ambiguity(s, eps, K, calib, tau, causal=True):
    """Per (b,h,row): True if some decision of the row could go either way
    within the score error bound (extremum order/ties, an interval or level
    boundary, the FWM cut)."""
    B, H, T, _ = s.shape
    amb = np.zeros((B, H, T), dtype=bool)
    for b in range(B):
        for h in range(H):
            for i in range(T):
                n = i + 1 if causal else T
                row, e = s[b, h, i, :n], eps[b, h, i, :n]
                a = int(np.argmax(row))
                M, eM = row[a], e[a]
                near = (M - row <= e + eM) & (row != M)
                bad = near.any()
                if calib == "minmax":
                    c = int(np.argmin(row))
                    m, em = row[c], e[c]
                    bad |= ((row - m <= e + em) & (row != m)).any()
                    span = M - m
                    if span <= 1e-12:
                        amb[b, h, i] = bad
                        continue
                    u = K * (row - m) / span
                    du = K / span * (e + em + u / K * (eM + em)) * 2
                    lo = 1
                else:
                    u = K * (row - M + tau) / tau
                    du = K / tau * (e + eM) * 2
                    lo = 0
                v2 = 2 * u
                nn = np.rint(v2)
                interior = (nn >= lo) & (nn <= 2 * K - 1)
                bad |= (interior & (np.abs(v2 - nn) <= 2 * du)).any()
                amb[b, h, i] = bad
    return amb


def device_scores(q, k, causal=1):
    """The kernels' canonical fp32 scores of (q, k) [B,H,T,d] (fp32 or
    bfloat16 inputs), through kia_debug_scores, as a host float32 array."""
    B, H, T, _ = q.shape
    out = torch.empty((B, H, T, T), dtype=torch.float32, device="cuda")
    kia.kia_debug_scores(q.cuda(), k.cuda(), out, causal)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def given_scores_check(oracle_mod, name, n_slices, bf16=False, variant=None):
    """Unrounded N(0,1) inputs at the workload's full size, every row of the
    sampled slices: the oracle takes the kernels' own fp32 scores (App. A:
    the operator acts on rows of fp32 scores), so every decision must agree
    bit for bit (codes, stored decisions, extrema, tie counts) and O, dQ,
    dK, dV meet the usual bar (bf16 inputs: 2e-2). The scores themselves are
    checked against the fp64 product q k^T within the fp32 MFMA bound."""
    import test_gpu_bf16 as B16
    w = dict(WORKLOADS[name])
    if variant:
        w.update(variant)
    B, H, T, d = w["B"], w["H"], w["T"], w["d"]
    q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], qk_scale=w["qk_scale"])
    args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"], 1)
    sl = sample_slices(B, H, n_slices, w["seed"])
    idx = [b * H + h for (b, h) in sl]
    flush(f"case given-scores {name} {variant} bf16={bf16} slices={len(sl)}")
    if bf16:
        (qb, kb, vb, db), (q, k, v, dO) = B16.bf16_inputs(q, k, v, dO)
        g = B16.run_gpu16(qb, kb, vb, db, *args, keep=idx)
        qs16, ks16 = (x.reshape(-1, T, d)[idx].unsqueeze(0) for x in (qb, kb))
        S = device_scores(qs16, ks16)
    else:
        g = run_gpu(q, k, v, dO, *args, keep=idx)
        S = device_scores(*(x.reshape(-1, T, d)[idx].unsqueeze(0) for x in (q, k)))
    qs, ks, vs, ds = restrict(q, k, v, dO, sl)
    if not bf16:
        s64, eps = fp32_scores_and_bound(qs, ks)
        valid = np.tril(np.ones((T, T), dtype=bool))
        assert np.all((np.abs(S - s64) <= eps)[..., valid]), "kernel scores off the bound"
    r = run_oracle_given(oracle_mod, qs, ks, vs, ds, S, *args)
    gs = {key: (val.reshape(-1, *val.shape[2:])[idx][None]
                if isinstance(val, np.ndarray) and not key.startswith("codes") else val)
          for key, val in g.items()}
    sl0 = [(0, i) for i in range(len(sl))]
    if bf16:
        return B16.compare16(gs, r, oracle_mod, w["calib"], sl0, exact=True,
                             tag=f"given-scores bf16 {name}")
    return compare(gs, r, oracle_mod, w["calib"], sl0, tag=f"given-scores {name}")


def run_oracle_given(oracle, q, k, v, dO, S, K, calib, tau, recon, ste, detach, causal):
    args = [x.double().numpy() for x in (q, k, v)]
    o, info, _, cd = oracle.attn_fwd(*args, K=K, calib=calib, tau=tau, recon=recon,
                                     causal=causal, want_codes=True, scores=S)
    dq, dk, dv, _, _ = oracle.attn_bwd(*args, dO.double().numpy(), K=K, calib=calib,
                                       tau=tau, recon=recon, ste=ste, detach=detach,
                                       causal=causal, scores=S)
    return dict(o=o, dq=dq, dk=dk, dv=dv, info=info, codes=cd)


def test_given_scores_bench_workload_every_slice(oracle_mod):
    """The bench workload exactly as bench.py runs it (N(0,1) inputs, B8 H12
    T1024 d64, FWM, Nearest, Prob-STE, K=4): all 96 slices, every row."""
    given_scores_check(oracle_mod, "gpt2_124m", n_slices=96)


def test_given_scores_long_context(oracle_mod):
    """The long-context workload (B1 H16 T8192 d128, q, k x 2), MinMax and
    FWM, two sampled slices, every row."""
    for calib in ("minmax", "fwm"):
        given_scores_check(oracle_mod, "long_8k", n_slices=2, variant=dict(calib=calib))


def test_given_scores_1b_scale_bf16(oracle_mod):
    """The 1B-scale workload with bf16 inputs (B4 H16 T2048 d128), two
    sampled slices, every row: decisions bit-exact, outputs within 2e-2."""
    given_scores_check(oracle_mod, "scale_1b", n_slices=2, bf16=True)


def test_unrounded_inputs_row_parity(oracle_mod):
    """The bench workload (N(0,1), GPT-2-124M shape) and the tiny workload:
    rows whose every decision is clear of the score error compare exactly
    (codes, argmax/argmin, tie counts) and within tolerance (O, dQ rows);
    the extrema of every row agree to the score error bound."""
    for name, n_slices in (("tiny", 1), ("gpt2_124m", 96)):
        w = WORKLOADS[name]
        B, H, T, d = w["B"], w["H"], w["T"], w["d"]
        q, k, v, dO = make_inputs(B, H, T, d, seed=w["seed"], qk_scale=w["qk_scale"])
        args = (w["K"], w["calib"], w["tau"], w["recon"], w["ste"], w["detach"], 1)
        flush(f"case unrounded {name}")
        g = run_gpu(q, k, v, dO, *args)
        sl = sample_slices(B, H, n_slices, w["seed"])
        qs, ks, vs, ds = restrict(q, k, v, dO, sl)
        r = run_oracle(oracle_mod, qs, ks, vs, ds, *args)
        s, eps = fp32_scores_and_bound(qs, ks)
        amb = ambiguity(s, eps, w["K"], w["calib"], w["tau"])
        RI = oracle_mod.RI
        for n, (b, h) in enumerate(sl):
            clean = ~amb[0, n]
            assert clean.mean() > 0.5, (name, clean.mean())
            info = r["info"][0, n]
            rows = np.arange(T)
            eM = eps[0, n][rows, info[:, RI["amax"]].astype(int)]
            assert np.all(np.abs(g["M"][b, h] - info[:, RI["M"]]) <= eM)
            assert np.array_equal(g["amax"][b, h][clean], info[clean, RI["amax"]].astype(np.int32))
            assert np.array_equal(g["nmax"][b, h][clean], info[clean, RI["nmax"]].astype(np.int32))
            assert np.array_equal(g["codes"][b, h][clean], r["codes"][0, n][clean])
            assert np.array_equal(g["codes_stored"][b, h][clean], r["codes"][0, n][clean])
            for key, tol in (("o", O_TOL), ("dq", G_TOL)):
                den = np.max(np.abs(r[key][0, n]))
                err = np.max(np.abs(g[key][b, h][clean] - r[key][0, n][clean])) / den
                assert err <= tol, (name, key, err)
            flush(f"  slice {(b, h)}: {int((~clean).sum())} of {T} rows near a boundary")


# ---------------------------------------------------------------------------
# Invariants at full size (no oracle needed)
# ---------------------------------------------------------------------------

def _gpt2_inputs(seed=1):
    w = WORKLOADS["gpt2_124m"]
    q, k, v, dO = make_inputs(w["B"], w["H"], w["T"], w["d"], seed=seed)
    return [x.cuda() for x in (q, k, v, dO)]


@pytest.mark.parametrize("calib", ("minmax", "fwm", "resolved"))
def test_rows_sum_to_one_on_device(calib):
    """P = w / sum w: with V = 1 every output entry is 1 (App. A
    normalization). W and sum_j w_j v_j are two fp32 sums of up to T terms in
    different orders, so the bound is T * 2^-23 (the paper's 1e-6 is for its
    short degenerate rows, checked by the oracle pins)."""
    q, k, _, _ = _gpt2_inputs()
    T = q.shape[2]
    ones = torch.ones_like(q)
    for recon in ("lerp", "nearest"):
        o, _ = kia.forward(q, k, ones, 4, calib, 8.0, recon, "weight", False, True)
        assert torch.max(torch.abs(o - 1)).item() <= T * 2.0 ** -23


def test_forward_is_independent_of_surrogate_and_detach():
    """Strict hard forward: Weight- and Prob-STE and full/detach give the
    same forward bit for bit (App. forward audits (iii); detach changes the
    backward only)."""
    q, k, v, _ = _gpt2_inputs()
    for calib in ("minmax", "fwm"):
        for recon in ("lerp", "nearest"):
            ref, st0 = kia.forward(q, k, v, 4, calib, 8.0, recon, "weight", False, True)
            for ste, det in (("prob", False), ("weight", True), ("prob", True)):
                o, st = kia.forward(q, k, v, 4, calib, 8.0, recon, ste, det, True)
                assert torch.equal(o, ref)
            o2, _ = kia.forward(q, k, v, 4, calib, 8.0, recon, "weight", False, True)
            assert torch.equal(o2, ref)  # deterministic


def test_backward_identities_on_device():
    """LERP makes the surrogate placement irrelevant; Prob-STE's dQ/dK equal
    the LERP operator's (the Jacobian of normalize(w^L)); dV differs (it uses
    the hard P) (Sec. 3, App. B)."""
    q, k, v, dO = _gpt2_inputs()
    for calib in ("minmax", "fwm"):
        res = {}
        for recon, ste in (("lerp", "weight"), ("lerp", "prob"), ("nearest", "prob")):
            o, st = kia.forward(q, k, v, 4, calib, 8.0, recon, ste, False, True)
            res[(recon, ste)] = kia.backward(q, k, v, o, dO, st, 4, calib, 8.0, recon, ste, False, True)
        a, b, c = res[("lerp", "weight")], res[("lerp", "prob")], res[("nearest", "prob")]
        for x, y in zip(a, b):
            assert torch.max(torch.abs(x - y)).item() <= 1e-6 * torch.max(torch.abs(x)).item()
        for x, y in zip(a[:2], c[:2]):
            assert torch.max(torch.abs(x - y)).item() <= 1e-5 * torch.max(torch.abs(x)).item()
        assert torch.max(torch.abs(a[2] - c[2])).item() > 1e-3 * torch.max(torch.abs(a[2])).item()


@pytest.mark.parametrize("calib", ("minmax", "fwm", "resolved"))
def test_zero_sum_of_key_gradients(calib):
    """Full gradient: sum_j dS_ij = 0, so sum_j dK_j = scale sum_i q_i
    sum_j dS_ij = 0 per (b,h); detaching the extrema breaks it (Sec. 3
    zero-sum identity; App. B detach)."""
    q, k, v, dO = _gpt2_inputs()
    for recon, ste in (("lerp", "weight"), ("nearest", "weight"), ("nearest", "prob")):
        rel = {}
        for det in (False, True):
            o, st = kia.forward(q, k, v, 4, calib, 8.0, recon, ste, det, True)
            _, dk, _ = kia.backward(q, k, v, o, dO, st, 4, calib, 8.0, recon, ste, det, True)
            colsum = dk.double().sum(dim=2)
            rel[det] = (colsum.abs().max() / dk.double().abs().sum(dim=2).max()).item()
        assert rel[False] < 1e-5, rel
        assert rel[True] > 1e-3, rel


def test_full_size_long_context_exact_scores(oracle_mod):
    """Long-context workload (B1 H16 T8192 d128, q,k x2 so row spans exceed
    tau; LERP, Weight-STE, K=4) for both calibrations, one sampled slice."""
    for calib in ("minmax", "fwm"):
        full_size_check(oracle_mod, "long_8k", variant=dict(calib=calib), n_slices=1)


def test_full_size_1b_shape_fp32_exact_scores(oracle_mod):
    """1B-scale shape (B4 H16 T2048 d128; FWM, Nearest, Prob-STE, K=16) on the
    fp32 path, two sampled slices, codes included."""
    full_size_check(oracle_mod, "scale_1b", n_slices=2)


def test_resolved_long_context_keeps_the_tail(oracle_mod):
    """The resolved grid at the long-context shape (B1 H16 T8192 d128, q,k x2:
    row spans ~30 nats, far beyond tau = 8, so most keys sit below the
    window on negative intervals), one sampled slice, codes included."""
    full_size_check(oracle_mod, "long_8k", variant=dict(calib="resolved", recon="nearest"),
                    n_slices=1)
