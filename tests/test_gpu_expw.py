"""GPU parity of the exponential weight functions (exact softmax of App. A;
BF16-exp and FP8-rounded exp of App. D) through the C-ABI against the fp64
oracle, plus the textbook softmax attention as an independent reference.

Bar: the quantized weight of every (query, key) pair (its bf16 bit pattern
or E4M3 byte, from kia_debug_codes) bit-exact; argmax and tie counts
bit-exact; O within 1e-4; dQ/dK/dV within 1e-3 (max |x - ref| / max |ref|
per (b,h) slice) on exact-score inputs (dyadic q, k or given scores), the
same bar as the K-interval variants.

BF16-exp also rounds the gradient: dz = bf16(bf16(dL/dw) w). dL/dw is an
fp32 value on both sides but not the same one (the kernel's fp32 dot
products and fma against the oracle's fp64 value rounded once), so where it
lies within a few fp32 ulp of a bf16 midpoint the two round it to
neighbouring bf16 values, one bf16 ulp of dL/dw apart (2^-8 to 2^-7 of
it). The products with w differ by as much relative, and their own
rounding to bf16 can then land them up to two bf16 ulps of dz apart
(2^-6 of dz at the bottom of a binade). The elements are pinned through the
score-gradient export: equal to the oracle's bit for bit except for a rare
few (< 0.1%), each within 2^-6 of itself plus the 1e-5 (of the slice's
largest dz) that bounds the unrounded modes (where g_j nearly equals <g>,
dL/dw is known only to an absolute fp32 error, and its bf16 rounding
inherits it). dQ/dK are then held to the fp32 bar of 1e-3 against the
oracle's corrected by exactly those flipped elements: each flip F_ij enters
dS_ij, and through the gradient mode the maximum's channel (-sum_j F_ij on
the argmax keys, split over ties) or the P1 row mean.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import given_score_inputs, make_inputs  # noqa: E402
import test_gpu_parity as P  # noqa: E402

MODES = ("softmax", "bf16_exp", "fp8_exp")
O_TOL, G_TOL = 1e-4, 1e-3


def run(oracle_mod, q, k, v, dO, recon, grad, causal, codes=True, slices=None):
    # K, calib, tau and ste are not used by the exponential weight functions
    b16 = recon == "bf16_exp"
    g = P.run_gpu(q, k, v, dO, 4, "fwm", 8.0, recon, "weight", grad, causal, codes=codes,
                  want_gself=b16)
    r = P.run_oracle(oracle_mod, q, k, v, dO, 4, "fwm", 8.0, recon, "weight", grad, causal,
                     slices=slices, codes=codes)
    if b16:
        r = flip_corrected(oracle_mod, q, k, v, dO, grad, causal, g["g_self"], r)
    return g, r


def flip_corrected(oracle_mod, q, k, v, dO, grad, causal, g_self, r):
    """The oracle's dQ, dK with the kernel's BF16-exp rounding flips of dz
    (module docstring) carried through: F = dz_kernel - dz_oracle, pinned
    elementwise here (rare: < 1% of a slice even where the weights are bf16
    subnormals; each one bf16 ulp of dz or within the
    fp32 cancellation error), is added to dS together with what the
    gradient mode derives from it, then multiplied by K resp. Q in fp64."""
    args = [x.double().numpy() for x in (q, k, v)]
    _, _, _, info, dz = oracle_mod.attn_bwd(*args, dO.double().numpy(), K=4, calib="fwm",
                                            tau=8.0, recon="bf16_exp", ste="weight",
                                            detach=True, causal=causal, want_dS=True)
    B, H, T, d = q.shape
    valid = np.tril(np.ones((T, T), dtype=bool)) if causal else np.ones((T, T), dtype=bool)
    F = np.where(valid, g_self - dz, 0.0)
    # g_ij = dO_i . v_j: gamma = (g - <g>) / W cancels to an absolute fp32
    # error of the order of 2^-24 times the dot products' own scale
    # sum_k |dO_ik v_jk| (which exceeds |g_ij| where the dot product itself
    # cancels; a single key: g - <g> = 0 exactly in the oracle, a residue of
    # two fp32 evaluations of dO . v in the kernel)
    gmax = np.max((np.abs(dO.double().numpy()) @ np.swapaxes(np.abs(v.double().numpy()), -1, -2)) *
                  valid, axis=-1, keepdims=True)
    for b in range(B):
        for h in range(H):
            big = np.max(np.abs(dz[b, h]))
            # the fp32 error alone (a one-hot row's argmax key: g - <g> is a
            # rounding residue, one per row) is no rounding flip
            floor = 1e-5 * big + 2.0 ** -20 * gmax[b, h]
            flips = np.count_nonzero(np.abs(F[b, h]) > floor)
            assert flips <= max(2, 1e-2 * valid.sum()), (b, h, flips)
            bound = 2.0 ** -6 * np.abs(dz[b, h]) + floor
            assert np.all(np.abs(F[b, h]) <= bound), (b, h, np.max(np.abs(F[b, h]) - bound))
    mode = P.oracle_grad(grad)
    if mode in ("full", "max_only"):
        # the maximum's channel -sum_j dz_j moves by -sum_j F_ij, split over
        # the keys equal to M (the row maximum's ties)
        S = P.oracle_scores(q, k)
        M = info[..., oracle_mod.RI["M"]]
        top = (S == M[..., None]) & valid
        F = F - top * (F.sum(axis=-1, keepdims=True) / top.sum(axis=-1, keepdims=True))
    elif mode == "p1":
        n = valid.sum(axis=-1, keepdims=True)
        F = np.where(valid, F - F.sum(axis=-1, keepdims=True) / n, 0.0)
    sc = 1.0 / math.sqrt(d)
    qd, kd = (x.double().numpy() for x in (q, k))
    out = dict(r)
    out["dq"] = r["dq"] + sc * F @ kd
    out["dk"] = r["dk"] + sc * np.swapaxes(F, -1, -2) @ qd
    return out


def check(g, r, oracle_mod, sl, tag, check_codes=True, g_tol=G_TOL, floors=None):
    RI = oracle_mod.RI
    for (b, h) in sl:
        info = r["info"][b, h]
        assert np.array_equal(g["M"][b, h].astype(np.float64), info[:, RI["M"]]), tag
        assert np.array_equal(g["amax"][b, h], info[:, RI["amax"]].astype(np.int32)), tag
        assert np.array_equal(g["nmax"][b, h], info[:, RI["nmax"]].astype(np.int32)), tag
        w_err = np.max(np.abs(g["W"][b, h] - info[:, RI["W"]]) / info[:, RI["W"]])
        assert w_err < O_TOL, (tag, w_err)
        if check_codes:
            for key in ("codes", "codes_stored"):
                bad = np.argwhere(g[key][b, h] != r["codes"][b, h])
                assert bad.size == 0, (tag, key, len(bad), bad[:5], g[key][b, h][tuple(bad[0])],
                                       r["codes"][b, h][tuple(bad[0])])
    floors = floors or {}
    errs = {key: P.rel_err(g[key], r[key], sl, floors.get(key)) for key in ("o", "dq", "dk", "dv")}
    P.flush(f"  {tag}: " + " ".join(f"{k_}={v_:.2e}" for k_, v_ in errs.items()))
    assert errs["o"] <= O_TOL, (tag, errs)
    assert max(errs["dq"], errs["dk"], errs["dv"]) <= g_tol, (tag, errs)


@pytest.mark.parametrize("grad", ("full", "detach", "p1"))
@pytest.mark.parametrize("mode", MODES)
def test_exp_modes_exact_score_parity(oracle_mod, mode, grad):
    """Every head size, ragged tails, T = 1, causal and not (the K-interval
    parity shapes), dyadic q and k."""
    for i, (B, H, T, d, _K, causal, sc) in enumerate(P.SHAPES):
        tag = f"{mode} {grad} B{B} H{H} T{T} d{d} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=500 + i, qk_scale=sc * 2, dyadic=True)
        g, r = run(oracle_mod, q, k, v, dO, mode, grad, causal)
        check(g, r, oracle_mod, [(b, h) for b in range(B) for h in range(H)], tag,
              g_tol=G_TOL)


# (seed, B, H, T, d, qk_scale, weight function, gradient mode), causal:
# two-key rows whose dQ cancels to a rounding-size fraction (slices that
# random sweeps of exact-score cases of these modes met)
ONE_HOT_EXP = [(12385, 1, 2, 2, 16, 5.0, "fp8_exp", "detach"),
               (10765, 2, 1, 2, 64, 3.0, "fp8_exp", "detach"),
               (11010, 2, 3, 2, 16, 5.0, "fp8_exp", "p1"),
               (11131, 1, 1, 2, 32, 5.0, "softmax", "p1"),
               (11377, 2, 1, 2, 128, 5.0, "fp8_exp", "p1")]


@pytest.mark.parametrize("case", ONE_HOT_EXP, ids=lambda c: f"seed{c[0]}")
def test_exp_modes_near_one_hot_slices_at_the_fp32_floor(oracle_mod, case):
    """As test_gpu_parity.test_near_one_hot_slices_at_the_fp32_floor for the
    exponential weight functions: the 1e-3 bar of a dQ or dK cancelled
    below the fp32 rounding bound of its inputs taken against that floor;
    everything else at the usual bars."""
    seed, B, H, T, d, sc, mode, grad = case
    P.flush(f"case exp one-hot seed{seed}")
    q, k, v, dO = make_inputs(B, H, T, d, seed=seed, qk_scale=sc, dyadic=True)
    g, r = run(oracle_mod, q, k, v, dO, mode, grad, 1)
    sl = [(b, h) for b in range(B) for h in range(H)]
    floors = P.cancellation_floors(q, k, v, dO, sl)
    assert any(np.abs(r["dq"][b, h]).max() < floors["dq"][(b, h)] for (b, h) in sl)
    check(g, r, oracle_mod, sl, f"exp one-hot seed{seed}", floors=floors)


def given_rows(values, T=64):
    """Rows of T fp32 scores for given-score inputs: key 0 holds 0 (the row
    maximum, so z = s exactly) and keys 1..T-1 the test values in order;
    returns [n_slices, T, T] score matrices (non-causal use)."""
    vals = np.asarray(values, dtype=np.float32)
    per = T - 1
    nrows = -(-len(vals) // per)
    rows = np.zeros((nrows, T), dtype=np.float32)
    flat = rows[:, 1:].reshape(-1)
    flat[:len(vals)] = vals
    rows[:, 1:] = flat.reshape(nrows, per)
    nsl = -(-nrows // T)
    S = np.zeros((nsl * T, T), dtype=np.float32)
    S[:nrows] = rows
    return S.reshape(nsl, T, T)


def given_inputs(S, seed):
    d = S.shape[-1]
    qs, ks = zip(*(given_score_inputs(S[i], d) for i in range(S.shape[0])))
    q, k = torch.cat(qs, dim=1), torch.cat(ks, dim=1)
    g = torch.Generator().manual_seed(seed)
    v = torch.randn(q.shape, generator=g)
    dO = torch.randn(q.shape, generator=g)
    return q, k, v, dO


def test_bf16_exp_codes_exhaustive(oracle_mod):
    """Every bf16 shift z in [-128, 0] (17153 values, including those whose
    exponential is a subnormal bf16 or 0) through the forward: each weight's
    bf16 pattern equals the oracle's, then O and the gradients."""
    bits = np.arange(0x8000, 0xC301, dtype=np.uint32)
    z = (bits << 16).view(np.float32)
    S = given_rows(z)
    q, k, v, dO = given_inputs(S, 11)
    P.flush(f"case bf16_exp exhaustive: {len(z)} shifts in {S.shape[0]} slices")
    g, r = run(oracle_mod, q, k, v, dO, "bf16_exp", "full", 0)
    check(g, r, oracle_mod, [(0, h) for h in range(S.shape[0])], "bf16_exp exhaustive",
          g_tol=G_TOL)


def e4m3_grid():
    """float8_e4m3fn values in [0, 1]: subnormal m 2^-9, normal (1 + m/8) 2^(e-7)."""
    out = []
    for c in range(0x39):
        e, m = c >> 3, c & 7
        out.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    return np.array(out)


def test_fp8_exp_codes_near_rounding_midpoints(oracle_mod):
    """Shifts z whose fp32 exponential lies on or within a few ulp of a
    midpoint between neighbouring E4M3 values (the 2^-10 underflow point
    included), and uniform shifts in [-12, 0]: each weight's E4M3 byte equals
    the oracle's."""
    grid = e4m3_grid()
    mids = (grid[:-1] + grid[1:]) / 2
    z0 = np.log(mids).astype(np.float32)
    vals = []
    for z in z0:
        x = z
        for _ in range(12):
            x = np.nextafter(x, np.float32(-np.inf))
        for _ in range(25):
            vals.append(x)
            x = np.nextafter(x, np.float32(np.inf))
    rng = np.random.default_rng(12)
    vals = np.concatenate([np.array(vals, dtype=np.float32),
                           (-12 * rng.random(4000)).astype(np.float32)])
    vals = np.minimum(vals, np.float32(0))
    S = given_rows(vals)
    q, k, v, dO = given_inputs(S, 13)
    P.flush(f"case fp8_exp midpoints: {len(vals)} shifts in {S.shape[0]} slices")
    g, r = run(oracle_mod, q, k, v, dO, "fp8_exp", "full", 0)
    check(g, r, oracle_mod, [(0, h) for h in range(S.shape[0])], "fp8_exp midpoints")


def textbook_attention(q, k, v, dO, causal):
    """Softmax attention by its definition in fp64 on the CPU (torch
    autograd): S = q k^T / sqrt(d), P = softmax over the valid keys,
    O = P V; gradients of sum(dO * O)."""
    q, k, v = (x.double().clone().requires_grad_(True) for x in (q, k, v))
    d, T = q.shape[-1], q.shape[-2]
    S = (q @ k.transpose(-1, -2).contiguous()) * float(np.float32(1.0 / math.sqrt(d)))
    if causal:
        S = S.masked_fill(torch.ones(T, T, dtype=torch.bool).triu(1), float("-inf"))
    O = torch.softmax(S, dim=-1) @ v
    (O * dO.double()).sum().backward()
    return O.detach().numpy(), q.grad.numpy(), k.grad.numpy(), v.grad.numpy()


@pytest.mark.parametrize("grad", ("full", "detach"))
def test_softmax_mode_is_textbook_softmax_attention(grad):
    """The softmax weight function is ordinary attention: shift invariance
    makes the maximum's channel vanish, so full and detach both equal the
    textbook gradients."""
    for (B, H, T, d, causal) in ((1, 2, 100, 64, 1), (1, 1, 77, 16, 0), (2, 1, 130, 128, 1)):
        P.flush(f"case textbook softmax {grad} B{B} H{H} T{T} d{d} causal{causal}")
        q, k, v, dO = make_inputs(B, H, T, d, seed=600 + T, qk_scale=2.0, dyadic=True)
        g = P.run_gpu(q, k, v, dO, 4, "fwm", 8.0, "softmax", "weight", grad, causal,
                      codes=False)
        ref = dict(zip(("o", "dq", "dk", "dv"), textbook_attention(q, k, v, dO, causal)))
        sl = [(b, h) for b in range(B) for h in range(H)]
        assert P.rel_err(g["o"], ref["o"], sl) <= O_TOL
        for key in ("dq", "dk", "dv"):
            assert P.rel_err(g[key], ref[key], sl) <= G_TOL, key


def score_grad_gpu(q, k, v, dO, mode, causal):
    """g_self (the detached dS = dz as the backward computed it) and the
    maximum channel's row sum cM, after a full-gradient backward."""
    B, H, T, d = q.shape
    qg, kg, vg, dg = (x.cuda() for x in (q, k, v, dO))
    o, st = kia.forward(qg, kg, vg, 4, "fwm", 8.0, mode, "weight", "full", causal)
    kia.backward(qg, kg, vg, o, dg, st, 4, "fwm", 8.0, mode, "weight", "full", causal)
    gs = torch.zeros((B, H, T, T), dtype=torch.float32, device="cuda")
    cM = torch.zeros((B, H, T), dtype=torch.float32, device="cuda")
    cm = torch.zeros_like(cM)
    kia.kia_debug_score_grad(st, gs, cM, cm, B, H, T, d, "fwm", mode, "weight", causal)
    torch.cuda.synchronize()
    return gs.cpu().double().numpy(), cM.cpu().double().numpy(), cm.cpu().double().numpy()


@pytest.mark.parametrize("mode", MODES)
def test_exp_modes_score_gradient_elements(oracle_mod, mode):
    """Element level: dz of every valid pair against the oracle's detached
    dS, and the maximum's channel cM = -sum_j dz_j. Softmax and FP8-exp
    (no rounding in the backward): within 1e-5 of the slice's largest |dz|.
    BF16-exp: bit-exact except a rare few pairs (< 0.1%) within 2^-6."""
    bits = np.arange(0x8000, 0xC301, 3, dtype=np.uint32)
    S = given_rows((bits << 16).view(np.float32))
    cases = [given_inputs(S, 21) + (0,),
             make_inputs(1, 2, 300, 64, seed=22, qk_scale=2.0, dyadic=True) + (1,)]
    for q, k, v, dO, causal in cases:
        B, H, T, d = q.shape
        P.flush(f"case score-gradient elements {mode} B{B} H{H} T{T} causal{causal}")
        gs, cM, cm = score_grad_gpu(q, k, v, dO, mode, causal)
        args = [x.double().numpy() for x in (q, k, v)]
        _, _, _, info, dz = oracle_mod.attn_bwd(*args, dO.double().numpy(), K=4, calib="fwm",
                                                tau=8.0, recon=mode, ste="weight",
                                                detach=True, causal=causal, want_dS=True)
        _, _, _, info_full, _ = oracle_mod.attn_bwd(*args, dO.double().numpy(), K=4,
                                                    calib="fwm", tau=8.0, recon=mode,
                                                    ste="weight", detach=False, causal=causal)
        valid = np.tril(np.ones((T, T), dtype=bool)) if causal else np.ones((T, T), dtype=bool)
        assert np.all(cm == 0)
        for b in range(B):
            for h in range(H):
                x, ref = gs[b, h][valid], dz[b, h][valid]
                scale = np.max(np.abs(ref))
                cref = info_full[b, h][:, oracle_mod.RI["cM"]]
                # cM = -sum_j dz_j: a flipped dz of BF16-exp moves its row's cM by
                # the same amount
                flips = np.sum(np.abs(gs[b, h] - dz[b, h]) * valid, axis=1)
                tol = 1e-5 * max(np.max(np.abs(cref)), scale) + 1.01 * flips
                assert np.all(np.abs(cM[b, h] - cref) <= tol)
                if mode == "bf16_exp":
                    diff = x != ref
                    P.flush(f"  slice {(b, h)}: {int(diff.sum())} of {x.size} dz differ")
                    assert diff.mean() < 1e-3
                    # at most two bf16 ulps of dz (one of dL/dw, then the second
                    # rounding), or where dL/dw nearly cancels (g close to <g>)
                    # its fp32 absolute error, as for the unrounded modes
                    assert np.all(np.abs(x - ref) <= 2.0 ** -6 * np.abs(ref) + 1e-5 * scale)
                else:
                    assert np.max(np.abs(x - ref)) <= 1e-5 * scale


@pytest.mark.parametrize("mode", MODES)
def test_exp_modes_full_size_gpt2_shape(oracle_mod, mode):
    """The GPT-2-124M attention shape (B8 H12 T1024 d64, dyadic q, k), one
    sampled slice against the oracle, codes included."""
    B, H, T, d = 8, 12, 1024, 64
    q, k, v, dO = make_inputs(B, H, T, d, seed=1, dyadic=True)
    P.flush(f"case full-size gpt2 {mode}")
    b16 = mode == "bf16_exp"
    g = P.run_gpu(q, k, v, dO, 4, "fwm", 8.0, mode, "weight", "full", 1, want_gself=b16)
    sl = P.sample_slices(B, H, 1, 1)
    qs, ks, vs, ds = P.restrict(q, k, v, dO, sl)
    r = P.run_oracle(oracle_mod, qs, ks, vs, ds, 4, "fwm", 8.0, mode, "weight", "full", 1)
    idx = [b * H + h for (b, h) in sl]
    gs = {key: val.reshape(-1, *val.shape[2:])[idx][None] for key, val in g.items()}
    if b16:
        r = flip_corrected(oracle_mod, qs, ks, vs, ds, "full", 1, gs["g_self"], r)
    check(gs, r, oracle_mod, [(0, i) for i in range(len(sl))], f"full-size {mode}",
          g_tol=G_TOL)


@pytest.mark.parametrize("mode", MODES)
def test_exp_modes_rows_sum_to_one(mode):
    """P = w / sum w: with V = 1 every output is 1 within the two fp32 sums'
    rounding (T * 2^-23), at the GPT-2-124M shape with N(0,1) inputs."""
    q, k, _, _ = (x.cuda() for x in make_inputs(8, 12, 1024, 64, seed=1))
    o, _ = kia.forward(q, k, torch.ones_like(q), 4, "fwm", 8.0, mode, "weight", False, True)
    assert torch.max(torch.abs(o - 1)).item() <= 1024 * 2.0 ** -23
