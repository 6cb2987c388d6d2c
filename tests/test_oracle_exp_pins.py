"""Pins of the oracle's exponential weight functions (App. A, Softmax; App. D,
reduced-precision exponential baselines) against independent references.

The references are library routines that the definitions name: PyTorch's
fp32 -> bfloat16 and fp32 -> float8_e4m3fn casts and its bfloat16 exp, and
PyTorch CPU autograd through those casts (the paper defines the BF16-exp
backward as native autograd through the casts, and the FP8 backward as an
identity surrogate around the rounding with the fp32 exponential's
derivative). Counting pins come from the paper's own statements: 56 nonzero
E4M3 weights in (0, 1] (49 normal, 7 subnormal) and underflow to 0 at
w <= 2^-10. CPU only.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

MODES = ("softmax", "bf16_exp", "fp8_exp")


def f32(x):
    return np.asarray(x, dtype=np.float32)


def rn32_exp(z):
    """fp32 rounding of e^z for fp32 z (numpy's fp64 exp, then the cast)."""
    return np.exp(f32(z).astype(np.float64)).astype(np.float32)


def torch_e4m3(y):
    return torch.from_numpy(f32(y)).to(torch.float8_e4m3fn).float().numpy().astype(np.float64)


def torch_bf16(y):
    return torch.from_numpy(f32(y)).to(torch.bfloat16).float().numpy().astype(np.float64)


def low16_near_tie(y, slack=2):
    """fp32 values whose bfloat16 rounding an fp32 exp error of `slack` ulps
    could flip (low 16 bits within `slack` of the tie 0x8000)."""
    b = f32(y).view(np.uint32).astype(np.int64)
    return np.abs((b & 0xFFFF) - 0x8000) <= slack


# --------------------------------------------------------------------------
# Elementwise weight functions
# --------------------------------------------------------------------------

def test_softmax_weight_is_exp(oracle_mod):
    z = -np.random.default_rng(1).exponential(3.0, size=4000).astype(np.float32)
    z[:3] = [0.0, -1e-30, -80.0]
    w, wE, code = oracle_mod.expw(z, "softmax")
    ref = np.exp(z.astype(np.float64))
    assert np.all(np.abs(w - ref) <= 1e-15 * ref)
    assert np.array_equal(w, wE) and not code.any()


def test_fp8_weights_take_56_nonzero_values(oracle_mod):
    """E4M3 has 56 nonzero values in (0, 1]: 49 normal (exponents -6..0) and
    7 subnormal multiples of 2^-9 (App. D); a dense sweep of z reaches all."""
    z = np.linspace(-8.0, 0.0, 400001).astype(np.float32)
    w, wE, code = oracle_mod.expw(z, "fp8_exp")
    vals = np.unique(w[w > 0])
    assert vals.size == 56
    assert w.max() == 1.0
    normal, sub = vals[vals >= 2.0 ** -6], vals[vals < 2.0 ** -6]
    assert normal.size == 49 and sub.size == 7
    assert np.array_equal(sub, np.arange(1, 8) * 2.0 ** -9)
    assert np.all(np.log2(normal) >= -6) and np.all(np.log2(normal) <= 0)
    # the code is the E4M3 byte of the value
    assert np.array_equal(torch.tensor(code.astype(np.uint8)).view(torch.float8_e4m3fn)
                          .float().numpy().astype(np.float64), w)
    # monotone in z
    assert np.all(np.diff(w) >= 0)


def test_fp8_underflow_boundary(oracle_mod):
    """Round-to-nearest sends w <= 2^-10 to 0 (the tie at 2^-10 goes to the
    even code 0) and anything above it to 2^-9: z below about -6.93 (App. D)."""
    z0 = np.float32(math.log(2.0 ** -10))
    zs = z0 + np.arange(-200, 201, dtype=np.float32) * np.spacing(z0)
    zs = zs.astype(np.float32)
    w, _, _ = oracle_mod.expw(zs, "fp8_exp")
    y = rn32_exp(zs).astype(np.float64)
    assert np.array_equal(w[y <= 2.0 ** -10], np.zeros(int((y <= 2.0 ** -10).sum())))
    assert np.all(w[y > 2.0 ** -10] == 2.0 ** -9)
    assert abs(float(z0) + 6.93) < 0.01


def test_fp8_rounding_matches_torch_cast(oracle_mod):
    """w = e4m3(fp32(e^z)), bit for bit against PyTorch's float8_e4m3fn cast,
    on random z and on z windows around every E4M3 midpoint in (0, 1]."""
    rng = np.random.default_rng(2)
    zs = [-rng.exponential(2.0, size=200000).astype(np.float32)]
    vals = np.unique(np.concatenate([np.arange(0, 8) * 2.0 ** -9] +
                                    [(1 + np.arange(8) / 8) * 2.0 ** e for e in range(-6, 0)] +
                                    [[1.0]]))
    mids = (vals[1:] + vals[:-1]) / 2
    for mk in mids:
        c = np.float32(math.log(mk))
        zs.append((c + np.arange(-300, 301, dtype=np.float32) * np.spacing(c)).astype(np.float32))
    z = np.minimum(np.concatenate(zs), np.float32(0.0))
    w, wE, code = oracle_mod.expw(z, "fp8_exp")
    y = rn32_exp(z)
    assert np.array_equal(wE, y.astype(np.float64))
    assert np.array_equal(w, torch_e4m3(y))


def bf16_grid(lo=-95.0):
    """Every bfloat16 value in [lo, 0]."""
    b = np.arange(0x8000, 0x10000, dtype=np.uint32)
    v = (b << 16).view(np.float32)
    return v[(v >= lo) & np.isfinite(v)]


def test_bf16_exp_exhaustive_against_torch(oracle_mod):
    """w = bf16(e^{bf16(z)}) on every bfloat16 input in [-95, 0] against
    PyTorch's bfloat16 exp (fp32 evaluation, then the cast). The two may
    differ only where the fp32 exponential lands within 2 ulps of a
    bfloat16 tie (PyTorch's fp32 exp is not correctly rounded)."""
    zb = bf16_grid()
    w, _, code = oracle_mod.expw(zb, "bf16_exp")
    ref = torch.exp(torch.from_numpy(zb).to(torch.bfloat16)).float().numpy().astype(np.float64)
    y = rn32_exp(zb)
    diff = w != ref
    assert np.all(low16_near_tie(y)[diff])
    assert diff.sum() <= 8
    # within half a bfloat16 ulp of the exact value (rounding to nearest)
    e = np.exp(zb.astype(np.float64))
    pos = w > 0
    ulp = np.spacing(w[pos].astype(np.float32)).astype(np.float64) * 65536
    assert np.all(np.abs(w[pos] - e[pos]) <= 0.5 * ulp * (1 + 1e-6))
    assert np.array_equal((code << 16).astype(np.uint32).view(np.float32).astype(np.float64), w)


def test_bf16_exp_rounds_the_input_first(oracle_mod):
    """The input z is cast to bfloat16 before the exponential (App. D): w(z)
    equals w at PyTorch's bfloat16 cast of z, and differs from rounding only
    the output where the two orders disagree."""
    rng = np.random.default_rng(3)
    z = -rng.exponential(3.0, size=100000).astype(np.float32)
    w, _, _ = oracle_mod.expw(z, "bf16_exp")
    zb = torch_bf16(z).astype(np.float32)
    wb, _, _ = oracle_mod.expw(zb, "bf16_exp")
    assert np.array_equal(w, wb)
    out_only = torch_bf16(rn32_exp(z))
    assert (w != out_only).mean() > 0.1


# --------------------------------------------------------------------------
# Rows against PyTorch autograd
# --------------------------------------------------------------------------

def torch_row(s, g, mode):
    """The three operators in the paper's fp32 form, through autograd."""
    st = torch.tensor(f32(s), requires_grad=True)
    gt = torch.tensor(f32(g))
    M = st.max()
    z = st - M
    if mode == "softmax":
        w = torch.exp(z)
    elif mode == "bf16_exp":
        w = torch.exp(z.to(torch.bfloat16)).float()
    else:
        # w^fp8 is a constant: the rounding's only gradient is the identity
        # surrogate on w^exp (the native cast backward is a separate
        # diagnostic of the paper, not this operator)
        we = torch.exp(z)
        w = we.detach().to(torch.float8_e4m3fn).float() + (we - we.detach())
    P = w / w.sum()
    (P * gt).sum().backward()
    return P.detach().numpy().astype(np.float64), st.grad.numpy().astype(np.float64)


def rand_scores(rng, n, sigma):
    s = rng.normal(0.0, sigma, size=n).astype(np.float32)
    while np.sum(s == s.max()) > 1:
        s = rng.normal(0.0, sigma, size=n).astype(np.float32)
    return s.astype(np.float64)


@pytest.mark.parametrize("mode", MODES)
def test_rows_match_torch_autograd(oracle_mod, mode):
    rng = np.random.default_rng(4)
    for n in (1, 2, 5, 64, 300):
        for sigma in (0.5, 3.0, 10.0):
            s = rand_scores(rng, n, sigma)
            g = rng.normal(size=n)
            g32 = f32(g).astype(np.float64)
            out = oracle_mod.row(s, g32, recon=mode, calib="minmax", K=4)
            Pt, dSt = torch_row(s, g32, mode)
            assert np.abs(out["P"] - Pt).max() <= 2e-6 * max(1.0, Pt.max())
            scale = np.abs(dSt).sum() + 1e-30
            if mode == "bf16_exp":
                # one bfloat16 rounding of dL/dw and one of the product:
                # fp32 vs fp64 inputs to them may flip either by one ulp
                j = np.argmax(s)
                others = np.arange(n) != j
                err = np.abs(out["dS"] - dSt)
                assert np.all(err[others] <= 2.0 ** -7 * np.abs(dSt[others]) + 1e-7 * scale)
                assert err[j] <= 2.0 ** -7 * scale
            else:
                assert np.abs(out["dS"] - dSt).max() <= 1e-5 * scale


@pytest.mark.parametrize("mode", MODES)
def test_rows_are_zero_sum_with_max_on_path(oracle_mod, mode):
    """The row maximum stays on the gradient path, so each row of dS sums
    to zero (App. D). Detached, softmax still sums to zero (its max channel
    vanishes in exact arithmetic), BF16-exp up to its bfloat16 roundings, and
    FP8-exp not at all (the slope weights w^exp differ from the rounded
    weights that normalize)."""
    rng = np.random.default_rng(5)
    for n in (2, 17, 200):
        s = rand_scores(rng, n, 4.0)
        g = rng.normal(size=n)
        full = oracle_mod.row(s, g, recon=mode, detach="full")
        det = oracle_mod.row(s, g, recon=mode, detach="detach")
        tot = np.abs(full["dS"]).sum()
        assert abs(full["dS"].sum()) <= 1e-14 * tot
        # the channel is -sum of the self term, on the argmax key only
        d = full["dS"] - det["dS"]
        j = np.argmax(s)
        assert np.all(d[np.arange(n) != j] == 0)
        assert abs(d[j] + det["dS"].sum()) <= 1e-15 * tot
        if mode == "softmax":
            assert abs(det["dS"].sum()) <= 1e-14 * tot
        elif mode == "bf16_exp":
            assert abs(det["dS"].sum()) <= 2.0 ** -7 * tot
        else:
            assert abs(det["dS"].sum()) > 1e-6 * tot


def test_softmax_row_is_textbook(oracle_mod):
    """P = softmax(s), dS = P (g - P.g) (App. A, Softmax)."""
    rng = np.random.default_rng(6)
    for n in (1, 3, 50):
        s = rand_scores(rng, n, 2.0)
        g = rng.normal(size=n)
        out = oracle_mod.row(s, g, recon="softmax")
        e = np.exp(s - s.max())
        P = e / e.sum()
        assert np.abs(out["P"] - P).max() <= 1e-7
        ref = P * (g - P @ g)
        assert np.abs(out["dS"] - ref).max() <= 1e-6 * np.abs(ref).max() + 1e-300


# --------------------------------------------------------------------------
# Attention level
# --------------------------------------------------------------------------

def torch_attention(q, k, v, dO, mode, causal):
    """fp32 PyTorch attention with the given weight function; scores are
    fl32(fl32(q.k) * fl32(1/sqrt(d))) as in the paper's fp32 path."""
    B, H, T, d = q.shape
    qt, kt, vt = (torch.tensor(f32(x), requires_grad=True) for x in (q, k, v))
    scale = torch.tensor(np.float32(1.0 / math.sqrt(d)))
    S = torch.matmul(qt.double(), kt.double().transpose(-1, -2).contiguous()).float() * scale
    if causal:
        mask = torch.ones(T, T, dtype=torch.bool).tril()
        S = S.masked_fill(~mask, -float("inf"))
    M = S.max(dim=-1, keepdim=True).values
    z = S - M
    if mode == "softmax":
        w = torch.exp(z)
    elif mode == "bf16_exp":
        w = torch.exp(z.to(torch.bfloat16)).float()
    else:
        we = torch.exp(z)
        w = we.detach().to(torch.float8_e4m3fn).float() + (we - we.detach())
    P = w / w.sum(dim=-1, keepdim=True)
    O = torch.matmul(P, vt)
    (O * torch.tensor(f32(dO))).sum().backward()
    return [x.detach().numpy().astype(np.float64) for x in (O, qt.grad, kt.grad, vt.grad)]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("causal", (1, 0))
def test_attention_matches_torch(oracle_mod, mode, causal):
    rng = np.random.default_rng(7)
    B, H, T, d = 1, 2, 48, 16
    q, k, v, dO = (rng.normal(size=(B, H, T, d)).astype(np.float32) for _ in range(4))
    q *= 2.0
    o, _, _, _ = oracle_mod.attn_fwd(q, k, v, 4, "minmax", 8.0, mode, causal=causal)
    dq, dk, dv, _, _ = oracle_mod.attn_bwd(q, k, v, dO, 4, "minmax", 8.0, mode, "weight",
                                           "full", causal=causal)
    ref = torch_attention(q, k, v, dO, mode, causal)
    tol = {"softmax": 1e-5, "fp8_exp": 1e-5, "bf16_exp": 4e-3}[mode]
    for x, r in zip((o, dq, dk, dv), ref):
        assert np.abs(x - r).max() <= tol * np.abs(r).max()
