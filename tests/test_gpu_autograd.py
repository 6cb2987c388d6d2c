"""The autograd operation k_interval_attention on the device.

1. Inside a small attention block (q, k, v and output projections, strided
   [B,H,T,d] views of the projections as inputs), the loss gradients of
   every parameter and of the block's input match the same block run on
   the CPU in fp64 with the oracle's forward and backward as its attention
   (O 1e-4, gradients 1e-3, the operator's parity bars). The projections
   are exact in fp32 (small multiples of 1/8), so both sides see the same
   scores and take the same index decisions.
2. Under kia_set_deterministic(True), its output and gradients are bitwise
   those of direct forward()/backward() calls on the same tensors, for
   float32 and for bfloat16 (the bf16-output entry points); the bfloat16
   gradients also meet the 2e-2 bar against the oracle.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402
import test_gpu_bf16 as B16  # noqa: E402
import test_gpu_parity as P  # noqa: E402

# (calib, recon, ste, gradient mode)
VARIANTS = [("fwm", "nearest", "prob", "full"), ("minmax", "lerp", "weight", "full"),
            ("minmax", "nearest", "weight", "detach"), ("fwm", "lerp", "prob", "max_only")]


def oracle_attention(oracle, K, calib, tau, recon, ste, mode, causal):
    """fp64 CPU autograd operation whose forward and backward are the
    oracle's (test reference only)."""

    class OracleAttention(torch.autograd.Function):
        @staticmethod
        def forward(ctx, q, k, v):
            args = [x.detach().contiguous().numpy() for x in (q, k, v)]
            o, _, _, _ = oracle.attn_fwd(*args, K=K, calib=calib, tau=tau, recon=recon,
                                         causal=causal, want_codes=False)
            ctx.save_for_backward(q, k, v)
            return torch.from_numpy(np.ascontiguousarray(o))

        @staticmethod
        def backward(ctx, dO):
            args = [x.detach().contiguous().numpy() for x in ctx.saved_tensors]
            dq, dk, dv, _, _ = oracle.attn_bwd(*args, dO.contiguous().numpy(), K=K,
                                               calib=calib, tau=tau, recon=recon, ste=ste,
                                               detach=mode, causal=causal)
            return tuple(torch.from_numpy(np.ascontiguousarray(x)) for x in (dq, dk, dv))

    return OracleAttention.apply


def block_params(B, T, H, d, seed):
    """x and the projection weights (fp64 CPU): x in {-2..2}, Wq and Wk in
    {-1/8, 0, 1/8} (q and k multiples of 1/8 with |q|, |k| <= 8, exact in
    fp32 for C <= 32), Wv, Wo and the loss weights r N(0, 1)-scaled."""
    g = torch.Generator().manual_seed(seed)
    C = H * d
    x = torch.randint(-2, 3, (B, T, C), generator=g).double()
    wq, wk = (torch.randint(-1, 2, (C, C), generator=g).double() / 8 for _ in range(2))
    wv, wo = (torch.randn(C, C, generator=g, dtype=torch.float64) / C ** 0.5 for _ in range(2))
    r = torch.randn(B, T, C, generator=g, dtype=torch.float64)
    return dict(x=x, wq=wq, wk=wk, wv=wv, wo=wo), r


def block_loss(p, r, attn, H, d):
    """sum(r * (attn(q, k, v) Wo)), q = x Wq (and k, v) viewed [B,H,T,d]."""
    x = p["x"]
    B, T, C = x.shape

    def heads(w):
        return (x @ w).view(B, T, H, d).transpose(1, 2)  # a strided view

    o = attn(heads(p["wq"]), heads(p["wk"]), heads(p["wv"]))
    y = o.transpose(1, 2).reshape(B, T, C) @ p["wo"]
    return (y * r).sum(), y


def rel(x, ref):
    return float((x - ref).abs().max() / ref.abs().max())


@pytest.mark.parametrize("variant", VARIANTS, ids=lambda v: "-".join(v))
def test_autograd_block_against_oracle(oracle_mod, variant):
    calib, recon, ste, mode = variant
    B, T, H, d = 2, 45, 2, 16
    for causal in (1, 0):
        tag = f"autograd block {variant} causal{causal}"
        P.flush("case " + tag)
        p64, r64 = block_params(B, T, H, d, seed=7 + causal)
        ref = {n: t.clone().requires_grad_() for n, t in p64.items()}
        lref, yref = block_loss(ref, r64, oracle_attention(oracle_mod, 4, calib, 8.0, recon, ste,
                                                           mode, causal), H, d)
        lref.backward()
        gpu = {n: t.float().cuda().requires_grad_() for n, t in p64.items()}
        attn = lambda q, k, v: kia.k_interval_attention(q, k, v, 4, calib, 8.0, recon, ste,
                                                        mode, causal)
        loss, y = block_loss(gpu, r64.float().cuda(), attn, H, d)
        loss.backward()
        torch.cuda.synchronize()
        assert rel(y.detach().cpu().double(), yref.detach()) <= P.O_TOL, (tag, "y")
        for n in p64:
            err = rel(gpu[n].grad.cpu().double(), ref[n].grad)
            assert err <= P.G_TOL, (tag, n, err)


@pytest.fixture
def deterministic():
    kia.kia_set_deterministic(True)
    try:
        yield
    finally:
        kia.kia_set_deterministic(False)


@pytest.mark.parametrize("dtype", ("float32", "bfloat16"))
def test_autograd_equals_direct_calls(oracle_mod, deterministic, dtype):
    dt = getattr(torch, dtype)
    for i, (B, H, T, d, causal) in enumerate([(1, 2, 300, 64, 1), (2, 1, 77, 32, 0),
                                              (1, 1, 130, 128, 1)]):
        tag = f"autograd direct {dtype} B{B} H{H} T{T} d{d} causal{causal}"
        P.flush("case " + tag)
        q, k, v, dO = make_inputs(B, H, T, d, seed=990 + i, qk_scale=1.5, dyadic=True)
        q, k, v, dO = (x.to(dt).cuda() for x in (q, k, v, dO))
        args = (4, "fwm", 8.0, "nearest", "prob", False, causal)
        qa, ka, va = (x.clone().requires_grad_() for x in (q, k, v))
        o = kia.k_interval_attention(qa, ka, va, *args)
        o.backward(dO)
        b16 = dt == torch.bfloat16
        od, st = kia.forward(q, k, v, *args, out_dtype=torch.bfloat16 if b16 else None)
        gd = kia.backward(q, k, v, od, dO, st, *args)
        torch.cuda.synchronize()
        assert o.dtype == dt and torch.equal(o.detach(), od), tag
        for name, x, y in zip(("dq", "dk", "dv"), (qa.grad, ka.grad, va.grad), gd):
            assert x.dtype == dt and torch.equal(x, y), (tag, name)
        if b16:
            r = P.run_oracle(oracle_mod, *(x.float().cpu() for x in (q, k, v, dO)), *args,
                             codes=False)
            sl = [(b, h) for b in range(B) for h in range(H)]
            for name, x in zip(("dq", "dk", "dv"), gd):
                err = P.rel_err(x.float().cpu().double().numpy(), r[name], sl)
                assert err <= B16.B16_TOL, (tag, name, err)
