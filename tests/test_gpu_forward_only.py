"""The forward-only gradient mode (KIA_GRAD_NONE, "none") on the device.

A forward-only forward leaves out what the backward alone reads (O^L, the
Prob-STE Nearest forward's third product, and the decisions stored in U)
and is otherwise the forward of every mode: O and the row statistics (M, m,
W, W^L, first extremum indices, tie counts) are bitwise equal to a forward
with the full gradient mode, on fp32, bf16-input and bf16-output entry
points and for the exponential weight functions. A backward or a decode of
stored decisions on its stats is refused by the binding, and a backward
asked for mode "none" by the C ABI; the autograd operation takes this path
where no gradient can be taken.
"""
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402
import test_gpu_parity as P  # noqa: E402

FIELDS = ("M", "m", "W", "WL", "amax", "amin", "nmax", "nmin")
# (calib, recon, ste)
OPS = [("fwm", "nearest", "prob"), ("minmax", "nearest", "prob"), ("minmax", "lerp", "weight"),
       ("resolved", "nearest", "weight"), ("fwm", "softmax", "weight")]
SHAPES = [(1, 2, 300, 64, 1), (2, 1, 77, 32, 0), (1, 1, 130, 128, 1), (1, 1, 1, 16, 1)]


def fields(st, shape):
    return {f: kia.stats_field(st, *shape, f).clone() for f in FIELDS}


# the exponential weight functions take fp32 inputs only
CASES = [(op, dt) for op in OPS for dt in ("f32", "bf16", "bf16o")
         if dt == "f32" or op[1] != "softmax"]


@pytest.mark.parametrize("op,dtype", CASES, ids=lambda x: x if isinstance(x, str) else "-".join(x))
def test_forward_only_equals_the_training_forward(op, dtype):
    calib, recon, ste = op
    exp = recon == "softmax"
    for i, (B, H, T, d, causal) in enumerate(SHAPES):
        tag = f"forward-only {op} {dtype} B{B} H{H} T{T} d{d} causal{causal}"
        P.flush("case " + tag)
        q, k, v, _ = make_inputs(B, H, T, d, seed=1100 + i, qk_scale=1.5, dyadic=True)
        dt = torch.float32 if dtype == "f32" else torch.bfloat16
        q, k, v = (x.to(dt).cuda() for x in (q, k, v))
        out = torch.bfloat16 if dtype == "bf16o" else None
        args = (4, calib, 8.0, recon, ste)
        runs = {}
        for mode in ("full", "none"):
            o, st = kia.forward(q, k, v, *args, mode, causal, out_dtype=out)
            torch.cuda.synchronize()
            runs[mode] = (o, st, fields(st, (B, H, T, d)))
        (o0, _, f0), (o1, st1, f1) = runs["full"], runs["none"]
        assert torch.equal(o0, o1), tag
        # FWM (and the exponential weights, which calibrate like it) keeps no
        # minimum: m, amin and nmin are not written there
        kept = FIELDS if calib != "fwm" else ("M", "W", "WL", "amax", "nmax")
        for f in kept:
            assert torch.equal(f0[f], f1[f]), (tag, f)
        if not exp:
            codes = torch.zeros((B, H, T, T), dtype=torch.int16, device="cuda")
            with pytest.raises(kia.KiaError, match="forward-only"):
                kia.kia_debug_codes_stored(st1, codes, B, H, T, d, *args, causal)
        # no backward on the forward-only stats: the binding refuses it
        dO = torch.ones_like(q)  # the input dtype
        with pytest.raises(kia.KiaError, match="forward-only"):
            kia.backward(q, k, v, o1, dO, st1, *args, "full", causal)
        # and the C ABI refuses a backward asked for mode "none"
        o2, st2 = kia.forward(q, k, v, *args, "full", causal, out_dtype=out)
        with pytest.raises(kia.KiaError, match="gradient mode"):
            kia.backward(q, k, v, o2, dO, st2, *args, "none", causal)


def test_autograd_op_without_gradients_runs_forward_only():
    """Under torch.no_grad (or with no input requiring grad) the autograd
    operation returns the forward-only output, equal to the training
    forward's; with gradients it still takes the full forward."""
    q, k, v, dO = (x.cuda() for x in make_inputs(1, 2, 200, 64, seed=1200, dyadic=True))
    args = (4, "fwm", 8.0, "nearest", "prob", False, True)
    ref, _ = kia.forward(q, k, v, *args)
    with torch.no_grad():
        o = kia.k_interval_attention(q.requires_grad_(), k, v, *args)
    assert not o.requires_grad and torch.equal(o, ref)
    q.requires_grad_(False)
    o = kia.k_interval_attention(q, k, v, *args)
    assert not o.requires_grad and torch.equal(o, ref)
    qa = q.clone().requires_grad_()
    o = kia.k_interval_attention(qa, k, v, *args)
    assert o.requires_grad and torch.equal(o.detach(), ref)
    o.backward(dO)
    assert qa.grad is not None and torch.isfinite(qa.grad).all()
