"""The no-allocation entry point kia_attn_fwd_bwd_static (statistics in the
library's static device scratch) against the allocating pair kia_attn_fwd +
kia_attn_bwd, through the C ABI: two calls in a row, the second with a
smaller problem (so it runs on what the first left in the scratch), each
held to the parity bar (O within 1e-4, dQ/dK/dV within 1e-3, max |x - ref| /
max |ref| per (b,h) slice). The forward output is deterministic, so O is
also compared bit for bit. A problem beyond the scratch is refused on the
host before any launch."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2609_33591_amd as kia  # noqa: E402
from paper_2609_33591_amd.inputs import make_inputs  # noqa: E402

O_TOL, G_TOL = 1e-4, 1e-3


def rel(x, ref):
    x, ref = x.double(), ref.double()
    num = (x - ref).abs().flatten(2).amax(dim=2)
    den = ref.abs().flatten(2).amax(dim=2).clamp_min(1e-300)
    return (num / den).max().item()


@pytest.mark.gpu
def test_static_scratch_matches_the_allocating_entry_points():
    cases = [((1, 12, 1024, 64), dict(K=4, calib="fwm", tau=8.0, recon="nearest", ste="prob",
                                      detach="full")),
             ((1, 3, 300, 32), dict(K=16, calib="minmax", tau=8.0, recon="lerp", ste="weight",
                                    detach="full"))]
    for n, ((B, H, T, d), op) in enumerate(cases):
        print(f"case static scratch B{B} H{H} T{T} d{d} {op}", flush=True)
        q, k, v, dO = (x.cuda() for x in make_inputs(B, H, T, d, seed=70 + n, qk_scale=1.5))
        a = (op["K"], op["calib"], op["tau"], op["recon"], op["ste"], op["detach"], True)
        o_ref, st = kia.forward(q, k, v, *a)
        ref = kia.backward(q, k, v, o_ref, dO, st, *a)
        outs = [torch.full_like(q, float("nan")) for _ in range(4)]
        kia.kia_attn_fwd_bwd_static(q, k, v, dO, *outs, *a)
        torch.cuda.synchronize()
        o, dq, dk, dv = outs
        assert torch.equal(o, o_ref)
        assert rel(o, o_ref) <= O_TOL
        for name, x, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
            e = rel(x, r)
            print(f"  {name}: {e:.2e}", flush=True)
            assert torch.isfinite(x).all() and e <= G_TOL, (name, e)


def test_static_scratch_refuses_problems_beyond_its_size():
    """Statistics larger than KIA_STATIC_BYTES: KIA_ERR_SCRATCH, decided on
    the host (no GPU touched; the pointers are never dereferenced)."""
    lib = kia.load()
    p = ctypes.c_void_p(256)
    need = kia.kia_stats_bytes(8, 12, 1024, 64, "nearest", "prob", True)
    assert need > 128 << 20
    rc = lib.kia_attn_fwd_bwd_static(p, p, p, p, p, p, p, p, 8, 12, 1024, 64, 4, 1, 8.0, 1, 1,
                                     0, 1, None)
    assert rc == -9
    assert "static scratch" in kia.kia_strerror(rc)
    assert kia.kia_stats_bytes(1, 24, 1024, 64, "nearest", "prob", True) <= 128 << 20
