"""GPU parity at the paper's own attention call shapes: micro-batch 1,
T = 1024, d_h = 64 with the 124M model's 12 heads and the 1B model's 24
heads (the paper trains with micro-batch 1 and gradient accumulation).
Every slice is compared against the oracle on exact-score (dyadic) inputs,
for the bench operator and for MinMax LERP, at the bar of the other parity
tests (codes and extrema bit-exact, O 1e-4, dQ/dK/dV 1e-3)."""
import pytest

pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import test_gpu_parity as P  # noqa: E402


@pytest.mark.parametrize("name", ("paper_124m_mb1", "paper_1b_mb1"))
@pytest.mark.parametrize("variant", (None, dict(calib="minmax", recon="lerp", ste="weight")),
                         ids=("bench-operator", "minmax-lerp"))
def test_paper_call_shapes(oracle_mod, name, variant):
    H = P.WORKLOADS[name]["H"]
    P.full_size_check(oracle_mod, name, variant=variant, n_slices=H)
