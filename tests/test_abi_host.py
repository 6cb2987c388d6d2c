"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports
every entry point include/kia.h declares, sizes the stats buffer as the
header documents, and rejects bad arguments before any launch."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kia.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2609_33591_amd as kia
    if not os.path.exists(kia.LIB_PATH):
        from paper_2609_33591_amd import build
        build.build()
    return kia.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kia_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"kia_attn_fwd", "kia_attn_bwd", "kia_attn_fwd_bf16", "kia_attn_bwd_bf16",
            "kia_stats_bytes", "kia_strerror"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_stats_layout_matches_header(lib):
    import paper_2609_33591_amd as kia
    B, H, T, d = 2, 3, 100, 64
    R = B * H * T
    a256 = lambda x: (x + 255) // 256 * 256
    nq = (T + 31) // 32
    for causal, ntile in ((1, nq * (nq + 1) // 2), (0, nq * nq)):
        dsb = B * H * ntile * 4096
        # O^L is present for every operator (only Nearest + Prob-STE writes
        # it), so no offset depends on recon or ste
        for recon, ste, ol in (("nearest", "prob", R * d * 4), ("lerp", "weight", R * d * 4),
                               ("lerp", "prob", R * d * 4), ("nearest", "weight", R * d * 4),
                               ("softmax", "prob", R * d * 4), ("bf16_exp", "weight", R * d * 4),
                               ("fp8_exp", "prob", R * d * 4)):
            offs = [kia.kia_stats_offset(B, H, T, d, recon, ste, causal, f) for f in range(15)]
            # the deterministic backward's row-sum partials (2 x ceil(T/128) x R),
            # which then hold its calibration records (4 x R)
            part = max(2 * ((T + 127) // 128), 4) * R * 4
            sizes = [R * 4] * 8 + [R * 64, R * 4, R * 4, ol, dsb, dsb, part]
            exp = [sum(a256(s) for s in sizes[:f]) for f in range(16)]
            assert offs == exp[:15]
            assert all(o % 256 == 0 for o in offs)
            assert kia.kia_stats_bytes(B, H, T, d, recon, ste, causal) == exp[15]


ARGS = dict(B=1, H=1, T=64, d=64, K=4, calib=0, tau=8.0, recon=0, ste=0, detach=0, causal=1)


def call_fwd(lib, **kw):
    a = dict(ARGS, **kw)
    fake = ctypes.c_void_p(4096)  # never dereferenced: validation fails first
    return lib.kia_attn_fwd(fake, fake, fake, fake, fake, a["B"], a["H"], a["T"], a["d"],
                            a["K"], a["calib"], a["tau"], a["recon"], a["ste"],
                            a["detach"], a["causal"], None)


def call_bwd(lib, **kw):
    a = dict(ARGS, **kw)
    fake = ctypes.c_void_p(4096)
    return lib.kia_attn_bwd(*([fake] * 9), a["B"], a["H"], a["T"], a["d"], a["K"],
                            a["calib"], a["tau"], a["recon"], a["ste"], a["detach"],
                            a["causal"], None)


def call_fwd16(lib, **kw):
    a = dict(ARGS, **kw)
    fake = ctypes.c_void_p(4096)
    return lib.kia_attn_fwd_bf16(fake, fake, fake, fake, fake, a["B"], a["H"], a["T"], a["d"],
                                 a["K"], a["calib"], a["tau"], a["recon"], a["ste"],
                                 a["detach"], a["causal"], None)


def call_bwd16(lib, **kw):
    a = dict(ARGS, **kw)
    fake = ctypes.c_void_p(4096)
    return lib.kia_attn_bwd_bf16(*([fake] * 9), a["B"], a["H"], a["T"], a["d"], a["K"],
                                 a["calib"], a["tau"], a["recon"], a["ste"], a["detach"],
                                 a["causal"], None)


@pytest.mark.parametrize("call", (call_fwd, call_bwd, call_fwd16, call_bwd16))
def test_invalid_arguments_are_rejected_on_the_host(lib, call):
    assert call(lib, d=48) == -3
    assert call(lib, d=256) == -3
    assert call(lib, B=0) == -2
    assert call(lib, T=0) == -2
    assert call(lib, T=65537) == -2
    assert call(lib, B=1 << 14, H=1 << 10, T=1 << 10) == -2   # size overflow
    assert call(lib, K=0) == -4
    assert call(lib, K=65) == -4
    assert call(lib, calib=3) == -5
    assert call(lib, calib=-1) == -5
    assert call(lib, recon=-1) == -5
    assert call(lib, ste=3) == -5
    assert call(lib, detach=6) == -5
    assert call(lib, detach=-1) == -5
    assert call(lib, causal=7) == -5
    assert call(lib, calib=1, tau=0.0) == -6
    assert call(lib, calib=1, tau=-1.0) == -6
    assert call(lib, calib=1, tau=float("inf")) == -6
    assert call(lib, calib=1, tau=float("nan")) == -6
    assert call(lib, calib=2, tau=0.0) == -6
    assert call(lib, calib=2, tau=float("nan")) == -6


def test_null_and_alignment_checks(lib):
    a = ARGS
    good = ctypes.c_void_p(4096)
    rc = lib.kia_attn_fwd(None, good, good, good, good, a["B"], a["H"], a["T"], a["d"],
                          a["K"], 0, 8.0, 0, 0, 0, 1, None)
    assert rc == -1
    odd = ctypes.c_void_p(4096 + 4)
    rc = lib.kia_attn_fwd(odd, good, good, good, good, a["B"], a["H"], a["T"], a["d"],
                          a["K"], 0, 8.0, 0, 0, 0, 1, None)
    assert rc == -7
    rc = lib.kia_attn_fwd(good, good, good, good, ctypes.c_void_p(4096 + 16), a["B"], a["H"],
                          a["T"], a["d"], a["K"], 0, 8.0, 0, 0, 0, 1, None)
    assert rc == -7


def test_strerror_names_every_code(lib):
    import paper_2609_33591_amd as kia
    for code in range(0, -9, -1):
        assert kia.kia_strerror(code) != "unknown error code"
    assert kia.kia_strerror(-99) == "unknown error code"


def test_exponential_weight_functions_are_validated_on_the_host(lib):
    """recon 2-4 (softmax, BF16-exp, FP8-exp) do not use K, calib, tau or ste;
    the bf16-input entry points reject them; recon 5 does not exist."""
    for call in (call_fwd, call_bwd, call_fwd16, call_bwd16):
        assert call(lib, recon=5) == -5
    for call in (call_fwd16, call_bwd16):
        for recon in (2, 3, 4):
            assert call(lib, recon=recon) == -5
    for call in (call_fwd, call_bwd):
        for recon in (2, 3, 4):
            assert call(lib, recon=recon, detach=6) == -5
            assert call(lib, recon=recon, causal=2) == -5
            assert call(lib, recon=recon, d=48) == -3
    good = ctypes.c_void_p(4096)
    for recon in (2, 3, 4):
        # K, calib, tau, ste unused: validation passes, the NULL q is caught
        rc = lib.kia_attn_fwd(None, good, good, good, good, 1, 1, 64, 64, 0, 9,
                              float("nan"), recon, 7, 0, 1, None)
        assert rc == -1
        rc = lib.kia_attn_bwd(None, *([good] * 8), 1, 1, 64, 64, 99, -3, -1.0, recon, 5,
                              0, 1, None)
        assert rc == -1
        n = ctypes.c_size_t(0)
        assert lib.kia_stats_bytes(1, 1, 64, 64, recon, 0, 1, ctypes.byref(n)) == 0
        assert n.value > 0


def test_forward_only_mode(lib):
    """KIA_GRAD_NONE (5) passes the forward's checks (the NULL q is what
    stops it here) and is refused by every backward entry point and by the
    static forward + backward before anything is enqueued."""
    good = ctypes.c_void_p(4096)
    a = ARGS
    for recon, ste in ((1, 1), (0, 0), (2, 0)):
        rc = lib.kia_attn_fwd(None, good, good, good, good, a["B"], a["H"], a["T"], a["d"],
                              a["K"], 1, 8.0, recon, ste, 5, 1, None)
        assert rc == -1
        if recon < 2:
            assert lib.kia_attn_fwd_bf16(None, good, good, good, good, a["B"], a["H"], a["T"],
                                         a["d"], a["K"], 1, 8.0, recon, ste, 5, 1, None) == -1
        assert call_bwd(lib, recon=recon, ste=ste, calib=1, detach=5) == -5
        assert call_bwd16(lib, recon=min(recon, 1), ste=ste, calib=1, detach=5) == -5
        rc = lib.kia_attn_fwd_bwd_static(*([good] * 8), a["B"], a["H"], a["T"], a["d"], a["K"], 1,
                                         8.0, recon, ste, 5, 1, None)
        assert rc == -5


def test_grid_policy_values(lib):
    """auto / wide / split are accepted (host state only), anything else is
    an enum error; the policy is left at auto."""
    import paper_2609_33591_amd as kia
    try:
        for p in (1, 2, 0):
            assert lib.kia_set_grid_policy(p) == 0
        for p in (-1, 3, 99):
            assert lib.kia_set_grid_policy(p) == -5
        with pytest.raises(kia.KiaError):
            kia.kia_set_grid_policy(7)
        kia.kia_set_grid_policy("split")
    finally:
        kia.kia_set_grid_policy("auto")


def test_deterministic_switch_values(lib):
    """0 and 1 are accepted (host state only), anything else is an enum
    error; the switch is left off."""
    import paper_2609_33591_amd as kia
    try:
        for v in (1, 0):
            assert lib.kia_set_deterministic(v) == 0
        for v in (-1, 2, 99):
            assert lib.kia_set_deterministic(v) == -5
        with pytest.raises(kia.KiaError):
            kia.kia_set_deterministic("yes")
        kia.kia_set_deterministic(True)
    finally:
        kia.kia_set_deterministic(False)


def test_mfma_probe_arguments_are_checked_on_the_host(lib):
    good = ctypes.c_void_p(4096)
    assert lib.kia_mfma_peak_probe(None, 1, 1, None) == -1
    assert lib.kia_mfma_peak_probe(ctypes.c_void_p(4096 + 4), 1, 1, None) == -7
    for wg, iters in ((0, 1), (1, 0), (1 << 21, 1), (1, 1 << 21), (-1, 5)):
        assert lib.kia_mfma_peak_probe(good, wg, iters, None) == -2
