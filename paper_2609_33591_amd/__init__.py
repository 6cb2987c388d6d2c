"""K-interval attention on MI355X (gfx950): thin Python binding of libkia.

The functions below carry the names of the C-ABI entry points declared in
``include/kia.h`` and only marshal arguments: torch device tensors become
pointers and shapes, the current HIP stream is passed through, and a
nonzero return code raises ``KiaError``. Every step of the operator runs in
the HIP kernels of ``csrc/``; there is no CPU fallback. If ``libkia.so`` is
missing, the first call raises.

Operator (Zhu, Hu, Kozlowski, "Pretraining Transformers with Quantized
Softmax in Attention", Sec. 3 and App. A/B): causal attention whose
exponential is rebuilt from K+1 grid values, MinMax or FWM calibration,
LERP or Nearest reconstruction, Weight- or Prob-STE surrogate, full or
detached calibration gradient.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkia.so")

# calibrations; "resolved" is the tail-policy diagnostic (FWM's step and origin,
# the grid continued below -tau, no zero tail)
CALIB = {"minmax": 0, "fwm": 1, "resolved": 2}
# K-interval reconstructions, then the exponential weight functions of the
# baselines (exact softmax, BF16-exp, FP8-rounded exp; K, calib, tau and ste
# unused)
RECON = {"lerp": 0, "nearest": 1, "softmax": 2, "bf16_exp": 3, "fp8_exp": 4}
STE = {"weight": 0, "prob": 1}
GRID = {"auto": 0, "wide": 1, "split": 2}
# gradient modes of the backward's `detach` argument (KIA_GRAD_*)
GRAD = {"full": 0, "detach": 1, "max_only": 2, "min_only": 3, "p1": 4}

# stats fields (KIA_STAT_* of kia.h)
STAT_FIELDS = {"M": 0, "m": 1, "W": 2, "WL": 3, "amax": 4, "amin": 5,
               "nmax": 6, "nmin": 7, "rowrec": 8, "sself": 9, "cM": 10, "OL": 11,
               "dS": 12, "U": 13}

_lib = None


class KiaError(RuntimeError):
    pass


def load():
    """Load libkia.so (built in-tree by build.py); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise KiaError(f"{LIB_PATH} is missing: run paper_2609_33591_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        P, I, F, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        lib.kia_stats_bytes.argtypes = [I] * 7 + [ctypes.POINTER(S)]
        lib.kia_stats_offset.argtypes = [I] * 8 + [ctypes.POINTER(S)]
        lib.kia_attn_fwd.argtypes = [P, P, P, P, P] + [I] * 6 + [F] + [I] * 4 + [P]
        lib.kia_attn_bwd.argtypes = [P] * 9 + [I] * 6 + [F] + [I] * 4 + [P]
        lib.kia_debug_codes.argtypes = [P] * 4 + [I] * 6 + [F] + [I, I] + [P]
        lib.kia_attn_fwd_bf16.argtypes = lib.kia_attn_fwd.argtypes
        lib.kia_attn_bwd_bf16.argtypes = lib.kia_attn_bwd.argtypes
        lib.kia_debug_codes_bf16.argtypes = lib.kia_debug_codes.argtypes
        lib.kia_debug_score_grad.argtypes = [P, I, P, P, P] + [I] * 8 + [P]
        lib.kia_geometry_probe.argtypes = [P] * 4 + [I] * 6 + [F] + [I, I] + [P]
        lib.kia_set_grid_policy.argtypes = [I]
        lib.kia_mfma_peak_probe.argtypes = [P, I, I, P]
        lib.kia_timing_enable.argtypes = [I]
        lib.kia_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(I)]
        lib.kia_strerror.argtypes = [I]
        lib.kia_strerror.restype = ctypes.c_char_p
        for fn in ("kia_stats_bytes", "kia_stats_offset", "kia_attn_fwd",
                   "kia_attn_bwd", "kia_debug_codes", "kia_attn_fwd_bf16",
                   "kia_attn_bwd_bf16", "kia_debug_codes_bf16", "kia_debug_score_grad",
                   "kia_geometry_probe", "kia_set_grid_policy", "kia_mfma_peak_probe",
                   "kia_timing_enable",
                   "kia_timing_read"):
            getattr(lib, fn).restype = I
        _lib = lib
    return _lib


def _check(rc: int) -> None:
    if rc != 0:
        raise KiaError(f"libkia error {rc}: {load().kia_strerror(rc).decode()}")


def _ptr(t, dtypes):
    import torch
    if not t.is_cuda:
        raise KiaError("libkia takes device tensors only")
    if t.dtype not in dtypes:
        raise KiaError(f"unexpected dtype {t.dtype}")
    if not t.is_contiguous():
        raise KiaError("tensors must be contiguous [B,H,T,d]")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _enum(x, table):
    return table[x] if isinstance(x, str) else int(x)


def _grad(mode) -> int:
    """False/True (full/detach), a GRAD name, or its integer code."""
    if isinstance(mode, str):
        return GRAD[mode]
    return int(mode)


def kia_strerror(code: int) -> str:
    return load().kia_strerror(int(code)).decode()


def kia_stats_bytes(B, H, T, d, recon, ste, causal) -> int:
    n = ctypes.c_size_t(0)
    _check(load().kia_stats_bytes(B, H, T, d, _enum(recon, RECON), _enum(ste, STE),
                                  int(bool(causal)), ctypes.byref(n)))
    return n.value


def kia_stats_offset(B, H, T, d, recon, ste, causal, field) -> int:
    n = ctypes.c_size_t(0)
    f = STAT_FIELDS[field] if isinstance(field, str) else int(field)
    _check(load().kia_stats_offset(B, H, T, d, _enum(recon, RECON), _enum(ste, STE),
                                   int(bool(causal)), f, ctypes.byref(n)))
    return n.value


def kia_attn_fwd(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
                 stream=None):
    import torch
    B, H, T, d = q.shape
    f32 = (torch.float32,)
    _check(load().kia_attn_fwd(_ptr(q, f32), _ptr(k, f32), _ptr(v, f32), _ptr(o, f32),
                               _ptr(stats, (torch.uint8,)), B, H, T, d, int(K),
                               _enum(calib, CALIB), float(tau), _enum(recon, RECON),
                               _enum(ste, STE), _grad(detach), int(bool(causal)),
                               _stream(stream)))


def kia_attn_bwd(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
                 detach, causal, stream=None):
    import torch
    B, H, T, d = q.shape
    f32 = (torch.float32,)
    _check(load().kia_attn_bwd(_ptr(q, f32), _ptr(k, f32), _ptr(v, f32), _ptr(o, f32),
                               _ptr(dO, f32), _ptr(stats, (torch.uint8,)), _ptr(dq, f32),
                               _ptr(dk, f32), _ptr(dv, f32), B, H, T, d, int(K),
                               _enum(calib, CALIB), float(tau), _enum(recon, RECON),
                               _enum(ste, STE), _grad(detach), int(bool(causal)),
                               _stream(stream)))


def kia_debug_codes(q, k, stats, codes, K, calib, tau, recon, causal, stream=None):
    import torch
    B, H, T, d = q.shape
    f32 = (torch.float32,)
    _check(load().kia_debug_codes(_ptr(q, f32), _ptr(k, f32), _ptr(stats, (torch.uint8,)),
                                  _ptr(codes, (torch.int16, torch.uint16)), B, H, T, d,
                                  int(K), _enum(calib, CALIB), float(tau),
                                  _enum(recon, RECON), int(bool(causal)), _stream(stream)))


def kia_attn_fwd_bf16(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
                      stream=None):
    """bf16-input forward: q, k, v torch.bfloat16; o fp32."""
    import torch
    B, H, T, d = q.shape
    b16, f32 = (torch.bfloat16,), (torch.float32,)
    _check(load().kia_attn_fwd_bf16(_ptr(q, b16), _ptr(k, b16), _ptr(v, b16), _ptr(o, f32),
                                    _ptr(stats, (torch.uint8,)), B, H, T, d, int(K),
                                    _enum(calib, CALIB), float(tau), _enum(recon, RECON),
                                    _enum(ste, STE), _grad(detach), int(bool(causal)),
                                    _stream(stream)))


def kia_attn_bwd_bf16(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
                      detach, causal, stream=None):
    """bf16-input backward: q, k, v, dO torch.bfloat16; o, dq, dk, dv fp32."""
    import torch
    B, H, T, d = q.shape
    b16, f32 = (torch.bfloat16,), (torch.float32,)
    _check(load().kia_attn_bwd_bf16(_ptr(q, b16), _ptr(k, b16), _ptr(v, b16), _ptr(o, f32),
                                    _ptr(dO, b16), _ptr(stats, (torch.uint8,)), _ptr(dq, f32),
                                    _ptr(dk, f32), _ptr(dv, f32), B, H, T, d, int(K),
                                    _enum(calib, CALIB), float(tau), _enum(recon, RECON),
                                    _enum(ste, STE), _grad(detach), int(bool(causal)),
                                    _stream(stream)))


def kia_debug_codes_bf16(q, k, stats, codes, K, calib, tau, recon, causal, stream=None):
    import torch
    B, H, T, d = q.shape
    b16 = (torch.bfloat16,)
    _check(load().kia_debug_codes_bf16(_ptr(q, b16), _ptr(k, b16), _ptr(stats, (torch.uint8,)),
                                       _ptr(codes, (torch.int16, torch.uint16)), B, H, T, d,
                                       int(K), _enum(calib, CALIB), float(tau),
                                       _enum(recon, RECON), int(bool(causal)), _stream(stream)))


def kia_debug_score_grad(stats, g_self, cM, cm, B, H, T, d, calib, recon, ste, causal,
                         input_bf16=False, stream=None):
    """Score-gradient decomposition after a backward in mode full, max_only
    or min_only: g_self [B,H,T,T], cM and cm [B,H,T] (fp32 device tensors)."""
    import torch
    f32 = (torch.float32,)
    _check(load().kia_debug_score_grad(_ptr(stats, (torch.uint8,)), int(bool(input_bf16)),
                                       _ptr(g_self, f32), _ptr(cM, f32), _ptr(cm, f32),
                                       B, H, T, d, _enum(calib, CALIB), _enum(recon, RECON),
                                       _enum(ste, STE), int(bool(causal)), _stream(stream)))


# columns of kia_geometry_probe's per-row record (KIA_GEO_* of kia.h)
GEO_FIELDS = {"span": 0, "h": 1, "zq001": 2, "qnorm": 3, "knorm": 4, "entropy": 5,
              "frac_z_lt_m6": 6, "top_mass": 7, "eff_buckets": 8, "tv": 9}


def kia_geometry_probe(q, k, stats, out, K, calib, tau, recon, causal, stream=None):
    """Per-row geometry statistics out [B,H,T,10] (fp32 device) after
    kia_attn_fwd with the same arguments on `stats`."""
    import torch
    B, H, T, d = q.shape
    f32 = (torch.float32,)
    _check(load().kia_geometry_probe(_ptr(q, f32), _ptr(k, f32), _ptr(stats, (torch.uint8,)),
                                     _ptr(out, f32), B, H, T, d, int(K), _enum(calib, CALIB),
                                     float(tau), _enum(recon, RECON), int(bool(causal)),
                                     _stream(stream)))


def kia_set_grid_policy(policy) -> None:
    """Launch-shape policy: "auto" (split only grids too small to fill the
    chip), "wide" (never split) or "split" (always split)."""
    _check(load().kia_set_grid_policy(_enum(policy, GRID)))


def kia_mfma_peak_probe(out, workgroups: int, iters: int, stream=None) -> None:
    """Launch the fp32 matrix-core probe (workgroups x 4 x iters x 4 MFMAs of
    4096 flops) on `stream`; out is a device int64 tensor of 4 that receives
    the shader-clock and 100 MHz counters of workgroup 0 around its loop."""
    import torch
    if not out.is_cuda or out.dtype != torch.int64 or out.numel() < 4:
        raise KiaError("out must be a device int64 tensor of at least 4 elements")
    _check(load().kia_mfma_peak_probe(ctypes.c_void_p(out.data_ptr()), int(workgroups),
                                      int(iters), _stream(stream)))


def kia_timing_enable(on: bool) -> None:
    _check(load().kia_timing_enable(int(bool(on))))


def kia_timing_read(name: str):
    """(total milliseconds, launch count) of the kernels called `name`."""
    ms, n = ctypes.c_double(0.0), ctypes.c_int(0)
    _check(load().kia_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ---------------------------------------------------------------- helpers
def new_stats(B, H, T, d, recon, ste, causal=True, device="cuda"):
    """Caller-owned stats buffer (uint8 device tensor, 256-byte aligned)."""
    import torch
    n = kia_stats_bytes(B, H, T, d, recon, ste, causal)
    buf = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + n]


def stats_field(stats, B, H, T, d, field, recon="lerp", ste="weight", causal=True):
    """Typed view [B,H,T] (or [B,H,T,16] / [B,H,T,d]) of one stats field
    (fields M .. cM do not depend on recon/ste/causal)."""
    import torch
    f = STAT_FIELDS[field]
    if f in (12, 13):
        raise KiaError(f"stats field {field} is a tile scratch with no per-row view")
    off = kia_stats_offset(B, H, T, d, recon, ste, causal, f)
    R = B * H * T
    width = {8: 16, 11: d}.get(f, 1)
    dtype = torch.int32 if f in (4, 5, 6, 7) else torch.float32
    view = stats[off:off + R * width * 4].view(dtype)
    return view.view(B, H, T, width) if width > 1 else view.view(B, H, T)


def forward(q, k, v, K, calib, tau, recon, ste="weight", detach=False, causal=True):
    """Allocate o (fp32) and stats, run kia_attn_fwd (kia_attn_fwd_bf16 for
    bfloat16 inputs); returns (o, stats)."""
    import torch
    B, H, T, d = q.shape
    o = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    stats = new_stats(B, H, T, d, recon, ste, causal, device=q.device)
    fwd = kia_attn_fwd_bf16 if q.dtype == torch.bfloat16 else kia_attn_fwd
    fwd(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal)
    return o, stats


def backward(q, k, v, o, dO, stats, K, calib, tau, recon, ste="weight",
             detach=False, causal=True):
    """Allocate dq, dk, dv (fp32) and run kia_attn_bwd (kia_attn_bwd_bf16 for
    bfloat16 inputs); returns (dq, dk, dv)."""
    import torch
    dq, dk, dv = (torch.empty(q.shape, dtype=torch.float32, device=q.device) for _ in range(3))
    bwd = kia_attn_bwd_bf16 if q.dtype == torch.bfloat16 else kia_attn_bwd
    bwd(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste, detach, causal)
    return dq, dk, dv
