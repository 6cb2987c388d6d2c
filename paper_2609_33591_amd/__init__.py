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
import functools
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
# (the forward also takes "none": no backward will read its stats)
GRAD = {"full": 0, "detach": 1, "max_only": 2, "min_only": 3, "p1": 4, "none": 5}

# stats fields (KIA_STAT_* of kia.h)
STAT_FIELDS = {"M": 0, "m": 1, "W": 2, "WL": 3, "amax": 4, "amin": 5,
               "nmax": 6, "nmin": 7, "rowrec": 8, "sself": 9, "cM": 10, "OL": 11,
               "dS": 12, "U": 13, "part": 14}

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
        lib.kia_attn_fwd_bf16o.argtypes = lib.kia_attn_fwd.argtypes
        lib.kia_attn_bwd_bf16o.argtypes = lib.kia_attn_bwd.argtypes
        lib.kia_stats_bytes_bf16o.argtypes = lib.kia_stats_bytes.argtypes
        lib.kia_debug_codes_bf16.argtypes = lib.kia_debug_codes.argtypes
        lib.kia_debug_codes_stored.argtypes = [P, P] + [I] * 6 + [F] + [I] * 3 + [P]
        lib.kia_debug_scores.argtypes = [P, P, P] + [I] * 5 + [P]
        lib.kia_debug_scores_bf16.argtypes = lib.kia_debug_scores.argtypes
        lib.kia_debug_score_grad.argtypes = [P, I, P, P, P] + [I] * 8 + [P]
        lib.kia_attn_fwd_bwd_static.argtypes = [P] * 8 + [I] * 6 + [F] + [I] * 4 + [P]
        lib.kia_geometry_probe.argtypes = [P] * 4 + [I] * 6 + [F] + [I, I] + [P]
        lib.kia_set_grid_policy.argtypes = [I]
        lib.kia_set_deterministic.argtypes = [I]
        lib.kia_mfma_peak_probe.argtypes = [P, I, I, P]
        lib.kia_timing_enable.argtypes = [I]
        lib.kia_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(I)]
        lib.kia_strerror.argtypes = [I]
        lib.kia_strerror.restype = ctypes.c_char_p
        for fn in ("kia_stats_bytes", "kia_stats_offset", "kia_attn_fwd",
                   "kia_attn_bwd", "kia_debug_codes", "kia_attn_fwd_bf16",
                   "kia_attn_bwd_bf16", "kia_debug_codes_bf16", "kia_debug_score_grad",
                   "kia_debug_codes_stored", "kia_debug_scores", "kia_debug_scores_bf16",
                   "kia_attn_fwd_bf16o", "kia_attn_bwd_bf16o", "kia_stats_bytes_bf16o",
                   "kia_attn_fwd_bwd_static",
                   "kia_geometry_probe", "kia_set_grid_policy", "kia_set_deterministic",
                   "kia_mfma_peak_probe",
                   "kia_timing_enable",
                   "kia_timing_read"):
            getattr(lib, fn).restype = I
        _lib = lib
    return _lib


def _check(rc: int) -> None:
    if rc != 0:
        raise KiaError(f"libkia error {rc}: {load().kia_strerror(rc).decode()}")


def _ptr(t, dtypes):
    """Device pointer of a contiguous tensor of one of `dtypes`."""
    if not t.is_cuda:
        raise KiaError("libkia takes device tensors only")
    if t.dtype not in dtypes:
        raise KiaError(f"unexpected dtype {t.dtype}")
    if not t.is_contiguous():
        raise KiaError("tensors must be contiguous [B,H,T,d]")
    return ctypes.c_void_p(t.data_ptr())


def _shape(q):
    if q.dim() != 4:
        raise KiaError(f"q must be [B,H,T,d], got shape {tuple(q.shape)}")
    return tuple(int(x) for x in q.shape)


def _same(q, named):
    """Every (name, tensor, dtypes) has q's [B,H,T,d] shape and device, one
    of `dtypes` and a contiguous layout (the C ABI takes sizes from q only,
    so a short buffer would become an out-of-bounds device access)."""
    shape = _shape(q)
    for name, t, dtypes in named:
        if tuple(t.shape) != shape:
            raise KiaError(f"{name} has shape {tuple(t.shape)}, q has {shape}")
        if t.dtype not in dtypes:
            raise KiaError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
        if t.device != q.device:
            raise KiaError(f"{name} is on {t.device}, q on {q.device}")
        if not t.is_contiguous():
            raise KiaError(f"{name} must be contiguous")
    return shape


def _check_stats(stats, q, shape, recon, ste, causal, nbytes=None):
    """stats is a flat uint8 buffer on q's device, 256-byte aligned, holding
    at least kia_stats_bytes (or `nbytes`) bytes."""
    import torch
    B, H, T, d = shape
    need = kia_stats_bytes(B, H, T, d, recon, ste, causal) if nbytes is None else nbytes
    if stats.dtype != torch.uint8 or stats.dim() != 1 or not stats.is_contiguous():
        raise KiaError("stats must be a contiguous 1-D uint8 tensor")
    if stats.device != q.device:
        raise KiaError(f"stats is on {stats.device}, q on {q.device}")
    if stats.numel() < need:
        raise KiaError(f"stats holds {stats.numel()} bytes, the problem needs {need}")
    if stats.data_ptr() % 256:
        raise KiaError("stats must be 256-byte aligned")


# The flags of the forward that last filled each stats buffer, keyed by its
# device and address: a backward (or a decode of the stored decisions) with
# other flags is rejected before the call (the C ABI leaves it undefined).
_FWD_FLAGS = {}


def _op_flags(shape, K, calib, tau, recon, ste, causal, in_dtype, nograd=False):
    """What a forward's statistics depend on: shape, causal mask, input
    type, the weight function and, for the K-interval ones, K, the
    calibration (tau unless MinMax) and, for Nearest, the surrogate; and
    whether the forward ran forward-only (gradient mode "none": no state
    for a backward)."""
    r = _enum(recon, RECON)
    c = _enum(calib, CALIB)
    grid = r in (RECON["lerp"], RECON["nearest"])
    return dict(shape=tuple(shape), causal=int(bool(causal)), input=str(in_dtype), recon=r,
                K=int(K) if grid else None, calib=c if grid else None,
                tau=float(tau) if grid and c != CALIB["minmax"] else None,
                ste=_enum(ste, STE) if r == RECON["nearest"] else None, nograd=bool(nograd))


def _stats_key(stats):
    return (str(stats.device), int(stats.data_ptr()))


def _record_forward(stats, flags):
    _FWD_FLAGS[_stats_key(stats)] = flags


def _check_forward(stats, flags, keys=None):
    """Raise if the forward that filled `stats` ran with other flags (only
    the `keys` given, default all)."""
    have = _FWD_FLAGS.get(_stats_key(stats))
    if have is None:
        return
    keys = keys or flags.keys()
    if "nograd" in keys and have["nograd"] and not flags["nograd"]:
        raise KiaError("stats were filled by a forward-only forward (gradient mode \"none\"), "
                       "which keeps no state for a backward or its stored decisions")
    diff = {k: (have[k], flags[k]) for k in keys if have[k] != flags[k]}
    if diff:
        raise KiaError("stats were filled by a forward with other arguments "
                       f"(forward, this call): {diff}")


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


@functools.lru_cache(maxsize=256)
def kia_stats_bytes(B, H, T, d, recon, ste, causal) -> int:
    n = ctypes.c_size_t(0)
    _check(load().kia_stats_bytes(B, H, T, d, _enum(recon, RECON), _enum(ste, STE),
                                  int(bool(causal)), ctypes.byref(n)))
    return n.value


@functools.lru_cache(maxsize=256)
def kia_stats_bytes_bf16o(B, H, T, d, recon, ste, causal) -> int:
    """Stats size for the bf16-output entry points (adds the fp32 dQ, dK
    accumulators; serves every other entry point too)."""
    n = ctypes.c_size_t(0)
    _check(load().kia_stats_bytes_bf16o(B, H, T, d, _enum(recon, RECON), _enum(ste, STE),
                                        int(bool(causal)), ctypes.byref(n)))
    return n.value


def kia_stats_offset(B, H, T, d, recon, ste, causal, field) -> int:
    n = ctypes.c_size_t(0)
    f = STAT_FIELDS[field] if isinstance(field, str) else int(field)
    _check(load().kia_stats_offset(B, H, T, d, _enum(recon, RECON), _enum(ste, STE),
                                   int(bool(causal)), f, ctypes.byref(n)))
    return n.value


def _fwd(fn, q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal, stream,
         in_dtype, o_dtypes):
    import torch
    shape = _same(q, [("k", k, (in_dtype,)), ("v", v, (in_dtype,)), ("o", o, o_dtypes)])
    _check_stats(stats, q, shape, _enum(recon, RECON), _enum(ste, STE), causal)
    B, H, T, d = shape
    ip = (in_dtype,)
    _check(fn(_ptr(q, ip), _ptr(k, ip), _ptr(v, ip), _ptr(o, o_dtypes),
              _ptr(stats, (torch.uint8,)), B, H, T, d, int(K), _enum(calib, CALIB),
              float(tau), _enum(recon, RECON), _enum(ste, STE), _grad(detach),
              int(bool(causal)), _stream(stream)))
    _record_forward(stats, _op_flags(shape, K, calib, tau, recon, ste, causal, in_dtype,
                                     nograd=_grad(detach) == GRAD["none"]))


def _bwd(fn, q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste, detach, causal,
         stream, in_dtype, o_dtypes, nbytes=None):
    import torch
    shape = _same(q, [("k", k, (in_dtype,)), ("v", v, (in_dtype,)), ("o", o, o_dtypes),
                      ("dO", dO, (in_dtype,)), ("dq", dq, o_dtypes), ("dk", dk, o_dtypes),
                      ("dv", dv, o_dtypes)])
    if nbytes is not None:
        nbytes = nbytes(*shape, _enum(recon, RECON), _enum(ste, STE), causal)
    _check_stats(stats, q, shape, _enum(recon, RECON), _enum(ste, STE), causal, nbytes)
    _check_forward(stats, _op_flags(shape, K, calib, tau, recon, ste, causal, in_dtype))
    B, H, T, d = shape
    ip = (in_dtype,)
    _check(fn(_ptr(q, ip), _ptr(k, ip), _ptr(v, ip), _ptr(o, o_dtypes), _ptr(dO, ip),
              _ptr(stats, (torch.uint8,)), _ptr(dq, o_dtypes), _ptr(dk, o_dtypes),
              _ptr(dv, o_dtypes), B, H, T, d, int(K), _enum(calib, CALIB), float(tau),
              _enum(recon, RECON), _enum(ste, STE), _grad(detach), int(bool(causal)),
              _stream(stream)))


def kia_attn_fwd(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
                 stream=None):
    """Forward (fp32): q, k, v, o [B,H,T,d] float32 device tensors; stats a
    uint8 device buffer of kia_stats_bytes bytes (see new_stats)."""
    import torch
    _fwd(load().kia_attn_fwd, q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
         stream, torch.float32, (torch.float32,))


def kia_attn_bwd(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
                 detach, causal, stream=None):
    """Backward (fp32) on the stats a forward with the same arguments
    filled; `detach` is the gradient mode (the backward's own choice)."""
    import torch
    _bwd(load().kia_attn_bwd, q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
         detach, causal, stream, torch.float32, (torch.float32,))


def kia_attn_fwd_bf16(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
                      stream=None):
    """bf16-input forward: q, k, v torch.bfloat16; o fp32."""
    import torch
    _fwd(load().kia_attn_fwd_bf16, q, k, v, o, stats, K, calib, tau, recon, ste, detach,
         causal, stream, torch.bfloat16, (torch.float32,))


def kia_attn_bwd_bf16(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
                      detach, causal, stream=None):
    """bf16-input backward: q, k, v, dO torch.bfloat16; o, dq, dk, dv fp32."""
    import torch
    _bwd(load().kia_attn_bwd_bf16, q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon,
         ste, detach, causal, stream, torch.bfloat16, (torch.float32,))


def kia_attn_fwd_bwd_static(q, k, v, dO, o, dq, dk, dv, K, calib, tau, recon, ste, detach,
                            causal, stream=None):
    """Forward and backward in one call with the statistics in the
    library's static device scratch (no stats buffer, nothing allocated):
    q, k, v, dO in, o, dq, dk, dv out, all [B,H,T,d] float32 on the device.
    Calls that overlap on one GPU race (one array per GPU)."""
    import torch
    f32 = (torch.float32,)
    shape = _same(q, [(n, x, f32) for n, x in (("k", k), ("v", v), ("dO", dO), ("o", o),
                                                ("dq", dq), ("dk", dk), ("dv", dv))])
    B, H, T, d = shape
    _check(load().kia_attn_fwd_bwd_static(*(_ptr(x, f32) for x in (q, k, v, dO, o, dq, dk, dv)),
                                          B, H, T, d, int(K), _enum(calib, CALIB), float(tau),
                                          _enum(recon, RECON), _enum(ste, STE), _grad(detach),
                                          int(bool(causal)), _stream(stream)))


def kia_attn_fwd_bf16o(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal,
                       stream=None):
    """bf16-output forward: q, k, v and o torch.bfloat16 (o the nearest-even
    rounding of the fp32 output)."""
    import torch
    _fwd(load().kia_attn_fwd_bf16o, q, k, v, o, stats, K, calib, tau, recon, ste, detach,
         causal, stream, torch.bfloat16, (torch.bfloat16,))


def kia_attn_bwd_bf16o(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste,
                       detach, causal, stream=None):
    """bf16-output backward: every tensor torch.bfloat16; stats of at least
    kia_stats_bytes_bf16o bytes (its last field accumulates dQ, dK in fp32)."""
    import torch
    _bwd(load().kia_attn_bwd_bf16o, q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon,
         ste, detach, causal, stream, torch.bfloat16, (torch.bfloat16,),
         nbytes=kia_stats_bytes_bf16o)


def _codes(fn, q, k, stats, codes, K, calib, tau, recon, causal, stream, in_dtype):
    import torch
    shape = _same(q, [("k", k, (in_dtype,))])
    B, H, T, d = shape
    if tuple(codes.shape) != (B, H, T, T) or codes.dtype not in (torch.int16, torch.uint16):
        raise KiaError(f"codes must be [B,H,T,T] int16/uint16, got {tuple(codes.shape)} "
                       f"{codes.dtype}")
    _check_stats(stats, q, shape, _enum(recon, RECON), 0, causal)
    flags = _op_flags(shape, K, calib, tau, recon, 0, causal, in_dtype)
    _check_forward(stats, flags, ("shape", "causal", "input", "recon", "K", "calib", "tau"))
    ip = (in_dtype,)
    _check(fn(_ptr(q, ip), _ptr(k, ip), _ptr(stats, (torch.uint8,)),
              _ptr(codes, (torch.int16, torch.uint16)), B, H, T, d, int(K),
              _enum(calib, CALIB), float(tau), _enum(recon, RECON), int(bool(causal)),
              _stream(stream)))


def kia_debug_codes(q, k, stats, codes, K, calib, tau, recon, causal, stream=None):
    """Index codes recomputed from q, k by the forward's device code."""
    import torch
    _codes(load().kia_debug_codes, q, k, stats, codes, K, calib, tau, recon, causal, stream,
           torch.float32)


def kia_debug_codes_bf16(q, k, stats, codes, K, calib, tau, recon, causal, stream=None):
    import torch
    _codes(load().kia_debug_codes_bf16, q, k, stats, codes, K, calib, tau, recon, causal,
           stream, torch.bfloat16)


def kia_debug_codes_stored(stats, codes, B, H, T, d, K, calib, tau, recon, ste, causal,
                           stream=None):
    """Code words of the decisions the forward stored in stats (field U),
    decoded without recomputing a score: codes [B,H,T,T] int16/uint16."""
    import torch
    if tuple(codes.shape) != (B, H, T, T) or codes.dtype not in (torch.int16, torch.uint16):
        raise KiaError(f"codes must be [B,H,T,T] int16/uint16, got {tuple(codes.shape)} "
                       f"{codes.dtype}")
    _check_stats(stats, codes, (B, H, T, d), _enum(recon, RECON), _enum(ste, STE), causal)
    have = _FWD_FLAGS.get(_stats_key(stats))
    if have is not None:
        flags = _op_flags((B, H, T, d), K, calib, tau, recon, ste, causal, have["input"])
        _check_forward(stats, flags)
    _check(load().kia_debug_codes_stored(_ptr(stats, (torch.uint8,)),
                                         _ptr(codes, (torch.int16, torch.uint16)), B, H, T, d,
                                         int(K), _enum(calib, CALIB), float(tau),
                                         _enum(recon, RECON), _enum(ste, STE),
                                         int(bool(causal)), _stream(stream)))


def kia_debug_scores(q, k, scores, causal, stream=None):
    """The canonical fp32 scores of every pair, scores [B,H,T,T] float32
    (0 where a key is not valid); bfloat16 q, k use the bf16 sub-tile."""
    import torch
    in_dtype = q.dtype
    if in_dtype not in (torch.float32, torch.bfloat16):
        raise KiaError(f"unexpected dtype {in_dtype}")
    shape = _same(q, [("k", k, (in_dtype,))])
    B, H, T, d = shape
    if tuple(scores.shape) != (B, H, T, T):
        raise KiaError(f"scores must be [B,H,T,T], got {tuple(scores.shape)}")
    fn = load().kia_debug_scores if in_dtype == torch.float32 else load().kia_debug_scores_bf16
    ip = (in_dtype,)
    _check(fn(_ptr(q, ip), _ptr(k, ip), _ptr(scores, (torch.float32,)), B, H, T, d,
              int(bool(causal)), _stream(stream)))


def kia_debug_score_grad(stats, g_self, cM, cm, B, H, T, d, calib, recon, ste, causal,
                         input_bf16=False, stream=None):
    """Score-gradient decomposition after a backward in mode full, max_only
    or min_only: g_self [B,H,T,T], cM and cm [B,H,T] (fp32 device tensors)."""
    import torch
    if tuple(g_self.shape) != (B, H, T, T) or tuple(cM.shape) != (B, H, T) or \
            tuple(cm.shape) != (B, H, T):
        raise KiaError("g_self must be [B,H,T,T] and cM, cm [B,H,T]")
    _check_stats(stats, g_self, (B, H, T, d), _enum(recon, RECON), _enum(ste, STE), causal)
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
    f32 = (torch.float32,)
    shape = _same(q, [("k", k, f32)])
    B, H, T, d = shape
    if tuple(out.shape) != (B, H, T, 10):
        raise KiaError(f"out must be [B,H,T,10], got {tuple(out.shape)}")
    _check_stats(stats, q, shape, _enum(recon, RECON), 0, causal)
    _check_forward(stats, _op_flags(shape, K, calib, tau, recon, 0, causal, torch.float32),
                   ("shape", "causal", "input", "recon", "K", "calib", "tau"))
    _check(load().kia_geometry_probe(_ptr(q, f32), _ptr(k, f32), _ptr(stats, (torch.uint8,)),
                                     _ptr(out, f32), B, H, T, d, int(K), _enum(calib, CALIB),
                                     float(tau), _enum(recon, RECON), int(bool(causal)),
                                     _stream(stream)))


def kia_set_grid_policy(policy) -> None:
    """Launch-shape policy: "auto" (split only grids too small to fill the
    chip), "wide" (never split) or "split" (always split)."""
    _check(load().kia_set_grid_policy(_enum(policy, GRID)))


def kia_set_deterministic(on) -> None:
    """Deterministic backward on (True) or off (False, the default): with it
    on, repeated backward calls on the same inputs give bitwise equal
    gradients (every reduction in a fixed order)."""
    if not isinstance(on, (bool, int)):
        raise KiaError("kia_set_deterministic takes a bool")
    _check(load().kia_set_deterministic(int(on)))


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
def new_stats(B, H, T, d, recon, ste, causal=True, device="cuda", bf16_out=False):
    """Caller-owned stats buffer (uint8 device tensor, 256-byte aligned);
    bf16_out sizes it for the bf16-output entry points."""
    import torch
    size = kia_stats_bytes_bf16o if bf16_out else kia_stats_bytes
    n = size(B, H, T, d, recon, ste, causal)
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


def forward(q, k, v, K, calib, tau, recon, ste="weight", detach=False, causal=True,
            out_dtype=None):
    """Allocate o and stats, run kia_attn_fwd (kia_attn_fwd_bf16 for bfloat16
    inputs; kia_attn_fwd_bf16o for out_dtype=torch.bfloat16); returns
    (o, stats)."""
    import torch
    B, H, T, d = q.shape
    b16o = out_dtype == torch.bfloat16
    o = torch.empty(q.shape, dtype=torch.bfloat16 if b16o else torch.float32, device=q.device)
    stats = new_stats(B, H, T, d, recon, ste, causal, device=q.device, bf16_out=b16o)
    if b16o:
        fwd = kia_attn_fwd_bf16o
    else:
        fwd = kia_attn_fwd_bf16 if q.dtype == torch.bfloat16 else kia_attn_fwd
    fwd(q, k, v, o, stats, K, calib, tau, recon, ste, detach, causal)
    return o, stats


def backward(q, k, v, o, dO, stats, K, calib, tau, recon, ste="weight",
             detach=False, causal=True):
    """Allocate dq, dk, dv (the dtype of o) and run kia_attn_bwd
    (kia_attn_bwd_bf16 for bfloat16 inputs, kia_attn_bwd_bf16o for a
    bfloat16 o); returns (dq, dk, dv)."""
    import torch
    dq, dk, dv = (torch.empty(q.shape, dtype=o.dtype, device=q.device) for _ in range(3))
    if o.dtype == torch.bfloat16:
        bwd = kia_attn_bwd_bf16o
    else:
        bwd = kia_attn_bwd_bf16 if q.dtype == torch.bfloat16 else kia_attn_bwd
    bwd(q, k, v, o, dO, stats, dq, dk, dv, K, calib, tau, recon, ste, detach, causal)
    return dq, dk, dv


@functools.lru_cache(maxsize=1)
def _attention_function():
    """The torch.autograd.Function over forward/backward (built on first use,
    so that importing this module does not import torch)."""
    import torch

    class KIntervalAttention(torch.autograd.Function):
        """K-interval attention as an autograd operation (the paper's
        attention operator of Sec. 3, its backward of App. B).

        Inputs q, k, v [B,H,T,d] on one device, all float32 (o and the
        gradients float32) or all bfloat16 (the bf16-output entry points: o
        and the gradients bfloat16). Non-contiguous inputs and incoming
        gradients are copied to contiguous ones; everything else runs in the
        library's kernels. The forward's stats buffer is kept for the
        backward. Not twice differentiable."""

        @staticmethod
        def forward(ctx, q, k, v, K, calib, tau, recon, ste, detach, causal):
            q, k, v = (x.contiguous() for x in (q, k, v))
            o, stats = forward(q, k, v, K, calib, tau, recon, ste, detach, causal,
                               out_dtype=_attention_out_dtype(q, k, v))
            ctx.save_for_backward(q, k, v, o, stats)
            ctx.args = (K, calib, tau, recon, ste, detach, causal)
            return o

        @staticmethod
        @torch.autograd.function.once_differentiable
        def backward(ctx, dO):
            q, k, v, o, stats = ctx.saved_tensors
            dq, dk, dv = backward(q, k, v, o, dO.contiguous(), stats, *ctx.args)
            return dq, dk, dv, None, None, None, None, None, None, None

    return KIntervalAttention


def k_interval_attention(q, k, v, K=4, calib="fwm", tau=8.0, recon="nearest", ste="prob",
                         detach=False, causal=True):
    """Differentiable K-interval attention: o = attention of q, k, v [B,H,T,d]
    (float32, or bfloat16 with bfloat16 output), with the gradients of
    loss(o) with respect to q, k and v from the library's backward. The
    arguments are those of forward(); `detach` selects the gradient mode
    (False/True, or a KIA_GRAD_* name such as "max_only"). Where no
    gradient can be taken (grad mode off, or no input requiring grad) the
    forward runs forward-only (gradient mode "none") and o is returned as
    is."""
    import torch
    out_dtype = _attention_out_dtype(q, k, v)
    if not (torch.is_grad_enabled() and any(x.requires_grad for x in (q, k, v))):
        q, k, v = (x.contiguous() for x in (q, k, v))
        return forward(q, k, v, K, calib, tau, recon, ste, "none", causal, out_dtype=out_dtype)[0]
    if _grad(detach) == GRAD["none"]:
        raise KiaError('gradient mode "none" keeps no state for a backward; '
                       "call under torch.no_grad for a forward-only pass")
    return _attention_function().apply(q, k, v, K, calib, tau, recon, ste, detach, causal)


def _attention_out_dtype(q, k, v):
    """The forward's out_dtype for the autograd operation's inputs: None
    (float32 output) for float32, bfloat16 for bfloat16; anything else
    raises."""
    import torch
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in (torch.float32, torch.bfloat16):
        raise KiaError("q, k, v must be all float32 or all bfloat16, got "
                       f"{q.dtype}, {k.dtype}, {v.dtype}")
    return torch.bfloat16 if q.dtype == torch.bfloat16 else None
