"""fp64 CPU oracle of causal K-interval attention (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path never does: it shares
no code with ``paper_2609_33591_amd`` and neither imports the other.

The arithmetic lives in ``kia_oracle.c`` (plain C, fp64, OpenMP over rows or
(b,h) slices); this module only compiles it and marshals numpy arrays.
Passages followed: Sec. 3 (calibration, reconstruction, Eq. calgrad, Eq. full,
Eq. wste, Eq. pste), App. A (operator definitions, edge-case table, the
softmax operator), App. B (gradient derivations) and App. D (reduced-precision
exponential baselines) of the paper.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kia_oracle.c")
_LIB = os.path.join(_HERE, "libkia_oracle.so")

# calibrations; "resolved" is the tail-policy diagnostic of the appendix (FWM's
# step and origin, the grid continued below -tau, no zero tail)
CALIB = {"minmax": 0, "fwm": 1, "resolved": 2}
# K-interval reconstructions, then the exponential weight functions (exact
# softmax, BF16-exp, FP8-rounded exp), which ignore K, calib and ste
RECON = {"lerp": 0, "nearest": 1, "softmax": 2, "bf16_exp": 3, "fp8_exp": 4}
EXP_MODES = ("softmax", "bf16_exp", "fp8_exp")
STE = {"weight": 0, "prob": 1}
# gradient modes: full, detach, single extremum channel, detach + P1
GRAD = {"full": 0, "detach": 1, "max_only": 2, "min_only": 3, "p1": 4}


def _grad(mode) -> int:
    """False/True (full/detach), a GRAD name, or its integer code."""
    if isinstance(mode, str):
        return GRAD[mode]
    if isinstance(mode, (bool, np.bool_)):
        return int(bool(mode))
    return int(mode)

# Column meaning of the per-row record (``info``), matching kia_oracle.c.
RI = dict(M=0, m=1, amax=2, nmax=3, amin=4, nmin=5, degen=6, h=7, WN=8, WL=9,
          W=10, cM=11, cm=12, sself=13, nvalid=14)
ROWINFO = 16


def build(force: bool = True) -> str:
    """Compile kia_oracle.c into libkia_oracle.so (gcc, fp64, no contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", "-shared", "-fPIC", _SRC,
               "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        up = ctypes.POINTER(ctypes.c_uint16)
        c_int, c_double = ctypes.c_int, ctypes.c_double
        lib.kio_row.argtypes = [c_int, dp, dp, c_int, c_int, c_double, c_int,
                                c_int, c_int, dp, dp, dp, ip, ip, ip, dp, dp, dp]
        lib.kio_row.restype = c_int
        fp = ctypes.POINTER(ctypes.c_float)
        lib.kio_attn_fwd.argtypes = [dp, dp, dp, dp, dp, dp, up] + [c_int] * 6 + \
            [c_double, c_int, c_int, c_int, c_int, c_int, fp]
        lib.kio_attn_fwd.restype = c_int
        lib.kio_attn_bwd.argtypes = [dp, dp, dp, dp, dp, dp, dp, dp, dp] + \
            [c_int] * 6 + [c_double] + [c_int] * 7 + [fp]
        lib.kio_attn_bwd.restype = c_int
        lib.kio_expw.argtypes = [c_int, ctypes.POINTER(ctypes.c_float), c_int, dp, dp, ip]
        lib.kio_expw.restype = c_int
        lib.kio_geometry.argtypes = [dp, dp, dp] + [c_int] * 6 + [c_double, c_int, c_int]
        lib.kio_geometry.restype = c_int
        lib.kio_max_threads.argtypes = []
        lib.kio_max_threads.restype = c_int
        _lib = lib
    return _lib


def _p(a, ctype=ctypes.c_double):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def row(s, g=None, K=4, calib="minmax", tau=8.0, recon="lerp", ste="weight",
        detach=False):
    """Forward (and backward if ``g`` is given) of one row of valid scores.

    Returns a dict with P, wL, wN, r, l, tail, u, dS (if g), and the row
    record fields (M, m, amax, nmax, amin, nmin, degen, h, WN, WL, W, cM, cm,
    sself) of the oracle.
    """
    lib = _load()
    s = _f64(s)
    n = s.shape[0]
    out = {k: np.zeros(n) for k in ("P", "wL", "wN", "u")}
    for k in ("r", "l", "tail"):
        out[k] = np.zeros(n, dtype=np.int32)
    info = np.zeros(ROWINFO)
    gg = None if g is None else _f64(g)
    dS = np.zeros(n) if g is not None else None
    rc = lib.kio_row(n, _p(s), _p(gg), int(K), CALIB[calib], float(tau),
                     RECON[recon], STE[ste], _grad(detach), _p(out["P"]),
                     _p(out["wL"]), _p(out["wN"]), _p(out["r"], ctypes.c_int32),
                     _p(out["l"], ctypes.c_int32),
                     _p(out["tail"], ctypes.c_int32), _p(out["u"]), _p(dS),
                     _p(info))
    if rc != 0:
        raise ValueError("kio_row rejected its arguments")
    if dS is not None:
        out["dS"] = dS
    for k, i in RI.items():
        out[k] = info[i]
    return out


def _given(scores, B, H, T):
    """Given fp32 scores [B,H,T,T] (App. A: the operator acts on rows of fp32
    scores) as a C-contiguous float32 array, or None."""
    if scores is None:
        return None
    g = np.ascontiguousarray(np.asarray(scores, dtype=np.float32))
    if g.shape != (B, H, T, T):
        raise ValueError(f"scores must be [B,H,T,T] = {(B, H, T, T)}, got {g.shape}")
    return g


def attn_fwd(q, k, v, K, calib, tau, recon, causal=True, round_scores=True,
             want_ol=False, want_codes=False, slices=None, scores=None):
    """O = P V for [B,H,T,d] inputs (any float dtype, converted exactly to fp64).

    Returns (o, info[B,H,T,16], ol or None, codes[B,H,T,T] uint16 or None).
    ``slices=(lo, hi)`` restricts work to flattened (b,h) slices [lo,hi).
    ``scores`` [B,H,T,T]: take these fp32 scores instead of forming them
    from q and k (which then serve only the products of the backward).
    """
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, T, d = q.shape
    given = _given(scores, B, H, T)
    o = np.zeros_like(q)
    ol = np.zeros_like(q) if want_ol else None
    info = np.zeros((B, H, T, ROWINFO))
    codes = np.zeros((B, H, T, T), dtype=np.uint16) if want_codes else None
    lo, hi = slices if slices is not None else (0, B * H)
    rc = lib.kio_attn_fwd(_p(q), _p(k), _p(v), _p(o), _p(ol), _p(info),
                          _p(codes, ctypes.c_uint16), B, H, T, d, int(K),
                          CALIB[calib], float(tau), RECON[recon], int(causal),
                          int(round_scores), int(lo), int(hi), _p(given, ctypes.c_float))
    if rc != 0:
        raise ValueError("kio_attn_fwd rejected its arguments")
    return o, info, ol, codes


def attn_bwd(q, k, v, dO, K, calib, tau, recon, ste, detach, causal=True,
             round_scores=True, want_dS=False, slices=None, scores=None):
    """Gradients of L = sum(dO * O) w.r.t. q, k, v ([B,H,T,d], fp64).

    Returns (dq, dk, dv, info[B,H,T,16], dS[B,H,T,T] or None). ``scores``
    as in attn_fwd.
    """
    lib = _load()
    q, k, v, dO = _f64(q), _f64(k), _f64(v), _f64(dO)
    B, H, T, d = q.shape
    given = _given(scores, B, H, T)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(q), np.zeros_like(q)
    info = np.zeros((B, H, T, ROWINFO))
    dS = np.zeros((B, H, T, T)) if want_dS else None
    lo, hi = slices if slices is not None else (0, B * H)
    rc = lib.kio_attn_bwd(_p(q), _p(k), _p(v), _p(dO), _p(dq), _p(dk), _p(dv),
                          _p(dS), _p(info), B, H, T, d, int(K), CALIB[calib],
                          float(tau), RECON[recon], STE[ste], _grad(detach),
                          int(causal), int(round_scores), int(lo), int(hi),
                          _p(given, ctypes.c_float))
    if rc != 0:
        raise ValueError("kio_attn_bwd rejected its arguments")
    return dq, dk, dv, info, dS


def expw(z, recon):
    """Exponential weight function on fp32 shifts ``z`` (array, cast to fp32).

    Returns (w, wE, code): the forward weight, the value whose derivative the
    backward uses, and the quantized weight's bit pattern (bf16 bits or the
    E4M3 byte; 0 for softmax).
    """
    lib = _load()
    z = np.ascontiguousarray(np.asarray(z, dtype=np.float32)).ravel()
    n = z.shape[0]
    w, wE = np.zeros(n), np.zeros(n)
    code = np.zeros(n, dtype=np.int32)
    rc = lib.kio_expw(n, _p(z, ctypes.c_float), RECON[recon], _p(w), _p(wE),
                      _p(code, ctypes.c_int32))
    if rc != 0:
        raise ValueError("kio_expw rejected its arguments")
    return w, wE, code


def max_threads() -> int:
    """Threads the oracle's OpenMP loops run on (omp_get_max_threads)."""
    return int(_load().kio_max_threads())


# Columns of the geometry-probe record, matching kia_oracle.c.
GEO = dict(span=0, h=1, zq001=2, qnorm=3, knorm=4, entropy=5, frac_z_lt_m6=6,
           top_mass=7, eff_buckets=8, tv=9)


def geometry(q, k, K, calib, tau, recon, causal=True):
    """Per-row geometry-probe statistics [B,H,T,10] (columns: GEO) of the
    operator's fp32 scores of q, k (any float dtype, converted to fp64)."""
    lib = _load()
    q, k = _f64(q), _f64(k)
    B, H, T, d = q.shape
    out = np.zeros((B, H, T, len(GEO)))
    rc = lib.kio_geometry(_p(q), _p(k), _p(out), B, H, T, d, int(K), CALIB[calib],
                          float(tau), RECON[recon], int(causal))
    if rc != 0:
        raise ValueError("kio_geometry rejected its arguments")
    return out
