"""fp64 CPU oracle for the seven credit-assignment estimators.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package. The GPU library never loads it, and it shares no
code with the GPU library.

The arithmetic lives in ``rlcs_oracle.c`` (sequential recurrences, one step at a time, in
fp64). This module only widens the inputs to fp64 and marshals them through ctypes:
float32 arrays are widened exactly, and uint16 arrays are read as bfloat16 bit patterns and
widened exactly. Scalar parameters are taken as float32 first (the precision the GPU entry
points receive) and then widened.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "rlcs_oracle.c")
_HDR = os.path.join(_HERE, "rlcs_oracle.h")
_LIB = os.path.join(_HERE, "liboracle.so")

__all__ = [
    "build", "gae", "td_lambda", "discounted", "vtrace", "retrace", "retrace_full", "elig_trace",
    "elig_trace_vec", "gae_masked", "normalize_advantages", "episodic_prefix", "affine_scan",
    "time_major", "widen", "param",
]


def build(force: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (plain -O2, no FMA contraction, no fast-math): always
    when force, else only if it does not exist yet."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-shared", "-fPIC", "-Wall", "-Werror", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        D = ctypes.POINTER(ctypes.c_double)
        U8 = ctypes.POINTER(ctypes.c_uint8)
        I64, F64, INT = ctypes.c_int64, ctypes.c_double, ctypes.c_int
        sigs = {
            "oracle_gae": [D, D, U8, U8, D, D, D, D, I64, I64, F64, F64],
            "oracle_td_lambda": [D, D, U8, U8, D, D, D, I64, I64, F64, F64],
            "oracle_discounted": [D, U8, U8, D, D, D, I64, I64, F64],
            "oracle_vtrace": [D, D, D, U8, U8, D, D, D, D, I64, I64, F64, F64, F64],
            "oracle_retrace": [D, D, D, D, U8, U8, D, D, D, D, I64, I64, F64, F64, F64],
            "oracle_retrace_full": [D, D, D, ctypes.POINTER(ctypes.c_int32), D, U8, U8, D, D, D,
                                    D, I64, I64, I64, F64, F64, F64],
            "oracle_elig_trace": [D, U8, U8, D, I64, I64, F64, F64],
            "oracle_elig_trace_vec": [D, U8, U8, D, I64, I64, I64, F64, F64],
            "oracle_gae_masked": [D, D, U8, U8, U8, D, D, D, D, I64, I64, F64, F64],
            "oracle_episodic_prefix": [D, U8, U8, D, I64, I64, INT],
            "oracle_affine_scan": [D, D, D, D, I64, I64, INT],
        }
        for name, argtypes in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = argtypes
            fn.restype = None
        _lib = lib
    return _lib


def widen(a) -> Optional[np.ndarray]:
    """Exact widening to fp64: float32/float64 as is, uint16 as bfloat16 bit patterns."""
    if a is None:
        return None
    a = np.asarray(a)
    if a.dtype == np.uint16:
        a = (a.astype(np.uint32) << 16).view(np.float32)
    if a.dtype not in (np.float32, np.float64):
        raise TypeError(f"oracle data arrays must be float32, float64 or bf16 bits, got {a.dtype}")
    return np.ascontiguousarray(a, dtype=np.float64)


def param(x: float) -> float:
    """A scalar parameter as the GPU receives it: rounded to float32, then widened."""
    return float(np.float32(x))


def _flags(f) -> Optional[np.ndarray]:
    if f is None:
        return None
    f = np.asarray(f)
    if f.dtype == np.bool_:
        f = f.view(np.uint8)
    if f.dtype != np.uint8:
        raise TypeError(f"flag arrays must be uint8 or bool, got {f.dtype}")
    return np.ascontiguousarray(f)


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _shape(a):
    a = np.asarray(a)
    if a.ndim != 2:
        raise ValueError(f"expected a 2-D [N, T] array, got shape {a.shape}")
    return a.shape


def _check(N, T, *arrays):
    for a in arrays:
        if a is not None and a.size != N * T:
            raise ValueError(f"array of size {a.size} does not match [N={N}, T={T}]")


def gae(r, v, term=None, trunc=None, bv=None, boot=None, *, gamma, lam):
    """Returns (advantages, returns), both fp64 [N, T]."""
    N, T = _shape(r)
    r, v, bv, boot = widen(r), widen(v), widen(bv), widen(boot)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, v, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    adv = np.empty((N, T)); ret = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_gae(_ptr(r, D), _ptr(v, D), _ptr(term, U), _ptr(trunc, U), _ptr(bv, D),
                       _ptr(boot, D), _ptr(adv, D), _ptr(ret, D), N, T,
                       param(gamma), param(lam))
    return adv, ret


def td_lambda(r, v, term=None, trunc=None, bv=None, boot=None, *, gamma, lam):
    N, T = _shape(r)
    r, v, bv, boot = widen(r), widen(v), widen(bv), widen(boot)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, v, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    out = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_td_lambda(_ptr(r, D), _ptr(v, D), _ptr(term, U), _ptr(trunc, U), _ptr(bv, D),
                             _ptr(boot, D), _ptr(out, D), N, T, param(gamma), param(lam))
    return out


def discounted(r, term=None, trunc=None, bv=None, boot=None, *, gamma):
    N, T = _shape(r)
    r, bv, boot = widen(r), widen(bv), widen(boot)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    out = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_discounted(_ptr(r, D), _ptr(term, U), _ptr(trunc, U), _ptr(bv, D),
                              _ptr(boot, D), _ptr(out, D), N, T, param(gamma))
    return out


def vtrace(r, v, log_rho, term=None, trunc=None, bv=None, boot=None, *, gamma,
           rho_bar=1.0, c_bar=1.0):
    """Returns (vs, pg), both fp64 [N, T]."""
    N, T = _shape(r)
    r, v, log_rho, bv, boot = widen(r), widen(v), widen(log_rho), widen(bv), widen(boot)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, v, log_rho, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    vs = np.empty((N, T)); pg = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_vtrace(_ptr(r, D), _ptr(v, D), _ptr(log_rho, D), _ptr(term, U),
                          _ptr(trunc, U), _ptr(bv, D), _ptr(boot, D), _ptr(vs, D), _ptr(pg, D),
                          N, T, param(gamma), param(rho_bar), param(c_bar))
    return vs, pg


def retrace(r, q, eq, log_rho, term=None, trunc=None, bv=None, boot=None, *, gamma, lam,
            c_bar=1.0):
    """Returns (delta, q_ret), both fp64 [N, T]."""
    N, T = _shape(r)
    r, q, eq, log_rho = widen(r), widen(q), widen(eq), widen(log_rho)
    bv, boot = widen(bv), widen(boot)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, q, eq, log_rho, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    delta = np.empty((N, T)); q_ret = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_retrace(_ptr(r, D), _ptr(q, D), _ptr(eq, D), _ptr(log_rho, D),
                           _ptr(term, U), _ptr(trunc, U), _ptr(bv, D), _ptr(boot, D),
                           _ptr(delta, D), _ptr(q_ret, D), N, T,
                           param(gamma), param(lam), param(c_bar))
    return delta, q_ret


def retrace_full(r, q, pi, actions, mu, term=None, trunc=None, bv=None, boot=None, *, gamma,
                 lam, c_bar=1.0):
    """Full-form Retrace: q and pi are [N, T, A], actions int32 [N, T], mu [N, T] (behaviour
    probability of the taken action). Returns (delta, q_ret), both fp64 [N, T]."""
    N, T = _shape(r)
    q3 = np.asarray(q)
    if q3.ndim != 3 or q3.shape[:2] != (N, T) or np.asarray(pi).shape != q3.shape:
        raise ValueError("q and pi must be [N, T, A] arrays matching r")
    A = q3.shape[2]
    r, q3, pi3, mu, bv, boot = widen(r), widen(q3), widen(pi), widen(mu), widen(bv), widen(boot)
    act = np.ascontiguousarray(actions, dtype=np.int32)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, mu, act, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    delta = np.empty((N, T)); q_ret = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_retrace_full(_ptr(r, D), _ptr(q3, D), _ptr(pi3, D), _ptr(act, ctypes.c_int32),
                                _ptr(mu, D), _ptr(term, U), _ptr(trunc, U), _ptr(bv, D),
                                _ptr(boot, D), _ptr(delta, D), _ptr(q_ret, D), N, T, A,
                                param(gamma), param(lam), param(c_bar))
    return delta, q_ret


def elig_trace(x, term=None, trunc=None, *, gamma, lam):
    N, T = _shape(x)
    x = widen(x)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, term, trunc)
    out = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_elig_trace(_ptr(x, D), _ptr(term, U), _ptr(trunc, U), _ptr(out, D), N, T,
                              param(gamma), param(lam))
    return out


def elig_trace_vec(x, term=None, trunc=None, *, gamma, lam):
    """Eligibility traces of F-vectors: x is [N, T, F], the flags [N, T]. Returns fp64 z
    [N, T, F]."""
    x3 = np.asarray(x)
    if x3.ndim != 3:
        raise ValueError(f"expected a 3-D [N, T, F] array, got shape {x3.shape}")
    N, T, F = x3.shape
    x3 = widen(x3)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, term, trunc)
    out = np.empty((N, T, F))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_elig_trace_vec(_ptr(x3, D), _ptr(term, U), _ptr(trunc, U), _ptr(out, D), N, T,
                                  F, param(gamma), param(lam))
    return out


def gae_masked(r, v, mask=None, term=None, trunc=None, bv=None, boot=None, *, gamma, lam):
    """GAE with observation-skip masking (see rlcs_oracle.h). Returns fp64 (adv, ret)."""
    N, T = _shape(r)
    r, v, bv, boot = widen(r), widen(v), widen(bv), widen(boot)
    mask, term, trunc = _flags(mask), _flags(term), _flags(trunc)
    _check(N, T, v, mask, term, trunc, bv)
    if trunc is not None and bv is None:
        raise ValueError("bv is required when trunc is given")
    adv = np.empty((N, T)); ret = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_gae_masked(_ptr(r, D), _ptr(v, D), _ptr(mask, U), _ptr(term, U), _ptr(trunc, U),
                              _ptr(bv, D), _ptr(boot, D), _ptr(adv, D), _ptr(ret, D), N, T,
                              param(gamma), param(lam))
    return adv, ret


def normalize_advantages(adv, mask=None, *, eps):
    """Whitening over the steps that take part (mask nonzero; all when mask is None):
    (adv - mean) / sqrt(var + eps) with the sample mean and the unbiased sample variance of
    those steps (variance 0 when fewer than two take part), applied to every step. fp64."""
    a = np.asarray(adv, dtype=np.float64)
    sel = a.reshape(-1) if mask is None else a[np.asarray(mask) != 0]
    n = sel.size
    mean = float(np.sum(sel)) / n if n > 0 else 0.0
    var = float(np.sum((sel - mean) ** 2)) / (n - 1) if n > 1 else 0.0
    return (a - mean) / np.sqrt(var + param(eps))


def time_major(fn, *args, **kw):
    """Estimator `fn` (one of the functions above) on time-major inputs: every 2-D argument is
    [T, N] (step t of environment n at [t, n]); 1-D arguments (bootstraps) are [N]. The oracle
    is the row-major one applied to the transposed arrays; the outputs come back as [T, N]."""
    def tr(a):
        if isinstance(a, np.ndarray) and a.ndim == 2:
            return np.ascontiguousarray(a.T)
        return a
    out = fn(*(tr(a) for a in args), **{k: tr(v) for k, v in kw.items()})
    if isinstance(out, tuple):
        return tuple(np.ascontiguousarray(o.T) for o in out)
    return np.ascontiguousarray(out.T)


def episodic_prefix(x, term=None, trunc=None, *, boundary="ends_at"):
    if boundary not in ("ends_at", "starts_at"):
        raise ValueError(f"boundary must be 'ends_at' or 'starts_at', got {boundary!r}")
    N, T = _shape(x)
    x = widen(x)
    term, trunc = _flags(term), _flags(trunc)
    _check(N, T, term, trunc)
    out = np.empty((N, T))
    D, U = ctypes.c_double, ctypes.c_uint8
    _load().oracle_episodic_prefix(_ptr(x, D), _ptr(term, U), _ptr(trunc, U), _ptr(out, D),
                                   N, T, 1 if boundary == "starts_at" else 0)
    return out


def affine_scan(alpha, beta, carry=None, *, reverse=True):
    N, T = _shape(alpha)
    alpha, beta, carry = widen(alpha), widen(beta), widen(carry)
    _check(N, T, beta)
    out = np.empty((N, T))
    D = ctypes.c_double
    _load().oracle_affine_scan(_ptr(alpha, D), _ptr(beta, D), _ptr(carry, D), _ptr(out, D),
                               N, T, 1 if reverse else 0)
    return out
