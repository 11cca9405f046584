"""rlcs: RL credit-assignment scans for AMD MI355X (gfx950).

Thin PyTorch binding over the C ABI of ``include/rlcs.h``: every function below checks its
tensors, passes their device pointers, sizes and the current HIP stream to the function of the
same name in ``librlcs.so``, and returns the output tensors. All arithmetic runs in the HIP
kernels; there is no other code path.

Tensors: data inputs are ``[N, T]`` contiguous float32 or bfloat16 (all of one call share the
dtype), flags are ``[N, T]`` uint8 or bool, ``boot`` / ``carry`` are ``[N]`` of the data dtype,
outputs are float32 ``[N, T]`` (allocated when not given). All tensors must live on the same
GPU. ``ws`` is an optional zero-initialised uint8 workspace (see ``make_workspace``).
"""
from __future__ import annotations

import contextlib
from typing import Optional, Tuple

import torch

from . import _native
from ._native import RlcsError

__all__ = [
    "rlcs_gae", "rlcs_vtrace", "rlcs_retrace", "rlcs_retrace_full", "rlcs_td_lambda", "rlcs_discounted",
    "rlcs_elig_trace", "rlcs_episodic_prefix", "rlcs_affine_scan", "rlcs_workspace_size",
    "rlcs_version", "testing_set_variant", "make_workspace", "RlcsError",
    "rlcs_gae_strided", "rlcs_vtrace_strided", "rlcs_retrace_strided", "rlcs_td_lambda_strided",
    "rlcs_discounted_strided", "rlcs_elig_trace_strided", "rlcs_episodic_prefix_strided",
    "rlcs_elig_trace_vec",
    "rlcs_workspace_size_columns", "make_workspace_columns", "rlcs_gae_masked",
    "rlcs_workspace_size_masked", "rlcs_gae_masked_noalloc",
]

_DTYPES = {torch.float32: _native.RLCS_F32, torch.bfloat16: _native.RLCS_BF16}


def _dev(t: torch.Tensor) -> torch.device:
    return t.device


def _check_data(name, t, N, T, dtype, device, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    exp = shape if shape is not None else (N, T)
    if tuple(t.shape) != tuple(exp):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(exp)}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype} like the other data inputs")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _check_flags(name, t, N, T, device):
    if t is None:
        return None
    if t.dtype not in (torch.uint8, torch.bool):
        raise TypeError(f"{name} must be uint8 or bool, got {t.dtype}")
    if tuple(t.shape) != (N, T):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {(N, T)}")
    if t.device != device or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous tensor on {device}")
    return t


def _out(name, t, N, T, device):
    if t is None:
        return torch.empty((N, T), dtype=torch.float32, device=device)
    if t.dtype != torch.float32 or tuple(t.shape) != (N, T) or t.device != device \
            or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 [N, T] tensor on {device}")
    return t


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _ws(ws: Optional[torch.Tensor], device):
    if ws is None:
        return None, 0
    if ws.device != device or not ws.is_contiguous():
        raise ValueError(f"ws must be a contiguous tensor on {device}")
    return ws.data_ptr(), ws.numel() * ws.element_size()


def _prep(x: torch.Tensor):
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("data inputs must be 2-D [N, T] tensors")
    if x.dtype not in _DTYPES:
        raise TypeError(f"data inputs must be float32 or bfloat16, got {x.dtype}")
    if x.device.type != "cuda":
        raise ValueError("tensors must be on a GPU")
    N, T = x.shape
    return int(N), int(T), x.dtype, x.device


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(device):
    """The current HIP stream of `device` as a raw handle (the direct accessor when this
    PyTorch has it: building a Stream object costs more than the kernel launch)."""
    if _raw_stream is not None:
        return _raw_stream(device.index)
    return torch.cuda.current_stream(device).cuda_stream


_SAME_DEVICE = contextlib.nullcontext()


def _on(device):
    """Context that makes `device` current for the call (nothing to do when it already is)."""
    return _SAME_DEVICE if device.index == torch.cuda.current_device() else torch.cuda.device(device)


def _call(fn: str, *args):
    code = getattr(_native.load(), fn)(*args)
    if code != _native.RLCS_OK:
        raise RlcsError(fn, code)


def make_workspace(N: int, T: int, device) -> torch.Tensor:
    """Zero-filled workspace for calls of shape [N, T] (lets long rows span workgroups)."""
    n = int(_native.load().rlcs_workspace_size(int(N), int(T)))
    return torch.zeros(max(n, 64), dtype=torch.uint8, device=device)


def rlcs_workspace_size(N: int, T: int) -> int:
    return int(_native.load().rlcs_workspace_size(int(N), int(T)))


def rlcs_version() -> int:
    return int(_native.load().rlcs_version())


def testing_set_variant(variant: int) -> None:
    """Test hook: force a kernel variant for this thread's later calls (0 = automatic)."""
    _call("rlcs_testing_set_variant", int(variant))


def rlcs_gae(r, v, term=None, trunc=None, bv=None, boot=None, adv=None, ret=None, *,
             gamma: float, lam: float, ws=None, want_ret: bool = True) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    N, T, dt, dev = _prep(r)
    _check_data("v", v, N, T, dt, dev); _check_data("bv", bv, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    adv = _out("adv", adv, N, T, dev)
    ret = _out("ret", ret, N, T, dev) if (want_ret or ret is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_gae", _ptr(r), _ptr(v), _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot),
              _ptr(adv), _ptr(ret), N, T, gamma, lam, _DTYPES[dt], wp, wb, _stream(dev))
    return adv, ret


def rlcs_vtrace(r, v, log_rho, term=None, trunc=None, bv=None, boot=None, vs=None, pg=None, *,
                gamma: float, rho_bar: float = 1.0, c_bar: float = 1.0, ws=None,
                want_pg: bool = True):
    N, T, dt, dev = _prep(r)
    _check_data("v", v, N, T, dt, dev); _check_data("log_rho", log_rho, N, T, dt, dev)
    _check_data("bv", bv, N, T, dt, dev); _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    vs = _out("vs", vs, N, T, dev)
    pg = _out("pg", pg, N, T, dev) if (want_pg or pg is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_vtrace", _ptr(r), _ptr(v), _ptr(log_rho), _ptr(term), _ptr(trunc), _ptr(bv),
              _ptr(boot), _ptr(vs), _ptr(pg), N, T, gamma, rho_bar, c_bar, _DTYPES[dt], wp, wb,
              _stream(dev))
    return vs, pg


def rlcs_retrace(r, q, eq, log_rho, term=None, trunc=None, bv=None, boot=None, delta=None,
                 q_ret=None, *, gamma: float, lam: float, c_bar: float = 1.0, ws=None,
                 want_q_ret: bool = True):
    N, T, dt, dev = _prep(r)
    for name, t in (("q", q), ("eq", eq), ("log_rho", log_rho), ("bv", bv)):
        _check_data(name, t, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    delta = _out("delta", delta, N, T, dev)
    q_ret = _out("q_ret", q_ret, N, T, dev) if (want_q_ret or q_ret is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_retrace", _ptr(r), _ptr(q), _ptr(eq), _ptr(log_rho), _ptr(term), _ptr(trunc),
              _ptr(bv), _ptr(boot), _ptr(delta), _ptr(q_ret), N, T, gamma, lam, c_bar,
              _DTYPES[dt], wp, wb, _stream(dev))
    return delta, q_ret


def rlcs_retrace_full(r, q, pi, actions, mu, term=None, trunc=None, bv=None, boot=None,
                      delta=None, q_ret=None, *, gamma: float, lam: float, c_bar: float = 1.0,
                      want_q_ret: bool = True, ws=None):
    """Full-form Retrace: q, pi [N, T, A] (data dtype), actions int32 [N, T], mu [N, T]. With a
    zero-filled `ws` of at least 64 bytes, a call that meets an action outside [0, A) sets the
    int32 at byte 8 of `ws` to 2 (the step takes Q and pi as 0)."""
    N, T, dt, dev = _prep(r)
    if not isinstance(q, torch.Tensor) or q.dim() != 3 or tuple(q.shape[:2]) != (N, T):
        raise ValueError("q must be a [N, T, A] tensor")
    A = int(q.shape[2])
    _check_data("q", q, N, T, dt, dev, shape=(N, T, A))
    _check_data("pi", pi, N, T, dt, dev, shape=(N, T, A))
    _check_data("mu", mu, N, T, dt, dev); _check_data("bv", bv, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    if not isinstance(actions, torch.Tensor) or actions.dtype != torch.int32 \
            or tuple(actions.shape) != (N, T) or actions.device != dev or not actions.is_contiguous():
        raise ValueError(f"actions must be a contiguous int32 [N, T] tensor on {dev}")
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    delta = _out("delta", delta, N, T, dev)
    q_ret = _out("q_ret", q_ret, N, T, dev) if (want_q_ret or q_ret is not None) else None
    with _on(dev):
        _call("rlcs_retrace_full", _ptr(r), _ptr(q), _ptr(pi), _ptr(actions), _ptr(mu),
              _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot), _ptr(delta), _ptr(q_ret), N, T, A,
              gamma, lam, c_bar, _DTYPES[dt], *_ws(ws, dev), _stream(dev))
    return delta, q_ret


def rlcs_td_lambda(r, v, term=None, trunc=None, bv=None, boot=None, ret=None, *, gamma: float,
                   lam: float, ws=None) -> torch.Tensor:
    N, T, dt, dev = _prep(r)
    _check_data("v", v, N, T, dt, dev); _check_data("bv", bv, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    ret = _out("ret", ret, N, T, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_td_lambda", _ptr(r), _ptr(v), _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot),
              _ptr(ret), N, T, gamma, lam, _DTYPES[dt], wp, wb, _stream(dev))
    return ret


def rlcs_discounted(r, term=None, trunc=None, bv=None, boot=None, ret=None, *, gamma: float,
                    ws=None) -> torch.Tensor:
    N, T, dt, dev = _prep(r)
    _check_data("bv", bv, N, T, dt, dev); _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    ret = _out("ret", ret, N, T, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_discounted", _ptr(r), _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot), _ptr(ret),
              N, T, gamma, _DTYPES[dt], wp, wb, _stream(dev))
    return ret


def rlcs_elig_trace(x, term=None, trunc=None, z=None, *, gamma: float, lam: float,
                    ws=None) -> torch.Tensor:
    N, T, dt, dev = _prep(x)
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    z = _out("z", z, N, T, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_elig_trace", _ptr(x), _ptr(term), _ptr(trunc), _ptr(z), N, T, gamma, lam,
              _DTYPES[dt], wp, wb, _stream(dev))
    return z


def rlcs_episodic_prefix(x, term=None, trunc=None, c=None, *, boundary: str = "ends_at",
                         ws=None) -> torch.Tensor:
    N, T, dt, dev = _prep(x)
    if boundary not in ("ends_at", "starts_at"):
        raise ValueError(f"boundary must be 'ends_at' or 'starts_at', got {boundary!r}")
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    c = _out("c", c, N, T, dev)
    wp, wb = _ws(ws, dev)
    b = _native.RLCS_STARTS_AT if boundary == "starts_at" else _native.RLCS_ENDS_AT
    with _on(dev):
        _call("rlcs_episodic_prefix", _ptr(x), _ptr(term), _ptr(trunc), _ptr(c), N, T, b,
              _DTYPES[dt], wp, wb, _stream(dev))
    return c


def rlcs_affine_scan(alpha, beta, carry=None, out=None, *, reverse: bool = True,
                     ws=None) -> torch.Tensor:
    N, T, dt, dev = _prep(alpha)
    _check_data("beta", beta, N, T, dt, dev); _check_data("carry", carry, N, T, dt, dev, shape=(N,))
    out = _out("out", out, N, T, dev)
    wp, wb = _ws(ws, dev)
    d = _native.RLCS_BACKWARD if reverse else _native.RLCS_FORWARD
    with _on(dev):
        _call("rlcs_affine_scan", _ptr(alpha), _ptr(beta), _ptr(carry), _ptr(out), N, T, d,
              _DTYPES[dt], wp, wb, _stream(dev))
    return out


# ---------------------------------------------------------------- strided layouts
# Every [N, T] tensor of the row-major functions may be any 2-D view with strides
# (stride_n, stride_t) in elements, the same for every [N, T] tensor of the call: a time-major
# [T, N] buffer is passed as its transpose ``x.t()`` (strides (1, ld)), a view of the first T
# steps of wider rows as is (strides (ld, 1)). Outputs not given are allocated with the inputs'
# strides.

def _strides(t: torch.Tensor):
    """(stride_n, stride_t) of a 2-D view, with the stride of a size-1 dimension chosen so that
    the dimensions nest (it never multiplies an index other than 0)."""
    N, T = int(t.shape[0]), int(t.shape[1])
    sn, st = int(t.stride(0)), int(t.stride(1))
    if T == 1:
        st = max(1, N * max(sn, 1))
    if N == 1:
        sn = max(1, T * max(st, 1))
    return sn, st


def _prep_strided(x: torch.Tensor):
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("data inputs must be 2-D [N, T] tensors")
    if x.dtype not in _DTYPES:
        raise TypeError(f"data inputs must be float32 or bfloat16, got {x.dtype}")
    if x.device.type != "cuda":
        raise ValueError("tensors must be on a GPU")
    N, T = int(x.shape[0]), int(x.shape[1])
    sn, st = _strides(x)
    return N, T, sn, st, x.dtype, x.device


def _check_strided(name, t, N, T, sn, st, device, dtype=None, flags=False):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if tuple(t.shape) != (N, T):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {(N, T)}")
    if flags:
        if t.dtype not in (torch.uint8, torch.bool):
            raise TypeError(f"{name} must be uint8 or bool, got {t.dtype}")
    elif dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if _strides(t) != (sn, st):
        raise ValueError(f"{name} has strides {t.stride()}, expected ({sn}, {st}) like the first input")
    return t


def _out_strided(name, t, N, T, sn, st, device):
    if t is None:
        return torch.empty_strided((N, T), (sn, st), dtype=torch.float32, device=device)
    if t.dtype != torch.float32:
        raise ValueError(f"{name} must be float32")
    return _check_strided(name, t, N, T, sn, st, device)


def _boot_strided(boot, N, dtype, device):
    return _check_data("boot", boot, 1, N, dtype, device, shape=(N,))


def make_workspace_columns(columns: int, T: int, device) -> torch.Tensor:
    """Zero-filled workspace for strided calls (columns = N) and rlcs_elig_trace_vec
    (columns = N * F) over T steps."""
    n = int(_native.load().rlcs_workspace_size_columns(int(columns), int(T)))
    return torch.zeros(max(n, 64), dtype=torch.uint8, device=device)


def rlcs_workspace_size_columns(columns: int, T: int) -> int:
    return int(_native.load().rlcs_workspace_size_columns(int(columns), int(T)))


def rlcs_gae_strided(r, v, term=None, trunc=None, bv=None, boot=None, adv=None, ret=None, *,
                     gamma: float, lam: float, ws=None, want_ret: bool = True):
    N, T, sn, st, dt, dev = _prep_strided(r)
    _check_strided("v", v, N, T, sn, st, dev, dt); _check_strided("bv", bv, N, T, sn, st, dev, dt)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    _boot_strided(boot, N, dt, dev)
    adv = _out_strided("adv", adv, N, T, sn, st, dev)
    ret = _out_strided("ret", ret, N, T, sn, st, dev) if (want_ret or ret is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_gae_strided", _ptr(r), _ptr(v), _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot),
              _ptr(adv), _ptr(ret), N, T, sn, st, gamma, lam, _DTYPES[dt], wp, wb, _stream(dev))
    return adv, ret


def rlcs_vtrace_strided(r, v, log_rho, term=None, trunc=None, bv=None, boot=None, vs=None,
                        pg=None, *, gamma: float, rho_bar: float = 1.0, c_bar: float = 1.0,
                        ws=None, want_pg: bool = True):
    N, T, sn, st, dt, dev = _prep_strided(r)
    for name, t in (("v", v), ("log_rho", log_rho), ("bv", bv)):
        _check_strided(name, t, N, T, sn, st, dev, dt)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    _boot_strided(boot, N, dt, dev)
    vs = _out_strided("vs", vs, N, T, sn, st, dev)
    pg = _out_strided("pg", pg, N, T, sn, st, dev) if (want_pg or pg is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_vtrace_strided", _ptr(r), _ptr(v), _ptr(log_rho), _ptr(term), _ptr(trunc),
              _ptr(bv), _ptr(boot), _ptr(vs), _ptr(pg), N, T, sn, st, gamma, rho_bar, c_bar,
              _DTYPES[dt], wp, wb, _stream(dev))
    return vs, pg


def rlcs_retrace_strided(r, q, eq, log_rho, term=None, trunc=None, bv=None, boot=None,
                         delta=None, q_ret=None, *, gamma: float, lam: float, c_bar: float = 1.0,
                         ws=None, want_q_ret: bool = True):
    N, T, sn, st, dt, dev = _prep_strided(r)
    for name, t in (("q", q), ("eq", eq), ("log_rho", log_rho), ("bv", bv)):
        _check_strided(name, t, N, T, sn, st, dev, dt)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    _boot_strided(boot, N, dt, dev)
    delta = _out_strided("delta", delta, N, T, sn, st, dev)
    q_ret = _out_strided("q_ret", q_ret, N, T, sn, st, dev) if (want_q_ret or q_ret is not None) else None
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_retrace_strided", _ptr(r), _ptr(q), _ptr(eq), _ptr(log_rho), _ptr(term),
              _ptr(trunc), _ptr(bv), _ptr(boot), _ptr(delta), _ptr(q_ret), N, T, sn, st, gamma,
              lam, c_bar, _DTYPES[dt], wp, wb, _stream(dev))
    return delta, q_ret


def rlcs_td_lambda_strided(r, v, term=None, trunc=None, bv=None, boot=None, ret=None, *,
                           gamma: float, lam: float, ws=None) -> torch.Tensor:
    N, T, sn, st, dt, dev = _prep_strided(r)
    _check_strided("v", v, N, T, sn, st, dev, dt); _check_strided("bv", bv, N, T, sn, st, dev, dt)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    _boot_strided(boot, N, dt, dev)
    ret = _out_strided("ret", ret, N, T, sn, st, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_td_lambda_strided", _ptr(r), _ptr(v), _ptr(term), _ptr(trunc), _ptr(bv),
              _ptr(boot), _ptr(ret), N, T, sn, st, gamma, lam, _DTYPES[dt], wp, wb, _stream(dev))
    return ret


def rlcs_discounted_strided(r, term=None, trunc=None, bv=None, boot=None, ret=None, *,
                            gamma: float, ws=None) -> torch.Tensor:
    N, T, sn, st, dt, dev = _prep_strided(r)
    _check_strided("bv", bv, N, T, sn, st, dev, dt)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    _boot_strided(boot, N, dt, dev)
    ret = _out_strided("ret", ret, N, T, sn, st, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_discounted_strided", _ptr(r), _ptr(term), _ptr(trunc), _ptr(bv), _ptr(boot),
              _ptr(ret), N, T, sn, st, gamma, _DTYPES[dt], wp, wb, _stream(dev))
    return ret


def rlcs_elig_trace_strided(x, term=None, trunc=None, z=None, *, gamma: float, lam: float,
                            ws=None) -> torch.Tensor:
    N, T, sn, st, dt, dev = _prep_strided(x)
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    z = _out_strided("z", z, N, T, sn, st, dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_elig_trace_strided", _ptr(x), _ptr(term), _ptr(trunc), _ptr(z), N, T, sn, st,
              gamma, lam, _DTYPES[dt], wp, wb, _stream(dev))
    return z


def rlcs_episodic_prefix_strided(x, term=None, trunc=None, c=None, *, boundary: str = "ends_at",
                                 ws=None) -> torch.Tensor:
    N, T, sn, st, dt, dev = _prep_strided(x)
    if boundary not in ("ends_at", "starts_at"):
        raise ValueError(f"boundary must be 'ends_at' or 'starts_at', got {boundary!r}")
    _check_strided("term", term, N, T, sn, st, dev, flags=True)
    _check_strided("trunc", trunc, N, T, sn, st, dev, flags=True)
    c = _out_strided("c", c, N, T, sn, st, dev)
    wp, wb = _ws(ws, dev)
    b = _native.RLCS_STARTS_AT if boundary == "starts_at" else _native.RLCS_ENDS_AT
    with _on(dev):
        _call("rlcs_episodic_prefix_strided", _ptr(x), _ptr(term), _ptr(trunc), _ptr(c), N, T, sn,
              st, b, _DTYPES[dt], wp, wb, _stream(dev))
    return c


# ---------------------------------------------------------------- vector eligibility traces

def rlcs_elig_trace_vec(x, term=None, trunc=None, z=None, *, gamma: float, lam: float,
                        ws=None) -> torch.Tensor:
    """x: contiguous [N, T, F] float32 / bfloat16; flags [N, T]; returns float32 z [N, T, F]."""
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError("x must be a 3-D [N, T, F] tensor")
    if x.dtype not in _DTYPES:
        raise TypeError(f"x must be float32 or bfloat16, got {x.dtype}")
    if x.device.type != "cuda" or not x.is_contiguous():
        raise ValueError("x must be a contiguous tensor on a GPU")
    N, T, F = (int(s) for s in x.shape)
    dev = x.device
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    if z is None:
        z = torch.empty((N, T, F), dtype=torch.float32, device=dev)
    elif z.dtype != torch.float32 or tuple(z.shape) != (N, T, F) or z.device != dev \
            or not z.is_contiguous():
        raise ValueError(f"z must be a contiguous float32 [N, T, F] tensor on {dev}")
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_elig_trace_vec", _ptr(x), _ptr(term), _ptr(trunc), _ptr(z), N, T, F, gamma,
              lam, _DTYPES[x.dtype], wp, wb, _stream(dev))
    return z


# ---------------------------------------------------------------- masked GAE

def rlcs_workspace_size_masked(N: int, T: int) -> int:
    return int(_native.load().rlcs_workspace_size_masked(int(N), int(T)))


def rlcs_gae_masked(r, v, mask=None, term=None, trunc=None, bv=None, boot=None, adv=None,
                    ret=None, *, gamma: float, lam: float, normalize: bool = False,
                    eps: float = 1e-8, ws=None, want_ret: bool = True):
    """GAE with observation-skip masking (mask nonzero = the step takes part), optionally with
    the advantages whitened over the steps that take part. A zero-filled workspace for
    whitening is allocated when none is given (a workspace passed in must have been zero-filled
    before its first use)."""
    N, T, dt, dev = _prep(r)
    _check_data("v", v, N, T, dt, dev); _check_data("bv", bv, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("mask", mask, N, T, dev)
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    adv = _out("adv", adv, N, T, dev)
    ret = _out("ret", ret, N, T, dev) if (want_ret or ret is not None) else None
    if normalize and ws is None:
        ws = torch.zeros(max(rlcs_workspace_size_masked(N, T), 64), dtype=torch.uint8, device=dev)
    wp, wb = _ws(ws, dev)
    with _on(dev):
        _call("rlcs_gae_masked", _ptr(r), _ptr(v), _ptr(mask), _ptr(term), _ptr(trunc), _ptr(bv),
              _ptr(boot), _ptr(adv), _ptr(ret), N, T, gamma, lam, 1 if normalize else 0, eps,
              _DTYPES[dt], wp, wb, _stream(dev))
    return adv, ret


def rlcs_gae_masked_noalloc(r, v, mask=None, term=None, trunc=None, bv=None, boot=None, adv=None,
                            ret=None, *, gamma: float, lam: float, normalize: bool = False,
                            eps: float = 1e-8, want_ret: bool = True):
    """rlcs_gae_masked with the library's built-in whitening workspace (N <= 65536): the C call
    allocates nothing. Pass `adv` (and `ret`) to keep this wrapper from allocating them."""
    N, T, dt, dev = _prep(r)
    _check_data("v", v, N, T, dt, dev); _check_data("bv", bv, N, T, dt, dev)
    _check_data("boot", boot, N, T, dt, dev, shape=(N,))
    _check_flags("mask", mask, N, T, dev)
    _check_flags("term", term, N, T, dev); _check_flags("trunc", trunc, N, T, dev)
    adv = _out("adv", adv, N, T, dev)
    ret = _out("ret", ret, N, T, dev) if (want_ret or ret is not None) else None
    with _on(dev):
        _call("rlcs_gae_masked_noalloc", _ptr(r), _ptr(v), _ptr(mask), _ptr(term), _ptr(trunc),
              _ptr(bv), _ptr(boot), _ptr(adv), _ptr(ret), N, T, gamma, lam, 1 if normalize else 0,
              eps, _DTYPES[dt], _stream(dev))
    return adv, ret
