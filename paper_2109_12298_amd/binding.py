"""Thin ctypes binding of libdpgrad.so (declared in include/dpgrad.h).

Each function has the name and argument order of its C entry point and only
marshals arguments: device pointers may be given as torch tensors (their
``data_ptr()``), raw integer addresses or None; ``ws_bytes`` is taken from the
workspace tensor; ``stream`` defaults to torch's current HIP stream.  A status
other than DP_OK raises :class:`DPError`.  There is no fallback: if the
library is not built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdpgrad.so")

DP_OK, DP_EINVAL, DP_EDTYPE, DP_EUNSUPPORTED, DP_ECAP, DP_EHIP = range(6)
DP_F32, DP_BF16 = 0, 1
DP_FLAG_BAD_INDEX, DP_FLAG_NONFINITE, DP_FLAG_CAP, DP_FLAG_WAIT = 1, 2, 4, 8

# (name, restype, argtypes) of every exported entry point
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_F = ctypes.c_float
_SZ = ctypes.c_size_t
_I32 = ctypes.c_int32
_U32 = ctypes.c_uint32
_U64 = ctypes.c_uint64
_ST = ctypes.c_int

SIGNATURES = {
    "dp_status_string": (ctypes.c_char_p, [_ST]),
    "dp_abi_version": (ctypes.c_int, []),
    "dp_grad_sample_linear_workspace_bytes": (_SZ, [_I64, _I64, _I64, _I64, _ST]),
    "dp_grad_sample_linear": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _I64, _F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dp_grad_sample_linear_noalloc_max_bytes": (_SZ, []),
    "dp_grad_sample_linear_noalloc": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _I64, _F, _P, _P, _P, _P, _P]),
    "dp_grad_sample_conv2d_workspace_bytes": (_SZ, [_I64] * 11),
    "dp_grad_sample_conv2d": (_ST, [_P, _P, _ST] + [_I64] * 16 + [_F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dp_conv2d_set_path": (ctypes.c_int, [ctypes.c_int]),
    "dp_conv2d_kernel_choice": (_I32, [_I64] * 11),
    "dp_grad_sample_many_grouped": (_I32, [_P, _ST, _I64]),
    "dp_grad_sample_many_workspace_bytes": (_SZ, [_P, _I32, _ST, _I64]),
    "dp_grad_sample_many": (_ST, [_P, _I32, _ST, _I64, _P, _P, _SZ, _P]),
    "dp_grad_sample_embedding_workspace_bytes": (_SZ, [_I64, _I64]),
    "dp_grad_sample_embedding": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _I64, _F, _P, _P, _P, _I64, _P,
                                       _P, _P, _SZ, _P]),
    "dp_grad_sample_layernorm_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
    "dp_grad_sample_layernorm": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dp_grad_sample_groupnorm_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
    "dp_grad_sample_groupnorm": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dp_lstm_backward": (_ST, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _P, _P, _P]),
    "dp_per_sample_norms": (_ST, [_P, _I32, _I64, _P, _P, _P]),
    "dp_per_sample_norms_active": (_ST, [_P, _I32, _I64, _P, _P, _P, _P]),
    "dp_ghost_norm_linear_workspace_bytes": (_SZ, [_I64, _I64, _I64, _I64]),
    "dp_ghost_norm_linear": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _I64, _F, _I32, _P, _P, _P, _SZ, _P]),
    "dp_ghost_norm_linear_many_workspace_bytes": (_SZ, [_P, _I32, _I64]),
    "dp_grad_sample_layernorm_many_workspace_bytes": (_SZ, [_P, _I32, _I64, _ST]),
    "dp_grad_sample_layernorm_many": (_ST, [_P, _I32, _ST, _I64, _P, _P, _SZ, _P]),
    "dp_ghost_norm_linear_many": (_ST, [_P, _I32, _ST, _I64, _P, _P, _SZ, _P]),
    "dp_sqnorm_from_grads": (_ST, [_P, _I64, _I64, _P, _P, _P]),
    "dp_clip_factors": (_ST, [_P, _I64, _F, _P, _P, _P]),
    "dp_clip_accumulate_workspace_bytes": (_SZ, [_I64, _I64]),
    "dp_clip_accumulate": (_ST, [_P, _P, _F, _I64, _I64, _P, _P, _P, _P, _SZ, _P]),
    "dp_clip_accumulate_linear_workspace_bytes": (_SZ, [_I64, _I64, _I64, _I64, _ST]),
    "dp_clip_accumulate_linear": (_ST, [_P, _P, _ST, _I64, _I64, _I64, _I64, _F, _P, _F, _P, _P, _P, _P,
                                        _SZ, _P]),
    "dp_clip_accumulate_linear_many_workspace_bytes": (_SZ, [_P, _I32, _ST, _I64]),
    "dp_clip_accumulate_linear_many": (_ST, [_P, _I32, _ST, _I64, _P, _F, _P, _P, _SZ, _P]),
    "dp_clip_accumulate_embedding_workspace_bytes": (_SZ, [_I64, _I64]),
    "dp_clip_accumulate_embedding": (_ST, [_P, _P, _P, _I64, _P, _F, _I64, _I64, _I64, _P, _P, _P, _SZ, _P]),
    "dp_clip_noise_many_workspace_bytes": (_SZ, [_P, _I32, _I64]),
    "dp_clip_noise_many": (_ST, [_P, _I32, _I64, _P, _F, _U64, _U64, _P, _F, _F, _P, _P, _SZ, _P]),
    "dp_norms_clip_noise_workspace_bytes": (_SZ, [_P, _I32, _I64]),
    "dp_norms_clip_noise": (_ST, [_P, _I32, _P, _I32, _I64, _P, _F, _U64, _U64, _P, _F, _F, _P, _P, _SZ, _P]),
    "dp_norms_clip_noise_sched": (_ST, [_P, _I32, _P, _I32, _I64, _P, _F, _U64, _U64, _P, _P, _I64, _P, _F, _P, _P,
                                        _SZ, _P]),
    "dp_step_advance": (_ST, [_P, _U64, _P]),
    "dp_add_noise": (_ST, [_P, _P, _I64, _U64, _U64, _U32, _F, _F, _F, _P, _P]),
    "dp_philox_normals": (_ST, [_P, _P, _I64, _U64, _U64, _U32, _P]),
}


class DPParam(ctypes.Structure):
    """struct dp_param of dpgrad.h."""
    _fields_ = [("grad_sample", ctypes.c_void_p), ("sum", ctypes.c_void_p), ("out", ctypes.c_void_p),
                ("numel", ctypes.c_int64), ("param_index", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("accum", ctypes.c_void_p)]


DP_PARAM_REDUCE = 1


def make_params(entries):
    """A dp_param array from (grad_sample, sum, out, numel, param_index[, accum]) tuples.

    grad_sample None means the sum is already formed (no DP_PARAM_REDUCE);
    an empty tensor (N = 0) still asks for the reduction.  accum (optional,
    default None) is the running sum of a virtual step."""
    arr = (DPParam * max(len(entries), 1))()
    for i, ent in enumerate(entries):
        g, s, o, numel, pidx = ent[:5]
        arr[i].accum = _ptr(ent[5]) if len(ent) > 5 else None
        arr[i].grad_sample = _ptr(g)
        arr[i].sum = _ptr(s)
        arr[i].out = _ptr(o)
        arr[i].numel = int(numel)
        arr[i].param_index = int(pidx)
        arr[i].flags = DP_PARAM_REDUCE if g is not None else 0
    return arr


class DPLinearClip(ctypes.Structure):
    """struct dp_linear_clip of dpgrad.h."""
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("T", ctypes.c_int64), ("d_in", ctypes.c_int64),
                ("d_out", ctypes.c_int64), ("scale", ctypes.c_float), ("sumW", ctypes.c_void_p),
                ("sumb", ctypes.c_void_p)]


def make_linear_clips(entries):
    """A dp_linear_clip array from (A, B, T, d_in, d_out, scale, sumW, sumb) tuples."""
    arr = (DPLinearClip * max(len(entries), 1))()
    for i, (A, B, T, d_in, d_out, scale, sumW, sumb) in enumerate(entries):
        arr[i].A = _ptr(A)
        arr[i].B = _ptr(B)
        arr[i].T, arr[i].d_in, arr[i].d_out = int(T), int(d_in), int(d_out)
        arr[i].scale = float(scale)
        arr[i].sumW = _ptr(sumW)
        arr[i].sumb = _ptr(sumb)
    return arr


DP_LAYER_LINEAR, DP_LAYER_CONV2D = 0, 1


class DPLayerGrad(ctypes.Structure):
    """struct dp_layer_grad of dpgrad.h."""
    _fields_ = [("kind", ctypes.c_int32), ("A", ctypes.c_void_p), ("B", ctypes.c_void_p)] + \
               [(f, ctypes.c_int64) for f in ("T", "d_in", "d_out", "Cin", "H", "W", "Cout", "Ho", "Wo", "kh", "kw",
                                              "sh", "sw", "ph", "pw")] + \
               [("scale", ctypes.c_float), ("gW", ctypes.c_void_p), ("gb", ctypes.c_void_p),
                ("sqnorm", ctypes.c_void_p)]


def linear_grad_item(A, B, T, d_in, d_out, scale, gW, gb=None, sqnorm=None):
    """The dp_layer_grad fields of a Linear layer (a dict for make_layer_grads)."""
    return dict(kind=DP_LAYER_LINEAR, A=A, B=B, T=T, d_in=d_in, d_out=d_out, scale=scale, gW=gW, gb=gb,
                sqnorm=sqnorm)


def conv2d_grad_item(X, GY, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, scale, gW, gb=None, sqnorm=None):
    """The dp_layer_grad fields of a Conv2d layer (a dict for make_layer_grads)."""
    return dict(kind=DP_LAYER_CONV2D, A=X, B=GY, Cin=Cin, H=H, W=W, Cout=Cout, Ho=Ho, Wo=Wo, kh=kh, kw=kw, sh=sh,
                sw=sw, ph=ph, pw=pw, scale=scale, gW=gW, gb=gb, sqnorm=sqnorm)


def make_layer_grads(entries):
    """A dp_layer_grad array from linear_grad_item / conv2d_grad_item dicts."""
    arr = (DPLayerGrad * max(len(entries), 1))()
    for i, e in enumerate(entries):
        for k, v in e.items():
            if k in ("A", "B", "gW", "gb", "sqnorm"):
                setattr(arr[i], k, _ptr(v))
            elif k == "scale":
                arr[i].scale = float(v)
            else:
                setattr(arr[i], k, int(v))
    return arr


class DPGhostLayer(ctypes.Structure):
    """struct dp_ghost_layer of dpgrad.h."""
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("T", ctypes.c_int64), ("d_in", ctypes.c_int64),
                ("d_out", ctypes.c_int64), ("scale", ctypes.c_float), ("bias", ctypes.c_int32),
                ("sqnorm", ctypes.c_void_p)]


def make_ghost_layers(entries):
    """A dp_ghost_layer array from (A, B, T, d_in, d_out, scale, bias, sqnorm) tuples."""
    arr = (DPGhostLayer * max(len(entries), 1))()
    for i, (A, B, T, d_in, d_out, scale, bias, sqnorm) in enumerate(entries):
        arr[i].A = _ptr(A)
        arr[i].B = _ptr(B)
        arr[i].T, arr[i].d_in, arr[i].d_out = int(T), int(d_in), int(d_out)
        arr[i].scale = float(scale)
        arr[i].bias = 1 if bias else 0
        arr[i].sqnorm = _ptr(sqnorm)
    return arr


class DPLayerNormLayer(ctypes.Structure):
    """struct dp_layernorm_layer of dpgrad.h."""
    _fields_ = [("xhat", ctypes.c_void_p), ("B", ctypes.c_void_p), ("T", ctypes.c_int64), ("D", ctypes.c_int64),
                ("scale", ctypes.c_float), ("ggamma", ctypes.c_void_p), ("gbeta", ctypes.c_void_p),
                ("sqnorm", ctypes.c_void_p)]


def make_layernorm_layers(entries):
    """A dp_layernorm_layer array from (xhat, B, T, D, scale, ggamma, gbeta, sqnorm) tuples."""
    arr = (DPLayerNormLayer * max(len(entries), 1))()
    for i, (xh, B, T, D, scale, gg, gb, sq) in enumerate(entries):
        arr[i].xhat = _ptr(xh)
        arr[i].B = _ptr(B)
        arr[i].T, arr[i].D = int(T), int(D)
        arr[i].scale = float(scale)
        arr[i].ggamma = _ptr(gg)
        arr[i].gbeta = _ptr(gb)
        arr[i].sqnorm = _ptr(sq)
    return arr


class DPError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__("%s: %s" % (where, status_string(code)))


_lib = None


def lib():
    """Load libdpgrad.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libdpgrad.so is not built (%s); run `python -m paper_2109_12298_amd.build`"
                               % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().dp_status_string(code).decode()


def dp_status_string(code: int) -> str:
    return status_string(code)


def dp_abi_version() -> int:
    return lib().dp_abi_version()


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _nbytes(x) -> int:
    if x is None:
        return 0
    return x.numel() * x.element_size()


def _numel(x) -> int:
    return 0 if x is None else x.numel()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def dtype_of(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return DP_F32
    if t.dtype == torch.bfloat16:
        return DP_BF16
    raise TypeError("unsupported dtype %s" % t.dtype)


def _check(code: int, where: str):
    if code != DP_OK:
        raise DPError(code, where)


# ---------------------------------------------------------------------------
# per-sample gradients
# ---------------------------------------------------------------------------

def dp_grad_sample_linear_workspace_bytes(N, T, d_in, d_out, dt) -> int:
    return lib().dp_grad_sample_linear_workspace_bytes(N, T, d_in, d_out, dt)


def dp_grad_sample_linear(A, B, dt, N, T, d_in, d_out, scale, gW, gb=None, sqnorm=None, status=None,
                          ws=None, stream=None):
    _check(lib().dp_grad_sample_linear(_ptr(A), _ptr(B), dt, N, T, d_in, d_out, scale, _ptr(gW), _ptr(gb),
                                       _ptr(sqnorm), _ptr(status), _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_grad_sample_linear")


def dp_grad_sample_linear_noalloc_max_bytes() -> int:
    return lib().dp_grad_sample_linear_noalloc_max_bytes()


def dp_grad_sample_linear_noalloc(A, B, dt, N, T, d_in, d_out, scale, gW, gb=None, sqnorm=None, status=None,
                                  stream=None):
    _check(lib().dp_grad_sample_linear_noalloc(_ptr(A), _ptr(B), dt, N, T, d_in, d_out, scale, _ptr(gW),
                                               _ptr(gb), _ptr(sqnorm), _ptr(status), _stream(stream)),
           "dp_grad_sample_linear_noalloc")


def dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw) -> int:
    return lib().dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw)


def dp_grad_sample_conv2d(X, GY, dt, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw, dh, dw, groups,
                          scale, gW, gb=None, sqnorm=None, status=None, ws=None, stream=None):
    _check(lib().dp_grad_sample_conv2d(_ptr(X), _ptr(GY), dt, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph,
                                       pw, dh, dw, groups, scale, _ptr(gW), _ptr(gb), _ptr(sqnorm),
                                       _ptr(status), _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_grad_sample_conv2d")


DP_CONV_AUTO, DP_CONV_TILED, DP_CONV_ROWS = 0, 1, 2


def dp_conv2d_set_path(path: int) -> int:
    """Process-wide kernel choice of dp_grad_sample_conv2d; returns the previous one."""
    prev = lib().dp_conv2d_set_path(path)
    if prev < 0:
        raise ValueError("unknown conv2d path %r" % (path,))
    return prev


DP_CONV_KERNEL_SMALL, DP_CONV_KERNEL_ROWS, DP_CONV_KERNEL_TILED = 0, 1, 2


def dp_conv2d_kernel_choice(N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw) -> int:
    """The conv kernel dp_grad_sample_conv2d would run for this shape now."""
    return lib().dp_conv2d_kernel_choice(N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw)


def dp_grad_sample_embedding_workspace_bytes(N, T) -> int:
    return lib().dp_grad_sample_embedding_workspace_bytes(N, T)


def dp_grad_sample_embedding(ids, B, dt, N, T, V, D, scale, row_ptr, uniq_ids, rows, cap, sqnorm=None,
                             status=None, ws=None, stream=None):
    _check(lib().dp_grad_sample_embedding(_ptr(ids), _ptr(B), dt, N, T, V, D, scale, _ptr(row_ptr),
                                          _ptr(uniq_ids), _ptr(rows), cap, _ptr(sqnorm), _ptr(status),
                                          _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_grad_sample_embedding")


def dp_lstm_backward(gates, c, W_hh, dh_out, dh_last, N, T, H, delta, status=None, stream=None):
    _check(lib().dp_lstm_backward(_ptr(gates), _ptr(c), _ptr(W_hh), _ptr(dh_out), _ptr(dh_last), N, T, H,
                                  _ptr(delta), _ptr(status), _stream(stream)), "dp_lstm_backward")


def dp_grad_sample_layernorm_workspace_bytes(N, T, D) -> int:
    return lib().dp_grad_sample_layernorm_workspace_bytes(N, T, D)


def dp_grad_sample_layernorm(xhat, B, dt, N, T, D, scale, ggamma, gbeta, sqnorm=None, status=None, ws=None,
                             stream=None):
    _check(lib().dp_grad_sample_layernorm(_ptr(xhat), _ptr(B), dt, N, T, D, scale, _ptr(ggamma), _ptr(gbeta),
                                          _ptr(sqnorm), _ptr(status), _ptr(ws), _nbytes(ws),
                                          _stream(stream)),
           "dp_grad_sample_layernorm")


def dp_grad_sample_groupnorm_workspace_bytes(N, C, P) -> int:
    return lib().dp_grad_sample_groupnorm_workspace_bytes(N, C, P)


def dp_grad_sample_groupnorm(xhat, B, dt, N, C, P, scale, ggamma, gbeta=None, sqnorm=None, status=None, ws=None,
                             stream=None):
    _check(lib().dp_grad_sample_groupnorm(_ptr(xhat), _ptr(B), dt, N, C, P, scale, _ptr(ggamma), _ptr(gbeta),
                                          _ptr(sqnorm), _ptr(status), _ptr(ws), _nbytes(ws),
                                          _stream(stream)),
           "dp_grad_sample_groupnorm")


# ---------------------------------------------------------------------------
# norms and clipping
# ---------------------------------------------------------------------------

def dp_per_sample_norms(sqnorm, n_layers, N, norm, status=None, stream=None):
    _check(lib().dp_per_sample_norms(_ptr(sqnorm), n_layers, N, _ptr(norm), _ptr(status), _stream(stream)),
           "dp_per_sample_norms")


def dp_per_sample_norms_active(sqnorm, n_layers, N, n_active, norm, status=None, stream=None):
    _check(lib().dp_per_sample_norms_active(_ptr(sqnorm), n_layers, N, _ptr(n_active), _ptr(norm), _ptr(status),
                                            _stream(stream)), "dp_per_sample_norms_active")


def dp_sqnorm_from_grads(G, N, numel, sqnorm, status=None, stream=None):
    _check(lib().dp_sqnorm_from_grads(_ptr(G), N, numel, _ptr(sqnorm), _ptr(status), _stream(stream)),
           "dp_sqnorm_from_grads")


def dp_clip_factors(norm, N, C, c, status=None, stream=None):
    _check(lib().dp_clip_factors(_ptr(norm), N, C, _ptr(c), _ptr(status), _stream(stream)), "dp_clip_factors")


def dp_clip_accumulate_workspace_bytes(N, numel) -> int:
    return lib().dp_clip_accumulate_workspace_bytes(N, numel)


def dp_clip_accumulate(G, norm, C, N, numel, sum, c_out=None, status=None, ws=None, stream=None):
    _check(lib().dp_clip_accumulate(_ptr(G), _ptr(norm), C, N, numel, _ptr(sum), _ptr(c_out), _ptr(status),
                                    _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_clip_accumulate")


def dp_clip_accumulate_linear_workspace_bytes(N, T, d_in, d_out, dt) -> int:
    return lib().dp_clip_accumulate_linear_workspace_bytes(N, T, d_in, d_out, dt)


def dp_clip_accumulate_linear(A, B, dt, N, T, d_in, d_out, scale, norm, C, sumW, sumb=None, status=None,
                              ws=None, stream=None):
    _check(lib().dp_clip_accumulate_linear(_ptr(A), _ptr(B), dt, N, T, d_in, d_out, scale, _ptr(norm), C,
                                           _ptr(sumW), _ptr(sumb), _ptr(status), _ptr(ws), _nbytes(ws),
                                           _stream(stream)),
           "dp_clip_accumulate_linear")


def dp_clip_accumulate_linear_many_workspace_bytes(items, count, dt, N) -> int:
    return lib().dp_clip_accumulate_linear_many_workspace_bytes(ctypes.cast(items, ctypes.c_void_p), count, dt, N)


def dp_clip_accumulate_linear_many(items, count, dt, N, norm, C, status=None, ws=None, stream=None):
    _check(lib().dp_clip_accumulate_linear_many(ctypes.cast(items, ctypes.c_void_p), count, dt, N, _ptr(norm), C,
                                                _ptr(status), _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_clip_accumulate_linear_many")


def dp_ghost_norm_linear_workspace_bytes(N, T, d_in, d_out) -> int:
    return lib().dp_ghost_norm_linear_workspace_bytes(N, T, d_in, d_out)


def dp_ghost_norm_linear(A, B, dt, N, T, d_in, d_out, scale, bias, sqnorm, status=None, ws=None, stream=None):
    _check(lib().dp_ghost_norm_linear(_ptr(A), _ptr(B), dt, N, T, d_in, d_out, scale, 1 if bias else 0,
                                      _ptr(sqnorm), _ptr(status), _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_ghost_norm_linear")


def dp_ghost_norm_linear_many_workspace_bytes(items, count, N) -> int:
    return lib().dp_ghost_norm_linear_many_workspace_bytes(ctypes.cast(items, ctypes.c_void_p), count, N)


def dp_ghost_norm_linear_many(items, count, dt, N, status=None, ws=None, stream=None):
    _check(lib().dp_ghost_norm_linear_many(ctypes.cast(items, ctypes.c_void_p), count, dt, N, _ptr(status),
                                           _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_ghost_norm_linear_many")


def dp_grad_sample_layernorm_many_workspace_bytes(items, count, N, dt) -> int:
    return lib().dp_grad_sample_layernorm_many_workspace_bytes(ctypes.cast(items, ctypes.c_void_p), count, N, dt)


def dp_grad_sample_layernorm_many(items, count, dt, N, status=None, ws=None, stream=None):
    _check(lib().dp_grad_sample_layernorm_many(ctypes.cast(items, ctypes.c_void_p), count, dt, N, _ptr(status),
                                               _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_grad_sample_layernorm_many")


def dp_grad_sample_many_grouped(items, k, dt, N) -> bool:
    """Whether layer k of a dp_layer_grad array goes into the grouped launch."""
    return bool(lib().dp_grad_sample_many_grouped(ctypes.cast(ctypes.byref(items[k]), ctypes.c_void_p), dt, N))


def dp_grad_sample_many_workspace_bytes(items, count, dt, N) -> int:
    return lib().dp_grad_sample_many_workspace_bytes(ctypes.cast(items, ctypes.c_void_p), count, dt, N)


def dp_grad_sample_many(items, count, dt, N, status=None, ws=None, stream=None):
    _check(lib().dp_grad_sample_many(ctypes.cast(items, ctypes.c_void_p), count, dt, N, _ptr(status), _ptr(ws),
                                     _nbytes(ws), _stream(stream)),
           "dp_grad_sample_many")


def dp_clip_accumulate_embedding_workspace_bytes(N, V) -> int:
    return lib().dp_clip_accumulate_embedding_workspace_bytes(N, V)


def dp_clip_accumulate_embedding(row_ptr, uniq_ids, rows, cap, norm, C, N, V, D, sum, status=None, ws=None,
                                 stream=None):
    _check(lib().dp_clip_accumulate_embedding(_ptr(row_ptr), _ptr(uniq_ids), _ptr(rows), cap, _ptr(norm), C, N,
                                              V, D, _ptr(sum), _ptr(status), _ptr(ws), _nbytes(ws),
                                              _stream(stream)),
           "dp_clip_accumulate_embedding")


# ---------------------------------------------------------------------------
# grouped clip + noise
# ---------------------------------------------------------------------------

def dp_clip_noise_many_workspace_bytes(params, count, N) -> int:
    return lib().dp_clip_noise_many_workspace_bytes(ctypes.cast(params, ctypes.c_void_p), count, N)


def dp_clip_noise_many(params, count, N, norm, C, seed, step, step_dev, sigma, denom, status=None, ws=None,
                       stream=None):
    _check(lib().dp_clip_noise_many(ctypes.cast(params, ctypes.c_void_p), count, N, _ptr(norm), C, seed, step,
                                    _ptr(step_dev), sigma, denom, _ptr(status), _ptr(ws), _nbytes(ws),
                                    _stream(stream)),
           "dp_clip_noise_many")


def dp_norms_clip_noise_workspace_bytes(params, count, N) -> int:
    return lib().dp_norms_clip_noise_workspace_bytes(ctypes.cast(params, ctypes.c_void_p), count, N)


def dp_norms_clip_noise(sqnorm, n_layers, params, count, N, norm, C, seed, step, step_dev, sigma, denom,
                        status=None, ws=None, stream=None):
    _check(lib().dp_norms_clip_noise(_ptr(sqnorm), n_layers, ctypes.cast(params, ctypes.c_void_p), count, N,
                                     _ptr(norm), C, seed, step, _ptr(step_dev), sigma, denom, _ptr(status),
                                     _ptr(ws), _nbytes(ws), _stream(stream)),
           "dp_norms_clip_noise")


def dp_norms_clip_noise_sched(sqnorm, n_layers, params, count, N, norm, C, seed, step, step_dev, sigma_table,
                              denom, status=None, ws=None, stream=None, n_active=None):
    """dp_norms_clip_noise with the noise multiplier of step t read from
    sigma_table[min(t, len - 1)] (a device float tensor) on the device, and
    optionally the active batch size from n_active (a device int64)."""
    _check(lib().dp_norms_clip_noise_sched(_ptr(sqnorm), n_layers, ctypes.cast(params, ctypes.c_void_p), count, N,
                                           _ptr(norm), C, seed, step, _ptr(step_dev), _ptr(sigma_table),
                                           _numel(sigma_table), _ptr(n_active), denom, _ptr(status), _ptr(ws),
                                           _nbytes(ws), _stream(stream)),
           "dp_norms_clip_noise_sched")


def dp_step_advance(step_dev, by=1, stream=None):
    _check(lib().dp_step_advance(_ptr(step_dev), by, _stream(stream)), "dp_step_advance")


# ---------------------------------------------------------------------------
# noise
# ---------------------------------------------------------------------------

def dp_add_noise(sum, out, numel, seed, step, param_index, sigma, C, denom, status=None, stream=None):
    _check(lib().dp_add_noise(_ptr(sum), _ptr(out), numel, seed, step, param_index, sigma, C, denom,
                              _ptr(status), _stream(stream)),
           "dp_add_noise")


def dp_philox_normals(z, raw, numel, seed, step, param_index, stream=None):
    _check(lib().dp_philox_normals(_ptr(z), _ptr(raw), numel, seed, step, param_index, _stream(stream)),
           "dp_philox_normals")
