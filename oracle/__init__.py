"""CPU oracle of the DeaMoE decode layer: TEST INFRASTRUCTURE ONLY.

ctypes front end of oracle/deamoe_oracle.c (plain C, fp64 accumulation).
Only tests/, the smoke check and the benchmark's CPU-baseline leg use it; the
product path never does.  It takes plain tensors / arrays and any object with
the layer-config attributes (hidden, n_experts, n_depts, top_k, top_k_dept,
d_shared, d_private, d_shared_expert, form, score, renorm, sigma, route_scale,
w_dtype, act_dtype, optionally dept_cover); it imports nothing from the HIP package.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None

_KEYS = ("dept_gate", "dept_up", "dept_down", "priv_gate", "priv_up", "priv_down",
         "se_gate", "se_up", "se_down")


class _Config(C.Structure):
    _fields_ = [(f, C.c_int) for f in ("hidden", "n_experts", "n_depts", "top_k", "top_k_dept",
                                       "d_shared", "d_private", "d_shared_expert",
                                       "form", "score", "renorm", "sigma")] + \
               [("route_scale", C.c_double), ("w_dtype", C.c_int), ("act_dtype", C.c_int),
                ("dept_cover", C.c_int)]


class _Weights(C.Structure):
    _fields_ = [("router", C.c_void_p), ("mat", C.c_void_p * 9), ("scale", C.c_void_p * 9)]


class _Routing(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("logits", "topk_ids", "topk_w", "tok_depts",
                                          "tok_dept_w", "tok_ndept", "dept_count", "dept_offset",
                                          "dept_tokens", "exp_count", "exp_offset", "exp_tokens")]


def _open(path: str):
    """Load an oracle build and declare its signatures."""
    L = C.CDLL(path)
    L.oref_num_threads.restype = C.c_int
    L.oref_set_num_threads.argtypes = [C.c_int]
    L.oref_fp8_value.restype = C.c_double
    L.oref_fp8_value.argtypes = [C.c_uint8]
    L.oref_fp8_decode.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p]
    L.oref_route.argtypes = [C.POINTER(_Config), C.c_int, C.c_void_p, C.c_void_p,
                             C.c_void_p, C.c_void_p, C.POINTER(_Routing)]
    L.oref_layer_naive.argtypes = [C.POINTER(_Config), C.c_int, C.c_void_p,
                                   C.POINTER(_Weights), C.c_void_p, C.c_void_p,
                                   C.c_int, C.c_void_p, C.c_void_p]
    L.oref_layer_two_stage.argtypes = [C.POINTER(_Config), C.c_int, C.c_void_p,
                                       C.POINTER(_Weights), C.c_void_p, C.c_void_p,
                                       C.c_void_p]
    L.oref_step_weight_bytes.restype = C.c_int64
    L.oref_step_weight_bytes.argtypes = [C.POINTER(_Config), C.c_void_p, C.c_void_p]
    return L


def lib():
    """The oracle library: oracle/liboracle.so, or the build named by
    DEAMOE_ORACLE_LIB (the sanitizer build of the CPU tests)."""
    global _lib
    if _lib is None:
        path = os.environ.get("DEAMOE_ORACLE_LIB", _build.LIB)
        if path == _build.LIB and not os.path.exists(path):
            _build.build()
        _lib = _open(path)
    return _lib


_DT = {"f32": 0, "bf16": 1, "fp8": 2}


def _config(cfg) -> _Config:
    return _Config(hidden=cfg.hidden, n_experts=cfg.n_experts, n_depts=cfg.n_depts,
                   top_k=cfg.top_k, top_k_dept=cfg.top_k_dept, d_shared=cfg.d_shared,
                   d_private=cfg.d_private, d_shared_expert=cfg.d_shared_expert,
                   form={"slice": 0, "factored": 1}[cfg.form],
                   score={"softmax": 0, "sigmoid": 1}[cfg.score],
                   renorm=int(bool(cfg.renorm)),
                   sigma={"silu": 0, "none": 1, "gelu": 2, "rmsnorm": 3}[cfg.sigma],
                   route_scale=float(cfg.route_scale), w_dtype=_DT[cfg.w_dtype],
                   act_dtype=_DT[cfg.act_dtype], dept_cover=int(getattr(cfg, "dept_cover", 0)))


def _host(a, keep: list):
    """Raw host bytes of a tensor / array (bf16 as its bit pattern); kept alive in `keep`."""
    if a is None:
        return None
    try:
        import torch
        if isinstance(a, torch.Tensor):
            t = a.detach().to("cpu").contiguous()
            if t.dtype == torch.bfloat16:
                t = t.view(torch.int16)
            a = t.numpy()
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(a)
    keep.append(a)
    return a.ctypes.data


def _weights(w: dict, keep: list) -> _Weights:
    W = _Weights()
    W.router = _host(w["router"], keep)
    for i, k in enumerate(_KEYS):
        W.mat[i] = _host(w.get(k), keep)
        W.scale[i] = _host(w.get(k + "_scale"), keep)
    return W


def _f32(a, keep):
    if a is None:
        return None
    try:
        import torch
        if isinstance(a, torch.Tensor):
            a = a.detach().to("cpu", torch.float32).numpy()
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(a, dtype=np.float32)
    keep.append(a)
    return a.ctypes.data


def route(cfg, x, router, logits_in=None, bias=None, T: int | None = None) -> dict:
    """Eq. 2 routing plus department bookkeeping for all tokens."""
    keep = []
    if T is None:
        T = int(x.shape[0]) if x is not None else int(logits_in.shape[0])
    n, m, k = cfg.n_experts, cfg.n_depts, cfg.top_k
    out = {"logits": np.zeros((T, n), np.float32), "topk_ids": np.zeros((T, k), np.int32),
           "topk_w": np.zeros((T, k), np.float64), "tok_depts": np.zeros((T, k), np.int32),
           "tok_dept_w": np.zeros((T, k), np.float64), "tok_ndept": np.zeros(T, np.int32),
           "dept_count": np.zeros(m, np.int32), "dept_offset": np.zeros(m + 1, np.int32),
           "dept_tokens": np.zeros(max(T * k, 1), np.int32), "exp_count": np.zeros(n, np.int32),
           "exp_offset": np.zeros(n + 1, np.int32), "exp_tokens": np.zeros(max(T * k, 1), np.int32)}
    R = _Routing(**{key: arr.ctypes.data for key, arr in out.items()})
    c = _config(cfg)
    rc = lib().oref_route(C.byref(c), T, _host(x, keep), _host(router, keep),
                          _f32(logits_in, keep), _f32(bias, keep), C.byref(R))
    if rc:
        raise ValueError("oracle rejected the configuration")
    out["dept_tokens"] = out["dept_tokens"][: out["dept_offset"][m]]
    out["exp_tokens"] = out["exp_tokens"][: out["exp_offset"][n]]
    return out


def layer(cfg, x, weights: dict, logits_in=None, bias=None, tokens=None) -> np.ndarray:
    """Naive Eq. 3 output (fp64) for the given token indices (default: all)."""
    keep = []
    T = int(x.shape[0])
    sel = None
    n_sel = T
    if tokens is not None:
        sel = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
        keep.append(sel)
        n_sel = len(sel)
    y = np.zeros((n_sel, cfg.hidden), np.float64)
    c = _config(cfg)
    W = _weights(weights, keep)
    rc = lib().oref_layer_naive(C.byref(c), T, _host(x, keep), C.byref(W),
                                _f32(logits_in, keep), _f32(bias, keep), n_sel,
                                None if sel is None else sel.ctypes.data, y.ctypes.data)
    if rc:
        raise ValueError("oracle rejected the configuration")
    return y


def layer_two_stage(cfg, x, weights: dict, logits_in=None, bias=None) -> np.ndarray:
    """The same output computed in the two-stage order of Sec. 3.2 (fp64)."""
    keep = []
    T = int(x.shape[0])
    y = np.zeros((T, cfg.hidden), np.float64)
    c = _config(cfg)
    W = _weights(weights, keep)
    rc = lib().oref_layer_two_stage(C.byref(c), T, _host(x, keep), C.byref(W),
                                    _f32(logits_in, keep), _f32(bias, keep), y.ctypes.data)
    if rc:
        raise ValueError("oracle rejected the configuration")
    return y


def set_num_threads(n: int) -> None:
    """Threads of the naive layer's token loop for later calls."""
    lib().oref_set_num_threads(int(n))


def num_threads() -> int:
    """Threads the oracle's token loop runs on."""
    return int(lib().oref_num_threads())


def fp8_decode(codes) -> np.ndarray:
    keep = []
    codes = np.ascontiguousarray(np.asarray(codes, dtype=np.uint8))
    out = np.zeros(codes.shape, np.float64)
    lib().oref_fp8_decode(_host(codes, keep), codes.size, out.ctypes.data)
    return out


def step_weight_bytes(cfg, dept_count, exp_count) -> int:
    keep = []
    dc = np.ascontiguousarray(np.asarray(dept_count, np.int32))
    ec = np.ascontiguousarray(np.asarray(exp_count, np.int32))
    keep += [dc, ec]
    c = _config(cfg)
    return int(lib().oref_step_weight_bytes(C.byref(c), dc.ctypes.data, ec.ctypes.data))
