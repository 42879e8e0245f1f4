"""Python binding of libdeamoe.so (the C ABI in include/deamoe.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  PyTorch provides device memory and the current stream.  The module
raises at import of the library when libdeamoe.so is missing; there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdeamoe.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4
F32, BF16, FP8_E4M3_B128 = 0, 1, 2
FORM_SLICE, FORM_FACTORED = 0, 1
SCORE_SOFTMAX, SCORE_SIGMOID = 0, 1
SIGMA_SILU, SIGMA_NONE, SIGMA_GELU, SIGMA_RMSNORM = 0, 1, 2, 3
MAX_TOKENS = 128
SCRATCH_BYTES = 64 << 20   # library-owned workspace of deamoe_layer_forward_noalloc, per GPU

EXPORTS = ("deamoe_status_string", "deamoe_workspace_bytes", "deamoe_route",
           "deamoe_layer_forward", "deamoe_layer_forward_traced", "deamoe_baseline_forward",
           "deamoe_loaded_bytes", "deamoe_trace_points", "deamoe_layer_forward_noalloc")


class DeamoeError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class deamoe_config(C.Structure):
    _fields_ = [(f, C.c_int32) for f in ("hidden", "n_experts", "n_depts", "top_k", "top_k_dept",
                                         "d_shared", "d_private", "d_shared_expert", "form",
                                         "score", "renorm", "sigma")] + \
               [("route_scale", C.c_float), ("w_dtype", C.c_int32), ("act_dtype", C.c_int32),
                ("max_tokens", C.c_int32), ("dept_cover", C.c_int32)]


class deamoe_weights(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("router", "dept_gate", "dept_up", "dept_down",
                                          "priv_gate", "priv_up", "priv_down", "se_gate", "se_up",
                                          "se_down")] + [("scale", C.c_void_p * 9)]


ROUTING_FIELDS = ("topk_ids", "topk_w", "tok_depts", "tok_dept_w", "tok_ndept", "dept_count",
                  "dept_offset", "dept_tokens", "exp_count", "exp_offset", "exp_tokens", "logits")


class deamoe_routing(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ROUTING_FIELDS]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with "
                              "`python -m paper_2608_14385_amd.build`")
        L = C.CDLL(LIB_PATH)
        cfgp, vp, i32 = C.POINTER(deamoe_config), C.c_void_p, C.c_int32
        L.deamoe_status_string.restype = C.c_char_p
        L.deamoe_status_string.argtypes = [C.c_int]
        L.deamoe_workspace_bytes.argtypes = [cfgp, C.POINTER(C.c_size_t)]
        L.deamoe_route.argtypes = [cfgp, i32, vp, vp, vp, vp, C.POINTER(deamoe_routing), vp,
                                   C.c_size_t, vp]
        layer_args = [cfgp, i32, vp, C.POINTER(deamoe_weights), vp, vp, C.POINTER(deamoe_routing),
                      vp, vp, C.c_size_t, vp]
        L.deamoe_layer_forward.argtypes = layer_args
        L.deamoe_baseline_forward.argtypes = layer_args
        L.deamoe_layer_forward_traced.argtypes = layer_args + [C.POINTER(C.c_void_p), i32]
        L.deamoe_layer_forward_noalloc.argtypes = [cfgp, i32, vp, C.POINTER(deamoe_weights), vp, vp,
                                                   C.POINTER(deamoe_routing), vp, vp]
        L.deamoe_trace_points.argtypes = [cfgp, i32, C.POINTER(C.c_int32)]
        L.deamoe_loaded_bytes.argtypes = [cfgp, i32, vp, vp, C.POINTER(C.c_int64),
                                          C.POINTER(C.c_int64)]
        for f in EXPORTS:
            getattr(L, f).restype = C.c_int if f != "deamoe_status_string" else C.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().deamoe_status_string(status).decode()


def _check(status: int, what: str):
    if status != OK:
        raise DeamoeError(status, what)


_DT = {"f32": F32, "bf16": BF16, "fp8": FP8_E4M3_B128}


def make_config(cfg, max_tokens: int) -> deamoe_config:
    """C config from a layer description (workloads.LayerConfig or alike)."""
    return deamoe_config(hidden=cfg.hidden, n_experts=cfg.n_experts, n_depts=cfg.n_depts,
                         top_k=cfg.top_k, top_k_dept=cfg.top_k_dept, d_shared=cfg.d_shared,
                         d_private=cfg.d_private, d_shared_expert=cfg.d_shared_expert,
                         form={"slice": FORM_SLICE, "factored": FORM_FACTORED}[cfg.form],
                         score={"softmax": SCORE_SOFTMAX, "sigmoid": SCORE_SIGMOID}[cfg.score],
                         renorm=int(bool(cfg.renorm)),
                         sigma={"silu": SIGMA_SILU, "none": SIGMA_NONE, "gelu": SIGMA_GELU,
                                "rmsnorm": SIGMA_RMSNORM}[cfg.sigma],
                         route_scale=float(cfg.route_scale), w_dtype=_DT[cfg.w_dtype],
                         act_dtype=_DT[cfg.act_dtype], max_tokens=int(max_tokens),
                         dept_cover=int(getattr(cfg, "dept_cover", 0)))


_WKEYS = ("dept_gate", "dept_up", "dept_down", "priv_gate", "priv_up", "priv_down",
          "se_gate", "se_up", "se_down")


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def make_weights(w: dict) -> deamoe_weights:
    """C weight table from a dict of device tensors (keys as in workloads.weight_shapes)."""
    W = deamoe_weights()
    W.router = _ptr(w.get("router"))
    for i, k in enumerate(_WKEYS):
        setattr(W, k, _ptr(w.get(k)))
        W.scale[i] = _ptr(w.get(k + "_scale"))
    return W


def workspace_bytes(c: deamoe_config) -> int:
    n = C.c_size_t(0)
    _check(lib().deamoe_workspace_bytes(C.byref(c), C.byref(n)), "deamoe_workspace_bytes")
    return int(n.value)


def alloc_workspace(c: deamoe_config, device="cuda") -> torch.Tensor:
    return torch.empty(workspace_bytes(c), dtype=torch.uint8, device=device)


@dataclass
class Routing:
    """Device tensors receiving the routing of one step."""
    tensors: dict

    @classmethod
    def alloc(cls, cfg, T: int, device="cuda") -> "Routing":
        n, m, k = cfg.n_experts, cfg.n_depts, cfg.top_k
        i32, f32 = torch.int32, torch.float32
        shapes = {"topk_ids": ((T, k), i32), "topk_w": ((T, k), f32),
                  "tok_depts": ((T, k), i32), "tok_dept_w": ((T, k), f32),
                  "tok_ndept": ((T,), i32), "dept_count": ((m,), i32),
                  "dept_offset": ((m + 1,), i32), "dept_tokens": ((max(T * k, 1),), i32),
                  "exp_count": ((n,), i32), "exp_offset": ((n + 1,), i32),
                  "exp_tokens": ((max(T * k, 1),), i32), "logits": ((T, n), f32)}
        return cls({key: torch.full(s, -7, dtype=dt, device=device)
                    for key, (s, dt) in shapes.items()})

    def struct(self) -> deamoe_routing:
        return deamoe_routing(**{k: self.tensors[k].data_ptr() for k in ROUTING_FIELDS})

    def host(self) -> dict:
        """Host copies, with the CSR token lists cut to their used length."""
        h = {k: v.cpu().numpy() for k, v in self.tensors.items()}
        h["dept_tokens"] = h["dept_tokens"][: h["dept_offset"][-1]]
        h["exp_tokens"] = h["exp_tokens"][: h["exp_offset"][-1]]
        return h


def _stream(stream) -> int | None:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def deamoe_route(c: deamoe_config, x, router_w, routing: Routing, ws: torch.Tensor,
                 logits_in=None, router_bias=None, T: int | None = None, stream=None):
    T = int(x.shape[0]) if T is None else T
    r = routing.struct()
    _check(lib().deamoe_route(C.byref(c), T, _ptr(x), _ptr(router_w), _ptr(logits_in),
                              _ptr(router_bias), C.byref(r), _ptr(ws), ws.numel(),
                              _stream(stream)), "deamoe_route")


def _layer(fn, c, x, W, y, ws, logits_in, router_bias, routing, stream, *extra):
    r = routing.struct() if routing is not None else None
    _check(fn(C.byref(c), int(x.shape[0]), _ptr(x), C.byref(W), _ptr(logits_in),
              _ptr(router_bias), C.byref(r) if r is not None else None, _ptr(y), _ptr(ws),
              ws.numel(), _stream(stream), *extra), fn.__name__)


def deamoe_layer_forward(c: deamoe_config, x, W: deamoe_weights, y, ws, logits_in=None,
                         router_bias=None, routing: Routing | None = None, stream=None):
    _layer(lib().deamoe_layer_forward, c, x, W, y, ws, logits_in, router_bias, routing, stream)


def deamoe_layer_forward_traced(c: deamoe_config, x, W: deamoe_weights, y, ws, events: list,
                                logits_in=None, router_bias=None, routing: Routing | None = None,
                                stream=None):
    """events: raw hipEvent_t handles (ints) recorded at the stage boundaries."""
    arr = (C.c_void_p * len(events))(*events)
    _layer(lib().deamoe_layer_forward_traced, c, x, W, y, ws, logits_in, router_bias, routing,
           stream, arr, len(events))


def deamoe_layer_forward_noalloc(c: deamoe_config, x, W: deamoe_weights, y, logits_in=None,
                                 router_bias=None, routing: Routing | None = None, stream=None):
    """deamoe_layer_forward on the library's own per-GPU scratch array (no workspace)."""
    r = routing.struct() if routing is not None else None
    _check(lib().deamoe_layer_forward_noalloc(
        C.byref(c), int(x.shape[0]), _ptr(x), C.byref(W), _ptr(logits_in), _ptr(router_bias),
        C.byref(r) if r is not None else None, _ptr(y), _stream(stream)),
        "deamoe_layer_forward_noalloc")


def deamoe_baseline_forward(c: deamoe_config, x, W: deamoe_weights, y, ws, logits_in=None,
                            router_bias=None, routing: Routing | None = None, stream=None):
    _layer(lib().deamoe_baseline_forward, c, x, W, y, ws, logits_in, router_bias, routing, stream)


def deamoe_loaded_bytes(c: deamoe_config, T: int, dept_count, exp_count) -> tuple:
    import numpy as np
    dc = np.ascontiguousarray(np.asarray(dept_count, dtype=np.int32))
    ec = np.ascontiguousarray(np.asarray(exp_count, dtype=np.int32))
    wb, tb = C.c_int64(0), C.c_int64(0)
    _check(lib().deamoe_loaded_bytes(C.byref(c), T, dc.ctypes.data, ec.ctypes.data, C.byref(wb),
                                     C.byref(tb)), "deamoe_loaded_bytes")
    return int(wb.value), int(tb.value)


def deamoe_trace_points(c: deamoe_config, T: int) -> int:
    n = C.c_int32(0)
    _check(lib().deamoe_trace_points(C.byref(c), T, C.byref(n)), "deamoe_trace_points")
    return int(n.value)


class Layer:
    """Owns the config, weight table and workspace of one layer on one device."""

    def __init__(self, cfg, weights: dict, max_tokens: int, device="cuda", baseline=False):
        self.cfg = cfg
        self.c = make_config(cfg, max_tokens)
        self.weights = weights
        self.W = make_weights(weights)
        self.ws = alloc_workspace(self.c, device)
        self.baseline = baseline

    def __call__(self, x, logits_in=None, router_bias=None, routing=None, y=None, stream=None):
        if y is None:
            y = torch.empty_like(x)
        fn = deamoe_baseline_forward if self.baseline else deamoe_layer_forward
        fn(self.c, x, self.W, y, self.ws, logits_in=logits_in, router_bias=router_bias,
           routing=routing, stream=stream)
        return y
