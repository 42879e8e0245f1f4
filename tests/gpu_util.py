"""Helpers of the GPU parity tests: run a case through the C ABI and through
the oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2608_14385_amd import deamoe as D
from paper_2608_14385_amd import workloads as W

TOL = {"f32": 1e-4, "bf16": 2e-2, "fp8": 6e-2}
ROUTE_EXACT = ("topk_ids", "tok_ndept", "tok_depts", "dept_count", "dept_offset", "dept_tokens",
               "exp_count", "exp_offset", "exp_tokens")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


class Case:
    """Seeded inputs of one layer run, on the device and (lazily) on the host."""

    def __init__(self, cfg, T, seed=0, gate_exact=True, logits=None, bias=None,
                 identity_private=False, max_tokens=None, weights=None):
        self.cfg, self.T = cfg, T
        self.max_tokens = max_tokens or max(T, 1)
        self.w = weights if weights is not None else W.make_weights(
            cfg, seed, device="cuda", gate_exact=gate_exact, identity_private=identity_private)
        self.x = W.make_tokens(cfg, T, seed, device="cuda", gate_exact=gate_exact)
        self.logits = None
        if logits == "uniform":
            self.logits = W.make_logits(cfg, T, seed, "uniform", device="cuda")
        elif logits == "gumbel":
            self.logits = W.make_logits(cfg, T, seed, "gumbel", device="cuda",
                                        bias=W.make_zipf_bias(cfg, seed))
        self.bias = W.make_zipf_bias(cfg, seed).cuda() if bias == "zipf" else None
        self._host = None

    def host(self):
        if self._host is None:
            self._host = {k: v.cpu() for k, v in self.w.items()}
        return self._host

    def run_gpu(self, baseline=False, routing=True):
        layer = D.Layer(self.cfg, self.w, self.max_tokens, baseline=baseline)
        rt = D.Routing.alloc(self.cfg, self.T) if routing else None
        y = torch.full_like(self.x, float("nan"))
        layer(self.x, logits_in=self.logits, router_bias=self.bias, routing=rt, y=y)
        torch.cuda.synchronize()
        return y, rt, layer

    def run_oracle(self, tokens=None):
        return oracle.layer(self.cfg, self.x.cpu(), self.host(), logits_in=self._cpu(self.logits),
                            bias=self._cpu(self.bias), tokens=tokens)

    def route_oracle(self):
        return oracle.route(self.cfg, self.x.cpu(), self.host()["router"],
                            logits_in=self._cpu(self.logits), bias=self._cpu(self.bias), T=self.T)

    @staticmethod
    def _cpu(t):
        return None if t is None else t.cpu()


def compare_routing(got: dict, ref: dict, T: int, k: int, exact_logits=True):
    for key in ROUTE_EXACT:
        a, b = np.asarray(got[key]), np.asarray(ref[key])
        if key in ("topk_ids", "tok_depts"):
            a, b = a.reshape(T, k), b.reshape(T, k)
        assert a.shape == b.shape, (key, a.shape, b.shape)
        assert np.array_equal(a, b), f"routing field {key} differs: first at {np.argwhere(a != b)[:4]}"
    np.testing.assert_allclose(got["topk_w"], ref["topk_w"], rtol=1e-5, atol=1e-7)
    np.testing.assert_allclose(got["tok_dept_w"], ref["tok_dept_w"], rtol=1e-5, atol=1e-7)
    if exact_logits:
        assert np.array_equal(got["logits"], ref["logits"]), "logits not bit-identical"


def compare_outputs(y_gpu: torch.Tensor, y_ref: np.ndarray, dtype: str, rows=None):
    y = y_gpu.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        y = y[rows]
    assert np.isfinite(y).all(), "non-finite output"
    err = np.abs(y - y_ref).max()
    scale = np.abs(y_ref).max()
    tol = TOL[dtype] * scale
    say(f"    max|err| = {err:.3e}   max|ref| = {scale:.3e}   ratio = {err / max(scale, 1e-30):.2e}"
        f"   (tol {TOL[dtype]:.0e})")
    assert err <= tol, f"max|err| {err:.4e} > {TOL[dtype]} * max|ref| ({scale:.4e})"
    return err / max(scale, 1e-30)


class WeightCache:
    """One weight draw of a full-size layer shared by the batches that test it
    (device tensors and their host copies).  Holds one draw at a time, so the
    device and host memory of a preset is released when the next one is
    drawn, and all of it by clear()."""

    def __init__(self):
        self.key, self.w, self.hw = None, None, None

    def get(self, cfg, seed: int, gate_exact: bool = True, host: bool = True):
        key = (cfg, seed, gate_exact)
        if key != self.key:
            self.clear()
            self.w = W.make_weights(cfg, seed, device="cuda", gate_exact=gate_exact)
            self.key = key
        if host and self.hw is None:
            self.hw = {k: v.cpu() for k, v in self.w.items()}
        return self.w, self.hw

    def case(self, cfg, T, seed, weight_seed, gate_exact=True, **kw) -> "Case":
        w, hw = self.get(cfg, weight_seed, gate_exact)
        c = Case(cfg, T, seed=seed, gate_exact=gate_exact, weights=w, **kw)
        c._host = hw
        return c

    def clear(self):
        self.key, self.w, self.hw = None, None, None
        torch.cuda.empty_cache()
