"""Seeded synthetic workloads for the DeaMoE decode layer.

This module only *describes and draws* inputs: layer shapes (presets), weights,
token activations, injected router logits and router biases.  It holds none of
the layer's arithmetic (no routing, no projections, no combine), so both the
HIP path and the CPU oracle can take their inputs from it without sharing any
of the method.

Shapes follow the paper's notation (Sec. 2.1 and Sec. 3.1):
  h        hidden size
  n        routed experts, grouped into m departments of E_d = n / m experts
  k        experts per token (Eq. 2), k_dept optional cap on departments per token
  d_s      intermediate size of the department-shared part
  d_p      intermediate size of each expert's private part (SLICE form)
  d        for the FACTORED form (Sec. 3.1, Eq. 4) the department intermediate
           size; the private A matrices are d x d
  d_se     always-on shared expert (0 = none)

Storage convention for every matrix: row-major [out, in].  The department down
projection is stored as (W_d^j)^T, shape [h, d_s]; in the FACTORED form the
private down matrix is stored as (A_d^i)^T, shape [d, d].

Weights are N(0, 1/sqrt(fan_in)) with fan_in = in-features of the matrix,
rounded to the storage dtype.  fp8 weights are OCP e4m3fn codes with one fp32
scale per 128 x 128 block of each [out, in] matrix: s = max|w| / 448 over the
block and q = e4m3(clamp(w / s, -448, 448)) (round to nearest even).
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import torch

FP8_MAX = 448.0
FP8_BLOCK = 128

_TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class LayerConfig:
    name: str
    hidden: int
    n_experts: int
    n_depts: int
    top_k: int
    top_k_dept: int = 0
    d_shared: int = 0
    d_private: int = 0
    d_shared_expert: int = 0
    form: str = "slice"          # "slice" | "factored"
    score: str = "softmax"       # "softmax" | "sigmoid"
    renorm: bool = True
    sigma: str = "silu"          # FACTORED interface nonlinearity: "silu" | "none" | "gelu" | "rmsnorm"
    route_scale: float = 1.0
    w_dtype: str = "f32"         # "f32" | "bf16" | "fp8"
    act_dtype: str = "f32"       # "f32" | "bf16"
    dept_cover: int = 0          # 1: strict department coverage (exactly top_k_dept per token)

    @property
    def experts_per_dept(self) -> int:
        return self.n_experts // self.n_depts

    def replace(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


@dataclass(frozen=True)
class Workload:
    """A layer config, its vanilla-MoE comparator and the batch sizes it runs at."""
    layer: LayerConfig
    baseline: LayerConfig
    batches: tuple
    routing: str = "gaussian"    # "gaussian" | "uniform_logits" | "zipf_bias"


def _vanilla(cfg: LayerConfig, name: str, n: int, k: int, f: int) -> LayerConfig:
    # Eq. 1-3: n independent SwiGLU experts of intermediate f.  Expressed as a
    # layer whose departments hold one expert each and no private part.
    return cfg.replace(name=name, n_experts=n, n_depts=n, top_k=k, top_k_dept=0,
                       d_shared=f, d_private=0, form="slice")


def _make_presets() -> dict:
    p = {}
    # Tiny fp32 SLICE layer (parity only).
    c1 = LayerConfig("tiny_f32", hidden=256, n_experts=16, n_depts=4, top_k=2,
                     d_shared=512, d_private=64, score="softmax", renorm=True,
                     w_dtype="f32", act_dtype="f32")
    p["tiny_f32"] = Workload(c1, _vanilla(c1, "tiny_f32_vanilla", 16, 2, 576), (4,))
    # Tiny FACTORED layer (Eq. 4) with the same router shape.
    tf = LayerConfig("tiny_factored", hidden=256, n_experts=16, n_depts=4, top_k=2,
                     d_shared=128, form="factored", score="softmax", renorm=True,
                     sigma="silu", w_dtype="f32", act_dtype="f32")
    p["tiny_factored"] = Workload(tf, _vanilla(tf, "tiny_factored_vanilla", 16, 2, 128), (4,))
    # 7B-class bf16 SLICE layer with an always-on shared expert.
    c2 = LayerConfig("7b_bf16", hidden=2048, n_experts=64, n_depts=8, top_k=6,
                     d_shared=1152, d_private=128, d_shared_expert=2816,
                     score="softmax", renorm=True, w_dtype="bf16", act_dtype="bf16")
    p["7b_bf16"] = Workload(c2, _vanilla(c2, "7b_bf16_vanilla", 64, 6, 1280), (1, 4, 16),
                            routing="uniform_logits")
    # DeepSeek-V3-shaped bf16 SLICE layer.
    c3 = LayerConfig("dsv3_bf16", hidden=7168, n_experts=256, n_depts=32, top_k=8,
                     d_shared=1792, d_private=256, score="sigmoid", renorm=True,
                     w_dtype="bf16", act_dtype="bf16")
    p["dsv3_bf16"] = Workload(c3, _vanilla(c3, "dsv3_bf16_vanilla", 256, 8, 2048),
                              (1, 2, 4, 8, 16, 32, 64))
    # Same shape, routing skewed towards few departments (Zipf s=1.2 bias).
    c4 = c3.replace(name="dsv3_skew")
    p["dsv3_skew"] = Workload(c4, _vanilla(c4, "dsv3_skew_vanilla", 256, 8, 2048),
                              (16, 32, 64, 128), routing="zipf_bias")
    # Same shape, fp8 e4m3 weights with 128x128 block scales.
    c5 = c3.replace(name="dsv3_fp8", w_dtype="fp8")
    p["dsv3_fp8"] = Workload(c5, _vanilla(c5, "dsv3_fp8_vanilla", 256, 8, 2048),
                             (1, 2, 4, 8, 16, 32))
    # The paper's budget-matched DeepSeek-V3 DeaMoE row of Table 1, FACTORED form.
    m6 = LayerConfig("dsv3_factored", hidden=7168, n_experts=864, n_depts=8, top_k=10,
                     top_k_dept=5, d_shared=2048, form="factored", score="sigmoid",
                     renorm=True, sigma="silu", w_dtype="bf16", act_dtype="bf16")
    p["dsv3_factored"] = Workload(m6, _vanilla(m6, "dsv3_vanilla_256x2048", 256, 8, 2048),
                                  (1, 2, 4, 8, 16, 32, 64))
    # The Qwen3-235B-A22B and Baseline-7B rows of Table 1 (Sec. 3.3), FACTORED
    # form, each against its MoE baseline; softmax with renormalised top-k.
    qw = LayerConfig("qwen3_factored", hidden=4096, n_experts=320, n_depts=8, top_k=8,
                     top_k_dept=5, d_shared=1536, form="factored", score="softmax",
                     renorm=True, sigma="silu", w_dtype="bf16", act_dtype="bf16")
    p["qwen3_factored"] = Workload(qw, _vanilla(qw, "qwen3_vanilla_128x1536", 128, 8, 1536),
                                   (1, 4, 16, 64))
    b7 = LayerConfig("base7b_factored", hidden=1024, n_experts=672, n_depts=8, top_k=10,
                     top_k_dept=4, d_shared=384, form="factored", score="softmax",
                     renorm=True, sigma="silu", w_dtype="bf16", act_dtype="bf16")
    p["base7b_factored"] = Workload(b7, _vanilla(b7, "base7b_vanilla_256x384", 256, 8, 384),
                                    (1, 4, 16, 64))
    # The DeepSeek-V2 and Kimi-K2 rows of Table 1.  DeepSeek-V2 keeps its own
    # gate (softmax over all experts, top-k weights not renormalised); Kimi-K2
    # follows DeepSeek-V3 (sigmoid, renormalised).
    v2 = LayerConfig("dsv2_factored", hidden=5120, n_experts=512, n_depts=8, top_k=10,
                     top_k_dept=5, d_shared=1536, form="factored", score="softmax",
                     renorm=False, sigma="silu", w_dtype="bf16", act_dtype="bf16")
    p["dsv2_factored"] = Workload(v2, _vanilla(v2, "dsv2_vanilla_160x1536", 160, 6, 1536),
                                  (1, 4, 16, 64))
    km = LayerConfig("kimik2_factored", hidden=7168, n_experts=1280, n_depts=16, top_k=10,
                     top_k_dept=5, d_shared=2048, form="factored", score="sigmoid",
                     renorm=True, sigma="silu", w_dtype="bf16", act_dtype="bf16")
    p["kimik2_factored"] = Workload(km, _vanilla(km, "kimik2_vanilla_384x2048", 384, 8, 2048),
                                    (1, 4, 16, 64))
    return p


PRESETS = _make_presets()


# ----------------------------------------------------------------------------
# weight shapes


def weight_shapes(cfg: LayerConfig) -> dict:
    """[out, in] shapes of every weight tensor, stacked over departments/experts."""
    h, n, m = cfg.hidden, cfg.n_experts, cfg.n_depts
    d = cfg.d_shared
    s = {"router": (n, h),
         "dept_gate": (m, d, h), "dept_up": (m, d, h), "dept_down": (m, h, d)}
    if cfg.form == "factored":
        s.update(priv_gate=(n, d, d), priv_up=(n, d, d), priv_down=(n, d, d))
    elif cfg.d_private > 0:
        p = cfg.d_private
        s.update(priv_gate=(n, p, h), priv_up=(n, p, h), priv_down=(n, h, p))
    if cfg.d_shared_expert > 0:
        e = cfg.d_shared_expert
        s.update(se_gate=(e, h), se_up=(e, h), se_down=(h, e))
    return s


EXPERT_KEYS = ("dept_gate", "dept_up", "dept_down", "priv_gate", "priv_up", "priv_down",
               "se_gate", "se_up", "se_down")


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _quant_fp8_blocks(w: torch.Tensor):
    """[.., out, in] fp32 -> (e4m3 codes as uint8, fp32 scales [.., ceil(out/128), ceil(in/128)])."""
    *lead, R, C = w.shape
    Rb, Cb = -(-R // FP8_BLOCK), -(-C // FP8_BLOCK)
    pad = torch.zeros(*lead, Rb * FP8_BLOCK, Cb * FP8_BLOCK, dtype=torch.float32, device=w.device)
    pad[..., :R, :C] = w
    blk = pad.reshape(*lead, Rb, FP8_BLOCK, Cb, FP8_BLOCK)
    amax = blk.abs().amax(dim=(-3, -1))                       # [.., Rb, Cb]
    scale = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax))
    q = (blk / scale[..., :, None, :, None]).clamp_(-FP8_MAX, FP8_MAX)
    codes = q.reshape(*lead, Rb * FP8_BLOCK, Cb * FP8_BLOCK)[..., :R, :C]
    codes = codes.contiguous().to(torch.float8_e4m3fn).view(torch.uint8)
    return codes, scale.contiguous()


def gate_exact_scale(hidden: int) -> float:
    """Power of two near 4*sqrt(h): router weights are integers over this scale."""
    return float(2 ** round(math.log2(4.0 * math.sqrt(hidden))))


def make_weights(cfg: LayerConfig, seed: int = 0, device="cpu", gate_exact: bool = False,
                 identity_private: bool = False) -> dict:
    """Draw every weight of the layer.

    Draw order: router, department gate/up/down, private gate/up/down, shared
    expert.  Returns tensors in storage dtype; fp8 matrices come as uint8 codes
    with a companion '<key>_scale' fp32 tensor.

    gate_exact: router weights are integers |q| <= 15 over 2^s ~ 4 sqrt(h), so
    that (with gate-exact tokens) every logit is exact in fp32 whatever the
    summation order.
    identity_private: FACTORED only, every private A matrix is the identity
    (the paper's identity initialisation, Sec. 3.4).
    """
    g = _gen(seed, device)
    shapes = weight_shapes(cfg)
    out = {}
    act = _TORCH_DTYPE[cfg.act_dtype]
    for key, shp in shapes.items():
        fan_in = shp[-1]
        w = torch.randn(*shp, generator=g, device=device, dtype=torch.float32)
        w.mul_(1.0 / math.sqrt(fan_in))
        if key == "router":
            if gate_exact:
                sc = gate_exact_scale(cfg.hidden)
                w = torch.round(w * sc).clamp_(-15, 15) / sc
            out[key] = w.to(act).contiguous()
            continue
        if identity_private and key.startswith("priv_"):
            assert cfg.form == "factored"
            w = torch.eye(shp[-1], device=device).expand(*shp).contiguous()
        if cfg.w_dtype == "fp8":
            codes, scale = _quant_fp8_blocks(w)
            out[key] = codes
            out[key + "_scale"] = scale
        else:
            out[key] = w.to(_TORCH_DTYPE[cfg.w_dtype]).contiguous()
        del w
    return out


def make_tokens(cfg: LayerConfig, T: int, seed: int = 0, device="cpu",
                gate_exact: bool = False) -> torch.Tensor:
    """x [T, h] ~ N(0, 1) in the activation dtype (gate_exact: on a 1/8 grid, |x| <= 4)."""
    g = _gen(seed + 1_000_003, device)
    x = torch.randn(T, cfg.hidden, generator=g, device=device, dtype=torch.float32)
    if gate_exact:
        x = torch.round(x * 8.0).clamp_(-32, 32) / 8.0
    return x.to(_TORCH_DTYPE[cfg.act_dtype]).contiguous()


def make_logits(cfg: LayerConfig, T: int, seed: int = 0, kind: str = "uniform",
                device="cpu", bias: torch.Tensor | None = None) -> torch.Tensor:
    """Injected router logits [T, n] fp32.

    uniform: i.i.d. U(0, 1).
    gumbel:  i.i.d. Gumbel(0, 1) plus an optional per-expert offset; top-k of
             Gumbel + log w draws k experts without replacement with probability
             proportional to w.
    """
    g = _gen(seed + 2_000_003, device)
    u = torch.rand(T, cfg.n_experts, generator=g, device=device, dtype=torch.float32)
    if kind == "uniform":
        return u.contiguous()
    if kind == "gumbel":
        u = u.clamp_(1e-12, 1.0 - 1e-7)
        l = -torch.log(-torch.log(u))
        if bias is not None:
            l = l + bias.to(device)
        return l.contiguous()
    raise ValueError(kind)


def make_zipf_bias(cfg: LayerConfig, seed: int = 0, s: float = 1.2) -> torch.Tensor:
    """Per-expert fp32 router bias b_e = log w_dept(e), w_j proportional to rank_j^-s.

    Department ranks come from a seeded permutation, so the popular departments
    are not simply the first ones.
    """
    g = _gen(seed + 3_000_003, "cpu")
    m, E = cfg.n_depts, cfg.experts_per_dept
    rank = torch.empty(m, dtype=torch.float64)
    rank[torch.randperm(m, generator=g)] = torch.arange(1, m + 1, dtype=torch.float64)
    w = rank.pow(-s)
    w = w / w.sum()
    return torch.log(w).repeat_interleave(E).to(torch.float32).contiguous()
