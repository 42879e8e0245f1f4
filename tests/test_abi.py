"""The C ABI on the host: exports, validation before any launch, accounting.

No call here reaches a kernel launch: every call is rejected by validation or
has T == 0, so the tests run without a GPU.
"""
import ctypes as C
import os
import re
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import oracle_pins  # noqa: E402
from paper_2608_14385_amd import deamoe as D  # noqa: E402
from paper_2608_14385_amd import workloads as W  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7f0000000000  # never dereferenced: validation rejects first


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(D.LIB_PATH):
        from paper_2608_14385_amd import build
        build.build()


def header_functions():
    src = open(os.path.join(ROOT, "include", "deamoe.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(deamoe_\w+)\s*\(", src, re.M)))


def test_exports_match_header():
    declared = header_functions()
    assert declared, "no declarations parsed"
    assert sorted(D.EXPORTS) == declared
    L = D.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings():
    for s in (D.OK, D.ERR_INVALID, D.ERR_UNSUPPORTED, D.ERR_WORKSPACE, D.ERR_HIP):
        assert D.status_string(s)
    assert D.status_string(12345) == "unknown status"


def cfg_c3(**kw):
    return D.make_config(W.PRESETS["dsv3_bf16"].layer.replace(**kw), 64)


def ws_status(c):
    n = C.c_size_t(0)
    return D.lib().deamoe_workspace_bytes(C.byref(c) if c is not None else None, C.byref(n)), n.value


@pytest.mark.parametrize("mut,expect", [
    (dict(n_depts=7), D.ERR_INVALID),                       # n % m != 0
    (dict(top_k=0), D.ERR_INVALID),
    (dict(top_k=300), D.ERR_INVALID),                        # k > n
    (dict(top_k_dept=1), D.ERR_INVALID),                     # k > k_dept * E_d (8 > 1 * 8 is ok) -> see below
    (dict(top_k_dept=40), D.ERR_INVALID),                    # k_dept > m
    (dict(d_shared=0), D.ERR_INVALID),
    (dict(d_private=-1), D.ERR_INVALID),
    (dict(score="softmax", renorm=False), D.OK),
    (dict(hidden=7168 + 64), D.ERR_UNSUPPORTED),             # not a multiple of 128 (bf16)
    (dict(d_private=192), D.ERR_UNSUPPORTED),
    (dict(w_dtype="f32"), D.ERR_UNSUPPORTED),                # fp32 weights with bf16 activations
    (dict(n_experts=4096, n_depts=32), D.ERR_UNSUPPORTED),
    (dict(top_k=40), D.ERR_UNSUPPORTED),
    (dict(hidden=65536 + 128), D.ERR_UNSUPPORTED),           # beyond DEAMOE_MAX_WIDTH
    (dict(d_shared=65536 + 128), D.ERR_UNSUPPORTED),
    (dict(top_k_dept=4, dept_cover=1), D.OK),
    (dict(dept_cover=1), D.ERR_INVALID),                     # strict coverage needs top_k_dept > 0
    (dict(top_k_dept=9, n_depts=32, top_k=8, dept_cover=1), D.ERR_INVALID),   # k < k_dept
    (dict(sigma="gelu"), D.OK),
    (dict(sigma="rmsnorm"), D.OK),
    (dict(w_dtype="fp8", hidden=8192), D.OK),
    (dict(w_dtype="fp8", hidden=8192 + 128), D.ERR_UNSUPPORTED),   # more than 64 fp8 scale blocks
    (dict(w_dtype="fp8", d_shared=8192 + 128), D.ERR_UNSUPPORTED),
    (dict(hidden=8192 + 128), D.OK),                                # bf16 has no such limit
])
def test_config_validation(mut, expect):
    if mut == dict(top_k_dept=1):
        mut = dict(top_k_dept=1, top_k=9)                    # 9 > 1 * 8
    st, _ = ws_status(cfg_c3(**mut))
    assert st == expect, (mut, D.status_string(st))


def test_config_validation_struct_fields():
    c = cfg_c3()
    assert ws_status(c)[0] == D.OK
    for field, val, expect in [("max_tokens", 0, D.ERR_INVALID), ("max_tokens", 129, D.ERR_UNSUPPORTED),
                               ("form", 5, D.ERR_INVALID), ("score", 2, D.ERR_INVALID),
                               ("renorm", 3, D.ERR_INVALID), ("sigma", 9, D.ERR_INVALID),
                               ("sigma", -1, D.ERR_INVALID), ("dept_cover", 2, D.ERR_INVALID),
                               ("w_dtype", 7, D.ERR_INVALID), ("act_dtype", 2, D.ERR_INVALID)]:
        c = cfg_c3()
        setattr(c, field, val)
        assert ws_status(c)[0] == expect, field
    c = cfg_c3()
    c.route_scale = float("nan")
    assert ws_status(c)[0] == D.ERR_INVALID
    assert D.lib().deamoe_workspace_bytes(None, None) == D.ERR_INVALID


def test_workspace_grows_with_tokens():
    cfg = W.PRESETS["dsv3_bf16"].layer
    sizes = [D.workspace_bytes(D.make_config(cfg, T)) for T in (1, 16, 128)]
    assert sizes[0] < sizes[1] < sizes[2]
    assert sizes[2] < 256 << 20   # modest next to 288 GB


def weights_struct(cfg):
    Wt = D.deamoe_weights()
    for k in W.weight_shapes(cfg):
        setattr(Wt, k, FAKE)
    if cfg.w_dtype == "fp8":
        for i in range(9):
            Wt.scale[i] = FAKE
    return Wt


def call_layer(c, T=4, x=FAKE, Wt=None, y=FAKE, ws=FAKE, ws_bytes=None, routing=None, fn=None):
    fn = fn or D.lib().deamoe_layer_forward
    ws_bytes = D.workspace_bytes(c) if ws_bytes is None else ws_bytes
    return fn(C.byref(c), T, x, C.byref(Wt) if Wt is not None else None, None, None,
              C.byref(routing) if routing is not None else None, y, ws, ws_bytes, None)


def test_layer_validation_paths():
    cfg = W.PRESETS["dsv3_bf16"].layer
    c = D.make_config(cfg, 16)
    Wt = weights_struct(cfg)
    assert call_layer(c, T=0, Wt=Wt) == D.OK                     # empty batch: no work
    assert call_layer(c, T=0, Wt=None, x=None, y=None, ws=None) == D.OK
    assert call_layer(c, T=-1, Wt=Wt) == D.ERR_INVALID
    assert call_layer(c, T=17, Wt=Wt) == D.ERR_UNSUPPORTED       # beyond max_tokens
    assert call_layer(c, Wt=None) == D.ERR_INVALID
    assert call_layer(c, Wt=Wt, y=None) == D.ERR_INVALID
    assert call_layer(c, Wt=Wt, x=None) == D.ERR_INVALID
    assert call_layer(c, Wt=Wt, ws=None) == D.ERR_WORKSPACE
    assert call_layer(c, Wt=Wt, ws_bytes=D.workspace_bytes(c) - 1) == D.ERR_WORKSPACE
    assert call_layer(c, Wt=Wt, ws=FAKE + 8) == D.ERR_WORKSPACE   # misaligned
    W2 = weights_struct(cfg)
    W2.priv_up = None
    assert call_layer(c, Wt=W2) == D.ERR_INVALID
    W3 = weights_struct(cfg)
    W3.dept_down = FAKE + 4                                       # misaligned matrix
    assert call_layer(c, Wt=W3) == D.ERR_INVALID
    W4 = weights_struct(cfg)
    W4.router = None                                              # router needed without logits_in
    assert call_layer(c, Wt=W4) == D.ERR_INVALID
    r = D.deamoe_routing()                                        # incomplete routing outputs
    assert call_layer(c, Wt=Wt, routing=r) == D.ERR_INVALID


def test_noalloc_validation_before_any_hip_call():
    """deamoe_layer_forward_noalloc rejects a configuration whose workspace
    exceeds the library's scratch array, and returns for T == 0, before any
    HIP call (so these run without a GPU)."""
    L = D.lib()
    cfg = W.PRESETS["dsv3_bf16"].layer

    def call(c, T):
        return L.deamoe_layer_forward_noalloc(C.byref(c), T, FAKE, None, None, None, None, FAKE,
                                              None)
    big = D.make_config(cfg.replace(hidden=14336), 128)
    assert D.workspace_bytes(big) > D.SCRATCH_BYTES
    assert call(big, 1) == D.ERR_WORKSPACE
    assert call(big, 0) == D.ERR_WORKSPACE
    ok = D.make_config(cfg, 128)
    assert D.workspace_bytes(ok) <= D.SCRATCH_BYTES
    assert call(ok, 0) == D.OK
    assert call(ok, -1) == D.ERR_INVALID
    assert call(ok, 129) == D.ERR_UNSUPPORTED
    assert call(D.make_config(cfg.replace(n_depts=7), 16), 1) == D.ERR_INVALID


def test_fp8_needs_scales():
    cfg = W.PRESETS["dsv3_fp8"].layer
    c = D.make_config(cfg, 4)
    Wt = weights_struct(cfg)
    assert call_layer(c, T=0, Wt=Wt) == D.OK
    Wt.scale[4] = None
    assert call_layer(c, Wt=Wt) == D.ERR_INVALID


def test_baseline_requires_vanilla_shape():
    wl = W.PRESETS["dsv3_bf16"]
    fn = D.lib().deamoe_baseline_forward
    c = D.make_config(wl.layer, 4)
    assert call_layer(c, Wt=weights_struct(wl.layer), fn=fn) == D.ERR_INVALID
    cb = D.make_config(wl.baseline, 4)
    assert call_layer(cb, T=0, Wt=weights_struct(wl.baseline), fn=fn) == D.OK
    assert fn(None, 0, None, None, None, None, None, None, None, 0, None) == D.ERR_INVALID


def test_route_validation():
    cfg = W.PRESETS["dsv3_bf16"].layer
    c = D.make_config(cfg, 8)
    L = D.lib()
    full = D.deamoe_routing(**{f: FAKE for f in D.ROUTING_FIELDS})
    n = D.workspace_bytes(c)
    assert L.deamoe_route(C.byref(c), 0, FAKE, FAKE, None, None, C.byref(full), FAKE, n, None) == D.OK
    assert L.deamoe_route(C.byref(c), 0, None, None, None, None, None, None, 0, None) == D.OK
    assert L.deamoe_route(C.byref(c), 2, None, FAKE, None, None, C.byref(full), FAKE, n, None) == D.ERR_INVALID
    assert L.deamoe_route(C.byref(c), 2, FAKE, FAKE, None, None, None, FAKE, n, None) == D.ERR_INVALID
    assert L.deamoe_route(C.byref(c), 9, FAKE, FAKE, None, None, C.byref(full), FAKE, n, None) == D.ERR_UNSUPPORTED
    assert L.deamoe_route(C.byref(c), 2, FAKE, FAKE, None, None, C.byref(full), FAKE, n - 256, None) == D.ERR_WORKSPACE


@pytest.mark.parametrize("name", ["tiny_f32", "tiny_factored", "7b_bf16", "dsv3_bf16", "dsv3_fp8",
                                  "dsv3_factored"])
def test_loaded_bytes_matches_oracle_accounting(name):
    wl = W.PRESETS[name]
    rng = np.random.default_rng(7)
    for cfg in (wl.layer, wl.baseline):
        c = D.make_config(cfg, 16)
        for _ in range(5):
            dc = (rng.random(cfg.n_depts) < 0.4).astype(np.int32) * rng.integers(1, 5, cfg.n_depts)
            ec = (rng.random(cfg.n_experts) < 0.2).astype(np.int32) * rng.integers(1, 3, cfg.n_experts)
            T = int(rng.integers(0, 17))
            wb, tb = D.deamoe_loaded_bytes(c, T, dc, ec)
            assert wb == oracle.step_weight_bytes(cfg, dc, ec)
            ab = 4 if cfg.act_dtype == "f32" else 2
            assert tb == wb + 2 * T * cfg.hidden * ab


def test_loaded_bytes_monte_carlo_matches_closed_form():
    """Uniform routing of the Table 1 DeepSeek-V3 DeaMoE row: the mean of the
    library's per-step accounting approaches the closed-form expected ratio
    (the one pinned against the Fig. 2 numbers)."""
    (name, kb, h, f, nb, m, n, kd, k, _, _) = oracle_pins._table1()[0]
    dea = W.LayerConfig("mc", hidden=h, n_experts=n, n_depts=m, top_k=k, top_k_dept=kd,
                        d_shared=f, form="factored", w_dtype="bf16", act_dtype="bf16")
    van = W.LayerConfig("mcv", hidden=h, n_experts=nb, n_depts=nb, top_k=kb, d_shared=f,
                        form="slice", w_dtype="bf16", act_dtype="bf16")
    cd, cv = D.make_config(dea, 16), D.make_config(van, 16)
    rng = np.random.default_rng(0)
    E = n // m
    for T in (4, 16):
        tot_d = tot_v = 0
        trials = 400
        for _ in range(trials):
            dc = np.zeros(m, np.int32)
            ec = np.zeros(n, np.int32)
            vc = np.zeros(nb, np.int32)
            for _t in range(T):
                depts = rng.choice(m, kd, replace=False)
                dc[depts] += 1
                ec[rng.choice(n, k, replace=False)] += 1
                vc[rng.choice(nb, kb, replace=False)] += 1
            tot_d += D.deamoe_loaded_bytes(cd, T, dc, ec)[0]
            tot_v += D.deamoe_loaded_bytes(cv, T, vc, vc)[0]
        assert abs(tot_d / tot_v - oracle_pins.expected_ratio(T)) < 0.01, T
    assert E == 108


def test_read_probe_library_exports():
    """The benchmark's read-bandwidth probe loads and exports its one entry point."""
    from paper_2608_14385_amd import build as B
    lib = C.CDLL(B.PROBE_LIB)
    assert hasattr(lib, "deamoe_probe_read")


def test_trace_points():
    """Stage boundaries of the traced call: small batches run the last down
    stage and the combine as one kernel; SLICE batches of at most 4 tokens
    also route inside the gate/up launch."""
    c = cfg_c3()
    assert [D.deamoe_trace_points(c, T) for T in (1, 4, 5, 16, 17, 32, 33, 64)] == \
        [4, 4, 5, 5, 5, 5, 6, 6]
    s7 = D.make_config(W.PRESETS["7b_bf16"].layer, 64)     # h 2048: fused up to 24 tokens
    assert [D.deamoe_trace_points(s7, T) for T in (1, 4, 5, 16, 24, 25)] == [4, 4, 5, 5, 5, 6]
    # routers of more than 1024 experts keep the separate routing kernel
    assert D.deamoe_trace_points(cfg_c3(n_experts=2048, n_depts=32), 1) == 5
    f = D.make_config(W.PRESETS["dsv3_factored"].layer, 64)
    # group-limited routing with long tiles routes inside the first stage
    # only while (nearly) all of its tiles fit in one round (one token here)
    assert [D.deamoe_trace_points(f, T) for T in (1, 2, 4, 5, 16, 17)] == [7, 8, 8, 8, 8, 9]
    q = D.make_config(W.PRESETS["qwen3_factored"].layer, 64)   # h 4096: fused up to 16 tokens
    assert [D.deamoe_trace_points(q, T) for T in (1, 16, 17)] == [7, 8, 9]
    b7 = D.make_config(W.PRESETS["base7b_factored"].layer, 64)   # h 1024: the same
    assert [D.deamoe_trace_points(b7, T) for T in (1, 16, 17)] == [7, 8, 9]
    k2 = D.make_config(W.PRESETS["kimik2_factored"].layer, 64)   # 1280 experts
    assert D.deamoe_trace_points(k2, 1) == 8
    # more active units than the fused kernel's table holds: separate stages
    big = cfg_c3(n_experts=2048, n_depts=64, top_k=32)
    assert [D.deamoe_trace_points(big, T) for T in (8, 16)] == [5, 6]
    # FACTORED fuses up to 16 tokens only
    assert D.deamoe_trace_points(D.make_config(W.PRESETS["kimik2_factored"].layer, 64), 32) == 9
    n = C.c_int32(0)
    for T in (0, 65):
        assert D.lib().deamoe_trace_points(C.byref(c), T, C.byref(n)) == D.ERR_INVALID
    assert D.lib().deamoe_trace_points(C.byref(c), 1, None) == D.ERR_INVALID
