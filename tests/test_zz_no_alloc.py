"""deamoe_layer_forward_noalloc, the entry point for callers that cannot
allocate: the library's own per-GPU scratch array in place of a caller
workspace.  Its outputs and routing must be bit-identical to
deamoe_layer_forward's on the same inputs (same kernels), on calls in a row
whose later ones are smaller and of another shape, so that the array holds
the previous call's contents when the next one starts."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_util import say  # noqa: E402
from paper_2608_14385_amd import deamoe as D  # noqa: E402
from paper_2608_14385_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.contiguous().view(torch.uint8)


def _both(cfg, w: dict, T: int, max_tokens: int, seed: int):
    """The layer through the workspace call and through the no-alloc call."""
    c = D.make_config(cfg, max_tokens)
    Wt = D.make_weights(w)
    x = W.make_tokens(cfg, T, seed, device="cuda")
    ws = D.alloc_workspace(c)
    rt_a, rt_b = D.Routing.alloc(cfg, T), D.Routing.alloc(cfg, T)
    y_a = torch.full_like(x, float("nan"))
    y_b = torch.full_like(x, float("nan"))
    D.deamoe_layer_forward(c, x, Wt, y_a, ws, routing=rt_a)
    D.deamoe_layer_forward_noalloc(c, x, Wt, y_b, routing=rt_b)
    torch.cuda.synchronize()
    assert torch.equal(_bits(y_a), _bits(y_b)), f"{cfg.name} T={T}: outputs differ"
    for key, v in rt_a.tensors.items():
        assert torch.equal(_bits(v), _bits(rt_b.tensors[key])), f"{cfg.name} T={T}: {key} differs"


def test_noalloc_matches_workspace_call():
    dsv3 = W.PRESETS["dsv3_bf16"].layer
    w = W.make_weights(dsv3, 7, device="cuda")
    for T, seed in ((64, 8), (9, 9)):   # second call smaller, same layer
        say(f"[gpu] no-alloc dsv3_bf16 T={T}")
        _both(dsv3, w, T, 64, seed)
    del w
    torch.cuda.empty_cache()
    tiny = W.PRESETS["tiny_factored"].layer   # then another shape and form
    say("[gpu] no-alloc tiny_factored T=3")
    _both(tiny, W.make_weights(tiny, 10, device="cuda"), 3, 4, 11)


def test_noalloc_rejects_oversize_workspace():
    cfg = W.PRESETS["dsv3_bf16"].layer.replace(hidden=14336)
    c = D.make_config(cfg, 128)
    assert D.workspace_bytes(c) > D.SCRATCH_BYTES
    with pytest.raises(D.DeamoeError) as e:
        D.deamoe_layer_forward_noalloc(c, torch.zeros(1, 14336, dtype=torch.bfloat16,
                                                      device="cuda"), D.deamoe_weights(),
                                       torch.zeros(1, 14336, dtype=torch.bfloat16, device="cuda"))
    assert e.value.status == D.ERR_WORKSPACE
