"""Shared helpers for the GPU parity tests (imported by tests/test_gpu_*.py)."""
from __future__ import annotations

import os

import numpy as np
import pytest
import torch

import oracle
from moe_inputs import as_f64, make_inputs, to_torch

TOL = {"f32": 1e-4, "bf16": 2e-2}  # max relative error: max|g - r| / max|r|


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def dev():
    return torch.device("cuda:0")


def max_rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def elem_rel_err(got, ref) -> float:
    """The element-wise measure reported beside max_rel_err: max_i |g_i - r_i|
    / max(|r_i|, 1e-3 max|r|), which shows errors on small entries that the
    max-normalised measure hides."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    floor = 1e-3 * float(np.max(np.abs(ref)))
    den = np.maximum(np.abs(ref), floor)
    if floor == 0.0:
        den = np.where(den == 0.0, 1.0, den)
    return float(np.max(np.abs(got - ref) / den))


# every assert_close of this session: (test, what, dtype, max-normalised, element-wise)
REPORT: list = []


def assert_close(got, ref, dtype: str, what: str, tol: float | None = None):
    t = TOL[dtype] if tol is None else tol
    err = max_rel_err(got, ref)
    REPORT.append((os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], what, dtype, err,
                   elem_rel_err(got, ref)))
    assert err <= t, f"{what}: max rel err {err:.3e} > {t:.1e}"


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float64 numpy (bf16 widened exactly)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        t = t.float()
    if t.dtype in (torch.int32, torch.int64):
        return t.numpy().astype(np.int64)
    return t.numpy().astype(np.float64)


def load_layer(layer, inp):
    """Copy generator inputs (storage form) into a MoELayer's tensors."""
    d = layer.x.device
    layer.x.copy_(to_torch(inp["x"], d))
    layer.w_gate.copy_(to_torch(inp["w_gate"], d))
    if inp.get("bias") is not None:
        layer.bias.copy_(torch.from_numpy(inp["bias"]).to(d))
    layer.w1.copy_(to_torch(inp["w1"], d))
    if inp.get("w3") is not None:
        layer.w3.copy_(to_torch(inp["w3"], d))
    layer.w2.copy_(to_torch(inp["w2"], d))
    if inp.get("dy") is not None:
        layer.dy.copy_(to_torch(inp["dy"], d))
    for name in ("b1", "b3", "b2"):  # the experts' biases (fp32)
        if inp.get(name) is not None:
            getattr(layer, name).copy_(torch.from_numpy(inp[name]).to(d))


def f64_inputs(inp):
    return {k: (None if v is None else (v.astype(np.float64) if v.dtype == np.float32 and
                                        k in ("bias", "b1", "b3", "b2") else as_f64(v)))
            for k, v in inp.items()}


def near_tie_check(own_logits, gpu_logits, gpu_idx, k):
    """The oracle's own routing (its fp64 logits) against the GPU's (its fp32
    logits): routing is a function of the logits, so the two may differ only
    on tokens whose fp64 logits have a near-tie among their top k + 1, a gap
    between consecutive sorted logits below 4 max|l_gpu - l_own|. Returns
    (tokens routed differently, tokens with such a near-tie, the bound);
    asserts that every differing token is a near-tie."""
    import oracle as _or
    own_logits = np.asarray(own_logits, dtype=np.float64)
    delta = float(np.max(np.abs(np.asarray(gpu_logits, dtype=np.float64) - own_logits)))
    bound = 4.0 * delta
    own_idx, _ = _or.topk_select(own_logits, k)
    srt = -np.sort(-own_logits, axis=1)[:, :min(k + 1, own_logits.shape[1])]
    gaps = srt[:, :-1] - srt[:, 1:] if srt.shape[1] > 1 else np.full((srt.shape[0], 1), np.inf)
    near = np.min(gaps, axis=1) < bound
    diff = np.any(np.asarray(gpu_idx) != own_idx, axis=1)
    assert not np.any(diff & ~near), (
        f"{int(np.sum(diff & ~near))} token(s) routed differently without a near-tie "
        f"(bound {bound:.3e})")
    return int(diff.sum()), int(near.sum()), bound


def oracle_for_layer(layer_inp64, cfg, R, layout, gpu_logits):
    """Oracle of the whole layer with routing taken from the GPU logits."""
    return oracle.layer_fwd_bwd(layer_inp64, k=cfg.k, f=cfg.f, act=cfg.act, R=R, layout=layout,
                                logits_for_routing=gpu_logits, gate=cfg.gate)


__all__ = ["TOL", "need_gpu", "dev", "max_rel_err", "elem_rel_err", "REPORT", "assert_close", "host", "load_layer",
           "f64_inputs", "oracle_for_layer", "make_inputs", "near_tie_check"]
