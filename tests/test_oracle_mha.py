"""Pins of the attention part of AT_r in the fp64 oracle (CPU only).

The oracle's MHA (Sec. 2.1: W^Q, W^K, W^V, W^O, heads of width d, scaled
dot-product attention) is checked against what does not share its code:
torch's fp64 scaled_dot_product_attention and its autograd gradients (a
library routine), central finite differences, and closed forms (W^Q = 0
gives uniform attention; one-token sequences give I W^V W^O); the chunked
layer with AT_r = attention + gate against a dense torch formulation of the
whole block.
"""
import math

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
from moe_inputs import as_f64, get_config, make_inputs
from test_oracle_pins import _brute_pos, _small_inputs, _torch_layer_grads  # noqa: F401


@pytest.fixture
def rng():
    return np.random.default_rng(20251000)


def _mha_inputs(rng, T, M, scale=0.4):
    return (rng.standard_normal((T, M)), rng.standard_normal((M, 3 * M)) * scale,
            rng.standard_normal((M, M)) * scale)


def _torch_mha(inp, w_qkv, w_o, seq_len, heads, causal):
    """The block's attention through torch's library routine, fp64."""
    T, M = inp.shape
    d = M // heads
    qkv = inp @ w_qkv
    B = T // seq_len

    def split(a):  # T x M -> B x heads x N x d
        return a.reshape(B, seq_len, heads, d).transpose(1, 2)

    q, k, v = (split(qkv[:, i * M:(i + 1) * M]) for i in range(3))
    a = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal)
    attn = a.transpose(1, 2).reshape(T, M)
    return qkv, attn, attn @ w_o


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("seq_len,heads", [(7, 2), (5, 4), (1, 2), (12, 1)])
def test_mha_forward_matches_torch_sdpa(rng, causal, seq_len, heads):
    M = 8 * heads if heads > 1 else 6
    T = 3 * seq_len
    inp, wqkv, wo = _mha_inputs(rng, T, M)
    ours = oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, causal)
    t = lambda a: torch.tensor(a, dtype=torch.float64)
    qkv, attn, out = _torch_mha(t(inp), t(wqkv), t(wo), seq_len, heads, causal)
    np.testing.assert_allclose(ours["qkv"], qkv.numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(ours["attn"], attn.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(ours["out"], out.numpy(), rtol=1e-12, atol=1e-13)
    # lse: scipy's logsumexp of the visible scores of each (sequence, head, row)
    d = M // heads
    for b in range(T // seq_len):
        for h in range(heads):
            for i in range(seq_len):
                t_i = b * seq_len + i
                js = range(b * seq_len, t_i + 1) if causal else range(b * seq_len, (b + 1) * seq_len)
                s = [qkv[t_i, h * d:(h + 1) * d].numpy() @ qkv[j, M + h * d:M + (h + 1) * d].numpy()
                     / math.sqrt(d) for j in js]
                assert ours["lse"][h, t_i] == pytest.approx(logsumexp(s), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("seq_len,heads", [(6, 2), (4, 1), (9, 3)])
def test_mha_backward_matches_torch_autograd(rng, causal, seq_len, heads):
    M = 4 * heads
    T = 2 * seq_len
    inp, wqkv, wo = _mha_inputs(rng, T, M)
    d_out = rng.standard_normal((T, M))
    ours_f = oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, causal)
    ours = oracle.mha_bwd(inp, wqkv, wo, ours_f, d_out, seq_len, heads, causal)
    leaf = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
    ti, tq, to = leaf(inp), leaf(wqkv), leaf(wo)
    qkv, attn, out = _torch_mha(ti, tq, to, seq_len, heads, causal)
    qkv.retain_grad()
    attn.retain_grad()
    (out * torch.tensor(d_out)).sum().backward()
    for key, ref in (("d_in", ti.grad), ("dw_qkv", tq.grad), ("dw_o", to.grad),
                     ("d_qkv", qkv.grad), ("d_attn", attn.grad)):
        np.testing.assert_allclose(ours[key], ref.numpy(), rtol=1e-11, atol=1e-12, err_msg=key)


@pytest.mark.parametrize("causal", [False, True])
def test_mha_finite_differences(rng, causal):
    seq_len, heads, M, T = 5, 2, 6, 10
    inp, wqkv, wo = _mha_inputs(rng, T, M)
    d_out = rng.standard_normal((T, M))
    loss = lambda i, q, o: float((oracle.mha_fwd(i, q, o, seq_len, heads, causal)["out"]
                                  * d_out).sum())
    g = oracle.mha_bwd(inp, wqkv, wo, oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, causal),
                       d_out, seq_len, heads, causal)
    eps = 1e-6
    for name, arr, grad in (("inp", inp, g["d_in"]), ("w_qkv", wqkv, g["dw_qkv"]),
                            ("w_o", wo, g["dw_o"])):
        for _ in range(6):
            idx = tuple(rng.integers(0, n) for n in arr.shape)
            a_p, a_m = arr.copy(), arr.copy()
            a_p[idx] += eps
            a_m[idx] -= eps
            args_p = {"inp": inp, "w_qkv": wqkv, "w_o": wo}
            args_m = dict(args_p)
            args_p[name], args_m[name] = a_p, a_m
            fd = (loss(args_p["inp"], args_p["w_qkv"], args_p["w_o"])
                  - loss(args_m["inp"], args_m["w_qkv"], args_m["w_o"])) / (2 * eps)
            assert grad[idx] == pytest.approx(fd, rel=1e-6, abs=1e-8), (name, idx)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_queries_give_uniform_attention(rng, causal):
    """W^Q = 0: every score is 0, so each row's weights are uniform over the
    visible tokens: attention = mean of V (prefix mean when causal) and
    lse = log(number of visible tokens)."""
    seq_len, heads, M, T = 6, 2, 8, 12
    inp, wqkv, wo = _mha_inputs(rng, T, M)
    wqkv[:, :M] = 0
    o = oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, causal)
    v = inp @ wqkv[:, 2 * M:]
    for b in range(T // seq_len):
        for i in range(seq_len):
            t = b * seq_len + i
            n_vis = i + 1 if causal else seq_len
            hi = t + 1 if causal else (b + 1) * seq_len
            np.testing.assert_allclose(o["attn"][t], v[b * seq_len:hi].mean(axis=0), rtol=1e-13,
                                       atol=1e-14)
            np.testing.assert_allclose(o["lse"][:, t], math.log(n_vis), rtol=1e-14)


def test_one_token_sequences_are_a_linear_map(rng):
    M, heads = 8, 4
    inp, wqkv, wo = _mha_inputs(rng, 5, M)
    for causal in (False, True):
        o = oracle.mha_fwd(inp, wqkv, wo, 1, heads, causal)
        np.testing.assert_allclose(o["out"], inp @ wqkv[:, 2 * M:] @ wo, rtol=1e-12, atol=1e-14)


def test_bidirectional_attention_is_permutation_equivariant(rng):
    seq_len, heads, M = 7, 2, 8
    inp, wqkv, wo = _mha_inputs(rng, 2 * seq_len, M)
    perm = np.concatenate([rng.permutation(seq_len), seq_len + rng.permutation(seq_len)])
    a = oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, False)
    b = oracle.mha_fwd(inp[perm], wqkv, wo, seq_len, heads, False)
    np.testing.assert_allclose(b["out"], a["out"][perm], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(b["lse"], a["lse"][:, perm], rtol=1e-13)


def test_causal_attention_ignores_later_tokens(rng):
    """Changing token j of a sequence changes no causal output before j."""
    seq_len, heads, M = 8, 2, 8
    inp, wqkv, wo = _mha_inputs(rng, seq_len, M)
    a = oracle.mha_fwd(inp, wqkv, wo, seq_len, heads, True)
    inp2 = inp.copy()
    inp2[5] += 1.0
    b = oracle.mha_fwd(inp2, wqkv, wo, seq_len, heads, True)
    np.testing.assert_array_equal(a["out"][:5], b["out"][:5])
    assert np.abs(a["out"][5:] - b["out"][5:]).min() > 0


# ---------------------------------------------------------------------------
# the chunked layer with AT_r = attention + gate (Sec. 3.2)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_layer_with_attention_matches_torch_block(rng, causal, act):
    """Attention (torch SDPA) then the dense masked MoE formulation, one
    autograd graph: y, the block input's gradient and every weight gradient."""
    seq_len, heads, M, H, E, k = 6, 2, 8, 6, 4, 2
    T = 4 * seq_len
    inp = _small_inputs(rng, T, M, H, E, act)
    inp["mha_in"], inp["w_qkv"], inp["w_o"] = _mha_inputs(rng, T, M, 0.3)
    mha = dict(seq_len=seq_len, heads=heads, causal=causal)
    for R, f in ((1, 1.0), (2, 1.0), (2, float(E))):
        out = oracle.layer_fwd_bwd(inp, k=k, f=f, act=act, R=R, mha=mha)
        Tr = T // R
        for r in range(R):
            sl = slice(r * Tr, (r + 1) * Tr)
            leaf = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
            ti, tq, to = leaf(inp["mha_in"][sl]), leaf(inp["w_qkv"]), leaf(inp["w_o"])
            _, _, x = _torch_mha(ti, tq, to, seq_len, heads, causal)
            sub = dict(inp, x=x.detach().numpy(), dy=inp["dy"][sl])
            ref = _torch_layer_grads(sub, k, out["C"], act, x=x)
            np.testing.assert_allclose(out["x"][sl], x.detach().numpy(), rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(out["y"][sl], ref["y"], rtol=1e-11, atol=1e-12)
            np.testing.assert_allclose(out["d_in"][sl], ti.grad.numpy(), rtol=1e-10, atol=1e-12)
            c = out["chunks"][r]
            np.testing.assert_allclose(c["dx"], x.grad.numpy(), rtol=1e-10, atol=1e-12)
        if R == 1:
            np.testing.assert_allclose(out["dw_qkv"], tq.grad.numpy(), rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(out["dw_o"], to.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_layer_with_attention_chunked_equals_unchunked_without_drops(rng):
    seq_len, heads, M, H, E, k = 4, 2, 8, 6, 4, 2
    T = 4 * seq_len
    inp = _small_inputs(rng, T, M, H, E, "swiglu")
    inp["mha_in"], inp["w_qkv"], inp["w_o"] = _mha_inputs(rng, T, M, 0.3)
    mha = dict(seq_len=seq_len, heads=heads, causal=True)
    one = oracle.layer_fwd_bwd(inp, k=k, f=float(E), act="swiglu", R=1, mha=mha)
    many = oracle.layer_fwd_bwd(inp, k=k, f=float(E), act="swiglu", R=4, mha=mha)
    for key in ("x", "y", "d_in", "dw_qkv", "dw_o", "dw1", "dw3", "dw2", "dw_gate"):
        np.testing.assert_allclose(many[key], one[key], rtol=1e-12, atol=1e-12, err_msg=key)
    assert many["lse"].shape == (4, heads, T // 4)


def test_mha_inputs_recipe():
    cfg = get_config("balanced", mha=True, T=1024)
    a = make_inputs(cfg, with_dy=False)
    assert a["mha_in"].shape == (1024, 1024) and a["w_qkv"].shape == (1024, 3072)
    assert a["w_o"].shape == (1024, 1024) and a["w_qkv"].dtype == np.uint16
    assert cfg.heads == 16 and cfg.seq_len == 512 and not cfg.causal
    w = as_f64(a["w_qkv"])
    assert abs(w.std() - 0.02) < 1e-3 and abs(as_f64(a["mha_in"]).std() - 1) < 1e-2
    b = make_inputs(cfg.replace(mha=False), with_dy=False)
    np.testing.assert_array_equal(a["x"], b["x"])  # the other tensors' streams are unchanged
    assert "mha_in" not in b
