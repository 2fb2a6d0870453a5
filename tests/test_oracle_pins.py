"""Pins of the fp64 oracle against things other than itself: a hand-worked
example, brute force on tiny inputs, closed forms, special cases that reduce
to textbook results, and an independent torch-fp64 autograd formulation.
Runs on the CPU only."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from scipy.special import softmax

import oracle
from moe_inputs import as_f64, get_config, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# capacity
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,E,k,f,C", [
    (256, 4, 2, 1.25, 160),      # tiny
    (4096, 8, 2, 1.2, 1229),     # 1228.8 rounds up
    (8192, 16, 1, 1.0, 512),
    (16384, 8, 2, 1.25, 5120),
    (4096, 64, 6, 1.5, 576),     # one of R = 4 chunks of 16384 tokens
    (500, 10, 2, 1.1, 110),      # exactly 110; naive float gives 110.00000000000001
    (3, 2, 1, 1.0, 2),
    (1, 64, 1, 1.0, 1),
    (4, 3, 2, 0.75, 2),
])
def test_capacity_hand_worked(T, E, k, f, C):
    assert oracle.capacity(T, E, k, f) == C


def test_capacity_is_least_integer_bound():
    # C is the least integer with C*E >= f*k*T, f = p/q as written in decimal
    for p in range(10, 16):
        f = p / 10
        for T in (1, 7, 64, 300, 4096):
            for E in (1, 3, 8, 64):
                for k in (1, 2, 6):
                    C = oracle.capacity(T, E, k, f)
                    assert C * E * 10 >= p * k * T
                    assert (C - 1) * E * 10 < p * k * T


# ---------------------------------------------------------------------------
# top-k selection and gate weights
# ---------------------------------------------------------------------------
def _key_beats(l, a, b):
    """a precedes b in the selection order: larger logit, then lower index."""
    return l[a] > l[b] or (l[a] == l[b] and a < b)


def test_topk_brute_force_with_ties(rng):
    for E in (1, 2, 3, 5, 6):
        for k in range(1, E + 1):
            # quantised logits force many ties; include signed zeros
            L = rng.integers(-2, 3, size=(40, E)).astype(np.float64) * 0.5
            L[L == 0] = rng.choice([0.0, -0.0], size=int((L == 0).sum()))
            idx, w = oracle.topk_select(L, k)
            for t in range(L.shape[0]):
                l = L[t]
                good = [S for S in itertools.combinations(range(E), k)
                        if all(_key_beats(l, a, b) for a in S for b in range(E) if b not in S)]
                assert len(good) == 1
                assert sorted(idx[t]) == sorted(good[0])
                for j in range(k - 1):
                    assert _key_beats(l, idx[t, j], idx[t, j + 1])


def test_topk_weights_closed_forms(rng):
    L = rng.standard_normal((64, 8)) * 3
    for k in (1, 2, 5, 8):
        idx, w = oracle.topk_select(L, k)
        np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-15)
        p = softmax(L, axis=1)
        for t in range(L.shape[0]):
            ps = p[t, idx[t]]
            np.testing.assert_allclose(w[t], ps / ps.sum(), rtol=1e-13, atol=0)
        if k == 1:
            assert np.all(w == 1.0)
    # k = 2: w0 is the logistic function of the logit gap
    idx, w = oracle.topk_select(L, 2)
    gap = L[np.arange(64), idx[:, 0]] - L[np.arange(64), idx[:, 1]]
    np.testing.assert_allclose(w[:, 0], 1.0 / (1.0 + np.exp(-gap)), rtol=1e-14)


def test_zero_token_routes_to_first_k_experts():
    cfg = get_config("tiny", T=8)
    inp = make_inputs(cfg, x_zero_rows=[0, 5])
    l = oracle.gate_logits(as_f64(inp["x"]), as_f64(inp["w_gate"]), None)
    assert np.all(l[0] == 0) and np.all(l[5] == 0)
    idx, w = oracle.topk_select(l, 3)
    for t in (0, 5):
        assert list(idx[t]) == [0, 1, 2]
        np.testing.assert_allclose(w[t], 1.0 / 3.0, rtol=1e-15)


# ---------------------------------------------------------------------------
# route: positions, counts, offsets, slot, row_src
# ---------------------------------------------------------------------------
def test_route_hand_worked_example():
    d = json.load(open(os.path.join(GOLDEN, "route_worked_example.json")))
    L = np.array(d["logits"], dtype=np.float64)
    # the -0.0 entry must survive JSON: rebuild it explicitly
    L[2, 1] = -0.0
    idx, _ = oracle.topk_select(L, d["k"])
    assert idx.tolist() == d["topk_idx"]
    for case in d["cases"]:
        assert oracle.capacity(d["T"], d["E"], d["k"], case["f"]) == case["C"]
        rt = oracle.route(idx, d["E"], case["C"], case["layout"])
        assert rt["pos"].tolist() == d["pos"]
        assert rt["demand"].tolist() == d["demand"]
        assert rt["counts"].tolist() == case["counts"]
        assert rt["offsets"].tolist() == case["offsets"]
        assert rt["slot"].tolist() == case["slot"]
        assert rt["row_src"].tolist() == case["row_src"]


def _brute_pos(idx):
    T, k = idx.shape
    pos = np.zeros_like(idx)
    for t in range(T):
        for j in range(k):
            e = idx[t, j]
            pos[t, j] = sum(1 for t2 in range(T) for j2 in range(k)
                            if idx[t2, j2] == e and (j2 < j or (j2 == j and t2 < t)))
    return pos


@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_route_brute_force_and_invariants(rng, layout):
    for (T, E, k) in [(1, 1, 1), (5, 3, 2), (17, 4, 3), (24, 8, 8), (30, 6, 1)]:
        L = rng.standard_normal((T, E))
        idx, _ = oracle.topk_select(L, k)
        for C in sorted({0, 1, 2, max(1, T * k // E), T * k, T * k + 3}):
            rt = oracle.route(idx, E, C, layout)
            assert np.array_equal(rt["pos"], _brute_pos(idx))
            kept = rt["pos"] < C
            assert np.array_equal(rt["kept"], kept)
            for t in range(T):
                assert len(set(idx[t].tolist())) == k          # k distinct experts
            assert np.all(rt["counts"] <= C)
            assert rt["counts"].sum() == kept.sum()
            for e in range(E):
                assert rt["counts"][e] == min(C, int((idx == e).sum()))
            # row_src o slot = id on kept assignments; the rest of row_src is -1
            live = rt["row_src"] >= 0
            assert live.sum() == kept.sum()
            for t in range(T):
                for j in range(k):
                    if kept[t, j]:
                        r = rt["slot"][t, j]
                        assert rt["row_src"][r] == t * k + j
                        e = idx[t, j]
                        assert rt["offsets"][e] <= r < rt["offsets"][e] + rt["counts"][e]
                    else:
                        assert rt["slot"][t, j] == -1
            if C >= T * k:
                assert kept.all()
            if C == 0:
                assert not kept.any()
            if layout == "padded":
                assert rt["rows"] == E * C
                assert rt["offsets"].tolist() == [e * C for e in range(E + 1)]
            else:
                assert rt["rows"] == min(T * k, E * C)
                assert rt["offsets"][E] == kept.sum()


# ---------------------------------------------------------------------------
# activations: closed-form derivatives vs finite differences and torch
# ---------------------------------------------------------------------------
def test_activation_derivatives():
    z = np.linspace(-8, 8, 2001)
    h = 1e-6
    np.testing.assert_allclose(oracle.gelu_grad(z), (oracle.gelu(z + h) - oracle.gelu(z - h)) / (2 * h),
                               atol=1e-8)
    np.testing.assert_allclose(oracle.silu_grad(z), (oracle.silu(z + h) - oracle.silu(z - h)) / (2 * h),
                               atol=1e-8)
    zt = torch.tensor(z, dtype=torch.float64)
    np.testing.assert_allclose(oracle.gelu(z), torch.nn.functional.gelu(zt).numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(oracle.silu(z), torch.nn.functional.silu(zt).numpy(), rtol=1e-14, atol=1e-15)
    # gelu(0) = silu(0) = 0 makes empty (zero) rows map to zero
    assert oracle.gelu(np.zeros(1))[0] == 0 and oracle.silu(np.zeros(1))[0] == 0


# ---------------------------------------------------------------------------
# dispatch / combine special cases
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_dispatch_copy_and_identity_combine(rng, layout):
    T, M, E, k = 40, 16, 5, 2
    x = rng.standard_normal((T, M))
    L = rng.standard_normal((T, E))
    idx, w = oracle.topk_select(L, k)
    for C in (3, 8, T * k):
        rt = oracle.route(idx, E, C, layout)
        xd = oracle.dispatch(x, rt["row_src"], k)
        for r, s in enumerate(rt["row_src"]):
            if s >= 0:
                assert np.array_equal(xd[r], x[s // k])
            else:
                assert not xd[r].any()
        y = oracle.combine(xd, rt["slot"], w)           # identity experts
        wk = (w * rt["kept"]).sum(axis=1)
        np.testing.assert_allclose(y, wk[:, None] * x, rtol=1e-14, atol=1e-14)
        if C >= T * k:
            np.testing.assert_allclose(y, x, rtol=1e-14, atol=1e-14)


def _ffn_dense(x, w1, w3, w2, act):
    h1 = x @ w1
    if act == "gelu":
        a = oracle.gelu(h1)
    else:
        a = oracle.silu(h1) * (x @ w3)
    return a @ w2


@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_k_equals_E_is_dense_softmax_mixture(rng, act):
    T, M, H, E = 12, 8, 6, 4
    x = rng.standard_normal((T, M))
    wg = rng.standard_normal((M, E)) * 0.5
    b = rng.standard_normal(E) * 0.1
    w1 = rng.standard_normal((E, M, H)) * 0.3
    w3 = rng.standard_normal((E, M, H)) * 0.3 if act == "swiglu" else None
    w2 = rng.standard_normal((E, H, M)) * 0.3
    inp = dict(x=x, w_gate=wg, bias=b, w1=w1, w3=w3, w2=w2, dy=None)
    out = oracle.layer_fwd_bwd(inp, k=E, f=float(E), act=act)
    p = softmax(x @ wg + b, axis=1)
    ref = sum(p[:, e:e + 1] * _ffn_dense(x, w1[e], None if w3 is None else w3[e], w2[e], act)
              for e in range(E))
    np.testing.assert_allclose(out["y"], ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------------------
# gradients: independent torch fp64 autograd of a dense masked formulation
# ---------------------------------------------------------------------------
def _torch_layer_grads(inp, k, C, act, gate="renorm", x=None):
    """Dense masked layer in torch fp64: the selection (torch.topk on
    continuous logits) and the keep mask (brute-force position count) are
    constants; y_t = sum_e keep_te * g_te * FFN_e(x_t) with g = softmax_S(l_t)
    (softmax over the selected logits) or, gate="full", softmax(l_t) over all
    experts masked to the selection. ``x``: a torch tensor to use as the
    layer input (computed from other leaves; its gradient is kept)."""
    t64 = lambda a: None if a is None else torch.tensor(a, dtype=torch.float64, requires_grad=True)
    if x is None:
        x = t64(inp["x"])
    else:
        x.retain_grad()
    wg, w1, w2 = t64(inp["w_gate"]), t64(inp["w1"]), t64(inp["w2"])
    w3 = t64(inp["w3"])
    b1, b3, b2 = t64(inp.get("b1")), t64(inp.get("b3")), t64(inp.get("b2"))
    b = t64(inp["bias"]) if inp["bias"] is not None else None
    T, E = x.shape[0], wg.shape[1]
    l = x @ wg + (b if b is not None else 0)
    sel = torch.topk(l.detach(), k, dim=1).indices.numpy()
    pos = _brute_pos(sel)
    sel_mask = torch.zeros(T, E, dtype=torch.float64)
    keep = torch.zeros(T, E, dtype=torch.float64)
    for t in range(T):
        for j in range(k):
            sel_mask[t, sel[t, j]] = 1
            if pos[t, j] < C:
                keep[t, sel[t, j]] = 1
    if gate == "full":
        g = torch.softmax(l, dim=1) * sel_mask * keep
    else:
        lm = l.masked_fill(sel_mask == 0, float("-inf"))
        g = torch.softmax(lm, dim=1) * keep
    y = torch.zeros_like(x)
    for e in range(E):
        h1 = x @ w1[e] + (b1[e] if b1 is not None else 0)
        if act == "gelu":
            a = torch.nn.functional.gelu(h1)
        else:
            a = torch.nn.functional.silu(h1) * (x @ w3[e] + (b3[e] if b3 is not None else 0))
        y = y + g[:, e:e + 1] * (a @ w2[e] + (b2[e] if b2 is not None else 0))
    dy = torch.tensor(inp["dy"], dtype=torch.float64)
    (y * dy).sum().backward()
    res = dict(y=y.detach().numpy(), dx=x.grad.numpy(), dw_gate=wg.grad.numpy(),
               dw1=w1.grad.numpy(), dw2=w2.grad.numpy())
    if w3 is not None:
        res["dw3"] = w3.grad.numpy()
    if b is not None:
        res["dbias"] = b.grad.numpy()
    for name, p in (("db1", b1), ("db3", b3), ("db2", b2)):
        if p is not None:
            res[name] = p.grad.numpy()
    return res


def _small_inputs(rng, T, M, H, E, act, bias=True, expert_bias=False):
    inp = dict(
        x=rng.standard_normal((T, M)),
        w_gate=rng.standard_normal((M, E)) * 0.3,
        bias=rng.standard_normal(E) * 0.2 if bias else None,
        w1=rng.standard_normal((E, M, H)) * 0.3,
        w3=rng.standard_normal((E, M, H)) * 0.3 if act == "swiglu" else None,
        w2=rng.standard_normal((E, H, M)) * 0.3,
        dy=rng.standard_normal((T, M)),
    )
    if expert_bias:
        inp.update(b1=rng.standard_normal((E, H)) * 0.3,
                   b3=rng.standard_normal((E, H)) * 0.3 if act == "swiglu" else None,
                   b2=rng.standard_normal((E, M)) * 0.3)
    return inp


@pytest.mark.parametrize("expert_bias", [False, True])
@pytest.mark.parametrize("gate", ["renorm", "full"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
@pytest.mark.parametrize("f", [0.5, 1.0, 4.0])
def test_layer_grads_match_torch_autograd(rng, act, layout, f, gate, expert_bias):
    T, M, H, E, k = 24, 8, 12, 4, 2
    inp = _small_inputs(rng, T, M, H, E, act, expert_bias=expert_bias)
    out = oracle.layer_fwd_bwd(inp, k=k, f=f, act=act, layout=layout, gate=gate)
    ref = _torch_layer_grads(inp, k, out["C"], act, gate)
    assert ("db1" in ref) == expert_bias and ("db2" in out) == expert_bias
    for key in ref:
        np.testing.assert_allclose(out[key], ref[key], rtol=1e-11, atol=1e-12, err_msg=key)


@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_biased_experts_with_zero_weights(rng, act, layout):
    """With every expert weight zero, FFN_e(x) = b2_e whatever the input (the
    first layer's output is multiplied by W2 = 0), so y_t is the kept gate
    weights times the chosen experts' b2 (Sec. 2.1 with constant experts);
    db2_e = sum of w_tj dy_t over e's kept assignments, dW2_e = a^T dY with
    a = act(b1_e) on every kept row, and dW1 = dW3 = db1 = db3 = 0 (dA = dY
    W2^T = 0). Rows past an expert's count stay zero in the padded layout."""
    T, M, H, E, k = 30, 6, 5, 4, 2
    inp = _small_inputs(rng, T, M, H, E, act, expert_bias=True)
    for w in ("w1", "w3", "w2"):
        if inp[w] is not None:
            inp[w] = np.zeros_like(inp[w])
    out = oracle.layer_fwd_bwd(inp, k=k, f=0.75, act=act, layout=layout)
    c = out["chunks"][0]
    idx, w, slot = c["topk_idx"], c["topk_w"], c["slot"]
    kept = slot >= 0
    assert kept.any() and not kept.all()
    y = np.zeros((T, M))
    db2 = np.zeros((E, M))
    for t in range(T):
        for j in range(k):
            if kept[t, j]:
                y[t] += w[t, j] * inp["b2"][idx[t, j]]
                db2[idx[t, j]] += w[t, j] * inp["dy"][t]
    np.testing.assert_allclose(out["y"], y, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(out["db2"], db2, rtol=1e-13, atol=1e-14)
    a = oracle.gelu(inp["b1"]) if act == "gelu" else oracle.silu(inp["b1"]) * inp["b3"]
    np.testing.assert_allclose(out["dw2"], a[:, :, None] * db2[:, None, :], rtol=1e-12, atol=1e-14)
    for name in ("dw1", "db1") + (("dw3", "db3") if act == "swiglu" else ()):
        assert not out[name].any(), name
    live = np.zeros(c["rows"], bool)
    for e in range(E):
        live[c["offsets"][e]:c["offsets"][e] + c["counts"][e]] = True
    assert not c["y_disp"][~live].any() and not c["h1"][~live].any()


def test_zero_capacity_leaves_only_gate_path(rng):
    T, M, H, E, k = 16, 8, 6, 4, 2
    inp = _small_inputs(rng, T, M, H, E, "gelu")
    out = oracle.layer_fwd_bwd(inp, k=k, f=1.0, act="gelu", C=0)
    assert not out["y"].any()
    assert not out["dw1"].any() and not out["dw2"].any()
    # no kept slot: dw = 0, so dl = 0 and dx = 0
    assert not out["dx"].any() and not out["dw_gate"].any()


@pytest.mark.parametrize("expert_bias", [False, True])
@pytest.mark.parametrize("gate", ["renorm", "full"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_layer_finite_differences(rng, act, gate, expert_bias):
    T, M, H, E, k = 10, 6, 5, 3, 2
    inp = _small_inputs(rng, T, M, H, E, act, expert_bias=expert_bias)
    out = oracle.layer_fwd_bwd(inp, k=k, f=1.0, act=act, gate=gate)
    # routing must be locally constant for the check to hold
    l = out["logits"]
    srt = np.sort(l, axis=1)
    assert np.min(srt[:, -k] - srt[:, -k - 1]) > 1e-3

    def loss(mod):
        o = oracle.layer_fwd_bwd(mod, k=k, f=1.0, act=act, C=out["C"], gate=gate)
        return float((o["y"] * inp["dy"]).sum())

    h = 1e-6
    names = ["x", "w_gate", "bias", "w1", "w2"] + (["w3"] if act == "swiglu" else [])
    if expert_bias:
        names += ["b1", "b2"] + (["b3"] if act == "swiglu" else [])
    gname = {"x": "dx", "w_gate": "dw_gate", "bias": "dbias", "w1": "dw1", "w2": "dw2", "w3": "dw3",
             "b1": "db1", "b2": "db2", "b3": "db3"}
    for name in names:
        a = inp[name]
        for flat in rng.choice(a.size, size=min(6, a.size), replace=False):
            ix = np.unravel_index(flat, a.shape)
            plus, minus = dict(inp), dict(inp)
            plus[name] = a.copy(); plus[name][ix] += h
            minus[name] = a.copy(); minus[name][ix] -= h
            fd = (loss(plus) - loss(minus)) / (2 * h)
            assert abs(fd - out[gname[name]][ix]) <= 1e-6 * max(1.0, abs(fd)), (name, ix)


def test_full_softmax_gate_closed_forms(rng):
    """gate="full": the selected experts' probabilities under the softmax over
    all experts. k = E reduces to the renormalised gate; k = 1 gives the
    largest probability 1 / sum_e exp(l_e - l_max); the weights of k < E
    experts sum to less than one."""
    L_ = rng.standard_normal((40, 6))
    i_full, w_full = oracle.topk_select(L_, 6, "full")
    i_ren, w_ren = oracle.topk_select(L_, 6)
    assert np.array_equal(i_full, i_ren)
    np.testing.assert_allclose(w_full, w_ren, rtol=1e-14)
    np.testing.assert_allclose(w_full, np.take_along_axis(softmax(L_, axis=1), i_full, 1), rtol=1e-14)
    _, w1 = oracle.topk_select(L_, 1, "full")
    np.testing.assert_allclose(w1[:, 0], softmax(L_, axis=1).max(axis=1), rtol=1e-14)
    _, w3 = oracle.topk_select(L_, 3, "full")
    assert np.all(w3.sum(axis=1) < 1.0)
    assert np.all(np.diff(w3, axis=1) <= 0)


@pytest.mark.parametrize("gate", ["renorm", "full"])
def test_gate_jacobian_rows_sum_to_zero(rng, gate):
    """The gate weights are softmax probabilities (of the selection or of all
    experts), so shifting every logit of a token changes nothing: each row of
    d_logits sums to zero."""
    T, M, E, k = 30, 5, 7, 3
    x, wg = rng.standard_normal((T, M)), rng.standard_normal((M, E))
    L_ = x @ wg
    idx, w = oracle.topk_select(L_, k, gate)
    dw = rng.standard_normal((T, k))
    g = oracle.gate_bwd(x, wg, idx, w, dw, L_, gate)
    np.testing.assert_allclose(g["d_logits"].sum(axis=1), 0.0, atol=1e-14)
    if gate == "full":  # every expert of every token has a gradient
        assert np.all(g["d_logits"] != 0.0)


def test_top1_full_softmax_gate_has_gradient(rng):
    """Unlike the renormalised top-1 gate (weight 1, no gradient), the
    Switch-style gate keeps the router trainable: d_logits = p (dw [e = S] - s)."""
    T, M, H, E = 20, 8, 6, 4
    inp = _small_inputs(rng, T, M, H, E, "gelu")
    out = oracle.layer_fwd_bwd(inp, k=1, f=1.0, act="gelu", gate="full")
    assert np.all(out["topk_w"] < 1.0)
    assert out["d_logits"].any() and out["dw_gate"].any()


def test_top1_gate_has_no_gradient(rng):
    T, M, H, E = 20, 8, 6, 4
    inp = _small_inputs(rng, T, M, H, E, "gelu")
    out = oracle.layer_fwd_bwd(inp, k=1, f=1.0, act="gelu")
    assert np.all(out["topk_w"] == 1.0)
    assert not out["d_logits"].any() and not out["dw_gate"].any()


# ---------------------------------------------------------------------------
# chunking (Sec. 3.2 partition; App. H microbatch equivalence)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_chunked_equals_unchunked_without_drops(rng, act):
    T, M, H, E, k, R = 32, 8, 6, 4, 2, 4
    inp = _small_inputs(rng, T, M, H, E, act)
    # capacity large enough that nothing is dropped in either split
    one = oracle.layer_fwd_bwd(inp, k=k, f=float(E), act=act, R=1)
    many = oracle.layer_fwd_bwd(inp, k=k, f=float(E), act=act, R=R)
    for key in ("y", "dx", "dw_gate", "dw1", "dw2", "dbias") + (("dw3",) if act == "swiglu" else ()):
        np.testing.assert_allclose(many[key], one[key], rtol=1e-12, atol=1e-12, err_msg=key)
    # and the chunked result is the concatenation of independent calls
    Tr = T // R
    for r in range(R):
        sub = {kk: (v[r * Tr:(r + 1) * Tr] if kk in ("x", "dy") else v) for kk, v in inp.items()}
        o = oracle.layer_fwd_bwd(sub, k=k, f=float(E), act=act)
        np.testing.assert_array_equal(many["y"][r * Tr:(r + 1) * Tr], o["y"])


def test_chunk_capacity_is_per_chunk(rng):
    T, E, k, R = 64, 4, 2, 4
    inp = _small_inputs(rng, T, 4, 4, E, "gelu")
    out = oracle.layer_fwd_bwd(inp, k=k, f=1.0, act="gelu", R=R)
    assert out["C"] == math.ceil(Fraction(1) * k * (T // R) / E)
    for c in out["chunks"]:
        assert c["counts"].max() <= out["C"]
