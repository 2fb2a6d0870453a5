"""Full-size parity: the four bf16 workloads at their real sizes, run exactly
as bench.py runs them (flowmoe_layer_fwd + flowmoe_layer_bwd, R chunks, two
streams, packed layout).

Checked against the fp64 oracle:
  * every gate logit (x W_g in fp64) within 1e-4 of max |logit|;
  * routing for every token and chunk, bit-exact: top-k indices from the
    GPU's fp32 logits, counts, offsets, slots, row sources, and the
    dispatched rows (bitwise copies of x);
  * the oracle's own fp64 routing differs from the GPU's only on tokens with
    a near-tie among their top k + 1 fp64 logits (a gap below 4 max|dl|);
    the count is printed;
  * sampled tokens: y, dx, d_topk_w, d_logits, and the rows of their kept
    assignments in y_disp, dy_disp and dx_disp, recomputed one token at a
    time through oracle.expert_ffn / combine_bwd / expert_ffn_bwd / gate_bwd
    on that token's kept assignments;
  * a sampled 32 x 32 block of dW1, dW2 (and dW3) of two experts: sums over
    the expert's rows of the oracle's per-row gradients, the tolerance
    scaled by the oracle block's largest entry;
  * dW_g and db: x^T d_logits and column sums of the GPU's own d_logits in
    fp64 (the reduction at full size; d_logits itself is sampled above).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_close, dev, host, load_layer, near_tie_check, need_gpu
from moe_inputs import as_f64, get_config, make_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

N_TOK = 24      # sampled tokens per workload
N_W = 32        # sampled rows and columns of the weight-gradient blocks


def _w64(a, e):
    """One expert's weight slice widened to fp64."""
    return as_f64(a[e])


def _run(cfg):
    from paper_2510_00207_amd.layer import MoELayer
    print(f"[fullsize] {cfg.name}: generating inputs", flush=True)
    inp = make_inputs(cfg)
    layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=cfg.R, f=cfg.f,
                     act=cfg.act, dtype=cfg.dtype, layout="packed", bias=cfg.zipf_bias,
                     device=dev())
    load_layer(layer, inp)
    sc = torch.cuda.current_stream()
    sm = torch.cuda.Stream()
    print(f"[fullsize] {cfg.name}: running layer (R={cfg.R})", flush=True)
    layer.forward(sc, sm)
    layer.backward(sc, sm)
    torch.cuda.synchronize()
    return layer, inp


@pytest.mark.parametrize("name", ["balanced", "skewed", "large", "fine"])
def test_fullsize_parity(name):
    need_gpu()
    cfg = get_config(name)
    layer, inp = _run(cfg)
    R, T, E, k, M = cfg.R, cfg.T, cfg.E, cfg.k, cfg.M
    Tr = T // R
    rng = np.random.default_rng(1000 + cfg.seed)
    x = inp["x"]
    bias = None if inp["bias"] is None else inp["bias"].astype(np.float64)
    wg = as_f64(inp["w_gate"])

    # ---- logits: all tokens ----
    print(f"[fullsize] {name}: logits", flush=True)
    x64 = as_f64(x)
    gl = host(layer.logits)
    own = oracle.gate_logits(x64, wg, bias)
    assert np.max(np.abs(gl - own)) <= 1e-4 * np.max(np.abs(own))

    # ---- routing and dispatch: all tokens, bit-exact ----
    print(f"[fullsize] {name}: routing", flush=True)
    idx_ref, w_ref = oracle.topk_select(gl, k)
    assert np.array_equal(host(layer.topk_idx), idx_ref)
    ndiff, nnear, bound = near_tie_check(own, gl, idx_ref, k)
    print(f"[fullsize] {name}: own fp64 routing differs on {ndiff} token(s); {nnear} token(s) "
          f"with a top-{k + 1} gap below {bound:.2e}", flush=True)
    np.testing.assert_allclose(host(layer.topk_w), w_ref, rtol=2e-6, atol=2e-7)
    C = oracle.capacity(Tr, E, k, cfg.f)
    assert layer.C == C
    slot_all = host(layer.slot)
    routes = []
    for r in range(R):
        rt = oracle.route(idx_ref[r * Tr:(r + 1) * Tr], E, C, "packed")
        routes.append(rt)
        assert np.array_equal(host(layer.counts[r]), rt["counts"])
        assert np.array_equal(host(layer.offsets[r]), rt["offsets"])
        assert np.array_equal(host(layer.load[r]), rt["demand"])
        assert np.array_equal(slot_all[r * Tr:(r + 1) * Tr], rt["slot"])
        live = int(rt["offsets"][-1])
        assert np.array_equal(host(layer.row_src[r][:live]), rt["row_src"][:live])
        xd = layer.x_disp[r][:live].view(torch.int16).cpu().numpy().view(np.uint16)
        src_tok = r * Tr + rt["row_src"][:live] // k
        assert np.array_equal(xd, x[src_tok]), f"x_disp chunk {r} is not a copy of x"
    kept_frac = sum(int(rt["offsets"][-1]) for rt in routes) / (T * k)
    print(f"[fullsize] {name}: C={C}, kept {kept_frac:.3f} of assignments", flush=True)

    # ---- sampled tokens: forward and backward through the oracle ----
    print(f"[fullsize] {name}: sampled tokens", flush=True)
    toks = np.sort(rng.choice(T, size=N_TOK, replace=False))
    dy64 = as_f64(inp["dy"][toks])
    y_gpu = host(layer.y[torch.from_numpy(toks).to(dev())])
    dx_gpu = host(layer.dx[torch.from_numpy(toks).to(dev())])
    dtw_gpu = host(layer.d_topk_w[torch.from_numpy(toks).to(dev())])
    dl_gpu = host(layer.d_logits[torch.from_numpy(toks).to(dev())])
    # per (token, j) kept assignment: expert, weight
    y_ref = np.zeros((N_TOK, M))
    dxd_ref = np.zeros((N_TOK, M))
    dw_ref = np.zeros((N_TOK, k))
    by_expert = {}
    for i, t in enumerate(toks):
        for j in range(k):
            if slot_all[t, j] >= 0:
                by_expert.setdefault(int(idx_ref[t, j]), []).append((i, j))
    # the GPU's rows of every sampled kept assignment, in by_expert order
    def rows_of(buf, items):
        out = []
        for i, j in items:
            t = int(toks[i])
            out.append(host(buf[t // Tr][int(slot_all[t, j])]))
        return np.stack(out)
    for e, items in by_expert.items():
        W1, W2 = _w64(inp["w1"], e)[None], _w64(inp["w2"], e)[None]
        W3 = _w64(inp["w3"], e)[None] if cfg.act == "swiglu" else None
        Xs = x64[[toks[i] for i, _ in items]]
        n = len(items)
        cnt, off = np.array([n]), np.array([0, n])
        sv = oracle.expert_ffn(Xs, cnt, off, W1, W3, W2, cfg.act)
        wt = np.array([w_ref[toks[i], j] for i, j in items])
        dys = np.stack([dy64[i] for i, _ in items])
        for q, (i, j) in enumerate(items):
            y_ref[i] += wt[q] * sv["y_disp"][q]
            dw_ref[i, j] = float(dys[q] @ sv["y_disp"][q])
        dyd, _ = oracle.combine_bwd(dys, sv["y_disp"], np.arange(n)[:, None], wt[:, None])
        dxd, _, _, _ = oracle.expert_ffn_bwd(dyd, Xs, sv, cnt, off, W1, W3, W2, cfg.act)
        for q, (i, _) in enumerate(items):
            dxd_ref[i] += dxd[q]
        assert_close(rows_of(layer.y_disp, items), sv["y_disp"], "bf16", f"{name} y_disp rows e={e}")
        assert_close(rows_of(layer.dy_disp, items), dyd, "bf16", f"{name} dy_disp rows e={e}")
        assert_close(rows_of(layer.dx_disp, items), dxd, "bf16", f"{name} dx_disp rows e={e}")
    g = oracle.gate_bwd(x64[toks], wg, idx_ref[toks], w_ref[toks], dw_ref)
    assert_close(y_gpu, y_ref, "bf16", f"{name} y (sampled)")
    assert_close(dtw_gpu, dw_ref, "bf16", f"{name} d_topk_w (sampled)")
    assert_close(dl_gpu, g["d_logits"], "bf16", f"{name} d_logits (sampled)")
    assert_close(dx_gpu, dxd_ref + g["dx_gate"], "bf16", f"{name} dx (sampled)")

    # ---- dW_g and db at full size from the GPU's d_logits ----
    dl_all = host(layer.d_logits)
    assert_close(host(layer.dw_gate), x64.T @ dl_all, "bf16", f"{name} dw_gate")
    if cfg.zipf_bias:
        assert_close(host(layer.dbias), dl_all.sum(axis=0), "bf16", f"{name} dbias")
    del x64, own, dl_all

    # ---- sampled expert weight-gradient entries ----
    print(f"[fullsize] {name}: sampled weight gradients", flush=True)
    dy_all = inp["dy"]
    for e in sorted(rng.choice(E, size=min(2, E), replace=False)):
        W1e, W2e = _w64(inp["w1"], e), _w64(inp["w2"], e)
        W3e = _w64(inp["w3"], e) if cfg.act == "swiglu" else None
        # all kept rows of expert e over the chunks: token, gate weight
        rows_t, rows_w = [], []
        for r, rt in enumerate(routes):
            lo, hi = rt["offsets"][e], rt["offsets"][e] + rt["counts"][e]
            for a in rt["row_src"][lo:hi]:
                t, j = r * Tr + a // k, a % k
                rows_t.append(t)
                rows_w.append(w_ref[t, j])
        if not rows_t:
            continue
        rows_t = np.array(rows_t)
        X = as_f64(x[rows_t])                                   # rows x M
        dY = np.array(rows_w)[:, None] * as_f64(dy_all[rows_t])  # rows x M (dy_disp)
        hs = np.sort(rng.choice(cfg.H, size=N_W, replace=False))
        ms = np.sort(rng.choice(M, size=N_W, replace=False))
        h1 = X @ W1e[:, hs]                                     # rows x N_W
        dA = dY @ W2e[hs, :].T                                  # rows x N_W
        if cfg.act == "gelu":
            a = oracle.gelu(h1)
            dH1 = dA * oracle.gelu_grad(h1)
        else:
            h3 = X @ W3e[:, hs]
            a = oracle.silu(h1) * h3
            dH1 = dA * h3 * oracle.silu_grad(h1)
            dH3 = dA * oracle.silu(h1)
        # blocks dW1[ms][:, hs] = X[:, ms]^T dH1 and dW2[hs][:, ms] = A^T dY[:, ms];
        # the tolerance is relative to the oracle block's largest entry
        hs_t, ms_t = torch.from_numpy(hs).to(dev()), torch.from_numpy(ms).to(dev())
        blk = lambda w, r, c: host(w[e].index_select(0, r).index_select(1, c))
        assert_close(blk(layer.dw1, ms_t, hs_t), X[:, ms].T @ dH1, "bf16", f"{name} dw1 block e={e}")
        assert_close(blk(layer.dw2, hs_t, ms_t), a.T @ dY[:, ms], "bf16", f"{name} dw2 block e={e}")
        if cfg.act == "swiglu":
            assert_close(blk(layer.dw3, ms_t, hs_t), X[:, ms].T @ dH3, "bf16",
                         f"{name} dw3 block e={e}")
    print(f"[fullsize] {name}: ok", flush=True)
