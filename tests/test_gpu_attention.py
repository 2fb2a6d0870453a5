"""Parity of the attention part of AT_r (flowmoe_attention_fwd/_bwd,
flowmoe_mha_fwd/_bwd) against the fp64 oracle, on seeded inputs: several
query/key tiles with ragged tails (sequence lengths that are not multiples
of the 128-query block, the 64-key tile or the 32-query step), one-token
sequences, both head widths, causal and bidirectional; and the full-size
large-layer attention (4 sequences of 4096 tokens, 32 heads of 128, causal)
on sampled (sequence, head) pairs. bf16 results within 2e-2 max relative
error, the float log-sum-exp within 1e-4."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_close, dev, host, need_gpu
from moe_inputs import as_f64, get_config, make_attention_inputs, make_inputs, to_torch

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2510_00207_amd import _lib as L
    return L


def run_core(T, M, seq_len, heads, causal, seed):
    L = _lib()
    d = dev()
    a = make_attention_inputs(seed, T, M)
    qkv = to_torch(a["qkv"], d)
    d_attn = to_torch(a["d_attn"], d)
    attn = torch.zeros(T, M, dtype=torch.bfloat16, device=d)
    lse = torch.zeros(heads, T, dtype=torch.float32, device=d)
    d_qkv = torch.zeros(T, 3 * M, dtype=torch.bfloat16, device=d)
    delta = torch.zeros(heads, T, dtype=torch.float32, device=d)
    s = L.make_shape(T, M, 64, 1, 1, 0, L.BF16)
    m = L.make_mha_shape(seq_len, heads, M // heads, causal)
    L.flowmoe_attention_fwd(s, m, qkv, attn, lse)
    L.flowmoe_attention_bwd(s, m, qkv, attn, lse, d_attn, d_qkv, delta)
    torch.cuda.synchronize()
    return a, dict(attn=host(attn), lse=host(lse), d_qkv=host(d_qkv), delta=host(delta))


CORE_CASES = [
    # (sequences, seq_len, heads, head_dim, causal)
    (2, 128, 2, 64, False),
    (2, 200, 2, 64, True),     # ragged: 200 = 128 + 72 queries, 3 key tiles + 8
    (1, 256, 2, 128, True),
    (2, 333, 1, 128, False),   # ragged in every tile size
    (3, 1, 2, 64, True),       # one-token sequences
    (3, 1, 1, 128, False),
    (1, 64, 4, 64, True),
    (1, 1000, 1, 128, True),   # 8 query blocks, 16 key tiles, the last ragged
    (2, 97, 3, 64, False),
    # grids of at least 512 blocks of 256 queries: the 8-wave forward blocks,
    # with ragged tails
    (4, 700, 48, 64, True),
    (2, 520, 96, 128, False),
]


@pytest.mark.parametrize("nseq,seq_len,heads,hd,causal", CORE_CASES)
def test_attention_core(nseq, seq_len, heads, hd, causal):
    need_gpu()
    T, M = nseq * seq_len, heads * hd
    print(f"[attn] core T={T} N={seq_len} heads={heads} d={hd} causal={causal}", flush=True)
    a, g = run_core(T, M, seq_len, heads, causal, seed=T + M + int(causal))
    qkv = as_f64(a["qkv"])
    d_attn = as_f64(a["d_attn"])
    attn, lse = oracle.attention(qkv, seq_len, heads, causal)
    assert_close(g["attn"], attn, "bf16", "attn")
    assert_close(g["lse"], lse, "f32", "lse")
    # delta = rowsum(d_attn * attn) per head (the GPU's from its own bf16 attn)
    d = hd
    ref_delta = np.stack([(d_attn[:, h * d:(h + 1) * d] * attn[:, h * d:(h + 1) * d]).sum(axis=1)
                          for h in range(heads)])
    assert_close(g["delta"], ref_delta, "bf16", "delta")
    d_qkv = oracle.attention_bwd(qkv, d_attn, seq_len, heads, causal)
    for name, sl in (("dQ", slice(0, M)), ("dK", slice(M, 2 * M)), ("dV", slice(2 * M, 3 * M))):
        assert_close(g["d_qkv"][:, sl], d_qkv[:, sl], "bf16", name)


def test_attention_causal_rows_ignore_later_tokens():
    """A change to the last token of a sequence leaves every causal output
    row before it bit-identical (the masked keys contribute exact zeros)."""
    need_gpu()
    L = _lib()
    d = dev()
    T, M, heads = 300, 128, 1
    a = make_attention_inputs(7, T, M)
    q0 = to_torch(a["qkv"], d)
    q1 = q0.clone()
    q1[T - 1, M:] = 0.5  # the last token's key and value
    s = L.make_shape(T, M, 64, 1, 1, 0, L.BF16)
    m = L.make_mha_shape(T, heads, M // heads, True)
    outs = []
    for q in (q0, q1):
        o = torch.zeros(T, M, dtype=torch.bfloat16, device=d)
        lse = torch.zeros(heads, T, device=d)
        L.flowmoe_attention_fwd(s, m, q, o, lse)
        outs.append((o, lse))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0][:T - 1], outs[1][0][:T - 1])
    assert torch.equal(outs[0][1][:, :T - 1], outs[1][1][:, :T - 1])
    assert not torch.equal(outs[0][0][T - 1], outs[1][0][T - 1])


def test_attention_is_deterministic():
    need_gpu()
    r1 = run_core(512, 256, 256, 2, True, 11)[1]
    r2 = run_core(512, 256, 256, 2, True, 11)[1]
    for k in r1:
        assert np.array_equal(r1[k], r2[k]), k


# ---------------------------------------------------------------------------
# the block's MHA: projections + core
# ---------------------------------------------------------------------------
MHA_CASES = {
    # reduced workloads: the balanced layer's bidirectional d = 64 heads and
    # the large layer's causal d = 128 heads, several tiles with ragged tails
    "balanced_s": get_config("balanced", T=640, M=256, mha=True, seq_len=320),
    "large_s": get_config("large", T=768, M=512, mha=True, seq_len=384),
    # 2048 rows of width 256: the weight gradients split their rows 4 ways
    "split_s": get_config("skewed", T=2048, M=256, mha=True, seq_len=256),
}


def _mha_bufs(T, M, heads, d):
    bf = dict(dtype=torch.bfloat16, device=d)
    return dict(qkv=torch.zeros(T, 3 * M, **bf), attn=torch.zeros(T, M, **bf),
                lse=torch.zeros(heads, T, device=d), out=torch.zeros(T, M, **bf),
                d_attn=torch.zeros(T, M, **bf), d_qkv=torch.zeros(T, 3 * M, **bf),
                delta=torch.zeros(heads, T, device=d), d_in=torch.zeros(T, M, **bf),
                dw_qkv=torch.zeros(M, 3 * M, device=d), dw_o=torch.zeros(M, M, device=d))


@pytest.mark.parametrize("name", list(MHA_CASES))
def test_mha_fwd_bwd(name):
    need_gpu()
    L = _lib()
    d = dev()
    cfg = MHA_CASES[name]
    print(f"[attn] mha {name}", flush=True)
    inp = make_inputs(cfg)
    T, M, heads = cfg.T, cfg.M, cfg.heads
    b = _mha_bufs(T, M, heads, d)
    t = {k: to_torch(inp[k], d) for k in ("mha_in", "w_qkv", "w_o", "dy")}
    s = L.make_shape(T, M, 64, 1, 1, 0, L.BF16)
    m = L.make_mha_shape(cfg.seq_len, heads, cfg.head_dim, cfg.causal)
    wsb = L.flowmoe_workspace_bytes(s, L.WS_MHA_BWD)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=d)
    L.flowmoe_mha_fwd(s, m, t["mha_in"], t["w_qkv"], t["w_o"], b["qkv"], b["attn"], b["lse"],
                      b["out"])
    # d_out: the generator's dy stands in for the gradient of I'
    L.flowmoe_mha_bwd(s, m, t["mha_in"], t["w_qkv"], t["w_o"], b["qkv"], b["attn"], b["lse"],
                      t["dy"], b["d_attn"], b["d_qkv"], b["delta"], b["d_in"], b["dw_qkv"],
                      b["dw_o"], 0, ws, wsb)
    torch.cuda.synchronize()
    i64 = {k: as_f64(inp[k]) for k in ("mha_in", "w_qkv", "w_o", "dy")}
    f = oracle.mha_fwd(i64["mha_in"], i64["w_qkv"], i64["w_o"], cfg.seq_len, heads, cfg.causal)
    r = oracle.mha_bwd(i64["mha_in"], i64["w_qkv"], i64["w_o"], f, i64["dy"], cfg.seq_len, heads,
                       cfg.causal)
    for key in ("qkv", "attn", "out"):
        assert_close(host(b[key]), f[key], "bf16", key)
    assert_close(host(b["lse"]), f["lse"], "bf16", "lse")  # (from the bf16-rounded Q, K)
    for key in ("d_attn", "d_qkv", "d_in", "dw_qkv", "dw_o"):
        assert_close(host(b[key]), r[key], "bf16", key)
    # accumulate adds the same weight gradients again
    dwq, dwo = b["dw_qkv"].clone(), b["dw_o"].clone()
    L.flowmoe_mha_bwd(s, m, t["mha_in"], t["w_qkv"], t["w_o"], b["qkv"], b["attn"], b["lse"],
                      t["dy"], b["d_attn"], b["d_qkv"], b["delta"], b["d_in"], b["dw_qkv"],
                      b["dw_o"], 1, ws, wsb)
    torch.cuda.synchronize()
    assert torch.allclose(b["dw_qkv"], 2 * dwq, rtol=1e-6, atol=1e-6)
    assert torch.allclose(b["dw_o"], 2 * dwo, rtol=1e-6, atol=1e-6)


# ---------------------------------------------------------------------------
# full size: the large layer's attention, sampled (sequence, head) pairs
# ---------------------------------------------------------------------------
def test_attention_full_size_large_sampled():
    """The large workload's attention at its real shape (T = 16384 = 4 x 4096,
    M = 4096: 32 heads of 128, causal) in the launch configuration the
    benchmark times; the oracle checks 3 whole (sequence, head) pairs."""
    need_gpu()
    cfg = get_config("large")
    T, M, N, heads = cfg.T, cfg.M, cfg.seq_len, cfg.heads
    print(f"[attn] full size T={T} M={M} N={N} heads={heads}", flush=True)
    a, g = run_core(T, M, N, heads, True, seed=cfg.seed)
    rng = np.random.default_rng(5)
    pairs = [(0, 0), (3, heads - 1), (int(rng.integers(4)), int(rng.integers(heads)))]
    D = cfg.head_dim
    for sq, h in pairs:
        rows = slice(sq * N, (sq + 1) * N)
        cols = [slice(i * M + h * D, i * M + (h + 1) * D) for i in range(3)]
        qkv_h = np.concatenate([as_f64(a["qkv"][rows, c]) for c in cols], axis=1)
        da_h = as_f64(a["d_attn"][rows, h * D:(h + 1) * D])
        attn, lse = oracle.attention(qkv_h, N, 1, True)
        assert_close(g["attn"][rows, h * D:(h + 1) * D], attn, "bf16", f"attn s{sq} h{h}")
        assert_close(g["lse"][h, rows], lse[0], "f32", f"lse s{sq} h{h}")
        d_qkv = oracle.attention_bwd(qkv_h, da_h, N, 1, True)
        for i, name in enumerate(("dQ", "dK", "dV")):
            assert_close(g["d_qkv"][rows, cols[i]], d_qkv[:, i * D:(i + 1) * D], "bf16",
                         f"{name} s{sq} h{h}")


# ---------------------------------------------------------------------------
# the layer with AT_r = attention + gate (Sec. 3.2)
# ---------------------------------------------------------------------------
LAYER_CASES = {
    "balanced_s": get_config("balanced", T=1024, M=256, H=416, mha=True, seq_len=256),
    "large_s": get_config("large", T=768, M=512, H=456, mha=True, seq_len=192),
    "fine_s": get_config("fine", T=1024, M=256, H=160, mha=True, seq_len=256),
}


def _mha_layer(cfg, R, inp):
    from paper_2510_00207_amd.layer import MoELayer
    from gpu_helpers import load_layer
    layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=R, f=cfg.f,
                     act=cfg.act, dtype=cfg.dtype, bias=cfg.zipf_bias, gate=cfg.gate,
                     mha=dict(seq_len=cfg.seq_len, head_dim=cfg.head_dim, causal=cfg.causal),
                     device=dev())
    load_layer(layer, inp)
    for k in ("mha_in", "w_qkv", "w_o"):
        getattr(layer, k).copy_(to_torch(inp[k], layer.x.device))
    return layer


@pytest.mark.parametrize("R", [1, 2])
@pytest.mark.parametrize("name", list(LAYER_CASES))
def test_layer_with_attention(name, R):
    need_gpu()
    from gpu_helpers import f64_inputs, near_tie_check
    cfg = LAYER_CASES[name]
    print(f"[attn] layer {name} R={R}", flush=True)
    inp = make_inputs(cfg)
    layer = _mha_layer(cfg, R, inp)
    sc = torch.cuda.current_stream()
    sm = torch.cuda.Stream()
    layer.forward(sc, sm)
    layer.backward(sc, sm)
    torch.cuda.synchronize()
    i64 = f64_inputs(inp)
    gl = host(layer.logits)
    mha = dict(seq_len=cfg.seq_len, heads=cfg.heads, causal=cfg.causal)
    ref = oracle.layer_fwd_bwd(i64, k=cfg.k, f=cfg.f, act=cfg.act, R=R, logits_for_routing=gl,
                               gate=cfg.gate, mha=mha)
    # AT_r's attention output is the MoE part's input
    assert_close(host(layer.x), ref["x"], "bf16", "x = I'")
    assert_close(host(layer.attn), ref["attn"], "bf16", "attn")
    assert_close(host(layer.lse), ref["lse"], "bf16", "lse")
    # routing on the GPU's logits is bit-exact; the oracle's own differs only on near-ties
    assert np.array_equal(host(layer.topk_idx), ref["topk_idx"])
    own = oracle.gate_logits(ref["x"], i64["w_gate"], i64["bias"])
    assert_close(gl, own, "bf16", "logits")
    ndiff, nnear, bound = near_tie_check(own, gl, host(layer.topk_idx), cfg.k)
    print(f"[attn] own-logit routing: {ndiff} differ, {nnear} near-ties below {bound:.2e}",
          flush=True)
    Tr = cfg.T // R
    for r, c in enumerate(ref["chunks"]):
        assert np.array_equal(host(layer.counts[r]), c["counts"]), f"counts chunk {r}"
        assert np.array_equal(host(layer.slot[r * Tr:(r + 1) * Tr]), c["slot"]), f"slot {r}"
    for key in ("y", "dx", "d_logits", "dw_gate", "dw1", "dw2", "d_in", "dw_qkv", "dw_o"):
        assert_close(host(getattr(layer, key)), ref[key], "bf16", key)
    if cfg.act == "swiglu":
        assert_close(host(layer.dw3), ref["dw3"], "bf16", "dw3")


def test_layer_with_attention_schedule():
    """Backward with the attention (R = 3 on two streams): the compute stream
    runs E_R..E_1, the expert weight gradients, the attention backward of
    chunks R..1 (each after its D_r: constraint 6d) and then the attention's
    weight gradients; tracing changes no result."""
    need_gpu()
    R = 3
    cfg = get_config("fine", T=256 * R, M=256, H=160, mha=True, seq_len=256)
    inp = make_inputs(cfg)
    sc, sm = torch.cuda.Stream(), torch.cuda.Stream()
    from paper_2510_00207_amd import _lib as L

    def ev(n):
        out = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in out:
            e.record(sc)
        return out

    fwd_ev, bwd_ev, (t0,) = ev(8 * R), ev(L.bwd_trace_len(R, True)), ev(1)
    torch.cuda.synchronize()
    traced, plain = _mha_layer(cfg, R, inp), _mha_layer(cfg, R, inp)
    plain.forward(sc, sm)
    plain.backward(sc, sm)
    torch.cuda.synchronize()
    t0.record(sc)
    traced.forward(sc, sm, trace=fwd_ev)
    traced.backward(sc, sm, trace=bwd_ev)
    plain.forward(sc, sm)
    plain.backward(sc, sm)
    torch.cuda.synchronize()
    t = lambda e: t0.elapsed_time(e)
    span = lambda i: (t(bwd_ev[i]), t(bwd_ev[i + 1]))
    D = {r: span(2 * (2 * R + r)) for r in range(R)}          # dispatch backward (task 2)
    E = {r: span(2 * (1 * R + r)) for r in range(R)}          # experts backward (task 1)
    W = span(8 * R)                                           # expert weight gradients
    A = {r: span(8 * R + 2 + 2 * r) for r in range(R)}        # attention backward of chunk r
    AW = span(10 * R + 2)                                     # attention weight gradients
    slack = 1e-3
    order = [E[r] for r in range(R - 1, -1, -1)] + [W] + [A[r] for r in range(R - 1, -1, -1)] + [AW]
    for a, b in zip(order, order[1:]):
        assert a[1] <= b[0] + slack
    for r in range(R):
        assert D[r][1] <= A[r][0] + slack, f"attention backward of chunk {r} before D_{r} ended"
    # the forward's AT_r spans include the attention: AT_r ends before D_r begins
    for r in range(R):
        assert t(fwd_ev[2 * r + 1]) <= t(fwd_ev[2 * (R + r)]) + slack
    for nm in ("y", "x", "d_in", "dw_qkv", "dw_o", "dw1", "dw_gate"):
        assert torch.equal(getattr(traced, nm), getattr(plain, nm)), nm


def test_layer_with_attention_deterministic_and_graph_replays():
    """The layer with the attention in AT_r (R = 2): two streams equal one
    stream bit for bit, two runs are bit-identical, and a fwd+bwd step
    captured in a HIP graph replays bit-identical to the eager step, replay
    after replay, with the outputs clobbered eagerly in between."""
    need_gpu()
    cfg = LAYER_CASES["fine_s"]
    R = 2
    inp = make_inputs(cfg)
    names = ("x", "qkv", "attn", "lse", "logits", "topk_idx", "y", "dx", "d_attn", "d_qkv",
             "delta", "d_in", "dw_qkv", "dw_o", "dw_gate", "dw1", "dw3", "dw2")

    def run(two):
        lay = _mha_layer(cfg, R, inp)
        sc = torch.cuda.current_stream()
        sm = torch.cuda.Stream() if two else sc
        lay.forward(sc, sm)
        lay.backward(sc, sm)
        torch.cuda.synchronize()
        return lay

    a, b, c = run(True), run(False), run(True)
    for nm in names:
        assert torch.equal(getattr(a, nm), getattr(b, nm)), f"{nm}: two streams differ from one"
        assert torch.equal(getattr(a, nm), getattr(c, nm)), f"{nm}: not deterministic"
    layer = _mha_layer(cfg, R, inp)
    bufs = layer.bufs()
    gs, sm = torch.cuda.Stream(), torch.cuda.Stream()
    layer.forward(gs, sm, bufs=bufs)  # (one-time set-up outside the capture)
    layer.backward(gs, sm, bufs=bufs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=gs):
        layer.forward(gs, sm, bufs=bufs)
        layer.backward(gs, sm, bufs=bufs)
    for rep in range(3):
        for nm in names:
            getattr(layer, nm).fill_(7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for nm in names:
            assert torch.equal(getattr(layer, nm), getattr(a, nm)), f"replay {rep}: {nm}"
