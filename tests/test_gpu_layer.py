"""Whole-layer parity: flowmoe_layer_fwd / flowmoe_layer_bwd (R chunks, two
streams) against the fp64 oracle, on seeded inputs spanning several tiles with
ragged tails. Routing (indices, counts, offsets, slots, permutation) must be
bit-exact against the oracle run on the GPU's fp32 logits; floating-point
outputs within 1e-4 (fp32) / 2e-2 (bf16) max relative error."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import (assert_close, dev, f64_inputs, host, load_layer, near_tie_check,
                         need_gpu, oracle_for_layer)
from moe_inputs import get_config, make_inputs
from paper_2510_00207_amd import _lib as L

pytestmark = pytest.mark.gpu

# reduced versions of the five workloads (same E, k, f, act, dtype, R), sized
# for the oracle; H and M leave ragged GEMM tiles. Widths that are multiples
# of 32 run the LDS-streaming GEMM everywhere; H = 456 (large_s) sends the
# row-mode GEMMs with K = H to the register-staged kernel.
CASES = {
    "tiny": get_config("tiny"),
    "balanced_s": get_config("balanced", T=512, M=256, H=416),
    "skewed_s": get_config("skewed", T=1024, M=256, H=256),
    "large_s": get_config("large", T=512, M=512, H=456),
    "fine_s": get_config("fine", T=1024, M=256, H=160),
}


def run_layer(cfg, layout, R=None, two_streams=True, inp=None):
    from paper_2510_00207_amd.layer import MoELayer
    R = cfg.R if R is None else R
    inp = make_inputs(cfg) if inp is None else inp
    layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=R, f=cfg.f, act=cfg.act,
                     dtype=cfg.dtype, layout=layout, bias=cfg.zipf_bias, gate=cfg.gate,
                     expert_bias=cfg.expert_bias, device=dev())
    load_layer(layer, inp)
    sc = torch.cuda.current_stream()
    sm = torch.cuda.Stream() if two_streams else sc
    layer.forward(sc, sm)
    layer.backward(sc, sm)
    torch.cuda.synchronize()
    return layer, inp


def check_against_oracle(cfg, layout, layer, inp, R):
    i64 = f64_inputs(inp)
    gl = host(layer.logits)
    ref = oracle_for_layer(i64, cfg, R, layout, gl)
    dt = cfg.dtype
    # gate logits vs the oracle's own fp64 logits
    own = oracle.gate_logits(i64["x"], i64["w_gate"], i64["bias"])
    dl = np.max(np.abs(gl - own))
    assert dl <= 1e-4 * np.max(np.abs(own)), f"logits off by {dl}"
    # routing is a function of the fp32 logits: bit-exact
    assert np.array_equal(host(layer.topk_idx), ref["topk_idx"])
    # the oracle's own fp64 routing differs only on near-ties
    ndiff, nnear, bound = near_tie_check(own, gl, host(layer.topk_idx), cfg.k)
    print(f"[layer] own-logit routing: {ndiff} token(s) differ, {nnear} near-tie(s) "
          f"below {bound:.2e}", flush=True)
    # (the full softmax gate divides by a sum over all E experts in fp32)
    wtol = dict(rtol=1e-5, atol=1e-7) if cfg.gate == "full" else dict(rtol=2e-6, atol=2e-7)
    np.testing.assert_allclose(host(layer.topk_w), ref["topk_w"], **wtol)
    Tr = cfg.T // R
    for r, c in enumerate(ref["chunks"]):
        assert np.array_equal(host(layer.counts[r]), c["counts"]), f"counts chunk {r}"
        assert np.array_equal(host(layer.offsets[r]), c["offsets"]), f"offsets chunk {r}"
        assert np.array_equal(host(layer.load[r]), c["demand"]), f"load chunk {r}"
        assert np.array_equal(host(layer.slot[r * Tr:(r + 1) * Tr]), c["slot"]), f"slot chunk {r}"
        live = c["rows"] if layout == "padded" else int(c["offsets"][-1])
        assert np.array_equal(host(layer.row_src[r][:c["rows"]])[:live], c["row_src"][:live])
        # dispatch is an exact copy
        assert np.array_equal(host(layer.x_disp[r][:live]), c["x_disp"][:live]), f"x_disp chunk {r}"
        # the backward has overwritten h_save with the hidden-layer gradient
        assert_close(host(layer.h_save[r][:live]), c["dh"][:live], dt, f"dH in h_save[{r}]")
        assert_close(host(layer.a_save[r][:live]), c["a"][:live], dt, f"a_save[{r}]")
        assert_close(host(layer.y_disp[r][:live]), c["y_disp"][:live], dt, f"y_disp[{r}]")
        assert_close(host(layer.dy_disp[r][:live]), c["dy_disp"][:live], dt, f"dy_disp[{r}]")
        assert_close(host(layer.dx_disp[r][:live]), c["dx_disp"][:live], dt, f"dx_disp[{r}]")
    assert_close(host(layer.y), ref["y"], dt, "y")
    assert_close(host(layer.d_topk_w), ref["d_topk_w"], dt, "d_topk_w")
    assert_close(host(layer.d_logits), ref["d_logits"], dt, "d_logits")
    assert_close(host(layer.dx), ref["dx"], dt, "dx")
    assert_close(host(layer.dw_gate), ref["dw_gate"], dt, "dw_gate")
    if cfg.zipf_bias:
        assert_close(host(layer.dbias), ref["dbias"], dt, "dbias")
    assert_close(host(layer.dw1), ref["dw1"], dt, "dw1")
    assert_close(host(layer.dw2), ref["dw2"], dt, "dw2")
    if cfg.act == "swiglu":
        assert_close(host(layer.dw3), ref["dw3"], dt, "dw3")
    if cfg.expert_bias:
        assert_close(host(layer.db1), ref["db1"], dt, "db1")
        assert_close(host(layer.db2), ref["db2"], dt, "db2")
        if cfg.act == "swiglu":
            assert_close(host(layer.db3), ref["db3"], dt, "db3")
    return ref


@pytest.mark.parametrize("layout", ["packed", "padded"])
@pytest.mark.parametrize("name", list(CASES))
def test_layer_parity(name, layout):
    need_gpu()
    cfg = CASES[name]
    print(f"[layer] {name} {layout} R={cfg.R}", flush=True)
    layer, inp = run_layer(cfg, layout)
    check_against_oracle(cfg, layout, layer, inp, cfg.R)


@pytest.mark.parametrize("R", [1, 2, 4])
def test_layer_chunks(R):
    need_gpu()
    cfg = CASES["balanced_s"]
    print(f"[layer] chunks R={R}", flush=True)
    layer, inp = run_layer(cfg, "packed", R=R)
    check_against_oracle(cfg, "packed", layer, inp, R)


def test_layer_many_chunks():
    """R = 70 chunks of 16 tokens: the weight-gradient GEMMs reduce over 70
    row segments per expert (the first 64 segments' ranges are loaded up
    front, one lane each, the later ones one by one), every step against
    the oracle."""
    need_gpu()
    cfg = get_config("balanced", T=70 * 16, M=128, H=96)
    print("[layer] many chunks R=70", flush=True)
    layer, inp = run_layer(cfg, "packed", R=70)
    check_against_oracle(cfg, "packed", layer, inp, 70)


@pytest.mark.parametrize("order", ["split", "joined"])
@pytest.mark.parametrize("name,R", [("fine_s", 4), ("balanced_m", 1)])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_layer_tile_orders(name, R, layout, order):
    """The layer with the grouped GEMM's row tiles in either order (the
    light tiles after every heavy one, or walked with their expert's heavy
    ones): every step matches the oracle, and the two orders give
    bit-identical results. fine_s has only light row tiles per chunk
    (~24 rows per expert), balanced_m experts of ~512 rows with and
    without a short third tile."""
    need_gpu()
    cfg = CASES[name] if name in CASES else get_config("balanced", T=2048, M=256, H=416)
    print(f"[layer] tile order {order} {name} {layout} R={R}", flush=True)
    try:
        L.flowmoe_set_tile_order(order)
        layer, inp = run_layer(cfg, layout, R=R)
        check_against_oracle(cfg, layout, layer, inp, R)
        other = "joined" if order == "split" else "split"
        L.flowmoe_set_tile_order(other)
        layer2, _ = run_layer(cfg, layout, R=R)
    finally:
        L.flowmoe_set_tile_order("auto")
    for nm in ("y", "dx", "dw_gate", "dw1", "dw2", "x_disp", "dx_disp"):
        assert torch.equal(getattr(layer, nm), getattr(layer2, nm)), nm


@pytest.mark.parametrize("R", [2, 4])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_layer_chunks_f32(R, act, layout):
    """fp32 layers in chunks: the weight gradients of all chunks come from one
    fp32 GEMM per weight whose reduction walks the chunks' rows in turn."""
    need_gpu()
    cfg = get_config("tiny", act=act)
    print(f"[layer] f32 {act} {layout} R={R}", flush=True)
    layer, inp = run_layer(cfg, layout, R=R)
    check_against_oracle(cfg, layout, layer, inp, R)


@pytest.mark.parametrize("name,R", [("balanced_s", 1), ("skewed_s", 1), ("fine_s", 4),
                                    ("large_s", 2)])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_layer_full_softmax_gate(name, R, layout):
    """The layer with the Switch-style gate (FLOWMOE_GATE_FULL): the skewed
    layer is top-1, whose renormalised gate has no gradient; here its router
    gets one, and every step still matches the oracle."""
    need_gpu()
    cfg = CASES[name].replace(gate="full")
    print(f"[layer] full gate {name} {layout} R={R}", flush=True)
    layer, inp = run_layer(cfg, layout, R=R)
    check_against_oracle(cfg, layout, layer, inp, R)
    # every expert's logit of a token with a kept assignment has a gradient
    # (a token whose assignments were all dropped has dw = 0, hence none)
    live = np.any(host(layer.d_topk_w) != 0.0, axis=1)
    assert live.any() and host(layer.dw_gate).any()
    assert np.all(host(layer.d_logits)[live] != 0.0)


@pytest.mark.parametrize("name,R", [("tiny", 1), ("tiny", 2), ("balanced_s", 1), ("skewed_s", 1),
                                    ("large_s", 2), ("fine_s", 4)])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_layer_biased_experts(name, R, layout):
    """Biased two-layer experts (b1, b3 on the first layer, b2 on the second)
    in the chunked layer: every output and gradient against the oracle, the
    bias gradients summed over the chunks; rows past an expert's count in
    the padded layout stay zero."""
    need_gpu()
    cfg = CASES[name].replace(expert_bias=True)
    print(f"[layer] biased experts {name} {layout} R={R}", flush=True)
    layer, inp = run_layer(cfg, layout, R=R)
    ref = check_against_oracle(cfg, layout, layer, inp, R)
    if layout == "padded":
        for r, c in enumerate(ref["chunks"]):
            live = np.zeros(c["rows"], bool)
            for e in range(cfg.E):
                live[c["offsets"][e]:c["offsets"][e] + c["counts"][e]] = True
            assert not host(layer.y_disp[r])[~live].any(), f"y_disp padding of chunk {r}"
            assert not host(layer.a_save[r])[~live].any(), f"a_save padding of chunk {r}"


def test_two_streams_equal_one_stream_and_deterministic():
    need_gpu()
    cfg = CASES["fine_s"]
    inp = make_inputs(cfg)
    a, _ = run_layer(cfg, "packed", two_streams=True, inp=inp)
    b, _ = run_layer(cfg, "packed", two_streams=False, inp=inp)
    c, _ = run_layer(cfg, "packed", two_streams=True, inp=inp)
    for name in ("logits", "topk_idx", "topk_w", "slot", "x_disp", "h_save", "a_save", "y_disp", "y",
                 "dy_disp", "d_topk_w", "dx_disp", "dx", "d_logits", "dw_gate", "dw1", "dw3", "dw2"):
        ta, tb, tc = getattr(a, name), getattr(b, name), getattr(c, name)
        assert torch.equal(ta, tb), f"{name}: two streams differ from one"
        assert torch.equal(ta, tc), f"{name}: not deterministic"


@pytest.mark.parametrize("name,R", [("balanced_s", 1), ("fine_s", 4)])
def test_layer_graph_replays_equal_eager(name, R):
    """A layer fwd+bwd step captured in a HIP graph (R chunks, two streams
    joined through the layer's events) replays bit-identical to the eager
    step, replay after replay, with eager work and synchronizations in
    between (nothing in the captured step is a memset node)."""
    need_gpu()
    cfg = CASES[name]
    inp = make_inputs(cfg)
    ref, _ = run_layer(cfg, "packed", R=R, inp=inp)
    from paper_2510_00207_amd.layer import MoELayer
    layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=R, f=cfg.f, act=cfg.act,
                     dtype=cfg.dtype, layout="packed", bias=cfg.zipf_bias, device=dev())
    load_layer(layer, inp)
    bufs = layer.bufs()
    gs, sm = torch.cuda.Stream(), torch.cuda.Stream()
    # eager run first (the library's one-time set-up happens outside the capture)
    layer.forward(gs, sm, bufs=bufs)
    layer.backward(gs, sm, bufs=bufs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=gs):
        layer.forward(gs, sm, bufs=bufs)
        layer.backward(gs, sm, bufs=bufs)
    names = ("logits", "topk_idx", "topk_w", "slot", "x_disp", "h_save", "a_save", "y_disp", "y",
             "dy_disp", "d_topk_w", "dx_disp", "dx", "d_logits", "dw_gate", "dw1", "dw2")
    # buffers in the dispatched layout: only the live rows of each chunk are
    # written (the packed tail past offsets[E] is not)
    disp = ("x_disp", "h_save", "a_save", "y_disp", "dy_disp", "dx_disp")
    live = [int(v) for v in ref.offsets[:, cfg.E].tolist()]
    for rep in range(3):
        for nm in names:  # clobber the outputs eagerly between replays
            getattr(layer, nm).fill_(7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for nm in names:
            a, b = getattr(layer, nm), getattr(ref, nm)
            if nm in disp:
                for r in range(R):
                    assert torch.equal(a[r, :live[r]], b[r, :live[r]]), f"replay {rep}: {nm} chunk {r}"
            else:
                assert torch.equal(a, b), f"replay {rep}: {nm}"
