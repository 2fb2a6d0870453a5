"""Per-call parity of the C ABI entry points against the oracle step they
implement, including edge cases: ties and signed zeros in the gate, T = 1,
E = 1, k = E, C = 0, C >= T*k, heavy drops, multi-tile scans."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_close, dev, host, need_gpu
from moe_inputs import as_f64, get_config, make_inputs, to_torch
from paper_2510_00207_amd import _lib as L

pytestmark = pytest.mark.gpu


def _shape(T, M, H, E, k, C, dtype="bf16", act="gelu", layout="packed", gate="renorm"):
    return L.make_shape(T, M, H, E, k, C, L.BF16 if dtype == "bf16" else L.F32,
                        L.SWIGLU if act == "swiglu" else L.GELU,
                        L.PADDED if layout == "padded" else L.PACKED,
                        L.GATE_FULL if gate == "full" else L.GATE_RENORM)


@pytest.mark.parametrize("E,k", [(1, 1), (3, 2), (4, 4), (8, 2), (16, 1), (24, 3), (32, 4), (33, 5), (64, 6),
                                 (64, 8)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gate_topk(E, k, dtype):
    need_gpu()
    cfg = get_config("balanced", T=300, M=136, H=8, E=E, k=k, dtype=dtype, seed=E * 10 + k)
    inp = make_inputs(cfg, with_dy=False, x_zero_rows=[0, 7])
    d = dev()
    x, wg = to_torch(inp["x"], d), to_torch(inp["w_gate"], d)
    bias = torch.linspace(-0.3, 0.3, E, device=d, dtype=torch.float32)
    logits = torch.empty(cfg.T, E, device=d)
    idx = torch.empty(cfg.T, k, dtype=torch.int32, device=d)
    w = torch.empty(cfg.T, k, device=d)
    s = _shape(cfg.T, cfg.M, 8, E, k, 0, dtype)
    L.flowmoe_gate_topk(s, x, wg, bias, logits, idx, w)
    torch.cuda.synchronize()
    own = oracle.gate_logits(as_f64(inp["x"]), as_f64(inp["w_gate"]), host(bias))
    gl = host(logits)
    assert np.max(np.abs(gl - own)) <= 1e-4 * np.max(np.abs(own))
    ref_i, ref_w = oracle.topk_select(gl, k)
    assert np.array_equal(host(idx), ref_i)
    np.testing.assert_allclose(host(w), ref_w, rtol=2e-6, atol=2e-7)
    # zero tokens: logits equal the bias, selection by bias then index
    assert np.allclose(gl[0], host(bias))


@pytest.mark.parametrize("T,M,E,k", [(77, 520, 64, 6), (130, 1000, 33, 3), (40, 4104, 8, 2),
                                   (200, 2056, 64, 6), (300, 1096, 8, 2)])
def test_gate_topk_chunked_weights(T, M, E, k):
    """W_g taller than one LDS chunk of the bf16 gate (32 KB of rows at a pitch
    of 16 * ceil(E / 16) + 8: 224 rows at E = 64, 288 at E = 33 (copied
    element by element), 672 at E = 8), with a ragged last chunk; M = 2056
    and 1096: 65 and 35 k steps of 32 over the waves of one-group blocks,
    the last step 8 rows deep."""
    need_gpu()
    cfg = get_config("balanced", T=T, M=M, H=8, E=E, k=k, dtype="bf16", seed=M + E)
    inp = make_inputs(cfg, with_dy=False)
    d = dev()
    x, wg = to_torch(inp["x"], d), to_torch(inp["w_gate"], d)
    logits = torch.empty(T, E, device=d)
    idx = torch.empty(T, k, dtype=torch.int32, device=d)
    w = torch.empty(T, k, device=d)
    L.flowmoe_gate_topk(_shape(T, M, 8, E, k, 0), x, wg, None, logits, idx, w)
    torch.cuda.synchronize()
    own = oracle.gate_logits(as_f64(inp["x"]), as_f64(inp["w_gate"]), None)
    gl = host(logits)
    assert np.max(np.abs(gl - own)) <= 1e-4 * np.max(np.abs(own))
    ref_i, ref_w = oracle.topk_select(gl, k)
    assert np.array_equal(host(idx), ref_i)
    np.testing.assert_allclose(host(w), ref_w, rtol=2e-6, atol=2e-7)


@pytest.mark.parametrize("T,M,E,k", [
    (16368, 64, 8, 2), (16400, 64, 8, 2), (65600, 32, 4, 1),
    (9000, 96, 64, 6),    # 563 groups: 2 per block, top-k on 8 lanes per token
    (16400, 128, 20, 3),  # 4 groups per block, two 16-expert blocks, 4 lanes per token
    (8200, 64, 40, 8),    # k = 8, three 16-expert blocks
])
def test_gate_topk_many_tokens(T, M, E, k):
    """Token counts around the group thresholds of the bf16 gate (512 and
    1024 groups of 16 tokens), ragged in the last block, and the wide-gate
    top-k at each lane count."""
    need_gpu()
    cfg = get_config("balanced", T=T, M=M, H=8, E=E, k=k, dtype="bf16", seed=T % 97)
    inp = make_inputs(cfg, with_dy=False)
    d = dev()
    x, wg = to_torch(inp["x"], d), to_torch(inp["w_gate"], d)
    bias = torch.linspace(-0.1, 0.1, E, device=d, dtype=torch.float32)
    logits = torch.empty(T, E, device=d)
    idx = torch.empty(T, k, dtype=torch.int32, device=d)
    w = torch.empty(T, k, device=d)
    L.flowmoe_gate_topk(_shape(T, M, 8, E, k, 0), x, wg, bias, logits, idx, w)
    torch.cuda.synchronize()
    own = oracle.gate_logits(as_f64(inp["x"]), as_f64(inp["w_gate"]), host(bias))
    gl = host(logits)
    assert np.max(np.abs(gl - own)) <= 1e-4 * np.max(np.abs(own))
    ref_i, ref_w = oracle.topk_select(gl, k)
    assert np.array_equal(host(idx), ref_i)
    np.testing.assert_allclose(host(w), ref_w, rtol=2e-6, atol=2e-7)


@pytest.mark.parametrize("T,E,k", [(600, 12, 4), (600, 40, 5), (9000, 64, 6), (16400, 24, 3)])
def test_gate_topk_ties(T, E, k):
    """Equal logits through the bf16 gate itself: W_g's columns repeat with
    period 8, so experts e and e + 8 get bit-identical logits (each column is
    reduced in the same order), and some tokens are all zero (every logit
    equal to zero). The selection must take the lower index of equal logits
    on every top-k path (segmented lanes for E <= 16, 16/8/4 lanes per token
    above)."""
    need_gpu()
    M = 64
    rng = np.random.default_rng(E * 1000 + k)
    d = dev()
    x = torch.from_numpy(rng.standard_normal((T, M)).astype(np.float32)).to(d).to(torch.bfloat16)
    x[::7] = 0
    base = rng.standard_normal((M, 8)).astype(np.float32) * 0.05
    wg_np = np.stack([base[:, e % 8] for e in range(E)], axis=1)
    wg = torch.from_numpy(wg_np).to(d).to(torch.bfloat16)
    logits = torch.empty(T, E, device=d)
    idx = torch.empty(T, k, dtype=torch.int32, device=d)
    w = torch.empty(T, k, device=d)
    L.flowmoe_gate_topk(_shape(T, M, 8, E, k, 0), x, wg, None, logits, idx, w)
    torch.cuda.synchronize()
    gl = host(logits)
    for e in range(8, E):  # the repeated columns really tie
        assert np.array_equal(gl[:, e], gl[:, e % 8])
    ref_i, ref_w = oracle.topk_select(gl, k)
    assert np.array_equal(host(idx), ref_i)
    np.testing.assert_allclose(host(w), ref_w, rtol=2e-6, atol=2e-7)
    assert list(host(idx)[0]) == list(range(k))  # token 0 is all zero


# the full softmax gate's weights divide by a sum over all E experts in fp32
FULL_W_TOL = dict(rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("T,M,E,k", [
    (700, 64, 4, 1), (700, 64, 8, 2), (700, 128, 16, 1), (700, 64, 24, 3), (700, 64, 64, 6),
    (700, 64, 64, 8), (9000, 96, 64, 6), (16400, 64, 8, 2), (8200, 64, 40, 1),
])
def test_gate_topk_full_softmax(T, M, E, k):
    """FLOWMOE_GATE_FULL: the same selection, weights = the selected experts'
    probabilities under the softmax over all E logits (every top-k path:
    segmented lanes for E <= 16, 16/8/4 lanes per token above)."""
    need_gpu()
    rng = np.random.default_rng(T + E + k)
    d = dev()
    x = torch.from_numpy(rng.standard_normal((T, M)).astype(np.float32)).to(d).to(torch.bfloat16)
    wg = torch.from_numpy((rng.standard_normal((M, E)) * 0.1).astype(np.float32)).to(d).to(
        torch.bfloat16)
    logits = torch.empty(T, E, device=d)
    idx = torch.empty(T, k, dtype=torch.int32, device=d)
    w = torch.empty(T, k, device=d)
    L.flowmoe_gate_topk(_shape(T, M, 8, E, k, 0, gate="full"), x, wg, None, logits, idx, w)
    torch.cuda.synchronize()
    gl = host(logits)
    ref_i, ref_w = oracle.topk_select(gl, k, "full")
    assert np.array_equal(host(idx), ref_i)
    np.testing.assert_allclose(host(w), ref_w, **FULL_W_TOL)
    if k < E:
        assert np.all(host(w).sum(axis=1) < 1.0)


def test_route_full_softmax_ties():
    need_gpu()
    rng = np.random.default_rng(11)
    d = dev()
    for E in (2, 5, 8, 17, 64):
        for k in sorted({1, min(E, 3)}):
            T = 257
            L_ = (rng.integers(-3, 4, size=(T, E)) * 0.25).astype(np.float32)
            L_[5, :] = 1.0
            lt = torch.from_numpy(L_).to(d)
            idx = torch.empty(T, k, dtype=torch.int32, device=d)
            w = torch.empty(T, k, device=d)
            L.flowmoe_route(_shape(T, 8, 8, E, k, 0, gate="full"), lt, idx, w)
            torch.cuda.synchronize()
            ref_i, ref_w = oracle.topk_select(L_.astype(np.float64), k, "full")
            assert np.array_equal(host(idx), ref_i), (E, k)
            np.testing.assert_allclose(host(w), ref_w, **FULL_W_TOL)
            np.testing.assert_allclose(host(w)[5], np.full(k, 1.0 / E), rtol=1e-6)


@pytest.mark.parametrize("T,M,E,k", [(333, 136, 8, 3), (700, 64, 16, 1), (1000, 256, 64, 6),
                                     (4100, 128, 24, 2)])
def test_gate_bwd_full_softmax(T, M, E, k):
    """FLOWMOE_GATE_FULL backward: dense d_logits (-p_e s off the selection),
    dW_g and db from them, and dx += d_logits W_g^T over all E experts (a
    GEMM of the bf16 hi/lo parts of d_logits against the stacked W_g^T)."""
    need_gpu()
    rng = np.random.default_rng(T * 3 + E)
    d = dev()
    td = torch.bfloat16
    rnd = lambda *s_, sc=1.0: host(torch.from_numpy(rng.standard_normal(s_) * sc).to(d).to(td))
    x64, wg64, dx0 = rnd(T, M), rnd(M, E, sc=0.05), rnd(T, M)
    gl = (x64 @ wg64).astype(np.float32).astype(np.float64)
    idx, w = oracle.topk_select(gl, k, "full")
    dtw = rng.standard_normal((T, k)).astype(np.float32)
    t = lambda a, dt=td: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    s = _shape(T, M, 8, E, k, 0, gate="full")
    nws = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    dlog = torch.empty(T, E, device=d)
    dwg = torch.full((M, E), 3.0, device=d)
    db = torch.full((E,), 3.0, device=d)
    dx = t(dx0)
    w32 = w.astype(np.float32)
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), t(gl, torch.float32), t(idx, torch.int32),
                            t(w32, torch.float32), t(dtw, torch.float32), dlog, dwg, db, dx, 0, ws,
                            nws)
    torch.cuda.synchronize()
    g = oracle.gate_bwd(x64, wg64, idx, w32.astype(np.float64), dtw.astype(np.float64), gl, "full")
    assert np.all(host(dlog) != 0.0)  # every expert has a gradient
    assert_close(host(dlog), g["d_logits"], "f32", "d_logits", tol=1e-5)
    assert_close(host(dwg), g["dw_gate"], "bf16", "dw_gate")
    assert_close(host(db), g["dbias"], "bf16", "dbias")
    assert_close(host(dx), dx0 + g["dx_gate"], "bf16", "dx + dense gate term")


def test_route_ties_and_signed_zeros():
    need_gpu()
    rng = np.random.default_rng(7)
    d = dev()
    for E in (2, 5, 8, 17, 64):
        for k in sorted({1, min(E, 3), min(E, 8)}):
            T = 257
            L_ = (rng.integers(-3, 4, size=(T, E)) * 0.25).astype(np.float32)
            z = L_ == 0
            L_[z] = rng.choice(np.array([0.0, -0.0], np.float32), size=int(z.sum()))
            L_[5, :] = 1.0                      # all equal
            L_[6, :] = -0.0
            lt = torch.from_numpy(L_).to(d)
            idx = torch.empty(T, k, dtype=torch.int32, device=d)
            w = torch.empty(T, k, device=d)
            L.flowmoe_route(_shape(T, 8, 8, E, k, 0, "f32"), lt, idx, w)
            torch.cuda.synchronize()
            ref_i, ref_w = oracle.topk_select(L_.astype(np.float64), k)
            assert np.array_equal(host(idx), ref_i), (E, k)
            np.testing.assert_allclose(host(w), ref_w, rtol=2e-6, atol=2e-7)
            assert list(host(idx)[5]) == list(range(k))


def _run_dispatch(T, M, E, k, C, layout, idx_np, x_t, with_ws=False):
    d = dev()
    s = _shape(T, M, 8, E, k, C, "bf16" if x_t.dtype == torch.bfloat16 else "f32", layout=layout)
    rows = L.flowmoe_rows_capacity(s)
    counts = torch.full((E,), -7, dtype=torch.int32, device=d)
    offsets = torch.full((E + 1,), -7, dtype=torch.int32, device=d)
    slot = torch.full((max(T * k, 1),), -7, dtype=torch.int32, device=d)
    row_src = torch.full((max(rows, 1),), -7, dtype=torch.int32, device=d)
    load = torch.full((E,), -7, dtype=torch.int32, device=d)
    x_disp = torch.full((max(rows, 1), M), 3.0, dtype=x_t.dtype, device=d)
    idx_t = torch.from_numpy(idx_np.astype(np.int32)).to(d)
    ws, nws = None, 0
    if with_ws:  # the tile-histogram scan (more than one tile of 1024 assignments)
        nws = L.flowmoe_workspace_bytes(s, L.WS_DISPATCH)
        assert (nws > 0) == (T * k > 1024)
        ws = torch.full((max(nws, 1),), 0x5A, dtype=torch.uint8, device=d)
    L.flowmoe_dispatch(s, idx_t, x_t, counts, offsets, slot, row_src, load, x_disp, ws, nws)
    torch.cuda.synchronize()
    return dict(counts=host(counts), offsets=host(offsets), slot=host(slot[:T * k]).reshape(T, k),
                row_src=host(row_src[:rows]), load=host(load), x_disp=x_disp[:rows], rows=rows)


@pytest.mark.parametrize("layout", ["packed", "padded"])
@pytest.mark.parametrize("T,E,k,cf", [
    (1, 1, 1, 1.0), (1, 4, 2, 1.0), (37, 1, 1, 1.0), (100, 4, 4, 1.0), (300, 8, 2, 1.2),
    (1000, 16, 1, 1.0), (2048, 64, 6, 1.5), (777, 7, 3, 0.3), (5000, 8, 2, 1.25),
    (13000, 4, 4, 1.1),  # T*k = 52000: more assignments than the scan stages in LDS
    (1024, 8, 1, 1.0), (1025, 8, 1, 1.0),  # one tile; two with a one-assignment tail
    (16384, 8, 1, 1.0), (16385, 8, 1, 1.0),
    (20000, 64, 2, 1.1), (40000, 16, 3, 0.8),
])
def test_dispatch(T, E, k, cf, layout):
    need_gpu()
    rng = np.random.default_rng(T + E)
    M = 72
    # skewed logits so that some experts overflow
    lg = rng.standard_normal((T, E)) + np.log(np.arange(1, E + 1))[::-1] * 0.7
    idx, _ = oracle.topk_select(lg, k)
    x = rng.standard_normal((T, M)).astype(np.float32)
    x_t = torch.from_numpy(x).to(dev()).to(torch.bfloat16)
    xb = host(x_t)
    for C in sorted({0, 1, oracle.capacity(T, E, k, cf), T * k}):
        g = _run_dispatch(T, M, E, k, C, layout, idx, x_t)
        ref = oracle.route(idx, E, C, layout)
        if T * k > 1024:  # both scans: the same integers
            h = _run_dispatch(T, M, E, k, C, layout, idx, x_t, with_ws=True)
            for key in ("counts", "offsets", "slot", "load", "row_src"):
                assert np.array_equal(h[key], g[key]), (key, C)
            assert torch.equal(h["x_disp"], g["x_disp"]), C
        assert np.array_equal(g["counts"], ref["counts"]), C
        assert np.array_equal(g["offsets"], ref["offsets"]), C
        assert np.array_equal(g["slot"], ref["slot"]), C
        assert np.array_equal(g["load"], ref["demand"]), C
        live = ref["rows"] if layout == "padded" else int(ref["offsets"][-1])
        assert np.array_equal(g["row_src"][:live], ref["row_src"][:live]), C
        xd = oracle.dispatch(xb, ref["row_src"], k)
        assert np.array_equal(host(g["x_disp"][:live]), xd[:live]), C


@pytest.fixture
def gemm_tiles():
    """Set the grouped-GEMM tile shape for one test; back to "auto" after it."""
    yield L.flowmoe_set_gemm_tiles
    L.flowmoe_set_gemm_tiles("auto")


@pytest.fixture
def tile_order():
    """Set the grouped-GEMM row-tile order for one test; back to "auto" after it."""
    yield L.flowmoe_set_tile_order
    L.flowmoe_set_tile_order("auto")


@pytest.mark.parametrize("biased", [False, True], ids=["nobias", "bias"])
@pytest.mark.parametrize("MHT", [(200, 264, "auto"), (224, 288, "wide"), (224, 288, "narrow")],
                         ids=["staged", "streaming-wide", "streaming-narrow"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_expert_ffn_fwd_bwd(dtype, act, layout, MHT, biased, gemm_tiles):
    """(200, 264): reductions not multiples of 32 (register-staged bf16 GEMM);
    (224, 288): multiples of 32 (LDS-streaming bf16 GEMM, 256 x 256 and
    256 x 128 tiles); all ragged. The counts give row tiles of every class:
    empty, a few rows, under and over half a tile, full. Biased experts: b1
    (b3) and b2 on the data rows only, and their gradients as per-expert
    column sums."""
    need_gpu()
    rng = np.random.default_rng(3)
    E, k = 6, 1
    M, H, tiles = MHT
    gemm_tiles(tiles)
    # per-expert counts spanning empty, tiny, tile-exact and ragged groups
    cnt = np.array([0, 1, 127, 128, 129, 300])
    C = 300
    T = int(cnt.sum())
    idx = np.repeat(np.arange(E), cnt)[:, None]
    rt = oracle.route(idx, E, C, layout)
    cfg = get_config("balanced", T=T, M=M, H=H, E=E, k=1, dtype=dtype, act=act, seed=11,
                     expert_bias=biased)
    inp = make_inputs(cfg)
    d = dev()
    bt = {kk: (None if inp[kk] is None else torch.from_numpy(inp[kk]).to(d))
          for kk in ("b1", "b3", "b2")}
    b64 = {kk: (None if inp[kk] is None else inp[kk].astype(np.float64)) for kk in ("b1", "b3", "b2")}
    xb = as_f64(inp["x"])
    x_disp64 = oracle.dispatch(xb, rt["row_src"], 1)
    rows = rt["rows"]
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    x_disp = torch.from_numpy(x_disp64).to(d).to(td)
    counts = torch.from_numpy(rt["counts"].astype(np.int32)).to(d)
    offsets = torch.from_numpy(rt["offsets"].astype(np.int32)).to(d)
    w1 = to_torch(inp["w1"], d)
    w3 = to_torch(inp["w3"], d) if act == "swiglu" else None
    w2 = to_torch(inp["w2"], d)
    HW = 2 * H if act == "swiglu" else H
    h_save = torch.full((rows, HW), 5.0, dtype=td, device=d)
    a_save = torch.full((rows, H), 5.0, dtype=td, device=d)
    y_disp = torch.full((rows, M), 5.0, dtype=td, device=d)
    s = _shape(T, M, H, E, 1, C, dtype, act, layout)
    assert L.flowmoe_rows_capacity(s) == rows
    L.flowmoe_expert_ffn(s, x_disp, counts, offsets, w1, w3, w2, h_save, a_save, y_disp, **bt)
    w64 = {kk: (None if inp[kk] is None else as_f64(inp[kk])) for kk in ("w1", "w3", "w2")}
    ref = oracle.expert_ffn(x_disp64, rt["counts"], rt["offsets"], w64["w1"], w64["w3"], w64["w2"], act,
                            **b64)
    # backward with a seeded upstream gradient on the live rows
    dy64 = rng.standard_normal((rows, M))
    live = np.zeros(rows, bool)
    for e in range(E):
        live[rt["offsets"][e]:rt["offsets"][e] + rt["counts"][e]] = True
    dy64[~live] = 0
    dy_t = torch.from_numpy(dy64).to(d).to(td)
    dy64 = host(dy_t)
    dx_disp = torch.full((rows, M), 5.0, dtype=td, device=d)
    dw1 = torch.full((E, M, H), 9.0, device=d)
    dw3 = torch.full((E, M, H), 9.0, device=d) if act == "swiglu" else None
    dw2 = torch.full((E, H, M), 9.0, device=d)
    db = {"db1": torch.full((E, H), 9.0, device=d), "db2": torch.full((E, M), 9.0, device=d),
          "db3": torch.full((E, H), 9.0, device=d) if act == "swiglu" else None}
    if not biased:  # the bias gradients are optional outputs
        db = {kk: None for kk in db}
    nws = L.flowmoe_workspace_bytes(s, L.WS_FFN_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    L.flowmoe_expert_ffn_bwd(s, dy_t, x_disp, h_save, a_save, counts, offsets, w1, w3, w2, dx_disp,
                             dw1, dw3, dw2, 0, ws, nws, **db)
    # accumulate = 1 adds a second identical gradient
    dw2b = dw2.clone()
    db2b = None if db["db2"] is None else db["db2"].clone()
    torch.cuda.synchronize()
    rdx, rdw1, rdw3, rdw2, rdh = oracle.expert_ffn_bwd(dy64, x_disp64, ref, rt["counts"],
                                                       rt["offsets"], w64["w1"], w64["w3"],
                                                       w64["w2"], act, return_dh=True)
    if biased:
        rdb1, rdb3, rdb2 = oracle.expert_bias_grads(dy64, rdh, rt["counts"], rt["offsets"], act)
        assert_close(host(db["db1"]), rdb1, dtype, "db1")
        assert_close(host(db["db2"]), rdb2, dtype, "db2")
        if act == "swiglu":
            assert_close(host(db["db3"]), rdb3, dtype, "db3")
    nl = rows if layout == "padded" else int(rt["offsets"][-1])
    hw = ref["h1"] if act == "gelu" else np.concatenate([ref["h1"], ref["h3"]], axis=1)
    assert_close(host(h_save)[:nl], hw[:nl], dtype, "h_save")
    assert_close(host(a_save)[:nl], ref["a"][:nl], dtype, "a_save")
    assert_close(host(y_disp)[:nl], ref["y_disp"][:nl], dtype, "y_disp")
    if layout == "padded":  # rows past each expert's count are zero
        assert not host(y_disp)[~live].any() and not host(h_save)[~live].any()
    assert_close(host(dx_disp)[:nl], rdx[:nl], dtype, "dx_disp")
    assert_close(host(dw1), rdw1, dtype, "dw1")
    assert_close(host(dw2), rdw2, dtype, "dw2")
    if act == "swiglu":
        assert_close(host(dw3), rdw3, dtype, "dw3")
    L.flowmoe_expert_ffn_bwd(s, dy_t, x_disp, h_save, a_save, counts, offsets, w1, w3, w2, dx_disp,
                             dw1, dw3, dw2, 1, ws, nws, **db)
    torch.cuda.synchronize()
    assert torch.equal(dw2, 2 * dw2b)
    if biased:
        assert torch.equal(db["db2"], 2 * db2b)


@pytest.mark.parametrize("M", [32, 64, 96, 160, 192])
@pytest.mark.parametrize("act", ["gelu", "swiglu"])
def test_expert_ffn_ring_depths(act, M, gemm_tiles):
    """Short reductions on the LDS-streaming GEMM (wide 256 x 256 tiles, a
    4-stage ring of 32-deep k-tiles): K = M of the first GEMM and of the
    input-gradient GEMM gives 1, 2, 3, 5 and 6 k-tiles, K = H = 96 and
    2H = 192 give 3 and 6, and the weight gradients reduce over expert row
    counts of 1 to 6 k-tiles (ragged ones among them): every prologue-only,
    partly steady and steady ring walk, each against the oracle."""
    need_gpu()
    gemm_tiles("wide")
    rng = np.random.default_rng(17)
    E, H = 5, 96
    cnt = np.array([32, 64, 95, 150, 192])
    C = int(cnt.max())
    T = int(cnt.sum())
    idx = np.repeat(np.arange(E), cnt)[:, None]
    rt = oracle.route(idx, E, C, "packed")
    cfg = get_config("balanced", T=T, M=M, H=H, E=E, k=1, dtype="bf16", act=act, seed=23)
    inp = make_inputs(cfg)
    d = dev()
    x_disp64 = oracle.dispatch(as_f64(inp["x"]), rt["row_src"], 1)
    rows = rt["rows"]
    x_disp = torch.from_numpy(x_disp64).to(d).to(torch.bfloat16)
    counts = torch.from_numpy(rt["counts"].astype(np.int32)).to(d)
    offsets = torch.from_numpy(rt["offsets"].astype(np.int32)).to(d)
    w1, w2 = to_torch(inp["w1"], d), to_torch(inp["w2"], d)
    w3 = to_torch(inp["w3"], d) if act == "swiglu" else None
    HW = 2 * H if act == "swiglu" else H
    h_save = torch.full((rows, HW), 5.0, dtype=torch.bfloat16, device=d)
    a_save = torch.full((rows, H), 5.0, dtype=torch.bfloat16, device=d)
    y_disp = torch.full((rows, M), 5.0, dtype=torch.bfloat16, device=d)
    s = _shape(T, M, H, E, 1, C, "bf16", act, "packed")
    L.flowmoe_expert_ffn(s, x_disp, counts, offsets, w1, w3, w2, h_save, a_save, y_disp)
    w64 = {kk: (None if inp[kk] is None else as_f64(inp[kk])) for kk in ("w1", "w3", "w2")}
    ref = oracle.expert_ffn(x_disp64, rt["counts"], rt["offsets"], w64["w1"], w64["w3"], w64["w2"], act)
    dy_t = torch.from_numpy(rng.standard_normal((rows, M))).to(d).to(torch.bfloat16)
    dy64 = host(dy_t)
    dx_disp = torch.full((rows, M), 5.0, dtype=torch.bfloat16, device=d)
    dw1 = torch.full((E, M, H), 9.0, device=d)
    dw3 = torch.full((E, M, H), 9.0, device=d) if act == "swiglu" else None
    dw2 = torch.full((E, H, M), 9.0, device=d)
    nws = L.flowmoe_workspace_bytes(s, L.WS_FFN_BWD)
    ws = torch.empty(max(1, nws), dtype=torch.uint8, device=d)
    L.flowmoe_expert_ffn_bwd(s, dy_t, x_disp, h_save, a_save, counts, offsets, w1, w3, w2, dx_disp,
                             dw1, dw3, dw2, 0, ws, nws)
    torch.cuda.synchronize()
    rdx, rdw1, rdw3, rdw2 = oracle.expert_ffn_bwd(dy64, x_disp64, ref, rt["counts"], rt["offsets"],
                                                  w64["w1"], w64["w3"], w64["w2"], act)
    hw = ref["h1"] if act == "gelu" else np.concatenate([ref["h1"], ref["h3"]], axis=1)
    assert_close(host(h_save), hw, "bf16", "h_save")
    assert_close(host(a_save), ref["a"], "bf16", "a_save")
    assert_close(host(y_disp), ref["y_disp"], "bf16", "y_disp")
    assert_close(host(dx_disp), rdx, "bf16", "dx_disp")
    assert_close(host(dw1), rdw1, "bf16", "dw1")
    assert_close(host(dw2), rdw2, "bf16", "dw2")
    if act == "swiglu":
        assert_close(host(dw3), rdw3, "bf16", "dw3")


@pytest.mark.parametrize("act", ["gelu", "swiglu"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_gemm_tile_shapes_agree(act, layout, gemm_tiles, tile_order):
    """256 x 256 and 256 x 128 tiles, each in the split and the joined
    row-tile order, over several row and column tiles with ragged edges,
    light last row tiles (one live row, four live rows) and an empty
    expert: all match the oracle, and as every output is accumulated in the
    same k order whatever the tile's shape or place in the walk, their
    outputs are bit-identical."""
    need_gpu()
    rng = np.random.default_rng(21)
    E, M, H = 4, 512, 800
    cnt = np.array([700, 513, 0, 260])
    C = 720
    T = int(cnt.sum())
    idx = np.repeat(np.arange(E), cnt)[:, None]
    rt = oracle.route(idx, E, C, layout)
    rows = rt["rows"]
    d = dev()
    bf = torch.bfloat16
    rnd = lambda *sh, sc=1.0: (torch.from_numpy(rng.standard_normal(sh) * sc).to(d).to(bf))
    x_disp, dy = rnd(rows, M), rnd(rows, M)
    live = torch.zeros(rows, dtype=torch.bool)
    for e in range(E):
        live[rt["offsets"][e]:rt["offsets"][e] + rt["counts"][e]] = True
    dy[~live.to(d)] = 0  # upstream gradient only on the live rows
    w1, w2 = rnd(E, M, H, sc=0.05), rnd(E, H, M, sc=0.05)
    w3 = rnd(E, M, H, sc=0.05) if act == "swiglu" else None
    counts = torch.from_numpy(rt["counts"].astype(np.int32)).to(d)
    offsets = torch.from_numpy(rt["offsets"].astype(np.int32)).to(d)
    s = _shape(T, M, H, E, 1, C, "bf16", act, layout)
    HW = 2 * H if act == "swiglu" else H
    nws = L.flowmoe_workspace_bytes(s, L.WS_FFN_BWD)
    out = {}
    for tiles, order in (("wide", "split"), ("narrow", "split"), ("wide", "joined"),
                         ("narrow", "joined")):
        gemm_tiles(tiles)
        tile_order(order)
        h = torch.full((rows, HW), 5.0, dtype=bf, device=d)
        a = torch.full((rows, H), 5.0, dtype=bf, device=d)
        y = torch.full((rows, M), 5.0, dtype=bf, device=d)
        L.flowmoe_expert_ffn(s, x_disp, counts, offsets, w1, w3, w2, h, a, y)
        dx = torch.full((rows, M), 5.0, dtype=bf, device=d)
        dw1 = torch.full((E, M, H), 9.0, device=d)
        dw3 = torch.full((E, M, H), 9.0, device=d) if act == "swiglu" else None
        dw2 = torch.full((E, H, M), 9.0, device=d)
        ws = torch.empty(nws, dtype=torch.uint8, device=d)
        L.flowmoe_expert_ffn_bwd(s, dy, x_disp, h, a, counts, offsets, w1, w3, w2, dx, dw1, dw3, dw2,
                                 0, ws, nws)
        torch.cuda.synchronize()
        out[(tiles, order)] = [t for t in (h, a, y, dx, dw1, dw3, dw2) if t is not None]
        if (tiles, order) == ("wide", "split"):
            x64, dy64 = host(x_disp), host(dy)
            w64 = [None if w is None else host(w) for w in (w1, w3, w2)]
            ref = oracle.expert_ffn(x64, rt["counts"], rt["offsets"], *w64, act)
            rdx, rdw1, rdw3, rdw2 = oracle.expert_ffn_bwd(dy64, x64, ref, rt["counts"], rt["offsets"],
                                                          *w64, act)
        nl = rows if layout == "padded" else int(rt["offsets"][-1])
        assert_close(host(y)[:nl], ref["y_disp"][:nl], "bf16", f"{tiles} {order} y")
        assert_close(host(dx)[:nl], rdx[:nl], "bf16", f"{tiles} {order} dx")
        assert_close(host(dw1), rdw1, "bf16", f"{tiles} {order} dw1")
        assert_close(host(dw2), rdw2, "bf16", f"{tiles} {order} dw2")
    names = [n for n in ("h", "a", "y", "dx", "dw1", "dw3", "dw2") if n != "dw3" or act == "swiglu"]
    first = out[("wide", "split")]
    for key, got in out.items():
        for name, p, q in zip(names, first, got):
            assert torch.equal(p, q), (key, name)


@pytest.mark.parametrize("T,M,E,k", [(3000, 520, 64, 6), (2000, 520, 20, 4), (9000, 1000, 3, 2),
                                     (1000, 264, 3, 2), (777, 1024, 16, 1), (40, 136, 8, 2),
                                     (4097, 2056, 64, 6), (1345, 200, 40, 8), (37, 72, 24, 3),
                                     (8193, 1024, 8, 2), (100, 64, 2, 2), (300, 8, 4, 2)])
def test_gate_bwd_shapes(T, M, E, k):
    """bf16 gate backward on the MFMA dW_g kernel (d_logits rows and dW_g
    partials in one launch, then the reduce): several token splits of whole
    64-token chunks and a ragged last chunk, 64-column x tiles with a ragged
    last one, fewer tokens than one chunk, E not a multiple of 4 and every
    row-tile count (2 E rounded up to 16, 32, 64, 128 rows of the hi/lo
    matrix), k from 1 to 8, the narrowest gates (E = k = 2) and rows of x
    (M = 8, one short column tile): d_logits, dW_g and db against the oracle within
    the fp32 bound (the kernel multiplies a hi + lo bf16 pair per d_logits
    value: about 16 significant bits)."""
    need_gpu()
    rng = np.random.default_rng(T + M + E)
    d = dev()
    x64 = host(torch.from_numpy(rng.standard_normal((T, M))).to(d).to(torch.bfloat16))
    wg64 = host(torch.from_numpy(rng.standard_normal((M, E)) * 0.05).to(d).to(torch.bfloat16))
    idx, w = oracle.topk_select(rng.standard_normal((T, E)), k)
    dtw64 = rng.standard_normal((T, k))
    t = lambda a, dt=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    s = _shape(T, M, 8, E, k, 0, "bf16")
    dlog = torch.empty(T, E, device=d)
    dwg = torch.full((M, E), 3.0, device=d)
    db = torch.full((E,), 3.0, device=d)
    nws = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), None, t(idx, torch.int32), t(w, torch.float32),
                            t(dtw64, torch.float32), dlog, dwg, db, None, 0, ws, nws)
    torch.cuda.synchronize()
    g = oracle.gate_bwd(x64, wg64, idx, host(t(w, torch.float32)), host(t(dtw64, torch.float32)))
    assert_close(host(dlog), g["d_logits"], "f32", "d_logits")
    assert_close(host(dwg), g["dw_gate"], "f32", "dw_gate")
    assert_close(host(db), g["dbias"], "f32", "dbias")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T,M,E,k", [(9000, 1000, 3, 2), (8200, 1032, 16, 4), (16400, 520, 12, 3),
                                     (4100, 4104, 8, 2), (70000, 136, 5, 5)])
def test_gate_bwd_long_inputs(T, M, E, k, dtype):
    """The renormalised gate's backward for E <= 16 over more than 8 M
    elements of x (bf16: the MFMA dW_g kernel over token splits; fp32: the
    register tiles), ragged column tiles and token splits; with the dx term
    and accumulation."""
    need_gpu()
    rng = np.random.default_rng(T + M + E + k)
    d = dev()
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    x64 = host(torch.from_numpy(rng.standard_normal((T, M))).to(d).to(td))
    wg64 = host(torch.from_numpy(rng.standard_normal((M, E)) * 0.05).to(d).to(td))
    idx, w = oracle.topk_select(rng.standard_normal((T, E)), k)
    dtw64 = rng.standard_normal((T, k))
    t = lambda a, dt=td: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    s = _shape(T, M, 8, E, k, 0, dtype)
    dlog = torch.full((T, E), 7.0, device=d)
    dwg = torch.full((M, E), 3.0, device=d)
    db = torch.full((E,), 3.0, device=d)
    dx0 = t(rng.standard_normal((T, M)))
    dx = dx0.clone()
    nws = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), None, t(idx, torch.int32), t(w, torch.float32),
                            t(dtw64, torch.float32), dlog, dwg, db, dx, 0, ws, nws)
    torch.cuda.synchronize()
    g = oracle.gate_bwd(x64, wg64, idx, host(t(w, torch.float32)), host(t(dtw64, torch.float32)))
    assert_close(host(dlog), g["d_logits"], "f32", "d_logits")
    assert_close(host(dwg), g["dw_gate"], "f32", "dw_gate")
    assert_close(host(db), g["dbias"], "f32", "dbias")
    assert_close(host(dx), host(dx0) + g["dx_gate"], dtype, "dx + gate term")
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), None, t(idx, torch.int32), t(w, torch.float32),
                            t(dtw64, torch.float32), dlog, dwg, db, None, 1, ws, nws)
    torch.cuda.synchronize()
    assert_close(host(dwg), 2 * g["dw_gate"], "f32", "dw_gate accumulated")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,E", [(1024, 16), (520, 64)])
def test_gate_bwd_top1_is_exactly_zero(dtype, M, E):
    """One selected expert under the renormalised gate: its weight is exactly
    1, so d_logits = w (dw - w dw) = 0 exactly (Sec. 2.1's gate with a
    single survivor), and so are dW_g, db and the dx term. The call writes
    those zeros over garbage, leaves accumulated gradients as they were and
    dx untouched, whichever dW_g path the shape would take; the oracle
    agrees."""
    need_gpu()
    rng = np.random.default_rng(M + E)
    d = dev()
    T = 777
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.from_numpy(rng.standard_normal((T, M))).to(d).to(dt)
    wg = torch.from_numpy(rng.standard_normal((M, E)) * 0.05).to(d).to(dt)
    idx, w = oracle.topk_select(rng.standard_normal((T, E)), 1)
    assert np.all(w == 1.0)
    dtw = rng.standard_normal((T, 1))
    t = lambda a, ty: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(ty)
    s = _shape(T, M, 8, E, 1, 0, dtype)
    nws = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    for acc in (0, 1):
        dlog = torch.full((T, E), 7.0, device=d)
        dwg = torch.full((M, E), 3.0, device=d)
        db = torch.full((E,), 3.0, device=d)
        dx = torch.from_numpy(rng.standard_normal((T, M))).to(d).to(dt)
        dx0 = dx.clone()
        L.flowmoe_gate_topk_bwd(s, x, wg, None, t(idx, torch.int32), t(w, torch.float32),
                                t(dtw, torch.float32), dlog, dwg, db, dx, acc, ws, nws)
        torch.cuda.synchronize()
        assert torch.all(dlog == 0)
        want = 3.0 if acc else 0.0
        assert torch.all(dwg == want) and torch.all(db == want)
        assert torch.equal(dx, dx0)
    g = oracle.gate_bwd(host(x), host(wg), idx, w, dtw)
    assert np.all(g["d_logits"] == 0) and np.all(g["dw_gate"] == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_combine_and_backward_steps(dtype, layout):
    need_gpu()
    rng = np.random.default_rng(5)
    T, M, E, k = 333, 136, 8, 3
    lg = rng.standard_normal((T, E))
    idx, w = oracle.topk_select(lg, k)
    C = oracle.capacity(T, E, k, 0.9)
    rt = oracle.route(idx, E, C, layout)
    rows = rt["rows"]
    d = dev()
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    rnd = lambda *s: host(torch.from_numpy(rng.standard_normal(s)).to(d).to(td))
    y_disp64, dy64, dx_disp64, x64 = rnd(rows, M), rnd(T, M), rnd(rows, M), rnd(T, M)
    wg64 = host(torch.from_numpy(rng.standard_normal((M, E)) * 0.05).to(d).to(td))
    t = lambda a, dt=td: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    s = _shape(T, M, 8, E, k, C, dtype, layout=layout)
    slot = t(rt["slot"], torch.int32)
    counts = t(rt["counts"], torch.int32)
    offsets = t(rt["offsets"], torch.int32)
    w_t = t(w, torch.float32)
    y = torch.empty(T, M, dtype=td, device=d)
    L.flowmoe_combine(s, t(y_disp64), slot, w_t, y)
    dy_disp = torch.full((rows, M), 7.0, dtype=td, device=d)
    dtw = torch.empty(T, k, device=d)
    L.flowmoe_combine_bwd(s, t(dy64), t(y_disp64), slot, w_t, counts, offsets, dy_disp, dtw)
    dx = torch.empty(T, M, dtype=td, device=d)
    L.flowmoe_dispatch_bwd(s, t(dx_disp64), slot, dx)
    torch.cuda.synchronize()
    assert_close(host(y), oracle.combine(y_disp64, rt["slot"], w), dtype, "y")
    rdy, rdw = oracle.combine_bwd(dy64, y_disp64, rt["slot"], w)
    live = rows if layout == "padded" else int(rt["offsets"][-1])
    assert_close(host(dy_disp)[:live], rdy[:live], dtype, "dy_disp")
    assert_close(host(dtw), rdw, dtype, "d_topk_w")
    rdx = oracle.dispatch_bwd(dx_disp64, rt["slot"])
    assert_close(host(dx), rdx, dtype, "dx")
    # gate backward, with dx accumulation and chunk accumulation of dW_g
    dlog = torch.empty(T, E, device=d)
    dwg = torch.full((M, E), 3.0, device=d)
    db = torch.full((E,), 3.0, device=d)
    nws = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    ws = torch.empty(nws, dtype=torch.uint8, device=d)
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), None, t(idx, torch.int32), w_t, dtw, dlog, dwg, db,
                            dx, 0, ws, nws)
    torch.cuda.synchronize()
    g = oracle.gate_bwd(x64, wg64, idx, w, host(dtw))
    assert_close(host(dlog), g["d_logits"], dtype, "d_logits")
    assert_close(host(dwg), g["dw_gate"], dtype, "dw_gate")
    assert_close(host(db), g["dbias"], dtype, "dbias")
    assert_close(host(dx), rdx + g["dx_gate"], dtype, "dx + gate")
    L.flowmoe_gate_topk_bwd(s, t(x64), t(wg64), None, t(idx, torch.int32), w_t, dtw, dlog, dwg, db,
                            None, 1, ws, nws)
    torch.cuda.synchronize()
    assert_close(host(dwg), 2 * g["dw_gate"], dtype, "dw_gate accumulated")
