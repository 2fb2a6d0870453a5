"""Row kernels (dispatch gather/scatter, combine, combine backward, dispatch
backward and its fusion with the gate's dx term) in both row-stream kinds,
forced through flowmoe_set_row_streams at sizes the oracle checks element by
element: non-temporal streams are otherwise taken only by calls that move at
least 256 MB. Every kind must match the oracle (Sec. 2.1 dispatch and
combine, and their backward) and the two kinds must agree bitwise. Also the
calls with no rows at all (C = 0, null row buffers)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_close, dev, host, need_gpu
from paper_2510_00207_amd import _lib as L

pytestmark = pytest.mark.gpu


@pytest.fixture
def row_streams():
    yield L.flowmoe_set_row_streams
    L.flowmoe_set_row_streams("auto")


def _shape(T, M, E, k, C, layout, dtype="bf16"):
    return L.make_shape(T, M, 8, E, k, C, L.BF16 if dtype == "bf16" else L.F32, L.GELU,
                        L.PADDED if layout == "padded" else L.PACKED, L.GATE_RENORM)


# k = 1: row gather; k = 2: scatter, and the combine kernels' four-step loads
# (tokens of at most two experts); k = 6: per-token arrays of 8. M = 2056 has
# four 512-element steps and a ragged 8-element tail, M = 1000 fewer than two.
@pytest.mark.parametrize("layout", ["packed", "padded"])
@pytest.mark.parametrize("k,E,M", [(1, 8, 2056), (2, 8, 2056), (2, 16, 1000), (6, 64, 1000),
                                   (6, 16, 2056), (3, 8, 520)])
def test_row_kernels_both_stream_kinds(k, E, M, layout, row_streams):
    need_gpu()
    rng = np.random.default_rng(100 * k + E + M)
    T = 611
    d = dev()
    bf = torch.bfloat16
    lg = rng.standard_normal((T, E)) + np.log(np.arange(1, E + 1))[::-1] * 0.5
    idx, w = oracle.topk_select(lg, k)
    C = oracle.capacity(T, E, k, 1.0)  # skewed logits: some experts overflow
    rt = oracle.route(idx, E, C, layout)
    rows = rt["rows"]
    live = rows if layout == "padded" else int(rt["offsets"][-1])
    assert 0 < live and not rt["kept"].all()
    t = lambda a, dt=bf: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    rnd = lambda *s: host(t(rng.standard_normal(s)))
    x64, y_disp64, dy64, dx_disp64 = rnd(T, M), rnd(rows, M), rnd(T, M), rnd(rows, M)
    wg64 = host(t(rng.standard_normal((M, E)) * 0.05))
    dtw64 = rng.standard_normal((T, k)).astype(np.float32).astype(np.float64)
    s = _shape(T, M, E, k, C, layout)
    i32 = lambda a: t(a, torch.int32)
    w_t = t(w, torch.float32)
    w32 = host(w_t)
    idx_t = i32(idx)
    ref_xd = oracle.dispatch(x64, rt["row_src"], k)
    ref_y = oracle.combine(y_disp64, rt["slot"], w32)
    ref_dyd, ref_dw = oracle.combine_bwd(dy64, y_disp64, rt["slot"], w32)
    ref_dx = oracle.dispatch_bwd(dx_disp64, rt["slot"])
    g = oracle.gate_bwd(x64, wg64, idx, w32, dtw64)
    out = {}
    for mode in ("nt", "cached"):
        row_streams(mode)
        counts = torch.full((E,), -7, dtype=torch.int32, device=d)
        offsets = torch.full((E + 1,), -7, dtype=torch.int32, device=d)
        slot = torch.full((T, k), -7, dtype=torch.int32, device=d)
        row_src = torch.full((rows,), -7, dtype=torch.int32, device=d)
        x_disp = torch.full((rows, M), 3.0, dtype=bf, device=d)
        L.flowmoe_dispatch(s, idx_t, t(x64), counts, offsets, slot, row_src, None, x_disp)
        y = torch.full((T, M), 3.0, dtype=bf, device=d)
        L.flowmoe_combine(s, t(y_disp64), slot, w_t, y)
        dy_disp = torch.full((rows, M), 3.0, dtype=bf, device=d)
        dtw = torch.full((T, k), 3.0, device=d)
        L.flowmoe_combine_bwd(s, t(dy64), t(y_disp64), slot, w_t, counts, offsets, dy_disp, dtw)
        dx = torch.full((T, M), 3.0, dtype=bf, device=d)
        L.flowmoe_dispatch_bwd(s, t(dx_disp64), slot, dx)
        torch.cuda.synchronize()
        assert np.array_equal(host(slot), rt["slot"]), mode
        assert np.array_equal(host(x_disp)[:live], ref_xd[:live]), f"{mode}: x_disp not a copy"
        if layout == "padded":  # rows past each expert's count are zero
            assert not host(x_disp)[host(row_src) < 0].any(), mode
        assert_close(host(y), ref_y, "bf16", f"{mode} y")
        assert_close(host(dy_disp)[:live], ref_dyd[:live], "bf16", f"{mode} dy_disp")
        assert_close(host(dtw), ref_dw, "bf16", f"{mode} d_topk_w")
        assert_close(host(dx), ref_dx, "bf16", f"{mode} dx")
        out[mode] = (x_disp, y, dy_disp, dtw, dx)
    for name, a, b in zip(("x_disp", "y", "dy_disp", "d_topk_w", "dx"), out["nt"], out["cached"]):
        assert torch.equal(a, b), f"{name}: the two row-stream kinds differ"


@pytest.mark.parametrize("k,E", [(1, 8), (2, 8), (6, 64)])
def test_layer_dispatch_bwd_with_gate_term_both_kinds(k, E, row_streams):
    """The layer's dispatch backward fused with the gate's dx term
    (dx = sum of dx_disp rows + d_logits W_g^T) in both row-stream kinds,
    through flowmoe_layer_bwd, against the oracle's dx."""
    need_gpu()
    from gpu_helpers import f64_inputs, load_layer, oracle_for_layer
    from moe_inputs import get_config, make_inputs
    from paper_2510_00207_amd.layer import MoELayer
    cfg = get_config("fine", T=768, M=2056, H=64, E=E, k=k, f=1.0, R=1, seed=7 + k)
    inp = make_inputs(cfg)
    res = {}
    for mode in ("nt", "cached"):
        row_streams(mode)
        layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=1, f=cfg.f,
                         act=cfg.act, dtype=cfg.dtype, device=dev())
        load_layer(layer, inp)
        layer.forward()
        layer.backward()
        torch.cuda.synchronize()
        res[mode] = layer
    ref = oracle_for_layer(f64_inputs(inp), cfg, 1, "packed", host(res["nt"].logits))
    for mode, layer in res.items():
        assert np.array_equal(host(layer.topk_idx), ref["topk_idx"])
        assert_close(host(layer.y), ref["y"], "bf16", f"{mode} y")
        assert_close(host(layer.dx), ref["dx"], "bf16", f"{mode} dx")
        assert_close(host(layer.d_topk_w), ref["d_topk_w"], "bf16", f"{mode} d_topk_w")
    for name in ("x_disp", "y", "dy_disp", "d_topk_w", "dx"):
        assert torch.equal(getattr(res["nt"], name), getattr(res["cached"], name)), name


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["packed", "padded"])
def test_no_rows_null_buffers(dtype, layout):
    """C = 0: every assignment is dropped and the calls have no rows, so the
    row buffers may be null. Dispatch writes counts 0 and slots -1; combine
    writes y = 0; the combine backward d_topk_w = 0; the dispatch backward
    dx = 0 (Sec. 2.1 with every assignment over capacity)."""
    need_gpu()
    T, M, E, k = 300, 136, 8, 2
    rng = np.random.default_rng(3)
    d = dev()
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    idx, w = oracle.topk_select(rng.standard_normal((T, E)), k)
    s = _shape(T, M, E, k, 0, layout, dtype)
    assert L.flowmoe_rows_capacity(s) == 0
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(d).to(dt)
    counts = torch.full((E,), -7, dtype=torch.int32, device=d)
    offsets = torch.full((E + 1,), -7, dtype=torch.int32, device=d)
    slot = torch.full((T, k), -7, dtype=torch.int32, device=d)
    x = t(rng.standard_normal((T, M)), td)
    L.flowmoe_dispatch(s, t(idx, torch.int32), x, counts, offsets, slot, None, None, None)
    y = torch.full((T, M), 3.0, dtype=td, device=d)
    L.flowmoe_combine(s, None, slot, t(w, torch.float32), y)
    dtw = torch.full((T, k), 3.0, device=d)
    L.flowmoe_combine_bwd(s, t(rng.standard_normal((T, M)), td), None, slot, t(w, torch.float32),
                          counts, offsets, None, dtw)
    dx = torch.full((T, M), 3.0, dtype=td, device=d)
    L.flowmoe_dispatch_bwd(s, None, slot, dx)
    torch.cuda.synchronize()
    ref = oracle.route(idx, E, 0, layout)
    assert np.array_equal(host(counts), ref["counts"]) and not ref["counts"].any()
    assert np.array_equal(host(offsets), ref["offsets"])
    assert np.all(host(slot) == -1)
    assert torch.all(y == 0) and torch.all(dtw == 0) and torch.all(dx == 0)
