"""Host-side checks of the C ABI: every declared symbol is exported, host
utilities agree with the oracle's definitions, and argument validation
rejects bad calls before anything is enqueued (no GPU needed)."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2510_00207_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "flowmoe.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(flowmoe_[a-z0-9_]+)\s*\(", src)))


def test_header_symbols_exported(flowmoe_lib):
    names = declared_functions()
    assert len(names) >= 16
    raw = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n
    assert L.flowmoe_version().startswith("flowmoe")


def test_capacity_matches_oracle(flowmoe_lib):
    for f in (0.5, 1.0, 1.1, 1.2, 1.25, 1.5, 2.0):
        for T in (1, 7, 100, 500, 4096, 16384):
            for E in (1, 3, 8, 10, 64):
                for k in (1, 2, 6):
                    assert L.flowmoe_capacity(T, E, k, f) == oracle.capacity(T, E, k, f), (T, E, k, f)
    assert L.flowmoe_capacity(4096, 8, 2, 1.2) == 1229
    assert L.flowmoe_capacity(-1, 8, 2, 1.2) == -1
    assert L.flowmoe_capacity(8, 0, 2, 1.2) == -1
    assert L.flowmoe_capacity(8, 8, 2, 0.0) == -1


def test_rows_capacity(flowmoe_lib):
    for layout in ("packed", "padded"):
        for (T, E, k, C) in [(256, 4, 2, 160), (4096, 8, 2, 1229), (8192, 16, 1, 512), (10, 4, 2, 0)]:
            s = L.make_shape(T, 64, 64, E, k, C, L.BF16, L.GELU, L.PADDED if layout == "padded" else L.PACKED)
            assert L.flowmoe_rows_capacity(s) == oracle.rows_capacity(T, E, k, C, layout)


def test_workspace_sizes(flowmoe_lib):
    s = L.make_shape(4096, 1024, 4096, 8, 2, 1229, L.BF16, L.GELU, L.PACKED)
    # one tile of 1024 assignments: no histograms
    assert L.flowmoe_workspace_bytes(L.make_shape(512, 1024, 4096, 8, 2, 160, L.BF16, L.GELU,
                                                  L.PACKED), L.WS_DISPATCH) == 0
    # more tiles: one E-wide int32 histogram per tile, 256-byte aligned
    for T, E, k in [(513, 8, 2), (4096, 8, 2), (20000, 64, 2), (49152, 16, 2)]:
        sd = L.make_shape(T, 1024, 4096, E, k, 1229, L.BF16, L.GELU, L.PACKED)
        tiles = -(-T * k // 1024)
        want = -(-tiles * E * 4 // 256) * 256
        assert L.flowmoe_workspace_bytes(sd, L.WS_DISPATCH) == want
        assert L.flowmoe_workspace_bytes(sd, L.WS_LAYER_BWD) >= want
    assert L.flowmoe_workspace_bytes(s, L.WS_FFN_BWD) >= 8192 * 4096 * 2
    assert L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD) >= 1024 * 8 * 4
    # the layer keeps dH in h_save: its workspace serves the gate backward and
    # the forward's dispatch scan
    assert L.flowmoe_workspace_bytes(s, L.WS_LAYER_BWD) == max(
        L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD), L.flowmoe_workspace_bytes(s, L.WS_DISPATCH))
    sw = L.make_shape(4096, 1024, 4096, 8, 2, 1229, L.BF16, L.SWIGLU, L.PACKED)
    assert L.flowmoe_workspace_bytes(sw, L.WS_FFN_BWD) >= 8192 * 8192 * 2


FAKE = 0x10000  # never dereferenced: every case below fails validation first


@pytest.mark.parametrize("field,value,status", [
    ("E", 0, L.ERR_INVALID), ("E", 65, L.ERR_UNSUPPORTED), ("k", 0, L.ERR_INVALID),
    ("k", 9, L.ERR_INVALID), ("M", 12, L.ERR_INVALID), ("M", 0, L.ERR_INVALID),
    ("T", -1, L.ERR_INVALID), ("dtype", 7, L.ERR_INVALID), ("act", 3, L.ERR_INVALID),
    ("layout", 2, L.ERR_INVALID),
])
def test_gate_validation(flowmoe_lib, field, value, status):
    s = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16)
    setattr(s, field, value)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk(s, FAKE, FAKE, None, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == status
    assert L.flowmoe_last_error()


def test_k_above_8_unsupported(flowmoe_lib):
    s = L.make_shape(16, 64, 64, 16, 9, 8, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_route(s, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_UNSUPPORTED


def test_null_pointers_rejected(flowmoe_lib):
    s = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk(s, None, FAKE, None, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "x" in str(ei.value)
    with pytest.raises(L.FlowMoEError):
        L.flowmoe_dispatch(s, FAKE, FAKE, None, FAKE, FAKE, FAKE, None, FAKE, stream=0)
    with pytest.raises(L.FlowMoEError):
        L.flowmoe_combine(s, FAKE, None, FAKE, FAKE, stream=0)
    sw = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16, L.SWIGLU)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_expert_ffn(sw, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert "w3" in str(ei.value)


def test_h_and_c_validation(flowmoe_lib):
    s = L.make_shape(16, 64, 60, 4, 2, 8, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_expert_ffn(s, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "H" in str(ei.value)
    s = L.make_shape(16, 64, 64, 4, 2, -1, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_dispatch(s, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID


def test_workspace_checked_before_launch(flowmoe_lib):
    s = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16)
    need = L.flowmoe_workspace_bytes(s, L.WS_FFN_BWD)
    assert need > 0
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_expert_ffn_bwd(s, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                 None, FAKE, 0, None, 0, stream=0)
    assert ei.value.status == L.ERR_WORKSPACE
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk_bwd(s, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, FAKE, 1,
                                stream=0)
    assert ei.value.status == L.ERR_WORKSPACE


def test_dispatch_workspace_checked(flowmoe_lib):
    # 18000 assignments: 18 tiles of 1024, so the scan may use 18 x 8 int32
    # histograms; a workspace that is given must hold them (null: no histograms)
    s = L.make_shape(9000, 64, 64, 8, 2, 2250, L.BF16)
    need = L.flowmoe_workspace_bytes(s, L.WS_DISPATCH)
    assert need == 768
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_dispatch(s, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, need - 1,
                           stream=0)
    assert ei.value.status == L.ERR_WORKSPACE and "flowmoe_dispatch" in str(ei.value)
    b = L.LayerBufs()
    for name in L._LAYER_FIELDS:
        if name != "mha":  # (a host struct: None = no attention)
            setattr(b, name, FAKE)
    b.ws_bytes = need - 256
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_layer_fwd(s, 1, b, s_compute=0, s_comm=0)
    assert ei.value.status == L.ERR_WORKSPACE and "flowmoe_layer_fwd" in str(ei.value)


def test_layer_validation(flowmoe_lib):
    s = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16)
    b = L.LayerBufs()
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_layer_fwd(s, 0, b, s_compute=0, s_comm=0)
    assert ei.value.status == L.ERR_INVALID
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_layer_fwd(s, 1, b, s_compute=0, s_comm=0)
    assert "w_gate" in str(ei.value)


def test_misaligned_tensors_rejected(flowmoe_lib):
    # layer-dtype tensors are moved in 16-byte vectors: a misaligned one is an
    # argument error, caught before anything is enqueued
    s = L.make_shape(16, 64, 64, 4, 2, 8, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk(s, FAKE + 8, FAKE, None, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "aligned" in str(ei.value)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk(s, FAKE, FAKE + 2, None, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "w_gate" in str(ei.value)
    need = L.flowmoe_workspace_bytes(s, L.WS_GATE_BWD)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_gate_topk_bwd(s, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE + 4, 0, FAKE,
                                need, stream=0)
    assert ei.value.status == L.ERR_INVALID and "dx" in str(ei.value)


def test_gemm_tiles_setting(flowmoe_lib):
    for t in ("wide", "narrow", "auto"):
        L.flowmoe_set_gemm_tiles(t)
    raw = ctypes.CDLL(L.LIB_PATH)
    raw.flowmoe_set_gemm_tiles.argtypes = [ctypes.c_int32]
    assert raw.flowmoe_set_gemm_tiles(3) == L.ERR_INVALID
    assert raw.flowmoe_set_gemm_tiles(-1) == L.ERR_INVALID


def test_tile_order_setting(flowmoe_lib):
    for o in ("joined", "split", "auto"):
        L.flowmoe_set_tile_order(o)
    raw = ctypes.CDLL(L.LIB_PATH)
    raw.flowmoe_set_tile_order.argtypes = [ctypes.c_int32]
    assert raw.flowmoe_set_tile_order(3) == L.ERR_INVALID
    assert raw.flowmoe_set_tile_order(-1) == L.ERR_INVALID


def test_capacity_exact_on_adversarial_factors(flowmoe_lib):
    """C = ceil(f k T / E) on the decimal value of f, exactly as the oracle's
    rational arithmetic: factors with many digits, factors just above and
    below products that are integers, and large T (a double product with a
    relative slack would round some of these the wrong way)."""
    cases = [(1 << 20, 1, 1, 1.000000000001), (1 << 20, 1, 1, 0.999999999999),
             (1 << 30, 1, 1, 1.0000000001), (1 << 30, 3, 1, 1.0000000001),
             (4096, 8, 2, 1.2), (10, 1, 1, 1.1), (3, 1, 1, 0.1 + 0.2), (1 << 30, 1, 2, 0.5),
             (100, 7, 3, 1.0 / 3.0), (2147483647, 64, 8, 0.123456789012345),
             (2147483647, 1, 1, 1e-300), (12345, 17, 5, 123.456), (1, 64, 1, 5e-324)]
    rng = __import__("numpy").random.default_rng(17)
    for _ in range(300):
        digits = int(rng.integers(1, 17))
        f = float(f"{rng.integers(1, 10**digits)}e{int(rng.integers(-digits - 1, 2))}")
        cases.append((int(rng.integers(0, 1 << 31)), int(rng.integers(1, 65)),
                      int(rng.integers(1, 9)), f))
    for T, E, k, f in cases:
        want = oracle.capacity(T, E, k, f)
        got = L.flowmoe_capacity(T, E, k, f)
        assert got == (want if want <= 2**31 - 1 else -1), (T, E, k, f, got, want)
    assert L.flowmoe_capacity(1 << 20, 1, 1, 1.000000000001) == (1 << 20) + 1
    assert L.flowmoe_capacity(8, 1, 1, float("inf")) == -1
    assert L.flowmoe_capacity(8, 1, 1, float("nan")) == -1
    assert L.flowmoe_capacity(2147483647, 1, 8, 1.0) == -1  # above INT32_MAX


def test_row_streams_setting(flowmoe_lib):
    for m in ("nt", "cached", "auto"):
        L.flowmoe_set_row_streams(m)
    raw = ctypes.CDLL(L.LIB_PATH)
    raw.flowmoe_set_row_streams.argtypes = [ctypes.c_int32]
    assert raw.flowmoe_set_row_streams(3) == L.ERR_INVALID
    assert raw.flowmoe_set_row_streams(-1) == L.ERR_INVALID


# ---------------------------------------------------------------------------
# the attention part of AT_r
# ---------------------------------------------------------------------------
def test_mha_validation(flowmoe_lib):
    s = L.make_shape(1024, 1024, 64, 4, 2, 8, L.BF16)
    m = L.make_mha_shape(512, 16, 64, True)
    cases = [
        (L.make_shape(1024, 1024, 64, 4, 2, 8, L.F32), m, L.ERR_UNSUPPORTED, "BF16"),
        (s, L.make_mha_shape(512, 8, 96, True), L.ERR_UNSUPPORTED, "head_dim"),
        (s, L.make_mha_shape(512, 8, 64, True), L.ERR_INVALID, "heads * head_dim"),
        (s, L.make_mha_shape(384, 16, 64, True), L.ERR_INVALID, "whole number of sequences"),
        (s, L.make_mha_shape(0, 16, 64, True), L.ERR_INVALID, "seq_len"),
        (s, L.MhaShape(512, 16, 64, 2), L.ERR_INVALID, "causal"),
    ]
    for shape, mha, status, text in cases:
        for call in (lambda: L.flowmoe_attention_fwd(shape, mha, FAKE, FAKE, FAKE, stream=0),
                     lambda: L.flowmoe_mha_fwd(shape, mha, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                               stream=0),
                     lambda: L.flowmoe_mha_bwd(shape, mha, *([FAKE] * 13), 0, stream=0)):
            with pytest.raises(L.FlowMoEError) as ei:
                call()
            assert ei.value.status == status and text in str(ei.value), str(ei.value)
    # null and misaligned tensors
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_attention_fwd(s, m, FAKE, None, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "attn is null" in str(ei.value)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_attention_bwd(s, m, FAKE, FAKE, FAKE + 2, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "lse is not 4-byte aligned" in str(ei.value)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_mha_fwd(s, m, FAKE, FAKE + 8, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == L.ERR_INVALID and "w_qkv is not 16-byte aligned" in str(ei.value)
    # no tokens: nothing to do, no tensor needed (the backward's weight gradients still are)
    s0 = L.make_shape(0, 1024, 64, 4, 2, 8, L.BF16)
    L.flowmoe_attention_fwd(s0, m, None, None, None, stream=0)
    L.flowmoe_mha_fwd(s0, m, None, None, None, None, None, None, None, stream=0)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_mha_bwd(s0, m, *([None] * 13), 0, stream=0)
    assert "dw_qkv is null" in str(ei.value)


def test_mha_workspace(flowmoe_lib):
    # the attention's weight gradients split their token rows into partial
    # sums when their 256 x 256 output tiles are too few for the 256 CUs:
    # M = 1024: dW_qkv has 4 x 12 tiles -> 6 splits of 1024 x 3072 floats
    # (dW_o: 4 x 4 -> 8 splits, fewer bytes); M = 4096 needs no split
    m = L.make_mha_shape(512, 16, 64, True)
    for M, need in ((1024, 6 * 1024 * 3072 * 4), (2048, 2 * 2048 * 6144 * 4), (4096, 0)):
        s = L.make_shape(1024, M, 64, 4, 2, 8, L.BF16)
        assert L.flowmoe_workspace_bytes(s, L.WS_MHA_BWD) == need, M
        assert L.flowmoe_workspace_bytes(s, L.WS_LAYER_BWD_MHA) >= max(
            need, L.flowmoe_workspace_bytes(s, L.WS_LAYER_BWD))
    s = L.make_shape(1024, 1024, 64, 4, 2, 8, L.BF16)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_mha_bwd(s, m, *([FAKE] * 13), 0, FAKE, 6 * 1024 * 3072 * 4 - 1, stream=0)
    assert ei.value.status == L.ERR_WORKSPACE and "flowmoe_mha_bwd" in str(ei.value)


def test_layer_mha_validation(flowmoe_lib):
    # the layer's chunk must hold whole sequences; its attention buffers are checked
    s = L.make_shape(768, 256, 64, 4, 2, 8, L.BF16)
    base = {n: FAKE for n in L._LAYER_FIELDS if n not in ("mha", "bias", "load", "w3", "dw3", "b1",
                                                             "b3", "b2", "db1", "db3", "db2", "dbias")}
    need = L.flowmoe_workspace_bytes(s, L.WS_LAYER_BWD_MHA)
    b = L.layer_bufs(ws_bytes=need, mha=L.make_mha_shape(512, 4, 64, True), **base)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_layer_fwd(s, 2, b, s_compute=0, s_comm=0)
    assert "whole number of sequences" in str(ei.value)
    bad = dict(base, delta=None)
    b = L.layer_bufs(ws_bytes=need, mha=L.make_mha_shape(256, 4, 64, True), **bad)
    with pytest.raises(L.FlowMoEError) as ei:
        L.flowmoe_layer_bwd(s, 2, b, s_compute=0, s_comm=0)
    assert "bufs->delta is null" in str(ei.value)
    with pytest.raises(ValueError):  # the binding checks the trace length first
        L.flowmoe_layer_bwd(s, 2, b, s_compute=0, s_comm=0, trace=[0] * (8 * 2 + 2))
    assert L.bwd_trace_len(2, True) == 24 and L.bwd_trace_len(2, False) == 18
