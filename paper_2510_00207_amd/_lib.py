"""ctypes binding of libflowmoe (include/flowmoe.h): argument marshalling only.

Every function here has the name of the C entry point it calls and forwards
its arguments: torch tensors (their data_ptr()), integers (raw device
addresses) or None (null). A non-OK status raises FlowMoEError with the
library's message. Streams default to torch's current stream. There is no
fallback: if libflowmoe.so has not been built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# FLOWMOE_LIB names another build of the library (the host-sanitized one)
LIB_PATH = os.environ.get("FLOWMOE_LIB") or os.path.join(_HERE, "libflowmoe.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_HIP, ERR_WORKSPACE = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
GELU, SWIGLU = 0, 1
PACKED, PADDED = 0, 1
GATE_RENORM, GATE_FULL = 0, 1
WS_DISPATCH, WS_FFN_BWD, WS_GATE_BWD, WS_LAYER_BWD, WS_MHA_BWD, WS_LAYER_BWD_MHA = 0, 1, 2, 3, 4, 5

_STATUS = {1: "FLOWMOE_ERR_INVALID", 2: "FLOWMOE_ERR_UNSUPPORTED", 3: "FLOWMOE_ERR_HIP",
           4: "FLOWMOE_ERR_WORKSPACE"}


class FlowMoEError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32)
                for n in ("T", "M", "H", "E", "k", "C", "dtype", "act", "layout", "gate")]


class MhaShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("seq_len", "heads", "head_dim", "causal")]


_VP = ctypes.c_void_p
_LAYER_FIELDS = [
    "w_gate", "bias", "w1", "w3", "w2", "b1", "b3", "b2",
    "x", "logits", "topk_idx", "topk_w", "counts", "offsets", "slot", "row_src", "load",
    "x_disp", "h_save", "a_save", "y_disp", "y",
    "dy", "dy_disp", "d_topk_w", "dx_disp", "dx", "d_logits", "dw_gate", "dbias", "dw1", "dw3",
    "dw2", "db1", "db3", "db2",
    "mha", "mha_in", "w_qkv", "w_o", "qkv", "attn", "lse", "d_attn", "d_qkv", "delta", "d_in",
    "dw_qkv", "dw_o", "ws",
]


class LayerBufs(ctypes.Structure):
    _fields_ = [(n, _VP) for n in _LAYER_FIELDS] + [("ws_bytes", ctypes.c_size_t)]


_lib = None


def load():
    """Load libflowmoe.so (built by paper_2510_00207_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    # torch ships its own HIP runtime with the same soname as the system one;
    # loading torch first makes libflowmoe bind to that single runtime, so the
    # streams and device pointers torch hands over are valid here.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2510_00207_amd.build` "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = _VP, ctypes.c_int32, ctypes.c_size_t
    SP = ctypes.POINTER(Shape)
    MP = ctypes.POINTER(MhaShape)
    sig = {
        "flowmoe_version": ([], ctypes.c_char_p),
        "flowmoe_last_error": ([], ctypes.c_char_p),
        "flowmoe_capacity": ([I32, I32, I32, ctypes.c_double], I32),
        "flowmoe_rows_capacity": ([SP], ctypes.c_int64),
        "flowmoe_workspace_bytes": ([SP, I32], SZ),
        "flowmoe_gate_topk": ([SP, P, P, P, P, P, P, P], I32),
        "flowmoe_route": ([SP, P, P, P, P], I32),
        "flowmoe_dispatch": ([SP, P, P, P, P, P, P, P, P, P, SZ, P], I32),
        "flowmoe_expert_ffn": ([SP, P, P, P, P, P, P, P, P, P, P, P, P, P], I32),
        "flowmoe_combine": ([SP, P, P, P, P, P], I32),
        "flowmoe_combine_bwd": ([SP, P, P, P, P, P, P, P, P, P], I32),
        "flowmoe_expert_ffn_bwd": ([SP, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, I32, P, SZ,
                                    P], I32),
        "flowmoe_dispatch_bwd": ([SP, P, P, P, P], I32),
        "flowmoe_gate_topk_bwd": ([SP, P, P, P, P, P, P, P, P, P, P, I32, P, SZ, P], I32),
        "flowmoe_gate_topk_bwd_noalloc": ([SP, P, P, P, P, P, P, P, P, P, P, I32, P], I32),
        "flowmoe_trace_start": ([P, P, I32, ctypes.c_uint32], I32),
        "flowmoe_trace_stop": ([], I32),
        "flowmoe_set_gemm_tiles": ([I32], I32),
        "flowmoe_set_row_streams": ([I32], I32),
        "flowmoe_set_tile_order": ([I32], I32),
        "flowmoe_attention_fwd": ([SP, MP, P, P, P, P], I32),
        "flowmoe_attention_bwd": ([SP, MP, P, P, P, P, P, P, P], I32),
        "flowmoe_mha_fwd": ([SP, MP, P, P, P, P, P, P, P, P], I32),
        "flowmoe_mha_bwd": ([SP, MP] + [P] * 13 + [I32, P, SZ, P], I32),
        "flowmoe_layer_fwd": ([SP, I32, ctypes.POINTER(LayerBufs), P, P, P], I32),
        "flowmoe_layer_bwd": ([SP, I32, ctypes.POINTER(LayerBufs), P, P, P], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def ptr(t) -> int | None:
    """Device address of a tensor, an integer address, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s) -> int | None:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(status: int) -> None:
    if status != OK:
        raise FlowMoEError(status, load().flowmoe_last_error().decode())


def make_shape(T, M, H, E, k, C, dtype=BF16, act=GELU, layout=PACKED, gate=GATE_RENORM) -> Shape:
    return Shape(T, M, H, E, k, C, dtype, act, layout, gate)


# ---- utilities ---------------------------------------------------------------
def flowmoe_version() -> str:
    return load().flowmoe_version().decode()


def flowmoe_last_error() -> str:
    return load().flowmoe_last_error().decode()


def flowmoe_capacity(T: int, E: int, k: int, f: float) -> int:
    return load().flowmoe_capacity(T, E, k, f)


def flowmoe_rows_capacity(shape: Shape) -> int:
    return load().flowmoe_rows_capacity(ctypes.byref(shape))


def flowmoe_workspace_bytes(shape: Shape, kind: int) -> int:
    return load().flowmoe_workspace_bytes(ctypes.byref(shape), kind)


# ---- forward -------------------------------------------------------------------
def flowmoe_gate_topk(shape, x, w_gate, bias, logits, topk_idx, topk_w, stream=None):
    _check(load().flowmoe_gate_topk(ctypes.byref(shape), ptr(x), ptr(w_gate), ptr(bias), ptr(logits),
                                    ptr(topk_idx), ptr(topk_w), _stream(stream)))


def flowmoe_route(shape, logits, topk_idx, topk_w, stream=None):
    _check(load().flowmoe_route(ctypes.byref(shape), ptr(logits), ptr(topk_idx), ptr(topk_w),
                                _stream(stream)))


def flowmoe_dispatch(shape, topk_idx, x, counts, offsets, slot, row_src, load_, x_disp,
                     ws=None, ws_bytes=0, stream=None):
    _check(load().flowmoe_dispatch(ctypes.byref(shape), ptr(topk_idx), ptr(x), ptr(counts),
                                   ptr(offsets), ptr(slot), ptr(row_src), ptr(load_), ptr(x_disp),
                                   ptr(ws), ws_bytes, _stream(stream)))


def flowmoe_expert_ffn(shape, x_disp, counts, offsets, w1, w3, w2, h_save, a_save, y_disp,
                       stream=None, b1=None, b3=None, b2=None):
    _check(load().flowmoe_expert_ffn(ctypes.byref(shape), ptr(x_disp), ptr(counts), ptr(offsets),
                                     ptr(w1), ptr(w3), ptr(w2), ptr(b1), ptr(b3), ptr(b2),
                                     ptr(h_save), ptr(a_save), ptr(y_disp), _stream(stream)))


def flowmoe_combine(shape, y_disp, slot, topk_w, y, stream=None):
    _check(load().flowmoe_combine(ctypes.byref(shape), ptr(y_disp), ptr(slot), ptr(topk_w), ptr(y),
                                  _stream(stream)))


# ---- backward ------------------------------------------------------------------
def flowmoe_combine_bwd(shape, dy, y_disp, slot, topk_w, counts, offsets, dy_disp, d_topk_w,
                        stream=None):
    _check(load().flowmoe_combine_bwd(ctypes.byref(shape), ptr(dy), ptr(y_disp), ptr(slot),
                                      ptr(topk_w), ptr(counts), ptr(offsets), ptr(dy_disp),
                                      ptr(d_topk_w), _stream(stream)))


def flowmoe_expert_ffn_bwd(shape, dy_disp, x_disp, h_save, a_save, counts, offsets, w1, w3, w2,
                           dx_disp, dw1, dw3, dw2, accumulate, ws, ws_bytes, stream=None,
                           db1=None, db3=None, db2=None):
    _check(load().flowmoe_expert_ffn_bwd(ctypes.byref(shape), ptr(dy_disp), ptr(x_disp),
                                         ptr(h_save), ptr(a_save), ptr(counts), ptr(offsets),
                                         ptr(w1), ptr(w3), ptr(w2), ptr(dx_disp), ptr(dw1),
                                         ptr(dw3), ptr(dw2), ptr(db1), ptr(db3), ptr(db2),
                                         int(accumulate), ptr(ws), ws_bytes, _stream(stream)))


def flowmoe_dispatch_bwd(shape, dx_disp, slot, dx, stream=None):
    _check(load().flowmoe_dispatch_bwd(ctypes.byref(shape), ptr(dx_disp), ptr(slot), ptr(dx),
                                       _stream(stream)))


def flowmoe_gate_topk_bwd(shape, x, w_gate, logits, topk_idx, topk_w, d_topk_w, d_logits, dw_gate,
                          dbias, dx, accumulate, ws, ws_bytes, stream=None):
    _check(load().flowmoe_gate_topk_bwd(ctypes.byref(shape), ptr(x), ptr(w_gate), ptr(logits),
                                        ptr(topk_idx), ptr(topk_w), ptr(d_topk_w), ptr(d_logits),
                                        ptr(dw_gate), ptr(dbias), ptr(dx), int(accumulate), ptr(ws),
                                        ws_bytes, _stream(stream)))


NOALLOC_SCRATCH_BYTES = 32 << 20


def flowmoe_gate_topk_bwd_noalloc(shape, x, w_gate, logits, topk_idx, topk_w, d_topk_w, d_logits,
                                  dw_gate, dbias, dx, accumulate, stream=None):
    _check(load().flowmoe_gate_topk_bwd_noalloc(ctypes.byref(shape), ptr(x), ptr(w_gate),
                                                ptr(logits), ptr(topk_idx), ptr(topk_w),
                                                ptr(d_topk_w), ptr(d_logits), ptr(dw_gate),
                                                ptr(dbias), ptr(dx), int(accumulate),
                                                _stream(stream)))


# ---- the attention part of AT_r ----------------------------------------------------
def make_mha_shape(seq_len, heads, head_dim, causal) -> MhaShape:
    return MhaShape(seq_len, heads, head_dim, int(bool(causal)))


def flowmoe_attention_fwd(shape, mha, qkv, attn, lse, stream=None):
    _check(load().flowmoe_attention_fwd(ctypes.byref(shape), ctypes.byref(mha), ptr(qkv), ptr(attn),
                                        ptr(lse), _stream(stream)))


def flowmoe_attention_bwd(shape, mha, qkv, attn, lse, d_attn, d_qkv, delta, stream=None):
    _check(load().flowmoe_attention_bwd(ctypes.byref(shape), ctypes.byref(mha), ptr(qkv), ptr(attn),
                                        ptr(lse), ptr(d_attn), ptr(d_qkv), ptr(delta),
                                        _stream(stream)))


def flowmoe_mha_fwd(shape, mha, inp, w_qkv, w_o, qkv, attn, lse, out, stream=None):
    _check(load().flowmoe_mha_fwd(ctypes.byref(shape), ctypes.byref(mha), ptr(inp), ptr(w_qkv),
                                  ptr(w_o), ptr(qkv), ptr(attn), ptr(lse), ptr(out),
                                  _stream(stream)))


def flowmoe_mha_bwd(shape, mha, inp, w_qkv, w_o, qkv, attn, lse, d_out, d_attn, d_qkv, delta, d_in,
                    dw_qkv, dw_o, accumulate, ws=None, ws_bytes=0, stream=None):
    _check(load().flowmoe_mha_bwd(ctypes.byref(shape), ctypes.byref(mha), ptr(inp), ptr(w_qkv),
                                  ptr(w_o), ptr(qkv), ptr(attn), ptr(lse), ptr(d_out), ptr(d_attn),
                                  ptr(d_qkv), ptr(delta), ptr(d_in), ptr(dw_qkv), ptr(dw_o),
                                  int(accumulate), ptr(ws), int(ws_bytes), _stream(stream)))


# ---- kernel tracing --------------------------------------------------------------
K_NAMES = ["gate", "route", "scan", "gather", "ffn1", "ffn2", "swiglu_act", "combine",
           "combine_bwd", "dgrad1", "wgrad2", "wgrad1", "dgrad2", "gate_bwd_wt", "gate_bwd_token",
           "gate_bwd_dw", "gate_bwd_reduce", "bias_grad", "attn_qkv", "attn_fwd", "attn_out",
           "attn_dgrad", "attn_bwd_dq", "attn_bwd_dkdv", "attn_wgrad"]
K = {n: i for i, n in enumerate(K_NAMES)}
K_GEMM = ("ffn1", "ffn2", "dgrad1", "wgrad2", "wgrad1", "dgrad2")


def kind_mask(names) -> int:
    m = 0
    for n in names:
        m |= 1 << K[n]
    return m


def flowmoe_trace_start(events, kinds, pairs: int, mask: int):
    """events: ctypes array of 2*pairs hipEvent_t; kinds: ctypes int32 array."""
    _check(load().flowmoe_trace_start(ctypes.cast(events, ctypes.c_void_p),
                                      ctypes.cast(kinds, ctypes.c_void_p), pairs, mask))


def flowmoe_trace_stop() -> int:
    return load().flowmoe_trace_stop()


TILES = {"auto": 0, "wide": 1, "narrow": 2}


def flowmoe_set_gemm_tiles(tiles: str | int) -> None:
    """Grouped-GEMM tile shape for later launches: "auto", "wide" (256 x 256)
    or "narrow" (256 x 128), or the FLOWMOE_TILES_* value."""
    _check(load().flowmoe_set_gemm_tiles(TILES[tiles] if isinstance(tiles, str) else tiles))


TILE_ORDERS = {"auto": 0, "split": 1, "joined": 2}


def flowmoe_set_tile_order(order: str | int) -> None:
    """Row-mode tile order of the grouped GEMM for later launches: "auto",
    "split" (light tiles after every heavy one) or "joined" (an expert's
    light tiles with its heavy ones), or the FLOWMOE_TILE_ORDER_* value."""
    _check(load().flowmoe_set_tile_order(TILE_ORDERS[order] if isinstance(order, str) else order))


ROW_STREAMS = {"auto": 0, "nt": 1, "cached": 2}


def flowmoe_set_row_streams(mode: str | int) -> None:
    """Row-stream kind of the dispatch/combine kernels for later launches:
    "auto", "nt" (non-temporal) or "cached", or the FLOWMOE_ROWS_* value."""
    _check(load().flowmoe_set_row_streams(ROW_STREAMS[mode] if isinstance(mode, str) else mode))


# ---- R-chunk layer ---------------------------------------------------------------
def layer_bufs(**tensors) -> LayerBufs:
    """LayerBufs from keyword tensors (names of the C struct fields)."""
    b = LayerBufs()
    for name, t in tensors.items():
        if name == "ws_bytes":
            b.ws_bytes = int(t)
        elif name == "mha":  # a MhaShape (or None), kept alive with the buffers
            b._mha = t
            b.mha = None if t is None else ctypes.addressof(t)
        elif name not in _LAYER_FIELDS:
            raise KeyError(name)
        else:
            setattr(b, name, ptr(t))
    return b


def _events(trace):
    if trace is None:
        return None
    arr = (ctypes.c_void_p * len(trace))(*[e.cuda_event if hasattr(e, "cuda_event") else int(e)
                                           for e in trace])
    return arr


def flowmoe_layer_fwd(shape, R, bufs, s_compute=None, s_comm=None, trace=None):
    if trace is not None and len(trace) < 8 * R:
        raise ValueError(f"the forward trace takes 8 * R = {8 * R} events, got {len(trace)}")
    sc = _stream(s_compute)
    sm = sc if s_comm is None else _stream(s_comm)
    _check(load().flowmoe_layer_fwd(ctypes.byref(shape), R, ctypes.byref(bufs), sc, sm,
                                    _events(trace)))


def bwd_trace_len(R: int, mha: bool) -> int:
    """Events of flowmoe_layer_bwd's trace: 8R + 2, or 10R + 4 with the attention."""
    return 10 * R + 4 if mha else 8 * R + 2


def flowmoe_layer_bwd(shape, R, bufs, s_compute=None, s_comm=None, trace=None):
    need = bwd_trace_len(R, bool(bufs.mha))
    if trace is not None and len(trace) < need:
        raise ValueError(f"the backward trace takes {need} events, got {len(trace)}")
    sc = _stream(s_compute)
    sm = sc if s_comm is None else _stream(s_comm)
    _check(load().flowmoe_layer_bwd(ctypes.byref(shape), R, ctypes.byref(bufs), sc, sm,
                                    _events(trace)))
