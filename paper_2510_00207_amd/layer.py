"""Device buffers for one MoE layer over R token chunks, and the calls that
run it through the C ABI (flowmoe_layer_fwd / flowmoe_layer_bwd).

torch provides device memory and streams only; every step runs in
libflowmoe's HIP kernels.
"""
from __future__ import annotations

import torch

from . import _lib as L

_TORCH_DTYPE = {L.F32: torch.float32, L.BF16: torch.bfloat16}


class MoELayer:
    """Buffers of a layer with T_total = R * T tokens.

    Parameters and inputs (w_gate, bias, w1, w3, w2, the experts' biases b1,
    b3, b2 when expert_bias, x, dy) are attributes the caller fills (or
    replaces with tensors of the same shape and dtype); everything else is
    allocated here. ``mha`` (dict seq_len, head_dim, causal): AT_r includes
    the block's attention; then mha_in, w_qkv and w_o are the caller's inputs
    and x is the attention output the forward writes.
    """

    def __init__(self, *, T_total: int, M: int, H: int, E: int, k: int, R: int = 1,
                 f: float | None = None, C: int | None = None, act: str = "gelu",
                 dtype: str = "bf16", layout: str = "packed", bias: bool = False,
                 gate: str = "renorm", expert_bias: bool = False, mha: dict | None = None,
                 device="cuda"):
        if T_total % R:
            raise ValueError("T_total must be a multiple of R")
        T = T_total // R
        if C is None:
            if f is None:
                raise ValueError("give the capacity C or the capacity factor f")
            C = L.flowmoe_capacity(T, E, k, f)
            if C < 0:
                raise ValueError("invalid capacity arguments")
        self.R, self.T_total = R, T_total
        self.dt = L.BF16 if dtype == "bf16" else L.F32
        self.shape = L.make_shape(T, M, H, E, k, C, self.dt,
                                  L.SWIGLU if act == "swiglu" else L.GELU,
                                  L.PADDED if layout == "padded" else L.PACKED,
                                  L.GATE_FULL if gate == "full" else L.GATE_RENORM)
        self.rows = L.flowmoe_rows_capacity(self.shape)
        if self.rows < 0:
            raise L.FlowMoEError(L.ERR_INVALID, L.flowmoe_last_error())
        td = _TORCH_DTYPE[self.dt]
        dev = torch.device(device)
        z = lambda *s, dtype=td: torch.zeros(*s, dtype=dtype, device=dev)
        i32 = torch.int32
        f32 = torch.float32
        HW = 2 * H if act == "swiglu" else H
        rows = self.rows
        # parameters
        self.w_gate = z(M, E)
        self.bias = z(E, dtype=f32) if bias else None
        self.w1 = z(E, M, H)
        self.w3 = z(E, M, H) if act == "swiglu" else None
        self.w2 = z(E, H, M)
        sw = act == "swiglu"
        self.b1 = z(E, H, dtype=f32) if expert_bias else None
        self.b3 = z(E, H, dtype=f32) if expert_bias and sw else None
        self.b2 = z(E, M, dtype=f32) if expert_bias else None
        # forward
        self.x = z(T_total, M)
        self.logits = z(T_total, E, dtype=f32)
        self.topk_idx = z(T_total, k, dtype=i32)
        self.topk_w = z(T_total, k, dtype=f32)
        self.counts = z(R, E, dtype=i32)
        self.offsets = z(R, E + 1, dtype=i32)
        self.slot = z(T_total, k, dtype=i32)
        self.row_src = z(R, max(rows, 1), dtype=i32)
        self.load = z(R, E, dtype=i32)
        self.x_disp = z(R, max(rows, 1), M)
        self.h_save = z(R, max(rows, 1), HW)
        self.a_save = z(R, max(rows, 1), H)
        self.y_disp = z(R, max(rows, 1), M)
        self.y = z(T_total, M)
        # backward
        self.dy = z(T_total, M)
        self.dy_disp = z(R, max(rows, 1), M)
        self.d_topk_w = z(T_total, k, dtype=f32)
        self.dx_disp = z(R, max(rows, 1), M)
        self.dx = z(T_total, M)
        self.d_logits = z(T_total, E, dtype=f32)
        self.dw_gate = z(M, E, dtype=f32)
        self.dbias = z(E, dtype=f32) if bias else None
        self.dw1 = z(E, M, H, dtype=f32)
        self.dw3 = z(E, M, H, dtype=f32) if act == "swiglu" else None
        self.dw2 = z(E, H, M, dtype=f32)
        self.db1 = z(E, H, dtype=f32) if expert_bias else None
        self.db3 = z(E, H, dtype=f32) if expert_bias and sw else None
        self.db2 = z(E, M, dtype=f32) if expert_bias else None
        # the attention part of AT_r
        if mha is not None:
            hd = mha["head_dim"]
            heads = M // hd
            self.mha = L.make_mha_shape(mha["seq_len"], heads, hd, mha.get("causal", True))
            self.mha_in = z(T_total, M)
            self.w_qkv = z(M, 3 * M)
            self.w_o = z(M, M)
            self.qkv = z(T_total, 3 * M)
            self.attn = z(T_total, M)
            self.lse = z(R, heads, T, dtype=f32)
            self.d_attn = z(T_total, M)
            self.d_qkv = z(T_total, 3 * M)
            self.delta = z(R, heads, T, dtype=f32)
            self.d_in = z(T_total, M)
            self.dw_qkv = z(M, 3 * M, dtype=f32)
            self.dw_o = z(M, M, dtype=f32)
        else:
            self.mha = None
            for n in ("mha_in", "w_qkv", "w_o", "qkv", "attn", "lse", "d_attn", "d_qkv", "delta",
                      "d_in", "dw_qkv", "dw_o"):
                setattr(self, n, None)
        self.ws_bytes = L.flowmoe_workspace_bytes(
            self.shape, L.WS_LAYER_BWD_MHA if mha is not None else L.WS_LAYER_BWD)
        self.ws = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)

    @property
    def C(self) -> int:
        return self.shape.C

    def bufs(self) -> L.LayerBufs:
        names = [n for n, _ in L.LayerBufs._fields_ if n != "ws_bytes"]
        return L.layer_bufs(ws_bytes=self.ws_bytes, **{n: getattr(self, n) for n in names})

    def forward(self, s_compute=None, s_comm=None, trace=None, bufs=None) -> None:
        L.flowmoe_layer_fwd(self.shape, self.R, bufs or self.bufs(), s_compute, s_comm, trace)

    def backward(self, s_compute=None, s_comm=None, trace=None, bufs=None) -> None:
        L.flowmoe_layer_bwd(self.shape, self.R, bufs or self.bufs(), s_compute, s_comm, trace)
