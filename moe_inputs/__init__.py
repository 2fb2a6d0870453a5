"""Seeded synthetic inputs for one MoE layer (forward + backward).

This module is shared by the fp64 oracle, the tests and the benchmark. It holds
workload descriptions and random-number recipes only: none of the layer's
arithmetic (gating, capacity, routing, experts, combine) lives here.

Workloads (shapes of the MoE layer of Section 2.1: T = B*N tokens of width M,
E experts of hidden size H, top-k routing, capacity factor f, pipelining
degree R of Section 3.2):

  tiny      fp32  T=256   M=64   H=128   E=4  k=2 f=1.25 GELU
  balanced  bf16  T=4096  M=1024 H=4096  E=8  k=2 f=1.2  GELU
  skewed    bf16  T=8192  M=1024 H=4096  E=16 k=1 f=1.0  GELU, Zipf gate bias
  large     bf16  T=16384 M=4096 H=14336 E=8  k=2 f=1.25 SwiGLU
  fine      bf16  T=16384 M=2048 H=1408  E=64 k=6 f=1.5  SwiGLU, R=4

Recipe (all tensors row-major):
  * every tensor has its own PCG64 stream, seeded by
    SeedSequence(entropy=seed, spawn_key=(tensor_id, block)), so tensors can be
    drawn block-parallel and a block's values do not depend on the thread count;
  * draws are standard normals in float32, scaled in float32, then rounded to
    the storage dtype (bf16 by round-to-nearest-even on the fp32 bits);
  * x ~ N(0,1) (T x M); W_g ~ N(0, 0.02^2) (M x E); W1, W3 ~ N(0, 0.02^2)
    (E x M x H); W2 ~ N(0, 0.02^2) (E x H x M); dy ~ N(0,1) (T x M);
  * the skewed workload adds a constant per-expert gate bias
    b_e = -1.2 * ln(rho_e), rho a seeded permutation of 1..E (log of a Zipf
    pmf with s = 1.2, up to a shift), so expert loads are heavy-tailed;
  * biased experts (expert_bias=True) add b1, b3 ~ N(0, 0.02^2) (E x H) and
    b2 ~ N(0, 0.02^2) (E x M) in float32;
  * with the block's attention in AT_r (mha=True): the block input
    mha_in ~ N(0,1) (T x M) in place of x as the layer's input, and
    w_qkv ~ N(0, 0.02^2) (M x 3M, [W^Q | W^K | W^V]), w_o ~ N(0, 0.02^2)
    (M x M); T/seq_len sequences of seq_len tokens, heads of width head_dim:
      tiny 4 x 64, d 64 causal; balanced 8 x 512, d 64 bidirectional
      (BERT-like); skewed 16 x 512, d 64 causal; large 4 x 4096, d 128 causal;
      fine 4 x 4096 (one sequence per chunk), d 128 causal.

bf16 tensors are held as numpy uint16 bit patterns; ``as_f64`` widens any
stored tensor exactly to float64.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

__all__ = [
    "MoEConfig", "CONFIGS", "get_config", "make_inputs", "as_f64",
    "bf16_round_bits", "bf16_bits_to_f32", "to_torch", "make_attention_inputs",
]

WEIGHT_STD = 0.02
ZIPF_S = 1.2

# tensor ids for the per-tensor streams
_TID = {"x": 0, "w_gate": 1, "bias": 2, "w1": 3, "w3": 4, "w2": 5, "dy": 6, "b1": 7, "b3": 8,
        "b2": 9, "mha_in": 10, "w_qkv": 11, "w_o": 12, "qkv": 13, "d_attn": 14}
_BLOCK = 1 << 22  # elements per independently seeded block


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    name: str
    T: int          # tokens (B*N)
    M: int          # model (embedding) width
    H: int          # expert hidden width
    E: int          # experts
    k: int          # experts per token
    f: float        # capacity factor
    act: str        # "gelu" | "swiglu"
    dtype: str      # "f32" | "bf16"
    R: int = 1      # token chunks (pipelining degree)
    zipf_bias: bool = False
    seed: int = 0
    gate: str = "renorm"  # gate weights: "renorm" (softmax over the selection) | "full"
    expert_bias: bool = False  # biased experts: b1, b3 (E x H), b2 (E x M), fp32
    mha: bool = False     # AT_r includes the block's multi-head attention
    seq_len: int = 0      # tokens per sequence (N of Sec. 2.1)
    head_dim: int = 0     # width d of an attention head (heads = M / d)
    causal: bool = True   # token i attends to tokens j <= i of its sequence

    def replace(self, **kw) -> "MoEConfig":
        return dataclasses.replace(self, **kw)

    @property
    def T_chunk(self) -> int:
        return self.T // self.R

    @property
    def heads(self) -> int:
        return self.M // self.head_dim if self.head_dim else 0


CONFIGS = {
    "tiny": MoEConfig("tiny", 256, 64, 128, 4, 2, 1.25, "gelu", "f32", seed=0,
                      seq_len=64, head_dim=64),
    "balanced": MoEConfig("balanced", 4096, 1024, 4096, 8, 2, 1.2, "gelu", "bf16", seed=1,
                          seq_len=512, head_dim=64, causal=False),
    "skewed": MoEConfig("skewed", 8192, 1024, 4096, 16, 1, 1.0, "gelu", "bf16",
                        zipf_bias=True, seed=2, seq_len=512, head_dim=64),
    "large": MoEConfig("large", 16384, 4096, 14336, 8, 2, 1.25, "swiglu", "bf16", seed=3,
                       seq_len=4096, head_dim=128),
    "fine": MoEConfig("fine", 16384, 2048, 1408, 64, 6, 1.5, "swiglu", "bf16", R=4, seed=4,
                      seq_len=4096, head_dim=128),
}


def get_config(name: str, **overrides) -> MoEConfig:
    cfg = CONFIGS[name]
    return cfg.replace(**overrides) if overrides else cfg


# ----------------------------------------------------------------------------
# bf16 bit helpers (storage format only)
# ----------------------------------------------------------------------------
def bf16_round_bits(a32: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern (uint16), round to nearest, ties to even.
    Inputs are finite (no NaN handling)."""
    u = np.ascontiguousarray(a32, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_f64(a: np.ndarray) -> np.ndarray:
    """Widen a stored tensor (float32, or uint16 bf16 bits) exactly to float64."""
    if a.dtype == np.uint16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------
# generation
# ----------------------------------------------------------------------------
def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normal(seed: int, tid: int, n: int, scale: float, dtype: str) -> np.ndarray:
    """n scaled standard normals, stored in ``dtype`` ('f32' or 'bf16')."""
    out = np.empty(n, dtype=np.float32 if dtype == "f32" else np.uint16)
    nblk = (n + _BLOCK - 1) // _BLOCK

    def fill(b: int) -> None:
        lo, hi = b * _BLOCK, min(n, (b + 1) * _BLOCK)
        ss = np.random.SeedSequence(entropy=seed, spawn_key=(tid, b))
        g = np.random.Generator(np.random.PCG64(ss))
        v = g.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            v *= np.float32(scale)
        out[lo:hi] = v if dtype == "f32" else bf16_round_bits(v)

    if nblk <= 1:
        for b in range(nblk):
            fill(b)
    else:
        with _cf.ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def _zipf_bias(seed: int, E: int) -> np.ndarray:
    ss = np.random.SeedSequence(entropy=seed, spawn_key=(_TID["bias"], 0))
    g = np.random.Generator(np.random.PCG64(ss))
    rho = g.permutation(np.arange(1, E + 1, dtype=np.float64))
    return (-ZIPF_S * np.log(rho)).astype(np.float32)


def make_inputs(cfg: MoEConfig, *, with_dy: bool = True, x_zero_rows=None) -> dict:
    """All layer inputs for ``cfg`` in storage form.

    Returns a dict with x (T,M), w_gate (M,E), bias (E,) float32 or None,
    w1 (E,M,H), w3 (E,M,H) or None, w2 (E,H,M), dy (T,M), and the experts'
    biases b1 (E,H), b3 (E,H), b2 (E,M) float32 (None unless
    cfg.expert_bias; b3 only for SwiGLU), and with cfg.mha the block input
    mha_in (T,M) and the attention weights w_qkv (M,3M), w_o (M,M).
    Storage arrays are float32 for
    dtype 'f32' and uint16 bf16 bits for 'bf16'.
    ``x_zero_rows`` (iterable of token indices) zeroes those rows of x, which
    makes their gate logits all tie (edge-case inputs).
    """
    T, M, H, E = cfg.T, cfg.M, cfg.H, cfg.E
    s, dt = cfg.seed, cfg.dtype
    out = {}
    out["x"] = _normal(s, _TID["x"], T * M, 1.0, dt).reshape(T, M)
    if x_zero_rows is not None:
        for t in x_zero_rows:
            out["x"][t, :] = 0
    out["w_gate"] = _normal(s, _TID["w_gate"], M * E, WEIGHT_STD, dt).reshape(M, E)
    out["bias"] = _zipf_bias(s, E) if cfg.zipf_bias else None
    out["w1"] = _normal(s, _TID["w1"], E * M * H, WEIGHT_STD, dt).reshape(E, M, H)
    out["w3"] = (_normal(s, _TID["w3"], E * M * H, WEIGHT_STD, dt).reshape(E, M, H)
                 if cfg.act == "swiglu" else None)
    out["w2"] = _normal(s, _TID["w2"], E * H * M, WEIGHT_STD, dt).reshape(E, H, M)
    out["dy"] = _normal(s, _TID["dy"], T * M, 1.0, dt).reshape(T, M) if with_dy else None
    if cfg.mha:
        out["mha_in"] = _normal(s, _TID["mha_in"], T * M, 1.0, dt).reshape(T, M)
        out["w_qkv"] = _normal(s, _TID["w_qkv"], M * 3 * M, WEIGHT_STD, dt).reshape(M, 3 * M)
        out["w_o"] = _normal(s, _TID["w_o"], M * M, WEIGHT_STD, dt).reshape(M, M)
    if cfg.expert_bias:  # fp32 like the gate bias
        out["b1"] = _normal(s, _TID["b1"], E * H, WEIGHT_STD, "f32").reshape(E, H)
        out["b3"] = (_normal(s, _TID["b3"], E * H, WEIGHT_STD, "f32").reshape(E, H)
                     if cfg.act == "swiglu" else None)
        out["b2"] = _normal(s, _TID["b2"], E * M, WEIGHT_STD, "f32").reshape(E, M)
    else:
        out["b1"] = out["b3"] = out["b2"] = None
    return out


def make_attention_inputs(seed: int, T: int, M: int) -> dict:
    """Inputs of the attention core alone: qkv ~ N(0,1) (T x 3M, [Q | K | V])
    and the gradient d_attn ~ N(0,1) (T x M), both bf16 bit patterns."""
    return dict(qkv=_normal(seed, _TID["qkv"], T * 3 * M, 1.0, "bf16").reshape(T, 3 * M),
                d_attn=_normal(seed, _TID["d_attn"], T * M, 1.0, "bf16").reshape(T, M))


def to_torch(a: np.ndarray, device=None):
    """Storage array -> torch tensor (bf16 bits become torch.bfloat16)."""
    import torch
    if a is None:
        return None
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device) if device is not None else t
