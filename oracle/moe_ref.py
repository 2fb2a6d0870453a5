"""fp64 reference of the MoE layer, step by step (test infrastructure only).

Notation follows Sec. 2.1 and the notation table of the appendix: T = B*N
tokens of width M, E experts with hidden width H, top-k gating, capacity
C = f*k*B*N/E, pipelining degree R (Sec. 3.2). Row-major arrays, float64.

Readings of points the paper leaves open (each one is listed in the design
notes with its reason):
  * gate = linear M x E map (Sec. 4.2), plus an optional constant bias b;
  * top-k selection by descending logit, ties to the lower expert index, with
    IEEE comparison (-0.0 == +0.0); selected weights are the softmax over the
    k selected logits (= full softmax renormalised over the selection), or,
    in the Switch-style variant (gate="full"), the selected experts' own
    probabilities under the softmax over all E logits, not renormalised;
  * C = ceil(f*k*T_r/E) in exact arithmetic on the decimal value of f, per
    chunk of T_r = T/R tokens (gating belongs to each chunk's subtask AT_r);
  * capacity priority: every first choice before any second choice, and
    ascending token order within a rank; weights are renormalised before the
    drop, so a token's kept weights may sum to less than one;
  * experts have no biases unless given (b1, b3 added to the first layer's
    pre-activations, b2 to the second layer's output, the biased two-layer
    experts that the parameter counts of Table 3 imply); GELU is the exact
    erf form, SwiGLU is silu(x W1 + b1) * (x W3 + b3) followed by W2;
  * routing is piecewise constant: selection and dropping carry no gradient.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
from scipy.special import erf, expit

PACKED, PADDED = "packed", "padded"


# ---------------------------------------------------------------------------
# capacity (Sec. 2.1)
# ---------------------------------------------------------------------------
def capacity(T_r: int, E: int, k: int, f: float) -> int:
    """C = ceil(f * k * T_r / E), with f taken as the decimal it is written as."""
    v = Fraction(repr(float(f))) * k * T_r / E
    return int(-((-v.numerator) // v.denominator))


def rows_capacity(T_r: int, E: int, k: int, C: int, layout: str) -> int:
    """Rows of the dispatched tensor: E*C for the padded E x C x M layout of
    Sec. 2.1, else the most rows that can be kept, min(T_r*k, E*C)."""
    return E * C if layout == PADDED else min(T_r * k, E * C)


# ---------------------------------------------------------------------------
# forward steps
# ---------------------------------------------------------------------------
def gate_logits(x, w_gate, bias=None):
    """Step 1: logits l = x W_g (+ b), a T x E matrix (linear gate, Sec. 4.2)."""
    l = x @ w_gate
    if bias is not None:
        l = l + np.asarray(bias, dtype=np.float64)[None, :]
    return l


def topk_select(logits, k, gate="renorm"):
    """Steps 2-3: per token, the k experts with the largest logits (ties go to
    the lower expert index) in descending order, and their gate weights:
    gate="renorm": w_j = exp(l_j - l_0) / sum_j' exp(l_j' - l_0), the softmax
    of Sec. 2.1 renormalised over the selected experts;
    gate="full": w_j = exp(l_j - l_0) / sum_e exp(l_e - l_0), the selected
    experts' probabilities under the softmax over all E logits (l_0 is the
    largest logit, so both are shifted by the row maximum)."""
    if gate not in ("renorm", "full"):
        raise ValueError(gate)
    T, E = logits.shape
    idx = np.zeros((T, k), dtype=np.int64)
    w = np.zeros((T, k), dtype=np.float64)
    for t in range(T):
        row = logits[t]
        order = sorted(range(E), key=lambda e: (-row[e], e))[:k]
        idx[t] = order
        sel = np.array([row[e] for e in order])
        ex = np.exp(sel - sel[0])
        den = ex.sum() if gate == "renorm" else np.exp(row - sel[0]).sum()
        w[t] = ex / den
    return idx, w


def route(topk_idx, E, C, layout=PACKED):
    """Steps 4-5: capacity-bounded positions and the dispatch permutation.

    Assignments (t, j) are taken in the order j = 0..k-1, then t = 0..T-1; an
    assignment's position is how many earlier assignments chose the same
    expert. It is kept iff position < C. Returns pos, kept, counts (E),
    offsets (E+1: packed prefix sums of counts, or e*C for the padded
    layout), slot (T x k, row or -1) and row_src (rows, t*k+j or -1)."""
    T, k = topk_idx.shape
    fill = [0] * E
    pos = np.zeros((T, k), dtype=np.int64)
    for j in range(k):
        for t in range(T):
            e = int(topk_idx[t, j])
            pos[t, j] = fill[e]
            fill[e] += 1
    kept = pos < C
    counts = np.array([min(c, C) for c in fill], dtype=np.int64)
    offsets = np.zeros(E + 1, dtype=np.int64)
    if layout == PADDED:
        offsets[:] = np.arange(E + 1) * C
    else:
        offsets[1:] = np.cumsum(counts)
    rows = rows_capacity(T, E, k, C, layout)
    slot = np.full((T, k), -1, dtype=np.int64)
    row_src = np.full(rows, -1, dtype=np.int64)
    for t in range(T):
        for j in range(k):
            if kept[t, j]:
                r = offsets[topk_idx[t, j]] + pos[t, j]
                slot[t, j] = r
                row_src[r] = t * k + j
    demand = np.array(fill, dtype=np.int64)
    return dict(pos=pos, kept=kept, counts=counts, offsets=offsets, slot=slot,
                row_src=row_src, demand=demand, rows=rows)


def dispatch(x, row_src, k):
    """Step 6: the dispatched tensor (the all-to-all send layout G(I') of
    Sec. 2.1): row r holds token row_src[r] // k, or zeros for an empty row."""
    out = np.zeros((row_src.shape[0], x.shape[1]), dtype=np.float64)
    for r, s in enumerate(row_src):
        if s >= 0:
            out[r] = x[s // k]
    return out


def gelu(z):
    """gelu(z) = z * Phi(z), Phi the standard normal CDF (exact erf form)."""
    return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))


def gelu_grad(z):
    """d gelu / dz = Phi(z) + z * phi(z)."""
    return 0.5 * (1.0 + erf(z / np.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / np.sqrt(2.0 * np.pi)


def silu(z):
    return z * expit(z)


def silu_grad(z):
    s = expit(z)
    return s * (1.0 + z * (1.0 - s))


def expert_ffn(x_disp, counts, offsets, w1, w3, w2, act, b1=None, b3=None, b2=None):
    """Step 7: each expert's two-layer FFN (Sec. 2.1: M x H then H x M) over
    its rows [offsets[e], offsets[e] + counts[e]), with optional biases
    (b1, b3: E x H on the first layer, b2: E x M on the second). Returns the
    pre-activations h1 (and h3 for SwiGLU), the activation a that feeds W2,
    and y_disp. Rows outside every expert's range stay zero."""
    rows, M = x_disp.shape
    H = w1.shape[2]
    h1 = np.zeros((rows, H))
    h3 = np.zeros((rows, H)) if act == "swiglu" else None
    a = np.zeros((rows, H))
    y = np.zeros((rows, M))
    for e in range(w1.shape[0]):
        lo, hi = int(offsets[e]), int(offsets[e]) + int(counts[e])
        if hi == lo:
            continue
        X = x_disp[lo:hi]
        h1[lo:hi] = X @ w1[e]
        if b1 is not None:
            h1[lo:hi] += b1[e]
        if act == "gelu":
            a[lo:hi] = gelu(h1[lo:hi])
        else:
            h3[lo:hi] = X @ w3[e]
            if b3 is not None:
                h3[lo:hi] += b3[e]
            a[lo:hi] = silu(h1[lo:hi]) * h3[lo:hi]
        y[lo:hi] = a[lo:hi] @ w2[e]
        if b2 is not None:
            y[lo:hi] += b2[e]
    return dict(h1=h1, h3=h3, a=a, y_disp=y)


def combine(y_disp, slot, w):
    """Step 8: y_t = sum over kept assignments of w_tj * y_disp[slot_tj]."""
    T, k = slot.shape
    y = np.zeros((T, y_disp.shape[1]))
    for t in range(T):
        for j in range(k):
            if slot[t, j] >= 0:
                y[t] += w[t, j] * y_disp[slot[t, j]]
    return y


# ---------------------------------------------------------------------------
# backward steps (reverse of the forward, Eqs. 5-6 order per chunk)
# ---------------------------------------------------------------------------
def combine_bwd(dy, y_disp, slot, w):
    """Step 9: dy_disp[slot] = w * dy_t and dw_tj = <dy_t, y_disp[slot]>;
    a dropped assignment has dw = 0 and no row."""
    T, k = slot.shape
    dy_disp = np.zeros_like(y_disp)
    dw = np.zeros((T, k))
    for t in range(T):
        for j in range(k):
            r = slot[t, j]
            if r >= 0:
                dy_disp[r] = w[t, j] * dy[t]
                dw[t, j] = float(dy[t] @ y_disp[r])
    return dy_disp, dw


def expert_ffn_bwd(dy_disp, x_disp, saved, counts, offsets, w1, w3, w2, act, return_dh=False):
    """Step 10: per expert, dA = dY W2^T, dW2 = A^T dY, then through the
    activation, dW1 = X^T dH1 (dW3 = X^T dH3) and dX = dH1 W1^T (+ dH3 W3^T).
    With return_dh, also the hidden-layer gradient per row: dH1 (GELU) or
    [dH1 | dH3] (SwiGLU), zero outside the experts' rows."""
    E, M, H = w1.shape
    dh = np.zeros((x_disp.shape[0], H if act == "gelu" else 2 * H))
    dx_disp = np.zeros_like(x_disp)
    dw1 = np.zeros_like(w1)
    dw3 = np.zeros_like(w1) if act == "swiglu" else None
    dw2 = np.zeros_like(w2)
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e]) + int(counts[e])
        if hi == lo:
            continue
        X, dY = x_disp[lo:hi], dy_disp[lo:hi]
        A, h1 = saved["a"][lo:hi], saved["h1"][lo:hi]
        dA = dY @ w2[e].T
        dw2[e] = A.T @ dY
        if act == "gelu":
            dH1 = dA * gelu_grad(h1)
            dw1[e] = X.T @ dH1
            dx_disp[lo:hi] = dH1 @ w1[e].T
            dh[lo:hi] = dH1
        else:
            h3 = saved["h3"][lo:hi]
            dH1 = dA * h3 * silu_grad(h1)
            dH3 = dA * silu(h1)
            dw1[e] = X.T @ dH1
            dw3[e] = X.T @ dH3
            dx_disp[lo:hi] = dH1 @ w1[e].T + dH3 @ w3[e].T
            dh[lo:hi, :H] = dH1
            dh[lo:hi, H:] = dH3
    if return_dh:
        return dx_disp, dw1, dw3, dw2, dh
    return dx_disp, dw1, dw3, dw2


def expert_bias_grads(dy_disp, dh, counts, offsets, act):
    """Step 10's bias part: each bias gradient is the sum over the expert's
    rows of the gradient of the pre-activation it is added to: db2_e = sum
    of dY rows, db1_e = sum of dH1 rows (db3_e = sum of dH3 rows), with dH
    as expert_ffn_bwd(..., return_dh=True) gives it."""
    E = counts.shape[0]
    M = dy_disp.shape[1]
    H = dh.shape[1] if act == "gelu" else dh.shape[1] // 2
    db1, db2 = np.zeros((E, H)), np.zeros((E, M))
    db3 = np.zeros((E, H)) if act == "swiglu" else None
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e]) + int(counts[e])
        db2[e] = dy_disp[lo:hi].sum(axis=0)
        db1[e] = dh[lo:hi, :H].sum(axis=0)
        if act == "swiglu":
            db3[e] = dh[lo:hi, H:].sum(axis=0)
    return db1, db3, db2


def dispatch_bwd(dx_disp, slot):
    """Step 11: dx_t = sum over kept assignments of dx_disp[slot_tj]."""
    T, k = slot.shape
    dx = np.zeros((T, dx_disp.shape[1]))
    for t in range(T):
        for j in range(k):
            if slot[t, j] >= 0:
                dx[t] += dx_disp[slot[t, j]]
    return dx


def gate_bwd(x, w_gate, topk_idx, w, dw, logits=None, gate="renorm"):
    """Steps 12-13: the Jacobian of the gate weights, with s = sum_j w_j dw_j.
    gate="renorm" (softmax over the selection): dl_{t,S_j} = w_j (dw_j - s),
    zero off the selection. gate="full" (w_j = p_{S_j}, p the softmax over
    all E logits, which ``logits`` gives): dl_{t,e} = p_e (dw_j - s) for
    e = S_j and -p_e s for every other expert. Then dW_g = x^T dl,
    db = sum_t dl_t and the gate's share of dx, dl W_g^T."""
    T, k = topk_idx.shape
    E = w_gate.shape[1]
    dl = np.zeros((T, E))
    for t in range(T):
        s = float(w[t] @ dw[t])
        if gate == "full":
            row = logits[t]
            p = np.exp(row - row.max())
            p /= p.sum()
            dl[t] = -p * s
        elif gate != "renorm":
            raise ValueError(gate)
        for j in range(k):
            dl[t, topk_idx[t, j]] = w[t, j] * (dw[t, j] - s)
    return dict(d_logits=dl, dw_gate=x.T @ dl, dbias=dl.sum(axis=0), dx_gate=dl @ w_gate.T)


# ---------------------------------------------------------------------------
# one chunk, and the chunked layer (Sec. 3.2 partition; App. H accumulation)
# ---------------------------------------------------------------------------
def layer_chunk(x, w_gate, bias, w1, w3, w2, dy, k, C, act, layout=PACKED,
                logits_for_routing=None, gate="renorm", b1=None, b3=None, b2=None):
    """Forward and backward of one chunk. ``logits_for_routing`` (the GPU's
    fp32 logits widened to fp64) replaces the oracle's own logits for
    selection and gate weights, so that floating-point parity is measured
    on the same routing. b1, b3, b2: the experts' biases (or None)."""
    E = w_gate.shape[1]
    logits = gate_logits(x, w_gate, bias)
    lr = logits if logits_for_routing is None else logits_for_routing
    idx, w = topk_select(lr, k, gate)
    rt = route(idx, E, C, layout)
    x_disp = dispatch(x, rt["row_src"], k)
    sv = expert_ffn(x_disp, rt["counts"], rt["offsets"], w1, w3, w2, act, b1, b3, b2)
    y = combine(sv["y_disp"], rt["slot"], w)
    out = dict(logits=logits, topk_idx=idx, topk_w=w, x_disp=x_disp, y=y, **rt, **sv)
    if dy is None:
        return out
    dy_disp, dw = combine_bwd(dy, sv["y_disp"], rt["slot"], w)
    dx_disp, dw1, dw3, dw2, dh = expert_ffn_bwd(dy_disp, x_disp, sv, rt["counts"], rt["offsets"],
                                                w1, w3, w2, act, return_dh=True)
    dx = dispatch_bwd(dx_disp, rt["slot"])
    g = gate_bwd(x, w_gate, idx, w, dw, lr, gate)
    out.update(dy_disp=dy_disp, d_topk_w=dw, dx_disp=dx_disp, dh=dh, dw1=dw1, dw3=dw3, dw2=dw2,
               d_logits=g["d_logits"], dw_gate=g["dw_gate"], dbias=g["dbias"],
               dx=dx + g["dx_gate"], dx_experts=dx)
    if b1 is not None or b3 is not None or b2 is not None:
        db1, db3, db2 = expert_bias_grads(dy_disp, dh, rt["counts"], rt["offsets"], act)
        out.update(db1=db1, db3=db3, db2=db2)
    return out


def layer_fwd_bwd(inp, k, f, act, R=1, layout=PACKED, logits_for_routing=None,
                  C=None, gate="renorm", mha=None):
    """The layer over T tokens split into R equal contiguous chunks, each an
    independent layer call with its own capacity; per-token outputs are
    concatenated and weight gradients summed over chunks. ``inp`` holds
    float64 arrays x, w_gate, bias (or None), w1, w3 (or None), w2, dy, and
    optionally the experts' biases b1, b3, b2.
    ``mha`` (dict seq_len, heads, causal): AT_r is the chunk's multi-head
    attention followed by the gate (Sec. 3.2); the MoE part's input x is
    then the attention output I' of inp["mha_in"] under inp["w_qkv"] and
    inp["w_o"], and the backward carries dx on through the attention to
    d_in, dw_qkv and dw_o (summed over chunks)."""
    if mha is not None:
        from .mha_ref import mha_fwd
        T = inp["mha_in"].shape[0]
        if T % R:
            raise ValueError("T must be a multiple of R")
        Tr = T // R
        fw = [mha_fwd(inp["mha_in"][r * Tr:(r + 1) * Tr], inp["w_qkv"], inp["w_o"],
                      mha["seq_len"], mha["heads"], mha["causal"]) for r in range(R)]
        inp = dict(inp, x=np.concatenate([m["out"] for m in fw], axis=0))
    x = inp["x"]
    T = x.shape[0]
    if T % R:
        raise ValueError("T must be a multiple of R")
    Tr = T // R
    E = inp["w_gate"].shape[1]
    if C is None:
        C = capacity(Tr, E, k, f)
    chunks = []
    for r in range(R):
        sl = slice(r * Tr, (r + 1) * Tr)
        lr = None if logits_for_routing is None else logits_for_routing[sl]
        dy = None if inp.get("dy") is None else inp["dy"][sl]
        chunks.append(layer_chunk(x[sl], inp["w_gate"], inp.get("bias"), inp["w1"],
                                  inp.get("w3"), inp["w2"], dy, k, C, act, layout, lr, gate,
                                  inp.get("b1"), inp.get("b3"), inp.get("b2")))
    res = dict(C=C, chunks=chunks)
    for key in ("logits", "topk_idx", "topk_w", "y", "dx", "d_topk_w", "d_logits"):
        if key in chunks[0]:
            res[key] = np.concatenate([c[key] for c in chunks], axis=0)
    for key in ("dw1", "dw3", "dw2", "dw_gate", "dbias", "db1", "db3", "db2"):
        if key in chunks[0] and chunks[0][key] is not None:
            res[key] = sum(c[key] for c in chunks)
    if mha is not None:
        from .mha_ref import mha_bwd
        res["x"] = x
        for key in ("qkv", "attn"):
            res[key] = np.concatenate([m[key] for m in fw], axis=0)
        res["lse"] = np.stack([m["lse"] for m in fw])  # R x heads x T_r
        if "dx" in res:
            bw = [mha_bwd(inp["mha_in"][r * Tr:(r + 1) * Tr], inp["w_qkv"], inp["w_o"], fw[r],
                          chunks[r]["dx"], mha["seq_len"], mha["heads"], mha["causal"])
                  for r in range(R)]
            for key in ("d_attn", "d_qkv", "d_in"):
                res[key] = np.concatenate([b[key] for b in bw], axis=0)
            res["dw_qkv"] = sum(b["dw_qkv"] for b in bw)
            res["dw_o"] = sum(b["dw_o"] for b in bw)
    return res
