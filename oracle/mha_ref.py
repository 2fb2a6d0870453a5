"""fp64 reference of the attention part of AT_r (test infrastructure only).

Sec. 2.1: a transformer block's MHA layer maps its input I (B x N x M, here
flattened to T = B*N rows of width M) with the Query, Key and Value matrices
W^Q, W^K, W^V (M x M) to attention data per token, and a linear map W^O
(M x M) gives its output I', which the gate and the experts consume.
Sec. 3.2 chunks the block's input into R equal parts, each an independent
subtask AT_r (MHA plus gating); a chunk therefore holds whole sequences.

Readings of what the paper leaves open (each listed in the design notes):
  * heads: the M columns split into `heads` heads of width d = M / heads,
    scaled dot-product attention per head with scale 1/sqrt(d), heads
    concatenated in column order before W^O;
  * the four matrices carry no biases and the block has no normalisation or
    residual inside AT_r (the parameter count 4 M^2 + M E of Sec. 4.2 counts
    only the four matrices and the gate);
  * the three input projections are stored side by side as one M x 3M
    matrix [W^Q | W^K | W^V], and their gradient likewise;
  * `causal`: token i attends to tokens j <= i of its own sequence (GPT-style
    models of Table 3); otherwise to every token of its sequence (BERT-style).

Every function is the definition written out with numpy matmuls per
(sequence, head); nothing is blocked, fused or reordered.
"""
from __future__ import annotations

import numpy as np


def _masked_scores(q, k, causal):
    """s_ij = q_i . k_j / sqrt(d), -inf where causal and j > i."""
    d = q.shape[1]
    s = (q @ k.T) / np.sqrt(d)
    if causal:
        n = s.shape[0]
        s = np.where(np.tril(np.ones((n, n), dtype=bool)), s, -np.inf)
    return s


def _softmax_rows(s):
    """Row softmax and the natural-log logsumexp of each row."""
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=1, keepdims=True)
    return e / z, (m + np.log(z))[:, 0]


def attention(qkv, seq_len, heads, causal):
    """The attention core per sequence and head: A_h = softmax(S) V_h with
    s_ij = q_i . k_j / sqrt(d) over the visible tokens. qkv: T x 3M = [Q|K|V].
    Returns attn (T x M, heads side by side) and lse (heads x T)."""
    T, M3 = qkv.shape
    M = M3 // 3
    if T % seq_len or M % heads:
        raise ValueError("T must hold whole sequences and M whole heads")
    d = M // heads
    attn = np.zeros((T, M))
    lse = np.zeros((heads, T))
    for b in range(T // seq_len):
        rows = slice(b * seq_len, (b + 1) * seq_len)
        for h in range(heads):
            cq = slice(h * d, (h + 1) * d)
            ck = slice(M + h * d, M + (h + 1) * d)
            cv = slice(2 * M + h * d, 2 * M + (h + 1) * d)
            p, l = _softmax_rows(_masked_scores(qkv[rows, cq], qkv[rows, ck], causal))
            attn[rows, cq] = p @ qkv[rows, cv]
            lse[h, rows] = l
    return attn, lse


def attention_bwd(qkv, d_attn, seq_len, heads, causal):
    """Gradient of attention() by the chain rule, per sequence and head, with
    P the softmax weights: dV = P^T dA, dP = dA V^T, dS = P * (dP -
    rowsum(P * dP)) (the softmax Jacobian), dQ = dS K / sqrt(d),
    dK = dS^T Q / sqrt(d). Returns d_qkv (T x 3M)."""
    T, M3 = qkv.shape
    M = M3 // 3
    d = M // heads
    d_qkv = np.zeros((T, 3 * M))
    for b in range(T // seq_len):
        rows = slice(b * seq_len, (b + 1) * seq_len)
        for h in range(heads):
            cq = slice(h * d, (h + 1) * d)
            ck = slice(M + h * d, M + (h + 1) * d)
            cv = slice(2 * M + h * d, 2 * M + (h + 1) * d)
            q, k, v = qkv[rows, cq], qkv[rows, ck], qkv[rows, cv]
            p, _ = _softmax_rows(_masked_scores(q, k, causal))
            da = d_attn[rows, cq]
            dp = da @ v.T
            ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
            d_qkv[rows, cq] = ds @ k / np.sqrt(d)
            d_qkv[rows, ck] = ds.T @ q / np.sqrt(d)
            d_qkv[rows, cv] = p.T @ da
    return d_qkv


def mha_fwd(inp, w_qkv, w_o, seq_len, heads, causal):
    """Forward of one chunk's MHA (Sec. 2.1).

    inp: T x M (T a multiple of seq_len: T / seq_len whole sequences),
    w_qkv: M x 3M = [W^Q | W^K | W^V], w_o: M x M.
    Returns qkv (T x 3M = [Q | K | V]), attn (T x M, the heads' outputs
    concatenated, before W^O), lse (heads x T, log of each softmax
    denominator with the row's scores), out = attn W^O (T x M)."""
    qkv = inp @ w_qkv
    attn, lse = attention(qkv, seq_len, heads, causal)
    return dict(qkv=qkv, attn=attn, lse=lse, out=attn @ w_o)


def mha_bwd(inp, w_qkv, w_o, saved, d_out, seq_len, heads, causal):
    """Backward of mha_fwd by the chain rule: d_attn = d_out W^O^T,
    dW^O = attn^T d_out, the attention core's gradient d_qkv, then
    d_inp = d_qkv [W^Q | W^K | W^V]^T and dW_qkv = inp^T d_qkv.
    Returns d_attn, d_qkv, d_in, dw_qkv, dw_o."""
    d_attn = d_out @ w_o.T
    d_qkv = attention_bwd(saved["qkv"], d_attn, seq_len, heads, causal)
    return dict(d_attn=d_attn, d_qkv=d_qkv, d_in=d_qkv @ w_qkv.T, dw_qkv=inp.T @ d_qkv,
                dw_o=saved["attn"].T @ d_out)
