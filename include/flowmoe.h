/*
 * flowmoe.h -- C ABI of the MoE-layer hot path (FlowMoE, arXiv 2510.00207).
 *
 * One MoE layer (Sec. 2.1): a linear gate with top-k softmax selection, the
 * capacity-bounded dispatch into the expert-major all-to-all send layout
 * G(I') (E x C x M, or its packed form), one two-layer FFN per expert, and the
 * weighted combine back to T x M; plus the backward of each step, and the
 * R-chunk two-stream schedule of Sec. 3.2 (Eqs. 3-6).
 *
 * Conventions for every call
 *  - All tensor pointers are DEVICE pointers owned by the caller, row-major
 *    and contiguous. The library never allocates or frees device memory and
 *    never synchronises the device: work is enqueued on the stream(s) given.
 *  - Tensors of the layer dtype (x, W_g, W1, W3, W2, the row buffers, y, dy,
 *    dx) must be 16-byte aligned (FLOWMOE_ERR_INVALID otherwise): kernels
 *    move them in 16-byte vectors.
 *  - "layer dtype" tensors are float (FLOWMOE_F32) or bf16 bit patterns
 *    (FLOWMOE_BF16, passed as uint16_t). Gate logits, gate weights, their
 *    gradients and all weight gradients are always float. Accumulation is
 *    always in float; bf16 results are rounded to nearest-even.
 *  - Arguments are validated on the host before anything is enqueued; on a
 *    non-OK status nothing was enqueued and flowmoe_last_error() (per host
 *    thread) describes the problem. Launch failures return FLOWMOE_ERR_HIP.
 *    Faults inside kernels surface at the caller's next synchronisation.
 *  - Inputs must be finite; NaN/Inf inputs give unspecified results.
 *  - Outputs are overwritten unless an `accumulate` flag is set.
 *  - Results are deterministic: no floating-point atomics anywhere.
 *  - Shapes: T tokens per call (one chunk), M model width, H expert hidden
 *    width, E experts (1..64), k experts per token (1..min(E, 8)), C the
 *    per-expert capacity (>= 0). M and H must be multiples of 8.
 *
 * Row buffers (x_disp, y_disp, dy_disp, dx_disp, h_save, a_save) hold
 * flowmoe_rows_capacity(shape) rows: min(T*k, E*C) for the packed layout,
 * E*C for the padded one. Expert e owns rows [offsets[e], offsets[e] +
 * counts[e]). In the padded layout, rows between counts[e] and C are written
 * as zeros by every producer; in the packed layout rows at or past
 * offsets[E] are left untouched.
 */
#ifndef FLOWMOE_H
#define FLOWMOE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FLOWMOE_OK = 0,
  FLOWMOE_ERR_INVALID = 1,     /* bad argument or shape */
  FLOWMOE_ERR_UNSUPPORTED = 2, /* valid, but not implemented (e.g. E > 64) */
  FLOWMOE_ERR_HIP = 3,         /* a HIP runtime call failed */
  FLOWMOE_ERR_WORKSPACE = 4    /* workspace missing or too small */
} flowmoe_status_t;

enum { FLOWMOE_F32 = 0, FLOWMOE_BF16 = 1 };      /* layer dtype */
enum { FLOWMOE_GELU = 0, FLOWMOE_SWIGLU = 1 };   /* expert activation */
enum { FLOWMOE_PACKED = 0, FLOWMOE_PADDED = 1 }; /* dispatch layout */
/* Gate weights of the k selected experts (Sec. 2.1's softmax gate):
 * RENORM: the softmax over the k selected logits (the full softmax
 *         renormalised over the selection; k = 1 gives weight 1);
 * FULL:   the selected experts' own probabilities under the softmax over all
 *         E logits, not renormalised (Switch-style: a top-1 router keeps a
 *         gradient); bf16 layers only. */
enum { FLOWMOE_GATE_RENORM = 0, FLOWMOE_GATE_FULL = 1 };

/* Shape of one layer call (one chunk of T tokens). */
typedef struct {
  int32_t T, M, H, E, k, C;
  int32_t dtype;  /* FLOWMOE_F32 | FLOWMOE_BF16 */
  int32_t act;    /* FLOWMOE_GELU | FLOWMOE_SWIGLU */
  int32_t layout; /* FLOWMOE_PACKED | FLOWMOE_PADDED */
  int32_t gate;   /* FLOWMOE_GATE_RENORM (0) | FLOWMOE_GATE_FULL */
} flowmoe_shape_t;

/* Workspace kinds for flowmoe_workspace_bytes(). */
enum {
  FLOWMOE_WS_DISPATCH = 0,
  FLOWMOE_WS_FFN_BWD = 1,
  FLOWMOE_WS_GATE_BWD = 2,
  FLOWMOE_WS_LAYER_BWD = 3,
  FLOWMOE_WS_MHA_BWD = 4,      /* flowmoe_mha_bwd (depends on shape->M only) */
  FLOWMOE_WS_LAYER_BWD_MHA = 5 /* flowmoe_layer_bwd with bufs->mha set */
};

/* ---- utilities ---------------------------------------------------------- */

/* Library version string, e.g. "flowmoe 0.1.0 gfx950". */
const char* flowmoe_version(void);

/* Message of the last non-OK status returned on this host thread ("" if none). */
const char* flowmoe_last_error(void);

/* Expert capacity C = ceil(f * k * T / E) (Sec. 2.1, C = f*k*B*N/E), computed
 * exactly on the decimal value of f: the shortest decimal that reads back
 * as f (1.1, not the binary value 1.10000000000000008882), so that products
 * that are integers in decimal arithmetic are not rounded up by binary
 * rounding error. Returns -1 for T < 0, E < 1, k < 1, f <= 0 or not finite,
 * or a capacity above INT32_MAX. */
int32_t flowmoe_capacity(int32_t T, int32_t E, int32_t k, double f);

/* Rows of the dispatched buffers for `shape`: E*C (padded) or
 * min(T*k, E*C) (packed). Returns -1 for an invalid shape. */
int64_t flowmoe_rows_capacity(const flowmoe_shape_t* shape);

/* Bytes of scratch the call of the given kind needs (0 = none). */
size_t flowmoe_workspace_bytes(const flowmoe_shape_t* shape, int32_t kind);

/* ---- forward (Sec. 2.1; one chunk's AT_r gating, D_r, E_r, C_r) ---------- */

/* Gate: logits = x W_g (+ bias), the linear M x E gate of Sec. 4.2, then per
 * token the k largest logits in descending order (ties to the lower expert
 * index, -0.0 == +0.0) and their weights: the softmax over the k selected
 * logits (FLOWMOE_GATE_RENORM: the softmax of Sec. 2.1 renormalised over the
 * selection) or the selected experts' probabilities under the softmax over
 * all E logits (FLOWMOE_GATE_FULL).
 *   x        T x M  layer dtype
 *   w_gate   M x E  layer dtype
 *   bias     E      float, nullable (constant per-expert logit offset)
 *   logits   T x E  float (out)
 *   topk_idx T x k  int32 (out)
 *   topk_w   T x k  float (out) */
flowmoe_status_t flowmoe_gate_topk(const flowmoe_shape_t* shape, const void* x,
                                   const void* w_gate, const float* bias, float* logits,
                                   int32_t* topk_idx, float* topk_w, hipStream_t stream);

/* The selection and weights of flowmoe_gate_topk from given float logits
 * (T x E); the same device routine. */
flowmoe_status_t flowmoe_route(const flowmoe_shape_t* shape, const float* logits,
                               int32_t* topk_idx, float* topk_w, hipStream_t stream);

/* Dispatch (D_r): capacity-bounded positions and the token permutation into
 * the expert-major send layout G(I') of Sec. 2.1. Assignments are ranked
 * every first choice before any second choice, ascending token within a
 * rank; assignment (t, j) is kept iff fewer than C earlier assignments chose
 * the same expert. Then x_disp[slot[t][j]] = x[t] for every kept one.
 *   topk_idx T x k int32 (in); an id outside [0, E) is treated as dropped
 *   x        T x M layer dtype (in)
 *   counts   E     int32 (out) kept rows per expert, min(demand, C)
 *   offsets  E+1   int32 (out) first row of each expert: prefix sums of
 *                  counts (packed) or e*C (padded); offsets[E] = end
 *   slot     T x k int32 (out) row of assignment (t, j), or -1 if dropped
 *   row_src  rows  int32 (out) t*k + j for the assignment in each row, -1
 *                  for an empty row (rows = flowmoe_rows_capacity)
 *   load     E     int32 (out, nullable) demand per expert before the drop
 *   x_disp   rows x M layer dtype (out)
 *   ws       nullable; flowmoe_workspace_bytes(shape, FLOWMOE_WS_DISPATCH)
 *            bytes (0 for T*k <= 1024). With it, inputs of more than 1024
 *            assignments count each 1024-assignment tile's experts once into
 *            the workspace instead of every tile recounting all others;
 *            results are identical. Non-null but too small:
 *            FLOWMOE_ERR_WORKSPACE. */
flowmoe_status_t flowmoe_dispatch(const flowmoe_shape_t* shape, const int32_t* topk_idx,
                                  const void* x, int32_t* counts, int32_t* offsets,
                                  int32_t* slot, int32_t* row_src, int32_t* load,
                                  void* x_disp, void* ws, size_t ws_bytes, hipStream_t stream);

/* Expert FFN (E_r), Sec. 2.1's two feed-forward layers M x H then H x M, on
 * each expert's rows (counts and offsets as flowmoe_dispatch writes them;
 * they are device data, so they are not checked on the host, but a range
 * they would take past the rows buffers is cut there), as one grouped GEMM
 * per layer, with optional biases (the biased two-layer experts that the
 * parameter counts of Table 3 imply):
 *   GELU:   h = X W1_e + b1_e,                         a = gelu(h) (exact erf)
 *   SwiGLU: h1 = X W1_e + b1_e, h3 = X W3_e + b3_e,    a = silu(h1) * h3
 *   y_disp = a W2_e + b2_e.
 *   w1, w3   E x M x H layer dtype (w3 used only for SwiGLU, else nullable)
 *   w2       E x H x M layer dtype
 *   b1, b3   E x H float, nullable (b3 used for SwiGLU only); b2 E x M
 *            float, nullable; 16-byte aligned. Rows past an expert's count
 *            (the padded layout) stay zero: no bias is added to them.
 *   h_save   rows x H (GELU) or rows x 2H ([h1 | h3], SwiGLU) (out)
 *   a_save   rows x H (out)  -- both kept for the backward
 *   y_disp   rows x M (out) */
flowmoe_status_t flowmoe_expert_ffn(const flowmoe_shape_t* shape, const void* x_disp,
                                    const int32_t* counts, const int32_t* offsets,
                                    const void* w1, const void* w3, const void* w2,
                                    const float* b1, const float* b3, const float* b2,
                                    void* h_save, void* a_save, void* y_disp,
                                    hipStream_t stream);

/* Combine (C_r): y[t] = sum over kept j of topk_w[t][j] * y_disp[slot[t][j]],
 * zero when no assignment of t is kept (Sec. 2.1). y is T x M layer dtype. */
flowmoe_status_t flowmoe_combine(const flowmoe_shape_t* shape, const void* y_disp,
                                 const int32_t* slot, const float* topk_w, void* y,
                                 hipStream_t stream);

/* ---- backward (reverse order, Eqs. 5-6) ----------------------------------- */

/* Combine backward: dy_disp[slot] = topk_w * dy[t] and
 * d_topk_w[t][j] = <dy[t], y_disp[slot[t][j]]> (0 for dropped assignments).
 * counts/offsets give the padded rows to zero. */
flowmoe_status_t flowmoe_combine_bwd(const flowmoe_shape_t* shape, const void* dy,
                                     const void* y_disp, const int32_t* slot,
                                     const float* topk_w, const int32_t* counts,
                                     const int32_t* offsets, void* dy_disp, float* d_topk_w,
                                     hipStream_t stream);

/* Expert FFN backward: dA = dY W2_e^T, dW2_e = A^T dY; through the
 * activation (GELU: dH = dA * gelu'(h); SwiGLU: dH1 = dA * h3 * silu'(h1),
 * dH3 = dA * silu(h1)); dW1_e = X^T dH1, dW3_e = X^T dH3,
 * dX = dH1 W1_e^T (+ dH3 W3_e^T); the biases' gradients are the column sums
 * over expert e's rows: db2_e = sum dY, db1_e = sum dH1, db3_e = sum dH3.
 *   dw1, dw3 E x M x H float; dw2 E x H x M float. With accumulate != 0 the
 *   weight (and bias) gradients are added to (sum over chunks, App. H),
 *   else written.
 *   db1, db3 E x H float, db2 E x M float: each nullable (not computed),
 *   16-byte aligned; they do not depend on whether the forward had biases
 *   (h_save holds the biased pre-activations).
 *   dx_disp rows x M layer dtype (out).
 *   ws: flowmoe_workspace_bytes(shape, FLOWMOE_WS_FFN_BWD) bytes. */
flowmoe_status_t flowmoe_expert_ffn_bwd(const flowmoe_shape_t* shape, const void* dy_disp,
                                        const void* x_disp, const void* h_save,
                                        const void* a_save, const int32_t* counts,
                                        const int32_t* offsets, const void* w1,
                                        const void* w3, const void* w2, void* dx_disp,
                                        float* dw1, float* dw3, float* dw2, float* db1,
                                        float* db3, float* db2, int32_t accumulate, void* ws,
                                        size_t ws_bytes, hipStream_t stream);

/* Dispatch backward: dx[t] = sum over kept j of dx_disp[slot[t][j]]
 * (zero for a token with no kept assignment). dx is T x M layer dtype. */
flowmoe_status_t flowmoe_dispatch_bwd(const flowmoe_shape_t* shape, const void* dx_disp,
                                      const int32_t* slot, void* dx, hipStream_t stream);

/* Gate backward: the Jacobian of the gate weights, with
 * s = sum_j w_j dw_j: FLOWMOE_GATE_RENORM d_logits[t][S_j] = w_j (dw_j - s),
 * zero off the selection; FLOWMOE_GATE_FULL d_logits[t][e] = -p_e s for
 * every expert (p the softmax of the token's logits, which `logits` gives:
 * T x E float, required in that mode, unused otherwise), except
 * w_j (dw_j - s) at e = S_j. dw_gate = x^T d_logits (M x E float);
 * dbias = column sums of d_logits (E float, nullable). If dx is given,
 * dx += d_logits W_g^T (T x M layer dtype, read-modify-write). accumulate
 * != 0 adds dw_gate and dbias to the existing values (sum over chunks).
 * With k = 1 under FLOWMOE_GATE_RENORM the single weight is exactly 1 and
 * d_logits is exactly zero: the call writes the zeros (d_logits; dw_gate
 * and dbias unless accumulating), leaves dx as it is and reads nothing of x.
 *   ws: flowmoe_workspace_bytes(shape, FLOWMOE_WS_GATE_BWD) bytes. */
flowmoe_status_t flowmoe_gate_topk_bwd(const flowmoe_shape_t* shape, const void* x,
                                       const void* w_gate, const float* logits,
                                       const int32_t* topk_idx, const float* topk_w,
                                       const float* d_topk_w, float* d_logits, float* dw_gate,
                                       float* dbias, void* dx, int32_t accumulate, void* ws,
                                       size_t ws_bytes, hipStream_t stream);

/* ---- the gate backward without a workspace --------------------------------- */

/* Bytes of device scratch the library holds for flowmoe_gate_topk_bwd_noalloc
 * (32 MiB per GPU it runs on, from its load until the process ends). */
#define FLOWMOE_NOALLOC_SCRATCH_BYTES (32u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the gate
 * backward of flowmoe_gate_topk_bwd, same arguments, same kernels and the
 * same results, without the workspace arguments. Its scratch is the
 * library's own static device array (FLOWMOE_NOALLOC_SCRATCH_BYTES per GPU);
 * the call allocates nothing. A shape whose flowmoe_workspace_bytes(shape,
 * FLOWMOE_WS_GATE_BWD) exceeds that size is rejected with
 * FLOWMOE_ERR_WORKSPACE before anything is enqueued. Every call on one GPU
 * shares that GPU's array: calls that may overlap on one GPU (on streams not
 * ordered with each other, or from several host threads) race and must not
 * be issued; calls in order on one stream are safe. */
flowmoe_status_t flowmoe_gate_topk_bwd_noalloc(const flowmoe_shape_t* shape, const void* x,
                                               const void* w_gate, const float* logits,
                                               const int32_t* topk_idx, const float* topk_w,
                                               const float* d_topk_w, float* d_logits,
                                               float* dw_gate, float* dbias, void* dx,
                                               int32_t accumulate, hipStream_t stream);

/* ---- kernel tracing ------------------------------------------------------- */

/* Kernel kinds (bit i of a trace mask selects kind i). */
enum {
  FLOWMOE_K_GATE = 0,            /* gate GEMV + top-k (flowmoe_gate_topk) */
  FLOWMOE_K_ROUTE = 1,           /* top-k from logits (flowmoe_route) */
  FLOWMOE_K_SCAN = 2,            /* capacity-bounded route scan (dispatch) */
  FLOWMOE_K_GATHER = 3,          /* row gather into x_disp (dispatch) */
  FLOWMOE_K_FFN1 = 4,            /* grouped GEMM h = X W1 (+ W3), activation epilogue */
  FLOWMOE_K_FFN2 = 5,            /* grouped GEMM y = a W2 */
  FLOWMOE_K_SWIGLU_ACT = 6,      /* fp32 SwiGLU activation */
  FLOWMOE_K_COMBINE = 7,         /* combine, and dispatch backward (gather-sum; in
                                    flowmoe_layer_bwd fused with dx += d_logits W_g^T) */
  FLOWMOE_K_COMBINE_BWD = 8,     /* combine backward */
  FLOWMOE_K_DGRAD1 = 9,          /* grouped GEMM dA = dY W2^T, activation' epilogue */
  FLOWMOE_K_WGRAD2 = 10,         /* grouped GEMM dW2 = A^T dY */
  FLOWMOE_K_WGRAD1 = 11,         /* grouped GEMM [dW1 | dW3] = X^T dH */
  FLOWMOE_K_DGRAD2 = 12,         /* grouped GEMM dX = dH W1^T (+ dH3 W3^T) */
  FLOWMOE_K_GATE_BWD_WT = 13,    /* stacked W_g^T of the full softmax gate's dense dx term */
  FLOWMOE_K_GATE_BWD_TOKEN = 14, /* dx += d_logits W_g^T (flowmoe_gate_topk_bwd with dx) */
  FLOWMOE_K_GATE_BWD_DW = 15,    /* d_logits, and dW_g / db split-T partials */
  FLOWMOE_K_GATE_BWD_REDUCE = 16, /* dW_g / db reduction over splits (+ W_g^T for the dx term) */
  FLOWMOE_K_BIAS_GRAD = 17,       /* the experts' bias gradients (column sums of dY, dH) */
  FLOWMOE_K_ATTN_QKV = 18,        /* attention: [Q | K | V] = I [W^Q | W^K | W^V] */
  FLOWMOE_K_ATTN_FWD = 19,        /* attention: softmax(Q K^T / sqrt(d)) V per head */
  FLOWMOE_K_ATTN_OUT = 20,        /* attention: I' = A W^O */
  FLOWMOE_K_ATTN_DGRAD = 21,      /* attention: dA = dI' W^O^T, dI = d[Q|K|V] [W^Q|W^K|W^V]^T */
  FLOWMOE_K_ATTN_BWD_DQ = 22,     /* attention backward: dQ and rowsum(dA * A) */
  FLOWMOE_K_ATTN_BWD_DKDV = 23,   /* attention backward: dK, dV */
  FLOWMOE_K_ATTN_WGRAD = 24       /* attention: dW^O, d[W^Q | W^K | W^V] */
};

/* Start tracing on the calling host thread: every later kernel launch whose
 * kind bit is set in `mask` records events[2i] on its stream just before the
 * launch and events[2i+1] just after, with kinds[i] (host memory) set to its
 * kind, for i = 0, 1, ... until `pairs` pairs are used (later launches are
 * not traced). Events are created by the caller (timing enabled). Tracing
 * only records events; it changes no result. */
flowmoe_status_t flowmoe_trace_start(hipEvent_t* events, int32_t* kinds, int32_t pairs,
                                     uint32_t mask);

/* Stop tracing; returns the number of pairs recorded since the start. */
int32_t flowmoe_trace_stop(void);

/* ---- grouped-GEMM tile shape ------------------------------------------------ */

/* Output tile shapes of the bf16 grouped GEMM (expert FFN forward and
 * backward). AUTO, the default: 256 x 256 tiles (one block per compute unit)
 * unless a launch would have at most 1.25 x 256 of them, then 256 x 128
 * tiles (up to two blocks per compute unit). WIDE and NARROW force one
 * shape (the SwiGLU forward always takes 256 x 256). Both shapes accumulate
 * every output in the same k order: results are bit-identical. */
enum { FLOWMOE_TILES_AUTO = 0, FLOWMOE_TILES_WIDE = 1, FLOWMOE_TILES_NARROW = 2 };

/* Set the tile shape for launches enqueued after the call, process-wide
 * (for tests and tuning). FLOWMOE_ERR_INVALID for another value. */
flowmoe_status_t flowmoe_set_gemm_tiles(int32_t tiles);

/* Order of the row-mode tiles of the bf16 grouped GEMM. An expert's row
 * tiles are heavy (at least half of 256 rows live) or light (its short last
 * tile). SPLIT runs every heavy tile before any light one (the light tiles
 * fill the last round of the compute units); JOINED walks an expert's light
 * tiles with its heavy ones, so that a light tile reads its weight panels
 * while the heavy tiles of the same expert have them in the L2 / Infinity
 * Cache. AUTO, the default: JOINED when the launch's expert weights exceed
 * the 256 MB Infinity Cache and the experts average at most eight row tiles
 * (rows capacity <= 2048 E), else SPLIT. Every output is computed by the
 * same tile code in the same k order: results are bit-identical. */
enum { FLOWMOE_TILE_ORDER_AUTO = 0, FLOWMOE_TILE_ORDER_SPLIT = 1, FLOWMOE_TILE_ORDER_JOINED = 2 };

/* Set the tile order for launches enqueued after the call, process-wide (for
 * tests and tuning). FLOWMOE_ERR_INVALID for another value. */
flowmoe_status_t flowmoe_set_tile_order(int32_t order);

/* ---- row streams of the dispatch and combine kernels ----------------------- */

/* How the row kernels (dispatch gather/scatter, combine, their backward and
 * the dispatch backward) move bf16 rows. AUTO, the default: non-temporal
 * loads and stores for calls that move at least 256 MB (more than the
 * Infinity Cache holds, so caching the stream only evicts data that is read
 * again), cached ones below. NT and CACHED force one kind for every bf16
 * call; fp32 calls always go through the caches. Results are identical. */
enum { FLOWMOE_ROWS_AUTO = 0, FLOWMOE_ROWS_NT = 1, FLOWMOE_ROWS_CACHED = 2 };

/* Set the row-stream kind for launches enqueued after the call, process-wide
 * (for tests and tuning). FLOWMOE_ERR_INVALID for another value. */
flowmoe_status_t flowmoe_set_row_streams(int32_t mode);

/* ---- the attention part of AT_r (Sec. 2.1 MHA, Sec. 3.2 AT_r) ------------- */

/* The block's multi-head attention. A call's shape->T tokens are
 * T / seq_len whole sequences of seq_len tokens (N of Sec. 2.1) each, and
 * M = heads * head_dim. Tensors are bf16 (shape->dtype must be
 * FLOWMOE_BF16) and 16-byte aligned; lse and delta are float, 4-byte
 * aligned. Only shape->T, shape->M and shape->dtype are used. */
typedef struct {
  int32_t seq_len;  /* tokens per sequence */
  int32_t heads;
  int32_t head_dim; /* 64 or 128 (else FLOWMOE_ERR_UNSUPPORTED) */
  int32_t causal;   /* 1: token i attends to tokens j <= i of its sequence;
                       0: to every token of its sequence */
} flowmoe_mha_shape_t;

/* Attention core (Sec. 2.1), per sequence and head h:
 *   A_h = softmax(Q_h K_h^T / sqrt(head_dim)) V_h  (a row per query)
 *   qkv   T x 3M (in): [Q | K | V], head h in columns h*head_dim .. of each
 *   attn  T x M (out): the heads' A_h side by side (head h in its columns)
 *   lse   heads x T float (out): the natural log of each row's softmax
 *         denominator sum_j exp(s_ij), s = Q_h K_h^T / sqrt(head_dim) over
 *         the row's visible tokens; the backward needs it
 * Probabilities are rounded to bf16 before they multiply V; sums in float. */
flowmoe_status_t flowmoe_attention_fwd(const flowmoe_shape_t* shape,
                                       const flowmoe_mha_shape_t* mha, const void* qkv,
                                       void* attn, float* lse, hipStream_t stream);

/* Attention core backward: d_qkv (T x 3M, out) = the gradients of Q, K and V
 * from d_attn (T x M, the gradient of attn) and the forward's qkv, attn and
 * lse. delta (heads x T float, out): rowsum(d_attn_h * attn_h) per head and
 * token, an intermediate of the softmax backward (written, then read). */
flowmoe_status_t flowmoe_attention_bwd(const flowmoe_shape_t* shape,
                                       const flowmoe_mha_shape_t* mha, const void* qkv,
                                       const void* attn, const float* lse, const void* d_attn,
                                       void* d_qkv, float* delta, hipStream_t stream);

/* The block's MHA (Sec. 2.1): qkv = in [W^Q | W^K | W^V], the attention
 * core, out = attn W^O (the I' that the gate and the experts consume).
 *   in     T x M;  w_qkv M x 3M ([W^Q | W^K | W^V] side by side); w_o M x M
 *   qkv    T x 3M, attn T x M, lse heads x T (out, kept for the backward)
 *   out    T x M (out) */
flowmoe_status_t flowmoe_mha_fwd(const flowmoe_shape_t* shape, const flowmoe_mha_shape_t* mha,
                                 const void* in, const void* w_qkv, const void* w_o, void* qkv,
                                 void* attn, float* lse, void* out, hipStream_t stream);

/* MHA backward: d_attn = d_out W^O^T (T x M, out), the attention backward
 * (d_qkv T x 3M and delta heads x T, out), d_in = d_qkv [W^Q|W^K|W^V]^T
 * (T x M, out), dw_o = attn^T d_out (M x M float) and dw_qkv = in^T d_qkv
 * (M x 3M float), overwritten or, with accumulate, added to.
 * ws: flowmoe_workspace_bytes(shape, FLOWMOE_WS_MHA_BWD) bytes (nullable
 * when that is 0): when the weight gradients have few output tiles for the
 * compute units (M <= 1024), their token rows are split into partial sums
 * there, which are then added in split order. */
flowmoe_status_t flowmoe_mha_bwd(const flowmoe_shape_t* shape, const flowmoe_mha_shape_t* mha,
                                 const void* in, const void* w_qkv, const void* w_o,
                                 const void* qkv, const void* attn, const float* lse,
                                 const void* d_out, void* d_attn, void* d_qkv, float* delta,
                                 void* d_in, float* dw_qkv, float* dw_o, int32_t accumulate,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- the R-chunk two-stream layer (Sec. 3.2, Eqs. 3-6) -------------------- */

/* Buffers of a whole layer over R chunks of shape->T tokens each. Per-token
 * tensors cover all R*T tokens; per-chunk tensors are R consecutive blocks
 * (routing indices inside a block are chunk-local). rows = rows_capacity. */
typedef struct {
  /* parameters */
  const void* w_gate; /* M x E */
  const float* bias;  /* E, nullable */
  const void* w1;     /* E x M x H */
  const void* w3;     /* E x M x H, SwiGLU only */
  const void* w2;     /* E x H x M */
  const float* b1;    /* E x H, nullable: the experts' biases (flowmoe_expert_ffn) */
  const float* b3;    /* E x H, nullable, SwiGLU only */
  const float* b2;    /* E x M, nullable */
  /* forward */
  void* x;            /* RT x M: the layer input; with `mha`, the attention
                         output I' (written by the forward) */
  float* logits;      /* RT x E */
  int32_t* topk_idx;  /* RT x k */
  float* topk_w;      /* RT x k */
  int32_t* counts;    /* R x E */
  int32_t* offsets;   /* R x (E+1) */
  int32_t* slot;      /* RT x k */
  int32_t* row_src;   /* R x rows */
  int32_t* load;      /* R x E, nullable */
  void* x_disp;       /* R x rows x M */
  void* h_save;       /* R x rows x H (x2 for SwiGLU); dH after flowmoe_layer_bwd */
  void* a_save;       /* R x rows x H */
  void* y_disp;       /* R x rows x M */
  void* y;            /* RT x M */
  /* backward */
  const void* dy;     /* RT x M */
  void* dy_disp;      /* R x rows x M */
  float* d_topk_w;    /* RT x k */
  void* dx_disp;      /* R x rows x M */
  void* dx;           /* RT x M */
  float* d_logits;    /* RT x E */
  float* dw_gate;     /* M x E, summed over chunks */
  float* dbias;       /* E, nullable */
  float* dw1;         /* E x M x H, summed over chunks */
  float* dw3;         /* E x M x H, SwiGLU only */
  float* dw2;         /* E x H x M */
  float* db1;         /* E x H, nullable: the experts' bias gradients, summed over chunks */
  float* db3;         /* E x H, nullable, SwiGLU only */
  float* db2;         /* E x M, nullable */
  /* the attention part of AT_r (flowmoe_mha_fwd / _bwd per chunk); all
     ignored when mha is null. Chunk r's sequences are its tokens, so
     shape->T must be a whole number of sequences */
  const flowmoe_mha_shape_t* mha;
  const void* mha_in; /* RT x M: the block input I */
  const void* w_qkv;  /* M x 3M */
  const void* w_o;    /* M x M */
  void* qkv;          /* RT x 3M (forward; kept for the backward) */
  void* attn;         /* RT x M (forward; kept) */
  float* lse;         /* R x heads x T (forward; kept) */
  void* d_attn;       /* RT x M (backward) */
  void* d_qkv;        /* RT x 3M (backward) */
  float* delta;       /* R x heads x T (backward) */
  void* d_in;         /* RT x M (backward): the block input's gradient */
  float* dw_qkv;      /* M x 3M, summed over chunks */
  float* dw_o;        /* M x M, summed over chunks */
  /* scratch */
  void* ws;           /* flowmoe_workspace_bytes(shape, FLOWMOE_WS_LAYER_BWD), or
                         FLOWMOE_WS_LAYER_BWD_MHA with mha;
                         nullable in the forward, which uses it as the
                         dispatch workspace of each chunk in turn */
  size_t ws_bytes;
} flowmoe_layer_bufs_t;

/* Forward of R chunks. Compute stream gets AT_1..AT_R (the chunk's
 * attention when bufs->mha is set, then its gate) then
 * E_1..E_R (experts) (Eq. 3); comm stream gets D_1..D_R then C_1..C_R
 * (Eq. 4); events make D_r wait for AT_r, E_r for D_r and C_r for E_r.
 * The call first makes s_comm wait for work already on s_compute and ends by
 * making s_compute wait for s_comm, so to the caller it is one operation on
 * s_compute. s_comm may equal s_compute (serial schedule, same results); with
 * R = 1 there is nothing to overlap and everything runs on s_compute.
 * trace (nullable): 8*R events, recorded at start/end of each task, at index
 * 2*(task*R + r) (+1 for the end), task 0 = AT_r (attention and gate),
 * 1 = dispatch, 2 = experts, 3 = combine. The events must be created by the
 * caller. */
flowmoe_status_t flowmoe_layer_fwd(const flowmoe_shape_t* shape, int32_t R,
                                   const flowmoe_layer_bufs_t* bufs, hipStream_t s_compute,
                                   hipStream_t s_comm, hipEvent_t* trace);

/* Backward of R chunks: comm stream gets C_R..C_1 (combine backward) then
 * D_R..D_1 (dispatch backward) (Eq. 6); compute stream gets E_R..E_1
 * (Eq. 5), with E_r after C_r and D_r after E_r (constraints 6b-6c). The
 * gating part of AT_r splits by what it reads: its parameter gradients
 * (d_logits, dW_g, db) need only C_r's d_topk_w and x, so AT_R..AT_1's share
 * runs on the comm stream right after C_1, while the compute stream is busy
 * with the expert backward; its input gradient dx += d_logits W_g^T is
 * fused into D_r. E_r computes the chunk's hidden-layer gradient dH and dX,
 * which D_r needs; the expert weight gradients, which no later task of the
 * layer needs, run once after E_1 as one GEMM per weight whose reduction
 * runs over the rows of chunks 1..R in that order (the same sums as R
 * per-chunk GEMMs, without R read-modify-write passes over the fp32
 * gradients); the experts' bias gradients (bufs->db1/db3/db2, column sums
 * of dH and dY over the rows of every chunk) run after D_1 on the comm
 * stream when both streams are in use, else after the weight gradients.
 * dW_g and db are summed over chunks in R..1 order.
 * bufs->h_save is consumed: each chunk's h_save is overwritten with its dH
 * (rows x H for GELU, rows x 2H = [dH1 | dH3] for SwiGLU).
 * trace (nullable): 8*R + 2 events, the first 8*R as for the forward with
 * task 0 = combine bwd, 1 = experts bwd (dH and dX of the chunk),
 * 2 = dispatch bwd (+ gate dx term), 3 = gate parameter gradients; the last
 * two (index 8*R, 8*R + 1) span the expert weight gradients.
 * With bufs->mha, the attention part of AT_R..AT_1 runs on the compute
 * stream after the expert weight gradients, chunk r's once D_r has made its
 * dx final (constraint 6d): flowmoe_mha_bwd's data part, dx being the
 * gradient of the attention output; then the attention's weight gradients
 * over all chunks, one GEMM per weight (dW^O, dW_qkv). The trace then holds
 * 10*R + 4 events: as above, then index 8*R + 2 + 2*r (+1) spanning chunk
 * r's attention backward and 10*R + 2 (+1) its weight gradients.
 * With R = 1 the two streams are used only for large layers (capacity rows
 * x M x H >= 2.5e11), where the expert GEMMs span many rounds of the compute
 * units; smaller ones run everything on s_compute. */
flowmoe_status_t flowmoe_layer_bwd(const flowmoe_shape_t* shape, int32_t R,
                                   const flowmoe_layer_bufs_t* bufs, hipStream_t s_compute,
                                   hipStream_t s_comm, hipEvent_t* trace);

#ifdef __cplusplus
}
#endif

#endif /* FLOWMOE_H */
