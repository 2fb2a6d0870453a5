// Shared device helpers and the internal launch interface of libflowmoe.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "flowmoe.h"

namespace flowmoe {

// ---------------------------------------------------------------------------
// scalar element access for the two layer dtypes
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;  // bf16 bit pattern

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// round to nearest, ties to even (v_cvt_pk_bf16_f32; inputs finite)
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
};

// 8 consecutive elements as float, from a 16-byte (bf16) or 2x16-byte (f32) load
__device__ __forceinline__ void load8(const bf16_t* p, float v[8]) {
  uint4 q = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float v[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(bf16_t* p, const float v[8]) {
  uint4 q;
  q.x = pack_bf16x2(v[0], v[1]);
  q.y = pack_bf16x2(v[2], v[3]);
  q.z = pack_bf16x2(v[4], v[5]);
  q.w = pack_bf16x2(v[6], v[7]);
  *reinterpret_cast<uint4*>(p) = q;
}
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// 8 consecutive elements in their stored form (bf16: one 16-byte vector;
// float: two), so that a kernel can issue all its loads before converting
// any of them (ext-vector types: arrays of them stay in registers)
typedef unsigned u32x4v_t __attribute__((ext_vector_type(4)));
struct Raw8b {
  u32x4v_t a;
};
struct Raw8f {
  u32x4v_t a, b;
};
__device__ __forceinline__ Raw8b raw8_load(const bf16_t* p) {
  return Raw8b{*reinterpret_cast<const u32x4v_t*>(p)};
}
__device__ __forceinline__ Raw8f raw8_load(const float* p) {
  return Raw8f{*reinterpret_cast<const u32x4v_t*>(p), *reinterpret_cast<const u32x4v_t*>(p + 4)};
}
// NT: non-temporal access (streams larger than the 256 MB Infinity Cache,
// whose lines would only evict data that is read again)
template <bool NT>
__device__ __forceinline__ u32x4v_t ld16(const u32x4v_t* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}
template <bool NT>
__device__ __forceinline__ void st16(u32x4v_t* p, const u32x4v_t& v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}
template <bool NT>
__device__ __forceinline__ Raw8b raw8_ld(const bf16_t* p) {
  return Raw8b{ld16<NT>(reinterpret_cast<const u32x4v_t*>(p))};
}
template <bool NT>
__device__ __forceinline__ Raw8f raw8_ld(const float* p) {
  return Raw8f{ld16<NT>(reinterpret_cast<const u32x4v_t*>(p)),
               ld16<NT>(reinterpret_cast<const u32x4v_t*>(p + 4))};
}
template <bool NT>
__device__ __forceinline__ void store8_t(bf16_t* p, const float v[8]) {
  u32x4v_t q;
  q.x = pack_bf16x2(v[0], v[1]);
  q.y = pack_bf16x2(v[2], v[3]);
  q.z = pack_bf16x2(v[4], v[5]);
  q.w = pack_bf16x2(v[6], v[7]);
  st16<NT>(reinterpret_cast<u32x4v_t*>(p), q);
}
template <bool NT>
__device__ __forceinline__ void store8_t(float* p, const float v[8]) {
  st16<NT>(reinterpret_cast<u32x4v_t*>(p),
           u32x4v_t{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                    __float_as_uint(v[3])});
  st16<NT>(reinterpret_cast<u32x4v_t*>(p + 4),
           u32x4v_t{__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]),
                    __float_as_uint(v[7])});
}
__device__ __forceinline__ void raw8_f32(const Raw8b& r, float v[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(r.a[i] << 16);
    v[2 * i + 1] = __uint_as_float(r.a[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void raw8_f32(const Raw8f& r, float v[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = __uint_as_float(r.a[i]);
    v[4 + i] = __uint_as_float(r.b[i]);
  }
}

// activations (fp32). erf follows Abramowitz & Stegun 7.1.26,
// erf(x) = 1 - (a1 t + ... + a5 t^5) exp(-x^2), t = 1 / (1 + p x), x >= 0,
// absolute error <= 1.5e-7; its exp(-x^2) term is also phi(z) * sqrt(2 pi)
// for x = z / sqrt(2), which the GELU derivative reuses. Reciprocals use the
// hardware's v_rcp_f32 (1 ulp), not a correctly rounded division: the
// epilogues evaluate these per output element, and the division sequence
// (about ten instructions each) made them a large share of a tile's time.
__device__ __forceinline__ float rcp_f(float x) { return __builtin_amdgcn_rcpf(x); }
struct ErfParts {
  float erf;   // erf(z / sqrt(2))
  float gexp;  // exp(-z^2 / 2)
};
__device__ __forceinline__ ErfParts erf_parts(float z) {
  const float x = fabsf(z) * 0.70710678118654752f;
  const float t = rcp_f(1.0f + 0.3275911f * x);
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float g = __expf(-x * x);
  const float ea = 1.0f - poly * g;
  return ErfParts{z < 0.0f ? -ea : ea, g};
}
// gelu(z) = z * Phi(z), Phi(z) = (1 + erf(z / sqrt(2))) / 2
__device__ __forceinline__ float gelu_f(float z) { return 0.5f * z * (1.0f + erf_parts(z).erf); }
// gelu'(z) = Phi(z) + z * phi(z)
__device__ __forceinline__ float gelu_grad_f(float z) {
  const ErfParts e = erf_parts(z);
  return 0.5f * (1.0f + e.erf) + z * 0.39894228040143268f * e.gexp;
}
__device__ __forceinline__ float sigmoid_f(float z) { return rcp_f(1.0f + __expf(-z)); }

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct Shape {
  int T, M, H, E, k, C, dtype, act, layout;
  int gate;   // FLOWMOE_GATE_RENORM | FLOWMOE_GATE_FULL
  long rows;  // rows capacity of the dispatched buffers
};

constexpr int kMaxE = 64;
constexpr int kMaxK = 8;

// internal launchers (return hipSuccess or the launch error)
hipError_t launch_gate_topk(const Shape& s, const void* x, const void* w_gate, const float* bias,
                            float* logits, int32_t* idx, float* w, hipStream_t st);
hipError_t launch_route(const Shape& s, const float* logits, int32_t* idx, float* w, hipStream_t st);
// dispatch workspace: per-tile expert histograms (0 bytes for one tile of
// 1024 assignments); ws may be null, then the scan recounts every tile
size_t dispatch_ws_bytes(const Shape& s);
hipError_t launch_dispatch(const Shape& s, const int32_t* idx, const void* x, int32_t* counts,
                           int32_t* offsets, int32_t* slot, int32_t* row_src, int32_t* load,
                           void* x_disp, void* ws, hipStream_t st);
hipError_t launch_combine(const Shape& s, const void* y_disp, const int32_t* slot, const float* w,
                          void* y, hipStream_t st);
hipError_t launch_combine_bwd(const Shape& s, const void* dy, const void* y_disp,
                              const int32_t* slot, const float* w, const int32_t* counts,
                              const int32_t* offsets, void* dy_disp, float* dw, hipStream_t st);
hipError_t launch_dispatch_bwd(const Shape& s, const void* dx_disp, const int32_t* slot, void* dx,
                               hipStream_t st);
// dx += the dispatch backward (the full softmax gate's layer path)
hipError_t launch_dispatch_bwd_add(const Shape& s, const void* dx_disp, const int32_t* slot,
                                   void* dx, hipStream_t st);
hipError_t launch_dispatch_bwd_gate(const Shape& s, const void* dx_disp, const int32_t* slot,
                                    const int32_t* idx, const float* w, const float* dw,
                                    const void* wgt, void* dx, hipStream_t st);
// gate backward workspace: [W_g^T, E x M in the layer dtype | dW_g partials]
size_t gate_bwd_ws_bytes(const Shape& s);
inline const void* gate_ws_wgt(const void* ws) { return ws; }
// logits: needed by the full softmax gate (nullable otherwise)
// One selected expert under the renormalised gate: its weight is exactly 1,
// so d_logits = w (dw - w dw) is exactly zero, and with it dW_g, db and the
// gate's share of dx; the gate backward then writes those zeros without
// reading x (the full softmax gate's top-1 has a nonzero gradient).
inline bool gate_grad_zero(const Shape& s) { return s.k == 1 && s.gate != FLOWMOE_GATE_FULL; }
// w_gate (nullable): the reduce launch also writes W_g^T at the front of ws
hipError_t launch_gate_dw(const Shape& s, const void* x, const float* logits, const int32_t* idx,
                          const float* w, const float* dw, float* d_logits, float* dw_gate,
                          float* dbias, int accumulate, void* ws, hipStream_t st,
                          const void* w_gate = nullptr);
hipError_t launch_gate_dx(const Shape& s, const int32_t* idx, const float* w, const float* dw,
                          const void* wgt, void* dx, hipStream_t st);
hipError_t launch_gate_bwd(const Shape& s, const void* x, const void* w_gate, const float* logits,
                           const int32_t* idx, const float* w, const float* dw, float* d_logits,
                           float* dw_gate, float* dbias, void* dx, int accumulate, void* ws,
                           hipStream_t st);
// full softmax gate: [W_g^T ; W_g^T] (bf16) into the gate workspace, then the
// dense dx term of the last launch_gate_dw on that workspace, stored into dx
// (add = false) or added to it
hipError_t launch_gate_wstack(const Shape& s, const void* w_gate, void* ws, hipStream_t st);
hipError_t launch_gate_dx_full(const Shape& s, void* ws, void* dx, bool add, hipStream_t st);
size_t ffn_bwd_ws_bytes(const Shape& s);
void set_gemm_tiles(int tiles);  // FLOWMOE_TILES_*, validated by the caller
void set_tile_order(int order);  // FLOWMOE_TILE_ORDER_*, validated by the caller
void set_row_streams(int mode);  // FLOWMOE_ROWS_*, validated by the caller
// dW_g partials of the bf16 gate backward: P[s] = X_s^T D_s (fp32, M x N)
// over token split s (rows offsets[s] .. + counts[s] of x (T x M, bf16) and
// of d (T x N, bf16)), on the grouped GEMM's weight-gradient path
hipError_t launch_gate_dw_gemm(const void* x, int T, int M, const void* d, int N,
                               const int32_t* counts, const int32_t* offsets, int S, float* P,
                               hipStream_t st);
// dx (T x M, bf16) = or += [hi | lo] (T x K) . wstack (K x M): the gate's
// dense dx term, the token splits as pseudo-experts sharing one B
hipError_t launch_gate_dx_gemm(const void* dlhl, int T, int K, const void* wstack, int M,
                               const int32_t* counts, const int32_t* offsets, int S, void* dx,
                               bool add, hipStream_t st);
// b1, b3 (E x H), b2 (E x M): float biases of the experts, each nullable
hipError_t launch_expert_ffn(const Shape& s, const void* x_disp, const int32_t* counts,
                             const int32_t* offsets, const void* w1, const void* w3,
                             const void* w2, const float* b1, const float* b3, const float* b2,
                             void* h_save, void* a_save, void* y_disp, hipStream_t st);
// input side of the expert backward of one chunk: dH (into dh, which may be
// h_save itself: each element's pre-activation is read before its gradient
// is written) and dX
hipError_t launch_expert_ffn_dgrad(const Shape& s, const void* dy_disp, const void* h_save,
                                   const int32_t* counts, const int32_t* offsets, const void* w1,
                                   const void* w3, const void* w2, void* dh, void* dx_disp,
                                   hipStream_t st);
// weight gradients summed over R chunks (chunk r's rows at r * rows of each
// row buffer, its counts and offsets at r * E and r * (E + 1)), one GEMM each,
// and the bias gradients (db1, db3, db2 nullable) as column sums of dH / dY
hipError_t launch_expert_ffn_wgrad(const Shape& s, int R, const void* dy_disp, const void* x_disp,
                                   const void* a_save, const void* dh, const int32_t* counts,
                                   const int32_t* offsets, float* dw1, float* dw3, float* dw2,
                                   float* db1, float* db3, float* db2, int accumulate,
                                   hipStream_t st);
hipError_t launch_expert_bias_grad(const Shape& s, int R, const void* dy_disp, const void* dh,
                                   const int32_t* counts, const int32_t* offsets, float* db1,
                                   float* db3, float* db2, int accumulate, hipStream_t st);
hipError_t launch_expert_ffn_bwd(const Shape& s, const void* dy_disp, const void* x_disp,
                                 const void* h_save, const void* a_save, const int32_t* counts,
                                 const int32_t* offsets, const void* w1, const void* w3,
                                 const void* w2, void* dx_disp, float* dw1, float* dw3,
                                 float* dw2, float* db1, float* db3, float* db2, int accumulate,
                                 void* ws, hipStream_t st);

// Dense GEMMs on the grouped GEMM (one expert of `rows` rows, bf16):
// C (rows x N, bf16, ldc) = A (rows x K, lda) B (K x N) with B[k][n] at
// B + n * ldb + k (b_kc) or B + k * ldb + n
hipError_t launch_dense_gemm(int kind, long rows, const void* A, long lda, int K, const void* B,
                             long ldb, bool b_kc, int N, void* C, long ldc, hipStream_t st);
// C (Mdim x N, fp32, ldc) = (or +=) the sum over nseg segments g, in order,
// of A_g^T B_g (A_g = A + g * a_sstride: rows x Mdim; B_g: rows x N). With
// `part` (mha_wgrad_ws_bytes, ldc = N), a launch with few output tiles splits
// every segment's rows into partial sums there, added in order afterwards.
hipError_t launch_dense_wgrad(int kind, long rows, int nseg, const void* A, long lda,
                              long a_sstride, int Mdim, const void* B, long ldb, long b_sstride,
                              int N, float* C, long ldc, int accumulate, float* part,
                              hipStream_t st);
// row splits of such a launch (1: none), and the partial-sum bytes the
// attention's two weight gradients (M x 3M, M x M) need at width M
int dense_wgrad_splits(int Mdim, int N, long rows);
size_t mha_wgrad_ws_bytes(int M);

// The attention of AT_r: T tokens = T / N sequences of N tokens, `heads`
// heads of width D (64 or 128), M = heads * D, bf16
struct AttnShape {
  int N, heads, D, causal;
};
hipError_t launch_attn_fwd(const AttnShape& m, int T, int M, const void* qkv, void* o, float* lse,
                           hipStream_t st);
hipError_t launch_attn_bwd(const AttnShape& m, int T, int M, const void* qkv, const void* o,
                           const float* lse, const void* d_o, void* d_qkv, float* delta,
                           hipStream_t st);
// projections + attention: qkv = in W_qkv, attention -> attn, out = attn W_o
hipError_t launch_mha_fwd(const AttnShape& m, int T, int M, const void* in, const void* w_qkv,
                          const void* w_o, void* qkv, void* attn, float* lse, void* out,
                          hipStream_t st);
// input side of the backward: d_attn = d_out W_o^T, the attention backward
// (d_qkv, delta), d_in = d_qkv W_qkv^T
hipError_t launch_mha_bwd_data(const AttnShape& m, int T, int M, const void* w_qkv,
                               const void* w_o, const void* qkv, const void* attn,
                               const float* lse, const void* d_out, void* d_attn, void* d_qkv,
                               float* delta, void* d_in, hipStream_t st);
// weight gradients over R chunks of T rows: dW_o = sum attn^T d_out,
// dW_qkv = sum in^T d_qkv
// (ws: mha_wgrad_ws_bytes(M) of scratch for the partial sums, or null)
hipError_t launch_mha_wgrad(int T, int M, int R, const void* in, const void* attn,
                            const void* d_out, const void* d_qkv, float* dw_qkv, float* dw_o,
                            int accumulate, void* ws, hipStream_t st);

// Kernel tracing (flowmoe_trace_start): record a begin/end event around a
// launch when the kind is selected. Defined in abi.hip.
hipError_t trace_mark(int kind, bool end, hipStream_t st);

// launch `f` bracketed by trace marks of `kind`
template <class F>
inline hipError_t traced(int kind, hipStream_t st, F&& f) {
  hipError_t e = trace_mark(kind, false, st);
  if (e != hipSuccess) return e;
  f();
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return trace_mark(kind, true, st);
}

inline size_t esize(int dtype) { return dtype == FLOWMOE_BF16 ? 2 : 4; }
inline size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

}  // namespace flowmoe
