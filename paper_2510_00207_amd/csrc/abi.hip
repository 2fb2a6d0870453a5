// C ABI front end of libflowmoe: argument validation, status codes, workspace
// queries, and the R-chunk two-stream layer schedule (Sec. 3.2, Eqs. 3-6).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "common.hpp"

using namespace flowmoe;

namespace {

thread_local char g_err[512] = "";

flowmoe_status_t fail(flowmoe_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

flowmoe_status_t ok() {
  g_err[0] = '\0';
  return FLOWMOE_OK;
}

flowmoe_status_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(FLOWMOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

long rows_of(const flowmoe_shape_t* s) {
  const long ec = (long)s->E * s->C;
  if (s->layout == FLOWMOE_PADDED) return ec;
  const long tk = (long)s->T * s->k;
  return tk < ec ? tk : ec;
}

enum { NEED_H = 1, NEED_C = 2 };

// Validate a shape; fills `out`. Returns OK or the failing status.
flowmoe_status_t check_shape(const flowmoe_shape_t* s, int need, Shape* out) {
  if (s == nullptr) return fail(FLOWMOE_ERR_INVALID, "shape is null");
  if (s->dtype != FLOWMOE_F32 && s->dtype != FLOWMOE_BF16)
    return fail(FLOWMOE_ERR_INVALID, "dtype %d is not FLOWMOE_F32 or FLOWMOE_BF16", s->dtype);
  if (s->act != FLOWMOE_GELU && s->act != FLOWMOE_SWIGLU)
    return fail(FLOWMOE_ERR_INVALID, "act %d is not FLOWMOE_GELU or FLOWMOE_SWIGLU", s->act);
  if (s->layout != FLOWMOE_PACKED && s->layout != FLOWMOE_PADDED)
    return fail(FLOWMOE_ERR_INVALID, "layout %d is not FLOWMOE_PACKED or FLOWMOE_PADDED", s->layout);
  if (s->gate != FLOWMOE_GATE_RENORM && s->gate != FLOWMOE_GATE_FULL)
    return fail(FLOWMOE_ERR_INVALID, "gate %d is not FLOWMOE_GATE_RENORM or FLOWMOE_GATE_FULL",
                s->gate);
  if (s->gate == FLOWMOE_GATE_FULL && s->dtype != FLOWMOE_BF16)
    return fail(FLOWMOE_ERR_UNSUPPORTED, "FLOWMOE_GATE_FULL needs FLOWMOE_BF16 layers");
  if (s->T < 0) return fail(FLOWMOE_ERR_INVALID, "T = %d < 0", s->T);
  if (s->M < 8 || s->M % 8) return fail(FLOWMOE_ERR_INVALID, "M = %d must be a positive multiple of 8", s->M);
  if (s->E < 1) return fail(FLOWMOE_ERR_INVALID, "E = %d < 1", s->E);
  if (s->E > kMaxE) return fail(FLOWMOE_ERR_UNSUPPORTED, "E = %d > %d", s->E, kMaxE);
  if (s->k < 1 || s->k > s->E) return fail(FLOWMOE_ERR_INVALID, "k = %d not in [1, E = %d]", s->k, s->E);
  if (s->k > kMaxK) return fail(FLOWMOE_ERR_UNSUPPORTED, "k = %d > %d", s->k, kMaxK);
  if ((need & NEED_H) && (s->H < 8 || s->H % 8))
    return fail(FLOWMOE_ERR_INVALID, "H = %d must be a positive multiple of 8", s->H);
  if ((need & NEED_C) && s->C < 0) return fail(FLOWMOE_ERR_INVALID, "C = %d < 0", s->C);
  const long tk = (long)s->T * s->k;
  if (tk > (1L << 30)) return fail(FLOWMOE_ERR_UNSUPPORTED, "T*k = %ld too large", tk);
  if ((need & NEED_C) && (long)s->E * s->C > (1L << 30))
    return fail(FLOWMOE_ERR_UNSUPPORTED, "E*C too large");
  const long rows = (need & NEED_C) ? rows_of(s) : 0;
  const long width = (need & NEED_H) ? 2L * (s->H > s->M ? s->H : s->M) : s->M;
  if (rows * width > (1L << 40) || (long)s->T * s->M > (1L << 40))
    return fail(FLOWMOE_ERR_UNSUPPORTED, "tensor too large");
  if (out) {
    out->T = s->T; out->M = s->M; out->H = s->H; out->E = s->E; out->k = s->k;
    out->C = s->C; out->dtype = s->dtype; out->act = s->act; out->layout = s->layout;
    out->gate = s->gate;
    out->rows = rows;
  }
  return FLOWMOE_OK;
}

#define REQUIRE(p, name) \
  if ((p) == nullptr) return fail(FLOWMOE_ERR_INVALID, "%s is null", name)

// a tensor of the layer dtype: non-null and 16-byte aligned (kernels move it
// in 16-byte vectors)
#define REQUIRE_T(p, name)                                                      \
  if ((p) == nullptr) return fail(FLOWMOE_ERR_INVALID, "%s is null", name);      \
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0)                                 \
    return fail(FLOWMOE_ERR_INVALID, "%s is not 16-byte aligned", name)

// the experts' biases (or their gradients, prefix "d"): each nullable, float,
// 16-byte aligned (moved in 16-byte vectors); b3 is used with SwiGLU only
flowmoe_status_t check_biases(const Shape& s, const float* b1, const float* b3, const float* b2,
                              const char* prefix) {
  const float* p[3] = {b1, s.act == FLOWMOE_SWIGLU ? b3 : nullptr, b2};
  const char* n[3] = {"b1", "b3", "b2"};
  for (int i = 0; i < 3; ++i)
    if (p[i] != nullptr && reinterpret_cast<uintptr_t>(p[i]) % 16 != 0)
      return fail(FLOWMOE_ERR_INVALID, "%s%s is not 16-byte aligned", prefix, n[i]);
  return FLOWMOE_OK;
}

flowmoe_status_t check_ws(void* ws, size_t have, size_t need, const char* call) {
  if (need == 0) return FLOWMOE_OK;
  if (ws == nullptr || have < need)
    return fail(FLOWMOE_ERR_WORKSPACE, "%s needs %zu workspace bytes, got %zu%s", call, need,
                ws == nullptr ? (size_t)0 : have, ws == nullptr ? " (null)" : "");
  return FLOWMOE_OK;
}

// per-thread, per-device pool of events for cross-stream ordering
struct EventPool {
  int device = -1;
  std::vector<hipEvent_t> ev;
};
thread_local std::vector<EventPool> g_pools;

hipError_t get_events(int n, hipEvent_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  EventPool* pool = nullptr;
  for (auto& p : g_pools)
    if (p.device == dev) pool = &p;
  if (pool == nullptr) {
    g_pools.push_back(EventPool());
    pool = &g_pools.back();
    pool->device = dev;
  }
  while ((int)pool->ev.size() < n) {
    hipEvent_t h;
    e = hipEventCreateWithFlags(&h, hipEventDisableTiming);
    if (e != hipSuccess) return e;
    pool->ev.push_back(h);
  }
  *out = pool->ev.data();
  return hipSuccess;
}

struct TraceState {
  hipEvent_t* ev = nullptr;
  int32_t* kinds = nullptr;
  int32_t pairs = 0;
  int32_t used = 0;
  uint32_t mask = 0;
  bool open = false;  // a begin was recorded for the current launch
};
thread_local TraceState g_trace;

inline const char* cptr(const void* p, long off) { return static_cast<const char*>(p) + off; }
inline char* mptr(void* p, long off) { return p == nullptr ? nullptr : static_cast<char*>(p) + off; }

}  // namespace

namespace flowmoe {
hipError_t trace_mark(int kind, bool end, hipStream_t st) {
  TraceState& t = g_trace;
  if (t.ev == nullptr || kind < 0 || kind >= 32 || !((t.mask >> kind) & 1u)) return hipSuccess;
  if (!end) {
    if (t.used >= t.pairs) return hipSuccess;
    t.open = true;
    t.kinds[t.used] = kind;
    return hipEventRecord(t.ev[2 * t.used], st);
  }
  if (!t.open) return hipSuccess;
  t.open = false;
  const hipError_t e = hipEventRecord(t.ev[2 * t.used + 1], st);
  ++t.used;
  return e;
}
}  // namespace flowmoe

extern "C" {

flowmoe_status_t flowmoe_trace_start(hipEvent_t* events, int32_t* kinds, int32_t pairs,
                                     uint32_t mask) {
  if (pairs < 0) return fail(FLOWMOE_ERR_INVALID, "pairs = %d < 0", pairs);
  if (pairs > 0 && (events == nullptr || kinds == nullptr))
    return fail(FLOWMOE_ERR_INVALID, "events and kinds must be given");
  g_trace = TraceState();
  g_trace.ev = pairs > 0 ? events : nullptr;
  g_trace.kinds = kinds;
  g_trace.pairs = pairs;
  g_trace.mask = mask;
  return ok();
}

int32_t flowmoe_trace_stop(void) {
  const int32_t n = g_trace.used;
  g_trace = TraceState();
  return n;
}

flowmoe_status_t flowmoe_set_gemm_tiles(int32_t tiles) {
  if (tiles != FLOWMOE_TILES_AUTO && tiles != FLOWMOE_TILES_WIDE && tiles != FLOWMOE_TILES_NARROW)
    return fail(FLOWMOE_ERR_INVALID, "tiles = %d is not a FLOWMOE_TILES_* value", tiles);
  set_gemm_tiles(tiles);
  return ok();
}

flowmoe_status_t flowmoe_set_tile_order(int32_t order) {
  if (order != FLOWMOE_TILE_ORDER_AUTO && order != FLOWMOE_TILE_ORDER_SPLIT &&
      order != FLOWMOE_TILE_ORDER_JOINED)
    return fail(FLOWMOE_ERR_INVALID, "order = %d is not a FLOWMOE_TILE_ORDER_* value", order);
  set_tile_order(order);
  return ok();
}

flowmoe_status_t flowmoe_set_row_streams(int32_t mode) {
  if (mode != FLOWMOE_ROWS_AUTO && mode != FLOWMOE_ROWS_NT && mode != FLOWMOE_ROWS_CACHED)
    return fail(FLOWMOE_ERR_INVALID, "mode = %d is not a FLOWMOE_ROWS_* value", mode);
  set_row_streams(mode);
  return ok();
}

const char* flowmoe_version(void) { return "flowmoe 0.2.0 gfx950"; }

const char* flowmoe_last_error(void) { return g_err; }

int32_t flowmoe_capacity(int32_t T, int32_t E, int32_t k, double f) {
  if (T < 0 || E < 1 || k < 1 || !(f > 0.0) || !isfinite(f)) return -1;
  // f as the shortest decimal that reads back as f: D * 10^x with D an
  // integer of p digits (printf rounds correctly; p = 17 always reads back)
  char buf[40];
  int p = 1;
  for (; p < 17; ++p) {
    snprintf(buf, sizeof(buf), "%.*e", p - 1, f);
    if (strtod(buf, nullptr) == f) break;
  }
  snprintf(buf, sizeof(buf), "%.*e", p - 1, f);
  unsigned long long D = 0;
  const char* c = buf;
  for (; *c != 'e'; ++c)
    if (*c >= '0' && *c <= '9') D = D * 10 + (unsigned long long)(*c - '0');
  const int x = atoi(c + 1) - (p - 1);
  // C = ceil(D * 10^x * k * T / E) in 128-bit integers (D < 10^17, k * T < 2^62)
  typedef unsigned __int128 u128;
  const u128 kMax = ~(u128)0;
  u128 num = (u128)D * (unsigned long long)k * (unsigned long long)T;
  if (num == 0) return 0;
  u128 den = (u128)(unsigned)E;
  if (x >= 0) {
    for (int i = 0; i < x; ++i) {
      if (num > kMax / 10) return -1;  // far beyond any int32 capacity
      num *= 10;
    }
  } else {
    for (int i = 0; i < -x; ++i) {
      if (den > num) return 1;  // 0 < value < 1
      den *= 10;
    }
  }
  const u128 c0 = num / den + (num % den != 0 ? 1 : 0);
  return c0 > (u128)2147483647 ? -1 : (int32_t)c0;
}

int64_t flowmoe_rows_capacity(const flowmoe_shape_t* shape) {
  Shape s;
  if (check_shape(shape, NEED_C, &s) != FLOWMOE_OK) return -1;
  return s.rows;
}

size_t flowmoe_workspace_bytes(const flowmoe_shape_t* shape, int32_t kind) {
  Shape s;
  if (check_shape(shape, NEED_H | NEED_C, &s) != FLOWMOE_OK) {
    if (check_shape(shape, 0, &s) != FLOWMOE_OK) return 0;
  }
  switch (kind) {
    case FLOWMOE_WS_DISPATCH: return dispatch_ws_bytes(s);
    case FLOWMOE_WS_FFN_BWD: return ffn_bwd_ws_bytes(s);
    case FLOWMOE_WS_GATE_BWD: return gate_bwd_ws_bytes(s);
    case FLOWMOE_WS_LAYER_BWD: {  // the backward's gate partials; the forward's scan histograms
      const size_t bwd = gate_bwd_ws_bytes(s), fwd = dispatch_ws_bytes(s);
      return bwd > fwd ? bwd : fwd;
    }
    case FLOWMOE_WS_MHA_BWD: return mha_wgrad_ws_bytes(s.M);
    case FLOWMOE_WS_LAYER_BWD_MHA: {  // (the attention's weight gradients run last)
      const size_t bwd = gate_bwd_ws_bytes(s), fwd = dispatch_ws_bytes(s);
      return std::max(std::max(bwd, fwd), mha_wgrad_ws_bytes(s.M));
    }
    default: return 0;
  }
}

flowmoe_status_t flowmoe_gate_topk(const flowmoe_shape_t* shape, const void* x,
                                   const void* w_gate, const float* bias, float* logits,
                                   int32_t* topk_idx, float* topk_w, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, 0, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(w_gate, "w_gate");
  if (s.T > 0) {
    REQUIRE_T(x, "x");
    REQUIRE(logits, "logits");
    REQUIRE(topk_idx, "topk_idx");
    REQUIRE(topk_w, "topk_w");
  }
  return hip_status(launch_gate_topk(s, x, w_gate, bias, logits, topk_idx, topk_w, stream),
                    "flowmoe_gate_topk");
}

flowmoe_status_t flowmoe_route(const flowmoe_shape_t* shape, const float* logits,
                               int32_t* topk_idx, float* topk_w, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, 0, &s);
  if (st != FLOWMOE_OK) return st;
  if (s.T > 0) {
    REQUIRE(logits, "logits");
    REQUIRE(topk_idx, "topk_idx");
    REQUIRE(topk_w, "topk_w");
  }
  return hip_status(launch_route(s, logits, topk_idx, topk_w, stream), "flowmoe_route");
}

flowmoe_status_t flowmoe_dispatch(const flowmoe_shape_t* shape, const int32_t* topk_idx,
                                  const void* x, int32_t* counts, int32_t* offsets,
                                  int32_t* slot, int32_t* row_src, int32_t* load, void* x_disp,
                                  void* ws, size_t ws_bytes, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE(counts, "counts");
  REQUIRE(offsets, "offsets");
  if (s.T > 0) {
    REQUIRE(topk_idx, "topk_idx");
    REQUIRE_T(x, "x");
    REQUIRE(slot, "slot");
  }
  if (s.rows > 0) {
    REQUIRE(row_src, "row_src");
    REQUIRE_T(x_disp, "x_disp");
  }
  if (ws != nullptr) {
    st = check_ws(ws, ws_bytes, dispatch_ws_bytes(s), "flowmoe_dispatch");
    if (st != FLOWMOE_OK) return st;
  }
  return hip_status(launch_dispatch(s, topk_idx, x, counts, offsets, slot, row_src, load, x_disp,
                                    ws, stream),
                    "flowmoe_dispatch");
}

flowmoe_status_t flowmoe_expert_ffn(const flowmoe_shape_t* shape, const void* x_disp,
                                    const int32_t* counts, const int32_t* offsets,
                                    const void* w1, const void* w3, const void* w2,
                                    const float* b1, const float* b3, const float* b2,
                                    void* h_save, void* a_save, void* y_disp,
                                    hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_H | NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE(counts, "counts");
  REQUIRE(offsets, "offsets");
  REQUIRE_T(w1, "w1");
  REQUIRE_T(w2, "w2");
  if (s.act == FLOWMOE_SWIGLU) REQUIRE_T(w3, "w3");
  st = check_biases(s, b1, b3, b2, "");
  if (st != FLOWMOE_OK) return st;
  if (s.rows > 0) {
    REQUIRE_T(x_disp, "x_disp");
    REQUIRE_T(h_save, "h_save");
    REQUIRE_T(a_save, "a_save");
    REQUIRE_T(y_disp, "y_disp");
  }
  return hip_status(launch_expert_ffn(s, x_disp, counts, offsets, w1, w3, w2, b1, b3, b2, h_save,
                                      a_save, y_disp, stream),
                    "flowmoe_expert_ffn");
}

flowmoe_status_t flowmoe_combine(const flowmoe_shape_t* shape, const void* y_disp,
                                 const int32_t* slot, const float* topk_w, void* y,
                                 hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  if (s.T > 0) {
    REQUIRE(slot, "slot");
    REQUIRE(topk_w, "topk_w");
    REQUIRE_T(y, "y");
    if (s.rows > 0) REQUIRE_T(y_disp, "y_disp");
  }
  return hip_status(launch_combine(s, y_disp, slot, topk_w, y, stream), "flowmoe_combine");
}

flowmoe_status_t flowmoe_combine_bwd(const flowmoe_shape_t* shape, const void* dy,
                                     const void* y_disp, const int32_t* slot,
                                     const float* topk_w, const int32_t* counts,
                                     const int32_t* offsets, void* dy_disp, float* d_topk_w,
                                     hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE(counts, "counts");
  if (s.T > 0) {
    REQUIRE_T(dy, "dy");
    REQUIRE(slot, "slot");
    REQUIRE(topk_w, "topk_w");
    REQUIRE(d_topk_w, "d_topk_w");
  }
  if (s.rows > 0) {
    REQUIRE_T(y_disp, "y_disp");
    REQUIRE_T(dy_disp, "dy_disp");
  }
  return hip_status(launch_combine_bwd(s, dy, y_disp, slot, topk_w, counts, offsets, dy_disp,
                                       d_topk_w, stream),
                    "flowmoe_combine_bwd");
}

flowmoe_status_t flowmoe_expert_ffn_bwd(const flowmoe_shape_t* shape, const void* dy_disp,
                                        const void* x_disp, const void* h_save,
                                        const void* a_save, const int32_t* counts,
                                        const int32_t* offsets, const void* w1,
                                        const void* w3, const void* w2, void* dx_disp,
                                        float* dw1, float* dw3, float* dw2, float* db1,
                                        float* db3, float* db2, int32_t accumulate, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_H | NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE(counts, "counts");
  REQUIRE(offsets, "offsets");
  REQUIRE_T(w1, "w1");
  REQUIRE_T(w2, "w2");
  REQUIRE(dw1, "dw1");
  REQUIRE(dw2, "dw2");
  if (s.act == FLOWMOE_SWIGLU) {
    REQUIRE_T(w3, "w3");
    REQUIRE(dw3, "dw3");
  }
  if (s.rows > 0) {
    REQUIRE_T(dy_disp, "dy_disp");
    REQUIRE_T(x_disp, "x_disp");
    REQUIRE_T(h_save, "h_save");
    REQUIRE_T(a_save, "a_save");
    REQUIRE_T(dx_disp, "dx_disp");
  }
  st = check_biases(s, db1, db3, db2, "d");
  if (st != FLOWMOE_OK) return st;
  st = check_ws(ws, ws_bytes, ffn_bwd_ws_bytes(s), "flowmoe_expert_ffn_bwd");
  if (st != FLOWMOE_OK) return st;
  return hip_status(launch_expert_ffn_bwd(s, dy_disp, x_disp, h_save, a_save, counts, offsets, w1,
                                          w3, w2, dx_disp, dw1, dw3, dw2, db1, db3, db2,
                                          accumulate != 0, ws, stream),
                    "flowmoe_expert_ffn_bwd");
}

flowmoe_status_t flowmoe_dispatch_bwd(const flowmoe_shape_t* shape, const void* dx_disp,
                                      const int32_t* slot, void* dx, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, NEED_C, &s);
  if (st != FLOWMOE_OK) return st;
  if (s.T > 0) {
    REQUIRE(slot, "slot");
    REQUIRE_T(dx, "dx");
    if (s.rows > 0) REQUIRE_T(dx_disp, "dx_disp");
  }
  return hip_status(launch_dispatch_bwd(s, dx_disp, slot, dx, stream), "flowmoe_dispatch_bwd");
}

flowmoe_status_t flowmoe_gate_topk_bwd(const flowmoe_shape_t* shape, const void* x,
                                       const void* w_gate, const float* logits,
                                       const int32_t* topk_idx, const float* topk_w,
                                       const float* d_topk_w,
                                       float* d_logits, float* dw_gate, float* dbias, void* dx,
                                       int32_t accumulate, void* ws, size_t ws_bytes,
                                       hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, 0, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(w_gate, "w_gate");
  REQUIRE(dw_gate, "dw_gate");
  if (s.T > 0) {
    REQUIRE_T(x, "x");
    REQUIRE(topk_idx, "topk_idx");
    REQUIRE(topk_w, "topk_w");
    REQUIRE(d_topk_w, "d_topk_w");
    REQUIRE(d_logits, "d_logits");
    if (s.gate == FLOWMOE_GATE_FULL) REQUIRE(logits, "logits");
  }
  if (dx != nullptr && reinterpret_cast<uintptr_t>(dx) % 16 != 0)
    return fail(FLOWMOE_ERR_INVALID, "dx is not 16-byte aligned");
  st = check_ws(ws, ws_bytes, gate_bwd_ws_bytes(s), "flowmoe_gate_topk_bwd");
  if (st != FLOWMOE_OK) return st;
  return hip_status(launch_gate_bwd(s, x, w_gate, logits, topk_idx, topk_w, d_topk_w, d_logits,
                                    dw_gate, dbias, dx, accumulate != 0, ws, stream),
                    "flowmoe_gate_topk_bwd");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// the gate backward without a caller workspace
// ---------------------------------------------------------------------------
namespace {

// The no-alloc gate backward's scratch: FLOWMOE_NOALLOC_SCRATCH_BYTES of
// device memory that every GPU the library runs on holds from the module's
// load until the process ends. Host code never uses this name as an address
// (on the host it is a stand-in, not device memory): the device address
// comes from hipGetSymbolAddress, once per device.
__device__ __align__(256) char scratch[FLOWMOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// device address of `scratch` on the current device
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

flowmoe_status_t flowmoe_gate_topk_bwd_noalloc(const flowmoe_shape_t* shape, const void* x,
                                               const void* w_gate, const float* logits,
                                               const int32_t* topk_idx, const float* topk_w,
                                               const float* d_topk_w, float* d_logits,
                                               float* dw_gate, float* dbias, void* dx,
                                               int32_t accumulate, hipStream_t stream) {
  Shape s;
  flowmoe_status_t st = check_shape(shape, 0, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(w_gate, "w_gate");
  REQUIRE(dw_gate, "dw_gate");
  if (s.T > 0) {
    REQUIRE_T(x, "x");
    REQUIRE(topk_idx, "topk_idx");
    REQUIRE(topk_w, "topk_w");
    REQUIRE(d_topk_w, "d_topk_w");
    REQUIRE(d_logits, "d_logits");
    if (s.gate == FLOWMOE_GATE_FULL) REQUIRE(logits, "logits");
  }
  if (dx != nullptr && reinterpret_cast<uintptr_t>(dx) % 16 != 0)
    return fail(FLOWMOE_ERR_INVALID, "dx is not 16-byte aligned");
  const size_t need = gate_bwd_ws_bytes(s);
  if (need > (size_t)FLOWMOE_NOALLOC_SCRATCH_BYTES)
    return fail(FLOWMOE_ERR_WORKSPACE,
                "flowmoe_gate_topk_bwd_noalloc: the shape needs %zu bytes of scratch, more than "
                "the %zu the library holds; call flowmoe_gate_topk_bwd with a workspace",
                need, (size_t)FLOWMOE_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return hip_status(e, "flowmoe_gate_topk_bwd_noalloc: scratch address");
  return hip_status(launch_gate_bwd(s, x, w_gate, logits, topk_idx, topk_w, d_topk_w, d_logits,
                                    dw_gate, dbias, dx, accumulate != 0, ws, stream),
                    "flowmoe_gate_topk_bwd_noalloc");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// R-chunk layer
// ---------------------------------------------------------------------------
namespace {

// The attention of T tokens of width M: bf16, whole sequences, M = heads *
// head_dim with head_dim 64 or 128
flowmoe_status_t check_mha(const flowmoe_shape_t* s, const flowmoe_mha_shape_t* m, AttnShape* out) {
  if (s == nullptr) return fail(FLOWMOE_ERR_INVALID, "shape is null");
  if (m == nullptr) return fail(FLOWMOE_ERR_INVALID, "mha is null");
  if (s->dtype != FLOWMOE_BF16)
    return fail(FLOWMOE_ERR_UNSUPPORTED, "the attention runs in FLOWMOE_BF16 only");
  if (s->T < 0) return fail(FLOWMOE_ERR_INVALID, "T = %d < 0", s->T);
  if (m->head_dim != 64 && m->head_dim != 128)
    return fail(FLOWMOE_ERR_UNSUPPORTED, "head_dim = %d is not 64 or 128", m->head_dim);
  if (m->heads < 1 || (long)m->heads * m->head_dim != s->M)
    return fail(FLOWMOE_ERR_INVALID, "heads * head_dim = %d * %d is not M = %d", m->heads,
                m->head_dim, s->M);
  if (m->seq_len < 1) return fail(FLOWMOE_ERR_INVALID, "seq_len = %d < 1", m->seq_len);
  if (s->T % m->seq_len)
    return fail(FLOWMOE_ERR_INVALID, "T = %d is not a whole number of sequences of %d tokens",
                s->T, m->seq_len);
  if (m->causal != 0 && m->causal != 1)
    return fail(FLOWMOE_ERR_INVALID, "causal = %d is not 0 or 1", m->causal);
  if ((long)s->T * 3 * s->M > (1L << 40) || s->T > (1 << 30))
    return fail(FLOWMOE_ERR_UNSUPPORTED, "tensor too large");
  if ((long)((m->seq_len + 127) / 128) * m->heads * (s->T / m->seq_len) > (1L << 31))
    return fail(FLOWMOE_ERR_UNSUPPORTED, "too many attention tiles");
  if (out) *out = AttnShape{m->seq_len, m->heads, m->head_dim, m->causal};
  return FLOWMOE_OK;
}

#define REQUIRE_F(p, name)                                                     \
  if ((p) == nullptr) return fail(FLOWMOE_ERR_INVALID, "%s is null", name);     \
  if (reinterpret_cast<uintptr_t>(p) % 4 != 0)                                 \
    return fail(FLOWMOE_ERR_INVALID, "%s is not 4-byte aligned", name)

}  // namespace

extern "C" {

flowmoe_status_t flowmoe_attention_fwd(const flowmoe_shape_t* shape,
                                       const flowmoe_mha_shape_t* mha, const void* qkv,
                                       void* attn, float* lse, hipStream_t stream) {
  AttnShape m;
  flowmoe_status_t st = check_mha(shape, mha, &m);
  if (st != FLOWMOE_OK) return st;
  if (shape->T == 0) return ok();
  REQUIRE_T(qkv, "qkv");
  REQUIRE_T(attn, "attn");
  REQUIRE_F(lse, "lse");
  return hip_status(launch_attn_fwd(m, shape->T, shape->M, qkv, attn, lse, stream),
                    "flowmoe_attention_fwd");
}

flowmoe_status_t flowmoe_attention_bwd(const flowmoe_shape_t* shape,
                                       const flowmoe_mha_shape_t* mha, const void* qkv,
                                       const void* attn, const float* lse, const void* d_attn,
                                       void* d_qkv, float* delta, hipStream_t stream) {
  AttnShape m;
  flowmoe_status_t st = check_mha(shape, mha, &m);
  if (st != FLOWMOE_OK) return st;
  if (shape->T == 0) return ok();
  REQUIRE_T(qkv, "qkv");
  REQUIRE_T(attn, "attn");
  REQUIRE_F(lse, "lse");
  REQUIRE_T(d_attn, "d_attn");
  REQUIRE_T(d_qkv, "d_qkv");
  REQUIRE_F(delta, "delta");
  return hip_status(launch_attn_bwd(m, shape->T, shape->M, qkv, attn, lse, d_attn, d_qkv, delta,
                                    stream),
                    "flowmoe_attention_bwd");
}

flowmoe_status_t flowmoe_mha_fwd(const flowmoe_shape_t* shape, const flowmoe_mha_shape_t* mha,
                                 const void* in, const void* w_qkv, const void* w_o, void* qkv,
                                 void* attn, float* lse, void* out, hipStream_t stream) {
  AttnShape m;
  flowmoe_status_t st = check_mha(shape, mha, &m);
  if (st != FLOWMOE_OK) return st;
  if (shape->T == 0) return ok();
  REQUIRE_T(in, "in");
  REQUIRE_T(w_qkv, "w_qkv");
  REQUIRE_T(w_o, "w_o");
  REQUIRE_T(qkv, "qkv");
  REQUIRE_T(attn, "attn");
  REQUIRE_F(lse, "lse");
  REQUIRE_T(out, "out");
  return hip_status(launch_mha_fwd(m, shape->T, shape->M, in, w_qkv, w_o, qkv, attn, lse, out,
                                   stream),
                    "flowmoe_mha_fwd");
}

flowmoe_status_t flowmoe_mha_bwd(const flowmoe_shape_t* shape, const flowmoe_mha_shape_t* mha,
                                 const void* in, const void* w_qkv, const void* w_o,
                                 const void* qkv, const void* attn, const float* lse,
                                 const void* d_out, void* d_attn, void* d_qkv, float* delta,
                                 void* d_in, float* dw_qkv, float* dw_o, int32_t accumulate,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  AttnShape m;
  flowmoe_status_t st = check_mha(shape, mha, &m);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(dw_qkv, "dw_qkv");
  REQUIRE_T(dw_o, "dw_o");
  if (shape->T > 0) {
    REQUIRE_T(in, "in");
    REQUIRE_T(w_qkv, "w_qkv");
    REQUIRE_T(w_o, "w_o");
    REQUIRE_T(qkv, "qkv");
    REQUIRE_T(attn, "attn");
    REQUIRE_F(lse, "lse");
    REQUIRE_T(d_out, "d_out");
    REQUIRE_T(d_attn, "d_attn");
    REQUIRE_T(d_qkv, "d_qkv");
    REQUIRE_F(delta, "delta");
    REQUIRE_T(d_in, "d_in");
  }
  st = check_ws(ws, ws_bytes, mha_wgrad_ws_bytes(shape->M), "flowmoe_mha_bwd");
  if (st != FLOWMOE_OK) return st;
  const int T = shape->T, M = shape->M;
  hipError_t e = launch_mha_bwd_data(m, T, M, w_qkv, w_o, qkv, attn, lse, d_out, d_attn, d_qkv,
                                     delta, d_in, stream);
  if (e == hipSuccess)
    e = launch_mha_wgrad(T, M, 1, in, attn, d_out, d_qkv, dw_qkv, dw_o, accumulate != 0, ws,
                         stream);
  return hip_status(e, "flowmoe_mha_bwd");
}

}  // extern "C"

namespace {

struct Chunk {
  const char *x, *dy;
  float *logits, *w, *dw, *dl;
  int32_t *idx, *counts, *offsets, *slot, *row_src, *load;
  char *x_disp, *h_save, *a_save, *y_disp, *y, *dy_disp, *dx_disp, *dx;
  // the attention part of AT_r (null without it); xw: x as written by it
  const char* in;
  char *xw, *qkv, *attn, *d_attn, *d_qkv, *d_in;
  float *lse, *delta;
};

Chunk chunk_of(const Shape& s, const flowmoe_layer_bufs_t* b, int r) {
  const long es = (long)esize(s.dtype);
  const long T = s.T, M = s.M, E = s.E, k = s.k, rows = s.rows;
  const long HW = (s.act == FLOWMOE_SWIGLU) ? 2L * s.H : s.H;
  Chunk c;
  c.x = b->x ? cptr(b->x, r * T * M * es) : nullptr;
  c.dy = b->dy ? cptr(b->dy, r * T * M * es) : nullptr;
  c.logits = b->logits ? b->logits + r * T * E : nullptr;
  c.w = b->topk_w ? b->topk_w + r * T * k : nullptr;
  c.dw = b->d_topk_w ? b->d_topk_w + r * T * k : nullptr;
  c.dl = b->d_logits ? b->d_logits + r * T * E : nullptr;
  c.idx = b->topk_idx ? b->topk_idx + r * T * k : nullptr;
  c.counts = b->counts ? b->counts + r * E : nullptr;
  c.offsets = b->offsets ? b->offsets + r * (E + 1) : nullptr;
  c.slot = b->slot ? b->slot + r * T * k : nullptr;
  c.row_src = b->row_src ? b->row_src + r * rows : nullptr;
  c.load = b->load ? b->load + r * E : nullptr;
  c.x_disp = mptr(b->x_disp, r * rows * M * es);
  c.h_save = mptr(b->h_save, r * rows * HW * es);
  c.a_save = mptr(b->a_save, r * rows * (long)s.H * es);
  c.y_disp = mptr(b->y_disp, r * rows * M * es);
  c.y = mptr(b->y, r * T * M * es);
  c.dy_disp = mptr(b->dy_disp, r * rows * M * es);
  c.dx_disp = mptr(b->dx_disp, r * rows * M * es);
  c.dx = mptr(b->dx, r * T * M * es);
  const long heads = b->mha ? b->mha->heads : 0;
  c.in = b->mha_in ? cptr(b->mha_in, r * T * M * es) : nullptr;
  c.xw = mptr(b->x, r * T * M * es);
  c.qkv = mptr(b->qkv, r * T * 3 * M * es);
  c.attn = mptr(b->attn, r * T * M * es);
  c.d_attn = mptr(b->d_attn, r * T * M * es);
  c.d_qkv = mptr(b->d_qkv, r * T * 3 * M * es);
  c.d_in = mptr(b->d_in, r * T * M * es);
  c.lse = b->lse ? b->lse + r * heads * T : nullptr;
  c.delta = b->delta ? b->delta + r * heads * T : nullptr;
  return c;
}

struct Sched {
  hipStream_t sc, sm;
  bool two;
  hipEvent_t* trace;
  int R;
  hipError_t err = hipSuccess;
  void mark(int task, int r, int end, hipStream_t st) { mark_at(2 * (task * R + r) + end, st); }
  void mark_at(int i, hipStream_t st) {
    if (trace != nullptr && err == hipSuccess) err = hipEventRecord(trace[i], st);
  }
  void signal(hipEvent_t ev, hipStream_t st) {
    if (two && err == hipSuccess) err = hipEventRecord(ev, st);
  }
  void wait(hipStream_t st, hipEvent_t ev) {
    if (two && err == hipSuccess) err = hipStreamWaitEvent(st, ev, 0);
  }
  void run(hipError_t e) {
    if (err == hipSuccess) err = e;
  }
};

flowmoe_status_t check_layer(const flowmoe_shape_t* shape, int32_t R, const flowmoe_layer_bufs_t* b,
                             Shape* s) {
  flowmoe_status_t st = check_shape(shape, NEED_H | NEED_C, s);
  if (st != FLOWMOE_OK) return st;
  if (b == nullptr) return fail(FLOWMOE_ERR_INVALID, "bufs is null");
  if (R < 1) return fail(FLOWMOE_ERR_INVALID, "R = %d < 1", R);
  if ((long)R * s->T > (1L << 30)) return fail(FLOWMOE_ERR_UNSUPPORTED, "R*T too large");
  return FLOWMOE_OK;
}

// the attention part of AT_r: shape and buffers (forward; backward adds its own)
flowmoe_status_t check_layer_mha(const flowmoe_shape_t* shape, const flowmoe_layer_bufs_t* b,
                                 bool bwd, AttnShape* m) {
  flowmoe_status_t st = check_mha(shape, b->mha, m);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(b->w_qkv, "bufs->w_qkv");
  REQUIRE_T(b->w_o, "bufs->w_o");
  if (bwd) {
    REQUIRE_T(b->dw_qkv, "bufs->dw_qkv");
    REQUIRE_T(b->dw_o, "bufs->dw_o");
  }
  if (shape->T > 0) {
    REQUIRE_T(b->mha_in, "bufs->mha_in");
    REQUIRE_T(b->qkv, "bufs->qkv");
    REQUIRE_T(b->attn, "bufs->attn");
    REQUIRE_F(b->lse, "bufs->lse");
    if (bwd) {
      REQUIRE_T(b->d_attn, "bufs->d_attn");
      REQUIRE_T(b->d_qkv, "bufs->d_qkv");
      REQUIRE_F(b->delta, "bufs->delta");
      REQUIRE_T(b->d_in, "bufs->d_in");
    }
  }
  return FLOWMOE_OK;
}

}  // namespace

extern "C" {

flowmoe_status_t flowmoe_layer_fwd(const flowmoe_shape_t* shape, int32_t R,
                                   const flowmoe_layer_bufs_t* b, hipStream_t s_compute,
                                   hipStream_t s_comm, hipEvent_t* trace) {
  Shape s;
  flowmoe_status_t st = check_layer(shape, R, b, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(b->w_gate, "bufs->w_gate");
  REQUIRE_T(b->w1, "bufs->w1");
  REQUIRE_T(b->w2, "bufs->w2");
  REQUIRE(b->counts, "bufs->counts");
  REQUIRE(b->offsets, "bufs->offsets");
  if (s.act == FLOWMOE_SWIGLU) REQUIRE_T(b->w3, "bufs->w3");
  st = check_biases(s, b->b1, b->b3, b->b2, "bufs->");
  if (st != FLOWMOE_OK) return st;
  AttnShape am = {};
  if (b->mha != nullptr) {
    st = check_layer_mha(shape, b, false, &am);
    if (st != FLOWMOE_OK) return st;
  }
  if (b->ws != nullptr) {  // optional here: the dispatch scan's tile histograms
    st = check_ws(b->ws, b->ws_bytes, dispatch_ws_bytes(s), "flowmoe_layer_fwd");
    if (st != FLOWMOE_OK) return st;
  }
  if (s.T > 0) {
    REQUIRE_T(b->x, "bufs->x"); REQUIRE(b->logits, "bufs->logits");
    REQUIRE(b->topk_idx, "bufs->topk_idx"); REQUIRE(b->topk_w, "bufs->topk_w");
    REQUIRE(b->slot, "bufs->slot"); REQUIRE_T(b->y, "bufs->y");
  }
  if (s.rows > 0) {
    REQUIRE(b->row_src, "bufs->row_src"); REQUIRE_T(b->x_disp, "bufs->x_disp");
    REQUIRE_T(b->h_save, "bufs->h_save"); REQUIRE_T(b->a_save, "bufs->a_save");
    REQUIRE_T(b->y_disp, "bufs->y_disp");
  }
  // With one chunk there is no overlap to gain and each cross-stream event
  // wait costs several microseconds: one chunk runs on s_compute only.
  if (R == 1) s_comm = s_compute;
  Sched sc{s_compute, s_comm, s_comm != s_compute, trace, R};
  hipEvent_t* ev = nullptr;
  sc.run(get_events(3 * R + 2, &ev));
  if (sc.err != hipSuccess) return hip_status(sc.err, "flowmoe_layer_fwd events");
  hipEvent_t *evG = ev, *evD = ev + R, *evF = ev + 2 * R, evStart = ev[3 * R], evEnd = ev[3 * R + 1];
  sc.signal(evStart, s_compute);
  sc.wait(s_comm, evStart);
  // AT_1..AT_R on the compute stream: the chunk's attention (which writes
  // its x), then the gate
  for (int r = 0; r < R; ++r) {
    Chunk c = chunk_of(s, b, r);
    sc.mark(0, r, 0, s_compute);
    if (b->mha != nullptr)
      sc.run(launch_mha_fwd(am, s.T, s.M, c.in, b->w_qkv, b->w_o, c.qkv, c.attn, c.lse, c.xw,
                            s_compute));
    sc.run(launch_gate_topk(s, c.x, b->w_gate, b->bias, c.logits, c.idx, c.w, s_compute));
    sc.mark(0, r, 1, s_compute);
    sc.signal(evG[r], s_compute);
  }
  // D_1..D_R on the comm stream
  for (int r = 0; r < R; ++r) {
    Chunk c = chunk_of(s, b, r);
    sc.wait(s_comm, evG[r]);
    sc.mark(1, r, 0, s_comm);
    sc.run(launch_dispatch(s, c.idx, c.x, c.counts, c.offsets, c.slot, c.row_src, c.load, c.x_disp,
                           b->ws, s_comm));
    sc.mark(1, r, 1, s_comm);
    sc.signal(evD[r], s_comm);
  }
  // E_1..E_R on the compute stream
  for (int r = 0; r < R; ++r) {
    Chunk c = chunk_of(s, b, r);
    sc.wait(s_compute, evD[r]);
    sc.mark(2, r, 0, s_compute);
    sc.run(launch_expert_ffn(s, c.x_disp, c.counts, c.offsets, b->w1, b->w3, b->w2, b->b1, b->b3,
                             b->b2, c.h_save, c.a_save, c.y_disp, s_compute));
    sc.mark(2, r, 1, s_compute);
    sc.signal(evF[r], s_compute);
  }
  // C_1..C_R on the comm stream
  for (int r = 0; r < R; ++r) {
    Chunk c = chunk_of(s, b, r);
    sc.wait(s_comm, evF[r]);
    sc.mark(3, r, 0, s_comm);
    sc.run(launch_combine(s, c.y_disp, c.slot, c.w, c.y, s_comm));
    sc.mark(3, r, 1, s_comm);
  }
  sc.signal(evEnd, s_comm);
  sc.wait(s_compute, evEnd);
  return hip_status(sc.err, "flowmoe_layer_fwd");
}

flowmoe_status_t flowmoe_layer_bwd(const flowmoe_shape_t* shape, int32_t R,
                                   const flowmoe_layer_bufs_t* b, hipStream_t s_compute,
                                   hipStream_t s_comm, hipEvent_t* trace) {
  Shape s;
  flowmoe_status_t st = check_layer(shape, R, b, &s);
  if (st != FLOWMOE_OK) return st;
  REQUIRE_T(b->w_gate, "bufs->w_gate");
  REQUIRE_T(b->w1, "bufs->w1");
  REQUIRE_T(b->w2, "bufs->w2");
  REQUIRE(b->counts, "bufs->counts");
  REQUIRE(b->offsets, "bufs->offsets");
  REQUIRE(b->dw_gate, "bufs->dw_gate");
  REQUIRE(b->dw1, "bufs->dw1");
  REQUIRE(b->dw2, "bufs->dw2");
  if (s.act == FLOWMOE_SWIGLU) {
    REQUIRE_T(b->w3, "bufs->w3");
    REQUIRE(b->dw3, "bufs->dw3");
  }
  st = check_biases(s, b->db1, b->db3, b->db2, "bufs->d");
  if (st != FLOWMOE_OK) return st;
  AttnShape am = {};
  const bool mha = b->mha != nullptr;
  if (mha) {
    st = check_layer_mha(shape, b, true, &am);
    if (st != FLOWMOE_OK) return st;
  }
  if (s.T > 0) {
    REQUIRE_T(b->x, "bufs->x"); REQUIRE_T(b->dy, "bufs->dy"); REQUIRE(b->topk_idx, "bufs->topk_idx");
    REQUIRE(b->topk_w, "bufs->topk_w"); REQUIRE(b->slot, "bufs->slot");
    REQUIRE(b->d_topk_w, "bufs->d_topk_w"); REQUIRE(b->d_logits, "bufs->d_logits");
    REQUIRE_T(b->dx, "bufs->dx");
    if (s.gate == FLOWMOE_GATE_FULL) REQUIRE(b->logits, "bufs->logits");
  }
  if (s.rows > 0) {
    REQUIRE_T(b->x_disp, "bufs->x_disp"); REQUIRE_T(b->h_save, "bufs->h_save");
    REQUIRE_T(b->a_save, "bufs->a_save"); REQUIRE_T(b->y_disp, "bufs->y_disp");
    REQUIRE_T(b->dy_disp, "bufs->dy_disp"); REQUIRE_T(b->dx_disp, "bufs->dx_disp");
  }
  const size_t need =
      flowmoe_workspace_bytes(shape, mha ? FLOWMOE_WS_LAYER_BWD_MHA : FLOWMOE_WS_LAYER_BWD);
  st = check_ws(b->ws, b->ws_bytes, need, "flowmoe_layer_bwd");
  if (st != FLOWMOE_OK) return st;
  // One chunk: the gate's parameter gradients and the dispatch backward can
  // still run beside the expert backward's GEMMs. That pays when those GEMMs
  // take many rounds of the CUs (the small kernels then cost them little);
  // with a few rounds the kernels beside them delay whole rounds, and the
  // event waits cost more than the overlap gains (measured: 2.3% faster for
  // a 1.9e12 rows*M*H layer, 3% slower for 3.4e10), so small layers run on
  // s_compute only.
  if (R == 1 && (double)s.rows * s.M * s.H < 2.5e11) s_comm = s_compute;
  Sched sc{s_compute, s_comm, s_comm != s_compute, trace, R};
  hipEvent_t* ev = nullptr;
  sc.run(get_events(4 * R + 2, &ev));
  if (sc.err != hipSuccess) return hip_status(sc.err, "flowmoe_layer_bwd events");
  hipEvent_t *evC = ev, *evE = ev + R, *evD = ev + 3 * R + 2, evStart = ev[3 * R],
             evEnd = ev[3 * R + 1];
  sc.signal(evStart, s_compute);
  sc.wait(s_comm, evStart);
  // The gate's own gradients (d_logits, dW_g, db) need only the combine
  // backward's d_topk_w, so they run on the comm stream while the expert
  // backward occupies the compute stream; its dx term is fused into the
  // dispatch backward. The workspace holds the gate's partials (the expert
  // backward keeps dH in h_save).
  void* ws_gate = b->ws;
  // C_R..C_1 (combine backward) on the comm stream
  for (int r = R - 1; r >= 0; --r) {
    Chunk c = chunk_of(s, b, r);
    sc.mark(0, r, 0, s_comm);
    sc.run(launch_combine_bwd(s, c.dy, c.y_disp, c.slot, c.w, c.counts, c.offsets, c.dy_disp, c.dw,
                              s_comm));
    sc.mark(0, r, 1, s_comm);
    sc.signal(evC[r], s_comm);
  }
  // gate parameter gradients of AT_R..AT_1, summed over chunks in that order;
  // W_g^T for the dx term (the gate workspace keeps it at its front) comes
  // with the first chunk's dW_g reduce.
  // The full softmax gate's d_logits is dense: its dx term is a GEMM over
  // all E experts, run per chunk right after that chunk's d_logits (whose
  // bf16 copy the next chunk's overwrites) and stored into dx, to which D_r
  // then adds the experts' part
  const bool full = s.gate == FLOWMOE_GATE_FULL;
  // (the sparse gate's W_g^T comes from the first chunk's dW_g reduce launch)
  if (s.T > 0 && full) sc.run(launch_gate_wstack(s, b->w_gate, ws_gate, s_comm));
  for (int r = R - 1; r >= 0; --r) {
    Chunk c = chunk_of(s, b, r);
    sc.mark(3, r, 0, s_comm);
    sc.run(launch_gate_dw(s, c.x, c.logits, c.idx, c.w, c.dw, c.dl, b->dw_gate, b->dbias,
                          r != R - 1, ws_gate, s_comm,
                          (r == R - 1 && !full && s.T > 0 && !gate_grad_zero(s)) ? b->w_gate
                                                                                : nullptr));
    if (full) sc.run(launch_gate_dx_full(s, ws_gate, c.dx, false, s_comm));
    sc.mark(3, r, 1, s_comm);
  }
  // E_R..E_1 on the compute stream: each chunk's dH (written over its h_save)
  // and dX, which D_r waits for; the weight gradients, which nothing in the
  // layer waits for, once after E_1 over the rows of all chunks (one GEMM per
  // weight instead of R read-modify-write passes over the fp32 gradients)
  for (int r = R - 1; r >= 0; --r) {
    Chunk c = chunk_of(s, b, r);
    sc.wait(s_compute, evC[r]);
    sc.mark(1, r, 0, s_compute);
    sc.run(launch_expert_ffn_dgrad(s, c.dy_disp, c.h_save, c.counts, c.offsets, b->w1, b->w3,
                                   b->w2, c.h_save, c.dx_disp, s_compute));
    sc.mark(1, r, 1, s_compute);
    sc.signal(evE[r], s_compute);
  }
  sc.mark(4, 0, 0, s_compute);  // (the trace's last pair: the weight gradients)
  // (with two streams the experts' bias gradients, which read dY and dH
  // only, run on the comm stream after D_1, beside these GEMMs)
  sc.run(launch_expert_ffn_wgrad(s, R, b->dy_disp, b->x_disp, b->a_save, b->h_save, b->counts,
                                 b->offsets, b->dw1, b->dw3, b->dw2, sc.two ? nullptr : b->db1,
                                 sc.two ? nullptr : b->db3, sc.two ? nullptr : b->db2, 0,
                                 s_compute));
  sc.mark(4, 0, 1, s_compute);
  // D_R..D_1 (dispatch backward, plus the gate's dx term) on the comm stream
  for (int r = R - 1; r >= 0; --r) {
    Chunk c = chunk_of(s, b, r);
    sc.wait(s_comm, evE[r]);
    sc.mark(2, r, 0, s_comm);
    // (d_logits = 0 for one selected expert: the dispatch backward alone)
    sc.run(full ? launch_dispatch_bwd_add(s, c.dx_disp, c.slot, c.dx, s_comm)
           : gate_grad_zero(s)
               ? launch_dispatch_bwd(s, c.dx_disp, c.slot, c.dx, s_comm)
               : launch_dispatch_bwd_gate(s, c.dx_disp, c.slot, c.idx, c.w, c.dw,
                                          gate_ws_wgt(ws_gate), c.dx, s_comm));
    sc.mark(2, r, 1, s_comm);
    if (mha) sc.signal(evD[r], s_comm);
  }
  if (sc.two)  // (after D_1, which waited for E_1: every chunk's dH and dY are final)
    sc.run(launch_expert_bias_grad(s, R, b->dy_disp, b->h_save, b->counts, b->offsets, b->db1,
                                   b->db3, b->db2, 0, s_comm));
  // the attention part of AT_R..AT_1 on the compute stream, each after D_r
  // has completed its x gradient (dx: the attention output's gradient),
  // then its weight gradients over all chunks (one GEMM per weight)
  if (mha) {
    for (int r = R - 1; r >= 0; --r) {
      Chunk c = chunk_of(s, b, r);
      sc.wait(s_compute, evD[r]);
      sc.mark_at(8 * R + 2 + 2 * r, s_compute);
      sc.run(launch_mha_bwd_data(am, s.T, s.M, b->w_qkv, b->w_o, c.qkv, c.attn, c.lse, c.dx,
                                 c.d_attn, c.d_qkv, c.delta, c.d_in, s_compute));
      sc.mark_at(8 * R + 3 + 2 * r, s_compute);
    }
    sc.mark_at(10 * R + 2, s_compute);
    sc.run(launch_mha_wgrad(s.T, s.M, R, b->mha_in, b->attn, b->dx, b->d_qkv, b->dw_qkv, b->dw_o,
                            0, b->ws, s_compute));
    sc.mark_at(10 * R + 3, s_compute);
  }
  sc.signal(evEnd, s_comm);
  sc.wait(s_compute, evEnd);
  return hip_status(sc.err, "flowmoe_layer_bwd");
}

}  // extern "C"
