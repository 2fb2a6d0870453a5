// Gate (the AT_r gating part of Sec. 2.1 / Sec. 4.2): logits = x W_g (+ b),
// top-k selection with renormalised softmax weights, and the gate backward.
//
// Wavefront layout: experts are spread over a segment of EP lanes (EP = next
// power of two >= E, E <= 64); a 64-wide wave holds 64/EP segments, each
// working on its own tokens. Top-k is k rounds of a segmented butterfly
// argmax on (logit, -index), so ties go to the lower expert index and
// -0.0 == +0.0 (IEEE compare).
#include <math.h>

#include "common.hpp"

namespace flowmoe {
namespace {

constexpr int kGateThreads = 256;
constexpr int kGateLdsFloats = 8192;  // x staging budget: 32 KB of LDS

__host__ __device__ inline int pow2_at_least(int e) {
  int p = 1;
  while (p < e) p <<= 1;
  return p;
}

// Segmented argmax across EP lanes. Larger value wins; equal values go to the
// smaller index.
__device__ __forceinline__ void seg_argmax(float& v, int& i, int EP) {
  for (int off = EP >> 1; off > 0; off >>= 1) {
    float ov = __shfl_xor(v, off, 64);
    int oi = __shfl_xor(i, off, 64);
    if (ov > v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
}

// Select the top-k of one token's logits held one per lane (lane expert e,
// invalid lanes pass valid=false), then write idx/w. All EP lanes of the
// segment take part; the first k lanes write.
__device__ __forceinline__ void topk_write(float logit, int e, bool valid, int EP, int k,
                                           int32_t* idx_out, float* w_out) {
  float top_v[kMaxK];
  int top_i[kMaxK];
  float mine = valid ? logit : -INFINITY;
  int my_i = valid ? e : (1 << 20) + e;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      float v = mine;
      int i = my_i;
      seg_argmax(v, i, EP);
      top_v[j] = v;
      top_i[j] = i;
      if (i == my_i) {  // this lane was selected: remove it
        mine = -INFINITY;
        my_i = (1 << 21) + e;
      }
    }
  }
  // softmax over the k selected logits, shifted by the largest
  float denom = 0.f;
  float ex[kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      ex[j] = expf(top_v[j] - top_v[0]);
      denom += ex[j];
    }
  }
  const int lane_in_seg = e;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k && lane_in_seg == j) {
      idx_out[j] = top_i[j];
      w_out[j] = ex[j] / denom;
    }
  }
}

// Fused gate: per block 4 waves; each wave has G = 64/EP segments, each
// segment TPG tokens. x rows of the block are staged in LDS as float.
template <typename TIn>
__global__ __launch_bounds__(kGateThreads) void gate_topk_kernel(
    const TIn* __restrict__ x, const TIn* __restrict__ wg, const float* __restrict__ bias,
    float* __restrict__ logits, int32_t* __restrict__ idx, float* __restrict__ w, int T, int M,
    int E, int k, int EP, int TPG, int xchunk) {
  extern __shared__ float xs[];  // [tokens_per_block][xchunk]
  const int G = 64 / EP;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int seg = lane / EP, e = lane % EP;
  const int tpb = 4 * G * TPG;  // tokens per block
  const int t0 = blockIdx.x * tpb;
  // token slot of (wave, seg, i) inside the block: wave-major
  const int base_slot = (wave * G + seg) * TPG;
  const bool evalid = e < E;

  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;

  for (int m0 = 0; m0 < M; m0 += xchunk) {
    const int mc = min(xchunk, M - m0);
    __syncthreads();
    // stage x[t0 .. t0+tpb) [m0 .. m0+mc) as float
    for (int q = threadIdx.x; q < tpb * mc; q += kGateThreads) {
      int tt = q / mc, mm = q % mc;
      int t = t0 + tt;
      xs[tt * xchunk + mm] = (t < T) ? Elem<TIn>::load(x + (size_t)t * M + m0 + mm) : 0.f;
    }
    __syncthreads();
    if (evalid) {
      const TIn* wcol = wg + (size_t)m0 * E + e;
      for (int mm = 0; mm < mc; ++mm) {
        float wv = Elem<TIn>::load(wcol + (size_t)mm * E);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (i < TPG) acc[i] += xs[(base_slot + i) * xchunk + mm] * wv;
      }
    }
  }
  const float b = (bias != nullptr && evalid) ? bias[e] : 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i < TPG) {
      const int t = t0 + base_slot + i;
      if (t < T) {  // uniform across the segment
        float l = acc[i] + b;
        if (evalid) logits[(size_t)t * E + e] = l;
        topk_write(l, e, evalid, EP, k, idx + (size_t)t * k, w + (size_t)t * k);
      }
    }
  }
}

// bf16 gate on MFMA (v_mfma_f32_16x16x32_bf16): a block of 4 waves owns 64
// tokens, each wave 16 of them, against all experts padded to 16-column
// blocks. x rows feed the A operand straight from global memory (16 bytes of
// one row per lane); W_g chunks of kGateKC rows are staged in LDS transposed
// (expert-major, K-contiguous) for the B operand. The logits tile goes
// through LDS to the wavefront top-k.
constexpr int kGateKC = 128;          // K rows of W_g staged per step
constexpr int kGateTok = 64;          // tokens per block
constexpr int kGateWtStride = kGateKC + 8;  // bf16 elements per staged expert row

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void gate_topk_mfma_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg, const float* __restrict__ bias,
    float* __restrict__ logits, int32_t* __restrict__ idx, float* __restrict__ w, int T, int M,
    int E, int k, int EP) {
  __shared__ __attribute__((aligned(16))) bf16_t wt[kMaxE * kGateWtStride];
  __shared__ float lg[kGateTok][kMaxE + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int NB = (E + 15) >> 4;  // 16-expert column blocks
  const int t0 = blockIdx.x * kGateTok + wave * 16;
  const int arow = t0 + (lane & 15);          // token whose A row this lane feeds
  const int kq = (lane >> 4) * 8;             // k offset of this lane inside a 32-step
  const bool arow_ok = arow < T;
  const bf16_t* xrow = x + (long)(arow_ok ? arow : 0) * M;
  floatx4_t acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < M; k0 += kGateKC) {
    // A fragments of this chunk, issued before the staging barrier
    uint4 av[kGateKC / 32];
#pragma unroll
    for (int s = 0; s < kGateKC / 32; ++s) {
      const int kk = k0 + s * 32 + kq;
      av[s] = (arow_ok && kk < M) ? *reinterpret_cast<const uint4*>(xrow + kk) : make_uint4(0, 0, 0, 0);
    }
    __syncthreads();  // previous chunk's readers of wt are done
    const int rows = min(kGateKC, M - k0);
    for (int q = tid; q < kGateKC * NB * 16; q += 256) {
      const int kk = q / (NB * 16), e = q % (NB * 16);
      const bf16_t v = (kk < rows && e < E) ? wg[(long)(k0 + kk) * E + e] : (bf16_t)0;
      wt[e * kGateWtStride + kk] = v;
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kGateKC / 32; ++s) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, av[s]);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        if (nb < NB) {
          const bf16x8_t b = *reinterpret_cast<const bf16x8_t*>(
              &wt[(nb * 16 + (lane & 15)) * kGateWtStride + s * 32 + kq]);
          acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[nb], 0, 0, 0);
        }
      }
    }
  }
  // acc[nb][r]: token (lane/16)*4 + r of this wave, expert nb*16 + lane%16
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    if (nb < NB) {
      const int e = nb * 16 + (lane & 15);
      const float b = (bias != nullptr && e < E) ? bias[e] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tt = wave * 16 + (lane >> 4) * 4 + r;
        const float l = acc[nb][r] + b;
        if (e < E) {
          lg[tt][e] = l;
          const int t = blockIdx.x * kGateTok + tt;
          if (t < T) logits[(long)t * E + e] = l;
        }
      }
    }
  }
  __syncthreads();
  // top-k: segments of EP lanes, one token per segment per round
  const int G = 64 / EP;
  const int seg = lane / EP, e = lane % EP;
  const bool evalid = e < E;
  for (int i = seg; i < 16; i += G) {
    const int tt = wave * 16 + i;
    const int t = blockIdx.x * kGateTok + tt;
    if (t >= T) break;  // uniform across the segment
    const float l = evalid ? lg[tt][e] : 0.f;
    topk_write(l, e, evalid, EP, k, idx + (long)t * k, w + (long)t * k);
  }
}

__global__ __launch_bounds__(kGateThreads) void route_kernel(const float* __restrict__ logits,
                                                             int32_t* __restrict__ idx,
                                                             float* __restrict__ w, int T, int E,
                                                             int k, int EP) {
  const int G = 64 / EP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int seg = lane / EP, e = lane % EP;
  const int t = (blockIdx.x * 4 + wave) * G + seg;
  if (t >= T) return;  // uniform per segment
  const bool evalid = e < E;
  float l = evalid ? logits[(size_t)t * E + e] : 0.f;
  topk_write(l, e, evalid, EP, k, idx + (size_t)t * k, w + (size_t)t * k);
}

// ---- backward ---------------------------------------------------------------

// W_g (M x E, layer dtype) -> W_g^T (E x M, float) in the workspace
template <typename TIn>
__global__ void transpose_wg_kernel(const TIn* __restrict__ wg, float* __restrict__ wgt, int M,
                                    int E) {
  const long n = (long)M * E;
  for (long q = blockIdx.x * (long)blockDim.x + threadIdx.x; q < n; q += (long)gridDim.x * blockDim.x) {
    const int e = (int)(q / M), m = (int)(q % M);
    wgt[q] = Elem<TIn>::load(wg + (size_t)m * E + e);
  }
}

// One wave per token: d_logits row, and optionally dx[t] += dl W_g^T.
template <typename TIn>
__global__ __launch_bounds__(256) void gate_bwd_token_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, const float* __restrict__ dw,
    const float* __restrict__ wgt, float* __restrict__ d_logits, TIn* __restrict__ dx, int T,
    int M, int E, int k) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  float wj[kMaxK], dl[kMaxK];
  int ij[kMaxK];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      wj[j] = w[(size_t)t * k + j];
      ij[j] = idx[(size_t)t * k + j];
      s += wj[j] * dw[(size_t)t * k + j];
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j)
    if (j < k) dl[j] = wj[j] * (dw[(size_t)t * k + j] - s);
  for (int e = lane; e < E; e += 64) {
    float v = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k && ij[j] == e) v = dl[j];
    d_logits[(size_t)t * E + e] = v;
  }
  if (dx == nullptr) return;
  // M is a multiple of 8 (checked on the host)
  TIn* row = dx + (size_t)t * M;
  for (int m = lane * 8; m < M; m += 64 * 8) {
    float v[8];
    load8(row + m, v);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        const float* wr = wgt + (size_t)ij[j] * M + m;
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] += dl[j] * wr[q];
      }
    }
    store8(row + m, v);
  }
}

// dW_g partials: block (m-tile of 256 rows of x^T plus the bias row, split s).
// Row m == M is the bias row (x = 1). P[s][m][e], m in [0, M].
template <typename TIn, int EP>
__global__ __launch_bounds__(256) void gate_bwd_dw_partial_kernel(
    const TIn* __restrict__ x, const float* __restrict__ d_logits, float* __restrict__ P, int T,
    int M, int E, int tokens_per_split) {
  __shared__ float dls[64][EP];
  const int m = blockIdx.x * 256 + threadIdx.x;
  const int s = blockIdx.y;
  const int tb = s * tokens_per_split, te = min(T, tb + tokens_per_split);
  float acc[EP];
#pragma unroll
  for (int e = 0; e < EP; ++e) acc[e] = 0.f;
  for (int c0 = tb; c0 < te; c0 += 64) {
    const int n = min(64, te - c0);
    __syncthreads();
    for (int q = threadIdx.x; q < 64 * EP; q += 256) {
      int tt = q / EP, e = q % EP;
      dls[tt][e] = (tt < n && e < E) ? d_logits[(size_t)(c0 + tt) * E + e] : 0.f;
    }
    __syncthreads();
    if (m <= M) {
      for (int tt = 0; tt < n; ++tt) {
        const float xv = (m < M) ? Elem<TIn>::load(x + (size_t)(c0 + tt) * M + m) : 1.0f;
#pragma unroll
        for (int e = 0; e < EP; ++e) acc[e] += xv * dls[tt][e];
      }
    }
  }
  if (m <= M) {
    float* out = P + ((size_t)s * (M + 1) + m) * E;
    for (int e = 0; e < E; ++e) out[e] = acc[e];
  }
}

__global__ void gate_bwd_dw_reduce_kernel(const float* __restrict__ P, float* __restrict__ dw_gate,
                                          float* __restrict__ dbias, int M, int E, int S,
                                          int accumulate) {
  const long n = (long)(M + 1) * E;
  for (long q = blockIdx.x * (long)blockDim.x + threadIdx.x; q < n; q += (long)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < S; ++s) v += P[(size_t)s * n + q];
    const int m = (int)(q / E);
    if (m < M) {
      dw_gate[q] = accumulate ? dw_gate[q] + v : v;
    } else if (dbias != nullptr) {
      const int e = (int)(q % E);
      dbias[e] = accumulate ? dbias[e] + v : v;
    }
  }
}

int gate_splits(const Shape& s) {
  // enough blocks to fill the chip, at least 64 tokens per split
  int by_tokens = (s.T + 63) / 64;
  int sp = 64;
  if (sp > by_tokens) sp = by_tokens;
  return sp < 1 ? 1 : sp;
}

}  // namespace

hipError_t launch_gate_topk(const Shape& s, const void* x, const void* w_gate, const float* bias,
                            float* logits, int32_t* idx, float* w, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int EP = pow2_at_least(s.E);
  if (s.dtype == FLOWMOE_BF16) {
    const int blocks = (s.T + kGateTok - 1) / kGateTok;
    return traced(FLOWMOE_K_GATE, st, [&] {
      hipLaunchKernelGGL(gate_topk_mfma_kernel, dim3(blocks), dim3(256), 0, st, (const bf16_t*)x,
                         (const bf16_t*)w_gate, bias, logits, idx, w, s.T, s.M, s.E, s.k, EP);
    });
  }
  const int G = 64 / EP;
  const int TPG = G >= 8 ? 1 : 8 / G;
  const int tpb = 4 * G * TPG;
  const int blocks = (s.T + tpb - 1) / tpb;
  int xchunk = kGateLdsFloats / tpb;
  if (xchunk > 256) xchunk = 256;
  const size_t lds = (size_t)tpb * xchunk * sizeof(float);
  return traced(FLOWMOE_K_GATE, st, [&] {
    hipLaunchKernelGGL(gate_topk_kernel<float>, dim3(blocks), dim3(kGateThreads), lds, st,
                       (const float*)x, (const float*)w_gate, bias, logits, idx, w, s.T, s.M,
                       s.E, s.k, EP, TPG, xchunk);
  });
}

hipError_t launch_route(const Shape& s, const float* logits, int32_t* idx, float* w, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int EP = pow2_at_least(s.E);
  const int per_block = 4 * (64 / EP);
  const int blocks = (s.T + per_block - 1) / per_block;
  return traced(FLOWMOE_K_ROUTE, st, [&] {
    hipLaunchKernelGGL(route_kernel, dim3(blocks), dim3(kGateThreads), 0, st, logits, idx, w, s.T,
                       s.E, s.k, EP);
  });
}

size_t gate_bwd_ws_bytes(const Shape& s) {
  const size_t wgt = align256((size_t)s.M * s.E * sizeof(float));
  const size_t part = align256((size_t)gate_splits(s) * (s.M + 1) * s.E * sizeof(float));
  return wgt + part;
}

hipError_t launch_gate_bwd(const Shape& s, const void* x, const void* w_gate, const int32_t* idx,
                           const float* w, const float* dw, float* d_logits, float* dw_gate,
                           float* dbias, void* dx, int accumulate, void* ws, hipStream_t st) {
  float* wgt = static_cast<float*>(ws);
  float* P = reinterpret_cast<float*>(static_cast<char*>(ws) +
                                      align256((size_t)s.M * s.E * sizeof(float)));
  const bool bf = s.dtype == FLOWMOE_BF16;
  const int S = gate_splits(s);
  hipError_t e = hipSuccess;
  if (s.T > 0) {
    if (dx != nullptr) {
      const int nb = (int)(((long)s.M * s.E + 255) / 256);
      e = traced(FLOWMOE_K_GATE_BWD_WT, st, [&] {
        if (bf)
          hipLaunchKernelGGL(transpose_wg_kernel<bf16_t>, dim3(nb), dim3(256), 0, st,
                             (const bf16_t*)w_gate, wgt, s.M, s.E);
        else
          hipLaunchKernelGGL(transpose_wg_kernel<float>, dim3(nb), dim3(256), 0, st,
                             (const float*)w_gate, wgt, s.M, s.E);
      });
      if (e != hipSuccess) return e;
    }
    const int tb = (s.T + 3) / 4;
    e = traced(FLOWMOE_K_GATE_BWD_TOKEN, st, [&] {
      if (bf)
        hipLaunchKernelGGL(gate_bwd_token_kernel<bf16_t>, dim3(tb), dim3(256), 0, st, idx, w, dw,
                           wgt, d_logits, (bf16_t*)dx, s.T, s.M, s.E, s.k);
      else
        hipLaunchKernelGGL(gate_bwd_token_kernel<float>, dim3(tb), dim3(256), 0, st, idx, w, dw,
                           wgt, d_logits, (float*)dx, s.T, s.M, s.E, s.k);
    });
    if (e != hipSuccess) return e;
    const int tps = (s.T + S - 1) / S;
    dim3 grid((s.M + 1 + 255) / 256, S);
    const int EP = pow2_at_least(s.E);
    e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
#define FLOWMOE_DW_LAUNCH(EPV)                                                                   \
  if (bf)                                                                                        \
    hipLaunchKernelGGL((gate_bwd_dw_partial_kernel<bf16_t, EPV>), grid, dim3(256), 0, st,        \
                       (const bf16_t*)x, d_logits, P, s.T, s.M, s.E, tps);                       \
  else                                                                                           \
    hipLaunchKernelGGL((gate_bwd_dw_partial_kernel<float, EPV>), grid, dim3(256), 0, st,         \
                       (const float*)x, d_logits, P, s.T, s.M, s.E, tps);
      if (EP <= 8) {
        FLOWMOE_DW_LAUNCH(8)
      } else if (EP <= 16) {
        FLOWMOE_DW_LAUNCH(16)
      } else if (EP <= 32) {
        FLOWMOE_DW_LAUNCH(32)
      } else {
        FLOWMOE_DW_LAUNCH(64)
      }
#undef FLOWMOE_DW_LAUNCH
    });
    if (e != hipSuccess) return e;
  }
  const long n = (long)(s.M + 1) * s.E;
  const int nb = (int)((n + 255) / 256);
  if (s.T == 0 && accumulate) return hipSuccess;
  // with no tokens the gradient is zero: a reduce over zero splits writes it
  const int splits = s.T > 0 ? S : 0;
  const int acc = s.T > 0 ? accumulate : 0;
  return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
    hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(nb), dim3(256), 0, st, P, dw_gate, dbias,
                       s.M, s.E, splits, acc);
  });
}

}  // namespace flowmoe
