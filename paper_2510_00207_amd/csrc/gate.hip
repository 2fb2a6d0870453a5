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

// bf16 gate on MFMA (v_mfma_f32_16x16x32_bf16). A block of 4 waves owns 16
// tokens; the reduction over M is split between the waves (wave w takes the
// 32-deep k steps s = w, w + 4, ...), so every wave has its x loads in flight
// at once: the kernel reads x in about one memory round trip. x rows feed the
// A operand straight from global memory (16 bytes of one row per lane). W_g
// rows are copied into LDS in chunks of KC rows (as stored, [k][E], one
// contiguous range) and each lane gathers its B fragment (8 consecutive k of
// one expert) with 2-byte LDS reads. The four partial logit tiles are summed
// in LDS in wave order (deterministic), the bias added, and each token's
// top-k taken by a segment of EP lanes.
constexpr int kGateTok = 16;            // tokens per block
constexpr int kGateWgBytes = 32768;     // LDS for one chunk of W_g rows
constexpr int kGateBatch = 8;           // x loads in flight per lane

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

// rows of W_g per LDS chunk: a multiple of 32 (whole k steps)
__host__ __device__ inline int gate_chunk_rows(int E) {
  int kc = kGateWgBytes / (2 * E);
  return kc - kc % 32;
}

template <int NB>  // 16-expert column blocks (E <= 16 * NB)
__global__ __launch_bounds__(256) void gate_topk_mfma_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg, const float* __restrict__ bias,
    float* __restrict__ logits, int32_t* __restrict__ idx, float* __restrict__ w, int T, int M,
    int E, int k, int EP) {
  __shared__ __attribute__((aligned(16))) bf16_t wgs[kGateWgBytes / 2];
  __shared__ float part[4][kGateTok][NB * 16 + 1];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t0 = blockIdx.x * kGateTok;
  const int arow = t0 + (lane & 15);  // token whose A row this lane feeds
  const int kq = (lane >> 4) * 8;     // k offset of this lane inside a step
  const bool arow_ok = arow < T;
  const bf16_t* xrow = x + (long)(arow_ok ? arow : 0) * M;
  const int KC = gate_chunk_rows(E);

  floatx4_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < M; k0 += KC) {
    const int kc = min(KC, M - k0);
    const int s_end = (k0 + kc + 31) / 32;  // k steps of this chunk: [k0/32, s_end)
    int s = k0 / 32 + wave;
    // this wave's first batch of x fragments, issued before the staging barrier
    uint4 av[kGateBatch];
    auto load_batch = [&](int s0) {
#pragma unroll
      for (int i = 0; i < kGateBatch; ++i) {
        const int kk = (s0 + 4 * i) * 32 + kq;
        av[i] = (arow_ok && s0 + 4 * i < s_end && kk < M)
                    ? *reinterpret_cast<const uint4*>(xrow + kk)
                    : make_uint4(0, 0, 0, 0);
      }
    };
    load_batch(s);
    __syncthreads();  // previous chunk's readers of wgs are done
    {
      // rows [k0, k0 + kc) of W_g are one contiguous range of kc * E values;
      // kc and M are multiples of 8, so it is a whole number of 16-byte units
      const uint4* src = reinterpret_cast<const uint4*>(wg + (long)k0 * E);
      uint4* dst = reinterpret_cast<uint4*>(wgs);
      const int n16 = kc * E / 8;  // <= 8 per thread (32 KB)
      uint4 tmp[kGateWgBytes / 16 / 256];
#pragma unroll
      for (int i = 0; i < kGateWgBytes / 16 / 256; ++i)
        if (tid + 256 * i < n16) tmp[i] = src[tid + 256 * i];
#pragma unroll
      for (int i = 0; i < kGateWgBytes / 16 / 256; ++i)
        if (tid + 256 * i < n16) dst[tid + 256 * i] = tmp[i];
    }
    __syncthreads();
    for (; s < s_end; s += 4 * kGateBatch) {
#pragma unroll
      for (int i = 0; i < kGateBatch; ++i) {
        const int si = s + 4 * i;
        if (si < s_end) {
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, av[i]);
          const int r0 = si * 32 - k0 + kq;  // first W_g row of this lane's fragment
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const int e = nb * 16 + (lane & 15);
            uint32_t u[4] = {0u, 0u, 0u, 0u};
            if (e < E) {
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int ra = r0 + 2 * q, rb = ra + 1;
                const uint32_t lo = (ra < kc) ? wgs[ra * E + e] : 0u;
                const uint32_t hi = (rb < kc) ? wgs[rb * E + e] : 0u;
                u[q] = lo | (hi << 16);
              }
            }
            const bf16x8_t b = __builtin_bit_cast(bf16x8_t, make_uint4(u[0], u[1], u[2], u[3]));
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[nb], 0, 0, 0);
          }
        }
      }
      if (s + 4 * kGateBatch < s_end) load_batch(s + 4 * kGateBatch);
    }
  }
  // acc[nb][r]: token (lane / 16) * 4 + r, expert nb * 16 + lane % 16
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 4; ++r) part[wave][(lane >> 4) * 4 + r][nb * 16 + (lane & 15)] = acc[nb][r];
  __syncthreads();
  // sum the four partial tiles in wave order; bias; logits out
  for (int q = tid; q < kGateTok * E; q += 256) {
    const int tt = q / E, e = q % E;
    float l = part[0][tt][e] + part[1][tt][e];
    l += part[2][tt][e];
    l += part[3][tt][e];
    if (bias != nullptr) l += bias[e];
    part[0][tt][e] = l;
    if (t0 + tt < T) logits[(long)(t0 + tt) * E + e] = l;
  }
  __syncthreads();
  // top-k: segments of EP lanes, one token per segment per round
  const int G = 64 / EP;
  const int seg = lane / EP, e = lane % EP;
  const bool evalid = e < E;
  for (int i = wave * G + seg; i < kGateTok; i += 4 * G) {
    const int t = t0 + i;
    if (t >= T) break;  // uniform across the segment
    const float l = evalid ? part[0][i][e] : 0.f;
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
//
// dl_{t, S_t[j]} = w_j (dw_j - sum_j' w_j' dw_j') and 0 off S_t (the Jacobian
// of the softmax over the k selected logits); dW_g = x^T dl, db = sum_t dl_t,
// dx_t += dl_t W_g^T.

// dl of one token for its k selected experts
__device__ __forceinline__ void token_dl(const int32_t* __restrict__ idx, const float* __restrict__ w,
                                         const float* __restrict__ dw, long t, int k,
                                         int (&ij)[kMaxK], float (&dl)[kMaxK]) {
  float wj[kMaxK], dwj[kMaxK];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      ij[j] = idx[t * k + j];
      wj[j] = w[t * k + j];
      dwj[j] = dw[t * k + j];
      s += wj[j] * dwj[j];
    } else {
      ij[j] = -1;
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) dl[j] = (j < k) ? wj[j] * (dwj[j] - s) : 0.f;
}

// W_g (M x E, layer dtype) -> W_g^T (E x M, float), so that the dx term reads
// 8 consecutive m of one expert as two 16-byte vectors
template <typename TIn>
__global__ __launch_bounds__(256) void transpose_wg_kernel(const TIn* __restrict__ wg,
                                                           float* __restrict__ wgt, int M, int E) {
  const long n = (long)M * E;
  for (long q = blockIdx.x * 256L + threadIdx.x; q < n; q += (long)gridDim.x * 256) {
    const int e = (int)(q / M), m = (int)(q % M);
    wgt[q] = Elem<TIn>::load(wg + (long)m * E + e);
  }
}

// dx[t] += dl_t W_g^T, one wave per token
template <typename TIn>
__global__ __launch_bounds__(256) void gate_bwd_dx_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, const float* __restrict__ dw,
    const float* __restrict__ wgt, TIn* __restrict__ dx, int T, int M, int k) {
  const int lane = threadIdx.x & 63;
  const long t = blockIdx.x * 4L + (threadIdx.x >> 6);
  if (t >= T) return;
  int ij[kMaxK];
  float dl[kMaxK];
  token_dl(idx, w, dw, t, k, ij, dl);
  TIn* row = dx + t * M;
  for (int m = lane * 8; m < M; m += 64 * 8) {  // M is a multiple of 8
    float v[8];
    load8(row + m, v);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        float g[8];
        load8(wgt + (long)ij[j] * M + m, g);
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] += dl[j] * g[q];
      }
    }
    store8(row + m, v);
  }
}

// dW_g partials. Block (m tile of 64 columns of x, token split s); thread
// (mg: 8 consecutive m, eg: 8 consecutive experts, tl: token lane) holds an
// 8 x 8 tile and walks the split's tokens t = tl, tl + TL, ...; the TL lanes
// are summed in LDS in lane order. P[s][m][e] for m < M; Pb[s][e] = sum of dl
// (the bias row) from the blocks of m tile 0, which also write d_logits.
template <typename TIn, int EG>
__global__ __launch_bounds__(256) void gate_bwd_dw_kernel(
    const TIn* __restrict__ x, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const float* __restrict__ dw, float* __restrict__ d_logits, float* __restrict__ P,
    float* __restrict__ Pb, int T, int M, int E, int k, int tokens_per_split) {
  constexpr int TL = 32 / EG;
  constexpr int NE = 8 * EG;  // experts covered by the block
  __shared__ float red[TL][64 + 1][NE];
  const int tid = threadIdx.x;
  const int mg = tid & 7, eg = (tid >> 3) % EG, tl = tid / (8 * EG);
  const int m0 = blockIdx.x * 64 + mg * 8;
  const int e0 = eg * 8;
  const int s = blockIdx.y;
  const long tb = (long)s * tokens_per_split;
  const long te = min((long)T, tb + tokens_per_split);
  const bool first_tile = blockIdx.x == 0;
  float acc[8][8], accb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    accb[i] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  }
  // tokens in batches of 4: every load of a batch is in flight together
  constexpr int TB = 4;
  for (long t0 = tb + tl; t0 < te; t0 += TB * TL) {
    float xv[TB][8], d[TB][8];
#pragma unroll
    for (int u = 0; u < TB; ++u) {
      const long t = t0 + u * TL;
#pragma unroll
      for (int q = 0; q < 8; ++q) xv[u][q] = d[u][q] = 0.f;
      if (t < te) {
        int ij[kMaxK];
        float dlk[kMaxK];
        token_dl(idx, w, dw, t, k, ij, dlk);
#pragma unroll
        for (int q = 0; q < 8; ++q)
#pragma unroll
          for (int j = 0; j < kMaxK; ++j)
            if (ij[j] == e0 + q) d[u][q] = dlk[j];
        if (m0 < M) load8(x + t * M + m0, xv[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < TB; ++u) {
      const long t = t0 + u * TL;
      if (t >= te) break;
      if (first_tile && mg == 0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (e0 + q < E) d_logits[t * E + e0 + q] = d[u][q];
          accb[q] += d[u][q];
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[i][q] += xv[u][i] * d[u][q];
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) red[tl][mg * 8 + i][e0 + q] = acc[i][q];
  if (first_tile && mg == 0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) red[tl][64][e0 + q] = accb[q];
  }
  __syncthreads();
  const int rows = first_tile ? 65 : 64;
  for (int q = tid; q < rows * NE; q += 256) {
    const int mm = q / NE, e = q % NE;
    if (e >= E) continue;
    float v = 0.f;
    for (int l = 0; l < TL; ++l) v += red[l][mm][e];
    if (mm == 64) {
      Pb[(long)s * E + e] = v;
    } else {
      const int m = blockIdx.x * 64 + mm;
      if (m < M) P[((long)s * M + m) * E + e] = v;
    }
  }
}

// dW_g[m][e] = sum over splits of P (split order), db likewise
__global__ __launch_bounds__(256) void gate_bwd_dw_reduce_kernel(
    const float* __restrict__ P, const float* __restrict__ Pb, float* __restrict__ dw_gate,
    float* __restrict__ dbias, int M, int E, int S, int accumulate) {
  const long n = (long)M * E;
  const long q = blockIdx.x * 256L + threadIdx.x;
  if (q >= n + E) return;
  if (q < n) {
    float v = 0.f;
#pragma unroll 8
    for (int s = 0; s < S; ++s) v += P[(long)s * n + q];
    dw_gate[q] = accumulate ? dw_gate[q] + v : v;
  } else if (q < n + E && dbias != nullptr) {
    const int e = (int)(q - n);
    float v = 0.f;
    for (int s = 0; s < S; ++s) v += Pb[(long)s * E + e];
    dbias[e] = accumulate ? dbias[e] + v : v;
  }
}

int gate_eg(int E) { return E <= 8 ? 1 : E <= 16 ? 2 : E <= 32 ? 4 : 8; }

// token splits: about two blocks per CU over the m tiles, at least one token
// per token lane
int gate_splits(const Shape& s) {
  const int mtiles = (s.M + 63) / 64;
  const int tl = 32 / gate_eg(s.E);
  int sp = (512 + mtiles - 1) / mtiles;
  const int by_tokens = (s.T + tl - 1) / tl;
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
    const int NB = (s.E + 15) / 16;
    return traced(FLOWMOE_K_GATE, st, [&] {
#define FLOWMOE_GATE_LAUNCH(NBV)                                                                  \
  hipLaunchKernelGGL(gate_topk_mfma_kernel<NBV>, dim3(blocks), dim3(256), 0, st,                  \
                     (const bf16_t*)x, (const bf16_t*)w_gate, bias, logits, idx, w, s.T, s.M, s.E, \
                     s.k, EP)
      if (NB == 1) FLOWMOE_GATE_LAUNCH(1);
      else if (NB == 2) FLOWMOE_GATE_LAUNCH(2);
      else if (NB == 3) FLOWMOE_GATE_LAUNCH(3);
      else FLOWMOE_GATE_LAUNCH(4);
#undef FLOWMOE_GATE_LAUNCH
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

// workspace: [W_g^T (E x M float) | P (S x M x E) | Pb (S x E)]
size_t gate_wt_bytes(const Shape& s) { return align256((size_t)s.M * s.E * sizeof(float)); }

size_t gate_bwd_ws_bytes(const Shape& s) {
  const int S = gate_splits(s);
  return gate_wt_bytes(s) + align256((size_t)S * s.M * s.E * sizeof(float)) +
         align256((size_t)S * s.E * sizeof(float));
}

hipError_t launch_gate_wt(const Shape& s, const void* w_gate, void* ws, hipStream_t st) {
  float* wgt = static_cast<float*>(ws);
  const long n = (long)s.M * s.E;
  const int nb = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  return traced(FLOWMOE_K_GATE_BWD_WT, st, [&] {
    if (s.dtype == FLOWMOE_BF16)
      hipLaunchKernelGGL(transpose_wg_kernel<bf16_t>, dim3(nb), dim3(256), 0, st,
                         (const bf16_t*)w_gate, wgt, s.M, s.E);
    else
      hipLaunchKernelGGL(transpose_wg_kernel<float>, dim3(nb), dim3(256), 0, st,
                         (const float*)w_gate, wgt, s.M, s.E);
  });
}

hipError_t launch_gate_dx(const Shape& s, const int32_t* idx, const float* w, const float* dw,
                          const float* wgt, void* dx, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int tb = (s.T + 3) / 4;
  return traced(FLOWMOE_K_GATE_BWD_TOKEN, st, [&] {
    if (s.dtype == FLOWMOE_BF16)
      hipLaunchKernelGGL(gate_bwd_dx_kernel<bf16_t>, dim3(tb), dim3(256), 0, st, idx, w, dw, wgt,
                         (bf16_t*)dx, s.T, s.M, s.k);
    else
      hipLaunchKernelGGL(gate_bwd_dx_kernel<float>, dim3(tb), dim3(256), 0, st, idx, w, dw, wgt,
                         (float*)dx, s.T, s.M, s.k);
  });
}

hipError_t launch_gate_dw(const Shape& s, const void* x, const int32_t* idx, const float* w,
                          const float* dw, float* d_logits, float* dw_gate, float* dbias,
                          int accumulate, void* ws, hipStream_t st) {
  const int S = gate_splits(s);
  float* P = reinterpret_cast<float*>(static_cast<char*>(ws) + gate_wt_bytes(s));
  float* Pb = reinterpret_cast<float*>(reinterpret_cast<char*>(P) +
                                       align256((size_t)S * s.M * s.E * sizeof(float)));
  const bool bf = s.dtype == FLOWMOE_BF16;
  if (s.T > 0) {
    const int tps = (s.T + S - 1) / S;
    const dim3 grid((s.M + 63) / 64, S);
    const int EG = gate_eg(s.E);
    hipError_t e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
#define FLOWMOE_DW_LAUNCH(EGV)                                                                   \
  if (bf)                                                                                        \
    hipLaunchKernelGGL((gate_bwd_dw_kernel<bf16_t, EGV>), grid, dim3(256), 0, st,                \
                       (const bf16_t*)x, idx, w, dw, d_logits, P, Pb, s.T, s.M, s.E, s.k, tps);  \
  else                                                                                           \
    hipLaunchKernelGGL((gate_bwd_dw_kernel<float, EGV>), grid, dim3(256), 0, st,                 \
                       (const float*)x, idx, w, dw, d_logits, P, Pb, s.T, s.M, s.E, s.k, tps);
      if (EG == 1) {
        FLOWMOE_DW_LAUNCH(1)
      } else if (EG == 2) {
        FLOWMOE_DW_LAUNCH(2)
      } else if (EG == 4) {
        FLOWMOE_DW_LAUNCH(4)
      } else {
        FLOWMOE_DW_LAUNCH(8)
      }
#undef FLOWMOE_DW_LAUNCH
    });
    if (e != hipSuccess) return e;
  }
  if (s.T == 0 && accumulate) return hipSuccess;
  // with no tokens the gradient is zero: a reduce over zero splits writes it
  const int splits = s.T > 0 ? S : 0;
  const int acc = s.T > 0 ? accumulate : 0;
  const long n = (long)s.M * s.E + s.E;
  const int nb = (int)((n + 255) / 256);
  return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
    hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(nb), dim3(256), 0, st, P, Pb, dw_gate,
                       dbias, s.M, s.E, splits, acc);
  });
}

hipError_t launch_gate_bwd(const Shape& s, const void* x, const void* w_gate, const int32_t* idx,
                           const float* w, const float* dw, float* d_logits, float* dw_gate,
                           float* dbias, void* dx, int accumulate, void* ws, hipStream_t st) {
  hipError_t e = launch_gate_dw(s, x, idx, w, dw, d_logits, dw_gate, dbias, accumulate, ws, st);
  if (e != hipSuccess || dx == nullptr || s.T == 0) return e;
  e = launch_gate_wt(s, w_gate, ws, st);
  if (e != hipSuccess) return e;
  return launch_gate_dx(s, idx, w, dw, gate_ws_wgt(ws), dx, st);
}

}  // namespace flowmoe
