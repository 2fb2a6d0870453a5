// Dispatch (D_r) and combine (C_r) of Sec. 2.1, with their backward.
//
// route_scan: capacity-bounded positions in the priority order "every first
//   choice, then every second choice, ..., ascending token within a rank",
//   i.e. a stable counting sort of the sequence s = j*T + t by expert. One
//   1024-thread workgroup walks the sequence in tiles; inside a wave, lanes
//   with the same expert are matched with 6 ballots (E <= 64), giving each
//   lane its rank among equal experts; per-expert wave counts are scanned in
//   LDS across the 16 waves and carried across tiles.
// gather / combine / scatter kernels move whole rows with 16-byte vectors,
//   one wave per row or token, accumulating in float in a fixed order.
#include "common.hpp"

namespace flowmoe {
namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / 64;

__global__ __launch_bounds__(kScanThreads) void route_scan_kernel(
    const int32_t* __restrict__ idx, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ slot, int32_t* __restrict__ row_src, int32_t* __restrict__ load, int T,
    int k, int E, int C, int padded, long rows) {
  __shared__ int wcnt[kScanWaves][kMaxE];
  __shared__ int running[kMaxE];
  __shared__ int offs[kMaxE + 1];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

  for (long r = tid; r < rows; r += kScanThreads) row_src[r] = -1;
  if (tid < kMaxE) running[tid] = 0;

  const long n = (long)T * k;
  // pass 1: positions
  for (long base = 0; base < n; base += kScanThreads) {
    __syncthreads();  // previous tile's readers of wcnt are done
    for (int q = tid; q < kScanWaves * kMaxE; q += kScanThreads) (&wcnt[0][0])[q] = 0;
    __syncthreads();
    const long s = base + tid;
    bool valid = s < n;
    int t = 0, j = 0, e = 0;
    if (valid) {
      j = (int)(s / T);
      t = (int)(s - (long)j * T);
      e = idx[(long)t * k + j];
      if ((unsigned)e >= (unsigned)E) {  // not an expert id: never kept
        valid = false;
        e = 0;
      }
    }
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 6; ++b) {
      const uint64_t m = __ballot(valid && ((e >> b) & 1));
      same &= ((e >> b) & 1) ? m : ~m;
    }
    const int rank = __popcll(same & lt_mask);
    if (valid && rank == 0) wcnt[wave][e] = __popcll(same);
    __syncthreads();
    if (tid < E) {
      int run = running[tid];
      for (int w = 0; w < kScanWaves; ++w) {
        const int c = wcnt[w][tid];
        wcnt[w][tid] = run;
        run += c;
      }
      running[tid] = run;
    }
    __syncthreads();
    if (valid) slot[(long)t * k + j] = wcnt[wave][e] + rank;
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int e = 0; e < E; ++e) {
      offs[e] = padded ? e * C : acc;
      acc += min(running[e], C);
    }
    offs[E] = padded ? E * C : acc;
  }
  __syncthreads();
  if (tid < E) {
    counts[tid] = min(running[tid], C);
    if (load != nullptr) load[tid] = running[tid];
  }
  if (tid <= E) offsets[tid] = offs[tid];
  __threadfence_block();
  __syncthreads();
  // pass 2: rows (each thread revisits exactly the elements it wrote)
  for (long base = 0; base < n; base += kScanThreads) {
    const long s = base + tid;
    if (s < n) {
      const int j = (int)(s / T);
      const int t = (int)(s - (long)j * T);
      const long a = (long)t * k + j;
      const int e = idx[a];
      const int pos = ((unsigned)e < (unsigned)E) ? slot[a] : C;
      if (pos < C) {
        const int r = offs[e] + pos;
        slot[a] = r;
        row_src[r] = (int)a;
      } else {
        slot[a] = -1;
      }
    }
  }
}

// x_disp[r] = x[row_src[r] / k] or zeros; rows [0, offsets[E]) (packed) or
// all rows (padded). One wave per row.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint4* __restrict__ x,
                                                          const int32_t* __restrict__ row_src,
                                                          const int32_t* __restrict__ offsets,
                                                          uint4* __restrict__ x_disp, int E, int k,
                                                          int vecs, long rows, int padded) {
  const long r = blockIdx.x * 4L + (threadIdx.x >> 6);
  const long live = padded ? rows : (long)offsets[E];
  if (r >= live) return;
  const int lane = threadIdx.x & 63;
  const int src = row_src[r];
  uint4* dst = x_disp + r * vecs;
  if (src >= 0) {
    const uint4* s = x + (long)(src / k) * vecs;
    for (int v = lane; v < vecs; v += 64) dst[v] = s[v];
  } else {
    const uint4 z = make_uint4(0, 0, 0, 0);
    for (int v = lane; v < vecs; v += 64) dst[v] = z;
  }
}

// y[t] = sum_j w[t][j] * src[slot[t][j]] over kept j (w == nullptr: weight 1).
// One wave per token, 8 elements per lane step.
template <typename TE>
__global__ __launch_bounds__(256) void combine_rows_kernel(const TE* __restrict__ src,
                                                           const int32_t* __restrict__ slot,
                                                           const float* __restrict__ w,
                                                           TE* __restrict__ y, int T, int M,
                                                           int k) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int lane = threadIdx.x & 63;
  int sl[kMaxK];
  float wt[kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      sl[j] = slot[(long)t * k + j];
      wt[j] = (w != nullptr) ? w[(long)t * k + j] : 1.0f;
    }
  }
  for (int m = lane * 8; m < M; m += 64 * 8) {
    float acc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k && sl[j] >= 0) {
        float v[8];
        load8(src + (long)sl[j] * M + m, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += wt[j] * v[q];
      }
    }
    store8(y + (long)t * M + m, acc);
  }
}

// combine backward, token part: dy_disp[slot] = w * dy[t], d_w = <dy[t], y_disp[slot]>
template <typename TE>
__global__ __launch_bounds__(256) void combine_bwd_kernel(
    const TE* __restrict__ dy, const TE* __restrict__ y_disp, const int32_t* __restrict__ slot,
    const float* __restrict__ w, const int32_t* __restrict__ counts, TE* __restrict__ dy_disp,
    float* __restrict__ dw, int T, int M, int k, int E, int C, int token_blocks) {
  const int lane = threadIdx.x & 63;
  if ((int)blockIdx.x >= token_blocks) {
    // padded layout: zero rows [e*C + counts[e], (e+1)*C)
    const long r = ((long)blockIdx.x - token_blocks) * 4 + (threadIdx.x >> 6);
    if (r >= (long)E * C) return;
    const int e = (int)(r / C), i = (int)(r % C);
    if (i < counts[e]) return;
    const float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int m = lane * 8; m < M; m += 64 * 8) store8(dy_disp + r * M + m, z);
    return;
  }
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int sl[kMaxK];
  float wt[kMaxK], dot[kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    dot[j] = 0.f;
    if (j < k) {
      sl[j] = slot[(long)t * k + j];
      wt[j] = w[(long)t * k + j];
    }
  }
  for (int m = lane * 8; m < M; m += 64 * 8) {
    float g[8];
    load8(dy + (long)t * M + m, g);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k && sl[j] >= 0) {
        float v[8], o[8];
        load8(y_disp + (long)sl[j] * M + m, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          dot[j] += g[q] * v[q];
          o[q] = wt[j] * g[q];
        }
        store8(dy_disp + (long)sl[j] * M + m, o);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      float d = dot[j];
      for (int off = 32; off > 0; off >>= 1) d += __shfl_xor(d, off, 64);
      if (lane == 0) dw[(long)t * k + j] = (sl[j] >= 0) ? d : 0.f;
    }
  }
}

}  // namespace

hipError_t launch_dispatch(const Shape& s, const int32_t* idx, const void* x, int32_t* counts,
                           int32_t* offsets, int32_t* slot, int32_t* row_src, int32_t* load,
                           void* x_disp, hipStream_t st) {
  const int padded = s.layout == FLOWMOE_PADDED;
  hipError_t err = traced(FLOWMOE_K_SCAN, st, [&] {
    hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(kScanThreads), 0, st, idx, counts, offsets,
                       slot, row_src, load, s.T, s.k, s.E, s.C, padded, s.rows);
  });
  if (err != hipSuccess || s.rows == 0) return err;
  const int vecs = (int)((long)s.M * esize(s.dtype) / 16);
  const long blocks = (s.rows + 3) / 4;
  return traced(FLOWMOE_K_GATHER, st, [&] {
    hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const uint4*)x, row_src, offsets, (uint4*)x_disp, s.E, s.k, vecs, s.rows,
                       padded);
  });
}

hipError_t launch_combine(const Shape& s, const void* y_disp, const int32_t* slot, const float* w,
                          void* y, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int blocks = (s.T + 3) / 4;
  return traced(FLOWMOE_K_COMBINE, st, [&] {
    if (s.dtype == FLOWMOE_BF16)
      hipLaunchKernelGGL(combine_rows_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st,
                         (const bf16_t*)y_disp, slot, w, (bf16_t*)y, s.T, s.M, s.k);
    else
      hipLaunchKernelGGL(combine_rows_kernel<float>, dim3(blocks), dim3(256), 0, st,
                         (const float*)y_disp, slot, w, (float*)y, s.T, s.M, s.k);
  });
}

hipError_t launch_dispatch_bwd(const Shape& s, const void* dx_disp, const int32_t* slot, void* dx,
                               hipStream_t st) {
  return launch_combine(s, dx_disp, slot, nullptr, dx, st);
}

hipError_t launch_combine_bwd(const Shape& s, const void* dy, const void* y_disp,
                              const int32_t* slot, const float* w, const int32_t* counts,
                              const int32_t* offsets, void* dy_disp, float* dw, hipStream_t st) {
  (void)offsets;
  const int token_blocks = (s.T + 3) / 4;
  const long fill_blocks = (s.layout == FLOWMOE_PADDED) ? ((long)s.E * s.C + 3) / 4 : 0;
  const long blocks = token_blocks + fill_blocks;
  if (blocks == 0) return hipSuccess;
  return traced(FLOWMOE_K_COMBINE_BWD, st, [&] {
    if (s.dtype == FLOWMOE_BF16)
      hipLaunchKernelGGL(combine_bwd_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, st,
                         (const bf16_t*)dy, (const bf16_t*)y_disp, slot, w, counts,
                         (bf16_t*)dy_disp, dw, s.T, s.M, s.k, s.E, s.C, token_blocks);
    else
      hipLaunchKernelGGL(combine_bwd_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st,
                         (const float*)dy, (const float*)y_disp, slot, w, counts,
                         (float*)dy_disp, dw, s.T, s.M, s.k, s.E, s.C, token_blocks);
  });
}

}  // namespace flowmoe
