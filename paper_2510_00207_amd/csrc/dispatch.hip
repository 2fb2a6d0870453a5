// Dispatch (D_r) and combine (C_r) of Sec. 2.1, with their backward.
//
// route_scan: capacity-bounded positions in the priority order "every first
//   choice, then every second choice, ..., ascending token within a rank",
//   i.e. a stable counting sort of the sequence s = j*T + t by expert. Block b
//   owns the 1024 positions [1024 b, 1024 b + 1024) of that sequence. It
//   counts, per expert, the assignments before its tile and after it (every
//   block reads all of topk_idx, from L2), so it knows both its tile's base
//   per expert and the totals (hence counts and offsets) without any
//   cross-block communication. Counting works on 64-position chunks: 6
//   ballots on the expert bits tell every lane which lanes share its expert
//   (its rank) and lane e how many lanes hold expert e. Inside the tile, the
//   16 waves' counts are scanned per expert with 16-lane shuffles.
//   That recount grows with the square of the input, so with more than one
//   tile and a workspace a first kernel (tile_hist) writes each tile's
//   per-expert counts and the scan sums those E-wide rows instead: the same
//   integers, from 1024/E times fewer reads (at 8 tiles already 10% faster
//   than the recount, at 96 tiles 3x).
// gather / combine / scatter kernels move whole rows with 16-byte vectors,
//   one wave per row or token, accumulating in float in a fixed order.
#include <atomic>

#include "common.hpp"

namespace flowmoe {
namespace {

template <int V>
struct KConst {
  static constexpr int value = V;
};
// f(KConst<KM>) with KM the smallest of 2, 4, 8 that is >= k
template <typename F>
__host__ void with_kmax(int k, F&& f) {
  if (k <= 2) f(KConst<2>{});
  else if (k <= 4) f(KConst<4>{});
  else f(KConst<8>{});
}

std::atomic<int> g_row_streams{FLOWMOE_ROWS_AUTO};

// f(true or false as a type): non-temporal row streams for bf16 calls that
// move at least 256 MB (the Infinity Cache): there every line of the stream
// is gone before it is read again, and caching it only evicts the rest.
// flowmoe_set_row_streams can force either kind for bf16 calls (fp32 calls
// always stream through the caches).
template <typename F>
__host__ void with_nt(const Shape& s, long rows, F&& f) {
  const int mode = g_row_streams.load(std::memory_order_relaxed);
  const bool big = (long)(rows + s.T) * s.M * 2 >= (256L << 20);
  const bool nt = s.dtype == FLOWMOE_BF16 &&
                  (mode == FLOWMOE_ROWS_NT || (mode == FLOWMOE_ROWS_AUTO && big));
  if (nt) f(std::true_type{});
  else f(std::false_type{});
}

constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / 64;
constexpr int kScanUnroll = 8;  // chunk loads in flight per lane
constexpr long kScanHistTiles = 1;  // more tiles than this: histogram pass

// expert of priority position s (j = s / T, t = s % T), or -1
__device__ __forceinline__ int scan_expert(const int32_t* __restrict__ idx, unsigned s, unsigned n,
                                           unsigned T, int k, int E) {
  if (s >= n) return -1;
  const unsigned j = s / T, t = s - j * T;
  const int e = idx[(long)t * k + j];
  return ((unsigned)e < (unsigned)E) ? e : -1;
}

// ballots over one 64-position chunk: rank of this lane's assignment among
// lanes with the same expert, and (for lane e) the chunk's count of expert e
__device__ __forceinline__ void chunk_match(int e, int lane, uint64_t lt_mask, int& rank,
                                            int& count) {
  const bool valid = e >= 0;
  const int ev = valid ? e : 0;
  const uint64_t vm = __ballot(valid);
  uint64_t same = vm, mine = vm;
#pragma unroll
  for (int b = 0; b < 6; ++b) {
    const uint64_t m = __ballot(valid && ((ev >> b) & 1));
    same &= ((ev >> b) & 1) ? m : ~m;
    mine &= ((lane >> b) & 1) ? m : ~m;
  }
  rank = __popcll(same & lt_mask);
  count = __popcll(mine);
}

// hist[b][e] = assignments of expert e among the tile's 1024 positions
__global__ __launch_bounds__(kScanThreads) void tile_hist_kernel(const int32_t* __restrict__ idx,
                                                                 int32_t* __restrict__ hist,
                                                                 int T, int k, int E) {
  __shared__ int part[kScanWaves][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const unsigned n = (unsigned)T * (unsigned)k;
  const int e = scan_expert(idx, blockIdx.x * (unsigned)kScanThreads + tid, n, T, k, E);
  int rank, cnt;
  chunk_match(e, lane, lt_mask, rank, cnt);
  part[wave][lane] = cnt;
  __syncthreads();
  if (wave == 0 && lane < E) {
    int sum = 0;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) sum += part[w][lane];
    hist[(long)blockIdx.x * E + lane] = sum;
  }
}

__global__ __launch_bounds__(kScanThreads) void route_scan_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ hist,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int32_t* __restrict__ slot,
    int32_t* __restrict__ row_src, int32_t* __restrict__ load, int T, int k, int E, int C,
    int padded, long rows) {
  __shared__ int own[kScanWaves][64];   // tile counts per wave, then element bases
  __shared__ int bef[kScanWaves][64];   // per-wave counts before the tile
  __shared__ int aft[kScanWaves][64];   // per-wave counts after the tile
  __shared__ int tot[64];
  __shared__ int offs[kMaxE + 1];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const unsigned n = (unsigned)T * (unsigned)k;  // <= 2^30 (host check)
  const unsigned tile0 = blockIdx.x * (unsigned)kScanThreads;

  // 1. counts outside the tile: wave w takes chunks c = i * 1024 + 64 w, or
  //    with the tile histograms (lane = expert) the tiles i = w mod 16
  int cb = 0, ca = 0;
  const unsigned nt = (n + kScanThreads - 1) / kScanThreads;  // tiles
  if (hist != nullptr) {
    for (unsigned i0 = wave; i0 < nt; i0 += kScanWaves * kScanUnroll) {
      int hv[kScanUnroll];
#pragma unroll
      for (int u = 0; u < kScanUnroll; ++u) {
        const unsigned i = i0 + u * kScanWaves;
        hv[u] = (i < nt && i != blockIdx.x && lane < E) ? hist[(long)i * E + lane] : 0;
      }
#pragma unroll
      for (int u = 0; u < kScanUnroll; ++u) {
        if (i0 + u * kScanWaves < blockIdx.x) cb += hv[u]; else ca += hv[u];
      }
    }
  } else for (unsigned i0 = 0; i0 < nt; i0 += kScanUnroll) {
    int ev[kScanUnroll];
#pragma unroll
    for (int u = 0; u < kScanUnroll; ++u) {
      const unsigned i = i0 + u;
      const unsigned s = i * kScanThreads + wave * 64 + lane;
      ev[u] = (i < nt && i != blockIdx.x) ? scan_expert(idx, s, n, T, k, E) : -1;
    }
#pragma unroll
    for (int u = 0; u < kScanUnroll; ++u) {
      const unsigned i = i0 + u;
      if (i < nt && i != blockIdx.x) {  // uniform
        int rank, cnt;
        chunk_match(ev[u], lane, lt_mask, rank, cnt);
        if (i < blockIdx.x) cb += cnt; else ca += cnt;
      }
    }
  }
  // 2. the tile itself
  const unsigned s = tile0 + tid;
  const int e = scan_expert(idx, s, n, T, k, E);
  int rank, cnt;
  chunk_match(e, lane, lt_mask, rank, cnt);
  own[wave][lane] = cnt;
  bef[wave][lane] = cb;
  aft[wave][lane] = ca;
  __syncthreads();
  {
    // thread (expert ex, wave w): element base = (assignments of ex before
    // the tile) + (in earlier waves of the tile); totals for the offsets
    const int ex = tid >> 4, w = tid & 15;
    const int c = own[w][ex];
    int inc = c, b4 = bef[w][ex], all = bef[w][ex] + c + aft[w][ex];
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const int o = __shfl_up(inc, off, 16);
      if (w >= off) inc += o;
      b4 += __shfl_xor(b4, off, 16);
      all += __shfl_xor(all, off, 16);
    }
    own[w][ex] = b4 + inc - c;
    if (w == 0) tot[ex] = all;
  }
  __syncthreads();
  if (wave == 0) {
    // offsets: exclusive prefix of min(total, C) over experts (lane = expert)
    const int kept = (lane < E) ? min(tot[lane], C) : 0;
    int inc = kept;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int o = __shfl_up(inc, off, 64);
      if (lane >= off) inc += o;
    }
    if (lane < E) offs[lane] = padded ? lane * C : inc - kept;
    if (lane == E - 1) offs[E] = padded ? E * C : inc;
    if (blockIdx.x == 0 && lane < E) {
      counts[lane] = kept;
      if (load != nullptr) load[lane] = tot[lane];
    }
  }
  __syncthreads();
  if (blockIdx.x == 0 && tid <= E) offsets[tid] = offs[tid];
  // 3. slot and row of this block's assignments
  if (s < n) {
    const unsigned j = s / (unsigned)T, t = s - j * (unsigned)T;
    const long a = (long)t * k + j;
    const int pos = (e >= 0) ? own[wave][e] + rank : C;
    if (pos < C) {
      const int r = offs[e] + pos;
      slot[a] = r;
      row_src[r] = (int)a;
    } else {
      slot[a] = -1;
    }
  }
  // 4. rows that no kept assignment fills: the packed tail, the padded gaps
  for (long r = (long)blockIdx.x * kScanThreads + tid; r < rows; r += (long)gridDim.x * kScanThreads) {
    bool empty;
    if (padded) {
      const int ee = (int)(r / C);
      empty = (int)(r - (long)ee * C) >= min(tot[ee], C);
    } else {
      empty = r >= offs[E];
    }
    if (empty) row_src[r] = -1;
  }
}

// x_disp[r] = x[row_src[r] / k] or zeros; rows [0, offsets[E]) (packed) or
// all rows (padded). One wave per row; each lane has 4 loads in flight.
template <bool NT>
__global__ __launch_bounds__(256) void gather_rows_kernel(const u32x4v_t* __restrict__ x,
                                                          const int32_t* __restrict__ row_src,
                                                          const int32_t* __restrict__ offsets,
                                                          u32x4v_t* __restrict__ x_disp, int E, int k,
                                                          int vecs, long rows, int padded) {
  constexpr int U = 4;
  const long r = blockIdx.x * 4L + (threadIdx.x >> 6);
  const long live = padded ? rows : (long)offsets[E];
  if (r >= live) return;
  const int lane = threadIdx.x & 63;
  const int src = row_src[r];
  u32x4v_t* dst = x_disp + r * vecs;
  if (src >= 0) {
    const u32x4v_t* s = x + (long)(src / k) * vecs;
    for (int v0 = lane; v0 < vecs; v0 += 64 * U) {
      u32x4v_t t[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int v = v0 + 64 * u;
        t[u] = ld16<NT>(s + (v < vecs ? v : v0));  // (every load issued, from in-bounds addresses)
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (v0 + 64 * u < vecs) st16<NT>(dst + v0 + 64 * u, t[u]);
    }
  } else {
    const u32x4v_t z = {0u, 0u, 0u, 0u};
    for (int v = lane; v < vecs; v += 64) st16<NT>(dst + v, z);
  }
}

// x_disp[slot[t][j]] = x[t] for every kept j: one wave per token, the row read
// once (4 loads in flight per lane) and written to each of its rows. Padded
// layout: blocks past the token blocks zero the rows past each expert's
// count. (Rows of the packed layout past offsets[E] are not written.)
template <int KM, bool NT>  // KM >= k
__global__ __launch_bounds__(256) void scatter_rows_kernel(
    const u32x4v_t* __restrict__ x, const int32_t* __restrict__ slot,
    const int32_t* __restrict__ counts, u32x4v_t* __restrict__ x_disp, int T, int k, int vecs,
    int E, int C, int token_blocks) {
  constexpr int U = 4;
  const int lane = threadIdx.x & 63;
  if ((int)blockIdx.x >= token_blocks) {
    const long r = ((long)blockIdx.x - token_blocks) * 4 + (threadIdx.x >> 6);
    if (r >= (long)E * C) return;
    const int e = (int)(r / C), i = (int)(r % C);
    if (i < counts[e]) return;
    const u32x4v_t z = {0u, 0u, 0u, 0u};
    for (int v = lane; v < vecs; v += 64) st16<NT>(x_disp + r * vecs + v, z);
    return;
  }
  const long t = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int sl[KM];
  bool any = false;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    sl[j] = j < k ? slot[t * k + j] : -1;
    any |= sl[j] >= 0;
  }
  if (!any) return;  // every assignment of the token dropped
  const u32x4v_t* src = x + t * vecs;
  for (int v0 = lane; v0 < vecs; v0 += 64 * U) {
    u32x4v_t q[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + 64 * u;
      q[u] = ld16<NT>(src + (v < vecs ? v : v0));  // (every load issued, from in-bounds addresses)
    }
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (sl[j] < 0) continue;
      u32x4v_t* dst = x_disp + (long)sl[j] * vecs;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (v0 + 64 * u < vecs) st16<NT>(dst + v0 + 64 * u, q[u]);
    }
  }
}

// y[t] = sum_j w[t][j] * src[slot[t][j]] over kept j (w == nullptr: weight 1).
// One wave per token, 8 elements per lane step; the k source rows of U
// steps are all loaded before any is used (every load issued, from
// in-bounds addresses), so each lane has k * U loads in flight. GATE
// (dispatch backward of the layer): also adds the gate's share dl_t W_g^T,
// with dl_t taken from the selection (gidx), its weights (gw) and their
// gradients (gdw), and W_g^T given transposed in float (wgt, E x M).
// ADD: y[t] += (the sum) instead of =, the old y loaded with the source rows.
// The source row of every slot j < kl is loaded, also of dropped ones (row 0,
// value unused), so that all loads of a step are in flight together; kl = 0
// when the call has no rows (C = 0: every slot dropped, src may be empty).
template <typename TE, bool GATE, int KM, bool ADD, bool NT>  // KM >= k: per-token array size
__global__ __launch_bounds__(256) void combine_rows_kernel(
    const TE* __restrict__ src, const int32_t* __restrict__ slot, const float* __restrict__ w,
    TE* __restrict__ y, int T, int M, int k, int kl, const int32_t* __restrict__ gidx,
    const float* __restrict__ gw, const float* __restrict__ gdw, const TE* __restrict__ wgt) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int lane = threadIdx.x & 63;
  int sl[KM];
  float wt[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < k) {
      sl[j] = slot[(long)t * k + j];
      wt[j] = (w != nullptr) ? w[(long)t * k + j] : 1.0f;
    }
  }
  int ge[KM];
  float gl[KM];
  if constexpr (GATE) {
    // dl over the selected experts: w_j (dw_j - sum_j' w_j' dw_j')
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < k) {
        ge[j] = gidx[(long)t * k + j];
        gl[j] = gw[(long)t * k + j];
        s += gl[j] * gdw[(long)t * k + j];
      }
    }
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (j < k) gl[j] = gl[j] * (gdw[(long)t * k + j] - s);
  }
  // steps of 512 elements loaded together: 4 in the non-temporal (>= 256 MB)
  // bf16 calls of tokens with at most two experts, else 2 (bf16) or 1
  constexpr int U = sizeof(TE) == 2 ? ((NT && KM <= 2) ? 4 : 2) : 1;
  for (int m0 = lane * 8; m0 < M; m0 += 64 * 8 * U) {
    decltype(raw8_load(src)) raw[U][KM];
    decltype(raw8_load(src)) yold[ADD ? U : 1];
    decltype(raw8_load(src)) graw[GATE ? U : 1][GATE ? KM : 1];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = m0 + 64 * 8 * u < M ? m0 + 64 * 8 * u : m0;
#pragma unroll
      for (int j = 0; j < KM; ++j)
        if (j < kl) raw[u][j] = raw8_ld<NT>(src + (long)(sl[j] >= 0 ? sl[j] : 0) * M + m);
      if constexpr (GATE) {
#pragma unroll
        for (int j = 0; j < KM; ++j)
          if (j < k) graw[u][j] = raw8_load(wgt + (long)ge[j] * M + m);
      }
      if constexpr (ADD) yold[u] = raw8_ld<NT>(y + (long)t * M + m);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = m0 + 64 * 8 * u;
      if (m >= M) break;
      float acc[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = 0.f;
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        if (j < k && sl[j] >= 0) {
          float v[8];
          raw8_f32(raw[u][j], v);
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[q] += wt[j] * v[q];
        }
      }
      if constexpr (GATE) {
#pragma unroll
        for (int j = 0; j < KM; ++j)
          if (j < k) {
            float g[8];
            raw8_f32(graw[u][j], g);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[q] += gl[j] * g[q];
          }
      }
      if constexpr (ADD) {
        float o[8];
        raw8_f32(yold[u], o);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += o[q];
      }
      store8_t<NT>(y + (long)t * M + m, acc);
    }
  }
}

// combine backward, token part: dy_disp[slot] = w * dy[t], d_w = <dy[t], y_disp[slot]>
// (kl as in combine_rows_kernel)
template <typename TE, int KM, bool NT>  // KM >= k: size of the per-token arrays
__global__ __launch_bounds__(256) void combine_bwd_kernel(
    const TE* __restrict__ dy, const TE* __restrict__ y_disp, const int32_t* __restrict__ slot,
    const float* __restrict__ w, const int32_t* __restrict__ counts, TE* __restrict__ dy_disp,
    float* __restrict__ dw, int T, int M, int k, int kl, int E, int C, int token_blocks) {
  const int lane = threadIdx.x & 63;
  if ((int)blockIdx.x >= token_blocks) {
    // padded layout: zero rows [e*C + counts[e], (e+1)*C)
    const long r = ((long)blockIdx.x - token_blocks) * 4 + (threadIdx.x >> 6);
    if (r >= (long)E * C) return;
    const int e = (int)(r / C), i = (int)(r % C);
    if (i < counts[e]) return;
    const float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int m = lane * 8; m < M; m += 64 * 8) store8_t<NT>(dy_disp + r * M + m, z);
    return;
  }
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int sl[KM];
  float wt[KM], dot[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    dot[j] = 0.f;
    if (j < k) {
      sl[j] = slot[(long)t * k + j];
      wt[j] = w[(long)t * k + j];
    }
  }
  // dy and the k rows of y_disp of U steps loaded before any is used
  // steps of 512 elements loaded together: 4 in the non-temporal (>= 256 MB)
  // bf16 calls of tokens with at most two experts, else 2 (bf16) or 1
  constexpr int U = sizeof(TE) == 2 ? ((NT && KM <= 2) ? 4 : 2) : 1;
  for (int m0 = lane * 8; m0 < M; m0 += 64 * 8 * U) {
    decltype(raw8_load(dy)) graw[U], raw[U][KM];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = m0 + 64 * 8 * u < M ? m0 + 64 * 8 * u : m0;
      graw[u] = raw8_ld<NT>(dy + (long)t * M + m);
#pragma unroll
      for (int j = 0; j < KM; ++j)
        if (j < kl) raw[u][j] = raw8_ld<NT>(y_disp + (long)(sl[j] >= 0 ? sl[j] : 0) * M + m);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = m0 + 64 * 8 * u;
      if (m >= M) break;
      float g[8];
      raw8_f32(graw[u], g);
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        if (j < k && sl[j] >= 0) {
          float v[8], o[8];
          raw8_f32(raw[u][j], v);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            dot[j] += g[q] * v[q];
            o[q] = wt[j] * g[q];
          }
          store8_t<NT>(dy_disp + (long)sl[j] * M + m, o);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < k) {
      float d = dot[j];
      for (int off = 32; off > 0; off >>= 1) d += __shfl_xor(d, off, 64);
      if (lane == 0) dw[(long)t * k + j] = (sl[j] >= 0) ? d : 0.f;
    }
  }
}

}  // namespace

void set_row_streams(int mode) { g_row_streams.store(mode, std::memory_order_relaxed); }

size_t dispatch_ws_bytes(const Shape& s) {
  const long tiles = ((long)s.T * s.k + kScanThreads - 1) / kScanThreads;
  return tiles > kScanHistTiles ? align256((size_t)tiles * s.E * sizeof(int32_t)) : 0;
}

hipError_t launch_dispatch(const Shape& s, const int32_t* idx, const void* x, int32_t* counts,
                           int32_t* offsets, int32_t* slot, int32_t* row_src, int32_t* load,
                           void* x_disp, void* ws, hipStream_t st) {
  const int padded = s.layout == FLOWMOE_PADDED;
  const long n = (long)s.T * s.k;
  const long tiles = (n + kScanThreads - 1) / kScanThreads;
  const long fill = (s.rows + kScanThreads - 1) / kScanThreads;  // blocks for the row fill
  const unsigned grid = (unsigned)(tiles > 0 ? tiles : (fill > 0 ? (fill < 64 ? fill : 64) : 1));
  int32_t* hist = (ws != nullptr && dispatch_ws_bytes(s) > 0) ? (int32_t*)ws : nullptr;
  hipError_t err = traced(FLOWMOE_K_SCAN, st, [&] {
    if (hist != nullptr)
      hipLaunchKernelGGL(tile_hist_kernel, dim3((unsigned)tiles), dim3(kScanThreads), 0, st, idx,
                         hist, s.T, s.k, s.E);
    hipLaunchKernelGGL(route_scan_kernel, dim3(grid), dim3(kScanThreads), 0, st, idx,
                       (const int32_t*)hist, counts, offsets, slot, row_src, load, s.T, s.k, s.E,
                       s.C, padded, s.rows);
  });
  if (err != hipSuccess || s.rows == 0) return err;
  const int vecs = (int)((long)s.M * esize(s.dtype) / 16);
  if (s.k == 1) {  // one row per token: walk the rows
    const long blocks = (s.rows + 3) / 4;
    return traced(FLOWMOE_K_GATHER, st, [&] {
      with_nt(s, s.rows, [&](auto ntc) {
        hipLaunchKernelGGL((gather_rows_kernel<decltype(ntc)::value>), dim3((unsigned)blocks),
                           dim3(256), 0, st, (const u32x4v_t*)x, row_src, offsets,
                           (u32x4v_t*)x_disp, s.E, s.k, vecs, s.rows, padded);
      });
    });
  }
  // k >= 2: walk the tokens, each x row read once for its k rows
  const int token_blocks = (s.T + 3) / 4;
  const long fill_blocks = padded ? ((long)s.E * s.C + 3) / 4 : 0;
  const long blocks = token_blocks + fill_blocks;
  if (blocks == 0) return hipSuccess;
  return traced(FLOWMOE_K_GATHER, st, [&] {
    with_kmax(s.k, [&](auto kc) {
      constexpr int KMV = decltype(kc)::value;
      with_nt(s, s.rows, [&](auto ntc) {
        hipLaunchKernelGGL((scatter_rows_kernel<KMV, decltype(ntc)::value>), dim3((unsigned)blocks),
                           dim3(256), 0, st, (const u32x4v_t*)x, slot, counts, (u32x4v_t*)x_disp,
                           s.T, s.k, vecs, s.E, s.C, token_blocks);
      });
    });
  });
}

hipError_t launch_combine(const Shape& s, const void* y_disp, const int32_t* slot, const float* w,
                          void* y, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int kl = s.rows > 0 ? s.k : 0;  // no rows: no source loads
  const int blocks = (s.T + 3) / 4;
  return traced(FLOWMOE_K_COMBINE, st, [&] {
    with_kmax(s.k, [&](auto kc) {
      constexpr int KMV = decltype(kc)::value;
      if (s.dtype == FLOWMOE_BF16)
        with_nt(s, s.rows, [&](auto ntc) {
          hipLaunchKernelGGL((combine_rows_kernel<bf16_t, false, KMV, false, decltype(ntc)::value>),
                             dim3(blocks), dim3(256), 0, st, (const bf16_t*)y_disp, slot, w,
                             (bf16_t*)y, s.T, s.M, s.k, kl, nullptr, nullptr, nullptr, nullptr);
        });
      else
        hipLaunchKernelGGL((combine_rows_kernel<float, false, KMV, false, false>), dim3(blocks),
                           dim3(256), 0, st, (const float*)y_disp, slot, w, (float*)y, s.T, s.M,
                           s.k, kl, nullptr, nullptr, nullptr, nullptr);
    });
  });
}

hipError_t launch_dispatch_bwd(const Shape& s, const void* dx_disp, const int32_t* slot, void* dx,
                               hipStream_t st) {
  return launch_combine(s, dx_disp, slot, nullptr, dx, st);
}

hipError_t launch_dispatch_bwd_add(const Shape& s, const void* dx_disp, const int32_t* slot,
                                   void* dx, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int kl = s.rows > 0 ? s.k : 0;  // no rows: no source loads
  const int blocks = (s.T + 3) / 4;
  return traced(FLOWMOE_K_COMBINE, st, [&] {
    with_kmax(s.k, [&](auto kc) {
      constexpr int KMV = decltype(kc)::value;
      if (s.dtype == FLOWMOE_BF16)
        with_nt(s, s.rows, [&](auto ntc) {
          hipLaunchKernelGGL((combine_rows_kernel<bf16_t, false, KMV, true, decltype(ntc)::value>),
                             dim3(blocks), dim3(256), 0, st, (const bf16_t*)dx_disp, slot, nullptr,
                             (bf16_t*)dx, s.T, s.M, s.k, kl, nullptr, nullptr, nullptr, nullptr);
        });
      else
        hipLaunchKernelGGL((combine_rows_kernel<float, false, KMV, true, false>), dim3(blocks),
                           dim3(256), 0, st, (const float*)dx_disp, slot, nullptr, (float*)dx,
                           s.T, s.M, s.k, kl, nullptr, nullptr, nullptr, nullptr);
    });
  });
}

hipError_t launch_dispatch_bwd_gate(const Shape& s, const void* dx_disp, const int32_t* slot,
                                    const int32_t* idx, const float* w, const float* dw,
                                    const void* wgt, void* dx, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int kl = s.rows > 0 ? s.k : 0;  // no rows: no source loads
  const int blocks = (s.T + 3) / 4;
  return traced(FLOWMOE_K_COMBINE, st, [&] {
    with_kmax(s.k, [&](auto kc) {
      constexpr int KMV = decltype(kc)::value;
      if (s.dtype == FLOWMOE_BF16)
        with_nt(s, s.rows, [&](auto ntc) {
          hipLaunchKernelGGL((combine_rows_kernel<bf16_t, true, KMV, false, decltype(ntc)::value>),
                             dim3(blocks), dim3(256), 0, st, (const bf16_t*)dx_disp, slot, nullptr,
                             (bf16_t*)dx, s.T, s.M, s.k, kl, idx, w, dw, (const bf16_t*)wgt);
        });
      else
        hipLaunchKernelGGL((combine_rows_kernel<float, true, KMV, false, false>), dim3(blocks),
                           dim3(256), 0, st, (const float*)dx_disp, slot, nullptr, (float*)dx,
                           s.T, s.M, s.k, kl, idx, w, dw, (const float*)wgt);
    });
  });
}

hipError_t launch_combine_bwd(const Shape& s, const void* dy, const void* y_disp,
                              const int32_t* slot, const float* w, const int32_t* counts,
                              const int32_t* offsets, void* dy_disp, float* dw, hipStream_t st) {
  (void)offsets;
  const int kl = s.rows > 0 ? s.k : 0;  // no rows: no source loads
  const int token_blocks = (s.T + 3) / 4;
  const long fill_blocks = (s.layout == FLOWMOE_PADDED) ? ((long)s.E * s.C + 3) / 4 : 0;
  const long blocks = token_blocks + fill_blocks;
  if (blocks == 0) return hipSuccess;
  return traced(FLOWMOE_K_COMBINE_BWD, st, [&] {
    with_kmax(s.k, [&](auto kc) {
      constexpr int KMV = decltype(kc)::value;
      if (s.dtype == FLOWMOE_BF16)
        with_nt(s, 2 * s.rows, [&](auto ntc) {
          hipLaunchKernelGGL((combine_bwd_kernel<bf16_t, KMV, decltype(ntc)::value>),
                             dim3((unsigned)blocks), dim3(256), 0, st, (const bf16_t*)dy,
                             (const bf16_t*)y_disp, slot, w, counts, (bf16_t*)dy_disp, dw, s.T, s.M,
                             s.k, kl, s.E, s.C, token_blocks);
        });
      else
        hipLaunchKernelGGL((combine_bwd_kernel<float, KMV, false>), dim3((unsigned)blocks),
                           dim3(256), 0, st, (const float*)dy, (const float*)y_disp, slot, w, counts,
                           (float*)dy_disp, dw, s.T, s.M, s.k, kl, s.E, s.C, token_blocks);
    });
  });
}

}  // namespace flowmoe
