// Expert FFN (E_r of Sec. 2.1) as grouped GEMMs over the dispatched rows.
//
// Two grouping modes:
//   ROWS  C_e[rows_e x N] = A[rows of e][K] * B_e[K x N]   (forward, dgrad):
//         the M dimension is ragged per expert (counts on the device), the
//         grid covers an upper bound of row tiles and each block finds its
//         expert by a prefix over the per-expert tile counts.
//   KSUM  C_e[Mdim x N]  = sum over rows r of e: A[r][.]^T B[r][.]  (wgrad):
//         the reduction length K = counts[e] is ragged.
//
// bf16 path: v_mfma_f32_32x32x16_bf16, 256 threads (2 x 2 waves), block tile
// BM x BN x 64, each wave 32*FM x 32*FN. Both operands are staged in LDS
// K-contiguous ([row][64] bf16 = 128 B per row) with the 16-byte chunk index
// XOR-swizzled by (row & 7), double-buffered with register prefetch of the
// next k-tile. Operands whose global layout is K-contiguous are copied with
// 16-byte loads; operands contiguous along M or N are loaded as KT x 8
// blocks and transposed in registers before the LDS write.
// fp32 path (correctness workloads): a plain LDS-tiled FMA kernel with the
// same modes and epilogues.
#include <math.h>

#include "common.hpp"

namespace flowmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

enum { MODE_ROWS = 0, MODE_KSUM = 1 };
enum {
  EPI_STORE = 0,       // C0 = acc
  EPI_GELU_FWD = 1,    // C0 = h = acc, C1 = a = gelu(acc)
  EPI_SWIGLU_FWD = 2,  // dual accumulators h1, h3: C0 = [h1 | h3], C1 = silu(h1) h3
  EPI_GELU_BWD = 3,    // C0 = acc * gelu'(aux h)
  EPI_SWIGLU_BWD = 4,  // C0 = [acc h3 silu'(h1) | acc silu(h1)] with aux = [h1 | h3]
  EPI_WGRAD = 5        // fp32 C0 (cols < nsplit) / C1 (cols >= nsplit), optional +=
};

struct GemmParams {
  const void* A;
  long lda;
  const void* B0;
  const void* B1;    // second B source: W3 (dual forward) or k >= ksplit (dgrad)
  long ldb;
  long b_estride;    // per-expert stride of B (ROWS mode)
  int ksplit;        // ROWS, K-contiguous B: k >= ksplit reads B1 at k - ksplit
  int Mdim, N, K;    // KSUM: Mdim rows of C; ROWS: K reduction length
  const int32_t* counts;
  const int32_t* offsets;
  int E;
  int padC;          // padded layout: every expert spans C rows (0 = packed)
  int mt_bound;      // ROWS: row tiles per column tile in the grid
  void* C0;
  void* C1;
  long ldc, ldc1;
  long c_estride;    // KSUM: per-expert stride of C
  int nsplit;        // EPI_WGRAD: first column that goes to C1
  int coloff;        // column offset added to C0 stores (fp32 split forward)
  const void* aux;   // h (GELU) or [h1 | h3] (SwiGLU), ld = ldaux
  long ldaux;
  int Hh;            // SwiGLU: H (offset of the second half)
  int accumulate;
};

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
constexpr int BK = 64;
constexpr int kThreads = 256;

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + (((chunk ^ (row & 7)) & 7) << 4);
}

// pack 16-bit column `col` of two 8 x bf16 rows into one dword (lo = r0)
__device__ __forceinline__ uint32_t pick2(const uint4& r0, const uint4& r1, int col) {
  const uint32_t* a = reinterpret_cast<const uint32_t*>(&r0);
  const uint32_t* b = reinterpret_cast<const uint32_t*>(&r1);
  const uint32_t x = a[col >> 1], y = b[col >> 1];
  return (col & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
}

// K-contiguous tile loader: ROWSxBK tile, 16-byte chunks, NP chunks/thread.
template <int ROWS>
struct KcLoader {
  static constexpr int NP = ROWS * 8 / kThreads;
  const bf16_t* p0[NP];  // row starts (k = 0)
  const bf16_t* p1[NP];  // second source (k >= ksplit)
  bool ok[NP];
  uint4 v[NP];
  int c;  // chunk of this thread
  __device__ __forceinline__ void load(int k0, int K, int ksplit) {
    const int k = k0 + c * 8;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (ok[p] && k < K) {
        const bf16_t* src = (k < ksplit) ? (p0[p] + k) : (p1[p] + (k - ksplit));
        v[p] = *reinterpret_cast<const uint4*>(src);
      } else {
        v[p] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int r0 = threadIdx.x >> 3;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int row = r0 + p * (kThreads / 8);
      *reinterpret_cast<uint4*>(lds + lds_off(row, c)) = v[p];
    }
  }
};

// MN-contiguous tile loader: element (row i, k) at col_ptr + k*ld, where each
// thread owns one group of 8 rows (g) and KT consecutive k (kg).
template <int ROWS>
struct MncLoader {
  static constexpr int KT = ROWS * BK / (8 * kThreads);  // 4 for 128 rows, 8 for 256
  static constexpr int KG = BK / KT;                    // k groups per tile
  const bf16_t* col;  // pointer to (k = 0, first row of my group)
  long ld;
  bool ok;
  int kg, g;
  uint4 v[KT];
  __device__ __forceinline__ void load(int k0, int Klim) {
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const int k = k0 + kg * KT + j;
      if (ok && k < Klim)
        v[j] = *reinterpret_cast<const uint4*>(col + (long)k * ld);
      else
        v[j] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int ii = 0; ii < 8; ++ii) {
      const int row = g * 8 + ii;
      if constexpr (KT == 8) {
        uint4 o;
        o.x = pick2(v[0], v[1], ii);
        o.y = pick2(v[2], v[3], ii);
        o.z = pick2(v[4], v[5], ii);
        o.w = pick2(v[6], v[7], ii);
        *reinterpret_cast<uint4*>(lds + lds_off(row, kg)) = o;
      } else {
        uint2 o;
        o.x = pick2(v[0], v[1], ii);
        o.y = pick2(v[2], v[3], ii);
        const int kin = kg * KT;  // element offset of my k group in the tile
        *reinterpret_cast<uint2*>(lds + lds_off(row, kin >> 3) + ((kin & 7) << 1)) = o;
      }
    }
  }
};

__device__ __forceinline__ float silu_f(float z) { return z * sigmoid_f(z); }

template <int MODE, bool A_KC, bool B_KC, int EPI, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_bf16_kernel(GemmParams p) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  static_assert(EPI != EPI_SWIGLU_FWD || FN == 2, "dual forward needs 64-column wave tiles");
  __shared__ __attribute__((aligned(16))) char smem[2 * (BM + BN) * 128];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- which tile --------------------------------------------------------
  int e = 0, mt = 0, nt = 0, row0 = 0, rows_e = 0, cnt_e = 0;
  if constexpr (MODE == MODE_ROWS) {
    nt = blockIdx.x / p.mt_bound;
    const int ml = blockIdx.x % p.mt_bound;
    int acc_t = 0;
    mt = -1;
    for (e = 0; e < p.E; ++e) {
      const int c = p.counts[e];
      const int r = p.padC ? p.padC : c;
      const int te = (r + BM - 1) / BM;
      if (ml < acc_t + te) {
        mt = ml - acc_t;
        rows_e = r;
        cnt_e = c;
        break;
      }
      acc_t += te;
    }
    if (mt < 0) return;
    row0 = p.offsets[e] + mt * BM;  // first global row of this tile
  } else {
    const int mtn = (p.Mdim + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
    e = blockIdx.x / (mtn * ntn);
    const int rem = blockIdx.x % (mtn * ntn);
    mt = rem / ntn;
    nt = rem % ntn;
    cnt_e = p.counts[e];
    row0 = p.offsets[e];
  }
  constexpr int NCOLS = (EPI == EPI_SWIGLU_FWD) ? BN / 2 : BN;  // distinct output columns per tile
  const int n0 = nt * NCOLS;

  // ---- loaders -------------------------------------------------------------
  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* B0 = static_cast<const bf16_t*>(p.B0);
  const bf16_t* B1 = static_cast<const bf16_t*>(p.B1);
  int Kred;  // reduction length
  if constexpr (MODE == MODE_ROWS) Kred = p.K; else Kred = cnt_e;

  KcLoader<BM> la;
  MncLoader<BM> lam;
  if constexpr (A_KC) {  // ROWS: A rows are the expert's rows
    la.c = tid & 7;
#pragma unroll
    for (int q = 0; q < KcLoader<BM>::NP; ++q) {
      const int i = (tid >> 3) + q * (kThreads / 8);
      const int li = mt * BM + i;
      la.ok[q] = li < cnt_e;
      la.p0[q] = A + (long)(row0 + i) * p.lda;
      la.p1[q] = la.p0[q];
    }
  } else {  // KSUM: A[i][k] = A[(row0 + k) * lda + m0 + i]
    lam.kg = tid % MncLoader<BM>::KG;
    lam.g = tid / MncLoader<BM>::KG;
    const int i0 = mt * BM + lam.g * 8;
    lam.ok = i0 < p.Mdim;
    lam.ld = p.lda;
    lam.col = A + (long)row0 * p.lda + i0;
  }
  KcLoader<BN> lb;
  MncLoader<BN> lbm;
  if constexpr (B_KC) {  // ROWS dgrad: B[k][n] at B + e*estride + n*ldb + k
    lb.c = tid & 7;
#pragma unroll
    for (int q = 0; q < KcLoader<BN>::NP; ++q) {
      const int i = (tid >> 3) + q * (kThreads / 8);
      const int n = n0 + i;
      lb.ok[q] = n < p.N;
      lb.p0[q] = B0 + (long)e * p.b_estride + (long)n * p.ldb;
      lb.p1[q] = (B1 != nullptr) ? B1 + (long)e * p.b_estride + (long)n * p.ldb : lb.p0[q];
    }
  } else {
    lbm.kg = tid % MncLoader<BN>::KG;
    lbm.g = tid / MncLoader<BN>::KG;
    lbm.ld = p.ldb;
    if constexpr (MODE == MODE_ROWS) {
      const bf16_t* base = B0;
      int n = n0 + lbm.g * 8;
      if constexpr (EPI == EPI_SWIGLU_FWD) {
        const int cc = lbm.g * 8;  // tile column
        base = ((cc >> 5) & 1) ? B1 : B0;
        n = n0 + (cc >> 6) * 32 + (cc & 31);
      }
      lbm.ok = n < p.N;
      lbm.col = base + (long)e * p.b_estride + n;
    } else {  // KSUM: B[k][n] = B[(row0 + k) * ldb + n]
      const int n = n0 + lbm.g * 8;
      lbm.ok = n < p.N;
      lbm.col = B0 + (long)row0 * p.ldb + n;
    }
  }

  auto load_tiles = [&](int k0) {
    if constexpr (A_KC) la.load(k0, Kred, 1 << 30); else lam.load(k0, Kred);
    if constexpr (B_KC) lb.load(k0, Kred, p.ksplit); else lbm.load(k0, Kred);
  };
  auto store_tiles = [&](int buf) {
    char* a_s = smem + buf * (BM + BN) * 128;
    char* b_s = a_s + BM * 128;
    if constexpr (A_KC) la.store(a_s); else lam.store(a_s);
    if constexpr (B_KC) lb.store(b_s); else lbm.store(b_s);
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (Kred + BK - 1) / BK;
  if (nk > 0) {
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) load_tiles((kt + 1) * BK);
    const char* a_s = smem + (kt & 1) * (BM + BN) * 128;
    const char* b_s = a_s + BM * 128;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = kk * 2 + (lane >> 5);
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(a_s + lds_off(wm * WM + i * 32 + (lane & 31), ch));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(b_s + lds_off(wn * WN + j * 32 + (lane & 31), ch));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_tiles((kt + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue ------------------------------------------------------------
  // acc[i][j][r] holds row  wm*WM + i*32 + 8*(r/4) + 4*(lane/32) + r%4,
  //                   col  wn*WN + j*32 + lane%32
  const int lcol = lane & 31, lhalf = lane >> 5;
  if constexpr (MODE == MODE_ROWS) {
    bf16_t* C0 = static_cast<bf16_t*>(p.C0);
    bf16_t* C1 = static_cast<bf16_t*>(p.C1);
    const bf16_t* aux = static_cast<const bf16_t*>(p.aux);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ti = wm * WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
        const int li = mt * BM + ti;  // row within the expert
        if (li >= rows_e) continue;
        const bool data = li < cnt_e;
        const long g = row0 + ti;
        if constexpr (EPI == EPI_SWIGLU_FWD) {
          const int n = n0 + wn * 32 + lcol;
          if (n < p.N) {
            const float h1 = data ? acc[i][0][r] : 0.f;
            const float h3 = data ? acc[i][1][r] : 0.f;
            C0[g * p.ldc + n] = f32_to_bf16(h1);
            C0[g * p.ldc + p.Hh + n] = f32_to_bf16(h3);
            C1[g * p.ldc1 + n] = f32_to_bf16(silu_f(h1) * h3);
          }
        } else {
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * WN + j * 32 + lcol;
            if (n >= p.N) continue;
            const float v = data ? acc[i][j][r] : 0.f;
            if constexpr (EPI == EPI_STORE) {
              C0[g * p.ldc + n] = f32_to_bf16(v);
            } else if constexpr (EPI == EPI_GELU_FWD) {
              C0[g * p.ldc + n] = f32_to_bf16(v);
              C1[g * p.ldc1 + n] = f32_to_bf16(gelu_f(v));
            } else if constexpr (EPI == EPI_GELU_BWD) {
              const float h = bf16_to_f32(aux[g * p.ldaux + n]);
              C0[g * p.ldc + n] = f32_to_bf16(v * gelu_grad_f(h));
            } else if constexpr (EPI == EPI_SWIGLU_BWD) {
              const float h1 = bf16_to_f32(aux[g * p.ldaux + n]);
              const float h3 = bf16_to_f32(aux[g * p.ldaux + p.Hh + n]);
              const float sg = sigmoid_f(h1);
              C0[g * p.ldc + n] = f32_to_bf16(v * h3 * sg * (1.f + h1 * (1.f - sg)));
              C0[g * p.ldc + p.Hh + n] = f32_to_bf16(v * h1 * sg);
            }
          }
        }
      }
    }
  } else {  // KSUM wgrad, fp32 out
    float* C0 = static_cast<float*>(p.C0);
    float* C1 = static_cast<float*>(p.C1);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = mt * BM + wm * WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
        if (m >= p.Mdim) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int n = n0 + wn * WN + j * 32 + lcol;
          if (n >= p.N) continue;
          float* dst = (n < p.nsplit) ? C0 + (long)e * p.c_estride + (long)m * p.ldc + n
                                      : C1 + (long)e * p.c_estride + (long)m * p.ldc + (n - p.nsplit);
          const float v = acc[i][j][r];
          *dst = p.accumulate ? *dst + v : v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 kernel: 64 x 64 tiles, 16-deep k steps, 4 x 4 outputs per thread
// ---------------------------------------------------------------------------
template <int MODE, bool B_KC, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmParams p) {
  constexpr int TB = 64, TK = 16;
  __shared__ float As[TK][TB + 1];
  __shared__ float Bs[TK][TB + 1];
  const int tid = threadIdx.x;
  int e = 0, mt = 0, nt = 0, row0 = 0, rows_e = 0, cnt_e = 0;
  if constexpr (MODE == MODE_ROWS) {
    nt = blockIdx.x / p.mt_bound;
    const int ml = blockIdx.x % p.mt_bound;
    int acc_t = 0;
    mt = -1;
    for (e = 0; e < p.E; ++e) {
      const int c = p.counts[e];
      const int r = p.padC ? p.padC : c;
      const int te = (r + TB - 1) / TB;
      if (ml < acc_t + te) {
        mt = ml - acc_t;
        rows_e = r;
        cnt_e = c;
        break;
      }
      acc_t += te;
    }
    if (mt < 0) return;
    row0 = p.offsets[e] + mt * TB;
  } else {
    const int mtn = (p.Mdim + TB - 1) / TB, ntn = (p.N + TB - 1) / TB;
    e = blockIdx.x / (mtn * ntn);
    const int rem = blockIdx.x % (mtn * ntn);
    mt = rem / ntn;
    nt = rem % ntn;
    cnt_e = p.counts[e];
    row0 = p.offsets[e];
  }
  const int n0 = nt * TB;
  const float* A = static_cast<const float*>(p.A);
  const float* B0 = static_cast<const float*>(p.B0);
  const float* B1 = static_cast<const float*>(p.B1);
  const int Kred = (MODE == MODE_ROWS) ? p.K : cnt_e;
  const int ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < Kred; k0 += TK) {
    for (int q = tid; q < TK * TB; q += 256) {
      const int kk = q / TB, ii = q % TB;
      const int k = k0 + kk;
      float av = 0.f, bv = 0.f;
      if (k < Kred) {
        if constexpr (MODE == MODE_ROWS) {
          if (mt * TB + ii < cnt_e) av = A[(long)(row0 + ii) * p.lda + k];
        } else {
          if (mt * TB + ii < p.Mdim) av = A[(long)(row0 + k) * p.lda + mt * TB + ii];
        }
        const int n = n0 + ii;
        if (n < p.N) {
          if constexpr (MODE == MODE_KSUM) {
            bv = B0[(long)(row0 + k) * p.ldb + n];
          } else if constexpr (B_KC) {
            bv = (k < p.ksplit) ? B0[(long)e * p.b_estride + (long)n * p.ldb + k]
                                : B1[(long)e * p.b_estride + (long)n * p.ldb + (k - p.ksplit)];
          } else {
            bv = B0[(long)e * p.b_estride + (long)k * p.ldb + n];
          }
        }
      }
      As[kk][ii] = av;
      Bs[kk][ii] = bv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
  float* C0 = static_cast<float*>(p.C0);
  float* C1 = static_cast<float*>(p.C1);
  const float* aux = static_cast<const float*>(p.aux);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ti = ty * 4 + i;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= p.N) continue;
      if constexpr (MODE == MODE_ROWS) {
        const int li = mt * TB + ti;
        if (li >= rows_e) continue;
        const float v = (li < cnt_e) ? acc[i][j] : 0.f;
        const long g = row0 + ti;
        if constexpr (EPI == EPI_STORE) {
          C0[g * p.ldc + p.coloff + n] = v;
        } else if constexpr (EPI == EPI_GELU_FWD) {
          C0[g * p.ldc + n] = v;
          C1[g * p.ldc1 + n] = gelu_f(v);
        } else if constexpr (EPI == EPI_GELU_BWD) {
          C0[g * p.ldc + n] = v * gelu_grad_f(aux[g * p.ldaux + n]);
        } else if constexpr (EPI == EPI_SWIGLU_BWD) {
          const float h1 = aux[g * p.ldaux + n], h3 = aux[g * p.ldaux + p.Hh + n];
          const float sg = sigmoid_f(h1);
          C0[g * p.ldc + n] = v * h3 * sg * (1.f + h1 * (1.f - sg));
          C0[g * p.ldc + p.Hh + n] = v * h1 * sg;
        }
      } else {
        const int m = mt * TB + ti;
        if (m >= p.Mdim) continue;
        float* dst = (n < p.nsplit) ? C0 + (long)e * p.c_estride + (long)m * p.ldc + n
                                    : C1 + (long)e * p.c_estride + (long)m * p.ldc + (n - p.nsplit);
        *dst = p.accumulate ? *dst + acc[i][j] : acc[i][j];
      }
    }
  }
}

// fp32 SwiGLU activation: a = silu(h1) * h3 over the live rows
__global__ void swiglu_act_f32_kernel(const float* __restrict__ h, float* __restrict__ a,
                                      const int32_t* __restrict__ offsets, int E, long rows,
                                      int padded, int H) {
  const long live = padded ? rows : (long)offsets[E];
  const long n = live * H;
  for (long q = blockIdx.x * (long)blockDim.x + threadIdx.x; q < n; q += (long)gridDim.x * blockDim.x) {
    const long r = q / H;
    const int c = (int)(q % H);
    const float h1 = h[r * 2 * H + c], h3 = h[r * 2 * H + H + c];
    a[q] = h1 * sigmoid_f(h1) * h3;
  }
}

// ---------------------------------------------------------------------------
// host helpers
// ---------------------------------------------------------------------------
int rows_tiles_bound(const Shape& s, int bm) {
  if (s.layout == FLOWMOE_PADDED) return s.E * ((s.C + bm - 1) / bm);
  return (int)((s.rows + bm - 1) / bm) + s.E;
}

GemmParams base_params(const Shape& s, const int32_t* counts, const int32_t* offsets) {
  GemmParams p = {};
  p.counts = counts;
  p.offsets = offsets;
  p.E = s.E;
  p.padC = (s.layout == FLOWMOE_PADDED) ? s.C : 0;
  p.ksplit = 1 << 30;
  p.nsplit = 1 << 30;
  p.Hh = s.H;
  return p;
}

template <int MODE, bool A_KC, bool B_KC, int EPI, int BM, int BN>
hipError_t run_bf16(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  long blocks;
  if (MODE == MODE_ROWS) {
    const int ncols = (EPI == EPI_SWIGLU_FWD) ? BN / 2 : BN;
    p.mt_bound = rows_tiles_bound(s, BM);
    blocks = (long)p.mt_bound * ((p.N + ncols - 1) / ncols);
  } else {
    blocks = (long)s.E * ((p.Mdim + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  }
  if (blocks == 0) return hipSuccess;
  return traced(kind, st, [&] {
    hipLaunchKernelGGL((gemm_bf16_kernel<MODE, A_KC, B_KC, EPI, BM, BN>), dim3((unsigned)blocks),
                       dim3(kThreads), 0, st, p);
  });
}

template <int MODE, bool B_KC, int EPI>
hipError_t run_f32(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  long blocks;
  if (MODE == MODE_ROWS) {
    p.mt_bound = rows_tiles_bound(s, 64);
    blocks = (long)p.mt_bound * ((p.N + 63) / 64);
  } else {
    blocks = (long)s.E * ((p.Mdim + 63) / 64) * ((p.N + 63) / 64);
  }
  if (blocks == 0) return hipSuccess;
  return traced(kind, st, [&] {
    hipLaunchKernelGGL((gemm_f32_kernel<MODE, B_KC, EPI>), dim3((unsigned)blocks), dim3(256), 0, st,
                       p);
  });
}

#define FLOWMOE_TRY(x)                 \
  do {                                 \
    hipError_t err_ = (x);             \
    if (err_ != hipSuccess) return err_; \
  } while (0)

}  // namespace

size_t ffn_bwd_ws_bytes(const Shape& s) {
  const int hw = (s.act == FLOWMOE_SWIGLU) ? 2 * s.H : s.H;
  return align256((size_t)s.rows * hw * esize(s.dtype));
}

hipError_t launch_expert_ffn(const Shape& s, const void* x_disp, const int32_t* counts,
                             const int32_t* offsets, const void* w1, const void* w3,
                             const void* w2, void* h_save, void* a_save, void* y_disp,
                             hipStream_t st) {
  if (s.rows == 0) return hipSuccess;
  const bool swiglu = s.act == FLOWMOE_SWIGLU;
  const int H = s.H, M = s.M;
  // layer 1: h = X W1 (and h3 = X W3)
  GemmParams p = base_params(s, counts, offsets);
  p.A = x_disp;
  p.lda = M;
  p.K = M;
  p.N = H;
  p.B0 = w1;
  p.B1 = w3;
  p.ldb = H;
  p.b_estride = (long)M * H;
  p.C0 = h_save;
  p.C1 = a_save;
  p.ldc = swiglu ? 2L * H : H;
  p.ldc1 = H;
  if (s.dtype == FLOWMOE_BF16) {
    if (swiglu)
      FLOWMOE_TRY((run_bf16<MODE_ROWS, true, false, EPI_SWIGLU_FWD, 128, 128>(FLOWMOE_K_FFN1, s, p, st)));
    else
      FLOWMOE_TRY((run_bf16<MODE_ROWS, true, false, EPI_GELU_FWD, 128, 128>(FLOWMOE_K_FFN1, s, p, st)));
  } else {
    if (swiglu) {
      p.B1 = nullptr;
      FLOWMOE_TRY((run_f32<MODE_ROWS, false, EPI_STORE>(FLOWMOE_K_FFN1, s, p, st)));
      p.B0 = w3;
      p.coloff = H;
      FLOWMOE_TRY((run_f32<MODE_ROWS, false, EPI_STORE>(FLOWMOE_K_FFN1, s, p, st)));
      FLOWMOE_TRY(traced(FLOWMOE_K_SWIGLU_ACT, st, [&] {
        hipLaunchKernelGGL(swiglu_act_f32_kernel, dim3(1024), dim3(256), 0, st,
                           (const float*)h_save, (float*)a_save, offsets, s.E, s.rows,
                           s.layout == FLOWMOE_PADDED, H);
      }));
    } else {
      FLOWMOE_TRY((run_f32<MODE_ROWS, false, EPI_GELU_FWD>(FLOWMOE_K_FFN1, s, p, st)));
    }
  }
  // layer 2: y = a W2
  GemmParams q = base_params(s, counts, offsets);
  q.A = a_save;
  q.lda = H;
  q.K = H;
  q.N = M;
  q.B0 = w2;
  q.ldb = M;
  q.b_estride = (long)H * M;
  q.C0 = y_disp;
  q.ldc = M;
  if (s.dtype == FLOWMOE_BF16)
    return run_bf16<MODE_ROWS, true, false, EPI_STORE, 128, 128>(FLOWMOE_K_FFN2, s, q, st);
  return run_f32<MODE_ROWS, false, EPI_STORE>(FLOWMOE_K_FFN2, s, q, st);
}

hipError_t launch_expert_ffn_bwd(const Shape& s, const void* dy_disp, const void* x_disp,
                                 const void* h_save, const void* a_save, const int32_t* counts,
                                 const int32_t* offsets, const void* w1, const void* w3,
                                 const void* w2, void* dx_disp, float* dw1, float* dw3,
                                 float* dw2, int accumulate, void* ws, hipStream_t st) {
  const bool swiglu = s.act == FLOWMOE_SWIGLU;
  const bool bf = s.dtype == FLOWMOE_BF16;
  const int H = s.H, M = s.M;
  const int HW = swiglu ? 2 * H : H;
  void* dH = ws;
  // 1. dA = dY W2^T, through the activation -> dH (rows x HW)
  if (s.rows > 0) {
    GemmParams p = base_params(s, counts, offsets);
    p.A = dy_disp;
    p.lda = M;
    p.K = M;
    p.N = H;
    p.B0 = w2;  // B[k=m][n=h] = W2[e][h][m]: K-contiguous
    p.ldb = M;
    p.b_estride = (long)H * M;
    p.C0 = dH;
    p.ldc = HW;
    p.aux = h_save;
    p.ldaux = HW;
    if (bf) {
      if (swiglu)
        FLOWMOE_TRY((run_bf16<MODE_ROWS, true, true, EPI_SWIGLU_BWD, 128, 128>(FLOWMOE_K_DGRAD1, s, p, st)));
      else
        FLOWMOE_TRY((run_bf16<MODE_ROWS, true, true, EPI_GELU_BWD, 128, 128>(FLOWMOE_K_DGRAD1, s, p, st)));
    } else {
      if (swiglu)
        FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_SWIGLU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
      else
        FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_GELU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
    }
  }
  // 2. dW2 = A^T dY  (H x M per expert)
  {
    GemmParams p = base_params(s, counts, offsets);
    p.A = a_save;
    p.lda = H;
    p.Mdim = H;
    p.B0 = dy_disp;
    p.ldb = M;
    p.N = M;
    p.C0 = dw2;
    p.ldc = M;
    p.c_estride = (long)H * M;
    p.accumulate = accumulate;
    if (bf)
      FLOWMOE_TRY((run_bf16<MODE_KSUM, false, false, EPI_WGRAD, 128, 128>(FLOWMOE_K_WGRAD2, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_KSUM, false, EPI_WGRAD>(FLOWMOE_K_WGRAD2, s, p, st)));
  }
  // 3. [dW1 | dW3] = X^T [dH1 | dH3]  (M x H per expert, each)
  {
    GemmParams p = base_params(s, counts, offsets);
    p.A = x_disp;
    p.lda = M;
    p.Mdim = M;
    p.B0 = dH;
    p.ldb = HW;
    p.N = HW;
    p.C0 = dw1;
    p.C1 = dw3;
    p.nsplit = H;
    p.ldc = H;
    p.c_estride = (long)M * H;
    p.accumulate = accumulate;
    if (bf)
      FLOWMOE_TRY((run_bf16<MODE_KSUM, false, false, EPI_WGRAD, 128, 128>(FLOWMOE_K_WGRAD1, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_KSUM, false, EPI_WGRAD>(FLOWMOE_K_WGRAD1, s, p, st)));
  }
  // 4. dX = dH1 W1^T (+ dH3 W3^T)
  if (s.rows > 0) {
    GemmParams p = base_params(s, counts, offsets);
    p.A = dH;
    p.lda = HW;
    p.K = HW;
    p.N = M;
    p.B0 = w1;  // B[k=h][n=m] = W1[e][m][h]: K-contiguous
    p.B1 = swiglu ? w3 : nullptr;
    p.ksplit = swiglu ? H : (1 << 30);
    p.ldb = H;
    p.b_estride = (long)M * H;
    p.C0 = dx_disp;
    p.ldc = M;
    if (bf)
      FLOWMOE_TRY((run_bf16<MODE_ROWS, true, true, EPI_STORE, 128, 128>(FLOWMOE_K_DGRAD2, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_STORE>(FLOWMOE_K_DGRAD2, s, p, st)));
  }
  return hipSuccess;
}

}  // namespace flowmoe
