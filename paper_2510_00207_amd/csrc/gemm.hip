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

#include <algorithm>
#include <atomic>

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
  EPI_WGRAD = 5,       // fp32 C0 (cols < nsplit) / C1 (cols >= nsplit), optional +=
  EPI_GATE_DW = 6,     // as EPI_WGRAD (its own instance: the gate's dW_g partials)
  EPI_ADD = 7          // C0 += acc (bf16; aux = C0 itself, prefetched like a pre-activation)
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
  int ntiles;        // ROWS: column tiles
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
  // KSUM: the reduction runs over nseg row segments (the chunks of a layer
  // call), in segment order; segment g's rows of expert e are those of
  // counts[g * E + e] and offsets[g * (E + 1) + e] in A + g * a_sstride and
  // B0 + g * b_sstride (elements)
  int nseg;
  long a_sstride, b_sstride;
  // rows of each row buffer (of each segment's): an expert's range
  // [offsets[e], offsets[e] + rows) is cut at it
  long rows_cap;
  // forward epilogues: per-expert float biases added to the data rows' outputs
  // (bias0 to C0's columns: b1 for h / h1, b2 for y; bias1: b3 for the dual
  // forward's h3), bias0[e * bias_estride + column]; null: none
  const float* bias0;
  const float* bias1;
  long bias_estride;
  // streaming kernel, row mode: an expert's light row tiles walked with its
  // heavy ones (1) or after every heavy tile (0)
  int joined;
};


// counts and offsets are device data: a range that inconsistent ones would
// take past the row buffers is cut there, not followed
__device__ __forceinline__ int clip_rows(long off, int n, long cap) {
  if (off < 0 || off >= cap || n <= 0) return 0;
  return (int)min((long)n, cap - off);
}

// Expert e's rows in segment g: counts[g * E + e] rows from row
// offsets[g * (E + 1) + e]. A dense launch (counts null: the attention's
// projections) splits the rows_cap rows of every segment into E equal
// parts, part e being rows [e rows_cap / E, (e + 1) rows_cap / E) (E = 1:
// all of them; E > 1: the token splits of a weight gradient).
__device__ __forceinline__ int seg_offset(const GemmParams& p, int g, int e) {
  return p.counts ? p.offsets[g * (p.E + 1) + e] : (int)(p.rows_cap * e / p.E);
}
__device__ __forceinline__ int seg_count(const GemmParams& p, int g, int e) {
  return p.counts ? p.counts[g * p.E + e]
                  : (int)(p.rows_cap * (e + 1) / p.E - p.rows_cap * e / p.E);
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
constexpr int BK = 64;

// LDS tile layout: 128-byte rows (64 bf16 of K), 16-byte chunks XOR-swizzled
// by (row / 2) % 8. A ds_read_b128 is serviced 16 lanes per cycle over 64
// banks; the 16 consecutive rows it touches then fall into 16 distinct
// 16-byte bank slots.
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + (((chunk ^ (row >> 1)) & 7) << 4);
}

// pack 16-bit column `col` of two 8 x bf16 rows into one dword (lo = r0)
__device__ __forceinline__ uint32_t pick2(const uint4& r0, const uint4& r1, int col) {
  const uint32_t* a = reinterpret_cast<const uint32_t*>(&r0);
  const uint32_t* b = reinterpret_cast<const uint32_t*>(&r1);
  const uint32_t x = a[col >> 1], y = b[col >> 1];
  return (col & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
}

// K-contiguous tile loader: ROWS x BK tile in 16-byte chunks. Thread t owns
// chunk c = t % 8 of rows r0 + p * NT/8 (r0 = t / 8), p < NP. Rows at or past
// `lim` and chunks at or past K load zeros. Chunks at k >= ksplit come from
// the second source at k - ksplit.
template <int ROWS, int NT>
struct KcLoader {
  static constexpr int NP = ROWS * 8 / NT;
  static constexpr int RSTEP = NT / 8;  // rows between a thread's chunks
  const bf16_t* base0;  // row r0, k = 0
  const bf16_t* base1;  // second source, row r0, k = 0
  long rstride;         // elements between rows r0 + p*RSTEP and r0 + (p+1)*RSTEP
  int lim, r0, c;
  uint4 v[NP];
  __device__ __forceinline__ void init(const bf16_t* b0, const bf16_t* b1, long ld, int limit) {
    r0 = threadIdx.x >> 3;
    c = threadIdx.x & 7;
    base0 = b0 + (long)r0 * ld;
    base1 = b1 + (long)r0 * ld;
    rstride = (long)RSTEP * ld;
    lim = limit;
  }
  __device__ __forceinline__ void load(int k0, int K, int ksplit) {
    const int k = k0 + c * 8;
    const bool second = k >= ksplit;
    const bf16_t* b = second ? base1 + (k - ksplit) : base0 + k;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (r0 + p * RSTEP < lim && k < K)
        v[p] = *reinterpret_cast<const uint4*>(b + p * rstride);
      else
        v[p] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
#pragma unroll
    for (int p = 0; p < NP; ++p)
      *reinterpret_cast<uint4*>(lds + lds_off(r0 + p * RSTEP, c)) = v[p];
  }
};

// MN-contiguous tile loader: element (row i, k) at col + k*ld, where each
// thread owns one group of 8 rows (g) and KT consecutive k (kg); the KT x 8
// block is transposed in registers before the LDS write.
template <int ROWS, int NT>
struct MncLoader {
  static constexpr int KT = ROWS * BK / (8 * NT);  // k rows per thread: 4 or 8
  static constexpr int KG = BK / KT;                    // k groups per tile
  const bf16_t* col;  // (k = 0, first row of my group)
  long ld;
  bool ok;
  int kg, g;
  uint4 v[KT];
  __device__ __forceinline__ void load(int k0, int Klim) {
    const bf16_t* b = col + (long)(k0 + kg * KT) * ld;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const int k = k0 + kg * KT + j;
      if (ok && k < Klim)
        v[j] = *reinterpret_cast<const uint4*>(b + (long)j * ld);
      else
        v[j] = make_uint4(0, 0, 0, 0);
    }
  }
  // Threads of odd groups store their rows in the order 1,0,3,2,..., so one
  // store instruction writes rows of both parities (both halves of the banks).
  __device__ __forceinline__ void store(char* lds) const {
    const bool odd = g & 1;
#pragma unroll
    for (int ii = 0; ii < 8; ++ii) {
      const int row = g * 8 + (ii ^ (int)odd);
      if constexpr (KT == 8) {
        uint4 a, b;  // column ii and column ii ^ 1 of the 8 x 8 block
        a.x = pick2(v[0], v[1], ii);      b.x = pick2(v[0], v[1], ii ^ 1);
        a.y = pick2(v[2], v[3], ii);      b.y = pick2(v[2], v[3], ii ^ 1);
        a.z = pick2(v[4], v[5], ii);      b.z = pick2(v[4], v[5], ii ^ 1);
        a.w = pick2(v[6], v[7], ii);      b.w = pick2(v[6], v[7], ii ^ 1);
        *reinterpret_cast<uint4*>(lds + lds_off(row, kg)) = odd ? b : a;
      } else {
        uint2 a, b;
        a.x = pick2(v[0], v[1], ii);      b.x = pick2(v[0], v[1], ii ^ 1);
        a.y = pick2(v[2], v[3], ii);      b.y = pick2(v[2], v[3], ii ^ 1);
        const int kin = kg * KT;  // element offset of my k group in the tile
        *reinterpret_cast<uint2*>(lds + lds_off(row, kin >> 3) + ((kin & 7) << 1)) = odd ? b : a;
      }
    }
  }
};

__device__ __forceinline__ float silu_f(float z) { return z * sigmoid_f(z); }

// Blocks are dispatched round-robin over the 8 XCDs (each with its own L2);
// renumber them so that every XCD works on one contiguous range of tiles.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int q = nblocks >> 3, rem = nblocks & 7;
  const int x = bid & 7, i = bid >> 3;
  return x * q + (x < rem ? x : rem) + i;
}

// Weight-gradient tile vbid (after xcd_remap, so that each XCD takes a
// contiguous range): expert e, then groups of 4 m tiles that walk the mtn x
// ntn grid m tile fastest. The 32 tiles that an XCD runs at once are 4 m x 8
// n tiles sharing 12 operand panels through its L2 (a walk along n alone
// shares 33: 1 A and 32 B panels); on the large layer's weight gradients
// that walk fetched ~12x their operands' bytes from HBM.
__device__ __forceinline__ void ksum_tile(int vbid, int mtn, int ntn, int& e, int& mt, int& nt) {
  constexpr int G = 4;
  e = vbid / (mtn * ntn);
  const int rem = vbid - e * (mtn * ntn);
  const int g = rem / (G * ntn), rg = rem - g * (G * ntn);
  const int gm = min(G, mtn - g * G);  // m tiles in this group
  nt = rg / gm;
  mt = g * G + (rg - nt * gm);
}

// Tile of dispatch position P (blocks go to the 8 XCDs round-robin: position
// P runs on XCD P % 8, as its (P / 8)-th block) in an nrows x ncols grid of
// output tiles walked in blocks of (at most) 16 x 16 tiles, row block by row
// block. XCD x takes a sub-block of each block, m tile fastest: split 4 x 2
// (rows (x % 4) r/4 .., columns (x / 4) c/2 ..) when the block's r rows and
// c columns allow it, else 8 x 1 or 1 x 8, else the block is walked m tile
// fastest. A full block's 256 tiles are one round of all 256 CUs: inside an
// XCD the 32 tiles running together share 12 operand panels through its L2,
// and across XCDs every B panel is read by four XCDs and every A panel by
// two at about the same time, so that the Infinity Cache serves the
// repeats instead of HBM (with each XCD on a range of its own, the XCDs
// stream eight different experts' weights at once). Every block starts at a
// multiple of 16, so its positions j have j % 8 == P % 8.
__device__ __forceinline__ void shared_block_tile(int P, int nrows, int ncols, int& mt, int& nt) {
  constexpr int SB = 16;
  const int rb = P / (SB * ncols);
  const int r = min(SB, nrows - rb * SB);   // rows of this row block
  const int Pr = P - rb * SB * ncols;       // position inside the row block
  const int cb = Pr / (r * SB);
  const int c = min(SB, ncols - cb * SB);   // columns of this block
  const int j = Pr - cb * r * SB;           // position inside the r x c block
  const int gr = (r % 4 == 0 && c % 2 == 0) ? 4 : (r % 8 == 0) ? 8 : (c % 8 == 0) ? 1 : 0;
  int lr, lc;
  if (gr != 0) {
    const int gc = 8 / gr, sr = r / gr, sc = c / gc;  // sub-block of sr x sc tiles per XCD
    const int x = j & 7, s = j >> 3;
    lr = (x % gr) * sr + s % sr;
    lc = (x / gr) * sc + s / sr;
  } else {
    lr = j % r;
    lc = j / r;
  }
  mt = rb * SB + lr;
  nt = cb * SB + lc;
}

// Epilogue shared by the bf16 kernels: the accumulators of wave (wm, wn)
// of the tile (each WM x WN, acc[i][j][4*g + q] = C[row wm*WM + i*32 + lane%32]
// [col wn*WN + j*32 + 8*g + 4*(lane/32) + q]) to global memory, staged
// through LDS (smem: SMEM free bytes, at least (NT/64)*64*WN floats).
template <int MODE, int EPI, int BM, int BN, int NT, int SMEM, int WM, int WN>
__device__ __forceinline__ void gemm_epilogue(const GemmParams& p, floatx16 (&acc)[WM / 32][WN / 32],
                                              char* smem, int e, int mt, int n0, int row0,
                                              int rows_e, int cnt_e, int wm, int wn) {
  constexpr int FM = WM / 32, FN = WN / 32;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // acc[i][j][4*g + q] is C[row wm*WM + i*32 + lane%32]
  //                        [col wn*WN + j*32 + 8*g + 4*(lane/32) + q], q = 0..3
  const int lrow = lane & 31, lcol = 4 * (lane >> 5);
  {
    // The wave's WM x WN tile goes out 64 rows at a time through its own LDS
    // region (fp32, 16-byte chunks XOR-swizzled by row), then each lane
    // writes 8 consecutive outputs of one row: full 128-byte lines (bf16
    // rows of the dispatched buffers, or fp32 rows of the weight gradients).
    // The main loop ended with a barrier, so the tile buffers are free.
    static_assert(FM % 2 == 0, "staged epilogue works on 64-row halves");
    constexpr int SCH = WN / 4;  // 16-byte chunks per staged row
    static_assert((NT / 64) * 64 * WN * 4 <= SMEM, "stage does not fit");
    float* stage = reinterpret_cast<float*>(smem) + wave * 64 * WN;
    bf16_t* C0 = static_cast<bf16_t*>(p.C0);
    bf16_t* C1 = static_cast<bf16_t*>(p.C1);
    const bf16_t* aux = static_cast<const bf16_t*>(p.aux);
    auto sidx = [&](int r, int c4) { return r * WN + ((c4 ^ (r & (SCH - 1))) << 2); };
    // forward biases: a lane's items all lie in one 8-column group (the item
    // index is it * 64 + lane and 64 is a multiple of the groups per row), so
    // its 8 (dual: 2 x 8) bias values are loaded once, before any store (a
    // wait for a load issued after stores would wait for those stores too)
    constexpr bool BIASED = MODE == MODE_ROWS && (EPI == EPI_STORE || EPI == EPI_GELU_FWD ||
                                                  EPI == EPI_SWIGLU_FWD);
    float bias0[8], bias1[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) bias0[q] = bias1[q] = 0.f;
    if constexpr (BIASED) {
      if (p.bias0 != nullptr || p.bias1 != nullptr) {
        int n;
        if constexpr (EPI == EPI_SWIGLU_FWD) {
          constexpr int G8 = WN / 16;
          static_assert(64 % G8 == 0, "one column group per lane");
          const int c8 = lane % G8;
          n = n0 + wn * (WN / 2) + (c8 >> 2) * 32 + (c8 & 3) * 8;
        } else {
          constexpr int G8 = WN / 8;
          static_assert(64 % G8 == 0, "one column group per lane");
          n = n0 + wn * WN + (lane % G8) * 8;
        }
        if (n < p.N) {
          if (p.bias0 != nullptr) load8(p.bias0 + (long)e * p.bias_estride + n, bias0);
          if (p.bias1 != nullptr) load8(p.bias1 + (long)e * p.bias_estride + n, bias1);
        }
      }
    }
#pragma unroll
    for (int hf = 0; hf < FM / 2; ++hf) {
      // activation-backward epilogues read the saved pre-activations: all of
      // this half's loads go out before the staging, and none waits behind
      // an output store (one memory round trip per half, not one per item)
      constexpr bool AUXB = MODE == MODE_ROWS &&
                            (EPI == EPI_GELU_BWD || EPI == EPI_SWIGLU_BWD || EPI == EPI_ADD);
      constexpr int AG8 = WN / 8, APER = AUXB ? AG8 : 1;
      Raw8b hr[APER], h3r[APER];
      if constexpr (AUXB) {
#pragma unroll
        for (int it = 0; it < APER; ++it) {
          const int item = it * 64 + lane;
          const int rr = item / AG8, c8 = item % AG8;
          const int ti = wm * WM + hf * 64 + rr;
          const int n = n0 + wn * WN + c8 * 8;
          const bool ok = mt * BM + ti < rows_e && n < p.N;
          const long off = ok ? (long)(row0 + ti) * p.ldaux + n : 0;  // (clamped: every load issued)
          hr[it] = raw8_load(aux + off);
          if constexpr (EPI == EPI_SWIGLU_BWD) h3r[it] = raw8_load(aux + off + (ok ? p.Hh : 0));
        }
      }
#pragma unroll
      for (int i2 = 0; i2 < 2; ++i2)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            const int r = i2 * 32 + lrow, c4 = (j * 32 + 8 * gq + lcol) >> 2;
            const floatx16& a = acc[hf * 2 + i2][j];
            *reinterpret_cast<float4*>(stage + sidx(r, c4)) =
                make_float4(a[4 * gq], a[4 * gq + 1], a[4 * gq + 2], a[4 * gq + 3]);
          }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      auto read8 = [&](int r, int c8, float v[8]) {
        const float4 lo = *reinterpret_cast<const float4*>(stage + sidx(r, 2 * c8));
        const float4 hi = *reinterpret_cast<const float4*>(stage + sidx(r, 2 * c8 + 1));
        v[0] = lo.x; v[1] = lo.y; v[2] = lo.z; v[3] = lo.w;
        v[4] = hi.x; v[5] = hi.y; v[6] = hi.z; v[7] = hi.w;
      };
      if constexpr (EPI == EPI_SWIGLU_FWD) {
        // column pairs (W1, W3) of 32 each: WN/2 distinct outputs per row
        constexpr int G8 = WN / 16;        // 8-column groups of distinct outputs per row
        constexpr int PER = 64 * G8 / 64;  // items per lane
#pragma unroll
        for (int it = 0; it < PER; ++it) {
          const int item = it * 64 + lane;
          const int rr = item / G8, c8 = item % G8;  // c8: 8-group among the distinct columns
          const int jp = c8 >> 2, cin = (c8 & 3) * 8;  // pair and offset inside its 32
          const int ti = wm * WM + hf * 64 + rr;
          const int li = mt * BM + ti;
          const int n = n0 + wn * (WN / 2) + jp * 32 + cin;
          if (li >= rows_e || n >= p.N) continue;
          const bool data = li < cnt_e;
          float h1[8], h3[8], a[8];
          read8(rr, (jp * 64 + cin) >> 3, h1);
          read8(rr, (jp * 64 + 32 + cin) >> 3, h3);
          if (data) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              h1[q] += bias0[q];
              h3[q] += bias1[q];
            }
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            if (!data) h1[q] = h3[q] = 0.f;
            a[q] = silu_f(h1[q]) * h3[q];
          }
          const long g = row0 + ti;
          store8(C0 + g * p.ldc + n, h1);
          store8(C0 + g * p.ldc + p.Hh + n, h3);
          store8(C1 + g * p.ldc1 + n, a);
        }
      } else if constexpr (MODE == MODE_KSUM) {  // fp32 weight gradient, C0 | C1 split at nsplit
        // 16-byte items of 4 columns, WN / 4 to a staged row: a row's WN * 4
        // bytes are written by consecutive lanes, so every store instruction
        // writes whole 128-byte lines (of 64 / (WN / 4) rows); items of 8
        // columns had left a 16-byte gap between the lanes of each store
        constexpr int G4 = WN / 4;
        constexpr int PER = 64 * G4 / 64;
        constexpr int PB = PER >= 8 ? 8 : PER;  // items per batch of accumulation loads
        float* D0 = static_cast<float*>(p.C0);
        float* D1 = static_cast<float*>(p.C1);
        auto dst_of = [&](int it, bool& ok) {
          const int item = it * 64 + lane;
          const int rr = item / G4, c4 = item % G4;
          const int m = mt * BM + wm * WM + hf * 64 + rr;
          const int n = n0 + wn * WN + c4 * 4;
          ok = m < p.Mdim && n < p.N;  // N and nsplit are multiples of 8
          return (n < p.nsplit) ? D0 + (long)e * p.c_estride + (long)m * p.ldc + n
                                : D1 + (long)e * p.c_estride + (long)m * p.ldc + (n - p.nsplit);
        };
#pragma unroll
        for (int b0 = 0; b0 < PER; b0 += PB) {
          // accumulation: the batch's old values are all loaded before any
          // store (from clamped addresses), one memory round trip per batch
          float4 old[PB];
          if (p.accumulate) {
#pragma unroll
            for (int i = 0; i < PB; ++i) {
              bool ok;
              float* d = dst_of(b0 + i, ok);
              old[i] = *reinterpret_cast<const float4*>(ok ? d : D0);
            }
          }
#pragma unroll
          for (int i = 0; i < PB; ++i) {
            const int it = b0 + i;
            bool ok;
            float* dst = dst_of(it, ok);
            if (!ok) continue;
            const int item = it * 64 + lane;
            float4 v = *reinterpret_cast<const float4*>(stage + sidx(item / G4, item % G4));
            if (p.accumulate) {
              v.x += old[i].x;
              v.y += old[i].y;
              v.z += old[i].z;
              v.w += old[i].w;
            }
            *reinterpret_cast<float4*>(dst) = v;
          }
        }
      } else {
        constexpr int G8 = WN / 8;
        constexpr int PER = 64 * G8 / 64;
#pragma unroll
        for (int it = 0; it < PER; ++it) {
          const int item = it * 64 + lane;
          const int rr = item / G8, c8 = item % G8;
          const int ti = wm * WM + hf * 64 + rr;
          const int li = mt * BM + ti;
          const int n = n0 + wn * WN + c8 * 8;
          if (li >= rows_e || n >= p.N) continue;
          const bool data = li < cnt_e;
          float v[8];
          read8(rr, c8, v);
          if (!data) {
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = 0.f;
          }
          if constexpr (EPI == EPI_STORE || EPI == EPI_GELU_FWD) {
            if (data) {
#pragma unroll
              for (int q = 0; q < 8; ++q) v[q] += bias0[q];
            }
          }
          const long g = row0 + ti;
          if constexpr (EPI == EPI_STORE) {
            store8(C0 + g * p.ldc + n, v);
          } else if constexpr (EPI == EPI_ADD) {
            float o[8];
            raw8_f32(hr[it], o);
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] += o[q];
            store8(C0 + g * p.ldc + n, v);
          } else if constexpr (EPI == EPI_GELU_FWD) {
            float a[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) a[q] = gelu_f(v[q]);
            store8(C0 + g * p.ldc + n, v);
            store8(C1 + g * p.ldc1 + n, a);
          } else if constexpr (EPI == EPI_GELU_BWD) {
            float h[8];
            raw8_f32(hr[it], h);
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] *= gelu_grad_f(h[q]);
            store8(C0 + g * p.ldc + n, v);
          } else if constexpr (EPI == EPI_SWIGLU_BWD) {
            float h1[8], h3[8], d3[8];
            raw8_f32(hr[it], h1);
            raw8_f32(h3r[it], h3);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              const float sg = sigmoid_f(h1[q]);
              d3[q] = v[q] * h1[q] * sg;
              v[q] = v[q] * h3[q] * sg * (1.f + h1[q] * (1.f - sg));
            }
            store8(C0 + g * p.ldc + n, v);
            store8(C0 + g * p.ldc + p.Hh + n, d3);
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
}

template <int MODE, bool A_KC, bool B_KC, int EPI, int BM, int BN, int NT>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmParams p) {
  constexpr int WGN = NT / 128;  // waves along N (two along M)
  constexpr int WM = BM / 2, WN = BN / WGN;
  constexpr int FM = WM / 32, FN = WN / 32;
  static_assert(EPI != EPI_SWIGLU_FWD || (FN % 2) == 0, "dual forward needs W1/W3 column pairs");
  __shared__ __attribute__((aligned(16))) char smem[2 * (BM + BN) * 128];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int vbid = xcd_remap(blockIdx.x, gridDim.x);

  // ---- which tile --------------------------------------------------------
  int e = 0, mt = 0, nt = 0, row0 = 0, rows_e = 0, cnt_e = 0;
  if constexpr (MODE == MODE_ROWS) {
    // column tiles fastest: concurrent blocks share the A rows of one tile
    const int ntn = p.ntiles;
    nt = vbid % ntn;
    const int ml = vbid / ntn;
    int acc_t = 0;
    mt = -1;
    for (e = 0; e < p.E; ++e) {
      const int c = seg_count(p, 0, e);
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
    rows_e = clip_rows(seg_offset(p, 0, e), rows_e, p.rows_cap);
    cnt_e = clip_rows(seg_offset(p, 0, e), cnt_e, p.rows_cap);
    row0 = seg_offset(p, 0, e) + mt * BM;  // first global row of this tile
  } else {
    ksum_tile(vbid, (p.Mdim + BM - 1) / BM, (p.N + BN - 1) / BN, e, mt, nt);
    cnt_e = clip_rows(seg_offset(p, 0, e), seg_count(p, 0, e), p.rows_cap);
    row0 = seg_offset(p, 0, e);
  }
  constexpr int NCOLS = (EPI == EPI_SWIGLU_FWD) ? BN / 2 : BN;  // distinct output columns per tile
  const int n0 = nt * NCOLS;

  // ---- loaders -------------------------------------------------------------
  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* B0 = static_cast<const bf16_t*>(p.B0);
  const bf16_t* B1 = static_cast<const bf16_t*>(p.B1);
  int Kred;  // reduction length
  if constexpr (MODE == MODE_ROWS) Kred = p.K; else Kred = cnt_e;

  KcLoader<BM, NT> la;
  MncLoader<BM, NT> lam;
  if constexpr (A_KC) {  // ROWS: A rows are the expert's rows
    const bf16_t* a0 = A + (long)row0 * p.lda;
    la.init(a0, a0, p.lda, cnt_e - mt * BM);
  } else {  // KSUM: A[i][k] = A[(row0 + k) * lda + m0 + i]
    lam.kg = tid % MncLoader<BM, NT>::KG;
    lam.g = tid / MncLoader<BM, NT>::KG;
    const int i0 = mt * BM + lam.g * 8;
    lam.ok = i0 < p.Mdim;
    lam.ld = p.lda;
    lam.col = A + (long)row0 * p.lda + i0;
  }
  KcLoader<BN, NT> lb;
  MncLoader<BN, NT> lbm;
  if constexpr (B_KC) {  // ROWS dgrad: B[k][n] at B + e*estride + n*ldb + k
    const bf16_t* b0 = B0 + (long)e * p.b_estride + (long)n0 * p.ldb;
    const bf16_t* b1 = (B1 != nullptr) ? B1 + (long)e * p.b_estride + (long)n0 * p.ldb : b0;
    lb.init(b0, b1, p.ldb, p.N - n0);
  } else {
    lbm.kg = tid % MncLoader<BN, NT>::KG;
    lbm.g = tid / MncLoader<BN, NT>::KG;
    lbm.ld = p.ldb;
    if constexpr (MODE == MODE_ROWS) {
      const bf16_t* base = B0;
      int n = n0 + lbm.g * 8;
      if constexpr (EPI == EPI_SWIGLU_FWD) {
        const int cc = lbm.g * 8;  // tile column: 32-column blocks alternate W1 / W3
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
    // fragments of step kk+1 are read while the MFMAs of step kk run
    bf16x8 af[2][FM], bfr[2][FN];
    auto read_frags = [&](int kk, int set) {
      const int ch = kk * 2 + (lane >> 5);
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[set][i] = *reinterpret_cast<const bf16x8*>(a_s + lds_off(wm * WM + i * 32 + (lane & 31), ch));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[set][j] = *reinterpret_cast<const bf16x8*>(b_s + lds_off(wn * WN + j * 32 + (lane & 31), ch));
    };
    read_frags(0, 0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      if (kk + 1 < BK / 16) read_frags(kk + 1, (kk + 1) & 1);
      // B as the first operand: the result tile is C^T, so each lane ends up
      // with 4 consecutive output columns of one row
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[kk & 1][j], af[kk & 1][i],
                                                              acc[i][j], 0, 0, 0);
    }
    if (more) store_tiles((kt + 1) & 1);
    __syncthreads();
  }

  gemm_epilogue<MODE, EPI, BM, BN, NT, (int)sizeof(smem), WM, WN>(p, acc, smem, e, mt, n0, row0, rows_e,
                                                                   cnt_e, wm, wn);
}

// ---------------------------------------------------------------------------
// bf16 kernel with direct-to-LDS operand streaming
// ---------------------------------------------------------------------------
// 256 x 256 block tile, 512 threads (2 x 4 waves of 128 x 64), BK = 32, a
// ring of 4 LDS stages (32 KB each: A then B). Operands go global -> LDS with
// bounds-checked buffer_load_dwordx4 ... lds (no staging registers; reads
// past a buffer's range return zeros, which masks ragged expert rows and the
// ragged reduction of the weight gradients). Each wave load fills one 1 KB
// block of LDS in lane order; the source chunk of each lane is chosen so the
// block holds the swizzled layout:
//   K-contiguous operand: [256 rows][32 k] (64 B rows), chunk c of row r at
//     physical chunk c ^ ((r / 4) % 4); fragments via ds_read_b128.
//   M/N-contiguous operand: panels of [32 k][PW cols] (PW*2 B rows), 16-byte
//     chunk m of row k at m ^ (4 * (k % 4)); fragments via two
//     ds_read_b64_tr_b16, which hand lane l' of each 16-lane group element
//     l' % 4 of lane 4q + l'/4 in slot q: lanes aimed at rows k0 + s/4,
//     columns c0 + 4 (s % 4) receive the K-contiguous 4-vectors the MFMA wants.
// Requires the reduction length of the row mode to be a multiple of 32.
constexpr int DBK = 32;
constexpr int kRowGroup = 4;  // row tiles per group of the row-mode tile order

template <int V>
struct IntC {
  static constexpr int value = V;
};

// inclusive prefix sum of v over the lanes of a wave
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  return v;
}

// Row-mode tile of the streaming kernel for block `bid`. The row tiles fall
// in two classes: heavy ones (at least half a tile of live rows) and light
// ones (an expert's short last tile, or padding only). Every XCD (blocks are
// dispatched round-robin over the 8 XCDs) takes an equal share of each class
// and runs its heavy tiles first, so that the light tiles make up the last,
// partial round on every XCD instead of a full-cost round on some. The heavy
// tiles (the experts' heavy row tiles one after the other x the column
// tiles) are walked in shared 16 x 16 blocks (shared_block_tile); inside the
// light class, consecutive tiles walk kRowGroup row tiles x the column
// tiles, row tiles fastest. Returns false for a block with no tile.
template <int BM>
__device__ __forceinline__ bool row_tile_of_block(const GemmParams& p, int bid, int& e, int& mt,
                                                  int& nt, int& rows_e, int& cnt_e, int& off_e) {
  // lane x holds expert x (E <= 64): its count and first row are loaded
  // together (one memory round trip), its tile counts per class summed over
  // the lanes by a prefix scan, and the block's expert found by a ballot
  // (a walk over the experts in scalar registers cost ~0.15 us per expert)
  const int lane = threadIdx.x & 63;
  const bool live = lane < p.E;
  const int c = live ? seg_count(p, 0, lane) : 0;
  const int o = live ? seg_offset(p, 0, lane) : 0;
  const int r = live ? (p.padC ? p.padC : c) : 0;
  const int te = (r + BM - 1) / BM;
  // heavy row tiles of this expert (joined order: all of them)
  const int he = p.joined ? te : min(te, (c + BM / 2) / BM);
  const int le = te - he;                     // light ones
  const int hin = wave_incl_scan(he), lin = wave_incl_scan(le);
  const int HR = __builtin_amdgcn_readlane(hin, 63), LR = __builtin_amdgcn_readlane(lin, 63);
  const int x = bid & 7, i = bid >> 3;
  const int H = HR * p.ntiles, L = LR * p.ntiles;
  const int hx = (H >> 3) + (x < (H & 7)), lx = (L >> 3) + (x < (L & 7));
  bool heavy;
  int ml;
  if (i < hx) {
    heavy = true;
    shared_block_tile(i * 8 + x, HR, p.ntiles, ml, nt);  // (i * 8 + x < H)
  } else if (i < hx + lx) {
    heavy = false;
    const int idx = x * (L >> 3) + min(x, L & 7) + (i - hx);
    const int gsz = kRowGroup * p.ntiles;
    const int g = idx / gsz, rg = idx - g * gsz;
    const int gm = min(kRowGroup, LR - g * kRowGroup);  // row tiles in this group
    nt = rg / gm;
    ml = g * kRowGroup + (rg - nt * gm);
  } else {
    return false;
  }
  // the expert whose range of class tiles holds ml: the one lane with
  // (inclusive sum - own count) <= ml < inclusive sum
  const int inc = heavy ? hin : lin, own = heavy ? he : le;
  const uint64_t hit = __ballot(live && ml < inc && ml >= inc - own);
  if (hit == 0) return false;
  e = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(hit));
  mt = (heavy ? 0 : __builtin_amdgcn_readlane(he, e)) + ml -
       (__builtin_amdgcn_readlane(inc, e) - __builtin_amdgcn_readlane(own, e));
  rows_e = __builtin_amdgcn_readlane(r, e);
  cnt_e = __builtin_amdgcn_readlane(c, e);
  off_e = __builtin_amdgcn_readlane(o, e);
  return true;
}

// grid of the streaming kernel in row mode: ceil(tiles / 8) + 1 blocks per
// XCD cover any split of the tile bound into the two classes
__host__ __device__ constexpr long row_mode_blocks(long tile_bound) { return 8 * ((tile_bound + 7) / 8 + 1); }

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;
typedef __attribute__((address_space(3))) void lds_void_t;

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (stride 0, byte offsets) whose range check covers
// `bytes` from `base`: loads past it return zeros.
__device__ __forceinline__ u32x4 make_rsrc(const void* base, long bytes) {
  const unsigned long a = reinterpret_cast<unsigned long>(base);
  const unsigned n = bytes <= 0 ? 0u : (bytes > 0x7FFFFFFFL ? 0x7FFFFFFFu : (unsigned)bytes);
  u32x4 d;
  d.x = __builtin_amdgcn_readfirstlane((unsigned)a);
  d.y = __builtin_amdgcn_readfirstlane((unsigned)(a >> 32) & 0xFFFFu);
  d.z = __builtin_amdgcn_readfirstlane(n);
  d.w = 0x00020000u;
  return d;
}

// One wave: 64 x 16 bytes from the buffer (per-lane byte offset voff) into
// the 1 KB LDS block at LDS byte address m0v (wave-uniform, computed in
// scalar registers: a vector-to-scalar move per load had put a dependent
// chain in front of every load), lane-ordered. Issued as inline assembly so
// that the compiler does not pair it with the LDS reads of other stages: the
// kernel orders them itself with s_waitcnt vmcnt and barriers.
__device__ __forceinline__ void dma16(u32x4 d, unsigned m0v, unsigned voff) {
  // the descriptor is wave-uniform; say so, so that it sits in scalar registers
  d.x = __builtin_amdgcn_readfirstlane(d.x);
  d.y = __builtin_amdgcn_readfirstlane(d.y);
  d.z = __builtin_amdgcn_readfirstlane(d.z);
  d.w = __builtin_amdgcn_readfirstlane(d.w);
  unsigned saved;  // m0 is reserved: keep the compiler's value intact
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(d), "s"(m0v)
      : "memory");
}


// wait until at most n vector-memory operations and no LDS operation of this
// wave are outstanding
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ int kc_off(int row, int chunk) {
  return row * 64 + (((chunk ^ (row >> 2)) & 3) << 4);
}

// K-contiguous fragment: row `row`, k16 step kk
__device__ __forceinline__ bf16x8 frag_kc(const char* region, int row, int kk, int lane) {
  return *reinterpret_cast<const bf16x8*>(region + kc_off(row, kk * 2 + (lane >> 5)));
}

// M/N-contiguous fragment of 32 columns starting at tile column cb
template <int PW>
__device__ __forceinline__ bf16x8 frag_mnc(const char* region, int cb, int kk, int lane) {
  const int G = lane >> 4, sl = lane & 15;
  const int col = cb + (G & 1) * 16 + 4 * (sl & 3);
  const int pc = col % PW;
  const char* pb = region + (col / PW) * (DBK * PW * 2);
  v4i16 h[2];
#pragma unroll
  for (int ins = 0; ins < 2; ++ins) {
    const int k = kk * 16 + (G >> 1) * 8 + 4 * ins + (sl >> 2);
    const char* a = pb + k * (PW * 2) + ((((pc >> 3) ^ ((k & 3) << 2))) << 4) + ((pc & 7) << 1);
    h[ins] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)a);
  }
  const v4i16 lo = h[0], hi = h[1];
  const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

template <int MODE, bool A_KC, bool B_KC, int EPI, bool NARROW>
__global__ __launch_bounds__(NARROW ? 256 : 512, 2) void gemm_dma_kernel(GemmParams p) {
  // Waves of 128 x 64 accumulators, two along M:
  //   wide:   256 x 256 tiles, 8 waves, 4 stages of the k-tile ring (128 KB
  //           of LDS, one block per CU);
  //   narrow: 256 x 128 tiles, 4 waves, 3 stages (72 KB, up to two blocks per
  //           CU), for launches whose wide tiles would leave CUs idle.
  constexpr int BM = 256, BN = NARROW ? 128 : 256, NT = NARROW ? 256 : 512;
  constexpr int WGM = 2, WGN = NARROW ? 2 : 4;
  constexpr int NW = NT / 64;          // waves
  constexpr int NST = NARROW ? 3 : 4;  // stages of the k-tile ring
  constexpr int A_BYTES = BM * DBK * 2, STB = A_BYTES + BN * DBK * 2;  // bytes per stage
  constexpr int BPA = (BM / 16) / NW, BPB = (BN / 16) / NW;  // 1 KB blocks per wave per stage
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  constexpr bool DUAL = EPI == EPI_SWIGLU_FWD;
  static_assert(!DUAL || !NARROW, "the dual forward pairs 128-column W1 and W3 panels");
  constexpr int PWB = DUAL ? 128 : BN;  // B panel width (M/N-contiguous B)
  // the k-tile ring, reused by the epilogue's staging (64 fp32 rows per wave)
  constexpr int SMEM = NST * STB > NW * 64 * WN * 4 ? NST * STB : NW * 64 * WN * 4;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // the LDS-DMA destinations in scalar registers: the ring's LDS address and
  // the wave index (both wave-uniform)
  const unsigned lds0 = __builtin_amdgcn_readfirstlane((unsigned)(size_t)(lds_void_t*)smem);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);

  // ---- which tile ----
  int e = 0, mt = 0, nt = 0, row0 = 0, rows_e = 0, cnt_e = 0;
  int seg_o = 0, seg_c = 0;  // KSUM: segment ranges, one lane per segment
  if constexpr (MODE == MODE_ROWS) {
    int off_e = 0;
    if (!row_tile_of_block<BM>(p, blockIdx.x, e, mt, nt, rows_e, cnt_e, off_e)) return;
    rows_e = clip_rows(off_e, rows_e, p.rows_cap);
    cnt_e = clip_rows(off_e, cnt_e, p.rows_cap);
    row0 = off_e + mt * BM;
  } else {
    // expert e's mtn x ntn tiles, walked in shared 16 x 16 blocks
    const int mtn = (p.Mdim + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
    e = blockIdx.x / (mtn * ntn);
    shared_block_tile(blockIdx.x - e * (mtn * ntn), mtn, ntn, mt, nt);
    // lane g holds segment g's first row and count of this expert (g < 64):
    // every segment's range in one memory round trip
    const int g = lane;
    seg_o = g < p.nseg ? seg_offset(p, g, e) : 0;
    seg_c = g < p.nseg ? seg_count(p, g, e) : 0;
    row0 = __builtin_amdgcn_readlane(seg_o, 0);
    cnt_e = clip_rows(row0, __builtin_amdgcn_readlane(seg_c, 0), p.rows_cap);
  }
  constexpr int NCOLS = DUAL ? BN / 2 : BN;
  const int n0 = nt * NCOLS;
  const int Kred = (MODE == MODE_ROWS) ? p.K : cnt_e;
  // a padding-only tile (padded layout) has nothing to reduce: zeros
  int nk = (MODE == MODE_ROWS && cnt_e <= mt * BM) ? 0 : (Kred + DBK - 1) / DBK;

  const bf16_t* A = static_cast<const bf16_t*>(p.A);
  const bf16_t* B0 = static_cast<const bf16_t*>(p.B0);
  const bf16_t* B1 = static_cast<const bf16_t*>(p.B1);

  // ---- buffer resources and per-lane source offsets (bytes, k0 = 0) ----
  // Each wave issues BPA A and BPB B block loads per stage: blocks wave + NW*i.
  // An M/N-contiguous panel of PW columns holds 64 / (PW / 8) k-rows per
  // block, 16-byte chunks XOR-swizzled by k-row.
  auto mnc_off = [&](int b, int pw, long ld) {
    const int cpr = pw / 8, kr = (64 / cpr) * b + lane / cpr;
    const int cm = (lane % cpr) ^ ((kr & 3) << 2);
    return (unsigned)(((long)kr * ld + cm * 8) * 2);
  };
  u32x4 ra, rb0, rb1;
  unsigned aoff[BPA], boff[BPB];
  int a_kstep, b_kstep;  // byte step per k-tile
  if constexpr (A_KC) {  // rows of the expert: [rows][K]
    const long valid = (long)(cnt_e - mt * BM) * p.lda;
    ra = make_rsrc(A + (long)row0 * p.lda, valid * 2);
#pragma unroll
    for (int i = 0; i < BPA; ++i) {
      const int b = wave + NW * i, row = 16 * b + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 2) & 3);
      aoff[i] = (unsigned)(((long)row * p.lda + c * 8) * 2);
    }
    a_kstep = DBK * 2;
  } else {  // KSUM: element (m, r) at A + (row0 + r) * lda + m; one panel of 256
    const int m0 = mt * BM;
    ra = make_rsrc(A + (long)row0 * p.lda + m0, ((long)cnt_e * p.lda - m0) * 2);
#pragma unroll
    for (int i = 0; i < BPA; ++i) aoff[i] = mnc_off(wave + NW * i, 256, p.lda);
    a_kstep = DBK * p.lda * 2;
  }
  if constexpr (B_KC) {  // rows n: [N][K] per expert; k >= ksplit from B1
    const long valid = (long)(p.N - n0) * p.ldb;
    rb0 = make_rsrc(B0 + (long)e * p.b_estride + (long)n0 * p.ldb, valid * 2);
    rb1 = (B1 != nullptr) ? make_rsrc(B1 + (long)e * p.b_estride + (long)n0 * p.ldb, valid * 2) : rb0;
#pragma unroll
    for (int i = 0; i < BPB; ++i) {
      const int b = wave + NW * i, row = 16 * b + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 2) & 3);
      boff[i] = (unsigned)(((long)row * p.ldb + c * 8) * 2);
    }
    b_kstep = DBK * 2;
  } else if constexpr (MODE == MODE_ROWS) {  // weights [K][N] per expert
    const long span = (long)p.K * p.ldb;
    if constexpr (DUAL) {  // panel 0: W1 columns n0.., panel 1: W3 columns n0..
      rb0 = make_rsrc(B0 + (long)e * p.b_estride + n0, (span - n0) * 2);
      rb1 = make_rsrc(B1 + (long)e * p.b_estride + n0, (span - n0) * 2);
#pragma unroll
      for (int i = 0; i < BPB; ++i) boff[i] = mnc_off((wave + NW * i) & 7, 128, p.ldb);
    } else {
      rb0 = make_rsrc(B0 + (long)e * p.b_estride + n0, (span - n0) * 2);
      rb1 = rb0;
#pragma unroll
      for (int i = 0; i < BPB; ++i) boff[i] = mnc_off(wave + NW * i, BN, p.ldb);
    }
    b_kstep = DBK * p.ldb * 2;
  } else {  // KSUM: element (r, n) at B + (row0 + r) * ldb + n
    rb0 = make_rsrc(B0 + (long)row0 * p.ldb + n0, ((long)cnt_e * p.ldb - n0) * 2);
    rb1 = rb0;
#pragma unroll
    for (int i = 0; i < BPB; ++i) boff[i] = mnc_off(wave + NW * i, BN, p.ldb);
    b_kstep = DBK * p.ldb * 2;
  }

  // KSUM: bind segment g (g >= 1) of the reduction: the expert's rows in the
  // g-th chunk's buffers (same per-lane offsets and k steps)
  auto bind_segment = [&](int g) {
    if constexpr (MODE == MODE_KSUM) {
      row0 = g < 64 ? __builtin_amdgcn_readlane(seg_o, g) : seg_offset(p, g, e);
      cnt_e = clip_rows(row0, g < 64 ? __builtin_amdgcn_readlane(seg_c, g) : seg_count(p, g, e),
                        p.rows_cap);
      const bf16_t* Ag = A + g * p.a_sstride;
      const bf16_t* Bg = B0 + g * p.b_sstride;
      const int m0 = mt * BM;
      ra = make_rsrc(Ag + (long)row0 * p.lda + m0, ((long)cnt_e * p.lda - m0) * 2);
      rb0 = make_rsrc(Bg + (long)row0 * p.ldb + n0, ((long)cnt_e * p.ldb - n0) * 2);
      rb1 = rb0;
      nk = (cnt_e + DBK - 1) / DBK;
    }
  };

  // Loads of k-tile kt into stage `stage`, in two parts: part 0 takes this
  // wave's first ceil(n / 2) of its n blocks of each operand, part 1 the rest.
  auto issue_part = [&](int kt, int stage, int q) {
    const unsigned sa = lds0 + (unsigned)(stage * STB), sb = sa + A_BYTES;
    const unsigned ka = (unsigned)kt * (unsigned)a_kstep;
    constexpr int HA = (BPA + 1) / 2, HB = (BPB + 1) / 2;
#pragma unroll
    for (int i = q ? HA : 0; i < (q ? BPA : HA); ++i) dma16(ra, sa + (wave_s + NW * i) * 1024, aoff[i] + ka);
#pragma unroll
    for (int i = q ? HB : 0; i < (q ? BPB : HB); ++i) {
      if constexpr (B_KC) {
        const int k0 = kt * DBK;
        const bool second = k0 >= p.ksplit;
        const unsigned kb = (unsigned)((second ? k0 - p.ksplit : k0) * 2);
        dma16(second ? rb1 : rb0, sb + (wave_s + NW * i) * 1024, boff[i] + kb);
      } else {
        const unsigned kb = (unsigned)kt * (unsigned)b_kstep;
        // blocks 8..15 hold the W3 panel
        const int blk = wave_s + NW * i;
        dma16((DUAL && blk >= 8) ? rb1 : rb0, sb + blk * 1024, boff[i] + kb);
      }
    }
  };
  auto issue = [&](int kt, int stage) {
    issue_part(kt, stage, 0);
    issue_part(kt, stage, 1);
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Ring of NST k-tiles: tile t lives in stage t % NST. Every wave loads its
  // share of each tile; a barrier after a wave's own loads of tile t have
  // landed (s_waitcnt vmcnt) makes the whole tile visible. Tile t's stage is
  // refilled (tile t + NST) only after the barrier that follows every wave's
  // last LDS read of tile t.
  auto prologue = [&] {
#pragma unroll
    for (int s = 0; s < NST; ++s)
      if (s < nk) issue(s, s);
  };

  // wait until this wave's loads of tile t have landed, given that the loads
  // of tiles up to min(t + ahead, nk - 1) have been issued
  constexpr int LPT = BPA + BPB;  // loads per wave per k-tile
  auto wait_tile = [&](int t, int ahead) {
    const int younger = min(ahead, nk - 1 - t);  // tiles issued after t
    if (younger >= 3) wait_vm_lgkm0<3 * LPT>();
    else if (younger == 2) wait_vm_lgkm0<2 * LPT>();
    else if (younger == 1) wait_vm_lgkm0<LPT>();
    else wait_vm_lgkm0<0>();
  };
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // The k loop for a wave whose first FML 32-row fragments hold live rows
  // (FML = FM for every wave of a tile with 256 live rows; the short last
  // tile of an expert skips the MFMAs and A reads of rows past its count).
  auto k_loop = [&](auto fml_c) {
    constexpr int FML = decltype(fml_c)::value;
    // Fragments of one 16-deep k step; two sets so that the LDS reads of the
    // next step are in flight while the MFMAs of the current one run.
    bf16x8 af[2][FM], bfr[2][FN];
    auto read_frags = [&](int stage, int kk, int set) {
      if constexpr (FML > 0) {
        const char* sa = smem + stage * STB;
        const char* sb = sa + A_BYTES;
#pragma unroll
        for (int i = 0; i < FML; ++i) {
          if constexpr (A_KC)
            af[set][i] = frag_kc(sa, wm * WM + i * 32 + (lane & 31), kk, lane);
          else
            af[set][i] = frag_mnc<256>(sa, wm * WM + i * 32, kk, lane);
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (B_KC)
            bfr[set][j] = frag_kc(sb, wn * WN + j * 32 + (lane & 31), kk, lane);
          else if constexpr (DUAL)  // pairs (h1, h3) of 32 columns: W1 panel, W3 panel
            bfr[set][j] = frag_mnc<PWB>(sb, (j & 1) * 128 + wn * (WN / 2) + (j >> 1) * 32, kk, lane);
          else
            bfr[set][j] = frag_mnc<PWB>(sb, wn * WN + j * 32, kk, lane);
        }
      }
    };
    // LDS read instructions per fragment set (ds_read_b128 for a K-contiguous
    // fragment, two ds_read_b64_tr_b16 for an M/N-contiguous one)
    constexpr int NRD = FML == 0 ? 0 : FML * (A_KC ? 1 : 2) + FN * (B_KC ? 1 : 2);
    constexpr int NMF = FML * FN;
    auto mfma_rows = [&](int set, int i0, int i1) {
#pragma unroll
      for (int i = i0; i < i1; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[set][j], af[set][i], acc[i][j], 0, 0, 0);
    };
    // One half k-step: the LDS reads of the next set interleaved with the
    // first half of this set's MFMAs, then one part of a k-tile's loads (if
    // any) between the two halves of the MFMAs, so that the memory pipe takes
    // the loads a few at a time while the matrix pipe stays busy. The
    // scheduling barriers keep the inline-asm loads where they are. A wave
    // issues the second half of its MFMAs at raised priority: of the two
    // waves of a SIMD the older one otherwise ran ahead and then waited at
    // the k-tile barrier for a quarter of the loop while the other finished
    // alone (large layer 32.0 -> 31.4 ms per step; raising it over both
    // halves or the whole half step measured slower).
    auto half_step = [&](int set, auto&& reads, auto&& loads) {
      reads();
      mfma_rows(set, 0, FML / 2);
      if constexpr (NRD > 0) {
#pragma unroll
        for (int q = 0; q < NRD; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, (NMF / 2 + NRD - 1) / NRD, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NMF / 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      loads();
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
      __builtin_amdgcn_sched_barrier(0);
      mfma_rows(set, FML / 2, FML);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
    };

    if (nk > 0) {
      wait_tile(0, NST - 1);
      barrier();
      read_frags(0, 0, 0);
    }
    // All tiles but the last: the barrier sits between the two k steps, so
    // each half pairs the MFMAs of one step with the reads of the next.
    // The loads of tile kt + NST go out in two parts: the first in the
    // second half of iteration kt (its stage was freed by that iteration's
    // barrier), the second in the first half of iteration kt + 1, both before
    // the wait that needs them (iteration kt + NST - 1).
    // Iteration kt of the ring. In the steady state (1 <= kt < nk - NST)
    // every load exists and the wait always leaves the loads of NST - 2
    // tiles in flight: that instance has no branches (a branch per
    // iteration for the wait's count and the loads' bounds cost ~2% on the
    // large layer).
    auto iter = [&](int kt, auto steady_c) {
      constexpr bool S = decltype(steady_c)::value == 1;
      const int stage = kt % NST;
      // step 1 of tile kt is read while step 0 runs; second part of tile kt + NST - 1
      half_step(
          0, [&] { read_frags(stage, 1, 1); },
          [&] {
            const int tl = kt + NST - 1;
            if (S || (tl >= NST && tl < nk)) issue_part(tl, tl % NST, 1);
          });
      // this wave's reads of tile kt are done (lgkmcnt 0) and its loads of
      // tile kt + 1 have landed; after the barrier every wave's have
      if constexpr (S) wait_vm_lgkm0<(NST - 2) * LPT>();
      else wait_tile(kt + 1, NST - 2);
      barrier();
      // step 0 of tile kt + 1 is read while step 1 of tile kt runs; first part
      // of tile kt + NST into the stage tile kt leaves
      half_step(
          1, [&] { read_frags((kt + 1) % NST, 0, 0); },
          [&] {
            if (S || kt + NST < nk) issue_part(kt + NST, stage, 0);
          });
    };
    int kt = 0;
    if (nk > 1) iter(kt++, IntC<0>{});
    for (; kt + NST < nk; ++kt) iter(kt, IntC<1>{});
    for (; kt + 1 < nk; ++kt) iter(kt, IntC<0>{});
    if (nk > 0) {
      read_frags((nk - 1) % NST, 1, 1);
      mfma_rows(0, 0, FML);
      if constexpr (NRD > 0) {
#pragma unroll
        for (int q = 0; q < NRD; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
          __builtin_amdgcn_sched_group_barrier(0x008, (NMF + NRD - 1) / NRD, 0);  // MFMAs
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NMF, 0);  // the rest of the MFMAs
      }
      mfma_rows(1, 0, FML);
    }
  };
  if constexpr (MODE == MODE_KSUM) {
    // every row of a weight-gradient tile is live; segments one after the
    // other into the same accumulators, the ring drained between them
    for (int g = 0; g < p.nseg; ++g) {
      if (g > 0) {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();  // all LDS reads of the last segment done before the refill
        bind_segment(g);
      }
      prologue();
      k_loop(IntC<FM>{});
    }
  } else {
    prologue();
    // live 32-row fragments of this wave (wave-uniform)
    const int live = min(BM, max(0, cnt_e - mt * BM));
    const int fml = __builtin_amdgcn_readfirstlane(min(FM, max(0, (live - wm * WM + 31) / 32)));
    if (fml > FM / 2) k_loop(IntC<FM>{});
    else if (fml > 0) k_loop(IntC<FM / 2>{});
    else k_loop(IntC<0>{});
  }
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();  // all LDS reads done before the epilogue reuses the stages
  gemm_epilogue<MODE, EPI, BM, BN, NT, SMEM, WM, WN>(p, acc, smem, e, mt, n0, row0, rows_e, cnt_e, wm,
                                                     wn);
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
      const int c = seg_count(p, 0, e);
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
    rows_e = clip_rows(seg_offset(p, 0, e), rows_e, p.rows_cap);
    cnt_e = clip_rows(seg_offset(p, 0, e), cnt_e, p.rows_cap);
    row0 = seg_offset(p, 0, e) + mt * TB;
  } else {
    const int mtn = (p.Mdim + TB - 1) / TB, ntn = (p.N + TB - 1) / TB;
    e = blockIdx.x / (mtn * ntn);
    const int rem = blockIdx.x % (mtn * ntn);
    mt = rem / ntn;
    nt = rem % ntn;
    cnt_e = clip_rows(seg_offset(p, 0, e), seg_count(p, 0, e), p.rows_cap);
    row0 = seg_offset(p, 0, e);
  }
  const int n0 = nt * TB;
  const float* A = static_cast<const float*>(p.A);
  const float* B0 = static_cast<const float*>(p.B0);
  const float* B1 = static_cast<const float*>(p.B1);
  const int ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  // KSUM: segments (chunks) one after the other into the same accumulators
  const int nseg = (MODE == MODE_KSUM) ? p.nseg : 1;
  for (int g = 0; g < nseg; ++g) {
    if (g > 0) {
      row0 = seg_offset(p, g, e);
      cnt_e = clip_rows(row0, seg_count(p, g, e), p.rows_cap);
      A = static_cast<const float*>(p.A) + g * p.a_sstride;
      B0 = static_cast<const float*>(p.B0) + g * p.b_sstride;
    }
    const int Kred = (MODE == MODE_ROWS) ? p.K : cnt_e;
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
        float v = (li < cnt_e) ? acc[i][j] : 0.f;
        if constexpr (EPI == EPI_STORE || EPI == EPI_GELU_FWD) {
          if (li < cnt_e && p.bias0 != nullptr) v += p.bias0[(long)e * p.bias_estride + n];
        }
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
  const long live = padded ? rows : min((long)offsets[E], rows);  // (cut at the buffers)
  const long n = live * H;
  for (long q = blockIdx.x * (long)blockDim.x + threadIdx.x; q < n; q += (long)gridDim.x * blockDim.x) {
    const long r = q / H;
    const int c = (int)(q % H);
    const float h1 = h[r * 2 * H + c], h3 = h[r * 2 * H + H + c];
    a[q] = h1 * sigmoid_f(h1) * h3;
  }
}

// Bias gradients of the experts: per-expert column sums,
// out[e][c] (+)= sum over expert e's rows r of src[r][c], over nseg row
// segments (the chunks of a layer call: segment g's rows of expert e are
// counts[g * E + e] rows from offsets[g * (E + 1) + e] of src + g * seg_stride)
// in segment order; columns at or past nsplit go to out1[e][c - nsplit]
// (SwiGLU's dH3 half), a null output is skipped. Block (512-column block,
// expert): 64 lanes of 8 columns, wave w summing the rows w, w + 4, ... of
// each segment in order (four rows in flight per lane), then the four
// waves' sums added in wave order: deterministic.
// C (+)= the S partial sums of P (S x n4 float4), added in split order
__global__ __launch_bounds__(256) void sum_splits_kernel(const float4* __restrict__ P, int S,
                                                         long n4, float4* __restrict__ C,
                                                         int accumulate) {
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
    float4 a = accumulate ? C[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int s = 0; s < S; ++s) {
      const float4 v = P[s * n4 + i];
      a.x += v.x;
      a.y += v.y;
      a.z += v.z;
      a.w += v.w;
    }
    C[i] = a;
  }
}

template <typename TE>
__global__ __launch_bounds__(256) void bias_grad_kernel(
    const TE* __restrict__ src, long ld, long seg_stride, const int32_t* __restrict__ counts,
    const int32_t* __restrict__ offsets, int E, int nseg, long rows_cap, int ncols, int nsplit,
    float* __restrict__ out0, float* __restrict__ out1, int accumulate) {
  __shared__ float part[4][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int e = blockIdx.y;
  const int c0 = blockIdx.x * 512 + lane * 8;  // ncols is a multiple of 8
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto add = [&](const auto& raw) {
    float v[8];
    raw8_f32(raw, v);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] += v[q];
  };
  if (c0 < ncols) {
    for (int g = 0; g < nseg; ++g) {
      const long off = offsets[g * (E + 1) + e];
      const int n = clip_rows(off, counts[g * E + e], rows_cap);
      const TE* base = src + g * seg_stride + off * ld + c0;
      int r = w;
      for (; r + 12 < n; r += 16) {
        const auto a0 = raw8_load(base + (long)r * ld);
        const auto a1 = raw8_load(base + (long)(r + 4) * ld);
        const auto a2 = raw8_load(base + (long)(r + 8) * ld);
        const auto a3 = raw8_load(base + (long)(r + 12) * ld);
        add(a0);
        add(a1);
        add(a2);
        add(a3);
      }
      for (; r < n; r += 4) add(raw8_load(base + (long)r * ld));
    }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) part[w][lane * 8 + q] = acc[q];
  __syncthreads();
  if (w == 0 && c0 < ncols) {
    float* dst = c0 < nsplit ? out0 : out1;
    if (dst == nullptr) return;
    dst += c0 < nsplit ? (long)e * nsplit + c0 : (long)e * (ncols - nsplit) + (c0 - nsplit);
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q)
      v[q] = ((part[0][lane * 8 + q] + part[1][lane * 8 + q]) + part[2][lane * 8 + q]) +
             part[3][lane * 8 + q];
    if (accumulate) {
      float o[8];
      load8(dst, o);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += o[q];
    }
    store8(dst, v);
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
  p.nseg = 1;
  p.rows_cap = s.rows;
  return p;
}

template <int MODE, bool A_KC, bool B_KC, int EPI, int BM, int BN, int NT>
hipError_t run_bf16(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  long blocks;
  if (MODE == MODE_ROWS) {
    const int ncols = (EPI == EPI_SWIGLU_FWD) ? BN / 2 : BN;
    p.mt_bound = rows_tiles_bound(s, BM);
    p.ntiles = (p.N + ncols - 1) / ncols;
    blocks = (long)p.mt_bound * p.ntiles;
  } else {
    blocks = (long)s.E * ((p.Mdim + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  }
  if (blocks == 0) return hipSuccess;
  return traced(kind, st, [&] {
    hipLaunchKernelGGL((gemm_bf16_kernel<MODE, A_KC, B_KC, EPI, BM, BN, NT>),
                       dim3((unsigned)blocks), dim3(NT), 0, st, p);
  });
}

// Tile shape of the streaming kernel: 256 x 256 unless those tiles would
// cover the launch in at most 1.25 rounds of the CUs, then 256 x 128.
constexpr int kCUs = 256;
std::atomic<int> g_tiles{FLOWMOE_TILES_AUTO};
std::atomic<int> g_tile_order{FLOWMOE_TILE_ORDER_AUTO};

template <int MODE, bool A_KC, bool B_KC, int EPI, bool NARROW>
hipError_t launch_dma(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  constexpr int BN = NARROW ? 128 : 256;
  long blocks;
  if (MODE == MODE_ROWS) {
    const int ncols = (EPI == EPI_SWIGLU_FWD) ? 128 : BN;
    p.mt_bound = rows_tiles_bound(s, 256);
    p.ntiles = (p.N + ncols - 1) / ncols;
    blocks = (s.rows == 0 || p.N == 0) ? 0 : row_mode_blocks((long)p.mt_bound * p.ntiles);
    // joined tile order: the experts' weights stream from HBM (more than the
    // Infinity Cache holds) and each expert spans few row tiles, so a light
    // tile run after all heavy ones would read its weight panels from HBM
    // again; with many row tiles per expert, or weights that stay cached,
    // running the light tiles last packs the rounds better (measured: fine
    // layer 7.63 -> 7.26 ms per step joined, balanced 0.68 -> 0.74 and large
    // 32.2 -> 32.7 ms)
    const double wbytes = 2.0 * s.E * (double)p.K * p.N * (EPI == EPI_SWIGLU_FWD ? 2 : 1);
    const int order = g_tile_order.load(std::memory_order_relaxed);
    p.joined = order == FLOWMOE_TILE_ORDER_JOINED ||
               (order == FLOWMOE_TILE_ORDER_AUTO && wbytes > 256.0 * 1024 * 1024 &&
                s.rows <= 2048L * s.E);
  } else {
    blocks = (long)s.E * ((p.Mdim + 255) / 256) * ((p.N + BN - 1) / BN);
  }
  if (blocks == 0) return hipSuccess;
  return traced(kind, st, [&] {
    hipLaunchKernelGGL((gemm_dma_kernel<MODE, A_KC, B_KC, EPI, NARROW>), dim3((unsigned)blocks),
                       dim3(NARROW ? 256 : 512), 0, st, p);
  });
}

template <int MODE, bool A_KC, bool B_KC, int EPI>
hipError_t run_dma(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  if constexpr (EPI == EPI_SWIGLU_FWD) {
    return launch_dma<MODE, A_KC, B_KC, EPI, false>(kind, s, p, st);
  } else {
    // wide tiles the launch would have (row mode: the live rows' tiles)
    const long rt = (MODE == MODE_ROWS) ? (s.rows + 255) / 256 : (long)s.E * ((p.Mdim + 255) / 256);
    const long wide = rt * ((p.N + 255) / 256);
    const int tiles = g_tiles.load(std::memory_order_relaxed);
    const bool narrow = tiles == FLOWMOE_TILES_NARROW ||
                        (tiles == FLOWMOE_TILES_AUTO && wide <= kCUs + kCUs / 4);
    if (narrow) return launch_dma<MODE, A_KC, B_KC, EPI, true>(kind, s, p, st);
    return launch_dma<MODE, A_KC, B_KC, EPI, false>(kind, s, p, st);
  }
}

// The streaming kernel needs the row-mode reduction length (and a K split)
// to be a multiple of its 32-deep k-tile; otherwise the register-staged
// kernel runs.
template <int MODE, bool A_KC, bool B_KC, int EPI>
hipError_t run_gemm_bf16(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  if (MODE == MODE_KSUM && p.nseg < 1) return hipErrorInvalidValue;  // (a launcher bug)
  const bool dma_ok = MODE == MODE_KSUM ||
                      (p.K % DBK == 0 && (p.ksplit >= p.K || p.ksplit % DBK == 0));
  if (dma_ok) return run_dma<MODE, A_KC, B_KC, EPI>(kind, s, p, st);
  return run_bf16<MODE, A_KC, B_KC, EPI, 256, 256, 512>(kind, s, p, st);
}

template <int MODE, bool B_KC, int EPI>
hipError_t run_f32(int kind, const Shape& s, GemmParams p, hipStream_t st) {
  if (MODE == MODE_KSUM && p.nseg < 1) return hipErrorInvalidValue;  // (a launcher bug)
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

void set_gemm_tiles(int tiles) { g_tiles.store(tiles, std::memory_order_relaxed); }
void set_tile_order(int order) { g_tile_order.store(order, std::memory_order_relaxed); }

hipError_t launch_gate_dw_gemm(const void* x, int T, int M, const void* d, int N,
                               const int32_t* counts, const int32_t* offsets, int S, float* P,
                               hipStream_t st) {
  Shape s2 = {};
  s2.E = S;
  GemmParams p = {};
  p.counts = counts;
  p.offsets = offsets;
  p.E = S;
  p.A = x;
  p.lda = M;
  p.B0 = d;
  p.ldb = N;
  p.Mdim = M;
  p.N = N;
  p.C0 = P;
  p.C1 = P;
  p.ldc = N;
  p.c_estride = (long)M * N;
  p.nsplit = 1 << 30;
  p.ksplit = 1 << 30;
  p.nseg = 1;
  p.rows_cap = T;
  // 256 x 256 tiles whatever the grid: these launches are bound by reading
  // x once, and the 8-wave tile's deeper ring (4 stages against 3) keeps
  // more of it in flight (the narrow tile took 1.2-1.7x as long)
  return launch_dma<MODE_KSUM, false, false, EPI_GATE_DW, false>(FLOWMOE_K_GATE_BWD_DW, s2, p, st);
}

hipError_t launch_gate_dx_gemm(const void* dlhl, int T, int K, const void* wstack, int M,
                               const int32_t* counts, const int32_t* offsets, int S, void* dx,
                               bool add, hipStream_t st) {
  Shape s2 = {};
  s2.T = T;
  s2.E = S;
  s2.rows = T;
  s2.layout = FLOWMOE_PACKED;
  GemmParams p = {};
  p.counts = counts;
  p.offsets = offsets;
  p.E = S;
  p.A = dlhl;
  p.lda = K;
  p.K = K;
  p.B0 = wstack;  // B[k][n] = wstack[k][n] for every token split (b_estride 0)
  p.ldb = M;
  p.N = M;
  p.C0 = dx;
  p.ldc = M;
  p.aux = dx;     // (EPI_ADD: the values added to)
  p.ldaux = M;
  p.ksplit = 1 << 30;
  p.nsplit = 1 << 30;
  p.nseg = 1;
  p.rows_cap = T;
  if (add)
    return run_gemm_bf16<MODE_ROWS, true, false, EPI_ADD>(FLOWMOE_K_GATE_BWD_TOKEN, s2, p, st);
  return run_gemm_bf16<MODE_ROWS, true, false, EPI_STORE>(FLOWMOE_K_GATE_BWD_TOKEN, s2, p, st);
}

hipError_t launch_dense_gemm(int kind, long rows, const void* A, long lda, int K, const void* B,
                             long ldb, bool b_kc, int N, void* C, long ldc, hipStream_t st) {
  if (rows == 0 || N == 0) return hipSuccess;
  Shape s2 = {};
  s2.T = (int)rows;
  s2.E = 1;
  s2.rows = rows;
  s2.layout = FLOWMOE_PACKED;
  GemmParams p = {};
  p.E = 1;  // (counts null: one expert of rows_cap rows)
  p.A = A;
  p.lda = lda;
  p.K = K;
  p.B0 = B;
  p.ldb = ldb;
  p.N = N;
  p.C0 = C;
  p.ldc = ldc;
  p.ksplit = 1 << 30;
  p.nsplit = 1 << 30;
  p.nseg = 1;
  p.rows_cap = rows;
  if (b_kc) return run_gemm_bf16<MODE_ROWS, true, true, EPI_STORE>(kind, s2, p, st);
  return run_gemm_bf16<MODE_ROWS, true, false, EPI_STORE>(kind, s2, p, st);
}

int dense_wgrad_splits(int Mdim, int N, long rows) {
  const long tiles = (long)((Mdim + 255) / 256) * ((N + 255) / 256);
  const long s = std::min<long>(8, (kCUs + tiles - 1) / tiles);
  return (int)std::max<long>(1, std::min<long>(s, rows / 512));
}

size_t mha_wgrad_ws_bytes(int M) {
  const long big = 1L << 40;  // (any number of rows)
  const int s3 = dense_wgrad_splits(M, 3 * M, big), s1 = dense_wgrad_splits(M, M, big);
  const size_t b3 = s3 > 1 ? (size_t)s3 * M * 3 * M * 4 : 0, b1 = s1 > 1 ? (size_t)s1 * M * M * 4 : 0;
  return align256(std::max(b3, b1));
}

hipError_t launch_dense_wgrad(int kind, long rows, int nseg, const void* A, long lda,
                              long a_sstride, int Mdim, const void* B, long ldb, long b_sstride,
                              int N, float* C, long ldc, int accumulate, float* part,
                              hipStream_t st) {
  // few output tiles for the CUs: the rows of every segment are split S ways
  // into partial sums in `part` (S x Mdim x N), which a reduction adds in
  // split order (deterministic)
  const int S = part ? dense_wgrad_splits(Mdim, N, rows * nseg) : 1;
  Shape s2 = {};
  s2.T = (int)rows;
  s2.E = S;
  s2.rows = rows;
  s2.layout = FLOWMOE_PACKED;
  GemmParams p = {};
  p.E = S;
  p.A = A;
  p.lda = lda;
  p.Mdim = Mdim;
  p.B0 = B;
  p.ldb = ldb;
  p.N = N;
  p.C0 = S > 1 ? part : C;
  p.C1 = p.C0;
  p.ldc = S > 1 ? N : ldc;
  p.c_estride = (long)Mdim * N;
  p.ksplit = 1 << 30;
  p.nsplit = 1 << 30;
  p.accumulate = S > 1 ? 0 : accumulate;
  p.nseg = nseg;
  p.a_sstride = a_sstride;
  p.b_sstride = b_sstride;
  p.rows_cap = rows;
  FLOWMOE_TRY((run_gemm_bf16<MODE_KSUM, false, false, EPI_WGRAD>(kind, s2, p, st)));
  if (S == 1) return hipSuccess;
  const long n4 = (long)Mdim * N / 4;  // (ldc == N here)
  return traced(kind, st, [&] {
    hipLaunchKernelGGL(sum_splits_kernel, dim3((unsigned)std::min<long>(2048, (n4 + 255) / 256)),
                       dim3(256), 0, st, reinterpret_cast<const float4*>(part), S, n4,
                       reinterpret_cast<float4*>(C), accumulate);
  });
}

size_t ffn_bwd_ws_bytes(const Shape& s) {
  const int hw = (s.act == FLOWMOE_SWIGLU) ? 2 * s.H : s.H;
  return align256((size_t)s.rows * hw * esize(s.dtype));
}

hipError_t launch_expert_ffn(const Shape& s, const void* x_disp, const int32_t* counts,
                             const int32_t* offsets, const void* w1, const void* w3,
                             const void* w2, const float* b1, const float* b3, const float* b2,
                             void* h_save, void* a_save, void* y_disp, hipStream_t st) {
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
  p.bias0 = b1;
  p.bias1 = swiglu ? b3 : nullptr;
  p.bias_estride = H;
  if (s.dtype == FLOWMOE_BF16) {
    if (swiglu)
      FLOWMOE_TRY((run_gemm_bf16<MODE_ROWS, true, false, EPI_SWIGLU_FWD>(FLOWMOE_K_FFN1, s, p, st)));
    else
      FLOWMOE_TRY((run_gemm_bf16<MODE_ROWS, true, false, EPI_GELU_FWD>(FLOWMOE_K_FFN1, s, p, st)));
  } else {
    if (swiglu) {
      p.B1 = nullptr;
      FLOWMOE_TRY((run_f32<MODE_ROWS, false, EPI_STORE>(FLOWMOE_K_FFN1, s, p, st)));
      p.B0 = w3;
      p.coloff = H;
      p.bias0 = b3;
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
  q.bias0 = b2;
  q.bias_estride = M;
  if (s.dtype == FLOWMOE_BF16)
    return run_gemm_bf16<MODE_ROWS, true, false, EPI_STORE>(FLOWMOE_K_FFN2, s, q, st);
  return run_f32<MODE_ROWS, false, EPI_STORE>(FLOWMOE_K_FFN2, s, q, st);
}

hipError_t launch_expert_ffn_dgrad(const Shape& s, const void* dy_disp, const void* h_save,
                                   const int32_t* counts, const int32_t* offsets, const void* w1,
                                   const void* w3, const void* w2, void* dh, void* dx_disp,
                                   hipStream_t st) {
  if (s.rows == 0) return hipSuccess;
  const bool swiglu = s.act == FLOWMOE_SWIGLU;
  const bool bf = s.dtype == FLOWMOE_BF16;
  const int H = s.H, M = s.M;
  const int HW = swiglu ? 2 * H : H;
  // 1. dA = dY W2^T, through the activation -> dH (rows x HW); an element's
  // pre-activation is read by the lane that then writes its gradient, so dh
  // may be h_save itself
  {
    GemmParams p = base_params(s, counts, offsets);
    p.A = dy_disp;
    p.lda = M;
    p.K = M;
    p.N = H;
    p.B0 = w2;  // B[k=m][n=h] = W2[e][h][m]: K-contiguous
    p.ldb = M;
    p.b_estride = (long)H * M;
    p.C0 = dh;
    p.ldc = HW;
    p.aux = h_save;
    p.ldaux = HW;
    if (bf) {
      if (swiglu)
        FLOWMOE_TRY((run_gemm_bf16<MODE_ROWS, true, true, EPI_SWIGLU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
      else
        FLOWMOE_TRY((run_gemm_bf16<MODE_ROWS, true, true, EPI_GELU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
    } else {
      if (swiglu)
        FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_SWIGLU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
      else
        FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_GELU_BWD>(FLOWMOE_K_DGRAD1, s, p, st)));
    }
  }
  // 2. dX = dH1 W1^T (+ dH3 W3^T)
  {
    GemmParams p = base_params(s, counts, offsets);
    p.A = dh;
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
      FLOWMOE_TRY((run_gemm_bf16<MODE_ROWS, true, true, EPI_STORE>(FLOWMOE_K_DGRAD2, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_ROWS, true, EPI_STORE>(FLOWMOE_K_DGRAD2, s, p, st)));
  }
  return hipSuccess;
}

hipError_t launch_expert_bias_grad(const Shape& s, int R, const void* dy_disp, const void* dh,
                                   const int32_t* counts, const int32_t* offsets, float* db1,
                                   float* db3, float* db2, int accumulate, hipStream_t st) {
  const bool swiglu = s.act == FLOWMOE_SWIGLU;
  const int H = s.H, M = s.M, HW = swiglu ? 2 * H : H;
  const long rows = s.rows;
  auto run = [&](const void* src, int ld, int ncols, int nsplit, float* o0, float* o1) {
    return traced(FLOWMOE_K_BIAS_GRAD, st, [&] {
      const dim3 grid((unsigned)((ncols + 511) / 512), (unsigned)s.E);
      if (s.dtype == FLOWMOE_BF16)
        hipLaunchKernelGGL(bias_grad_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)src,
                           (long)ld, rows * ld, counts, offsets, s.E, R, rows, ncols, nsplit, o0, o1,
                           accumulate);
      else
        hipLaunchKernelGGL(bias_grad_kernel<float>, grid, dim3(256), 0, st, (const float*)src,
                           (long)ld, rows * ld, counts, offsets, s.E, R, rows, ncols, nsplit, o0, o1,
                           accumulate);
    });
  };
  if (db2 != nullptr) FLOWMOE_TRY(run(dy_disp, M, M, M, db2, nullptr));
  if (db1 != nullptr || (swiglu && db3 != nullptr))
    FLOWMOE_TRY(run(dh, HW, HW, H, db1, swiglu ? db3 : nullptr));
  return hipSuccess;
}

hipError_t launch_expert_ffn_wgrad(const Shape& s, int R, const void* dy_disp, const void* x_disp,
                                   const void* a_save, const void* dh, const int32_t* counts,
                                   const int32_t* offsets, float* dw1, float* dw3, float* dw2,
                                   float* db1, float* db3, float* db2, int accumulate,
                                   hipStream_t st) {
  const bool swiglu = s.act == FLOWMOE_SWIGLU;
  const bool bf = s.dtype == FLOWMOE_BF16;
  const int H = s.H, M = s.M;
  const int HW = swiglu ? 2 * H : H;
  const long rows = s.rows;
  // 1. dW2 = sum over chunks of A^T dY  (H x M per expert)
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
    p.nseg = R;
    p.a_sstride = rows * H;
    p.b_sstride = rows * M;
    if (bf)
      FLOWMOE_TRY((run_gemm_bf16<MODE_KSUM, false, false, EPI_WGRAD>(FLOWMOE_K_WGRAD2, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_KSUM, false, EPI_WGRAD>(FLOWMOE_K_WGRAD2, s, p, st)));
  }
  // 2. [dW1 | dW3] = sum over chunks of X^T [dH1 | dH3]  (M x H per expert, each)
  {
    GemmParams p = base_params(s, counts, offsets);
    p.A = x_disp;
    p.lda = M;
    p.Mdim = M;
    p.B0 = dh;
    p.ldb = HW;
    p.N = HW;
    p.C0 = dw1;
    p.C1 = dw3;
    p.nsplit = H;
    p.ldc = H;
    p.c_estride = (long)M * H;
    p.accumulate = accumulate;
    p.nseg = R;
    p.a_sstride = rows * M;
    p.b_sstride = rows * HW;
    if (bf)
      FLOWMOE_TRY((run_gemm_bf16<MODE_KSUM, false, false, EPI_WGRAD>(FLOWMOE_K_WGRAD1, s, p, st)));
    else
      FLOWMOE_TRY((run_f32<MODE_KSUM, false, EPI_WGRAD>(FLOWMOE_K_WGRAD1, s, p, st)));
  }
  // 3. the biases' gradients: column sums of dY and dH over each expert's rows
  return launch_expert_bias_grad(s, R, dy_disp, dh, counts, offsets, db1, db3, db2, accumulate,
                                 st);
}

hipError_t launch_expert_ffn_bwd(const Shape& s, const void* dy_disp, const void* x_disp,
                                 const void* h_save, const void* a_save, const int32_t* counts,
                                 const int32_t* offsets, const void* w1, const void* w3,
                                 const void* w2, void* dx_disp, float* dw1, float* dw3,
                                 float* dw2, float* db1, float* db3, float* db2, int accumulate,
                                 void* ws, hipStream_t st) {
  // dH in the workspace (h_save is left as it is)
  FLOWMOE_TRY(launch_expert_ffn_dgrad(s, dy_disp, h_save, counts, offsets, w1, w3, w2, ws, dx_disp,
                                      st));
  return launch_expert_ffn_wgrad(s, 1, dy_disp, x_disp, a_save, ws, counts, offsets, dw1, dw3, dw2,
                                 db1, db3, db2, accumulate, st);
}

}  // namespace flowmoe
