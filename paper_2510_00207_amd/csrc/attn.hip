// The multi-head attention of AT_r (Sec. 2.1): per sequence and head,
// A = softmax(Q K^T / sqrt(d)) V with Q, K, V the head's columns of
// I [W^Q | W^K | W^V], then I' = A W^O. The projections run on the grouped
// GEMM as one dense expert; the attention runs in the kernels below, which
// stream K and V tiles through LDS and never store the N x N scores.
//
// Forward (one block: 128 queries of one sequence and head, 4 waves of 32):
// each wave computes S^T = K Q^T for a 64-key tile with
// v_mfma_f32_32x32x16_bf16, so that a lane's accumulator column is one query
// and the online-softmax statistics (running max and sum, base-2 exponents)
// live in the lane pair (l, l + 32) that holds that query's 64 scores. The
// bf16 probabilities P^T are then the second MFMA's column operand straight
// from the registers, and O^T += V^T P^T takes V^T from LDS by transposing
// reads (ds_read_b64_tr_b16). The log-sum-exp of each row is kept for the
// backward.
//
// Backward (no atomics; every sum in a fixed order):
//   dq kernel (blocks of 128 queries, loop over 32-key tiles): recomputes P
//     from S and the log-sum-exp, dP^T = V dO^T, dS = P (dP - delta) with
//     delta = rowsum(dO * O) (computed here and stored for the next kernel),
//     dQ^T += K^T dS^T;
//   dkdv kernel (blocks of 128 keys, loop over 32-query steps): S and dP with
//     the key as the accumulator column, dV^T += dO^T P, dK^T += Q^T dS.
#include <math.h>

#include "common.hpp"

namespace flowmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

struct AttnArgs {
  const bf16_t* qkv;  // T x 3M = [Q | K | V]; head h at columns h * D of each
  const bf16_t* o;    // T x M: the heads' outputs (backward)
  const bf16_t* d_o;  // T x M: their gradient (backward)
  bf16_t* out;        // forward: T x M
  bf16_t* d_qkv;      // backward: T x 3M
  float* lse;         // heads x T: natural log-sum-exp of each row's scores
  float* delta;       // heads x T: rowsum(dO * O) over the head's columns
  int T, M, N, heads, nseq;
  int pair;  // causal grid of one round of resident blocks: pair long and short tiles (decode)
  float c2;  // log2(e) / sqrt(D): a score times c2 is its base-2 exponent
  float rs;  // 1 / sqrt(D)
};

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// the LDS stage of a double-buffered loop as a compile-time constant: the
// loops run their steps in pairs (stage 0, stage 1), so every LDS address of
// a step is a register base plus an immediate offset
template <int S>
struct Stage {
  static constexpr int value = S;
};

__device__ __forceinline__ bf16x8 zero8() { return __builtin_bit_cast(bf16x8, u32x4{0, 0, 0, 0}); }

__device__ __forceinline__ floatx16 zero16() {
  floatx16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

// LDS tiles hold rows of D bf16 (2D bytes); the 16-byte chunk c of row r
// sits at chunk c ^ sw(r). For D = 128 (a row is one pass over the 64 banks)
// sw is one-to-one on any 16 consecutive rows, so a row read (16 lanes on 16
// rows, one chunk each) touches 16 distinct bank groups; sw / 2 takes 4
// distinct values of one parity on 4 aligned rows, so a transposing read
// (4 aligned rows x two adjacent 32-byte column pairs per 32 lanes) does too.
// For D = 64 (two rows per pass) the same holds with the row parity as the
// extra bank bit.
template <int D>
__device__ __forceinline__ int sw(int r) {
  if constexpr (D == 128) return 4 * (r & 3) + ((r >> 2) & 3);
  else return 4 * ((r >> 1) & 1) + 2 * ((r >> 2) & 1) + ((r >> 3) & 1);
}
template <int D>
__device__ __forceinline__ int toff(int r, int c) {
  return r * (2 * D) + ((c ^ sw<D>(r)) << 4);
}

// Two MFMA operand forms are read from these tiles:
//   row operand (d contiguous): lane l supplies row r0 + l % 32 of a 32-row
//     block at d = 16 ks + 8 (l / 32) .. + 7, one 16-byte read of chunk
//     2 ks + l / 32 (row_base, frag_row_x);
//   transposed operand: lane l supplies column cb + l % 32 of the tile at
//     the 8 rows of its k-slots, slot 4 i + j (i = 0, 1; j = 0..3) being row
//     rb + 4 (l / 32) + 8 i + j, as two transposing reads (tr_base,
//     frag_tr_x). Each ds_read_b64_tr_b16 hands lane l' of a 16-lane group
//     element l' % 4 of the 4 values that lane 4 q + l' / 4 addressed, in
//     slot q; lanes aimed at rows r0 + s / 4, columns c0 + 4 (s % 4) give
//     lane l' column c0 + l' at rows r0 .. r0 + 3.

// The swizzle lets a lane's fragment addresses be formed from three per-lane
// bases: a row read of row r0 + lq (r0 a multiple of 32) at k step ks is at
// r0 * 2D + (row_base ^ 32 ks), and a transposing read at rows rb (a
// multiple of 16) and columns cb (a multiple of 32) at
// rb * 2D + (tr_base_i ^ 2 cb) for its two halves i. The loops rebuild the
// XORs in every step from bases they mark as changed (opaque()): the
// compiler would otherwise keep every combination live across the loop and,
// short of registers, spill them and reload one before each LDS read.
template <int D>
__device__ __forceinline__ int row_base(int lq, int h2) {
  return toff<D>(lq, h2);
}
template <int D>
__device__ __forceinline__ int tr_base(int lane, int i) {
  const int G = lane >> 4, sl = lane & 15;
  const int col = (G & 1) * 16 + 4 * (sl & 3);
  const int r = 4 * (G >> 1) + 8 * i + (sl >> 2);
  return toff<D>(r, col >> 3) + ((col & 7) << 1);
}
template <int D>
__device__ __forceinline__ bf16x8 frag_row_x(const char* t, int base, int r0, int ks) {
  return *reinterpret_cast<const bf16x8*>(t + r0 * 2 * D + (base ^ (ks << 5)));
}
template <int D>
__device__ __forceinline__ bf16x8 frag_tr_x(const char* t, int b0, int b1, int rb, int cb) {
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(t + rb * 2 * D + (b0 ^ (2 * cb))));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(t + rb * 2 * D + (b1 ^ (2 * cb))));
  const short __attribute__((ext_vector_type(8))) s = {lo[0], lo[1], lo[2], lo[3],
                                                       hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, s);
}
__device__ __forceinline__ void opaque(int& a, int& b, int& c) {
  asm volatile("" : "+v"(a), "+v"(b), "+v"(c));
}

// Rows 16 s .. 16 s + 15 of a 32 x 32 accumulator (lane l: column l % 32,
// element 4 J + j = row 8 J + 4 (l / 32) + j) as an MFMA column operand in
// the transposed operand's slot order: slot 4 i + j <- element 8 s + 4 i + j.
__device__ __forceinline__ bf16x8 pfrag(const floatx16& a, int s) {
  bf16x8 r;
#pragma unroll
  for (int t = 0; t < 8; ++t) r[t] = (__bf16)a[8 * s + t];
  return r;
}

__device__ __forceinline__ floatx16 mfma(const bf16x8& a, const bf16x8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// store a 32-row block of a transposed accumulator (lane: column = token,
// rows = d) as bf16 row segments dst[8 J + 4 (l / 32) .. + 3] * scale
__device__ __forceinline__ void store_cols(bf16_t* dst, const floatx16& a, int h2, float scale) {
#pragma unroll
  for (int J = 0; J < 4; ++J) {
    uint2 v;
    v.x = pack_bf16x2(a[4 * J] * scale, a[4 * J + 1] * scale);
    v.y = pack_bf16x2(a[4 * J + 2] * scale, a[4 * J + 3] * scale);
    *reinterpret_cast<uint2*>(dst + 8 * J + 4 * h2) = v;
  }
}

// ROWS-row K and V tiles of one (sequence, head), double-buffered through
// registers: every thread moves ROWS * D / 2048 16-byte chunks of each per tile
template <int D, int ROWS = 64, int NT = 256>
struct KVTiles {
  static constexpr int CPR = D / 8;             // 16-byte chunks per row
  static constexpr int TB = ROWS * D * 2;       // bytes of one tile
  static constexpr int TOT = ROWS * CPR;        // chunks per tile
  static constexpr int LD = (TOT + NT - 1) / NT; // chunks per thread per tile
  u32x4 rk[LD], rv[LD];
  __device__ __forceinline__ void load(const bf16_t* Kg, const bf16_t* Vg, long ld, int key0, int N,
                                       int tid) {
#pragma unroll
    for (int u = 0; u < LD; ++u) {
      const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR, key = key0 + r;
      if (key < N && idx < TOT) {
        rk[u] = *reinterpret_cast<const u32x4*>(Kg + key * ld + 8 * c);
        rv[u] = *reinterpret_cast<const u32x4*>(Vg + key * ld + 8 * c);
      } else {
        rk[u] = u32x4{0, 0, 0, 0};
        rv[u] = u32x4{0, 0, 0, 0};
      }
    }
  }
  __device__ __forceinline__ void store(char* tk, char* tv, int tid) {
#pragma unroll
    for (int u = 0; u < LD; ++u) {
      const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR;
      if (TOT % NT == 0 || idx < TOT) {
        *reinterpret_cast<u32x4*>(tk + toff<D>(r, c)) = rk[u];
        *reinterpret_cast<u32x4*>(tv + toff<D>(r, c)) = rv[u];
      }
    }
  }
};

// block -> (query or key tile, head, sequence). Blocks are dispatched in
// order; u = blockIdx / (heads x sequences) ranks the tiles by their causal
// work, longest first (`rev`: tiles in descending order, the query tiles of
// the forward and of dQ; else ascending, the key tiles of dK/dV). With
// `a.pair` (every block resident at once, two to a CU: the second half of
// the grid lands on the CUs of the first half) the second half runs the
// shortest tiles first, so that a CU's two blocks have complementary work
// (ranks u and nt - 1 - u) instead of ranks u and u + nt / 2.
__device__ __forceinline__ void decode(const AttnArgs& a, bool rev, int& tile, int& hd, int& sq,
                                       int rows = 128) {
  const int per = a.heads * a.nseq, nt = (a.N + rows - 1) / rows;
  const int u = (int)(blockIdx.x / per), rest = (int)(blockIdx.x % per);
  const int h = (nt + 1) / 2;
  const int r = a.pair && u >= h ? nt - 1 - (u - h) : u;  // rank in work order
  tile = rev ? nt - 1 - r : r;
  hd = rest % a.heads;
  sq = rest / a.heads;
}

// NW waves (of 32 queries each) per forward block: every K/V tile that a
// block stages in LDS serves 32 NW queries (8 waves halve the staging
// traffic per MFMA of 4; the launch picks 4 when 8 would leave fewer than
// two blocks per CU)
template <int D, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void attn_fwd_kernel(AttnArgs a) {
  constexpr int KS = D / 16, DB = D / 32, QB = 32 * NW;
  using Tiles = KVTiles<D, 64, 64 * NW>;
  __shared__ __attribute__((aligned(16))) char lds[2 * 2 * Tiles::TB];
  // the wave index through readfirstlane: the compiler then knows it is
  // wave-uniform, and the branches on a wave's query or key range are
  // scalar branches instead of exec-mask ones (backward 7-10% faster)
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6),
            h2 = lane >> 5, lq = lane & 31;
  int qt, hd, sq;
  decode(a, CAUSAL, qt, hd, sq, QB);
  const long tok0 = (long)sq * a.N, ld = 3L * a.M;
  const bf16_t* Qg = a.qkv + tok0 * ld + (long)hd * D;
  const bf16_t* Kg = Qg + a.M;
  const bf16_t* Vg = Qg + 2L * a.M;
  const int q0 = qt * QB, qw = q0 + 32 * w + lq;

  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qf[ks] = qw < a.N ? *reinterpret_cast<const bf16x8*>(Qg + qw * ld + 16 * ks + 8 * h2) : zero8();
  floatx16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = zero16();
  float m = -INFINITY, l = 0.0f;

  const int kend = CAUSAL ? min(a.N, q0 + QB) : a.N;
  const int nk = (kend + 63) / 64;
  Tiles tl;
  tl.load(Kg, Vg, ld, 0, a.N, tid);
  tl.store(lds, lds + Tiles::TB, tid);
  __syncthreads();
  int rbase = row_base<D>(lq, h2), tb0 = tr_base<D>(lane, 0), tb1 = tr_base<D>(lane, 1);
  auto step = [&](const int kt, auto stc) {
    constexpr int st = decltype(stc)::value;
    opaque(rbase, tb0, tb1);
    if (kt + 1 < nk) tl.load(Kg, Vg, ld, (kt + 1) * 64, a.N, tid);
    const char* tk = lds + st * 2 * Tiles::TB;
    const char* tv = tk + Tiles::TB;
    const int kb0 = kt * 64;
    // (causal: a wave whose queries all precede the tile has nothing in it)
    if (!CAUSAL || kb0 <= q0 + 32 * w + 31) {
      floatx16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = zero16();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) s[kb] = mfma(frag_row_x<D>(tk, rbase, 32 * kb, ks), qf[ks], s[kb]);
      }
      const bool edge = kb0 + 64 > a.N || (CAUSAL && kb0 + 63 > q0 + 32 * w);
      if (edge) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kb0 + 32 * kb + 8 * (r >> 2) + 4 * h2 + (r & 3);
            if (key >= a.N || (CAUSAL && key > qw)) s[kb][r] = -INFINITY;
          }
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * a.c2;
      // The reference m of the exponents moves only when a score exceeds it
      // by more than 2^8 (then the sum and the accumulators are rescaled):
      // probabilities up to 256 stay exact in float and in bf16's exponent
      // range, and the final lse = m + log2(l) is the same. Every query sees
      // key 0 in the first tile, so m is finite from then on.
      const bool up = mx > m + 8.0f;
      if (__any(up)) {
        const float mn = up ? mx : m;
        const float al = exp2_fast(m - mn);
        l *= al;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= al;
        m = mn;
      }
      float rsum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = exp2_fast(fmaf(s[kb][r], a.c2, -m));
          s[kb][r] = pv;
          rsum += pv;
        }
      }
      rsum += __shfl_xor(rsum, 32);
      l += rsum;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const bf16x8 pb = pfrag(s[kb], s2);
#pragma unroll
          for (int db = 0; db < DB; ++db)
            o[db] = mfma(frag_tr_x<D>(tv, tb0, tb1, 32 * kb + 16 * s2, 32 * db), pb, o[db]);
        }
      }
    }
    if (kt + 1 < nk) {
      char* nk_ = lds + (st ^ 1) * 2 * Tiles::TB;
      tl.store(nk_, nk_ + Tiles::TB, tid);
    }
    __syncthreads();
    };
  for (int kt = 0; kt < nk; kt += 2) {
    step(kt, Stage<0>{});
    if (kt + 1 < nk) step(kt + 1, Stage<1>{});
  }
  if (qw < a.N) {
    const float inv = 1.0f / l;
    bf16_t* Og = a.out + (tok0 + qw) * a.M + (long)hd * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) store_cols(Og + 32 * db, o[db], h2, inv);
    if (h2 == 0) a.lse[(long)hd * a.T + tok0 + qw] = (m + log2f(l)) * kLn2;
  }
}

template <int D, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void attn_dq_kernel(AttnArgs a) {
  constexpr int KS = D / 16, DB = D / 32, QB = 32 * NW, NT = 64 * NW;
  constexpr int CPR = D / 8;
  using Tiles = KVTiles<D, 32, NT>;
  // 32-key K/V stages, then the dO rows of the block's 128 queries (read
  // from LDS each tile rather than held in registers): 64 KB of LDS at
  // D = 128, so two blocks share a CU, and the kernel fits in the 256 VGPRs
  // that leaves without moving values through the AGPRs every step
  __shared__ __attribute__((aligned(16))) char lds[2 * 2 * Tiles::TB + QB * D * 2];
  char* const gt = lds + 2 * 2 * Tiles::TB;
  // the wave index through readfirstlane: the compiler then knows it is
  // wave-uniform, and the branches on a wave's query or key range are
  // scalar branches instead of exec-mask ones (backward 7-10% faster)
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6),
            h2 = lane >> 5, lq = lane & 31;
  int qt, hd, sq;
  decode(a, CAUSAL, qt, hd, sq, QB);
  const long tok0 = (long)sq * a.N, ld = 3L * a.M;
  const bf16_t* Qg = a.qkv + tok0 * ld + (long)hd * D;
  const bf16_t* Kg = Qg + a.M;
  const bf16_t* Vg = Qg + 2L * a.M;
  const bf16_t* Gg = a.d_o + tok0 * a.M + (long)hd * D;
  const bf16_t* Og = a.o + tok0 * a.M + (long)hd * D;
  const int q0 = qt * QB, qw = q0 + 32 * w + lq;
  const bool live = qw < a.N;

#pragma unroll
  for (int u = 0; u < QB * CPR / NT; ++u) {
    const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR, q = q0 + r;
    *reinterpret_cast<u32x4*>(gt + toff<D>(r, c)) =
        q < a.N ? *reinterpret_cast<const u32x4*>(Gg + (long)q * a.M + 8 * c) : u32x4{0, 0, 0, 0};
  }
  bf16x8 qf[KS];
  float dl = 0.0f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = live ? *reinterpret_cast<const bf16x8*>(Qg + qw * ld + 16 * ks + 8 * h2) : zero8();
    const bf16x8 gv = live ? *reinterpret_cast<const bf16x8*>(Gg + (long)qw * a.M + 16 * ks + 8 * h2) : zero8();
    const bf16x8 ov = live ? *reinterpret_cast<const bf16x8*>(Og + (long)qw * a.M + 16 * ks + 8 * h2) : zero8();
#pragma unroll
    for (int t = 0; t < 8; ++t) dl += (float)gv[t] * (float)ov[t];
  }
  dl += __shfl_xor(dl, 32);
  const long srow = (long)hd * a.T + tok0 + qw;
  if (live && h2 == 0) a.delta[srow] = dl;
  const float l2 = live ? a.lse[srow] * kLog2e : 0.0f;
  floatx16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dq[db] = zero16();

  const int kend = CAUSAL ? min(a.N, q0 + QB) : a.N;
  const int nk = (kend + 31) / 32;
  Tiles tl;
  tl.load(Kg, Vg, ld, 0, a.N, tid);
  tl.store(lds, lds + Tiles::TB, tid);
  __syncthreads();
  int rbase = row_base<D>(lq, h2), tb0 = tr_base<D>(lane, 0), tb1 = tr_base<D>(lane, 1);
  auto step = [&](const int kt, auto stc) {
    constexpr int st = decltype(stc)::value;
    opaque(rbase, tb0, tb1);
    if (kt + 1 < nk) tl.load(Kg, Vg, ld, (kt + 1) * 32, a.N, tid);
    const char* tk = lds + st * 2 * Tiles::TB;
    const char* tv = tk + Tiles::TB;
    const int kb0 = kt * 32;
    if (!CAUSAL || kb0 <= q0 + 32 * w + 31) {
      floatx16 s = zero16(), dp = zero16();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) s = mfma(frag_row_x<D>(tk, rbase, 0, ks), qf[ks], s);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        dp = mfma(frag_row_x<D>(tv, rbase, 0, ks), frag_row_x<D>(gt, rbase, 32 * w, ks), dp);
      const bool edge = kb0 + 32 > a.N || (CAUSAL && kb0 + 31 > q0 + 32 * w);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float pv = exp2_fast(s[r] * a.c2 - l2);
        if (edge) {
          const int key = kb0 + 8 * (r >> 2) + 4 * h2 + (r & 3);
          if (key >= a.N || (CAUSAL && key > qw)) pv = 0.0f;
        }
        s[r] = pv * (dp[r] - dl);  // dS^T
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const bf16x8 pb = pfrag(s, s2);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          dq[db] = mfma(frag_tr_x<D>(tk, tb0, tb1, 16 * s2, 32 * db), pb, dq[db]);
      }
    }
    if (kt + 1 < nk) {
      char* nk_ = lds + (st ^ 1) * 2 * Tiles::TB;
      tl.store(nk_, nk_ + Tiles::TB, tid);
    }
    __syncthreads();
    };
  for (int kt = 0; kt < nk; kt += 2) {
    step(kt, Stage<0>{});
    if (kt + 1 < nk) step(kt + 1, Stage<1>{});
  }
  if (live) {
    bf16_t* dst = a.d_qkv + (tok0 + qw) * ld + (long)hd * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) store_cols(dst + 32 * db, dq[db], h2, a.rs);
  }
}

template <int D, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void attn_dkdv_kernel(AttnArgs a) {
  constexpr int KS = D / 16, DB = D / 32, CPR = D / 8, KB = 32 * NW, NT = 64 * NW;
  constexpr int TQ = 32 * D * 2;                // one 32-row tile
  constexpr int STG = 2 * TQ + 256;             // Q, dO, then 32 lse2 and 32 delta
  constexpr int TOT = 32 * CPR;                 // chunks per 32-row tile
  constexpr int LD = (TOT + NT - 1) / NT;       // chunks per thread per tile
  // two query stages, then the V rows of the block's 128 keys (read from
  // LDS each step rather than held in registers: the kernel then fits in the
  // 256 VGPRs without moving values through the AGPRs every step)
  __shared__ __attribute__((aligned(16))) char lds[2 * STG + KB * D * 2];
  char* const vt = lds + 2 * STG;
  // the wave index through readfirstlane: the compiler then knows it is
  // wave-uniform, and the branches on a wave's query or key range are
  // scalar branches instead of exec-mask ones (backward 7-10% faster)
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6),
            h2 = lane >> 5, lq = lane & 31;
  int kt, hd, sq;
  decode(a, false, kt, hd, sq, KB);
  const long tok0 = (long)sq * a.N, ld = 3L * a.M;
  const bf16_t* Qg = a.qkv + tok0 * ld + (long)hd * D;
  const bf16_t* Gg = a.d_o + tok0 * a.M + (long)hd * D;
  const long srow0 = (long)hd * a.T + tok0;
  const int k0 = kt * KB, kw = k0 + 32 * w + lq;
  const bool live = kw < a.N;

  bf16x8 kf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    kf[ks] = live ? *reinterpret_cast<const bf16x8*>(Qg + a.M + kw * ld + 16 * ks + 8 * h2) : zero8();
#pragma unroll
  for (int u = 0; u < KB * CPR / NT; ++u) {
    const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR, key = k0 + r;
    *reinterpret_cast<u32x4*>(vt + toff<D>(r, c)) =
        key < a.N ? *reinterpret_cast<const u32x4*>(Qg + 2L * a.M + key * ld + 8 * c)
                  : u32x4{0, 0, 0, 0};
  }
  floatx16 dv[DB], dk[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dv[db] = zero16();
    dk[db] = zero16();
  }
  // query steps of 32: causal keys k0.. are seen by queries >= k0 only
  const int qs0 = CAUSAL ? k0 : 0;
  const int nqs = (a.N - qs0 + 31) / 32;
  u32x4 rq[LD], rg[LD];
  float rstat = 0.0f;
  auto load = [&](int qb) {
#pragma unroll
    for (int u = 0; u < LD; ++u) {
      const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR, q = qb + r;
      if (q < a.N && idx < TOT) {
        rq[u] = *reinterpret_cast<const u32x4*>(Qg + q * ld + 8 * c);
        rg[u] = *reinterpret_cast<const u32x4*>(Gg + (long)q * a.M + 8 * c);
      } else {
        rq[u] = u32x4{0, 0, 0, 0};
        rg[u] = u32x4{0, 0, 0, 0};
      }
    }
    if (tid < 64) {
      const int q = qb + (tid & 31);
      rstat = q < a.N ? (tid < 32 ? a.lse[srow0 + q] * kLog2e : a.delta[srow0 + q]) : 0.0f;
    }
  };
  auto store = [&](char* stg) {
#pragma unroll
    for (int u = 0; u < LD; ++u) {
      const int idx = tid + NT * u, r = idx / CPR, c = idx % CPR;
      if (TOT % NT != 0 && idx >= TOT) continue;
      *reinterpret_cast<u32x4*>(stg + toff<D>(r, c)) = rq[u];
      *reinterpret_cast<u32x4*>(stg + TQ + toff<D>(r, c)) = rg[u];
    }
    if (tid < 64) reinterpret_cast<float*>(stg + 2 * TQ)[tid] = rstat;
  };
  if (nqs > 0) {
    load(qs0);
    store(lds);
  }
  __syncthreads();
  int rbase = row_base<D>(lq, h2), tb0 = tr_base<D>(lane, 0), tb1 = tr_base<D>(lane, 1);
  auto step = [&](const int it, auto stc) {
    constexpr int st = decltype(stc)::value;
    opaque(rbase, tb0, tb1);
    const int qb = qs0 + 32 * it;
    if (it + 1 < nqs) load(qb + 32);
    const char* tq = lds + st * STG;
    const char* tg = tq + TQ;
    const float* l2 = reinterpret_cast<const float*>(tq + 2 * TQ);
    const float* dls = l2 + 32;
    if (!CAUSAL || qb + 31 >= k0 + 32 * w) {
      floatx16 s = zero16(), dp = zero16();
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) s = mfma(frag_row_x<D>(tq, rbase, 0, ks), kf[ks], s);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        dp = mfma(frag_row_x<D>(tg, rbase, 0, ks), frag_row_x<D>(vt, rbase, 32 * w, ks), dp);
      const bool edge = qb + 32 > a.N || (CAUSAL && k0 + 32 * w + 31 > qb);
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        const float4 lv = *reinterpret_cast<const float4*>(l2 + 8 * J + 4 * h2);
        const float4 dv4 = *reinterpret_cast<const float4*>(dls + 8 * J + 4 * h2);
        const float lr[4] = {lv.x, lv.y, lv.z, lv.w}, dr[4] = {dv4.x, dv4.y, dv4.z, dv4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = 4 * J + j;
          float pv = exp2_fast(s[r] * a.c2 - lr[j]);
          if (edge) {
            const int q = qb + 8 * J + 4 * h2 + j;
            if (q >= a.N || (CAUSAL && kw > q)) pv = 0.0f;
          }
          s[r] = pv;
          dp[r] = pv * (dp[r] - dr[j]);  // dS
        }
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const bf16x8 pb = pfrag(s, s2), pd = pfrag(dp, s2);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dv[db] = mfma(frag_tr_x<D>(tg, tb0, tb1, 16 * s2, 32 * db), pb, dv[db]);
          dk[db] = mfma(frag_tr_x<D>(tq, tb0, tb1, 16 * s2, 32 * db), pd, dk[db]);
        }
      }
    }
    if (it + 1 < nqs) store(lds + (st ^ 1) * STG);
    __syncthreads();
    };
  for (int it = 0; it < nqs; it += 2) {
    step(it, Stage<0>{});
    if (it + 1 < nqs) step(it + 1, Stage<1>{});
  }
  if (live) {
    bf16_t* dst = a.d_qkv + (tok0 + kw) * ld + (long)hd * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      store_cols(dst + a.M + 32 * db, dk[db], h2, a.rs);
      store_cols(dst + 2L * a.M + 32 * db, dv[db], h2, 1.0f);
    }
  }
}

AttnArgs attn_args(const AttnShape& m, int T, int M) {
  AttnArgs a = {};
  a.T = T;
  a.M = M;
  a.N = m.N;
  a.heads = m.heads;
  a.nseq = m.N > 0 ? T / m.N : 0;
  a.c2 = kLog2e / sqrtf((float)m.D);
  a.rs = 1.0f / sqrtf((float)m.D);
  return a;
}

unsigned attn_blocks(const AttnArgs& a, int rows = 128) {
  return (unsigned)(((a.N + rows - 1) / rows) * a.heads * a.nseq);
}

// pair long and short causal tiles (decode) when the 4-wave grid (two
// blocks per CU) is resident all at once: then the makespan is a CU's two
// blocks together, not the longest-first order's
int attn_pair(const AttnShape& m, const AttnArgs& a, bool wide) {
  return m.causal && !wide && attn_blocks(a, 128) <= 2u * 256u ? 1 : 0;
}

#define FLOWMOE_ATTN_LAUNCH(KERNEL, a, st, ROWS, THREADS, ...)                                 \
  do {                                                                                          \
    const dim3 g(attn_blocks(a, ROWS)), b(THREADS);                                             \
    if (m.D == 128) {                                                                           \
      if (m.causal) hipLaunchKernelGGL((KERNEL<128, true, ##__VA_ARGS__>), g, b, 0, st, a);     \
      else hipLaunchKernelGGL((KERNEL<128, false, ##__VA_ARGS__>), g, b, 0, st, a);             \
    } else {                                                                                    \
      if (m.causal) hipLaunchKernelGGL((KERNEL<64, true, ##__VA_ARGS__>), g, b, 0, st, a);      \
      else hipLaunchKernelGGL((KERNEL<64, false, ##__VA_ARGS__>), g, b, 0, st, a);              \
    }                                                                                           \
  } while (0)

}  // namespace

hipError_t launch_attn_fwd(const AttnShape& m, int T, int M, const void* qkv, void* o, float* lse,
                           hipStream_t st) {
  AttnArgs a = attn_args(m, T, M);
  if (attn_blocks(a) == 0) return hipSuccess;
  a.qkv = static_cast<const bf16_t*>(qkv);
  a.out = static_cast<bf16_t*>(o);
  a.lse = lse;
  const bool wide = attn_blocks(a, 256) >= 2u * 256u;
  a.pair = attn_pair(m, a, wide);
  return traced(FLOWMOE_K_ATTN_FWD, st, [&] {
    if (wide) FLOWMOE_ATTN_LAUNCH(attn_fwd_kernel, a, st, 256, 512, 8);
    else FLOWMOE_ATTN_LAUNCH(attn_fwd_kernel, a, st, 128, 256, 4);
  });
}

hipError_t launch_attn_bwd(const AttnShape& m, int T, int M, const void* qkv, const void* o,
                           const float* lse, const void* d_o, void* d_qkv, float* delta,
                           hipStream_t st) {
  AttnArgs a = attn_args(m, T, M);
  if (attn_blocks(a) == 0) return hipSuccess;
  a.qkv = static_cast<const bf16_t*>(qkv);
  a.o = static_cast<const bf16_t*>(o);
  a.d_o = static_cast<const bf16_t*>(d_o);
  a.d_qkv = static_cast<bf16_t*>(d_qkv);
  a.lse = const_cast<float*>(lse);
  a.delta = delta;
  // 8-wave blocks (256 queries, or keys) when that grid still gives two
  // blocks per CU: each staged tile then serves twice the MFMA work
  const bool wide = attn_blocks(a, 256) >= 2u * 256u;
  a.pair = attn_pair(m, a, wide);
  hipError_t e = traced(FLOWMOE_K_ATTN_BWD_DQ, st, [&] {
    if (wide) FLOWMOE_ATTN_LAUNCH(attn_dq_kernel, a, st, 256, 512, 8);
    else FLOWMOE_ATTN_LAUNCH(attn_dq_kernel, a, st, 128, 256, 4);
  });
  if (e != hipSuccess) return e;
  return traced(FLOWMOE_K_ATTN_BWD_DKDV, st, [&] {
    if (wide) FLOWMOE_ATTN_LAUNCH(attn_dkdv_kernel, a, st, 256, 512, 8);
    else FLOWMOE_ATTN_LAUNCH(attn_dkdv_kernel, a, st, 128, 256, 4);
  });
}

hipError_t launch_mha_fwd(const AttnShape& m, int T, int M, const void* in, const void* w_qkv,
                          const void* w_o, void* qkv, void* attn, float* lse, void* out,
                          hipStream_t st) {
  if (T == 0) return hipSuccess;
  hipError_t e = launch_dense_gemm(FLOWMOE_K_ATTN_QKV, T, in, M, M, w_qkv, 3L * M, false, 3 * M,
                                   qkv, 3L * M, st);
  if (e != hipSuccess) return e;
  e = launch_attn_fwd(m, T, M, qkv, attn, lse, st);
  if (e != hipSuccess) return e;
  return launch_dense_gemm(FLOWMOE_K_ATTN_OUT, T, attn, M, M, w_o, M, false, M, out, M, st);
}

hipError_t launch_mha_bwd_data(const AttnShape& m, int T, int M, const void* w_qkv,
                               const void* w_o, const void* qkv, const void* attn,
                               const float* lse, const void* d_out, void* d_attn, void* d_qkv,
                               float* delta, void* d_in, hipStream_t st) {
  if (T == 0) return hipSuccess;
  // d_attn = d_out W^O^T: B[k][n] = W^O[n][k] (K-contiguous)
  hipError_t e = launch_dense_gemm(FLOWMOE_K_ATTN_DGRAD, T, d_out, M, M, w_o, M, true, M, d_attn,
                                   M, st);
  if (e != hipSuccess) return e;
  e = launch_attn_bwd(m, T, M, qkv, attn, lse, d_attn, d_qkv, delta, st);
  if (e != hipSuccess) return e;
  // d_in = d_qkv [W^Q | W^K | W^V]^T: B[k][n] = W_qkv[n][k] (K-contiguous)
  return launch_dense_gemm(FLOWMOE_K_ATTN_DGRAD, T, d_qkv, 3L * M, 3 * M, w_qkv, 3L * M, true, M,
                           d_in, M, st);
}

hipError_t launch_mha_wgrad(int T, int M, int R, const void* in, const void* attn,
                            const void* d_out, const void* d_qkv, float* dw_qkv, float* dw_o,
                            int accumulate, void* ws, hipStream_t st) {
  // dW^O = attn^T d_out and dW_qkv = in^T d_qkv, each summed over the R
  // chunks' rows in chunk order (through partial sums in ws when their
  // output tiles are too few for the CUs)
  float* part = static_cast<float*>(ws);
  hipError_t e = launch_dense_wgrad(FLOWMOE_K_ATTN_WGRAD, T, R, attn, M, (long)T * M, M, d_out, M,
                                    (long)T * M, M, dw_o, M, accumulate, part, st);
  if (e != hipSuccess) return e;
  return launch_dense_wgrad(FLOWMOE_K_ATTN_WGRAD, T, R, in, M, (long)T * M, M, d_qkv, 3L * M,
                            (long)T * 3 * M, 3 * M, dw_qkv, 3L * M, accumulate, part, st);
}

}  // namespace flowmoe
