// Gate (the AT_r gating part of Sec. 2.1 / Sec. 4.2): logits = x W_g (+ b),
// top-k selection with renormalised softmax weights, and the gate backward.
//
// Selection order: larger logit first, equal logits by the lower expert
// index, -0.0 == +0.0; every top-k path compares 64-bit keys that encode
// exactly this order. The fp32 gate and flowmoe_route spread a token's
// experts over a segment of EP lanes (EP = next power of two >= E, E <= 64;
// a 64-wide wave holds 64/EP segments) and take k rounds of a segmented
// butterfly maximum; the bf16 gate selects in its own epilogue.
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

// Selection key of (logit v, expert e): a larger key comes first in the
// order (larger value; equal values by the lower index; -0.0 == +0.0). The
// value's bits map monotonically onto an unsigned word (negative values:
// every bit flipped; others: the sign bit set), -0.0 taken as +0.0; the low
// word is 2^32 - 1 - e. Key 0 is below every logit (an empty slot or a lane
// past E); keys of one token's logits are distinct.
__device__ __forceinline__ uint64_t sel_key(float v, int e) {
  uint32_t b = __float_as_uint(v);
  b = (b == 0x80000000u) ? 0u : b;
  const uint32_t m = (b & 0x80000000u) ? 0xFFFFFFFFu : 0x80000000u;
  return ((uint64_t)(b ^ m) << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)e);
}
__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t s = (uint32_t)(key >> 32);
  return __uint_as_float((s & 0x80000000u) ? (s ^ 0x80000000u) : ~s);
}
__device__ __forceinline__ int key_index(uint64_t key) {
  return (int)(0xFFFFFFFFu - (uint32_t)key);
}
__device__ __forceinline__ uint64_t shfl_xor_key(uint64_t key, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)key, m), hi = __shfl_xor((uint32_t)(key >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

// the k selected (keys in order) -> idx and weights exp(l_j - l_0) / Z,
// shifted by the largest logit l_0: Z = the sum over the selection (zfull <
// 0: the renormalised gate) or zfull, the sum over all E experts (the full
// softmax gate)
template <int KM>
__device__ __forceinline__ void topk_store(const uint64_t (&top)[KM], int k, float zfull,
                                           int32_t* idx_out, float* w_out) {
  float ex[KM], denom = 0.f;
  const float v0 = key_value(top[0]);
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    ex[j] = j < k ? expf(key_value(top[j]) - v0) : 0.f;
    denom += ex[j];
  }
  if (zfull >= 0.f) denom = zfull;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < k) {
      idx_out[j] = key_index(top[j]);
      w_out[j] = ex[j] / denom;
    }
  }
}

// Top-k of one token's logits held one per lane by a segment of EP lanes
// (lane expert e; lanes past E pass valid = false): k rounds of a butterfly
// maximum of the keys, the winner's lane dropping out; with `full`, a
// butterfly sum of exp(l_e - l_0) over the segment for the full softmax.
// Lane 0 of the segment writes idx/w.
__device__ __forceinline__ void topk_write(float logit, int e, bool valid, int EP, int k,
                                           bool full, int32_t* idx_out, float* w_out) {
  uint64_t top[kMaxK];
  uint64_t mine = valid ? sel_key(logit, e) : 0ull;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    uint64_t best = mine;
    if (j < k) {
      for (int off = EP >> 1; off > 0; off >>= 1) {
        const uint64_t o = shfl_xor_key(best, off);
        best = o > best ? o : best;
      }
      mine = (best == mine) ? 0ull : mine;
    }
    top[j] = best;
  }
  float z = -1.f;
  if (full) {  // (uniform)
    z = valid ? expf(logit - key_value(top[0])) : 0.f;
    for (int off = EP >> 1; off > 0; off >>= 1) z += __shfl_xor(z, off);
  }
  if (e == 0) topk_store<kMaxK>(top, k, z, idx_out, w_out);
}

// Top-k of one token's E logits by P consecutive lanes (P a power of two
// <= 64). Lane p keeps the KM largest keys of logits p, p + P, ... in order
// (an insertion without branches); then log2(P) exchanges with a lane of
// the other half of ever wider lane groups (lane_partner below) merge two
// sorted lists (topk_merge). Every lane ends with the same list; lane p == 0
// writes.
template <int KM>
__device__ __forceinline__ void topk_insert(uint64_t key, uint64_t (&tk)[KM]) {
  bool b[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) b[j] = key > tk[j];
#pragma unroll
  for (int j = KM - 1; j >= 1; --j)  // b is monotone: b[j - 1] implies b[j]
    tk[j] = b[j] ? (b[j - 1] ? tk[j - 1] : key) : tk[j];
  tk[0] = b[0] ? key : tk[0];
}

// Exchange with a lane of the other half of an aligned group of 2 M lanes
// (M < 16: DPP moves inside a row, no LDS round trip: M = 1 and 2 swap
// neighbours and pairs of a quad, M = 4 and 8 mirror the halves of a row;
// wider: lane ^ M). After exchanges M = 1, 2, ..., P / 2 of lists that are
// merged (or values that are combined) at each step, every lane of an
// aligned P-lane group holds the result of the whole group. All lanes of
// the group must be active.
template <int M>
__device__ __forceinline__ uint32_t lane_partner(uint32_t v) {
  if constexpr (M == 1) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
  else if constexpr (M == 2) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
  else if constexpr (M == 4) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false);
  else if constexpr (M == 8) return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, false);
  else return __shfl_xor(v, M);
}
template <int M>
__device__ __forceinline__ uint64_t key_partner(uint64_t key) {
  const uint32_t lo = lane_partner<M>((uint32_t)key), hi = lane_partner<M>((uint32_t)(key >> 32));
  return ((uint64_t)hi << 32) | lo;
}
template <int M>
__device__ __forceinline__ float sum_partner(float z) {
  return z + __uint_as_float(lane_partner<M>(__float_as_uint(z)));
}

// one merge step: the partner's sorted list b, the larger of a[j] and
// b[KM - 1 - j] for every j (the KM largest of both as a bitonic
// sequence), then half-cleaners sort it
template <int KM, int M>
__device__ __forceinline__ void topk_merge(uint64_t (&tk)[KM]) {
  uint64_t o[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) o[j] = key_partner<M>(tk[j]);
#pragma unroll
  for (int j = 0; j < KM; ++j) tk[j] = tk[j] > o[KM - 1 - j] ? tk[j] : o[KM - 1 - j];
#pragma unroll
  for (int d = KM / 2; d >= 1; d >>= 1)
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if ((j & d) == 0) {
        const uint64_t a = tk[j], b = tk[j + d];
        const bool up = a > b;  // (one compare for both selects)
        tk[j] = up ? a : b;
        tk[j + d] = up ? b : a;
      }
}

template <int KM, int P>
__device__ __forceinline__ void topk_lanes(const float* logit, int E, int k, int p, bool full,
                                           int32_t* idx_out, float* w_out) {
  constexpr int NV = kMaxE / P;  // logits per lane at most
  float v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = p + i * P < E ? logit[p + i * P] : 0.f;  // reads first
  uint64_t tk[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) tk[j] = 0ull;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (p + i * P < E) topk_insert<KM>(sel_key(v[i], p + i * P), tk);
  if constexpr (P > 1) topk_merge<KM, 1>(tk);
  if constexpr (P > 2) topk_merge<KM, 2>(tk);
  if constexpr (P > 4) topk_merge<KM, 4>(tk);
  if constexpr (P > 8) topk_merge<KM, 8>(tk);
  if constexpr (P > 16) topk_merge<KM, 16>(tk);
  if constexpr (P > 32) topk_merge<KM, 32>(tk);
  float z = -1.f;
  if (full) {  // the full softmax's sum: each lane its logits, then the exchanges
    const float v0 = key_value(tk[0]);
    z = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (p + i * P < E) z += expf(v[i] - v0);
    if constexpr (P > 1) z = sum_partner<1>(z);
    if constexpr (P > 2) z = sum_partner<2>(z);
    if constexpr (P > 4) z = sum_partner<4>(z);
    if constexpr (P > 8) z = sum_partner<8>(z);
    if constexpr (P > 16) z = sum_partner<16>(z);
    if constexpr (P > 32) z = sum_partner<32>(z);
  }
  if (p == 0) topk_store<KM>(tk, k, z, idx_out, w_out);
}

// Top-k of one token's E logits by P >= 8 consecutive lanes (at most 8
// logits per lane), the same selection as topk_lanes in fewer steps: each
// lane sorts its own keys; then k rounds take the largest head over the
// group (the exchanges of lane_partner) and the one lane holding that key
// (keys are distinct) drops it. Lane p == 0 writes.
template <int KM, int P>
__device__ __forceinline__ void topk_extract(const float* logit, int E, int k, int p, bool full,
                                             int32_t* idx_out, float* w_out) {
  static_assert(P >= 8, "at most 8 logits per lane");
  constexpr int NV = kMaxE / P;
  float v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = p + i * P < E ? logit[p + i * P] : 0.f;  // reads first
  uint64_t own[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) own[i] = 0ull;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (p + i * P < E) topk_insert<NV>(sel_key(v[i], p + i * P), own);
  uint64_t tk[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    uint64_t best = own[0];
    if (j < k) {  // (uniform; k <= E, so best is a real key)
      uint64_t o;
      o = key_partner<1>(best), best = o > best ? o : best;
      o = key_partner<2>(best), best = o > best ? o : best;
      o = key_partner<4>(best), best = o > best ? o : best;
      if constexpr (P > 8) o = key_partner<8>(best), best = o > best ? o : best;
      if constexpr (P > 16) o = key_partner<16>(best), best = o > best ? o : best;
      if constexpr (P > 32) o = key_partner<32>(best), best = o > best ? o : best;
      const bool pop = own[0] == best;
#pragma unroll
      for (int i = 0; i + 1 < NV; ++i) own[i] = pop ? own[i + 1] : own[i];
      own[NV - 1] = pop ? 0ull : own[NV - 1];
    }
    tk[j] = best;  // (rounds past k are never stored)
  }
  float z = -1.f;
  if (full) {  // the full softmax's sum: each lane its logits, then the exchanges
    const float v0 = key_value(tk[0]);
    z = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (p + i * P < E) z += expf(v[i] - v0);
    z = sum_partner<1>(z);
    z = sum_partner<2>(z);
    z = sum_partner<4>(z);
    if constexpr (P > 8) z = sum_partner<8>(z);
    if constexpr (P > 16) z = sum_partner<16>(z);
    if constexpr (P > 32) z = sum_partner<32>(z);
  }
  if (p == 0) topk_store<KM>(tk, k, z, idx_out, w_out);
}

// Fused gate: per block 4 waves; each wave has G = 64/EP segments, each
// segment TPG tokens. x rows of the block are staged in LDS as float.
template <typename TIn>
__global__ __launch_bounds__(kGateThreads) void gate_topk_kernel(
    const TIn* __restrict__ x, const TIn* __restrict__ wg, const float* __restrict__ bias,
    float* __restrict__ logits, int32_t* __restrict__ idx, float* __restrict__ w, int T, int M,
    int E, int k, int EP, int TPG, int xchunk, int full) {
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
        topk_write(l, e, evalid, EP, k, full, idx + (size_t)t * k, w + (size_t)t * k);
      }
    }
  }
}

// bf16 gate on MFMA (v_mfma_f32_16x16x32_bf16). A block of NW waves owns TGB
// groups of 16 tokens; the reduction over M is split between the waves: wave
// w takes the 32-deep k steps s = w, w + NW, ... and needs only those steps'
// W_g rows, so each wave streams on its own, with no block barrier until the
// partial sums meet. Per step a lane loads 16 bytes of x for each token group
// (8 consecutive k of one token: the A fragment as it lies in memory) and up
// to NB 16-byte units of the step's 32 W_g rows; a ring of D steps of these
// loads stays in flight in registers, and no load is issued for a step past
// the wave's last. A step's W_g rows go to the wave's own LDS slice (two
// slices, alternating) one step ahead; each B fragment (8 consecutive k of
// one expert) comes back as two transposing reads (ds_read_b64_tr_b16),
// issued before the next step's rows are written, so that the MFMAs wait
// for those reads only. Loads use clamped in-bounds addresses; rows past M
// are staged as zeros and the slice columns past E are zeroed once, so the
// accumulator columns past E hold zeros and are never written. The NW
// partial logit tiles are summed in LDS in wave order (deterministic), the
// bias added, and each token's top-k taken by a segment of EP lanes (E <=
// 16) or by P = 256 / (16 TGB) lanes per token (wider gates) on the block's
// first 256 lanes.
constexpr int kGateTok = 16;  // tokens per group
constexpr int kGateDepth = 4; // k steps of loads in flight per wave

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef short gv4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) gv4i16_t lds_gv4i16_t;

// NB 16-expert column blocks (E <= 16 NB), TGB token groups per block, NW
// waves, VEC: E a multiple of 8 (W_g rows are whole 16-byte units)
template <int NB, int TGB, int NW, bool VEC>
__global__ __launch_bounds__(64 * NW) void gate_topk_mfma_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg, const float* __restrict__ bias,
    float* __restrict__ logits, int32_t* __restrict__ idx, float* __restrict__ w, int T, int M,
    int E, int k, int EP, int full) {
  constexpr int TB = kGateTok * TGB;           // tokens per block
  constexpr int PW = NB * 16 + 1;              // partial-tile row pitch (floats)
  constexpr int PART_BYTES = NW * TB * PW * 4; // the waves' partial tiles
  // W_g slice: 32 rows at a pitch of 16 NB + 8 bf16 (a multiple of 16
  // bytes, so every transposing read is 8-byte aligned; the 16 spare bytes
  // shift successive rows by 4 banks)
  constexpr int PITCH = 16 * NB + 8;
  constexpr int SLICE = 32 * PITCH + 8;  // bf16 per slice (+ a 16-byte slot for unused lanes)
  constexpr int SLICE_BYTES = NW * 2 * SLICE * 2;  // two slices per wave
  constexpr int SMEM = PART_BYTES > SLICE_BYTES ? PART_BYTES : SLICE_BYTES;
  constexpr int D = kGateDepth;
  constexpr int WU = NB;  // 16-byte W_g units per lane per step: 32 rows * E / 8 <= 64 NB
  typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  float(*part)[TB][PW] = reinterpret_cast<float(*)[TB][PW]>(smem);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  bf16_t* slices = reinterpret_cast<bf16_t*>(smem) + wave * 2 * SLICE;
  const int t0 = blockIdx.x * TB;
  const int kq = (lane >> 4) * 8;  // k offset of this lane inside a step
  const bf16_t* xrow[TGB];
#pragma unroll
  for (int g = 0; g < TGB; ++g) {
    const int arow = t0 + g * kGateTok + (lane & 15);  // token whose A row this lane feeds
    xrow[g] = x + (long)(arow < T ? arow : 0) * M;
  }
  const int S = (M + 31) / 32;                          // k steps
  const int nj = S > wave ? (S - wave + NW - 1) / NW : 0;  // this wave's steps: s = wave + NW j
  const int UR = E / 8;                                 // 16-byte units per W_g row
  const int n16 = 32 * UR;                              // units per step
  // transposing reads: in each 16-lane group q (= lane / 16) lane l aims at
  // slice row 8 q + l / 4 (+ 4 for the second read), columns 4 (l % 4) .. + 3
  // of a column block, and receives the group's 8 consecutive rows (k) of
  // column l of the block: its B fragment, in the x fragment's k order
  const int tr_off = ((8 * (lane >> 4) + ((lane & 15) >> 2)) * PITCH + 4 * (lane & 3)) * 2;

  // columns past E of both slices: zero (the staging never writes them)
  if (E < 16 * NB) {
    const int pad = 16 * NB - E;
    for (int q = lane; q < 64 * pad; q += 64) {
      const int rr = q / pad, c = E + (q - rr * pad);
      slices[(rr >> 5) * SLICE + (rr & 31) * PITCH + c] = (bf16_t)0;
    }
  }

  floatx4_t acc[TGB][NB];
#pragma unroll
  for (int g = 0; g < TGB; ++g)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[g][nb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  u32x4_t xr[D][TGB], wr[D][WU];
  // The wave's j-th step is s = wave + NW ((j + rot) mod nj): blocks start
  // at different k steps, so they do not all read the same W_g rows at once
  // (on 16384 tokens at E = 8 that hot spot made the gate 1.5x slower).
  const int rot = nj > 0 ? (int)(blockIdx.x % (unsigned)nj) : 0;
  auto step_of = [&](int j) {
    const int jj = j + rot;
    return wave + NW * (jj < nj ? jj : jj - nj);
  };
  // loads of step j into ring slot d; a step past the wave's last loads the
  // last one's addresses again (L2 hits, never used), so that every step
  // issues the same loads and the compiler's load counting stays exact. No
  // value is masked here (a select would wait for the load): x of tokens
  // past T only reaches logits that are not written, x past M meets W_g
  // rows that are zero in LDS, and the W_g units past the step's rows are
  // zeroed when staged.
  auto issue = [&](int d, int j) __attribute__((always_inline)) {
    const int s = step_of(j < nj ? j : nj - 1);
    const int kk = s * 32 + kq;
    const int ko = kk < M ? kk : 0;
#pragma unroll
    for (int g = 0; g < TGB; ++g) xr[d][g] = *reinterpret_cast<const u32x4_t*>(xrow[g] + ko);
    // rows [32 s, 32 s + 32) of W_g are one contiguous range of 32 E values
    // (16-byte aligned: 64 E bytes per step)
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(wg + (long)s * 32 * E);
    const int units = min(32, M - s * 32) * UR;  // whole 16-byte units inside W_g
#pragma unroll
    for (int u = 0; u < WU; ++u) {
      const int q = lane + 64 * u;
      wr[d][u] = src[q < units ? q : 0];
    }
  };
  // W_g rows of step j (< nj) into slice b (rows past M zero; columns past
  // E keep their zeros)
  auto stage = [&](int d, int j, int b) __attribute__((always_inline)) {
    bf16_t* dst = slices + b * SLICE;
    const int s = step_of(j);
    const int rows = min(32, M - s * 32);
    if constexpr (VEC) {
      const int units = rows * UR;
#pragma unroll
      for (int u = 0; u < WU; ++u) {
        const int q = lane + 64 * u;
        const int r = q / UR, cu = q - r * UR;
        // (lanes past the slice's units write the spare slot: no branch)
        bf16_t* p = dst + (q < n16 ? r * PITCH + cu * 8 : 32 * PITCH);
        if (rows == 32)  // (uniform: every step but a last partial one)
          *reinterpret_cast<u32x4_t*>(p) = wr[d][u];
        else
          *reinterpret_cast<u32x4_t*>(p) = q < units ? wr[d][u] : u32x4_t{0u, 0u, 0u, 0u};
      }
    } else {  // element by element (E not a multiple of 8)
      for (int q = lane; q < 32 * E; q += 64) {
        const int r = q / E, e = q - r * E;
        const int row = s * 32 + r;
        dst[r * PITCH + e] = row < M ? wg[(long)row * E + e] : (bf16_t)0;
      }
    }
  };
  // (the LDS operations of one wave complete in order; the fence keeps the
  // compiler from moving a slice's reads below the next writes to it, or
  // the writes above the reads)
  auto lds_fence = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  };

  if (nj > 0) {  // (uniform)
#pragma unroll
    for (int d = 0; d < D; ++d) issue(d, d);
    stage(0, 0, 0);
    lds_fence();
  }
  for (int j0 = 0; j0 < nj; j0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int j = j0 + d;
      if (j < nj) {  // (uniform)
        const char* sb = reinterpret_cast<const char*>(slices + (d & 1) * SLICE) + tr_off;
        bf16x8_t bfr[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const gv4i16_t lo =
              __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_gv4i16_t*)(sb + 32 * nb));
          const gv4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_gv4i16_t*)(sb + 32 * nb + 8 * PITCH));
          const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3],
                                                               hi[0], hi[1], hi[2], hi[3]};
          bfr[nb] = __builtin_bit_cast(bf16x8_t, v);
        }
        lds_fence();
        // next step's W_g rows into the other slice
        if (j + 1 < nj) stage((d + 1) % D, j + 1, (d + 1) & 1);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int g = 0; g < TGB; ++g)
            acc[g][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, xr[d][g]), bfr[nb], acc[g][nb], 0, 0, 0);
      }
      issue(d, j + D);
      lds_fence();
    }
  }
  // the slices overlap other waves' partial tiles
  __syncthreads();
  // acc[g][nb][r]: token g * 16 + (lane / 16) * 4 + r, expert nb * 16 + lane % 16
#pragma unroll
  for (int g = 0; g < TGB; ++g)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        part[wave][g * kGateTok + (lane >> 4) * 4 + r][nb * 16 + (lane & 15)] = acc[g][nb][r];
  __syncthreads();
  // sum the partial tiles in wave order; bias; logits out
  for (int q = tid; q < TB * E; q += 64 * NW) {
    const int tt = q / E, e = q % E;
    float l = part[0][tt][e];
#pragma unroll
    for (int v = 1; v < NW; ++v) l += part[v][tt][e];
    if (bias != nullptr) l += bias[e];
    part[0][tt][e] = l;
    if (t0 + tt < T) logits[(long)(t0 + tt) * E + e] = l;
  }
  __syncthreads();
  if (E > 16) {
    // top-k: the block's first 256 lanes, P per token, logits read from LDS
    constexpr int P = 256 / TB;
    const int tt = tid / P, p = tid % P, t = t0 + tt;
    if (tid < 256 && t < T) {  // (whole P-lane groups: T bounds tokens, P divides 64)
      int32_t* io = idx + (long)t * k;
      float* wo = w + (long)t * k;
      if constexpr (P >= 8) {
        if (k <= 2) topk_extract<2, P>(part[0][tt], E, k, p, full, io, wo);
        else if (k <= 4) topk_extract<4, P>(part[0][tt], E, k, p, full, io, wo);
        else topk_extract<8, P>(part[0][tt], E, k, p, full, io, wo);
      } else {
        if (k <= 2) topk_lanes<2, P>(part[0][tt], E, k, p, full, io, wo);
        else if (k <= 4) topk_lanes<4, P>(part[0][tt], E, k, p, full, io, wo);
        else topk_lanes<8, P>(part[0][tt], E, k, p, full, io, wo);
      }
    }
  } else {
    // top-k: segments of EP <= 16 lanes, one token per segment per round
    const int G = 64 / EP;
    const int seg = lane / EP, e = lane % EP;
    const bool evalid = e < E;
    for (int i = wave * G + seg; i < TB; i += NW * G) {
      const int t = t0 + i;
      if (t >= T) break;  // uniform across the segment
      const float l = evalid ? part[0][i][e] : 0.f;
      topk_write(l, e, evalid, EP, k, full, idx + (long)t * k, w + (long)t * k);
    }
  }
}

// token groups per block: every block reads all of W_g (from L2), so wide
// gates take as many tokens per block as still leave a block per CU; narrow
// ones (E <= 16) stop at two groups, leaving two blocks per CU on long
// inputs, so that one block's top-k overlaps another's loads
inline int gate_groups_per_block(int T, int E) {
  const int groups = (T + kGateTok - 1) / kGateTok;
  if (E <= 16) return groups >= 1024 ? 2 : 1;
  if (groups >= 1024) return 4;
  if (groups >= 512) return 2;
  return 1;
}

// waves per block: wide gates with blocks of one token group split M
// eight ways
inline int gate_waves(int T, int E, int tgb) {
  (void)T;
  return tgb == 1 && E > 16 ? 8 : 4;
}

__global__ __launch_bounds__(kGateThreads) void route_kernel(const float* __restrict__ logits,
                                                             int32_t* __restrict__ idx,
                                                             float* __restrict__ w, int T, int E,
                                                             int k, int EP, int full) {
  const int G = 64 / EP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int seg = lane / EP, e = lane % EP;
  const int t = (blockIdx.x * 4 + wave) * G + seg;
  if (t >= T) return;  // uniform per segment
  const bool evalid = e < E;
  float l = evalid ? logits[(size_t)t * E + e] : 0.f;
  topk_write(l, e, evalid, EP, k, full, idx + (size_t)t * k, w + (size_t)t * k);
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

// dx[t] += dl_t W_g^T, one wave per token (W_g^T: E x M in the layer dtype,
// so that each selected expert's 8 consecutive m are one 16-byte load)
template <typename TIn>
__global__ __launch_bounds__(256) void gate_bwd_dx_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, const float* __restrict__ dw,
    const TIn* __restrict__ wgt, TIn* __restrict__ dx, int T, int M, int k) {
  const int lane = threadIdx.x & 63;
  const long t = blockIdx.x * 4L + (threadIdx.x >> 6);
  if (t >= T) return;
  int ij[kMaxK];
  float dl[kMaxK];
  token_dl(idx, w, dw, t, k, ij, dl);
  TIn* row = dx + t * M;
  for (int m = lane * 8; m < M; m += 64 * 8) {  // M is a multiple of 8
    // this step's dx and W_g^T rows loaded before the add and the store
    const auto xr = raw8_load(row + m);
    decltype(raw8_load(wgt)) gr[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) gr[j] = raw8_load(wgt + (long)ij[j] * M + m);
    float v[8];
    raw8_f32(xr, v);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        float g[8];
        raw8_f32(gr[j], g);
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
  // partial tiles by token lane: row i of the 8 x 8 tile of column group mg
  // at red[tl * RS + (i * 8 + mg) * NE + e], so that the 8 lanes of one tl
  // (mg = 0..7) write 8 consecutive runs of NE floats, and the lanes of
  // successive tl start 4 banks apart; the bias row at i = 8, mg = 0
  constexpr int RS = 9 * 8 * NE + 4;
  __shared__ float red[TL * RS];
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
    for (int q = 0; q < 8; ++q) red[tl * RS + (i * 8 + mg) * NE + e0 + q] = acc[i][q];
  if (first_tile && mg == 0) {
#pragma unroll
    for (int q = 0; q < 8; ++q) red[tl * RS + 64 * NE + e0 + q] = accb[q];
  }
  __syncthreads();
  const int rows = first_tile ? 65 : 64;
  for (int q = tid; q < rows * NE; q += 256) {
    const int mm = q / NE, e = q % NE;
    if (e >= E) continue;
    // row mm = 8 mg + i of the m tile (mm = 64: the bias row)
    const int at = (mm == 64 ? 64 : (mm & 7) * 8 + (mm >> 3)) * NE + e;
    float v = 0.f;
    for (int l = 0; l < TL; ++l) v += red[l * RS + at];
    if (mm == 64) {
      Pb[(long)s * E + e] = v;
    } else {
      const int m = blockIdx.x * 64 + mm;
      if (m < M) P[((long)s * M + m) * E + e] = v;
    }
  }
}

// bf16 layers: d_logits of 64 tokens per block, written as float (the
// output) and, for the full softmax gate's GEMM path, as a bf16 pair hi + lo
// per value (hi = bf16(dl), lo = bf16(dl - hi): about 16 significant bits)
// in rows [hi(E4) | lo(E4)]; db partials per block (token order); block 0
// also writes the row counts and offsets of that GEMM's token splits.
constexpr int kDlTok = 64;
__device__ __forceinline__ void dl_rows(
    int blk, float (*tile)[kMaxE + 1], const int32_t* __restrict__ idx,
    const float* __restrict__ w, const float* __restrict__ dw, const float* __restrict__ logits,
    float* __restrict__ d_logits, bf16_t* __restrict__ dlhl, float* __restrict__ Pb,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int T, int E, int E4, int k,
    int S, int tps, int full) {
  // (dense tile of the block's d_logits rows; odd pitch: column sums and row
  // writes both spread over the banks)
  const int tid = threadIdx.x;
  const long t0 = (long)blk * kDlTok;
  for (int q = tid; q < kDlTok * (kMaxE + 1); q += 256) (&tile[0][0])[q] = 0.f;
  if (counts != nullptr && blk == 0 && tid < S) {
    const long r0 = (long)tid * tps;
    counts[tid] = (int32_t)(r0 < T ? min((long)tps, T - r0) : 0);
    offsets[tid] = (int32_t)(r0 < T ? r0 : T);
  }
  __syncthreads();
  if (tid < kDlTok && t0 + tid < T) {
    const long t = t0 + tid;
    int ij[kMaxK];
    float dl[kMaxK];
    token_dl(idx, w, dw, t, k, ij, dl);
    if (full) {
      // the full softmax gate: every expert gets -p_e s (p the softmax over
      // all E logits, shifted by their maximum; s = sum_j w_j dw_j), the
      // selected ones w_j (dw_j - s) next
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < kMaxK; ++j)
        if (j < k) s += w[t * k + j] * dw[t * k + j];
      const float* lr = logits + t * E;
      float vmax = lr[0];
      for (int e = 1; e < E; ++e) vmax = fmaxf(vmax, lr[e]);
      float z = 0.f;
      for (int e = 0; e < E; ++e) z += expf(lr[e] - vmax);
      const float f = -s / z;
      for (int e = 0; e < E; ++e) tile[tid][e] = expf(lr[e] - vmax) * f;
    }
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) tile[tid][ij[j]] = dl[j];  // the k selected experts are distinct
  }
  __syncthreads();
  for (int q = tid; q < kDlTok * E4; q += 256) {
    const int tt = q / E4, e = q % E4;
    const long t = t0 + tt;
    if (t >= T) break;
    const float v = tile[tt][e];
    if (e < E) d_logits[t * E + e] = v;
    if (dlhl != nullptr) {
      const bf16_t hi = f32_to_bf16(v);
      dlhl[t * 2 * E4 + e] = hi;
      dlhl[t * 2 * E4 + E4 + e] = f32_to_bf16(v - bf16_to_f32(hi));
    }
  }
  if (tid < E) {
    float v = 0.f;
    for (int tt = 0; tt < kDlTok; ++tt) v += tile[tt][tid];  // rows past T are zero
    Pb[(long)blk * E + tid] = v;
  }
}

__global__ __launch_bounds__(256) void gate_bwd_dl_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, const float* __restrict__ dw,
    const float* __restrict__ logits, float* __restrict__ d_logits, bf16_t* __restrict__ dlhl,
    float* __restrict__ Pb, int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int T,
    int E, int E4, int k, int S, int tps, int full) {
  __shared__ float tile[kDlTok][kMaxE + 1];
  dl_rows(blockIdx.x, tile, idx, w, dw, logits, d_logits, dlhl, Pb, counts, offsets, T, E, E4, k,
          S, tps, full);
}

// dW_g of the renormalised bf16 gate on MFMA (v_mfma_f32_16x16x32_bf16),
// one launch with the d_logits rows. Blocks [0, ndl) are dl_rows blocks
// (d_logits, db partials per 64 tokens). Each other block takes MT columns
// m0 .. m0 + MT - 1 of x (rows of dW_g) over one token split [tb, te) and
// computes, in chunks of 64 tokens,
//   Q[r][m] = sum over the chunk's tokens t of D[r][t] x[t][m],
// where row r = 2 e + h of D holds the bf16 part hi (h = 0) or the rest lo
// (h = 1) of d_logits[t][e] (hi = bf16(dl), lo = bf16(dl - hi): about 16
// significant bits; zero for experts a token did not select), and finally
// P[split][m][e] = Q[2 e][m] + Q[2 e + 1][m], summed over the splits in
// order by the reduce launch. Building a chunk: every thread computes the
// d_logits of its token's selection (4 threads a token, two entries each,
// the sum s over the k entries in entry order as token_dl takes it, the
// entries gathered from the quad by DPP), stores its part of the x tile
// (loaded kDwDepth chunks ahead in registers), clears the entries it wrote
// two chunks earlier into the same D buffer and writes its new ones (both
// D buffers start zero, so only entries are ever written). Multiplying a
// chunk: each wave takes its row tiles of D (A operand, 16-byte row reads:
// 8 consecutive tokens of one row) times its 16 columns of the x tile (B
// operand, two transposing reads: 8 consecutive tokens of one column). D
// and the x tile are double-buffered; each step multiplies chunk c and
// builds chunk c + 1, then meets the block at one barrier. Every load is
// issued unconditionally from a clamped address (tokens past the split: its
// first token, whose entries are not used; columns past M: column 0, whose
// results are not written). The block's partial rows go out through LDS as
// one contiguous range.
constexpr int kDwTok = 64;    // tokens per chunk
constexpr int kDwDepth = 4;   // chunks of loads in flight
constexpr int kDwDPitch = 72; // bf16 per row of D (64 tokens + 8: 16-byte aligned rows, 4 banks apart)

template <int S_>
__device__ __forceinline__ float quad_bcast(float v) {  // lane S_ of each quad
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), S_ * 0x55, 0xF, 0xF, false));
}

// NR 16-row tiles of D (2 E <= 16 NR); kDwCols columns of x per block, each
// wave one 16-column tile and every row tile (32 columns, each wave half of
// the row tiles, measured 5-10% slower at E = 64)
constexpr int kDwCols = 64;
template <int NR>
__global__ __launch_bounds__(256) void gate_dw_mfma_kernel(
    const bf16_t* __restrict__ x, const int32_t* __restrict__ idx, const float* __restrict__ w,
    const float* __restrict__ dw, float* __restrict__ d_logits, float* __restrict__ P,
    float* __restrict__ Pb, int T, int M, int E, int k, int tps, int mtiles, int ndl) {
  constexpr int MT = kDwCols;
  constexpr int XP = MT + 8;                // bf16 per x tile row
  constexpr int XT = kDwTok * XP;           // bf16 per x tile
  constexpr int DT = 16 * NR * kDwDPitch;   // bf16 per D tile
  constexpr int XPT = MT / 32;              // 16-byte x pieces per thread and chunk
  constexpr int CPR = MT / 8;               // 16-byte pieces per token row
  constexpr int CT = MT / 16;               // column tiles
  constexpr int WG = 4 / CT;                // wave groups over the row tiles
  constexpr int RT = NR / WG;               // row tiles per wave
  static_assert(RT >= 1 && RT * WG == NR, "row tiles split evenly over the wave groups");
  constexpr int DW_BYTES = 2 * (XT + DT) * 2;
  constexpr int DL_BYTES = kDlTok * (kMaxE + 1) * 4;
  constexpr int D = kDwDepth;
  typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) char smem[DW_BYTES > DL_BYTES ? DW_BYTES : DL_BYTES];
  if ((int)blockIdx.x < ndl) {  // (uniform)
    dl_rows(blockIdx.x, reinterpret_cast<float(*)[kMaxE + 1]>(smem), idx, w, dw, nullptr, d_logits,
            nullptr, Pb, nullptr, nullptr, T, E, E, k, 0, 0, 0);
    return;
  }
  const int blk = blockIdx.x - ndl;
  const int mt = blk % mtiles, sp = blk / mtiles;
  const int m0 = mt * MT;
  const int tb = sp * tps, te = min(T, tb + tps);  // (tb < T: every split holds tokens)
  const int nch = (te - tb + kDwTok - 1) / kDwTok;
  bf16_t* xt = reinterpret_cast<bf16_t*>(smem);  // [2][kDwTok][XP]: tokens x columns
  bf16_t* dt = xt + 2 * XT;                      // [2][16 NR][kDwDPitch]: rows r x tokens
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ct = wave % CT, rg = wave / CT;
  // x: XPT 16-byte pieces a thread, tokens tid / CPR + (256 / CPR) h of the
  // chunk, columns m0 + xc .. + 7
  const int xc = 8 * (tid % CPR);
  const int xm = m0 + xc < M ? m0 + xc : 0;
  // selection: token st of the chunk, entries q and q + 4
  const int st = tid >> 2, q = tid & 3;
  const int ja = q < k ? q : 0, jb = q + 4 < k ? q + 4 : 0;

  u32x4_t xr[D][XPT];
  int32_t ir[D][2];
  float wr[D][2], dr[D][2];
  auto issue = [&](int d, int c) __attribute__((always_inline)) {
    const int tc = tb + (c < nch ? c : nch - 1) * kDwTok;
#pragma unroll
    for (int h = 0; h < XPT; ++h) {
      const int t = tc + tid / CPR + (256 / CPR) * h;
      xr[d][h] = *reinterpret_cast<const u32x4_t*>(x + (long)(t < te ? t : tb) * M + xm);
    }
    const int t = tc + st;
    const long r = (long)(t < te ? t : tb) * k;
    ir[d][0] = idx[r + ja];
    ir[d][1] = idx[r + jb];
    wr[d][0] = w[r + ja];
    wr[d][1] = w[r + jb];
    dr[d][0] = dw[r + ja];
    dr[d][1] = dw[r + jb];
  };

  // both D buffers zero
  for (int u = tid; u < 2 * DT / 8; u += 256)
    reinterpret_cast<u32x4_t*>(dt)[u] = u32x4_t{0u, 0u, 0u, 0u};
  floatx4_t acc[RT];
#pragma unroll
  for (int i = 0; i < RT; ++i) acc[i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  // transposing reads of the x tile: lane l aims at token 8 (l / 16) + (l %
  // 16) / 4 (+ 4 for the second read) of a 32-token step, columns 16 ct +
  // 4 (l % 4) .. + 3, and receives 8 consecutive tokens of column 16 ct + l % 16
  const int tr_off = ((8 * (lane >> 4) + ((lane & 15) >> 2)) * XP + 16 * ct + 4 * (lane & 3)) * 2;
  // row reads of D: row l % 16 of a tile, tokens 8 (l / 16) .. + 7 of a step
  const int a_off = (((16 * RT * rg) + (lane & 15)) * kDwDPitch + 8 * (lane >> 4)) * 2;
  // D positions this thread wrote in each buffer for its last chunk there (-1: none)
  int pa0 = -1, pb0 = -1, pa1 = -1, pb1 = -1;

  // chunk c's x tile and D entries from ring slot d into buffers c & 1,
  // after clearing chunk c - 2's entries there (the same token columns:
  // only this thread's quad writes them, clears before sets in program
  // order; a token's selected experts are distinct)
  auto build = [&](int d, int c) __attribute__((always_inline)) {
    bf16_t* xb = xt + (c & 1) * XT;
    bf16_t* db = dt + (c & 1) * DT;
    // d_logits of this thread's two entries, as token_dl computes them
    float wv[kMaxK], dv[kMaxK];
    wv[0] = quad_bcast<0>(wr[d][0]), dv[0] = quad_bcast<0>(dr[d][0]);
    wv[1] = quad_bcast<1>(wr[d][0]), dv[1] = quad_bcast<1>(dr[d][0]);
    wv[2] = quad_bcast<2>(wr[d][0]), dv[2] = quad_bcast<2>(dr[d][0]);
    wv[3] = quad_bcast<3>(wr[d][0]), dv[3] = quad_bcast<3>(dr[d][0]);
    wv[4] = quad_bcast<0>(wr[d][1]), dv[4] = quad_bcast<0>(dr[d][1]);
    wv[5] = quad_bcast<1>(wr[d][1]), dv[5] = quad_bcast<1>(dr[d][1]);
    wv[6] = quad_bcast<2>(wr[d][1]), dv[6] = quad_bcast<2>(dr[d][1]);
    wv[7] = quad_bcast<3>(wr[d][1]), dv[7] = quad_bcast<3>(dr[d][1]);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) s += wv[j] * dv[j];
    const float dla = wr[d][0] * (dr[d][0] - s), dlb = wr[d][1] * (dr[d][1] - s);
    const bool live = tb + c * kDwTok + st < te;
    const int ea = ir[d][0], eb = ir[d][1];
    const int na = live && q < k && ea >= 0 && ea < E ? 2 * ea * kDwDPitch + st : -1;
    const int nb = live && q + 4 < k && eb >= 0 && eb < E ? 2 * eb * kDwDPitch + st : -1;
#pragma unroll
    for (int h = 0; h < XPT; ++h)
      *reinterpret_cast<u32x4_t*>(xb + (tid / CPR + (256 / CPR) * h) * XP + xc) = xr[d][h];
    int& qa = (c & 1) ? pa1 : pa0;
    int& qb = (c & 1) ? pb1 : pb0;
    if (qa >= 0) db[qa] = db[qa + kDwDPitch] = (bf16_t)0;
    if (qb >= 0) db[qb] = db[qb + kDwDPitch] = (bf16_t)0;
    if (na >= 0) {
      const bf16_t hi = f32_to_bf16(dla);
      db[na] = hi;
      db[na + kDwDPitch] = f32_to_bf16(dla - bf16_to_f32(hi));
    }
    if (nb >= 0) {
      const bf16_t hi = f32_to_bf16(dlb);
      db[nb] = hi;
      db[nb + kDwDPitch] = f32_to_bf16(dlb - bf16_to_f32(hi));
    }
    qa = na, qb = nb;
  };
  // chunk c: D times the x tile from buffers c & 1
  auto multiply = [&](int c) __attribute__((always_inline)) {
    const char* xbc = reinterpret_cast<const char*>(xt + (c & 1) * XT);
    const char* dbc = reinterpret_cast<const char*>(dt + (c & 1) * DT);
#pragma unroll
    for (int ks = 0; ks < kDwTok / 32; ++ks) {
      const char* bp = xbc + tr_off + ks * 32 * XP * 2;
      const gv4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_gv4i16_t*)bp);
      const gv4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_gv4i16_t*)(bp + 8 * XP));
      const short __attribute__((ext_vector_type(8))) bv = {lo[0], lo[1], lo[2], lo[3],
                                                            hi[0], hi[1], hi[2], hi[3]};
      const bf16x8_t bfr = __builtin_bit_cast(bf16x8_t, bv);
#pragma unroll
      for (int i = 0; i < RT; ++i) {
        const bf16x8_t afr = *reinterpret_cast<const bf16x8_t*>(
            dbc + a_off + (16 * i * kDwDPitch + 32 * ks) * 2);
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr, bfr, acc[i], 0, 0, 0);
      }
    }
  };

  // One barrier a chunk: iteration c multiplies chunk c, builds chunk c + 1
  // into the other buffers (last read by chunk c - 1, which every wave
  // finished before the previous barrier) and reloads that ring slot D
  // chunks ahead. Whole rounds of D chunks run without branches (the
  // compiler's load counting stays exact); the last chunks after the loop
  // load nothing more.
#pragma unroll
  for (int d = 0; d < D; ++d) issue(d, d);
  build(0, 0);
  issue(0, D);
  __syncthreads();
  int c0 = 0;
  for (; c0 + D < nch; c0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      multiply(c0 + d);
      build((d + 1) % D, c0 + d + 1);
      issue((d + 1) % D, c0 + d + 1 + D);
      __syncthreads();
    }
  }
#pragma unroll
  for (int d = 0; d < D; ++d) {
    if (c0 + d < nch) {  // (uniform)
      multiply(c0 + d);
      if (c0 + d + 1 < nch) build((d + 1) % D, c0 + d + 1);
      __syncthreads();
    }
  }
  // acc[i][j]: Q row 16 (RT rg + i) + 4 (lane / 16) + j, column m0 + 16 ct + lane % 16.
  // The block's partial rows P[split][m0 .. m0 + MT)[0 .. E) are one
  // contiguous range: staged in LDS (free after the loop's last barrier),
  // then written as whole 16-byte pieces (4-byte scattered stores of the
  // accumulators took 3 of the 16 us of a 4096-token chunk at E = 64).
  constexpr int PP = kMaxE + 4;  // staging row pitch (floats)
  static_assert(MT * PP * 4 <= DW_BYTES, "the staging fits the block's LDS");
  float* pt = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int i2 = 0; i2 < 2; ++i2) {
      const int e = 8 * (RT * rg + i) + 2 * (lane >> 4) + i2;
      if (e < E) pt[(16 * ct + (lane & 15)) * PP + e] = acc[i][2 * i2] + acc[i][2 * i2 + 1];
    }
  __syncthreads();
  const int rows = min(MT, M - m0), n = rows * E;
  float* pr = P + ((long)sp * M + m0) * E;
  if (E % 4 == 0) {
    for (int q4 = 4 * tid; q4 < n; q4 += 4 * 256) {
      const int r = q4 / E, e = q4 - r * E;
      *reinterpret_cast<float4*>(pr + q4) = *reinterpret_cast<const float4*>(pt + r * PP + e);
    }
  } else {
    for (int q1 = tid; q1 < n; q1 += 256) {
      const int r = q1 / E;
      pr[q1] = pt[r * PP + (q1 - r * E)];
    }
  }
}

// the full softmax gate's dense dx term takes dx += [hi | lo] B with
// B = [W_g^T ; W_g^T] (2 E4 x M, bf16; rows e >= E of each half zero)
__global__ __launch_bounds__(256) void gate_wstack_kernel(const bf16_t* __restrict__ wg,
                                                          bf16_t* __restrict__ wstack, int M,
                                                          int E, int E4) {
  const long n = 2L * E4 * M;
  for (long q = blockIdx.x * 256L + threadIdx.x; q < n; q += (long)gridDim.x * 256) {
    const long r = q / M, m = q - r * M;
    const int e = (int)(r % E4);
    wstack[q] = e < E ? wg[m * E + e] : (bf16_t)0;
  }
}

// dW_g[m][e] = sum over splits of P[s][m][e] (split order; rows of pitch
// ldp), plus the same sum over column lo_off + e when lo_off >= 0 (the lo
// halves of the bf16 path), one thread an element, in blocks [0, nw) (nw =
// ceil(M E / 256)); db[e] = sum over the SB rows of Pb, block nw + e: each
// thread the rows i, i + 256, ... in order, then a fixed pairwise tree (a
// lone thread's serial sum over thousands of rows took tens of us).
// Blocks past the reduction's (wt_block = nw + E and on, when wg is given)
// copy W_g (M x E) to W_g^T (E x M) in the layer dtype for the dx term: one
// launch less than a kernel of its own.
__global__ __launch_bounds__(256) void gate_bwd_dw_reduce_kernel(
    const float* __restrict__ P, const float* __restrict__ Pb, float* __restrict__ dw_gate,
    float* __restrict__ dbias, int M, int E, int S, int ldp, int lo_off, int SB, int accumulate,
    const void* __restrict__ wg, void* __restrict__ wgt, int wt_block, int bf) {
  const long n = (long)M * E;
  if (wg != nullptr && (int)blockIdx.x >= wt_block) {
    const long r = ((long)blockIdx.x - wt_block) * 256 + threadIdx.x;
    if (r >= n) return;
    const long e = r / M, m = r % M;
    if (bf)
      static_cast<bf16_t*>(wgt)[r] = static_cast<const bf16_t*>(wg)[m * E + e];
    else
      static_cast<float*>(wgt)[r] = static_cast<const float*>(wg)[m * E + e];
    return;
  }
  const int nw = (int)((n + 255) / 256);
  if ((int)blockIdx.x >= nw) {
    const int e = (int)blockIdx.x - nw;
    if (e >= E || dbias == nullptr) return;  // (uniform)
    __shared__ float red[256];
    const int tid = threadIdx.x;
    float v = 0.f;
    for (int s = tid; s < SB; s += 256) v += Pb[(long)s * E + e];
    red[tid] = v;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
      if (tid < off) red[tid] += red[tid + off];
      __syncthreads();
    }
    if (tid == 0) dbias[e] = accumulate ? dbias[e] + red[0] : red[0];
    return;
  }
  const long q = blockIdx.x * 256L + threadIdx.x;
  if (q < n) {
    const long m = q / E, e = q % E;
    const long stride = (long)M * ldp;
    const float* p = P + m * ldp + e;
    float v = 0.f;
#pragma unroll 8
    for (int s = 0; s < S; ++s) v += p[s * stride];
    if (lo_off >= 0) {
      float vl = 0.f;
#pragma unroll 8
      for (int s = 0; s < S; ++s) vl += p[s * stride + lo_off];
      v += vl;
    }
    dw_gate[q] = accumulate ? dw_gate[q] + v : v;
  }
}

__global__ __launch_bounds__(256) void zero_f32_kernel(float* __restrict__ p, long n) {
  for (long q = blockIdx.x * 256L + threadIdx.x; q < n; q += (long)gridDim.x * 256) p[q] = 0.f;
}

int gate_eg(int E) { return E <= 8 ? 1 : E <= 16 ? 2 : E <= 32 ? 4 : 8; }

// bf16 path: the GEMM's column count (hi and lo halves of E rounded up to 4)
int gate_dw_cols(int E) { return 2 * ((E + 3) / 4 * 4); }

// dW_g paths: the renormalised bf16 gate takes the MFMA kernel (d_logits
// rows and dW_g partials in one launch, then the reduce); the full softmax
// gate d_logits, then dW_g as a GEMM (its hi/lo rows also feed the dense dx
// GEMM); fp32 gates the register-tile kernel
bool gate_dw_on_mfma(const Shape& s) {
  return s.dtype == FLOWMOE_BF16 && s.gate != FLOWMOE_GATE_FULL;
}
bool gate_dw_on_gemm(const Shape& s) { return s.gate == FLOWMOE_GATE_FULL; }

// MFMA path: token splits (multiples of 64 tokens): about two blocks per
// CU over the 64-column tiles, partials (splits x M x E floats) at most a
// quarter of x's bytes
int gate_dwm_tps(const Shape& s) {
  const long mtiles = (s.M + kDwCols - 1) / kDwCols;
  long sp = (512 + mtiles - 1) / mtiles;
  const long by_bytes = s.T / (8L * s.E), by_chunks = (s.T + kDwTok - 1) / kDwTok;
  if (sp > by_bytes) sp = by_bytes;
  if (sp > by_chunks) sp = by_chunks;
  if (sp < 1) sp = 1;
  const long tps = (s.T + sp - 1) / sp;
  return (int)((tps + kDwTok - 1) / kDwTok * kDwTok);
}
int gate_dwm_splits(const Shape& s) {
  const int tps = gate_dwm_tps(s);
  return s.T > 0 ? (s.T + tps - 1) / tps : 1;
}

// GEMM path: token splits of the dW_g GEMM (its pseudo-experts): about 256
// blocks of 256 x 256 tiles, at least 128 tokens per split, at most 16 MB
// of fp32 partials
int gate_dw_splits(const Shape& s) {
  const long mt = (s.M + 255) / 256, nt = (gate_dw_cols(s.E) + 255) / 256;
  long sp = 256 / (mt * nt);
  const long by_tokens = s.T / 128, by_bytes = (16L << 20) / ((long)s.M * gate_dw_cols(s.E) * 4);
  if (sp > by_tokens) sp = by_tokens;
  if (sp > by_bytes) sp = by_bytes;
  if (sp > 64) sp = 64;
  return sp < 1 ? 1 : (int)sp;
}

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
  const int full = s.gate == FLOWMOE_GATE_FULL;
  if (s.dtype == FLOWMOE_BF16) {
    const int NB = (s.E + 15) / 16;
    const int TGB = gate_groups_per_block(s.T, s.E);
    const int blocks = (s.T + kGateTok * TGB - 1) / (kGateTok * TGB);
    const int NW = gate_waves(s.T, s.E, TGB);
    return traced(FLOWMOE_K_GATE, st, [&] {
#define FLOWMOE_GATE_KERNEL(NBV, TGBV, NWV, VECV)                                                 \
  hipLaunchKernelGGL((gate_topk_mfma_kernel<NBV, TGBV, NWV, VECV>), dim3(blocks), dim3(64 * NWV), \
                     0, st, (const bf16_t*)x, (const bf16_t*)w_gate, bias, logits, idx, w, s.T,   \
                     s.M, s.E, s.k, EP, full)
#define FLOWMOE_GATE_LAUNCH(NBV, TGBV, NWV)                          \
  do {                                                               \
    if (s.E % 8 == 0) FLOWMOE_GATE_KERNEL(NBV, TGBV, NWV, true);    \
    else FLOWMOE_GATE_KERNEL(NBV, TGBV, NWV, false);                \
  } while (0)
#define FLOWMOE_GATE_NB(TGBV, NWV)                     \
  if (NB == 1) FLOWMOE_GATE_LAUNCH(1, TGBV, NWV);      \
  else if (NB == 2) FLOWMOE_GATE_LAUNCH(2, TGBV, NWV); \
  else if (NB == 3) FLOWMOE_GATE_LAUNCH(3, TGBV, NWV); \
  else FLOWMOE_GATE_LAUNCH(4, TGBV, NWV);
      if (TGB == 1) {
        if (NW == 8) { FLOWMOE_GATE_NB(1, 8) }
        else { FLOWMOE_GATE_NB(1, 4) }
      } else if (TGB == 2) { FLOWMOE_GATE_NB(2, 4) }
      else { FLOWMOE_GATE_NB(4, 4) }
#undef FLOWMOE_GATE_NB
#undef FLOWMOE_GATE_LAUNCH
#undef FLOWMOE_GATE_KERNEL
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
                       s.E, s.k, EP, TPG, xchunk, full);
  });
}

hipError_t launch_route(const Shape& s, const float* logits, int32_t* idx, float* w, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int EP = pow2_at_least(s.E);
  const int per_block = 4 * (64 / EP);
  const int blocks = (s.T + per_block - 1) / per_block;
  return traced(FLOWMOE_K_ROUTE, st, [&] {
    hipLaunchKernelGGL(route_kernel, dim3(blocks), dim3(kGateThreads), 0, st, logits, idx, w, s.T,
                       s.E, s.k, EP, (int)(s.gate == FLOWMOE_GATE_FULL));
  });
}

// workspace: [W_g^T (E x M float) | P | Pb | GEMM path: dl hi/lo (T x N bf16),
// split counts and offsets (S int32 each)]; MFMA path: P (S x M x E), Pb
// (ceil(T/64) x E); register-tile path: P (S x M x E), Pb (S x E); GEMM path:
// P (S x M x N, N = gate_dw_cols(E)), Pb (ceil(T/64) x E)
size_t gate_wt_bytes(const Shape& s) { return align256((size_t)s.M * s.E * sizeof(float)); }

namespace {
struct GateWs {
  float* P;
  float* Pb;
  bf16_t* dlhl;
  int32_t* counts;
  int32_t* offsets;
  bf16_t* wstack;  // full softmax gate: [W_g^T ; W_g^T] (2 E4 x M) for the dx GEMM
  size_t bytes;    // from the start of the workspace
};
GateWs gate_ws(const Shape& s, void* ws) {
  char* base = static_cast<char*>(ws);
  size_t off = gate_wt_bytes(s);
  GateWs g = {};
  auto take = [&](size_t n) {
    char* p = base ? base + off : nullptr;
    off += align256(n);
    return p;
  };
  if (gate_dw_on_mfma(s)) {
    const int S = gate_dwm_splits(s);
    const long nb = (s.T + kDlTok - 1) / kDlTok;
    g.P = reinterpret_cast<float*>(take((size_t)S * s.M * s.E * sizeof(float)));
    g.Pb = reinterpret_cast<float*>(take((size_t)(nb > 0 ? nb : 1) * s.E * sizeof(float)));
  } else if (gate_dw_on_gemm(s)) {
    const int S = gate_dw_splits(s), N = gate_dw_cols(s.E);
    const long nb = (s.T + kDlTok - 1) / kDlTok;
    g.P = reinterpret_cast<float*>(take((size_t)S * s.M * N * sizeof(float)));
    g.Pb = reinterpret_cast<float*>(take((size_t)(nb > 0 ? nb : 1) * s.E * sizeof(float)));
    g.dlhl = reinterpret_cast<bf16_t*>(take((size_t)s.T * N * sizeof(bf16_t)));
    g.counts = reinterpret_cast<int32_t*>(take((size_t)S * sizeof(int32_t)));
    g.offsets = reinterpret_cast<int32_t*>(take((size_t)S * sizeof(int32_t)));
    if (s.gate == FLOWMOE_GATE_FULL)
      g.wstack = reinterpret_cast<bf16_t*>(take((size_t)N * s.M * sizeof(bf16_t)));
  } else {
    const int S = gate_splits(s);
    g.P = reinterpret_cast<float*>(take((size_t)S * s.M * s.E * sizeof(float)));
    g.Pb = reinterpret_cast<float*>(take((size_t)S * s.E * sizeof(float)));
  }
  g.bytes = off;
  return g;
}
}  // namespace

size_t gate_bwd_ws_bytes(const Shape& s) { return gate_ws(s, nullptr).bytes; }

hipError_t launch_gate_wstack(const Shape& s, const void* w_gate, void* ws, hipStream_t st) {
  const GateWs g = gate_ws(s, ws);
  const int E4 = gate_dw_cols(s.E) / 2;
  const long n = 2L * E4 * s.M;
  const int nb = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  return traced(FLOWMOE_K_GATE_BWD_WT, st, [&] {
    hipLaunchKernelGGL(gate_wstack_kernel, dim3(nb), dim3(256), 0, st, (const bf16_t*)w_gate,
                       g.wstack, s.M, s.E, E4);
  });
}

hipError_t launch_gate_dx_full(const Shape& s, void* ws, void* dx, bool add, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const GateWs g = gate_ws(s, ws);
  return launch_gate_dx_gemm(g.dlhl, s.T, gate_dw_cols(s.E), g.wstack, s.M, g.counts, g.offsets,
                             gate_dw_splits(s), dx, add, st);
}

hipError_t launch_gate_dx(const Shape& s, const int32_t* idx, const float* w, const float* dw,
                          const void* wgt, void* dx, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const int tb = (s.T + 3) / 4;
  return traced(FLOWMOE_K_GATE_BWD_TOKEN, st, [&] {
    if (s.dtype == FLOWMOE_BF16)
      hipLaunchKernelGGL(gate_bwd_dx_kernel<bf16_t>, dim3(tb), dim3(256), 0, st, idx, w, dw,
                         (const bf16_t*)wgt, (bf16_t*)dx, s.T, s.M, s.k);
    else
      hipLaunchKernelGGL(gate_bwd_dx_kernel<float>, dim3(tb), dim3(256), 0, st, idx, w, dw,
                         (const float*)wgt, (float*)dx, s.T, s.M, s.k);
  });
}

hipError_t launch_gate_dw(const Shape& s, const void* x, const float* logits, const int32_t* idx,
                          const float* w, const float* dw, float* d_logits, float* dw_gate,
                          float* dbias, int accumulate, void* ws, hipStream_t st,
                          const void* w_gate) {
  const GateWs g = gate_ws(s, ws);
  const bool bf = s.dtype == FLOWMOE_BF16;
  // reduce blocks: dW_g elements, then one block per db entry
  const int nred = (int)(((long)s.M * s.E + 255) / 256) + s.E;
  // with w_gate, the reduce launch also writes W_g^T at the front of ws
  const int ntr = w_gate != nullptr ? (int)(((long)s.M * s.E + 255) / 256) : 0;
  if (gate_grad_zero(s) && s.T > 0) {
    // d_logits is exactly zero: nothing of x is read
    const long nz = (long)s.T * s.E;
    hipError_t e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
      hipLaunchKernelGGL(zero_f32_kernel, dim3((unsigned)((nz + 255) / 256 < 1024 ? (nz + 255) / 256 : 1024)),
                         dim3(256), 0, st, d_logits, nz);
    });
    if (e != hipSuccess) return e;
  }
  if (s.T == 0 || gate_grad_zero(s)) {
    // with no tokens (or d_logits = 0) the gradient is zero: a reduce over
    // zero splits writes it
    if (accumulate && ntr == 0) return hipSuccess;
    return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
      hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(accumulate ? ntr : nred + ntr), dim3(256),
                         0, st, g.P, g.Pb, dw_gate, dbias, s.M, s.E, 0, s.E, -1, 0, 0, w_gate, ws,
                         accumulate ? 0 : nred, (int)bf);
    });
  }
  if (gate_dw_on_mfma(s)) {
    const int tps = gate_dwm_tps(s), S = gate_dwm_splits(s);
    const int mtiles = (s.M + kDwCols - 1) / kDwCols;
    const int ndl = (s.T + kDlTok - 1) / kDlTok;
    const int nr = (2 * s.E + 15) / 16;
    const dim3 grid(ndl + mtiles * S);
    hipError_t e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
#define FLOWMOE_DWM_LAUNCH(NRV)                                                                   \
  hipLaunchKernelGGL(gate_dw_mfma_kernel<NRV>, grid, dim3(256), 0, st, (const bf16_t*)x, idx, w,   \
                     dw, d_logits, g.P, g.Pb, s.T, s.M, s.E, s.k, tps, mtiles, ndl)
      if (nr <= 1) FLOWMOE_DWM_LAUNCH(1);
      else if (nr <= 2) FLOWMOE_DWM_LAUNCH(2);
      else if (nr <= 4) FLOWMOE_DWM_LAUNCH(4);
      else FLOWMOE_DWM_LAUNCH(8);
#undef FLOWMOE_DWM_LAUNCH
    });
    if (e != hipSuccess) return e;
    return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
      hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(nred + ntr), dim3(256), 0, st, g.P, g.Pb,
                         dw_gate, dbias, s.M, s.E, S, s.E, -1, ndl, accumulate, w_gate, ws, nred,
                         (int)bf);
    });
  }
  if (gate_dw_on_gemm(s)) {
    // d_logits (and its hi/lo copy), then dW_g = x^T [hi | lo] as a weight-
    // gradient GEMM whose pseudo-experts are the token splits, then the sum
    // over splits and halves
    const int S = gate_dw_splits(s), N = gate_dw_cols(s.E);
    const int tps = (s.T + S - 1) / S;
    const int nb = (s.T + kDlTok - 1) / kDlTok;
    hipError_t e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
      hipLaunchKernelGGL(gate_bwd_dl_kernel, dim3(nb), dim3(256), 0, st, idx, w, dw, logits,
                         d_logits, g.dlhl, g.Pb, g.counts, g.offsets, s.T, s.E, N / 2, s.k, S,
                         tps, (int)(s.gate == FLOWMOE_GATE_FULL));
    });
    if (e != hipSuccess) return e;
    e = launch_gate_dw_gemm(x, s.T, s.M, g.dlhl, N, g.counts, g.offsets, S, g.P, st);
    if (e != hipSuccess) return e;
    return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
      hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(nred + ntr), dim3(256), 0, st, g.P, g.Pb,
                         dw_gate, dbias, s.M, s.E, S, N, N / 2, nb, accumulate, w_gate, ws, nred,
                         (int)bf);
    });
  }
  const int S = gate_splits(s);
  const int tps = (s.T + S - 1) / S;
  const dim3 grid((s.M + 63) / 64, S);
  const int EG = gate_eg(s.E);
  hipError_t e = traced(FLOWMOE_K_GATE_BWD_DW, st, [&] {
#define FLOWMOE_DW_LAUNCH(EGV)                                                                    \
  if (bf)                                                                                         \
    hipLaunchKernelGGL((gate_bwd_dw_kernel<bf16_t, EGV>), grid, dim3(256), 0, st,                 \
                       (const bf16_t*)x, idx, w, dw, d_logits, g.P, g.Pb, s.T, s.M, s.E, s.k, tps); \
  else                                                                                            \
    hipLaunchKernelGGL((gate_bwd_dw_kernel<float, EGV>), grid, dim3(256), 0, st, (const float*)x, \
                       idx, w, dw, d_logits, g.P, g.Pb, s.T, s.M, s.E, s.k, tps);
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
  return traced(FLOWMOE_K_GATE_BWD_REDUCE, st, [&] {
    hipLaunchKernelGGL(gate_bwd_dw_reduce_kernel, dim3(nred + ntr), dim3(256), 0, st, g.P, g.Pb,
                       dw_gate, dbias, s.M, s.E, S, s.E, -1, S, accumulate, w_gate, ws, nred, (int)bf);
  });
}

hipError_t launch_gate_bwd(const Shape& s, const void* x, const void* w_gate, const float* logits,
                           const int32_t* idx, const float* w, const float* dw, float* d_logits,
                           float* dw_gate, float* dbias, void* dx, int accumulate, void* ws,
                           hipStream_t st) {
  const bool full = s.gate == FLOWMOE_GATE_FULL;
  // the sparse dx term reads W_g^T, which the dW_g reduce launch writes (with
  // d_logits = 0 the term is zero: dx is left as it is)
  if (gate_grad_zero(s)) dx = nullptr;
  const bool wt = dx != nullptr && s.T > 0 && !full;
  hipError_t e = launch_gate_dw(s, x, logits, idx, w, dw, d_logits, dw_gate, dbias, accumulate, ws,
                                st, wt ? w_gate : nullptr);
  if (e != hipSuccess || dx == nullptr || s.T == 0) return e;
  if (full) {  // dense d_logits: dx += [hi | lo] [W_g^T ; W_g^T]
    e = launch_gate_wstack(s, w_gate, ws, st);
    if (e != hipSuccess) return e;
    return launch_gate_dx_full(s, ws, dx, true, st);
  }
  return launch_gate_dx(s, idx, w, dw, gate_ws_wgt(ws), dx, st);
}

}  // namespace flowmoe
