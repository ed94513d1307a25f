// MFMA building blocks shared by the fused MoL kernels (scoring, rerank):
// the gating MLP + softmax + weighted sum for 16 items of one query held in
// the 16x16x32 register layout described below.
//
// Lane l of a wave: item column c = l % 16, group g = l / 16.  For one query
// the lane holds the component dot products s_p for the contiguous run
// p = base(g) + mu, mu < 2 Px, base(g) = 2 g Px.  This is the layout a
// 16x16x32 GEMM over rows r = 2 pq + q (two queries q) produces directly:
// lane group g receives rows 4 g .. 4 g + 3, i.e. pq in {2 g, 2 g + 1} of
// both queries (see mol_fused.hip).
//
//   GEMM2 (f16)   U^T[j][item] = W1'[j][:] . s[:, item] + b1'[j]
//                 s is the B operand: K slot 8g + e <-> p = base(g) + 8m + e.
//   SiLU          h'_j = u'_j / (1 + 2^{u'_j}),  u' = -log2(e) u
//   GEMM3 (f16)   l'^T[p][item] = -W2[p][:] . h'[:, item]
//                                 + log2(e) (a_x[item][p] + a_q[q][p] + b2[p])
//                 GEMM2's accumulators (row j = 16 jt + 4 g + i) are the B
//                 operand with K slot 8g + e of block m <-> j = 32 m +
//                 16 (e/4) + 4 g + e%4; W2's rows are ordered so that output
//                 row 16 pt + 4 g + i is p = base(g) + 4 pt + i, the lane's
//                 own s value.  log2(e) (a_x + a_q + b2) enters as the
//                 accumulator input (f32).
//   softmax, phi  w_p = 2^{l'_p}, phi = sum w_p s_p / sum w_p (s in f32),
//                 reduced over the 4 lanes of an item with permlane swaps.
// (Eq. 1 / Eq. 2 with the two-layer SiLU gating MLP of Appendix A.3.)
#pragma once

#include "mol_kernels.h"

namespace mol {
namespace tile {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x4_t mfma_bf16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_f16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
// (a, b) rounded to f16 (nearest-even) in the low / high half: one
// v_cvt_pk_f16_f32 on gfx950
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, f16x2_t));
}
// f16 bits of -scale * w (sign flipped on the integer side)
__device__ __forceinline__ uint32_t neg_bf16_to_f16_bits(bf16_t w, float scale) {
  const float v = scale * to_f32(static_cast<bf16_t>(w ^ 0x8000u));
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(v)));
}
// f16 hi + lo split of v, packed (hi in the low half)
__device__ __forceinline__ uint32_t split_f16(float v) {
  const float hi = static_cast<float>(static_cast<_Float16>(v));
  return pack_f16(hi, v - hi);
}

// Sum / max of x over the 4 lanes {c, c+16, c+32, c+48}, in all of them.
__device__ __forceinline__ float sum_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t v = __float_as_uint(y);
  auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float max_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(y);
  auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Margin of the bound phi <= max_p s_p under float32 rounding.  phi is
// formed as sum_p w_p s_p / sum_p w_p with w_p >= 0: each of the two sums of
// at most 64 terms is off by under 64 units of 2^-24 relative to
// sum_p w_p |s_p| (resp. sum_p w_p), and the reciprocal and product add a
// few more, so the computed phi exceeds max_p s_p by less than
// 140 * 2^-24 * max_p |s_p|.  The margin is 2^-12 (1 + max_p |s_p|), more
// than 100 times that.
__device__ __forceinline__ float bound_margin(float mabs) { return 0x1p-12f * (1.f + mabs); }

__device__ __forceinline__ int lane_base(int g, int PX) { return 2 * g * PX; }

// s_waitcnt immediate that waits until at most n vector-memory operations
// of this wave are outstanding (expcnt and lgkmcnt left unconstrained).
// Vector-memory loads complete in issue order, so after issuing the loads
// of later stages, vmcnt <= (their count) means every older load is done.
constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// LDS exchange point between lanes of one wave.  LDS operations of a wave
// execute in issue order, so waiting for the wave's own LDS accesses
// (lgkmcnt(0)) and stopping the compiler from moving memory accesses across
// is enough; a memory fence would also wait for every outstanding global
// load (vmcnt(0)), draining the LDS ring's prefetches.
__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));   // lgkmcnt(0) only
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// Workgroup barrier of the LDS ring: waits until at most VM of this wave's
// vector-memory operations are outstanding (its older direct-to-LDS copies
// have landed) and its LDS accesses are done, then joins the barrier.
// Unlike __syncthreads() it carries no memory fence, whose vmcnt(0) would
// also wait for the copies of later stages.
template <int VM>
__device__ __forceinline__ void ring_barrier() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wave priority around a chain of matrix instructions: while a wave issues
// its MFMAs it wins the SIMD's issue arbitration over the other wave's
// vector ALU stream, so the matrix pipe starts early and runs under that
// stream instead of after it.  Only the issue order changes.
__device__ __forceinline__ void mfma_priority_begin() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(1);
  __builtin_amdgcn_sched_barrier(0);
}
__device__ __forceinline__ void mfma_priority_end() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(0);
  __builtin_amdgcn_sched_barrier(0);
}

// Waits out the result latency of every matrix instruction issued before it
// (11 wait states: a v_mfma_f32_16x16x32 result is readable 7 issue slots
// after the MFMA, measured on gfx950; the kernels that use this issue no
// larger MFMA) at the end of a block whose successors read MFMA results.  The compiler's
// hazard padding does not cover every path into such a successor when the
// MFMAs are followed by scheduling-group pseudo-instructions: a skipped
// conditional block then left a GEMM3 result read with no wait states.
__device__ __forceinline__ void mfma_drain() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 2");
  __builtin_amdgcn_sched_barrier(0);
}

typedef __attribute__((address_space(3))) uint64_t lds_u64_t;

// LDS offset of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)(p)));
}

// One lane's 16 bytes of a direct global -> LDS copy of a 1 KB block: lane i
// writes LDS bytes [lds_block + 16 i, lds_block + 16 i + 16).  lds_block must
// be wave-uniform.  Issued as inline asm so that the compiler does not see
// an LDS store: it would otherwise make every later LDS read wait for all
// outstanding copies (vmcnt(0)), including the prefetches of later stages.
// The caller tracks completion with counted vmcnt waits (ring_barrier); M0
// is saved and restored around the copy.
__device__ __forceinline__ void copy16_to_lds(const void* src, uint32_t lds_block) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds_block)
      : "memory");
}

// Bitonic sort (descending) of SORT keys in LDS by one wave.
template <int SORT>
__device__ __noinline__ void wave_sort(lds_u64_t* r, int lane) {
  for (int size = 2; size <= SORT; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
      for (int t = 0; t < SORT / 128; ++t) {
        const int i = lane + 64 * t;
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const uint64_t a = r[lo], c = r[hi];
        if ((a < c) == desc) {
          r[lo] = c;
          r[hi] = a;
        }
      }
      wave_lds_sync();
    }
  }
}

// Running top-k of one query kept by one wave in LDS: list [0, 128) sorted
// descending, staging [128, 256); keys below the threshold are rejected.
struct WaveTopk {
  static constexpr int kList = 128;
  static constexpr int kStage = 128;
  uint64_t* reg;
  uint64_t theta;
  float theta_score;   // score of theta (-inf while the list is not full)
  int stg;
  int k;
  __device__ void init(uint64_t* region, int k_, int lane) {
    reg = region;
    theta = 0ull;
    theta_score = -__builtin_inff();
    stg = 0;
    k = k_;
    for (int i = lane; i < kList + kStage; i += 64) reg[i] = 0ull;
  }
  __device__ void merge(int lane) {
    wave_lds_sync();
    wave_sort<kList + kStage>((lds_u64_t*)reg, lane);
    for (int i = kList + lane; i < kList + kStage; i += 64) reg[i] = 0ull;
    wave_lds_sync();
    theta = reg[k - 1];
    theta_score = key_score(theta);
    stg = 0;
  }
  // offer one key per lane (0 = none); at most 16 lanes offer per call
  __device__ void offer(uint64_t key, int lane) {
    const bool pass = key > theta;
    const uint64_t mask = __ballot(pass);
    if (mask) {
      const int below = __popcll(mask & ((1ull << lane) - 1ull));
      if (pass) reg[kList + stg + below] = key;
      stg += __popcll(mask);
      if (stg > kStage - 16) merge(lane);
    }
  }
  // offer (score, item) from lanes with valid set: a float compare rejects
  // scores below the threshold's before any key is formed (a key beats
  // theta only if its score is at least theta's score)
  __device__ void offer_score(float score, int32_t item, bool valid, int lane) {
    const bool maybe = valid && score >= theta_score;
    if (__ballot(maybe) == 0ull) return;
    offer(maybe ? make_key(score, item) : 0ull, lane);
  }
  __device__ void flush(int lane) {
    if (stg > 0) merge(lane);
  }
};

// Sums over the 4 lanes {c, c+16, c+32, c+48} of an item of two (den,
// num) pairs a and b: three swaps, no copies.  The rows of 16 lanes end
// up holding a's sums (rows 0, 1) and b's (rows 2, 3); each lane returns
// the pair of its rows.  The additions pair rows (0 + 1) + (2 + 3), as
// sum_groups does.
__device__ __forceinline__ void row_sums(float da, float na, float db, float nb, float& den, float& num) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(da), __float_as_uint(na), false, false);
  const float sa = __uint_as_float(a[0]) + __uint_as_float(a[1]);   // rows: da01, na01, da23, na23
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(db), __float_as_uint(nb), false, false);
  const float sb = __uint_as_float(b[0]) + __uint_as_float(b[1]);   // rows: db01, nb01, db23, nb23
  auto u = __builtin_amdgcn_permlane32_swap(__float_as_uint(sa), __float_as_uint(sb), false, false);
  const float t = __uint_as_float(u[0]) + __uint_as_float(u[1]);    // rows: da, na, db, nb
  const uint32_t tb = __float_as_uint(t);
  auto v = __builtin_amdgcn_permlane16_swap(tb, tb, false, false);
  den = __uint_as_float(v[0]);                                       // rows: da, da, db, db
  num = __uint_as_float(v[1]);                                       // rows: na, na, nb, nb
}


// f32 pair -> bf16 pair (nearest-even), a in the low half
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}
// (a, b) as two bf16 terms: hi = bf16(x), lo = bf16(x - hi), so that hi + lo
// carries x to about 2^-17 relative (16 significant bits against f16's 11)
__device__ __forceinline__ void split_bf16(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = pack_bf16(a, b);
  lo = pack_bf16(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}

// Per-wave constants of the gating MLP in MFMA operand layouts.
//
// X2 (the two-term form): W1 and -W2 enter as their own bf16 values (exact),
// and the two operands computed on the way, -log2(e) s and h', as two bf16
// terms each (split_bf16), so GEMM2 and GEMM3 take two bf16 MFMAs per K
// block; the chain then holds phi to float32-like accuracy for gating
// weights far beyond the f16 form's range (Appendix A.3's MLP, unchanged).
template <int PX, int H, bool X2 = false>
struct MolMlp {
  static constexpr int P = 8 * PX;
  static constexpr int RUN = 2 * PX;
  static constexpr int KP = P / 32;   // K blocks of GEMM2
  static constexpr int JT = H / 16;   // output tiles of GEMM2
  static constexpr int KH = H / 32;   // K blocks of GEMM3
  static constexpr int PT = P / 16;   // output tiles of GEMM3
  static_assert(PT <= 4, "a_q + b2 operand holds at most 4 tiles");
  // first component of the run held by lane group g
  __device__ static int base(int g) { return lane_base(g, PX); }
  uint4 w1op[JT][KP];
  uint4 w2op[PT][KH];
  f32x4_t b1acc[JT];

  __device__ void load(const DevProb& pr, int c, int g) {
    const bf16_t* W1 = static_cast<const bf16_t*>(pr.W1);
    const bf16_t* W2 = static_cast<const bf16_t*>(pr.W2);
    const int base = lane_base(g, PX);
    // W1' = -log2(e) W1: row j, K slot 8g+e <-> p = base(g) + 8m + e
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const bf16_t* src = W1 + (16 * jt + c) * P + base + 8 * m;
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = X2 ? static_cast<uint32_t>(src[2 * e]) | (static_cast<uint32_t>(src[2 * e + 1]) << 16)
                    : neg_bf16_to_f16_bits(src[2 * e], kLog2e) |
                          (neg_bf16_to_f16_bits(src[2 * e + 1], kLog2e) << 16);
        w1op[jt][m] = make_uint4(w[0], w[1], w[2], w[3]);
      }
    // -W2: row 16 pt + c <-> p = base(c/4) + 4 pt + c%4; K slot 8g+e <-> j
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
      for (int m = 0; m < KH; ++m) {
        const int p = lane_base(c >> 2, PX) + 4 * pt + (c & 3);
        uint32_t w[4];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const int e0 = 2 * e2, e1 = 2 * e2 + 1;
          const int j0 = 32 * m + 16 * (e0 >> 2) + 4 * g + (e0 & 3);
          const int j1 = 32 * m + 16 * (e1 >> 2) + 4 * g + (e1 & 3);
          w[e2] = X2 ? (static_cast<uint32_t>(W2[p * H + j0]) ^ 0x8000u) |
                           ((static_cast<uint32_t>(W2[p * H + j1]) ^ 0x8000u) << 16)
                     : neg_bf16_to_f16_bits(W2[p * H + j0], 1.f) |
                           (neg_bf16_to_f16_bits(W2[p * H + j1], 1.f) << 16);
        }
        w2op[pt][m] = make_uint4(w[0], w[1], w[2], w[3]);
      }
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int i = 0; i < 4; ++i) b1acc[jt][i] = -kLog2e * pr.b1[16 * jt + 4 * g + i];
  }

  // The same for a problem with pr.P <= P components and pr.H <= H hidden
  // units: the missing rows and columns of W1, b1 and W2 are zero, so the
  // padded hidden units give h' = 0 and the padded components' logits keep
  // their accumulator input (set to -inf by the caller: zero weight).
  __device__ void load_padded(const DevProb& pr, int c, int g) {
    const bf16_t* W1 = static_cast<const bf16_t*>(pr.W1);
    const bf16_t* W2 = static_cast<const bf16_t*>(pr.W2);
    const int Pr = pr.P, Hr = pr.H;
    const int base = lane_base(g, PX);
    // every read is unconditional, from a clamped in-range index, and masked
    // afterwards: the reads are issued together instead of one branch (and
    // one wait) each
    auto w1 = [&](int j, int p) -> uint32_t {
      const bf16_t w = W1[min(j, Hr - 1) * Pr + min(p, Pr - 1)];
      const uint32_t keep = 0u - static_cast<uint32_t>((j < Hr) & (p < Pr));
      return (X2 ? static_cast<uint32_t>(w) : neg_bf16_to_f16_bits(w, kLog2e)) & keep;
    };
    auto w2 = [&](int p, int j) -> uint32_t {
      const bf16_t w = W2[min(p, Pr - 1) * Hr + min(j, Hr - 1)];
      const uint32_t keep = 0u - static_cast<uint32_t>((j < Hr) & (p < Pr));
      return (X2 ? static_cast<uint32_t>(w ^ 0x8000u) : neg_bf16_to_f16_bits(w, 1.f)) & keep;
    };
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        const int j = 16 * jt + c, p0 = base + 8 * m;
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = w1(j, p0 + 2 * e) | (w1(j, p0 + 2 * e + 1) << 16);
        w1op[jt][m] = make_uint4(w[0], w[1], w[2], w[3]);
      }
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
      for (int m = 0; m < KH; ++m) {
        const int p = lane_base(c >> 2, PX) + 4 * pt + (c & 3);
        uint32_t w[4];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const int e0 = 2 * e2, e1 = 2 * e2 + 1;
          const int j0 = 32 * m + 16 * (e0 >> 2) + 4 * g + (e0 & 3);
          const int j1 = 32 * m + 16 * (e1 >> 2) + 4 * g + (e1 & 3);
          w[e2] = w2(p, j0) | (w2(p, j1) << 16);
        }
        w2op[pt][m] = make_uint4(w[0], w[1], w[2], w[3]);
      }
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * jt + 4 * g + i;
        const float b = pr.b1[min(j, Hr - 1)];
        b1acc[jt][i] = j < Hr ? -kLog2e * b : 0.f;
      }
  }

  // The stages of the chain for one query, without scheduling fences.
  // s: the lane's run of s values; c0: log2(e) (a_x + a_q + b2) in the
  // GEMM3 accumulator layout (element i of tile pt <-> p = base(g) + 4 pt + i).
  __device__ static void pack_s(const float (&s)[RUN], uint4 (&sop)[KP]) {
#pragma unroll
    for (int m = 0; m < KP; ++m)
      sop[m] = make_uint4(pack_f16(s[8 * m + 0], s[8 * m + 1]), pack_f16(s[8 * m + 2], s[8 * m + 3]),
                          pack_f16(s[8 * m + 4], s[8 * m + 5]), pack_f16(s[8 * m + 6], s[8 * m + 7]));
  }
  __device__ void gemm2(const uint4 (&sop)[KP], f32x4_t (&u)[JT]) const {
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      u[jt] = b1acc[jt];
#pragma unroll
      for (int m = 0; m < KP; ++m) u[jt] = mfma_f16(w1op[jt][m], sop[m], u[jt]);
    }
  }
  __device__ static void silu(const f32x4_t (&u)[JT], uint4 (&hop)[KH]) {
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      float hv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = u[2 * m + (e >> 2)][e & 3];
        hv[e] = x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x));
      }
      hop[m] = make_uint4(pack_f16(hv[0], hv[1]), pack_f16(hv[2], hv[3]), pack_f16(hv[4], hv[5]),
                          pack_f16(hv[6], hv[7]));
    }
  }
  __device__ void gemm3(const uint4 (&hop)[KH], const f32x4_t (&c0)[PT], f32x4_t (&lg)[PT]) const {
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      lg[pt] = c0[pt];
#pragma unroll
      for (int m = 0; m < KH; ++m) lg[pt] = mfma_f16(w2op[pt][m], hop[m], lg[pt]);
    }
  }

  // Base-2 gating logits l' of one query for the lane's items (GEMM2 ->
  // SiLU -> GEMM3), each matrix chain issued at raised wave priority.
  __device__ void logits(const float (&s)[RUN], const f32x4_t (&c0)[PT], f32x4_t (&lg)[PT]) const {
    if constexpr (X2) {
      logits_x2(s, c0, lg);
      return;
    }
    uint4 sop[KP];
    pack_s(s, sop);
    f32x4_t u[JT];
    mfma_priority_begin();
    gemm2(sop, u);
    mfma_priority_end();
    uint4 hop[KH];
    silu(u, hop);
    mfma_priority_begin();
    gemm3(hop, c0, lg);
    mfma_priority_end();
  }

  // The two-term chain: x = -log2(e) s and h' = u' / (1 + 2^u') as hi + lo
  // bf16 pairs; each K block of GEMM2 and GEMM3 takes the hi and the lo
  // operand against the same exact weights.
  __device__ void logits_x2(const float (&s)[RUN], const f32x4_t (&c0)[PT], f32x4_t (&lg)[PT]) const {
    uint4 shi[KP], slo[KP];
#pragma unroll
    for (int m = 0; m < KP; ++m) {
      uint32_t h[4], l[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2)
        split_bf16(-kLog2e * s[8 * m + 2 * e2], -kLog2e * s[8 * m + 2 * e2 + 1], h[e2], l[e2]);
      shi[m] = make_uint4(h[0], h[1], h[2], h[3]);
      slo[m] = make_uint4(l[0], l[1], l[2], l[3]);
    }
    f32x4_t u[JT];
    mfma_priority_begin();
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      u[jt] = b1acc[jt];
#pragma unroll
      for (int m = 0; m < KP; ++m) {
        u[jt] = mfma_bf16(w1op[jt][m], shi[m], u[jt]);
        u[jt] = mfma_bf16(w1op[jt][m], slo[m], u[jt]);
      }
    }
    mfma_priority_end();
    uint4 hhi[KH], hlo[KH];
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      float hv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = u[2 * m + (e >> 2)][e & 3];
        hv[e] = x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x));
      }
      uint32_t h[4], l[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) split_bf16(hv[2 * e2], hv[2 * e2 + 1], h[e2], l[e2]);
      hhi[m] = make_uint4(h[0], h[1], h[2], h[3]);
      hlo[m] = make_uint4(l[0], l[1], l[2], l[3]);
    }
    mfma_priority_begin();
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      lg[pt] = c0[pt];
#pragma unroll
      for (int m = 0; m < KH; ++m) {
        lg[pt] = mfma_bf16(w2op[pt][m], hhi[m], lg[pt]);
        lg[pt] = mfma_bf16(w2op[pt][m], hlo[m], lg[pt]);
      }
    }
    mfma_priority_end();
  }

  // sum_p w_p and sum_p w_p s_p over the lane's p (w = 2^(l' - shift)),
  // two partial sums each to shorten the dependency chains
  __device__ static void weights(const f32x4_t (&lg)[PT], const float (&s)[RUN], float shift, float& den,
                                 float& num) {
    float d[2], n[2];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float w = __builtin_amdgcn_exp2f(lg[pt][i] - shift);
        if (pt == 0 && i < 2) {   // first term of each partial sum
          d[i] = w;
          n[i] = w * s[i];
        } else {
          d[i & 1] += w;
          n[i & 1] = fmaf(w, s[4 * pt + i], n[i & 1]);
        }
      }
    den = d[0] + d[1];
    num = n[0] + n[1];
  }

  // phi of two queries (out[q] valid in the lanes of rows 2q, 2q + 1), with
  // the two chains software-pipelined in one scheduling region: query 1's
  // GEMM2 issues between query 0's SiLU instructions, query 0's GEMM3
  // between query 1's, and query 1's GEMM3 between query 0's softmax terms,
  // so that each wave keeps its matrix core busy under its own vector ALU
  // work.  VA is the number of vector ALU instructions placed after each
  // matrix instruction.  The arithmetic is that of phi<2> (the same
  // instructions on the same operands), so the results are bit-identical;
  // a query whose sum left [2^-60, 2^60] is redone by phi<2>.
  template <int VA>
  __device__ void phi2_interleaved(const float (&s)[2][RUN], const f32x4_t (&c0)[2][PT], float (&out)[2]) const {
    static_assert(!X2, "the interleaved chain is the f16 form");
    uint4 sop[2][KP];
    f32x4_t u[2][JT];
    uint4 hop[2][KH];
    f32x4_t lg[2][PT];
    float den[2], num[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      pack_s(s[q], sop[q]);
      gemm2(sop[q], u[q]);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) silu(u[q], hop[q]);
#pragma unroll
    for (int q = 0; q < 2; ++q) gemm3(hop[q], c0[q], lg[q]);
#pragma unroll
    for (int q = 0; q < 2; ++q) weights(lg[q], s[q], 0.f, den[q], num[q]);
    // issue order: query 0's GEMM2 (JT KP matrix instructions), then the
    // three interleaved runs of JT KP, PT KH and PT KH matrix instructions,
    // each followed by VA vector ALU (transcendentals included) instructions
    constexpr int kMfma = 0x008, kValu = 0x002 | 0x400;
    __builtin_amdgcn_sched_group_barrier(kMfma, JT * KP, 0);
#pragma unroll
    for (int i = 0; i < JT * KP + 2 * PT * KH; ++i) {
      __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kValu, VA, 0);
    }
    float D, Nm;
    row_sums(den[0], num[0], den[1], num[1], D, Nm);
    const bool ok = D >= 0x1p-60f && D <= 0x1p60f;
    if (!__all(ok)) {
      phi<2>(s, c0, out);
      return;
    }
    const float v = Nm * __builtin_amdgcn_rcpf(D);
    out[0] = v;
    out[1] = v;
  }

  // The two-query chain split for a software-pipelined scan (the same
  // instructions on the same operands as phi2_interleaved and phi<2>, so the
  // sums are bit-identical).  Stage A: both queries' GEMM2 -> SiLU -> GEMM3
  // and query 0's softmax sums, scheduled as in phi2_interleaved for
  // H <= 64 and as two priority-raised chains (logits) for larger H, where
  // the matrix chains are long against the SiLU work; query 1's base-2
  // logits are handed to stage B, which the caller issues together with the
  // next step's GEMM1.
  template <int VA, int NDS = 0>
  __device__ void phi2_stage_a(const float (&s)[2][RUN], const f32x4_t (&c0)[2][PT], f32x4_t (&lg1)[PT],
                               float& den0, float& num0) const {
    static_assert(!X2, "the pipelined chain is the f16 form");
    if constexpr (H > 64) {
      f32x4_t lg0[PT];
      logits(s[0], c0[0], lg0);
      logits(s[1], c0[1], lg1);
      weights(lg0, s[0], 0.f, den0, num0);
      // query 1's logits are read after the caller's next branch
      mfma_drain();
      return;
    }
    uint4 sop[2][KP];
    f32x4_t u[2][JT];
    uint4 hop[2][KH];
    f32x4_t lg0[PT];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      pack_s(s[q], sop[q]);
      gemm2(sop[q], u[q]);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) silu(u[q], hop[q]);
    gemm3(hop[0], c0[0], lg0);
    gemm3(hop[1], c0[1], lg1);
    weights(lg0, s[0], 0.f, den0, num0);
    constexpr int kMfma = 0x008, kValu = 0x002 | 0x400, kDsRead = 0x100;
    // the caller's NDS LDS reads (the GEMM3 accumulator inputs) go first, so
    // that GEMM2 and the SiLU cover their latency
    if constexpr (NDS > 0) __builtin_amdgcn_sched_group_barrier(kDsRead, NDS, 0);
    __builtin_amdgcn_sched_group_barrier(kMfma, JT * KP, 0);
#pragma unroll
    for (int i = 0; i < JT * KP + 2 * PT * KH; ++i) {
      __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kValu, VA, 0);
    }
    // query 1's logits are read after the caller's next branch
    mfma_drain();
  }
  // Stage B: query 1's softmax sums and the sums over an item's four lanes
  // (D and Nm in the layout of row_sums).
  __device__ static void phi2_stage_b(const f32x4_t (&lg1)[PT], const float (&s1)[RUN], float den0, float num0,
                                      float& D, float& Nm) {
    float den1, num1;
    weights(lg1, s1, 0.f, den1, num1);
    row_sums(den0, num0, den1, num1, D, Nm);
  }

  // phi for the lane's item under NQ (1 or 2) queries: out[q] is valid in
  // the lanes of query q's rows (NQ = 2: rows 0-1 for query 0, rows 2-3 for
  // query 1; NQ = 1: every lane).  The queries' chains are independent and
  // branch-free, so they can be interleaved; a query whose max-free sum left
  // [2^-60, 2^60] (logits far from zero) is redone with the row maximum
  // subtracted.  c0[q]: log2(e) (a_x + a_q + b2) of query q in the GEMM3
  // accumulator layout.
  template <int NQ>
  __device__ void phi(const float (&s)[NQ][RUN], const f32x4_t (&c0)[NQ][PT], float (&out)[NQ]) const {
    static_assert(NQ == 1 || NQ == 2, "one or two queries per call");
    float den[NQ], num[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      f32x4_t lg[PT];
      logits(s[q], c0[q], lg);
      weights(lg, s[q], 0.f, den[q], num[q]);
    }
    float D, Nm;
    row_sums(den[0], num[0], den[NQ - 1], num[NQ - 1], D, Nm);
    const bool ok = D >= 0x1p-60f && D <= 0x1p60f;
    if (!__all(ok)) {
      const uint64_t okm = __ballot(ok);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const uint64_t rows = NQ == 1 ? ~0ull : q == 0 ? 0x00000000FFFFFFFFull : 0xFFFFFFFF00000000ull;
        if ((okm & rows) == rows) continue;
        f32x4_t lg[PT];
        logits(s[q], c0[q], lg);
        float mx = -__builtin_inff();
#pragma unroll
        for (int pt = 0; pt < PT; ++pt)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, lg[pt][i]);
        weights(lg, s[q], max_groups(mx), den[q], num[q]);
      }
      row_sums(den[0], num[0], den[NQ - 1], num[NQ - 1], D, Nm);
    }
    const float v = Nm * __builtin_amdgcn_rcpf(D);
#pragma unroll
    for (int q = 0; q < NQ; ++q) out[q] = v;
  }
};


// The gating chain for P <= 16 components: GEMM2 on 16x16x16 f16 MFMAs
// (K = 16 = P'), so lane (c, g) holds item c's components p = 4 g + e,
// e < 4, and GEMM3 has one output tile whose row 4 g + i is p = 4 g + i:
// no padding of P to 32.  Same interface as MolMlp (pr.P <= 16, pr.H <= H).
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
template <int H, bool X2 = false>
struct MolMlp16 {   // X2: the two-term chain, as in MolMlp
  static constexpr int P = 16;
  static constexpr int RUN = 4;
  static constexpr int JT = H / 16;   // output tiles of GEMM2
  static constexpr int KH = H / 32;   // K blocks of GEMM3
  static constexpr int PT = 1;        // output tiles of GEMM3
  uint2 w1op[JT];
  uint4 w2op[KH];
  f32x4_t b1acc[JT];
  __device__ static int base(int g) { return 4 * g; }

  __device__ void load_padded(const DevProb& pr, int c, int g) {
    const bf16_t* W1 = static_cast<const bf16_t*>(pr.W1);
    const bf16_t* W2 = static_cast<const bf16_t*>(pr.W2);
    const int Pr = pr.P, Hr = pr.H;
    // unconditional reads from clamped indices, masked afterwards
    auto w1 = [&](int j, int p) -> uint32_t {
      const bf16_t w = W1[min(j, Hr - 1) * Pr + min(p, Pr - 1)];
      const uint32_t keep = 0u - static_cast<uint32_t>((j < Hr) & (p < Pr));
      return (X2 ? static_cast<uint32_t>(w) : neg_bf16_to_f16_bits(w, kLog2e)) & keep;
    };
    auto w2 = [&](int p, int j) -> uint32_t {
      const bf16_t w = W2[min(p, Pr - 1) * Hr + min(j, Hr - 1)];
      const uint32_t keep = 0u - static_cast<uint32_t>((j < Hr) & (p < Pr));
      return (X2 ? static_cast<uint32_t>(w ^ 0x8000u) : neg_bf16_to_f16_bits(w, 1.f)) & keep;
    };
    // W1' = -log2(e) W1: row j = 16 jt + c, K slot 4 g + e <-> p = 4 g + e
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      const int j = 16 * jt + c;
      w1op[jt] = make_uint2(w1(j, 4 * g) | (w1(j, 4 * g + 1) << 16), w1(j, 4 * g + 2) | (w1(j, 4 * g + 3) << 16));
    }
    // -W2: row c <-> p = c; K slot 8 g + e of block m <-> j as in MolMlp
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      uint32_t w[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int e0 = 2 * e2, e1 = 2 * e2 + 1;
        const int j0 = 32 * m + 16 * (e0 >> 2) + 4 * g + (e0 & 3);
        const int j1 = 32 * m + 16 * (e1 >> 2) + 4 * g + (e1 & 3);
        w[e2] = w2(c, j0) | (w2(c, j1) << 16);
      }
      w2op[m] = make_uint4(w[0], w[1], w[2], w[3]);
    }
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * jt + 4 * g + i;
        const float b = pr.b1[min(j, Hr - 1)];
        b1acc[jt][i] = j < Hr ? -kLog2e * b : 0.f;
      }
  }

  __device__ void logits(const float (&s)[RUN], const f32x4_t (&c0)[PT], f32x4_t (&lg)[PT]) const {
    if constexpr (X2) {
      logits_x2(s, c0, lg);
      return;
    }
    const uint2 sop = make_uint2(pack_f16(s[0], s[1]), pack_f16(s[2], s[3]));
    f32x4_t u[JT];
    mfma_priority_begin();
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
      u[jt] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, w1op[jt]),
                                                    __builtin_bit_cast(f16x4_t, sop), b1acc[jt], 0, 0, 0);
    mfma_priority_end();
    uint4 hop[KH];
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      float hv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = u[2 * m + (e >> 2)][e & 3];
        hv[e] = x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x));
      }
      hop[m] = make_uint4(pack_f16(hv[0], hv[1]), pack_f16(hv[2], hv[3]), pack_f16(hv[4], hv[5]),
                          pack_f16(hv[6], hv[7]));
    }
    mfma_priority_begin();
    lg[0] = c0[0];
#pragma unroll
    for (int m = 0; m < KH; ++m) lg[0] = mfma_f16(w2op[m], hop[m], lg[0]);
    mfma_priority_end();
  }

  // The two-term chain (see MolMlp::logits_x2): GEMM2 on 16x16x16 bf16 MFMAs
  // with the hi and the lo operand of -log2(e) s, GEMM3 with those of h'.
  __device__ void logits_x2(const float (&s)[RUN], const f32x4_t (&c0)[PT], f32x4_t (&lg)[PT]) const {
    uint32_t s01h, s01l, s23h, s23l;
    split_bf16(-kLog2e * s[0], -kLog2e * s[1], s01h, s01l);
    split_bf16(-kLog2e * s[2], -kLog2e * s[3], s23h, s23l);
    const uint2 shi = make_uint2(s01h, s23h), slo = make_uint2(s01l, s23l);
    f32x4_t u[JT];
    mfma_priority_begin();
#pragma unroll
    for (int jt = 0; jt < JT; ++jt) {
      u[jt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4_t, w1op[jt]),
                                                       __builtin_bit_cast(bf16x4_t, shi), b1acc[jt], 0, 0, 0);
      u[jt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4_t, w1op[jt]),
                                                       __builtin_bit_cast(bf16x4_t, slo), u[jt], 0, 0, 0);
    }
    mfma_priority_end();
    uint4 hhi[KH], hlo[KH];
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      float hv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = u[2 * m + (e >> 2)][e & 3];
        hv[e] = x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x));
      }
      uint32_t h[4], l[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) split_bf16(hv[2 * e2], hv[2 * e2 + 1], h[e2], l[e2]);
      hhi[m] = make_uint4(h[0], h[1], h[2], h[3]);
      hlo[m] = make_uint4(l[0], l[1], l[2], l[3]);
    }
    mfma_priority_begin();
    lg[0] = c0[0];
#pragma unroll
    for (int m = 0; m < KH; ++m) {
      lg[0] = mfma_bf16(w2op[m], hhi[m], lg[0]);
      lg[0] = mfma_bf16(w2op[m], hlo[m], lg[0]);
    }
    mfma_priority_end();
  }

  __device__ static void weights(const f32x4_t (&lg)[PT], const float (&s)[RUN], float shift, float& den,
                                 float& num) {
    float d[2], n[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float w = __builtin_amdgcn_exp2f(lg[0][i] - shift);
      if (i < 2) {
        d[i] = w;
        n[i] = w * s[i];
      } else {
        d[i & 1] += w;
        n[i & 1] = fmaf(w, s[i], n[i & 1]);
      }
    }
    den = d[0] + d[1];
    num = n[0] + n[1];
  }

  template <int NQ>
  __device__ void phi(const float (&s)[NQ][RUN], const f32x4_t (&c0)[NQ][PT], float (&out)[NQ]) const {
    static_assert(NQ == 1 || NQ == 2, "one or two queries per call");
    float den[NQ], num[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      f32x4_t lg[PT];
      logits(s[q], c0[q], lg);
      weights(lg, s[q], 0.f, den[q], num[q]);
    }
    float D, Nm;
    row_sums(den[0], num[0], den[NQ - 1], num[NQ - 1], D, Nm);
    const bool ok = D >= 0x1p-60f && D <= 0x1p60f;
    if (!__all(ok)) {
      const uint64_t okm = __ballot(ok);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const uint64_t rows = NQ == 1 ? ~0ull : q == 0 ? 0x00000000FFFFFFFFull : 0xFFFFFFFF00000000ull;
        if ((okm & rows) == rows) continue;
        f32x4_t lg[PT];
        logits(s[q], c0[q], lg);
        float mx = fmaxf(fmaxf(lg[0][0], lg[0][1]), fmaxf(lg[0][2], lg[0][3]));
        weights(lg, s[q], max_groups(mx), den[q], num[q]);
      }
      row_sums(den[0], num[0], den[NQ - 1], num[NQ - 1], D, Nm);
    }
    const float v = Nm * __builtin_amdgcn_rcpf(D);
#pragma unroll
    for (int q = 0; q < NQ; ++q) out[q] = v;
  }
};

}  // namespace tile
}  // namespace mol
