// Fused MoL scoring on gfx950 matrix cores (bf16 embeddings, P_q = 8).
//
// One wave scores 2 queries against 16 items per step through three chained
// 16x16x32 MFMA products whose register layouts line up, so no accumulator
// is re-laid-out through LDS (lane l: item column c = l % 16, group
// g = l / 16):
//
//   GEMM1 (bf16)  S[(q,pq)][item] = Q[q][pq] . X[px][item], one per px.
//                 Rows 8 q + pq: a lane of group g holds query g/2, pq in
//                 {4(g%2) .. 4(g%2)+3}, all px.  One permlane32 swap per
//                 register pair then gives each query's 64 p values to all
//                 64 lanes: lane (c, g) holds the contiguous run
//                 p = base(g) + mu, mu < 2 Px, base(g) = (4(g%2) + 2(g/2)) Px.
//   GEMM2 (f16)   U^T[j][item] = W1'[j][:] . s[:, item] + b1'[j]; the run
//                 above is the B operand (K slot 8g + e <-> p = base(g)+8m+e).
//   SiLU          h'_j = u'_j / (1 + 2^{u'_j}),  u' = -log2(e) u.
//   GEMM3 (f16)   l'^T[p][item] = -W2[p][:] . h'[:, item]
//                                 + log2(e) (a_x[item][p] + a_q[q][p] + b2[p]);
//                 GEMM2's accumulators are the B operand up to a fixed
//                 permutation of K (folded into the staged W2), and W2's
//                 rows are ordered so each lane's logits are the p values
//                 of its own s run.  a_x is the accumulator input; a_q + b2
//                 enters as one extra K block split into f16 hi + lo.
//   softmax, phi  w_p = 2^{l'_p}, phi = sum w_p s_p / sum w_p, s in f32,
//                 summed over the 4 lanes of an item with two xor shuffles.
//
// (Eq. 1 / Eq. 2 of the paper with the two-layer SiLU gating MLP of its
// Appendix A.3.)  Epilogues: a running per-query top-k (Definition 1) kept
// in LDS with threshold rejection, or a dense phi store.
//
// Workgroup: 8 waves (2 per SIMD) = 16 queries sharing an LDS-staged,
// double-buffered stream of 32-item tiles loaded with direct global->LDS
// copies.
#include "mol_kernels.h"

namespace mol {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kTopkList = 128;   // list capacity per query (k <= 128)
constexpr int kTopkStage = 128;  // staging slots per query
constexpr int kWaves = 8;
constexpr int kQueriesPerWG = 2 * kWaves;
constexpr int kTile = 32;        // items per LDS stage (two 16-item steps)

__device__ __forceinline__ f32x4_t mfma_bf16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_f16(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(a))) |
         (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(b))) << 16);
}
__device__ __forceinline__ uint32_t neg_bf16_to_f16_bits(bf16_t w, float scale) {
  // f16 bits of -scale * w (sign flipped on the integer side)
  const float v = scale * to_f32(static_cast<bf16_t>(w ^ 0x8000u));
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(v)));
}

// Sum of x over the 4 lanes {c, c+16, c+32, c+48} (the 4 groups holding one
// item), returned in all of them; VALU lane permutes only.
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

// LDS fence for exchanges between lanes of one wave.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Bitonic sort (descending) of 256 keys held in LDS by one wave.
__device__ __noinline__ void wave_sort256(uint64_t* r, int lane) {
  for (int size = 2; size <= 256; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
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

template <int PX, int D, int H>
struct FusedShape {
  static constexpr int PQ = 8;
  static constexpr int P = PQ * PX;
  static constexpr int RUN = 2 * PX;     // s values per lane per query
  static constexpr int KD = D / 32;      // K blocks of GEMM1
  static constexpr int KP = P / 32;      // K blocks of GEMM2
  static constexpr int JT = H / 16;      // output tiles of GEMM2
  static constexpr int KH = H / 32;      // K blocks of GEMM3
  static constexpr int PT = P / 16;      // output tiles of GEMM3
  static constexpr int XROWCH = D / 8;   // 16-byte chunks per X row
  static constexpr int AROWCH = P / 4;   // 16-byte chunks per a_x row
  static constexpr int XSTAGE = PX * kTile * D * 2;   // bytes of one X stage
  static constexpr int ASTAGE = kTile * P * 4;        // bytes of one a_x stage
  static constexpr int LDS_X = 2 * XSTAGE;
  static constexpr int LDS_AX = 2 * ASTAGE;
  static constexpr int LDS_CB = kQueriesPerWG * P * 4;
  static constexpr int LDS_TOPK = kQueriesPerWG * (kTopkList + kTopkStage) * 8;
  static constexpr int LDS_TOTAL = LDS_X + LDS_AX + LDS_CB + LDS_TOPK;
  // 16-byte global->LDS copies per stage, in 1 KB blocks of one wave each
  static constexpr int XBLOCKS = XSTAGE / 1024;
  static constexpr int ABLOCKS = ASTAGE / 1024;
  static_assert(XBLOCKS % kWaves == 0, "X stage must split evenly over the waves");
};

__device__ __forceinline__ int lane_base(int g, int PX) { return (4 * (g & 1) + 2 * (g >> 1)) * PX; }

// WG -> (item range, query group); WGs on one XCD (WG id mod 8) share item
// ranges so that the corpus streams through each XCD's L2 once.
__device__ __forceinline__ void wg_coords(int g, int R, int G, int& r, int& qg) {
  if (R <= 8 && (8 % R) == 0 && ((R * G) % 8) == 0) {
    const int x = g & 7, i = g >> 3;
    r = x % R;
    qg = (x / R) * (R * G / 8) + i;
  } else {
    r = g % R;
    qg = g / R;
  }
}

template <int PX, int D, int H, bool DENSE>
__global__ __launch_bounds__(64 * kWaves, 1) void k_mol_fused(
    DevProb pr, int k, int R, int range_len, int G, int n_begin, int n_end,
    uint64_t* __restrict__ partial, float* __restrict__ phi_out, long phi_stride) {
  using S = FusedShape<PX, D, H>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  unsigned char* sAx = smem + S::LDS_X;
  uint32_t* sCb = reinterpret_cast<uint32_t*>(smem + S::LDS_X + S::LDS_AX);
  uint64_t* sTop = reinterpret_cast<uint64_t*>(smem + S::LDS_X + S::LDS_AX + S::LDS_CB);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 15, g = lane >> 4;
  const int base = lane_base(g, PX);
  int r, qg;
  wg_coords(blockIdx.x, R, G, r, qg);
  const int qwg = qg * kQueriesPerWG;     // first query of the workgroup
  const int qwv = qwg + 2 * wave;         // first of this wave's 2 queries
  const int nr0 = n_begin + r * range_len;
  const int nr1 = min(n_end, nr0 + range_len);
  const int ntiles = nr1 > nr0 ? (nr1 - nr0 + kTile - 1) / kTile : 0;
  const int N = pr.N;
  constexpr int P = S::P;

  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);
  const bf16_t* W1 = static_cast<const bf16_t*>(pr.W1);
  const bf16_t* W2 = static_cast<const bf16_t*>(pr.W2);

  // ---- stage tile t into LDS buffer buf with direct global->LDS copies ----
  // X stage layout [px][item][16-byte chunk ^ (item % XROWCH)], a_x stage
  // [item][16-byte chunk ^ (item % AROWCH)].  Lane i of a copy writes LDS
  // bytes 16 i of its 1 KB block, so the global side picks the chunk that
  // belongs there.  Items past the end are clamped to N-1 (valid memory,
  // masked later).
  auto stage = [&](int t, int buf) {
    const int n0 = nr0 + kTile * t;
#pragma unroll
    for (int cp = 0; cp < S::XBLOCKS / kWaves; ++cp) {
      const int blk = wave + kWaves * cp;
      const int pos = blk * 64 + lane;
      const int px = pos / (kTile * S::XROWCH);
      const int rem = pos % (kTile * S::XROWCH);
      const int n = rem / S::XROWCH, phys = rem % S::XROWCH;
      const int cc = phys ^ (n % S::XROWCH);
      const int item = min(n0 + n, N - 1);
      const bf16_t* src = X + (static_cast<long>(px) * N + item) * D + 8 * cc;
      unsigned char* dst = sX + buf * S::XSTAGE + blk * 1024;
      __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)dst, 16, 0, 0);
    }
    for (int blk = wave; blk < S::ABLOCKS; blk += kWaves) {
      const int pos = blk * 64 + lane;
      const int n = pos / S::AROWCH, phys = pos % S::AROWCH;
      const int cc = phys ^ (n % S::AROWCH);
      const int item = min(n0 + n, N - 1);
      const float* src = pr.a_x + static_cast<long>(item) * P + 4 * cc;
      unsigned char* dst = sAx + buf * S::ASTAGE + blk * 1024;
      __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)dst, 16, 0, 0);
    }
  };
  if (ntiles > 0) stage(0, 0);

  // ---- per-workgroup constants ----
  for (int i = tid; i < kQueriesPerWG * P; i += 64 * kWaves) {
    const int qi = i / P, p = i % P, b = qwg + qi;
    const float v = b < pr.B ? kLog2e * (pr.a_q[static_cast<long>(b) * P + p] + pr.b2[p]) : 0.f;
    const float hi = static_cast<float>(static_cast<_Float16>(v));
    sCb[i] = pack_f16(hi, v - hi);
  }
  uint64_t* myTop = sTop + wave * 2 * (kTopkList + kTopkStage);
  if (!DENSE)
    for (int i = lane; i < 2 * (kTopkList + kTopkStage); i += 64) myTop[i] = 0ull;

  // W1' = -log2(e) W1 as GEMM2 A operands: row j, K slot 8g+e <-> p = base(g)+8m+e
  uint4 w1op[S::JT][S::KP];
#pragma unroll
  for (int jt = 0; jt < S::JT; ++jt)
#pragma unroll
    for (int m = 0; m < S::KP; ++m) {
      const bf16_t* src = W1 + (16 * jt + c) * P + base + 8 * m;
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = neg_bf16_to_f16_bits(src[2 * e], kLog2e) |
               (neg_bf16_to_f16_bits(src[2 * e + 1], kLog2e) << 16);
      w1op[jt][m] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  // -W2 as GEMM3 A operands: row rho = 16 pt + c <-> p = base(c/4) + 4 pt + c%4;
  // K slot 8g+e <-> j = 32 m + 16 (e/4) + 4 g + e%4
  uint4 w2op[S::PT][S::KH];
#pragma unroll
  for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
    for (int m = 0; m < S::KH; ++m) {
      const int p = lane_base(c >> 2, PX) + 4 * pt + (c & 3);
      uint32_t w[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int e0 = 2 * e2, e1 = 2 * e2 + 1;
        const int j0 = 32 * m + 16 * (e0 >> 2) + 4 * g + (e0 & 3);
        const int j1 = 32 * m + 16 * (e1 >> 2) + 4 * g + (e1 & 3);
        w[e2] = neg_bf16_to_f16_bits(W2[p * H + j0], 1.f) |
                (neg_bf16_to_f16_bits(W2[p * H + j1], 1.f) << 16);
      }
      w2op[pt][m] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  // b1' in the GEMM2 accumulator layout (row j = 16 jt + 4 g + i)
  f32x4_t b1acc[S::JT];
#pragma unroll
  for (int jt = 0; jt < S::JT; ++jt)
#pragma unroll
    for (int i = 0; i < 4; ++i) b1acc[jt][i] = -kLog2e * pr.b1[16 * jt + 4 * g + i];
  // Q as GEMM1 A operands: row c = 8 q + pq, K slot 8g+e <-> d = 32 kk + 8 g + e
  uint4 qop[S::KD];
  {
    const int b = qwv + (c >> 3), pq = c & 7;
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk)
      qop[kk] = b < pr.B
                    ? *reinterpret_cast<const uint4*>(Q + (static_cast<long>(b) * 8 + pq) * D + 32 * kk + 8 * g)
                    : make_uint4(0, 0, 0, 0);
  }
  // constant B operand of the a_q + b2 K block: ones in K slots 0 and 1
  const uint4 ones = make_uint4(g == 0 ? 0x3C003C00u : 0u, 0u, 0u, 0u);

  // running top-k state of the wave's 2 queries (wave-uniform)
  uint64_t theta[2] = {0ull, 0ull};
  int stg[2] = {0, 0};
  auto merge = [&](int qb) {
    uint64_t* reg = myTop + qb * (kTopkList + kTopkStage);
    wave_lds_sync();
    wave_sort256(reg, lane);
    for (int i = kTopkList + lane; i < kTopkList + kTopkStage; i += 64) reg[i] = 0ull;
    wave_lds_sync();
    theta[qb] = reg[k - 1];
    stg[qb] = 0;
  };

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage(t + 1, buf ^ 1);
    const unsigned char* xs = sX + buf * S::XSTAGE;
    const unsigned char* as = sAx + buf * S::ASTAGE;

#pragma unroll
    for (int st = 0; st < kTile / 16; ++st) {
      const int n = 16 * st + c;            // item within the stage
      const int item = nr0 + kTile * t + n;
      const bool item_ok = item < nr1;

      // GEMM1: both queries x 16 items x all px
      f32x4_t acc1[PX];
#pragma unroll
      for (int px = 0; px < PX; ++px) {
        acc1[px] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const unsigned char* row = xs + (px * kTile + n) * (D * 2);
#pragma unroll
        for (int kk = 0; kk < S::KD; ++kk) {
          const int phys = (4 * kk + g) ^ (n % S::XROWCH);
          acc1[px] = mfma_bf16(qop[kk], *reinterpret_cast<const uint4*>(row + 16 * phys), acc1[px]);
        }
      }
      // separate the two queries: s0[mu], s1[mu] hold p = base(g) + mu
      float s0[S::RUN], s1[S::RUN];
#pragma unroll
      for (int mu = 0; mu < S::RUN; ++mu) {
        const float a = acc1[mu % PX][mu / PX];
        const float b = acc1[mu % PX][2 + mu / PX];
        auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
        s0[mu] = __uint_as_float(sw[0]);
        s1[mu] = __uint_as_float(sw[1]);
      }
      // a_x (scaled by log2 e) in the GEMM3 accumulator layout
      f32x4_t axr[S::PT];
#pragma unroll
      for (int q4 = 0; q4 < S::PT; ++q4) {
        const int phys = (base / 4 + q4) ^ (n % S::AROWCH);
        const float4 a = *reinterpret_cast<const float4*>(as + n * (P * 4) + 16 * phys);
        axr[q4] = f32x4_t{kLog2e * a.x, kLog2e * a.y, kLog2e * a.z, kLog2e * a.w};
      }

#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float s[S::RUN];
#pragma unroll
        for (int mu = 0; mu < S::RUN; ++mu) s[mu] = qb == 0 ? s0[mu] : s1[mu];
        // GEMM2
        uint4 sop[S::KP];
#pragma unroll
        for (int m = 0; m < S::KP; ++m)
          sop[m] = make_uint4(pack_f16(s[8 * m + 0], s[8 * m + 1]), pack_f16(s[8 * m + 2], s[8 * m + 3]),
                              pack_f16(s[8 * m + 4], s[8 * m + 5]), pack_f16(s[8 * m + 6], s[8 * m + 7]));
        f32x4_t u[S::JT];
#pragma unroll
        for (int jt = 0; jt < S::JT; ++jt) {
          u[jt] = b1acc[jt];
#pragma unroll
          for (int m = 0; m < S::KP; ++m) u[jt] = mfma_f16(w1op[jt][m], sop[m], u[jt]);
        }
        // SiLU, packed as GEMM3 B operands: K slot 8g+e of block m <-> (jt, i) = (2m + e/4, e%4)
        uint4 hop[S::KH];
#pragma unroll
        for (int m = 0; m < S::KH; ++m) {
          float hv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = u[2 * m + (e >> 2)][e & 3];
            hv[e] = x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x));
          }
          hop[m] = make_uint4(pack_f16(hv[0], hv[1]), pack_f16(hv[2], hv[3]), pack_f16(hv[4], hv[5]),
                              pack_f16(hv[6], hv[7]));
        }
        // GEMM3 with the a_q + b2 block
        f32x4_t lg[S::PT];
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt) {
          const int p = lane_base(c >> 2, PX) + 4 * pt + (c & 3);
          const uint32_t cb = g == 0 ? sCb[(2 * wave + qb) * P + p] : 0u;
          lg[pt] = mfma_f16(make_uint4(cb, 0u, 0u, 0u), ones, axr[pt]);
#pragma unroll
          for (int m = 0; m < S::KH; ++m) lg[pt] = mfma_f16(w2op[pt][m], hop[m], lg[pt]);
        }
        // softmax over p and phi
        float den = 0.f, num = 0.f;
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float w = __builtin_amdgcn_exp2f(lg[pt][i]);
            den += w;
            num = fmaf(w, s[4 * pt + i], num);
          }
        den = sum_groups(den);
        num = sum_groups(num);
        if (!__all(den >= 0x1p-60f && den <= 0x1p60f)) {
          // logits far from zero: subtract the row maximum first
          float mx = -__builtin_inff();
#pragma unroll
          for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, lg[pt][i]);
          mx = max_groups(mx);
          den = 0.f;
          num = 0.f;
#pragma unroll
          for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float w = __builtin_amdgcn_exp2f(lg[pt][i] - mx);
              den += w;
              num = fmaf(w, s[4 * pt + i], num);
            }
          den = sum_groups(den);
          num = sum_groups(num);
        }
        const float phi = num * __builtin_amdgcn_rcpf(den);
        const int b = qwv + qb;

        if constexpr (DENSE) {
          if (g == 0 && item_ok && b < pr.B) phi_out[b * phi_stride + (item - n_begin)] = phi;
        } else {
          const uint64_t key = (g == 0 && item_ok) ? make_key(phi, item) : 0ull;
          const bool pass = key > theta[qb];
          const uint64_t mask = __ballot(pass);
          if (mask) {
            uint64_t* reg = myTop + qb * (kTopkList + kTopkStage);
            const int below = __popcll(mask & ((1ull << lane) - 1ull));
            if (pass) reg[kTopkList + stg[qb] + below] = key;
            stg[qb] += __popcll(mask);
            if (stg[qb] > kTopkStage - 16) merge(qb);
          }
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  if constexpr (!DENSE) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      if (stg[qb] > 0) merge(qb);
      const int b = qwv + qb;
      if (b < pr.B) {
        const uint64_t* reg = myTop + qb * (kTopkList + kTopkStage);
        uint64_t* dst = partial + (static_cast<long>(b) * R + r) * k;
        for (int i = lane; i < k; i += 64) dst[i] = reg[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
bool fused_supported(const DevProb& pr, int k) {
  if (pr.dtype != MOL_BF16 || pr.Pq != 8) return false;
  if (!((pr.Px == 4 && pr.d == 128 && pr.H == 128) || (pr.Px == 4 && pr.d == 64 && pr.H == 64) ||
        (pr.Px == 8 && pr.d == 64 && pr.H == 64)))
    return false;
  return k <= kTopkList;
}

void fused_grid(const DevProb& pr, int n_count, int& R, int& range_len, int& G) {
  G = (pr.B + kQueriesPerWG - 1) / kQueriesPerWG;
  R = std::max(1, 256 / G);
  const int max_r = std::max(1, n_count / 512);
  R = std::min(R, max_r);
  range_len = (n_count + R - 1) / R;
  range_len = (range_len + kTile - 1) / kTile * kTile;
  R = (n_count + range_len - 1) / range_len;
}

template <int PX, int D, int H, bool DENSE>
static hipError_t launch_fused_t(const DevProb& pr, int k, int R, int range_len, int G, int n_begin,
                                 int n_end, uint64_t* partial, float* phi, long phi_stride,
                                 hipStream_t st) {
  using S = FusedShape<PX, D, H>;
  auto kern = &k_mol_fused<PX, D, H, DENSE>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS_TOTAL);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(R * G), dim3(64 * kWaves), S::LDS_TOTAL, st, pr, k, R, range_len,
                     G, n_begin, n_end, partial, phi, phi_stride);
  return hipGetLastError();
}

template <bool DENSE>
static hipError_t launch_fused_d(const DevProb& pr, int k, int R, int range_len, int G, int n_begin,
                                 int n_end, uint64_t* partial, float* phi, long phi_stride,
                                 hipStream_t st) {
  if (pr.Px == 8)
    return launch_fused_t<8, 64, 64, DENSE>(pr, k, R, range_len, G, n_begin, n_end, partial, phi, phi_stride, st);
  if (pr.d == 128)
    return launch_fused_t<4, 128, 128, DENSE>(pr, k, R, range_len, G, n_begin, n_end, partial, phi, phi_stride, st);
  return launch_fused_t<4, 64, 64, DENSE>(pr, k, R, range_len, G, n_begin, n_end, partial, phi, phi_stride, st);
}

hipError_t launch_fused_topk(const DevProb& pr, int k, int R, int range_len, int G,
                             uint64_t* partial, hipStream_t st) {
  return launch_fused_d<false>(pr, k, R, range_len, G, 0, pr.N, partial, nullptr, 0, st);
}

hipError_t launch_fused_dense(const DevProb& pr, int n_begin, int n_count, float* phi,
                              hipStream_t st) {
  int R, range_len, G;
  fused_grid(pr, n_count, R, range_len, G);
  return launch_fused_d<true>(pr, 1, R, range_len, G, n_begin, n_begin + n_count, nullptr, phi,
                              n_count, st);
}

}  // namespace mol
