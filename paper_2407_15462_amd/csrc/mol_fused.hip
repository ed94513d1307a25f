// Fused MoL scoring on gfx950 matrix cores (bf16 embeddings, P_q = 8).
//
// One wave scores 4 queries against a tile of 32 items per step, through
// three chained 32x32x16 MFMA products whose layouts line up so that no
// accumulator ever has to be re-laid-out through LDS:
//
//   GEMM1 (bf16):  S[(b,pq)][item] = Q[b][pq] . X[px][item]      one per px
//                  rows (b_local, pq) = 32, columns = 32 items.  A lane
//                  (item c = lane%32, half h = lane/32) ends up holding, for
//                  each of its 4 queries, s_p for pq in {4h..4h+3} and all px,
//                  i.e. p = 4 Px h + lambda, lambda = i Px + px in [0, 4 Px).
//   GEMM2 (f16):   U^T[j][item] = W1'[j][:] . s[:, item] + b1'[j]
//                  the s values above are exactly a B operand (column = item,
//                  K slot 8h+e <-> p = 4 Px h + 8m + e), so s only needs an
//                  f32 -> f16 conversion in registers.
//   SiLU:          h'_j = u'_j / (1 + 2^{u'_j})   (u' = -log2(e) u)
//   GEMM3 (f16):   l'^T[p][item] = -W2[p][:] . h'[:, item] + log2(e) (a_x + a_q + b2)
//                  the accumulator rows of GEMM2 are again a B operand up to a
//                  fixed permutation of the K index, which is folded into the
//                  staged W2; the output rows are ordered so that a lane's
//                  logits line up with the s values it already holds.
//   softmax, phi:  w_p = 2^{l'_p};  phi = sum_p w_p s_p / sum_p w_p  (s in f32)
//
// (Eq. 1 / Eq. 2 of the paper with the two-layer SiLU gating MLP of its
// Appendix A.3.)  The per-query logit a_q[b] + b2 enters GEMM3 through one
// extra K block holding it split into two f16 halves (hi + lo), so the
// per-item logit a_x can be the MFMA accumulator input.
//
// Epilogues: a running per-query top-k (Definition 1) kept by each wave in
// LDS with threshold rejection, or a dense phi store.
#include "mol_kernels.h"

namespace mol {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kTopkList = 128;   // list capacity per query (k <= 128)
constexpr int kTopkStage = 128;  // staging slots per query

__device__ __forceinline__ f32x16_t mfma_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma_f16(f16x8_t a, f16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// LDS fence for exchanges between lanes of one wave.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Bitonic sort (descending) of 256 keys held in LDS by one wave.
__device__ __forceinline__ void wave_sort256(uint64_t* r, int lane) {
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
  static constexpr int KD = D / 16;    // K blocks of GEMM1
  static constexpr int KP = P / 16;    // K blocks of GEMM2
  static constexpr int JT = H / 32;    // output tiles of GEMM2
  static constexpr int KH = H / 16;    // K blocks of GEMM3
  static constexpr int PT = P / 32;    // output tiles of GEMM3
  static constexpr int XCH = PX * D / 64;      // 16-byte X chunks per thread per tile
  static constexpr int ACH = P / 32;           // 16-byte a_x chunks per thread per tile
  static constexpr int XROWCH = D / 8;         // 16-byte chunks per X row
  static constexpr int AROWCH = P / 4;         // 16-byte chunks per a_x row
  static constexpr int LDS_X = 2 * PX * 32 * D * 2;
  static constexpr int LDS_AX = 2 * 32 * P * 4;
  static constexpr int LDS_W1 = JT * KP * 64 * 16;
  static constexpr int LDS_W2 = PT * KH * 64 * 16;
  static constexpr int LDS_CB = 16 * P * 4;
  static constexpr int LDS_TOPK = 4 * 4 * (kTopkList + kTopkStage) * 8;
  static constexpr int LDS_TOTAL = LDS_X + LDS_AX + LDS_W1 + LDS_W2 + LDS_CB + LDS_TOPK;
};

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
__global__ __launch_bounds__(256, 1) void k_mol_fused(
    DevProb pr, int k, int R, int range_len, int G, int n_begin, int n_end,
    uint64_t* __restrict__ partial, float* __restrict__ phi_out, long phi_stride) {
  using S = FusedShape<PX, D, H>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  float* sAx = reinterpret_cast<float*>(smem + S::LDS_X);
  uint4* sW1 = reinterpret_cast<uint4*>(smem + S::LDS_X + S::LDS_AX);
  uint4* sW2 = sW1 + S::JT * S::KP * 64;
  uint32_t* sCb = reinterpret_cast<uint32_t*>(sW2 + S::PT * S::KH * 64);
  uint64_t* sTop = reinterpret_cast<uint64_t*>(sCb + 16 * S::P);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  int r, qg;
  wg_coords(blockIdx.x, R, G, r, qg);
  const int qwg = qg * 16;                 // first query of the workgroup
  const int qwv = qwg + wave * 4;          // first query of this wave
  const int nr0 = n_begin + r * range_len;
  const int nr1 = min(n_end, nr0 + range_len);
  const int ntiles = nr1 > nr0 ? (nr1 - nr0 + 31) / 32 : 0;
  const int N = pr.N, P = S::P;

  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);
  const bf16_t* W1 = static_cast<const bf16_t*>(pr.W1);
  const bf16_t* W2 = static_cast<const bf16_t*>(pr.W2);

  // ---- stage the gating MLP operands (f16, pre-scaled, pre-permuted) ----
  for (int i = tid; i < S::JT * S::KP * 64; i += 256) {
    const int ln = i & 63, m = (i >> 6) % S::KP, jt = (i >> 6) / S::KP;
    const int j = 32 * jt + (ln & 31), hl = ln >> 5;
    f16x8_t v;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      v[e] = static_cast<_Float16>(kLog2e * to_f32(static_cast<bf16_t>(W1[j * P + 4 * PX * hl + 8 * m + e] ^ 0x8000u)));
    sW1[i] = __builtin_bit_cast(uint4, v);
  }
  for (int i = tid; i < S::PT * S::KH * 64; i += 256) {
    const int ln = i & 63, m = (i >> 6) % S::KH, pt = (i >> 6) / S::KH;
    const int rr = ln & 31, hl = ln >> 5;
    const int p = 4 * PX * ((rr & 7) >> 2) + 16 * pt + 4 * (rr >> 3) + (rr & 3);
    f16x8_t v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = 32 * (m >> 1) + 8 * (2 * (m & 1) + (e >> 2)) + 4 * hl + (e & 3);
      v[e] = static_cast<_Float16>(to_f32(static_cast<bf16_t>(W2[p * H + j] ^ 0x8000u)));
    }
    sW2[i] = __builtin_bit_cast(uint4, v);
  }
  for (int i = tid; i < 16 * P; i += 256) {
    const int qi = i / P, p = i % P, b = qwg + qi;
    const float c = b < pr.B ? kLog2e * (pr.a_q[static_cast<long>(b) * P + p] + pr.b2[p]) : 0.f;
    const _Float16 hi = static_cast<_Float16>(c);
    const _Float16 lo = static_cast<_Float16>(c - static_cast<float>(hi));
    sCb[i] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, hi)) |
             (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, lo)) << 16);
  }
  uint64_t* myTop = sTop + wave * 4 * (kTopkList + kTopkStage);
  if (!DENSE)
    for (int i = lane; i < 4 * (kTopkList + kTopkStage); i += 64) myTop[i] = 0ull;

  // b1' in the GEMM2 accumulator layout
  f32x16_t b1acc[S::JT];
#pragma unroll
  for (int jt = 0; jt < S::JT; ++jt)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      b1acc[jt][v] = -kLog2e * pr.b1[32 * jt + 8 * (v >> 2) + 4 * half + (v & 3)];

  // Q as GEMM1 A operands: row = b_local * 8 + pq
  uint4 qop[S::KD];
  {
    const int b = qwv + (col >> 3), pq = col & 7;
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk) {
      if (b < pr.B)
        qop[kk] = *reinterpret_cast<const uint4*>(Q + (static_cast<long>(b) * 8 + pq) * D + 16 * kk + 8 * half);
      else
        qop[kk] = make_uint4(0, 0, 0, 0);
    }
  }
  // constant B operand of the a_q + b2 K block: ones in K slots 0 and 1
  f16x8_t ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = static_cast<_Float16>((half == 0 && e < 2) ? 1.f : 0.f);

  // ---- tile staging: global -> registers -> LDS (double buffered) ----
  uint4 xr[S::XCH], ar[S::ACH];
  auto load_tile = [&](int t) {
    const int n0 = nr0 + 32 * t;
#pragma unroll
    for (int c = 0; c < S::XCH; ++c) {
      const int ch = tid + 256 * c;
      const int px = ch / (32 * S::XROWCH), rem = ch % (32 * S::XROWCH);
      const int n = min(n0 + rem / S::XROWCH, N - 1), cc = rem % S::XROWCH;
      xr[c] = *reinterpret_cast<const uint4*>(X + (static_cast<long>(px) * N + n) * D + 8 * cc);
    }
#pragma unroll
    for (int c = 0; c < S::ACH; ++c) {
      const int ch = tid + 256 * c;
      const int n = min(n0 + ch / S::AROWCH, N - 1), cc = ch % S::AROWCH;
      ar[c] = *reinterpret_cast<const uint4*>(pr.a_x + static_cast<long>(n) * P + 4 * cc);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int c = 0; c < S::XCH; ++c) {
      const int ch = tid + 256 * c;
      const int px = ch / (32 * S::XROWCH), rem = ch % (32 * S::XROWCH);
      const int n = rem / S::XROWCH, cc = rem % S::XROWCH;
      const int phys = cc ^ (n % S::XROWCH);
      *reinterpret_cast<uint4*>(sX + ((buf * PX + px) * 32 + n) * D * 2 + 16 * phys) = xr[c];
    }
#pragma unroll
    for (int c = 0; c < S::ACH; ++c) {
      const int ch = tid + 256 * c;
      const int n = ch / S::AROWCH, cc = ch % S::AROWCH;
      const int phys = cc ^ (n % S::AROWCH);
      *reinterpret_cast<uint4*>(sAx + (buf * 32 + n) * P + 4 * phys) = ar[c];
    }
  };

  // running top-k state of the wave's 4 queries (wave-uniform)
  uint64_t theta[4] = {0ull, 0ull, 0ull, 0ull};
  int stg[4] = {0, 0, 0, 0};
  auto merge = [&](int bl) {
    uint64_t* reg = myTop + bl * (kTopkList + kTopkStage);
    wave_lds_sync();
    wave_sort256(reg, lane);
    for (int i = kTopkList + lane; i < kTopkList + kTopkStage; i += 64) reg[i] = 0ull;
    wave_lds_sync();
    theta[bl] = reg[k - 1];
    stg[bl] = 0;
  };

  if (ntiles > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int n0 = nr0 + 32 * t;
    if (t + 1 < ntiles) load_tile(t + 1);

    // GEMM1: component dot products for 4 queries x 32 items, all px
    f32x16_t acc1[PX];
#pragma unroll
    for (int px = 0; px < PX; ++px) {
      acc1[px] = f32x16_t{};
      const unsigned char* rowp = sX + ((buf * PX + px) * 32 + col) * D * 2;
#pragma unroll
      for (int kk = 0; kk < S::KD; ++kk) {
        const int phys = (2 * kk + half) ^ (col % S::XROWCH);
        const uint4 xb = *reinterpret_cast<const uint4*>(rowp + 16 * phys);
        acc1[px] = mfma_bf16(qop[kk], xb, acc1[px]);
      }
    }
    // a_x (scaled by log2 e) as the GEMM3 accumulator input
    f32x16_t axr[S::PT];
#pragma unroll
    for (int pt = 0; pt < S::PT; ++pt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int logical = PX * half + 4 * pt + q4;
        const int phys = logical ^ (col % S::AROWCH);
        const float4 a = *reinterpret_cast<const float4*>(sAx + (buf * 32 + col) * P + 4 * phys);
        axr[pt][4 * q4 + 0] = kLog2e * a.x;
        axr[pt][4 * q4 + 1] = kLog2e * a.y;
        axr[pt][4 * q4 + 2] = kLog2e * a.z;
        axr[pt][4 * q4 + 3] = kLog2e * a.w;
      }
    }
    const int item = n0 + col;
    const bool item_ok = item < nr1;

#pragma unroll
    for (int bl = 0; bl < 4; ++bl) {
      // GEMM2 B operands: f16 copies of this query's s values
      f16x8_t sop[S::KP];
#pragma unroll
      for (int m = 0; m < S::KP; ++m)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int lam = 8 * m + e;
          sop[m][e] = static_cast<_Float16>(acc1[lam % PX][4 * bl + lam / PX]);
        }
      f32x16_t u[S::JT];
#pragma unroll
      for (int jt = 0; jt < S::JT; ++jt) {
        u[jt] = b1acc[jt];
#pragma unroll
        for (int m = 0; m < S::KP; ++m)
          u[jt] = mfma_f16(__builtin_bit_cast(f16x8_t, sW1[(jt * S::KP + m) * 64 + lane]), sop[m], u[jt]);
      }
      // SiLU (scaled): h' = u' / (1 + 2^{u'}), packed as GEMM3 B operands
      f16x8_t hop[S::KH];
#pragma unroll
      for (int m = 0; m < S::KH; ++m)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = u[m >> 1][8 * (m & 1) + e];
          const float den = 1.f + __builtin_amdgcn_exp2f(x);
          hop[m][e] = static_cast<_Float16>(x * __builtin_amdgcn_rcpf(den));
        }
      // a_q + b2 (hi/lo f16) as one extra K block
      f32x16_t lg[S::PT];
#pragma unroll
      for (int pt = 0; pt < S::PT; ++pt) {
        const int rr = col;
        const int p = 4 * PX * ((rr & 7) >> 2) + 16 * pt + 4 * (rr >> 3) + (rr & 3);
        const uint32_t cb = sCb[(wave * 4 + bl) * P + p];
        uint4 cbw = make_uint4(half == 0 ? cb : 0u, 0u, 0u, 0u);
        lg[pt] = mfma_f16(__builtin_bit_cast(f16x8_t, cbw), ones, axr[pt]);
#pragma unroll
        for (int m = 0; m < S::KH; ++m)
          lg[pt] = mfma_f16(__builtin_bit_cast(f16x8_t, sW2[(pt * S::KH + m) * 64 + lane]), hop[m], lg[pt]);
      }
      // softmax over p and phi = sum pi_p s_p; lane holds p = 4 Px half + lambda
      float den = 0.f, num = 0.f;
#pragma unroll
      for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int lam = 16 * pt + v;
          const float w = __builtin_amdgcn_exp2f(lg[pt][v]);
          den += w;
          num = fmaf(w, acc1[lam % PX][4 * bl + lam / PX], num);
        }
      den += __shfl_xor(den, 32);
      num += __shfl_xor(num, 32);
      const bool ok = den >= 0x1p-60f && den <= 0x1p60f;
      if (!__all(ok)) {
        // logits far from zero: subtract the row maximum first
        float mx = -__builtin_inff();
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
          for (int v = 0; v < 16; ++v) mx = fmaxf(mx, lg[pt][v]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        den = 0.f;
        num = 0.f;
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int lam = 16 * pt + v;
            const float w = __builtin_amdgcn_exp2f(lg[pt][v] - mx);
            den += w;
            num = fmaf(w, acc1[lam % PX][4 * bl + lam / PX], num);
          }
        den += __shfl_xor(den, 32);
        num += __shfl_xor(num, 32);
      }
      const float phi = num / den;
      const int b = qwv + bl;

      if constexpr (DENSE) {
        if (half == 0 && item_ok && b < pr.B) phi_out[b * phi_stride + (item - n_begin)] = phi;
      } else {
        const uint64_t key = (half == 0 && item_ok) ? make_key(phi, item) : 0ull;
        const bool pass = key > theta[bl];
        const uint64_t mask = __ballot(pass);
        if (mask) {
          uint64_t* reg = myTop + bl * (kTopkList + kTopkStage);
          const int below = __popcll(mask & ((1ull << lane) - 1ull));
          if (pass) reg[kTopkList + stg[bl] + below] = key;
          stg[bl] += __popcll(mask);
          if (stg[bl] > kTopkStage - 32) merge(bl);
        }
      }
    }

    if (t + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  if constexpr (!DENSE) {
#pragma unroll
    for (int bl = 0; bl < 4; ++bl) {
      if (stg[bl] > 0) merge(bl);
      const int b = qwv + bl;
      if (b < pr.B) {
        const uint64_t* reg = myTop + bl * (kTopkList + kTopkStage);
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
  G = (pr.B + 15) / 16;
  R = std::max(1, 256 / G);
  const int max_r = std::max(1, n_count / 512);
  R = std::min(R, max_r);
  range_len = (n_count + R - 1) / R;
  range_len = (range_len + 31) / 32 * 32;
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
  hipLaunchKernelGGL(kern, dim3(R * G), dim3(256), S::LDS_TOTAL, st, pr, k, R, range_len, G,
                     n_begin, n_end, partial, phi, phi_stride);
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
