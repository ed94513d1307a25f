// Per-component top-k' on gfx950 matrix cores (TopKDotProduct for every
// component, Algorithm 2's TopKPerEmbedding stage 1; with P_q = P_x = 1 on
// the averaged embeddings it is TopKAvg).
//
// Each (query vector f_pq(q), item table X_px) pair is one independent
// maximum-inner-product list.  A workgroup streams an item range of one
// component px through LDS; each wave multiplies every 32-item tile
// (A operand, read once from LDS) with NB blocks of 32 query vectors
// (B operands, in registers) on 32x32x16 bf16 MFMAs.  In the result
// D[item][query vector] lane (c = lane % 32, h = lane / 32) holds, per
// block, 16 items' scores for the single list of query vector c: every
// list is owned by two lanes, each seeing half of the items.  A lane keeps
// its list's running threshold (the k'-th best key merged so far) and
// appends the scores that reach it to its own staging region in the
// workspace; about k' (1 + ln(n / k')) keys per list survive over n items.
// A full staging region is merged into the list (also in the workspace) by
// a wave-wide bitonic sort in LDS.  Lists of several item ranges are merged
// afterwards by segmented sorts.
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kNB = 2;                       // query-vector blocks per wave
constexpr int kVecPerWave = 32 * kNB;
constexpr int kVecPerWG = kWaves * kVecPerWave;
constexpr int kStageBytes = 16384;           // bytes of one LDS item stage
constexpr int kRing = 4;                     // item stages in flight
constexpr int kSortKeys = 512;               // keys of one wave's merge sort
constexpr int kSGMax = (kSortKeys - 128) / 2;  // largest staging region per lane half

__device__ __forceinline__ f32x16_t mfma32_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

template <int D, int KL>
struct EmbdShape {
  static constexpr int KD = D / 16;                    // K blocks (32x32x16)
  static constexpr int ROWCH = D / 8;                  // 16-byte chunks per item row
  static constexpr int ST = kStageBytes / (2 * D);     // items per stage
  static constexpr int SORT = kSortKeys;
  static constexpr int SG = (kSortKeys - KL) / 2;      // staging slots per (list, lane half)
  static constexpr int LOADS = kStageBytes / 1024 / kWaves;   // copies per lane per stage
  static constexpr int LDS_X = kRing * kStageBytes;
  static constexpr int LDS_SORT = kWaves * SORT * 8;
  static constexpr int LDS_TOTAL = LDS_X + LDS_SORT;
  static_assert(ST % 32 == 0, "stage holds whole 32-item tiles");
  static_assert(KL + 2 * SG <= SORT && SG <= kSGMax, "sort region holds list + both staging halves");
};

}  // namespace

// Grid: WG -> (vector group, px, range).  WGs sharing (px, range) are placed
// on the same XCD (WG id mod 8) when the grid allows it.
// lists: [nvec * Px][R][KL] keys; stg: [nvec * Px][R][2][SG] keys.
template <int D, int KL>
__global__ __launch_bounds__(64 * kWaves, 1) void k_topk_per_embd(
    DevProb pr, int kp, int R, int range_len, int G, uint64_t* __restrict__ lists,
    uint64_t* __restrict__ stg) {
  using S = EmbdShape<D, KL>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  uint64_t* sSort = reinterpret_cast<uint64_t*>(smem + S::LDS_X);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int Px = pr.Px, N = pr.N;
  const int nvec = pr.B * pr.Pq;               // query vectors
  const int total = gridDim.x;
  int L = blockIdx.x;
  if (total % 8 == 0) L = (blockIdx.x >> 3) + (total >> 3) * (blockIdx.x & 7);
  const int rg = L % G, unit = L / G;
  const int px = unit % Px, r = unit / Px;
  const int vwave = rg * kVecPerWG + wave * kVecPerWave;   // first query vector of the wave
  const int nr0 = r * range_len, nr1 = min(N, nr0 + range_len);
  const int nstages = nr1 > nr0 ? (nr1 - nr0 + S::ST - 1) / S::ST : 0;

  const bf16_t* X = static_cast<const bf16_t*>(pr.X) + static_cast<long>(px) * N * D;
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);

  auto stage = [&](int t, int buf) {
    const int n0 = nr0 + S::ST * t;
    for (int blk = wave; blk < kStageBytes / 1024; blk += kWaves) {
      const int pos = blk * 64 + lane;
      const int n = pos / S::ROWCH, phys = pos % S::ROWCH;
      const int cc = phys ^ (n % S::ROWCH);
      const int item = min(n0 + n, N - 1);
      const bf16_t* src = X + static_cast<long>(item) * D + 8 * cc;
      __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)(sX + buf * kStageBytes + blk * 1024),
                                       16, 0, 0);
    }
  };
  for (int t = 0; t < kRing - 1 && t < nstages; ++t) stage(t, t);

  // query vectors as B operands: column = lane % 32 within each block
  uint4 qop[kNB][S::KD];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int v = vwave + 32 * nb + col;
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk)
      qop[nb][kk] = v < nvec ? *reinterpret_cast<const uint4*>(Q + static_cast<long>(v) * D + 16 * kk + 8 * half)
                             : make_uint4(0, 0, 0, 0);
  }
  uint64_t* mySort = sSort + wave * S::SORT;
  // list of (block nb, column c): query vector vwave + 32 nb + c, component px, range r
  auto list_idx = [&](int nb, int c) { return (static_cast<long>(vwave + 32 * nb + c) * Px + px) * R + r; };
  auto stg_ptr = [&](int nb, int c, int h) { return stg + (list_idx(nb, c) * 2 + h) * S::SG; };
  // per-lane list state: threshold (float score of the k'-th key) and staging count
  float th[kNB];
  int cnt[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const bool vok = vwave + 32 * nb + col < nvec;
    th[nb] = vok ? -__builtin_inff() : __builtin_inff();   // invalid vectors never pass
    cnt[nb] = 0;
    if (vok && half == 0) {
      uint64_t* lp = lists + list_idx(nb, col) * KL;
      for (int i = 0; i < KL; ++i) lp[i] = 0ull;
    }
  }
  // merge the staged keys of list (nb, c) into it; nb and c are wave-uniform
  auto merge = [&](int nb, int c) {
    // staged keys were written by other lanes of this wave: make them visible
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
    const int c0 = __builtin_amdgcn_readlane(cnt[nb], c);
    const int c1 = __builtin_amdgcn_readlane(cnt[nb], c + 32);
    uint64_t* lp = lists + list_idx(nb, c) * KL;
    const uint64_t* s0 = stg_ptr(nb, c, 0);
    const uint64_t* s1 = stg_ptr(nb, c, 1);
    // every slot loads from a valid address (branch-free, so all loads are
    // in flight together); slots past the staged counts are cleared
    uint64_t vals[S::SORT / 64];
#pragma unroll
    for (int j = 0; j < S::SORT / 64; ++j) {
      const int i = lane + 64 * j;
      const int a = i - KL, b = i - KL - S::SG;
      const uint64_t* src = i < KL ? lp + i : (a < S::SG ? s0 + max(a, 0) : s1 + min(max(b, 0), S::SG - 1));
      vals[j] = *src;
    }
#pragma unroll
    for (int j = 0; j < S::SORT / 64; ++j) {
      const int i = lane + 64 * j;
      const int a = i - KL, b = i - KL - S::SG;
      const bool keep = i < KL || (a < S::SG ? a < c0 : (b < S::SG && b < c1));
      mySort[i] = keep ? vals[j] : 0ull;
    }
    wave_lds_sync();
    wave_sort<S::SORT>((lds_u64_t*)mySort, lane);
    for (int i = lane; i < KL; i += 64) lp[i] = mySort[i];
    const float nth = key_score(mySort[kp - 1]);
    wave_lds_sync();
    if (col == c) {
      th[nb] = nth;
      cnt[nb] = 0;
    }
  };

  // stage 0 complete; the copies of later stages may still be in flight
  if (nstages >= kRing - 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm((kRing - 2) * S::LOADS));
  else if (nstages == 2) __builtin_amdgcn_s_waitcnt(waitcnt_vm(S::LOADS));
  else __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int t = 0; t < nstages; ++t) {
    const int buf = t % kRing;
    const unsigned char* xs = sX + buf * kStageBytes;
    for (int tt = 0; tt < S::ST / 32; ++tt) {
      const int n = 32 * tt + col;                    // A-operand row = item
      const int n0 = nr0 + S::ST * t + 32 * tt;       // first item of the tile
      f32x16_t acc[kNB];
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) acc[nb] = f32x16_t{};
      const unsigned char* rowp = xs + n * (2 * D);
#pragma unroll
      for (int kk = 0; kk < S::KD; ++kk) {
        const uint4 xa = *reinterpret_cast<const uint4*>(rowp + 16 * ((2 * kk + half) ^ (n % S::ROWCH)));
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) acc[nb] = mfma32_bf16(xa, qop[nb][kk], acc[nb]);
      }
      // lane (c, h) register v holds item n0 + (v/4)*8 + 4h + v%4 of list c
      if (n0 + 32 > nr1) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const bool ok = n0 + (v >> 2) * 8 + 4 * half + (v & 3) < nr1;
#pragma unroll
          for (int nb = 0; nb < kNB; ++nb) acc[nb][v] = ok ? acc[nb][v] : __builtin_nanf("");  // never passes
        }
      }
      uint64_t any = 0ull;
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int v = 0; v < 16; ++v) any |= __ballot(acc[nb][v] >= th[nb]);
      if (any == 0ull) continue;
      // append survivors to the lane's own staging region
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) {
        uint64_t* sp = stg_ptr(nb, col, half);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (acc[nb][v] >= th[nb]) {
            const int item = n0 + (v >> 2) * 8 + 4 * half + (v & 3);
            sp[cnt[nb]] = make_key(acc[nb][v], item);
            ++cnt[nb];
          }
        }
      }
      // merge lists whose staging could overflow on the next tile
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) {
        uint64_t need = __ballot(cnt[nb] > S::SG - 16);
        while (need) {
          const int c = __builtin_ctzll(need) & 31;
          need &= ~((1ull << c) | (1ull << (c + 32)));
          merge(nb, c);
        }
      }
    }
    // refill the buffer read in iteration t-1 (every wave finished it before
    // the barrier that ended iteration t-1), then wait for stage t+1
    if (t + kRing - 1 < nstages) {
      stage(t + kRing - 1, (t + kRing - 1) % kRing);
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((kRing - 2) * S::LOADS));
    } else {
      __builtin_amdgcn_s_waitcnt(0);
    }
    __syncthreads();
  }
  // flush the remaining staged keys
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    uint64_t need = __ballot(cnt[nb] > 0);
    while (need) {
      const int c = __builtin_ctzll(need) & 31;
      need &= ~((1ull << c) | (1ull << (c + 32)));
      merge(nb, c);
    }
  }
}

// ---------------------------------------------------------------------------
bool per_embd_supported(const DevProb& pr, int kp) {
  if (pr.dtype != MOL_BF16) return false;
  if (pr.d != 64 && pr.d != 128) return false;
  return kp <= 256;
}

int per_embd_list_cap(int kp) { return kp <= 128 ? 128 : 256; }
int per_embd_stage_cap() { return 2 * kSGMax; }

void per_embd_grid(const DevProb& pr, int& R, int& range_len, int& G) {
  const int nvec = pr.B * pr.Pq;
  G = (nvec + kVecPerWG - 1) / kVecPerWG;
  const int units = G * pr.Px;
  R = std::max(1, (256 + units - 1) / units);
  R = std::min(R, std::max(1, pr.N / 4096));
  range_len = (pr.N + R - 1) / R;
  range_len = (range_len + 127) / 128 * 128;
  R = (pr.N + range_len - 1) / range_len;
}

template <int D, int KL>
static hipError_t launch_pe_t(const DevProb& pr, int kp, int R, int range_len, int G, uint64_t* lists,
                              uint64_t* stg, hipStream_t st) {
  using S = EmbdShape<D, KL>;
  auto kern = &k_topk_per_embd<D, KL>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS_TOTAL);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(G * pr.Px * R), dim3(64 * kWaves), S::LDS_TOTAL, st, pr, kp, R,
                     range_len, G, lists, stg);
  return hipGetLastError();
}

hipError_t launch_per_embd(const DevProb& pr, int kp, int R, int range_len, int G, uint64_t* lists,
                           uint64_t* stg, hipStream_t st) {
  const int KL = per_embd_list_cap(kp);
  if (pr.d == 64)
    return KL == 128 ? launch_pe_t<64, 128>(pr, kp, R, range_len, G, lists, stg, st)
                     : launch_pe_t<64, 256>(pr, kp, R, range_len, G, lists, stg, st);
  return KL == 128 ? launch_pe_t<128, 128>(pr, kp, R, range_len, G, lists, stg, st)
                   : launch_pe_t<128, 256>(pr, kp, R, range_len, G, lists, stg, st);
}

}  // namespace mol
