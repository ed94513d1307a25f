// Per-component top-k' on gfx950 matrix cores (TopKDotProduct for every
// component, Algorithm 2's TopKPerEmbedding stage 1; with P_q = P_x = 1 on
// the averaged embeddings it is TopKAvg).
//
// Each (query vector f_pq(q), item table X_px) pair is one independent
// maximum-inner-product list.  A wave owns 32 query vectors and, for one
// item component px and one item range, streams 32-item tiles through a
// 32x32x16 bf16 MFMA: lane (item c = lane % 32, half h = lane / 32) then
// holds the dot products of its item with 16 of the 32 query vectors.  Each
// score is compared with its list's running threshold (the k'-th best key
// so far); the survivors (on average k' (1 + ln(n / k')) per list over n
// items) are appended to a per-list staging buffer in the workspace, and a
// full buffer is merged into the list by a wave-wide bitonic sort in LDS.
// Lists from several item ranges are merged afterwards by segmented sorts.
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWaves = 8;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWG = kWaves * kRowsPerWave;
constexpr int kStageBytes = 16384;  // bytes of one LDS item stage
constexpr int kSG = 224;            // staging slots per list (workspace)
constexpr int kRing = 4;            // item stages in flight

__device__ __forceinline__ f32x16_t mfma32_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

template <int D, int KL>
struct EmbdShape {
  static constexpr int KD = D / 16;                    // K blocks (32x32x16)
  static constexpr int ROWCH = D / 8;                  // 16-byte chunks per item row
  static constexpr int ST = kStageBytes / (2 * D);     // items per stage
  static constexpr int SORT = 512;                     // >= KL + kSG
  static constexpr int LDS_X = kRing * kStageBytes;
  static constexpr int LOADS = kStageBytes / 1024 / kWaves;   // copies per lane per stage
  static constexpr int LDS_SORT = kWaves * SORT * 8;
  static constexpr int LDS_META = kWaves * kRowsPerWave * (8 + 4);
  static constexpr int LDS_TOTAL = LDS_X + LDS_SORT + LDS_META;
  static_assert(ST % 64 == 0, "stage holds whole pairs of 32-item tiles");
  static_assert(KL + kSG <= SORT, "sort region holds list + staging");
  // a stage appends at most ST keys per list; merge before that can overflow
  static constexpr int MERGE_AT = kSG - ST;
  static_assert(MERGE_AT > 0, "staging must absorb one stage");
};

}  // namespace

// Grid: WG -> (row group, px, range).  WGs sharing (px, range) are placed
// on the same XCD (WG id mod 8) when the grid allows it.
// lists: [nvec * Px][R][KL] keys; stg: [nvec * Px][R][kSG] keys.
template <int D, int KL>
__global__ __launch_bounds__(64 * kWaves, 1) void k_topk_per_embd(
    DevProb pr, int kp, int R, int range_len, int G, uint64_t* __restrict__ lists,
    uint64_t* __restrict__ stg) {
  using S = EmbdShape<D, KL>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  uint64_t* sSort = reinterpret_cast<uint64_t*>(smem + S::LDS_X);
  uint64_t* sTh = reinterpret_cast<uint64_t*>(smem + S::LDS_X + S::LDS_SORT);
  int* sCnt = reinterpret_cast<int*>(sTh + kWaves * kRowsPerWave);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int Px = pr.Px, N = pr.N;
  const int nvec = pr.B * pr.Pq;               // query vectors
  const int total = gridDim.x;
  int L = blockIdx.x;
  if (total % 8 == 0) L = (blockIdx.x >> 3) + (total >> 3) * (blockIdx.x & 7);
  const int rg = L % G, unit = L / G;
  const int px = unit % Px, r = unit / Px;
  const int vbase = rg * kRowsPerWG + wave * kRowsPerWave;   // first query vector of the wave
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

  // query vectors as A operands: row = lane % 32
  uint4 qop[S::KD];
  {
    const int v = vbase + col;
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk)
      qop[kk] = v < nvec ? *reinterpret_cast<const uint4*>(Q + static_cast<long>(v) * D + 16 * kk + 8 * half)
                         : make_uint4(0, 0, 0, 0);
  }
  uint64_t* mySort = sSort + wave * S::SORT;
  uint64_t* myTh = sTh + wave * kRowsPerWave;
  int* myCnt = sCnt + wave * kRowsPerWave;
  // list and staging of wave row w: (query vector vbase + w, component px, range r)
  auto list_idx = [&](int w) { return (static_cast<long>(vbase + w) * Px + px) * R + r; };
  if (lane < kRowsPerWave) {
    myTh[lane] = 0ull;
    myCnt[lane] = 0;
  }
  for (int w = 0; w < kRowsPerWave; ++w) {
    if (vbase + w >= nvec) break;
    uint64_t* lp = lists + list_idx(w) * KL;
    for (int i = lane; i < KL; i += 64) lp[i] = 0ull;
  }
  // row of accumulator register v for this lane
  auto row_of = [&](int v) { return (v >> 2) * 8 + 4 * half + (v & 3); };
  // thresholds of the lane's 16 lists; rows past the last query vector never pass
  float thf[16];
  auto load_thresholds = [&]() {
#pragma unroll
    for (int v = 0; v < 16; ++v)
      thf[v] = vbase + row_of(v) < nvec ? key_score(myTh[row_of(v)]) : __builtin_inff();
  };
  auto merge = [&](int w) {
    // staged keys were written by other lanes of this wave: make them visible
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
    const int cnt = myCnt[w];
    uint64_t* lp = lists + list_idx(w) * KL;
    const uint64_t* sp = stg + list_idx(w) * kSG;
    for (int i = lane; i < S::SORT; i += 64) {
      uint64_t v = 0ull;
      if (i < KL) v = lp[i];
      else if (i - KL < cnt) v = sp[i - KL];
      mySort[i] = v;
    }
    wave_lds_sync();
    wave_sort<S::SORT>((lds_u64_t*)mySort, lane);
    for (int i = lane; i < KL; i += 64) lp[i] = mySort[i];
    if (lane == 0) {
      myTh[w] = mySort[kp - 1];
      myCnt[w] = 0;
    }
    wave_lds_sync();
  };

  // stage 0 complete; the loads of stages 1 .. issued-1 may still be in flight
  if (nstages >= kRing - 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm((kRing - 2) * S::LOADS));
  else if (nstages == 2) __builtin_amdgcn_s_waitcnt(waitcnt_vm(S::LOADS));
  else __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  load_thresholds();

  // survivors of one 32-item tile (scores in acc) are appended to staging
  auto append = [&](f32x16_t& acc, int item, bool item_ok) {
    if (!__all(item_ok)) {
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] = item_ok ? acc[v] : __builtin_nanf("");  // never passes
    }
    uint64_t mv[16];
    uint64_t any = 0ull;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      mv[v] = __ballot(acc[v] >= thf[v]);
      any |= mv[v];
    }
    if (any == 0ull) return;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const uint64_t m = mv[v];
      if (m == 0ull) continue;
      const int w = row_of(v);
      const uint32_t mh = half ? static_cast<uint32_t>(m >> 32) : static_cast<uint32_t>(m);
      const int base = myCnt[w];
      if ((mh >> col) & 1u) {
        const int below = __popc(mh & ((1u << col) - 1u));
        stg[list_idx(w) * kSG + base + below] = make_key(acc[v], item);
      }
      if (col == 0) myCnt[w] = base + __popc(mh);
    }
  };

  for (int t = 0; t < nstages; ++t) {
    const int buf = t % kRing;
    const unsigned char* xs = sX + buf * kStageBytes;
    for (int tt = 0; tt < S::ST / 64; ++tt) {
      // two independent 32-item tiles per step
      const int na = 64 * tt + col, nb = na + 32;
      const int itema = nr0 + S::ST * t + na, itemb = itema + 32;
      f32x16_t acca = {}, accb = {};
      const unsigned char* rowa = xs + na * (2 * D);
      const unsigned char* rowb = xs + nb * (2 * D);
#pragma unroll
      for (int kk = 0; kk < S::KD; ++kk) {
        const int pa = (2 * kk + half) ^ (na % S::ROWCH);
        const int pb = (2 * kk + half) ^ (nb % S::ROWCH);
        acca = mfma32_bf16(qop[kk], *reinterpret_cast<const uint4*>(rowa + 16 * pa), acca);
        accb = mfma32_bf16(qop[kk], *reinterpret_cast<const uint4*>(rowb + 16 * pb), accb);
      }
      append(acca, itema, itema < nr1);
      append(accb, itemb, itemb < nr1);
    }
    // merge lists whose staging could overflow during the next stage
    wave_lds_sync();
    uint64_t nm = __ballot(lane < kRowsPerWave && myCnt[lane] > S::MERGE_AT);
    if (nm) {
      while (nm) {
        const int w = __builtin_ctzll(nm);
        nm &= nm - 1;
        merge(w);
      }
      load_thresholds();
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
  uint64_t nm = __ballot(lane < kRowsPerWave && myCnt[lane] > 0 && vbase + lane < nvec);
  while (nm) {
    const int w = __builtin_ctzll(nm);
    nm &= nm - 1;
    merge(w);
  }
}

// ---------------------------------------------------------------------------
bool per_embd_supported(const DevProb& pr, int kp) {
  if (pr.dtype != MOL_BF16) return false;
  if (pr.d != 64 && pr.d != 128) return false;
  return kp <= 256;
}

int per_embd_list_cap(int kp) { return kp <= 128 ? 128 : 256; }
int per_embd_stage_cap() { return kSG; }

void per_embd_grid(const DevProb& pr, int& R, int& range_len, int& G) {
  const int nvec = pr.B * pr.Pq;
  G = (nvec + kRowsPerWG - 1) / kRowsPerWG;
  const int units = G * pr.Px;
  R = std::max(1, (256 + units - 1) / units);
  R = std::min(R, std::max(1, pr.N / 4096));
  range_len = (pr.N + R - 1) / R;
  range_len = (range_len + 63) / 64 * 64;
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
