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
// list is owned by two lanes, each seeing half of the items.
//
// Two passes over the same dot products:
//  1. the bucket scan keeps, per list, the maximum score over each bucket
//     of `bucket_tiles` tiles (both lanes of the list joined at the bucket
//     end) and stores the bucket maxima;
//  2. the k'-th largest bucket maximum T of a list is a lower bound of the
//     list's k'-th largest score (k' disjoint buckets each hold an item at
//     least that large), so only items scoring at least T can be in the
//     list, and they lie in the buckets whose maximum reaches T (about k'
//     of them).  For lists of up to 256 keys the pruned pass therefore
//     recomputes, per bucket, only the query vectors for which the bucket
//     is "hot" (gathered into 32-vector MFMA blocks; about k' / buckets of
//     the work of a full scan) and appends every score reaching T to the
//     list's key buffer; a sort per list finishes it.  Should a list
//     receive more keys than its buffer holds (massive ties), a device flag
//     switches the call to the threshold scan below for every list.
//     The threshold scan walks all items again from T: scores that reach
//     it are appended to the lane's staging region in the workspace; a full
//     staging region is merged into the list by a wave-wide bitonic sort in
//     LDS, and the threshold rises to the list's k'-th key.  Lists of
//     several item ranges are merged afterwards by segmented sorts.
// Every pass evaluates bit-identical dot products (the same instructions in
// the same accumulation order on the same tile rows; the pruned pass also
// lowers T by a few units in the last place, so a different MFMA column
// could not drop a key), so the bound is exact.
#include <type_traits>

#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// query-vector blocks of 32 per wave, chosen so that the B operands and two
// tiles' accumulators stay in registers: 4 in the bucket scan at d = 64,
// 2 otherwise (the threshold scan also keeps staging state)
constexpr int nb_for(int d, bool scan2) { return (d >= 128 || scan2) ? 2 : 4; }
// small batches (at most 256 query vectors) use one block per wave, so that
// no wave multiplies empty vector slots
constexpr int kSmallVectors = 256;
constexpr int nb_pick(int d, bool scan2, bool small) { return small ? 1 : nb_for(d, scan2); }
// waves per workgroup: 8, or 4 for lists of 512 / 1024 keys, whose merge
// sorts need 8 / 16 KB of LDS per wave
constexpr int waves_for(int kl) { return kl >= 512 ? 4 : 8; }
enum ScanMode { kScanBuckets = 0, kScanThreshold = 1, kScanPruned = 2 };
constexpr int kRing = 3;                     // item stages in flight
constexpr int kSGMax = 512;                  // largest staging region per lane half
constexpr int kMaxBuckets = 2048;            // bucket maxima per list (all ranges, both halves)

__device__ __forceinline__ f32x16_t mfma32_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// per-lane key slots of the pruned pass's LDS staging, per vector block
constexpr int kHitSlots = 2;

template <int D, int KL, bool SCAN2, bool SMALL, bool PRUNED = false>
struct EmbdShape {
  static constexpr int KD = D / 16;                    // K blocks (32x32x16)
  static constexpr int NB = nb_pick(D, SCAN2, SMALL);
  static constexpr int VEC_WAVE = 32 * NB;             // query vectors per wave
  static constexpr int WAVES = waves_for(KL);
  static constexpr int VEC_WG = WAVES * VEC_WAVE;
  static constexpr int STAGE_BYTES = WAVES == 8 ? 32768 : 16384;   // bytes of one LDS item stage
  static constexpr int ROWCH = D / 8;                  // 16-byte chunks per item row
  // XOR swizzle of a row's chunks: the 16 rows one 16-lane group reads land
  // on distinct 16-byte bank slots of each 256-byte LDS line
  static constexpr int RPL = D >= 128 ? 1 : 128 / D;   // rows per 256-byte line
  __device__ static int swz(int n) { return (n / RPL) % ROWCH; }
  static constexpr int ST = STAGE_BYTES / (2 * D);     // items per stage
  static constexpr int SORT = KL <= 256 ? 512 : 2 * KL;  // keys of one wave's merge sort
  static constexpr int SG = (SORT - KL) / 2;           // staging slots per (list, lane half)
  static constexpr int LOADS = STAGE_BYTES / 1024 / WAVES;   // copies per lane per stage
  static constexpr int LDS_X = kRing * STAGE_BYTES;
  static constexpr int LDS_SORT = SCAN2 ? WAVES * SORT * 8 : 0;   // the threshold scan's merge sorts
  // the pruned pass: kHitSlots keys per (wave, block, lane), lane-contiguous
  static constexpr int LDS_HIT = PRUNED ? WAVES * NB * kHitSlots * 64 * 8 : 0;
  static constexpr int LDS_TOTAL = LDS_X + LDS_SORT + LDS_HIT;
  static_assert(ST % 32 == 0, "stage holds whole 32-item tiles");
  static_assert(KL + 2 * SG <= SORT && SG <= kSGMax, "sort region holds list + both staging halves");
  static_assert(LDS_TOTAL <= 160 * 1024, "LDS budget");
};

}  // namespace

// Inputs and outputs of the pruned pass (and the flag the threshold scan
// and the final selection are gated on).
struct PrunedArgs {
  const int* work = nullptr;          // [groups * CH]: g * CH + chunk of each work item
  const uint32_t* work_total = nullptr;
  const int* hot_v = nullptr;         // [groups][nvec]: query vectors for which bucket g is hot
  const int* hot_n = nullptr;         // [groups]
  uint32_t* cnt = nullptr;            // [nvec * Px]: keys appended per list
  uint64_t* keys = nullptr;           // [nvec * Px][cap]
  uint32_t* flag = nullptr;           // set when some list received more than cap keys
  int cap = 0, CH = 0;
};

// Grid: WG -> (vector group, px, range).  WGs sharing (px, range) are placed
// on the same XCD (WG id mod 8) when the grid allows it.
// R, range_len, G: this scan's item ranges and query-vector groups.
// bmax: [Px][R][nbk][nvec] bucket maxima (bucket scan writes; for one
//   (component, range, bucket) the lists are contiguous, so a wave's store
//   covers one line);
// thr: [nvec * Px] starting thresholds (threshold scan and pruned pass read);
// lists: [nvec * Px][R][KL] keys; stg: [nvec * Px][R][2][SG] keys (threshold scan);
// gate: the threshold scan does nothing while *gate is zero (NULL: always runs);
// pa: the pruned pass's work list and outputs.  In the pruned pass R,
// range_len, bucket_tiles and nbk are the bucket scan's, whose buckets are
// the pass's work units.
template <int D, int KL, int MODE, bool SMALL>
__global__ __launch_bounds__(64 * waves_for(KL), 1) void k_topk_per_embd(
    DevProb pr, int kp, int R, int range_len, int G, int bucket_tiles, int nbk,
    float* __restrict__ bmax, const float* __restrict__ thr, uint64_t* __restrict__ lists,
    uint64_t* __restrict__ stg, const uint32_t* __restrict__ gate, PrunedArgs pa) {
  constexpr bool SCAN2 = MODE == kScanThreshold;
  constexpr bool PRUNED = MODE == kScanPruned;
  using S = EmbdShape<D, KL, SCAN2, SMALL, PRUNED>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  uint64_t* sSort = reinterpret_cast<uint64_t*>(smem + S::LDS_X);
  uint64_t* sHit = reinterpret_cast<uint64_t*>(smem + S::LDS_X + S::LDS_SORT);

  if (SCAN2 && gate && *gate == 0u) return;    // whole workgroup
  // one work unit: the workgroup's (vector group, px, range) of a full
  // scan, or work item wi of the pruned pass
  auto run = [&](int wi) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int col = lane & 31, half = lane >> 5;
  const int Px = pr.Px, N = pr.N;
  const int nvec = pr.B * pr.Pq;               // query vectors
  int px, r, nr0, nr1;
  int vwave = 0;                               // first query vector of the wave (full scans)
  int grp = 0, chunk = 0;                      // pruned pass: bucket group and vector chunk
  if constexpr (PRUNED) {
    const int item = pa.work[wi];
    grp = item / pa.CH;
    chunk = item - grp * pa.CH;
    px = grp / (R * nbk);
    r = (grp / nbk) % R;
    nr0 = r * range_len + (grp % nbk) * bucket_tiles * 32;
    nr1 = min(N, min(r * range_len + range_len, nr0 + bucket_tiles * 32));
  } else {
    const int total = gridDim.x;
    int L = wi;
    if (total % 8 == 0) L = (blockIdx.x >> 3) + (total >> 3) * (blockIdx.x & 7);
    const int rg = L % G, unit = L / G;
    px = unit % Px;
    r = unit / Px;
    vwave = rg * S::VEC_WG + wave * S::VEC_WAVE;
    nr0 = r * range_len;
    nr1 = min(N, nr0 + range_len);
  }
  const int nstages = nr1 > nr0 ? (nr1 - nr0 + S::ST - 1) / S::ST : 0;

  const bf16_t* X = static_cast<const bf16_t*>(pr.X) + static_cast<long>(px) * N * D;
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);

  auto stage = [&](int t, int buf) {
    const int n0 = nr0 + S::ST * t;
    for (int blk = wave; blk < S::STAGE_BYTES / 1024; blk += S::WAVES) {
      const int pos = blk * 64 + lane;
      const int n = pos / S::ROWCH, phys = pos % S::ROWCH;
      const int cc = phys ^ S::swz(n);
      const int item = min(n0 + n, N - 1);
      const bf16_t* src = X + static_cast<long>(item) * D + 8 * cc;
      copy16_to_lds(src, lds_addr(sX + buf * S::STAGE_BYTES + blk * 1024));
    }
  };
  for (int t = 0; t < kRing - 1 && t < nstages; ++t) stage(t, t);

  // the query vector of the lane's column in block nb (-1: none)
  int vv[S::NB];
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    if constexpr (PRUNED) {
      // slots interleaved over the waves: a chunk's hot vectors (about 80 %
      // of its slots) then load every wave alike, and the waves, which meet
      // at every stage's barrier, wait less for the one with the most hits
      // (exact_1m: 9.15 -> 8.89 ms for the call; hybrid_8m: 16.67 -> 16.79)
      const int slot = chunk * S::VEC_WG + (32 * nb + col) * S::WAVES + wave;
      vv[nb] = slot < pa.hot_n[grp] ? pa.hot_v[static_cast<long>(grp) * nvec + slot] : -1;
    } else {
      const int v = vwave + 32 * nb + col;
      vv[nb] = v < nvec ? v : -1;
    }
  }
  // query vectors as B operands: column = lane % 32 within each block
  uint4 qop[S::NB][S::KD];
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    const int v = vv[nb];
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk)
      qop[nb][kk] = v >= 0 ? *reinterpret_cast<const uint4*>(Q + static_cast<long>(v) * D + 16 * kk + 8 * half)
                           : make_uint4(0, 0, 0, 0);
  }
  uint64_t* mySort = sSort + wave * S::SORT;
  // list of (block nb, column c): query vector vwave + 32 nb + c, component px, range r
  auto list_idx = [&](int nb, int c) { return (static_cast<long>(vwave + 32 * nb + c) * Px + px) * R + r; };
  auto stg_ptr = [&](int nb, int c, int h) { return stg + (list_idx(nb, c) * 2 + h) * S::SG; };
  // per-lane state.  Scan 1: running bucket maximum.  Scan 2: threshold
  // (float score every appended key reaches), staging count, and whether the
  // list has been merged into (it is empty otherwise).
  bool vok[S::NB];
  float th[S::NB], bm[S::NB];
  int cnt[S::NB];
  bool merged[S::NB];
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    vok[nb] = vv[nb] >= 0;
    bm[nb] = -__builtin_inff();
    cnt[nb] = 0;
    merged[nb] = false;
    th[nb] = __builtin_inff();                      // invalid vectors never pass
    if (SCAN2 && vok[nb]) {
      th[nb] = thr[static_cast<long>(vv[nb]) * Px + px];
      if (half == 0) {
        uint64_t* lp = lists + list_idx(nb, col) * KL;
        for (int i = 0; i < KL; ++i) lp[i] = 0ull;
      }
    }
    if (PRUNED && vok[nb]) {
      // T lowered by a few units in the last place (see the file comment)
      const float t = thr[static_cast<long>(vv[nb]) * Px + px];
      th[nb] = t - 0x1p-20f * fmaxf(1.f, fabsf(t));
    }
  }
  // bucket maxima of (px, r): bucket bk of query vector v at bucket_row[bk * nvec + v]
  float* bucket_row = bmax + (static_cast<long>(px) * R + r) * nbk * nvec;
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
    constexpr int kBatch = 4;                     // loads in flight per lane
#pragma unroll
    for (int j0 = 0; j0 < S::SORT / 64; j0 += kBatch) {
      uint64_t vals[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = lane + 64 * (j0 + j);
        const int a = i - KL, b = i - KL - S::SG;
        const uint64_t* src = i < KL ? lp + i : (a < S::SG ? s0 + max(a, 0) : s1 + min(max(b, 0), S::SG - 1));
        vals[j] = *src;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int i = lane + 64 * (j0 + j);
        const int a = i - KL, b = i - KL - S::SG;
        const bool keep = i < KL || (a < S::SG ? a < c0 : (b < S::SG && b < c1));
        mySort[i] = keep ? vals[j] : 0ull;
      }
    }
    wave_lds_sync();
    wave_sort<S::SORT>((lds_u64_t*)mySort, lane);
    for (int i = lane; i < KL; i += 64) lp[i] = mySort[i];
    const float nth = key_score(mySort[kp - 1]);
    wave_lds_sync();
    if (col == c) {
      th[nb] = fmaxf(th[nb], nth);
      cnt[nb] = 0;
      merged[nb] = true;
    }
  };

  // stage 0 complete; the copies of later stages may still be in flight
  if (nstages >= kRing - 1) ring_barrier<(kRing - 2) * S::LOADS>();
  else if (nstages == 2) ring_barrier<S::LOADS>();
  else ring_barrier<0>();

  // Tiles are software-pipelined in pairs: the MFMAs of one tile are issued
  // before the threshold / bucket work of the previous one, so a wave keeps
  // its matrix core busy while its VALU works.  Stages hold an even number
  // of tiles, so a stage boundary always falls between pairs.
  constexpr int TPS = S::ST / 32;                  // tiles per stage
  static_assert(TPS % 2 == 0, "stages hold whole tile pairs");
  const int ntiles = nstages * TPS;               // includes masked tail tiles
  auto mma = [&](int j, f32x16_t(&acc)[S::NB]) {
    const unsigned char* xs = sX + ((j / TPS) % kRing) * S::STAGE_BYTES;
    const int n = 32 * (j % TPS) + col;             // A-operand row = item
    const unsigned char* rowp = xs + n * (2 * D);
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) acc[nb] = f32x16_t{};
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk) {
      const uint4 xa = *reinterpret_cast<const uint4*>(rowp + 16 * ((2 * kk + half) ^ S::swz(n)));
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb) acc[nb] = mfma32_bf16(xa, qop[nb][kk], acc[nb]);
    }
  };
  // Threshold / bucket work of tile j.  RAGGED: the tile may reach past the
  // range end (items there become -inf and are never staged).
  int bcount = 0, bk = 0;                         // bucket scan: tiles in the open bucket, its index
  uint32_t hitc = 0u;                             // pruned pass: LDS slots used, 8 bits per block
  // bucket scan: close bucket b of every block: the two lanes of a list
  // (items 4h .. 4h + 3 of every 8) join their maxima, half 0 stores
  auto store_buckets = [&](int b) {
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      const uint32_t u = __float_as_uint(bm[nb]);
      auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
      const float mm = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      if (vok[nb] && half == 0 && b < nbk) bucket_row[static_cast<long>(b) * nvec + vv[nb]] = mm;
      bm[nb] = -__builtin_inff();
    }
  };
  auto process = [&](auto ragged_tag, int j, f32x16_t(&acc)[S::NB]) {
    constexpr bool RAGGED = decltype(ragged_tag)::value;
    const int n0 = nr0 + 32 * j;                    // first item of the tile
    // lane (c, h) register v holds item n0 + (v/4)*8 + 4h + v%4 of list c
    uint32_t vmask = 0xFFFFu;
    if constexpr (RAGGED) {
      vmask = 0u;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const bool ok = n0 + (v >> 2) * 8 + 4 * half + (v & 3) < nr1;
        vmask |= ok ? (1u << v) : 0u;
#pragma unroll
        for (int nb = 0; nb < S::NB; ++nb) acc[nb][v] = ok ? acc[nb][v] : -__builtin_inff();
      }
    }
    float m[S::NB];
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      float a0 = fmaxf(fmaxf(acc[nb][0], acc[nb][1]), acc[nb][2]);
      float a1 = fmaxf(fmaxf(acc[nb][3], acc[nb][4]), acc[nb][5]);
      float a2 = fmaxf(fmaxf(acc[nb][6], acc[nb][7]), acc[nb][8]);
      float a3 = fmaxf(fmaxf(acc[nb][9], acc[nb][10]), acc[nb][11]);
      float a4 = fmaxf(fmaxf(acc[nb][12], acc[nb][13]), acc[nb][14]);
      m[nb] = fmaxf(fmaxf(fmaxf(a0, a1), a2), fmaxf(fmaxf(a3, a4), acc[nb][15]));
    }
    if constexpr (MODE == kScanBuckets) {
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb) bm[nb] = fmaxf(bm[nb], m[nb]);
      if (++bcount == bucket_tiles) {
        store_buckets(bk);
        bcount = 0;
        ++bk;
      }
      return;
    }
    if constexpr (PRUNED) {
      bool hit = false;
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb) hit = hit || m[nb] >= th[nb];
      if (__ballot(hit) == 0ull) return;
      // keys reaching the list's threshold go to the lane's LDS slots (the
      // item's end appends them with one atomic per lane); beyond the slots,
      // straight to the list's key buffer
      // a block is entered when one of its lanes reaches the threshold
      // (most blocks: about 5 lanes of a wave's 256 hit per tile); inside,
      // each group of three values is tested on its maximum first, so the
      // per-value tests run only in the groups that hold a hit
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb) {
        if (m[nb] >= th[nb]) {
#pragma unroll
          for (int g3 = 0; g3 < 6; ++g3) {
            const int v0 = 3 * g3, v1 = g3 < 5 ? v0 + 3 : 16;
            const float gmax = g3 < 5 ? fmaxf(fmaxf(acc[nb][v0], acc[nb][v0 + 1]), acc[nb][v0 + 2]) : acc[nb][15];
            if (gmax < th[nb]) continue;
#pragma unroll
            for (int v = v0; v < v1; ++v) {
              if (acc[nb][v] >= th[nb] && ((vmask >> v) & 1u)) {
                const int item = n0 + (v >> 2) * 8 + 4 * half + (v & 3);
                const uint64_t key = make_key(acc[nb][v], item);
                const int used = (hitc >> (8 * nb)) & 0xFF;
                if (used < kHitSlots) {
                  sHit[((wave * S::NB + nb) * kHitSlots + used) * 64 + lane] = key;
                  hitc += 1u << (8 * nb);
                } else {
                  const long list = static_cast<long>(vv[nb]) * Px + px;
                  const uint32_t slot = atomicAdd(pa.cnt + list, 1u);
                  if (slot < static_cast<uint32_t>(pa.cap)) pa.keys[list * pa.cap + slot] = key;
                  else *pa.flag = 1u;
                }
              }
            }
          }
        }
      }
      return;
    }
    bool hit = false;
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) hit = hit || m[nb] >= th[nb];
    if (__ballot(hit) == 0ull) return;
    // append survivors to the lane's own staging region (groups of three
    // values tested on their maximum first, as in the pruned pass)
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      if (m[nb] >= th[nb]) {
        uint64_t* sp = stg_ptr(nb, col, half);
#pragma unroll
        for (int g3 = 0; g3 < 6; ++g3) {
          const int v0 = 3 * g3, v1 = g3 < 5 ? v0 + 3 : 16;
          const float gmax = g3 < 5 ? fmaxf(fmaxf(acc[nb][v0], acc[nb][v0 + 1]), acc[nb][v0 + 2]) : acc[nb][15];
          if (gmax < th[nb]) continue;
#pragma unroll
          for (int v = v0; v < v1; ++v) {
            if (acc[nb][v] >= th[nb] && ((vmask >> v) & 1u)) {
              const int item = n0 + (v >> 2) * 8 + 4 * half + (v & 3);
              sp[cnt[nb]] = make_key(acc[nb][v], item);
              ++cnt[nb];
            }
          }
        }
      }
    }
    // merge lists whose staging could overflow on the next tile
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      uint64_t need = __ballot(cnt[nb] > S::SG - 16);
      while (need) {
        const int c = __builtin_ctzll(need) & 31;
        need &= ~((1ull << c) | (1ull << (c + 32)));
        merge(nb, c);
      }
    }
  };
  using Full = std::false_type;
  using Ragged = std::true_type;
  // end of stage t: refill the buffer of stage t-1 (every wave finished
  // reading it before the barrier that ended stage t-1), then wait for
  // stage t+1
  auto stage_end = [&](int t) {
    if (t + kRing - 1 < nstages) {
      stage(t + kRing - 1, (t + kRing - 1) % kRing);
      ring_barrier<(kRing - 2) * S::LOADS>();
    } else if (t + kRing - 2 < nstages) {
      ring_barrier<(kRing - 3) * S::LOADS>();   // stages t+2 .. end are in flight
    } else {
      ring_barrier<0>();
    }
  };

  // Main loop over tile pairs whose tiles (and the next one) hold items
  // only: the MFMAs of tile j+1 (j+2) are issued next to the threshold work
  // of tile j (j+1) in one basic block.  The tail (last pair, ragged tiles,
  // masked tiles of the last stage) runs unpipelined.
  f32x16_t accA[S::NB], accB[S::NB];
  const int nfull = (nr1 - nr0) / 32;             // tiles holding items only
  int j = 0;
  // every global load issued so far (thresholds, query operands) completes
  // here, once: the loop's first use of a threshold would otherwise carry a
  // compiler-inserted vmcnt(0), executed on every iteration, that also waits
  // for the LDS ring's prefetch copies
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  if (ntiles > 0) mma(0, accA);
  for (; j + 2 < nfull; j += 2) {
    mma(j + 1, accB);
    process(Full{}, j, accA);
    if ((j + 2) % TPS == 0) stage_end((j + 2) / TPS - 1);
    mma(j + 2, accA);
    process(Full{}, j + 1, accB);
  }
  if (ntiles > 0) {
    process(Ragged{}, j, accA);                   // tile j, computed above
    for (++j; j < ntiles; ++j) {
      if (j % TPS == 0) stage_end(j / TPS - 1);
      mma(j, accA);
      process(Ragged{}, j, accA);
    }
  }
  if constexpr (MODE == kScanBuckets) {
    // the last partial bucket, then -inf for buckets past the range end
    int b = bk;
    if (bcount != 0) store_buckets(b++);
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      if (!vok[nb] || half != 0) continue;
      for (int bb = b; bb < nbk; ++bb) bucket_row[static_cast<long>(bb) * nvec + vv[nb]] = -__builtin_inff();
    }
    return;
  }
  if constexpr (PRUNED) {
    // append the staged keys: one atomic per lane and block reserves them
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      const int used = (hitc >> (8 * nb)) & 0xFF;
      if (used > 0) {
        const long list = static_cast<long>(vv[nb]) * Px + px;
        const uint32_t base = atomicAdd(pa.cnt + list, static_cast<uint32_t>(used));
        for (int i = 0; i < used; ++i) {
          const uint32_t slot = base + i;
          const uint64_t key = sHit[((wave * S::NB + nb) * kHitSlots + i) * 64 + lane];
          if (slot < static_cast<uint32_t>(pa.cap)) pa.keys[list * pa.cap + slot] = key;
          else *pa.flag = 1u;
        }
      }
    }
    return;
  }
  // staged keys of lists never merged into go straight into the (empty)
  // list when they fit; the others are merged
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent");
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    const int other = __shfl_xor(cnt[nb], 32);
    const int c0 = half == 0 ? cnt[nb] : other;
    const int c1 = half == 0 ? other : cnt[nb];
    if (vok[nb] && !merged[nb] && c0 + c1 <= KL) {
      uint64_t* lp = lists + list_idx(nb, col) * KL + (half == 0 ? 0 : c0);
      const uint64_t* sp = stg_ptr(nb, col, half);
      for (int i = 0; i < cnt[nb]; ++i) lp[i] = sp[i];
      cnt[nb] = 0;
    }
  }
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    uint64_t need = __ballot(cnt[nb] > 0);
    while (need) {
      const int c = __builtin_ctzll(need) & 31;
      need &= ~((1ull << c) | (1ull << (c + 32)));
      merge(nb, c);
    }
  }
  };  // run
  if constexpr (PRUNED) {
    // persistent workgroups over the work list; every wave sees the same
    // length and leaves the loop together.  The barrier after each item
    // keeps the next item's LDS copies from overwriting a stage that a
    // slower wave still reads.
    const int total = static_cast<int>(*pa.work_total);
    for (int wi = blockIdx.x; wi < total; wi += gridDim.x) {
      run(wi);
      ring_barrier<0>();
    }
  } else {
    run(blockIdx.x);
  }
}

// k'-th largest bucket maximum of every list: the starting threshold T of
// the second pass.  A workgroup of kThrLists waves takes kThrLists
// consecutive query vectors of one component: their bucket maxima
// ([Px][R][nbk][nvec], so one (range, bucket) row of the block is
// kThrLists contiguous floats) are read coalesced and transposed through
// LDS to one row of per_list + 1 floats per list (an odd stride: a row's
// transposing stores hit distinct banks); then each wave runs a bitwise
// search over the order-preserving 32-bit images of its list's maxima
// (VPL per lane).  Fewer than k' finite maxima give -inf (no filtering).
constexpr int kThrLists = 16;
constexpr int kThrBits = 20;                 // bits the threshold search resolves
template <int VPL>
__global__ __launch_bounds__(64 * kThrLists) void k_bucket_threshold(const float* __restrict__ bmax, int nvec,
                                                                    int Px, int per_list, int kp,
                                                                    float* __restrict__ thr,
                                                                    float* __restrict__ thr_t) {
  extern __shared__ float sm[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nblk = (nvec + kThrLists - 1) / kThrLists;
  const int px = blockIdx.x / nblk, v0 = (blockIdx.x % nblk) * kThrLists;
  const int row_stride = per_list + 1;
  const float* base = bmax + static_cast<long>(px) * per_list * nvec + v0;
  const int nvalid = min(kThrLists, nvec - v0);
  // thread (row r, quarter q): lists 4q .. 4q + 3 of row r as one 16-byte
  // load when the block is whole and aligned, four loads in flight
  constexpr int kRowsPerPass = 64 * kThrLists / 4;
  const int q = tid & 3;
  const bool vec = nvalid == kThrLists && (nvec & 3) == 0;
  for (int r0 = tid >> 2; r0 < per_list; r0 += 4 * kRowsPerPass) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = r0 + u * kRowsPerPass;
      const float* src = base + static_cast<long>(min(row, per_list - 1)) * nvec + 4 * q;
      if (vec) {
        v[u] = *reinterpret_cast<const float4*>(src);
      } else {
        const float ninf = -__builtin_inff();
        v[u] = make_float4(4 * q + 0 < nvalid ? src[0] : ninf, 4 * q + 1 < nvalid ? src[1] : ninf,
                           4 * q + 2 < nvalid ? src[2] : ninf, 4 * q + 3 < nvalid ? src[3] : ninf);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = r0 + u * kRowsPerPass;
      if (row < per_list) {
        sm[(4 * q + 0) * row_stride + row] = v[u].x;
        sm[(4 * q + 1) * row_stride + row] = v[u].y;
        sm[(4 * q + 2) * row_stride + row] = v[u].z;
        sm[(4 * q + 3) * row_stride + row] = v[u].w;
      }
    }
  }
  __syncthreads();
  const int v = v0 + wave;
  if (v >= nvec) return;                       // wave-uniform
  const float* row = sm + wave * row_stride;
  uint32_t val[VPL];
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int i = lane + 64 * j;
    val[j] = i < per_list ? float_to_ordered(row[i]) : 0u;
  }
  // With at least k' finite maxima the k'-th largest image K lies between
  // the smallest finite image lo and the largest hi, so it shares their bits
  // above the highest bit where they differ; the search resolves kThrBits
  // bits from there down.  Any t <= K is a valid threshold: the bits left
  // zero only lower it, by under 2^-(kThrBits - 9) relative.  Fewer than k'
  // finite maxima: no filtering.
  const uint32_t ninf = float_to_ordered(-__builtin_inff());
  uint32_t hi = 0u, lo = 0xFFFFFFFFu;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    hi = max(hi, val[j]);
    lo = val[j] > ninf ? min(lo, val[j]) : lo;
  }
  for (int sh = 1; sh < 64; sh <<= 1) {
    hi = max(hi, static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), sh)));
    lo = min(lo, static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), sh)));
  }
  int nfin = 0;
#pragma unroll
  for (int j = 0; j < VPL; ++j) nfin += __popcll(__ballot(val[j] > ninf));
  uint32_t t = 0u;
  if (nfin >= kp) {
    const uint32_t diff = hi ^ lo;
    const int top = diff ? 31 - __clz(static_cast<int>(diff)) : -1;
    t = top >= 0 ? hi & ~((top == 31 ? 0u : 2u << top) - 1u) : hi;
    for (int bit = top; bit >= 0 && bit > top - kThrBits; --bit) {
      const uint32_t c = t | (1u << bit);
      int n = 0;
#pragma unroll
      for (int j = 0; j < VPL; ++j) n += __popcll(__ballot(val[j] >= c));
      if (n >= kp) t = c;
    }
  }
  // t is at most the k'-th largest image; images below that of -inf mean "none"
  const float f = t >= ninf ? ordered_to_float(t) : -__builtin_inff();
  if (lane == 0) {
    thr[static_cast<long>(v) * Px + px] = f;
    thr_t[static_cast<long>(px) * nvec + v] = f;
  }
}

// T lowered by a few units in the last place: the pruned pass's threshold
// (a bucket is hot when its maximum reaches twice the lowering below T)
__device__ __forceinline__ float lowered(float t, float times) {
  return t - times * 0x1p-20f * fmaxf(1.f, fabsf(t));
}

// Work list of the pruned pass.  One workgroup per bucket group g = (px,
// range, bucket): the query vectors whose lists have this bucket hot
// (maximum at least T, lowered) are compacted into hot_v[g], and the group's
// ceil(count / vec_wg) chunks are appended to the work list.
__global__ __launch_bounds__(256) void k_pe_hot(const float* __restrict__ bmax, const float* __restrict__ thr_t,
                                               int nvec, int per_list, int vec_wg, int CH,
                                               int* __restrict__ hot_v, int* __restrict__ hot_n,
                                               int* __restrict__ work, uint32_t* __restrict__ work_total) {
  __shared__ int s_cnt[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const long g = blockIdx.x;
  const int px = static_cast<int>(g / per_list);
  const float* row = bmax + g * nvec;
  const float* tp = thr_t + static_cast<long>(px) * nvec;
  int* out = hot_v + g * nvec;
  int base = 0;
  for (int v0 = 0; v0 < nvec; v0 += 256) {
    const int v = v0 + tid;
    bool hot = false;
    if (v < nvec) hot = row[v] >= lowered(tp[v], 2.f);
    const uint64_t m = __ballot(hot);
    if (lane == 0) s_cnt[wave] = __popcll(m);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += s_cnt[w];
    const int tot = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    if (hot) out[off + __popcll(m & ((1ull << lane) - 1ull))] = v;
    base += tot;
    __syncthreads();
  }
  if (tid == 0) {
    hot_n[g] = base;
    const int chunks = (base + vec_wg - 1) / vec_wg;
    if (chunks > 0) {
      const uint32_t at = atomicAdd(work_total, static_cast<uint32_t>(chunks));
      for (int c = 0; c < chunks; ++c) work[at + c] = static_cast<int>(g) * CH + c;
    }
  }
}

// Final selection of the pruned pass, one wave per list: the list's keys
// (count at most cap) sorted in LDS, the first k' decoded into the outputs.
// Lists with more keys than cap are left to the threshold-scan path (the
// device flag is then set and that path rewrites every list).
template <int SORT>
__global__ __launch_bounds__(256) void k_pe_select(const uint32_t* __restrict__ cnt, const uint64_t* __restrict__ keys,
                                                  int cap, int rows, int kp, float* __restrict__ out_dot,
                                                  int32_t* __restrict__ out_idx) {
  __shared__ uint64_t sk[4][SORT];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long row = static_cast<long>(blockIdx.x) * 4 + wave;
  if (row >= rows) return;                     // wave-uniform; the sort syncs only the wave
  const uint32_t n = cnt[row];
  if (n > static_cast<uint32_t>(cap)) return;
  const uint64_t* src = keys + row * cap;
  for (int i = lane; i < SORT; i += 64) sk[wave][i] = i < static_cast<int>(n) ? src[i] : 0ull;
  wave_lds_sync();
  wave_sort<SORT>((lds_u64_t*)sk[wave], lane);
  for (int i = lane; i < kp; i += 64) {
    const uint64_t key = sk[wave][i];
    out_dot[row * kp + i] = key_score(key);
    out_idx[row * kp + i] = key_item(key);
  }
}

// ---------------------------------------------------------------------------
// small-batch form (one 32-vector block per wave): lists of up to 256 keys
bool per_embd_small(const DevProb& pr, int kp) {
  return pr.B * pr.Pq <= kSmallVectors && per_embd_list_cap(kp) <= 256;
}

bool per_embd_supported(const DevProb& pr, int kp) {
  if (pr.dtype != MOL_BF16) return false;
  if (pr.d != 32 && pr.d != 64 && pr.d != 128) return false;
  return kp <= 1024;
}

int per_embd_list_cap(int kp) { return kp <= 128 ? 128 : kp <= 256 ? 256 : kp <= 512 ? 512 : 1024; }
int per_embd_stage_cap(int kp) {
  // 2 SG of the list capacity's merge sort: SORT - KL
  const int kl = per_embd_list_cap(kp);
  return (kl <= 256 ? 512 : 2 * kl) - kl;
}

// items of one LDS stage (EmbdShape::ST) for width d and list capacity kl
static int stage_items(int d, int kl) { return (waves_for(kl) == 8 ? 32768 : 16384) / (2 * d); }

static void scan_grid(const DevProb& pr, int kp, bool scan2, PerEmbdGrid::Scan& sc) {
  const int nvec = pr.B * pr.Pq;
  const int vec_wg = waves_for(per_embd_list_cap(kp)) * 32 * nb_pick(pr.d, scan2, per_embd_small(pr, kp));
  sc.G = (nvec + vec_wg - 1) / vec_wg;
  const int units = sc.G * pr.Px;
  // about one workgroup per CU, with ranges of at least 512 items
  int R = std::max(1, (256 + units - 1) / units);
  R = std::min(R, std::max(1, pr.N / 512));
  // whole stages per range: a range's tile walk then covers exactly
  // range_len / 32 tiles, the count the bucket layout is sized for
  const int unit = std::max(128, stage_items(pr.d, per_embd_list_cap(kp)));
  sc.range_len = (pr.N + R - 1) / R;
  sc.range_len = (sc.range_len + unit - 1) / unit * unit;
  sc.R = (pr.N + sc.range_len - 1) / sc.range_len;
}

void per_embd_grid(const DevProb& pr, int kp, PerEmbdGrid& g) {
  scan_grid(pr, kp, false, g.s1);
  scan_grid(pr, kp, true, g.s2);
  const int KL = per_embd_list_cap(kp);
  const int nvec = pr.B * pr.Pq;
  const int ntiles = g.s1.range_len / 32;
  const int tps = stage_items(pr.d, KL) / 32;
  g.vec_wg_pruned = waves_for(KL) * 32 * nb_pick(pr.d, false, false);
  g.CH = (nvec + g.vec_wg_pruned - 1) / g.vec_wg_pruned;
  g.key_cap = 2 * KL;
  // buckets per list.  The full-scan form: 1024 for k' <= 128 (about
  // k'^2 / 2048 <= 8 collisions among the k' largest items, so the bound
  // admits few more keys than 2048 would, at half the maxima stored and
  // searched), else 2048.  The pruned form: about k' + k'^2 / (2 B) of the
  // B buckets of a list are hot, so a bucket is hot for about nvec k' / B
  // vectors; B is chosen so that this fills 80 % of a workgroup's vector
  // slots (partly filled second chunks would cost a full pass), and at
  // least 4 k' buckets keep the pass at a quarter of a full scan or less.
  const bool can_prune = KL <= 256 && !per_embd_small(pr, kp);
  int target = kp <= 128 ? kMaxBuckets / 2 : kMaxBuckets;
  if (can_prune) {
    const long want = (5l * nvec * kp + 4l * g.vec_wg_pruned - 1) / (4l * g.vec_wg_pruned);
    target = static_cast<int>(std::min<long>(kMaxBuckets, std::max<long>(4l * kp, want)));
  }
  // buckets of whole LDS stages where they are at least one stage long
  // (rounded down: more buckets), so a work unit of the pruned pass starts
  // on a stage and walks no masked tiles
  g.bucket_tiles = std::max(1, (g.s1.R * ntiles + target - 1) / target);
  if (g.bucket_tiles >= tps) g.bucket_tiles = g.bucket_tiles / tps * tps;
  g.nbk = (ntiles + g.bucket_tiles - 1) / g.bucket_tiles;
  while (g.s1.R * g.nbk > kMaxBuckets) {
    g.bucket_tiles += g.bucket_tiles >= tps ? tps : 1;
    g.nbk = (ntiles + g.bucket_tiles - 1) / g.bucket_tiles;
  }
  g.pruned = can_prune && g.s1.R * g.nbk >= 4 * kp;
  g.groups = pr.Px * g.s1.R * g.nbk;
}

// compute units of the current device (the pruned pass runs one persistent
// workgroup per CU: 8 waves of up to 256 registers fill its four SIMDs)
static int resident_cus() {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
    ncu = 256;
  return ncu;
}

template <int D, int KL, int MODE, bool SMALL>
static hipError_t launch_pe_t(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b,
                              const uint32_t* gate, hipStream_t st) {
  using S = EmbdShape<D, KL, MODE == kScanThreshold, SMALL, MODE == kScanPruned>;
  const PerEmbdGrid::Scan& sc = MODE == kScanThreshold ? g.s2 : g.s1;
  auto kern = &k_topk_per_embd<D, KL, MODE, SMALL>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS_TOTAL);
  if (e != hipSuccess) return e;
  PrunedArgs pa;
  int grid = sc.G * pr.Px * sc.R;
  if (MODE == kScanPruned) {
    const int rows = pr.B * pr.Pq * pr.Px;
    pa.work = b.work;
    pa.work_total = b.ctl + rows + 1;
    pa.hot_v = b.hot_v;
    pa.hot_n = b.hot_n;
    pa.cnt = b.ctl;
    pa.keys = b.keys;
    pa.flag = b.ctl + rows;
    pa.cap = g.key_cap;
    pa.CH = g.CH;
    grid = std::min<long>(static_cast<long>(g.groups) * g.CH, resident_cus());   // persistent, one per CU
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * S::WAVES), S::LDS_TOTAL, st, pr, kp, sc.R, sc.range_len, sc.G,
                     g.bucket_tiles, g.nbk, b.bmax, b.thr, b.lists, b.stg, gate, pa);
  return hipGetLastError();
}

template <int D, int KL, bool SMALL>
static hipError_t launch_pe_s(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b,
                              hipStream_t st) {
  const int nvec = pr.B * pr.Pq, rows = nvec * pr.Px;
  hipError_t e;
  if (g.pruned) {
    // per-list key counts, the overflow flag and the work-list length start at zero
    e = launch_fill(reinterpret_cast<uint64_t*>(b.ctl), (rows + 2 + 1) / 2, 0ull, st);
    if (e != hipSuccess) return e;
  }
  e = launch_pe_t<D, KL, kScanBuckets, SMALL>(pr, kp, g, b, nullptr, st);
  if (e != hipSuccess) return e;
  const int nblk = (nvec + kThrLists - 1) / kThrLists;
  const int per_list = g.s1.R * g.nbk;
  const int lds = kThrLists * (per_list + 1) * 4;
  auto thr_kern = per_list <= 1024 ? &k_bucket_threshold<16>
                  : per_list <= 1536 ? &k_bucket_threshold<24> : &k_bucket_threshold<32>;
  static_assert(kMaxBuckets <= 32 * 64, "bucket maxima per list beyond the search's registers");
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(thr_kern), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(thr_kern, dim3(nblk * pr.Px), dim3(64 * kThrLists), lds, st, b.bmax, nvec, pr.Px, per_list, kp,
                     b.thr, b.thr_t);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if constexpr (KL <= 256 && !SMALL) {
    if (g.pruned) {
      hipLaunchKernelGGL(k_pe_hot, dim3(g.groups), dim3(256), 0, st, b.bmax, b.thr_t, nvec, per_list,
                         g.vec_wg_pruned, g.CH, b.hot_v, b.hot_n, b.work, b.ctl + rows + 1);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      e = launch_pe_t<D, KL, kScanPruned, false>(pr, kp, g, b, nullptr, st);
      if (e != hipSuccess) return e;
      // the threshold scan only where some list overflowed its key buffer
      return launch_pe_t<D, KL, kScanThreshold, false>(pr, kp, g, b, b.ctl + rows, st);
    }
  }
  return launch_pe_t<D, KL, kScanThreshold, SMALL>(pr, kp, g, b, nullptr, st);
}

template <int D, int KL>
static hipError_t launch_pe_d(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b,
                              hipStream_t st) {
  if constexpr (KL <= 256) {
    if (per_embd_small(pr, kp)) return launch_pe_s<D, KL, true>(pr, kp, g, b, st);
  }
  return launch_pe_s<D, KL, false>(pr, kp, g, b, st);
}

hipError_t launch_per_embd(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b, hipStream_t st) {
  const int KL = per_embd_list_cap(kp);
  if (pr.d == 32) {
    switch (KL) {
      case 128: return launch_pe_d<32, 128>(pr, kp, g, b, st);
      case 256: return launch_pe_d<32, 256>(pr, kp, g, b, st);
      case 512: return launch_pe_d<32, 512>(pr, kp, g, b, st);
      default: return launch_pe_d<32, 1024>(pr, kp, g, b, st);
    }
  }
  if (pr.d == 64) {
    switch (KL) {
      case 128: return launch_pe_d<64, 128>(pr, kp, g, b, st);
      case 256: return launch_pe_d<64, 256>(pr, kp, g, b, st);
      case 512: return launch_pe_d<64, 512>(pr, kp, g, b, st);
      default: return launch_pe_d<64, 1024>(pr, kp, g, b, st);
    }
  }
  switch (KL) {
    case 128: return launch_pe_d<128, 128>(pr, kp, g, b, st);
    case 256: return launch_pe_d<128, 256>(pr, kp, g, b, st);
    case 512: return launch_pe_d<128, 512>(pr, kp, g, b, st);
    default: return launch_pe_d<128, 1024>(pr, kp, g, b, st);
  }
}

hipError_t launch_per_embd_select(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b,
                                  float* out_dot, int32_t* out_idx, hipStream_t st) {
  const int rows = pr.B * pr.Pq * pr.Px;
  if (g.key_cap <= 256)
    hipLaunchKernelGGL(k_pe_select<256>, dim3((rows + 3) / 4), dim3(256), 0, st, b.ctl, b.keys, g.key_cap, rows, kp,
                       out_dot, out_idx);
  else
    hipLaunchKernelGGL(k_pe_select<512>, dim3((rows + 3) / 4), dim3(256), 0, st, b.ctl, b.keys, g.key_cap, rows, kp,
                       out_dot, out_idx);
  return hipGetLastError();
}

}  // namespace mol
