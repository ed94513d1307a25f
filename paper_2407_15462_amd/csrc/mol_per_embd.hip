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
// Two scans of the same dot products:
//  1. every lane keeps the maximum of its scores over buckets of
//     `bucket_tiles` tiles and stores the bucket maxima;
//  2. the k'-th largest bucket maximum of a list is a lower bound of the
//     list's k'-th largest score (k' disjoint buckets each hold an item at
//     least that large), so the second scan starts every list at that
//     threshold.  Scores that reach the threshold are appended to the
//     lane's staging region in the workspace; a full staging region is
//     merged into the list by a wave-wide bitonic sort in LDS, and the
//     threshold rises to the list's k'-th key.
// Both scans evaluate bit-identical dot products (same instructions, same
// accumulation order), so the bound is exact.  Lists of several item ranges
// are merged afterwards by segmented sorts.
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
constexpr int kRing = 3;                     // item stages in flight
constexpr int kSGMax = 512;                  // largest staging region per lane half
constexpr int kMaxBuckets = 2048;            // bucket maxima per list (all ranges, both halves)

__device__ __forceinline__ f32x16_t mfma32_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

template <int D, int KL, bool SCAN2, bool SMALL>
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
  static constexpr int LDS_SORT = WAVES * SORT * 8;
  static constexpr int LDS_TOTAL = LDS_X + LDS_SORT;
  static_assert(ST % 32 == 0, "stage holds whole 32-item tiles");
  static_assert(KL + 2 * SG <= SORT && SG <= kSGMax, "sort region holds list + both staging halves");
  static_assert(LDS_TOTAL <= 160 * 1024, "LDS budget");
};

}  // namespace

// Grid: WG -> (vector group, px, range).  WGs sharing (px, range) are placed
// on the same XCD (WG id mod 8) when the grid allows it.
// R, range_len, G: this scan's item ranges and query-vector groups.
// bmax: [Px][R][nbk][nvec][2] bucket maxima (scan 1 writes, scan 2 unused):
//   for one (component, range, bucket) the two lanes of every list are
//   adjacent and the lists contiguous, so a wave's store covers one line;
// thr: [nvec * Px] starting thresholds (scan 2 reads);
// lists: [nvec * Px][R][KL] keys; stg: [nvec * Px][R][2][SG] keys (scan 2).
template <int D, int KL, bool SCAN2, bool SMALL>
__global__ __launch_bounds__(64 * waves_for(KL), 1) void k_topk_per_embd(
    DevProb pr, int kp, int R, int range_len, int G, int bucket_tiles, int nbk,
    float* __restrict__ bmax, const float* __restrict__ thr, uint64_t* __restrict__ lists,
    uint64_t* __restrict__ stg) {
  using S = EmbdShape<D, KL, SCAN2, SMALL>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  uint64_t* sSort = reinterpret_cast<uint64_t*>(smem + S::LDS_X);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int col = lane & 31, half = lane >> 5;
  const int Px = pr.Px, N = pr.N;
  const int nvec = pr.B * pr.Pq;               // query vectors
  const int total = gridDim.x;
  int L = blockIdx.x;
  if (total % 8 == 0) L = (blockIdx.x >> 3) + (total >> 3) * (blockIdx.x & 7);
  const int rg = L % G, unit = L / G;
  const int px = unit % Px, r = unit / Px;
  const int vwave = rg * S::VEC_WG + wave * S::VEC_WAVE;   // first query vector of the wave
  const int nr0 = r * range_len, nr1 = min(N, nr0 + range_len);
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

  // query vectors as B operands: column = lane % 32 within each block
  uint4 qop[S::NB][S::KD];
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
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
  // per-lane state.  Scan 1: running bucket maximum.  Scan 2: threshold
  // (float score every appended key reaches), staging count, and whether the
  // list has been merged into (it is empty otherwise).
  bool vok[S::NB];
  float th[S::NB], bm[S::NB];
  int cnt[S::NB];
  bool merged[S::NB];
#pragma unroll
  for (int nb = 0; nb < S::NB; ++nb) {
    vok[nb] = vwave + 32 * nb + col < nvec;
    bm[nb] = -__builtin_inff();
    cnt[nb] = 0;
    merged[nb] = false;
    th[nb] = __builtin_inff();                      // invalid vectors never pass
    if (SCAN2 && vok[nb]) {
      th[nb] = thr[static_cast<long>(vwave + 32 * nb + col) * Px + px];
      if (half == 0) {
        uint64_t* lp = lists + list_idx(nb, col) * KL;
        for (int i = 0; i < KL; ++i) lp[i] = 0ull;
      }
    }
  }
  // bucket bk of the lane's list in block nb: bucket_ptr(nb)[bk * nv2]
  const long nv2 = 2l * nvec;
  auto bucket_ptr = [&](int nb) {
    return bmax + (static_cast<long>(px) * R + r) * nbk * nv2 + 2l * (vwave + 32 * nb + col) + half;
  };
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
  int bcount = 0, bk = 0;                         // scan 1: tiles in the open bucket, its index
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
    if constexpr (!SCAN2) {
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb) bm[nb] = fmaxf(bm[nb], m[nb]);
      if (++bcount == bucket_tiles) {
#pragma unroll
        for (int nb = 0; nb < S::NB; ++nb) {
          if (vok[nb] && bk < nbk) bucket_ptr(nb)[bk * nv2] = bm[nb];
          bm[nb] = -__builtin_inff();
        }
        bcount = 0;
        ++bk;
      }
      return;
    }
    bool hit = false;
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) hit = hit || m[nb] >= th[nb];
    if (__ballot(hit) == 0ull) return;
    // append survivors to the lane's own staging region
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      if (m[nb] >= th[nb]) {
        uint64_t* sp = stg_ptr(nb, col, half);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (acc[nb][v] >= th[nb] && ((vmask >> v) & 1u)) {
            const int item = n0 + (v >> 2) * 8 + 4 * half + (v & 3);
            sp[cnt[nb]] = make_key(acc[nb][v], item);
            ++cnt[nb];
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
  if (!SCAN2) {
    // the last partial bucket, then -inf for buckets past the range end
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) {
      if (!vok[nb]) continue;
      float* bp = bucket_ptr(nb);
      int b = bk;
      if (bcount != 0 && b < nbk) bp[b++ * nv2] = bm[nb];
      for (; b < nbk; ++b) bp[b * nv2] = -__builtin_inff();
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
}

// k'-th largest bucket maximum of every list: the starting threshold of the
// second scan.  A workgroup of kThrLists waves takes kThrLists consecutive
// query vectors of one component: their bucket maxima ([Px][R][nbk][nvec][2],
// so one (range, bucket) row of the block is 2 kThrLists contiguous floats)
// are read coalesced and transposed through LDS to one row of per_list + 1
// floats per list (an odd stride: a row's transposing stores hit distinct
// banks); then each wave runs a bitwise search over the order-preserving
// 32-bit images of its list's VPL * 64 maxima.  Fewer than k' finite maxima
// give -inf (no filtering).
constexpr int kThrLists = 16;
template <int VPL>
__global__ __launch_bounds__(64 * kThrLists) void k_bucket_threshold(const float* __restrict__ bmax, int nvec,
                                                                    int Px, int rows, int kp,
                                                                    float* __restrict__ thr) {
  extern __shared__ float sm[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nblk = (nvec + kThrLists - 1) / kThrLists;
  const int px = blockIdx.x / nblk, v0 = (blockIdx.x % nblk) * kThrLists;
  const int per_list = 2 * rows;               // maxima per list: rows x 2 lanes
  const int row_stride = per_list + 1;
  const long nv2 = 2l * nvec;
  const float* base = bmax + static_cast<long>(px) * rows * nv2 + 2l * v0;
  // element e of a block row: list v0 + e / 2, lane half e % 2
  constexpr int kRowElems = 2 * kThrLists;
  const int nvalid = 2 * min(kThrLists, nvec - v0);
  for (int i = tid; i < rows * kRowElems; i += 64 * kThrLists) {
    const int row = i / kRowElems, e = i % kRowElems;
    const float v = e < nvalid ? base[row * nv2 + e] : -__builtin_inff();
    sm[(e >> 1) * row_stride + 2 * row + (e & 1)] = v;
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
  uint32_t t = 0u;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    int n = 0;
#pragma unroll
    for (int j = 0; j < VPL; ++j) n += __popcll(__ballot(val[j] >= c));
    if (n >= kp) t = c;
  }
  // t is the k'-th largest image; images below that of -inf mean "none"
  const float f = t >= float_to_ordered(-__builtin_inff()) ? ordered_to_float(t) : -__builtin_inff();
  if (lane == 0) thr[static_cast<long>(v) * Px + px] = f;
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
  // buckets: as many as fit `cap` per list over all ranges and halves.  For
  // k' <= 128, 1024 buckets leave about k'^2 / 2048 <= 8 collisions among
  // the k' largest items, so the bound admits few more keys than 2048 do,
  // while the bucket scan stores and the threshold kernel reads half as
  // many maxima
  const int cap = kp <= 128 ? kMaxBuckets / 2 : kMaxBuckets;
  const int ntiles = g.s1.range_len / 32;
  g.bucket_tiles = std::max(1, (2 * g.s1.R * ntiles + cap - 1) / cap);
  g.nbk = (ntiles + g.bucket_tiles - 1) / g.bucket_tiles;
  while (2 * g.s1.R * g.nbk > cap) {
    ++g.bucket_tiles;
    g.nbk = (ntiles + g.bucket_tiles - 1) / g.bucket_tiles;
  }
}

template <int D, int KL, bool SCAN2, bool SMALL>
static hipError_t launch_pe_t(const DevProb& pr, int kp, const PerEmbdGrid& g, float* bmax, const float* thr,
                              uint64_t* lists, uint64_t* stg, hipStream_t st) {
  using S = EmbdShape<D, KL, SCAN2, SMALL>;
  const PerEmbdGrid::Scan& sc = SCAN2 ? g.s2 : g.s1;
  auto kern = &k_topk_per_embd<D, KL, SCAN2, SMALL>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS_TOTAL);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(sc.G * pr.Px * sc.R), dim3(64 * S::WAVES), S::LDS_TOTAL, st, pr, kp, sc.R,
                     sc.range_len, sc.G, g.bucket_tiles, g.nbk, bmax, thr, lists, stg);
  return hipGetLastError();
}

template <int D, int KL, bool SMALL>
static hipError_t launch_pe_s(const DevProb& pr, int kp, const PerEmbdGrid& g, float* bmax, float* thr,
                              uint64_t* lists, uint64_t* stg, hipStream_t st) {
  hipError_t e = launch_pe_t<D, KL, false, SMALL>(pr, kp, g, bmax, thr, lists, stg, st);
  if (e != hipSuccess) return e;
  const int nvec = pr.B * pr.Pq;
  const int nblk = (nvec + kThrLists - 1) / kThrLists;
  const int per_list = 2 * g.s1.R * g.nbk;
  const int lds = kThrLists * (per_list + 1) * 4;
  auto thr_kern = per_list <= kMaxBuckets / 2 ? &k_bucket_threshold<kMaxBuckets / 128>
                                              : &k_bucket_threshold<kMaxBuckets / 64>;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(thr_kern), hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(thr_kern, dim3(nblk * pr.Px), dim3(64 * kThrLists), lds, st, bmax, nvec, pr.Px,
                     g.s1.R * g.nbk, kp, thr);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_pe_t<D, KL, true, SMALL>(pr, kp, g, bmax, thr, lists, stg, st);
}

template <int D, int KL>
static hipError_t launch_pe_d(const DevProb& pr, int kp, const PerEmbdGrid& g, float* bmax, float* thr,
                              uint64_t* lists, uint64_t* stg, hipStream_t st) {
  if constexpr (KL <= 256) {
    if (per_embd_small(pr, kp)) return launch_pe_s<D, KL, true>(pr, kp, g, bmax, thr, lists, stg, st);
  }
  return launch_pe_s<D, KL, false>(pr, kp, g, bmax, thr, lists, stg, st);
}

hipError_t launch_per_embd(const DevProb& pr, int kp, const PerEmbdGrid& g, float* bmax, float* thr,
                           uint64_t* lists, uint64_t* stg, hipStream_t st) {
  const int KL = per_embd_list_cap(kp);
  if (pr.d == 32) {
    switch (KL) {
      case 128: return launch_pe_d<32, 128>(pr, kp, g, bmax, thr, lists, stg, st);
      case 256: return launch_pe_d<32, 256>(pr, kp, g, bmax, thr, lists, stg, st);
      case 512: return launch_pe_d<32, 512>(pr, kp, g, bmax, thr, lists, stg, st);
      default: return launch_pe_d<32, 1024>(pr, kp, g, bmax, thr, lists, stg, st);
    }
  }
  if (pr.d == 64) {
    switch (KL) {
      case 128: return launch_pe_d<64, 128>(pr, kp, g, bmax, thr, lists, stg, st);
      case 256: return launch_pe_d<64, 256>(pr, kp, g, bmax, thr, lists, stg, st);
      case 512: return launch_pe_d<64, 512>(pr, kp, g, bmax, thr, lists, stg, st);
      default: return launch_pe_d<64, 1024>(pr, kp, g, bmax, thr, lists, stg, st);
    }
  }
  switch (KL) {
    case 128: return launch_pe_d<128, 128>(pr, kp, g, bmax, thr, lists, stg, st);
    case 256: return launch_pe_d<128, 256>(pr, kp, g, bmax, thr, lists, stg, st);
    case 512: return launch_pe_d<128, 512>(pr, kp, g, bmax, thr, lists, stg, st);
    default: return launch_pe_d<128, 1024>(pr, kp, g, bmax, thr, lists, stg, st);
  }
}

}  // namespace mol
