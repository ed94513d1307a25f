// Component dot products of every query vector with a tile of items on
// gfx950 matrix cores, for the shapes the fused kernels do not cover
// (any P_q, P_x <= 64, d a multiple of 32 up to 1024, bf16): the first step
// of Eq. 1 / Eq. 2 as a plain GEMM, S_px = X_px Q^T per item component px.
//
// Workgroup: 4 waves on a 128-item x 64-vector output tile, each wave two
// 32 x 32 blocks (64 items x 32 vectors) on 32x32x16 bf16 MFMAs.  The K
// dimension (d) is walked 64 at a time through double-buffered LDS tiles
// [rows][64 K] whose 16-byte chunks are XOR-swizzled by row.  In each block
// D[item][vector] lane (c = lane % 32, h = lane / 32) holds vector c's dot
// products with items 8 j + 4 h + i (j, i < 4): four runs of 4 consecutive
// items.
//
// Gather form (items != NULL): block row y is query b and the tile's items
// are b's candidates items[b * item_stride + i], i < item_count[b]; the
// vector slots past b's P_q vectors are zero (the matrix core has work to
// spare at rerank sizes).
//
// Outputs, per mode:
//   kDotsToBuffer      s[p][b][i] float32 (p = pq * P_x + px, i = item - n0),
//                      the input of the pair-wise gating kernel;
//   kDotsToKeys        keys[(b * P + p) * key_stride + i], the per-component
//                      lists (TopKDotProduct) before selection.  With
//                      tile_stride > 1 only every tile_stride-th 128-item
//                      tile is computed (a sample), its keys stored
//                      compactly (tile j at 128 j) and slots past the range
//                      cleared to 0;
//   kDotsToMaxKeys     keys[b * key_stride + i] of m = max_p s_p (the
//                      components walked inside the workgroup; P_q divides
//                      64): the max-component score of every item;
//   kDotsToCandidates  the keys of list (b, p) that reach thr[(b * P + p) *
//                      thr_stride] are appended to its row of `keys`, the
//                      list's count advanced with one atomic add per wave
//                      and list, straight from the accumulators (the rows
//                      must hold every item).
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32x16_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// physical 16-byte chunk of logical chunk ch in row r (rows of 8 chunks,
// 128 B: two rows per 256 B of banks).  The 16 consecutive rows that one
// 16-lane group reads at the same logical chunk land in 16 distinct 16-byte
// bank slots: row parity picks the half, (r / 2) % 8 the slot within it.
__device__ __forceinline__ int dots_swz8(int r, int ch) { return ch ^ ((r >> 1) & 7); }

}  // namespace

// Grid: x = 128-item tiles of [n0, n0 + nt), y = TV-vector tiles of the
// B * P_q query vectors (gather form: query b), z = item component px.
// TV = 64 or 128 vectors per tile: each of the 4 waves owns 64 items x TV/2
// vectors (TV/64 pairs of 32 x 32 blocks); with TV = 128 the items are read
// once for twice as many vectors.  The result tile leaves through LDS in
// halves of 64 vector rows.
template <int MODE, int TV>
__global__ __launch_bounds__(256) void k_dots_mfma(DevProb pr, int n0, int nt, int tile_stride,
                                                   const int32_t* __restrict__ items,
                                                   const int32_t* __restrict__ item_count, long item_stride,
                                                   float* __restrict__ sbuf, long s_pstride, long s_bstride,
                                                   uint64_t* __restrict__ keys, long key_stride,
                                                   const uint64_t* __restrict__ thr, long thr_stride,
                                                   uint32_t* __restrict__ counts) {
  constexpr int TI = 128, KS = 64, CH = KS / 8;   // tile items, K per step, chunks per row
  constexpr int NBV = TV / 64;                    // 32-vector blocks per wave
  constexpr int BL = TV * CH / 256;               // vector-row chunks per thread and step
  constexpr int HALVES = TV / 64;                 // 64-row halves of the result tile
  // staging: items [2][TI][CH] (16 KB per buffer), then vectors [2][TV][CH];
  // after the K loop one 64-row half of the result tile [64][TR] floats
  constexpr int TR = TI + 4;
  __shared__ uint4 smem[2 * TI * CH + 2 * TV * CH];
  static_assert(64 * TR * 4 <= sizeof(smem), "result half-tile exceeds the staging area");
  uint4* sA = smem;
  uint4* sB = smem + 2 * TI * CH;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool gather = items != nullptr;
  const int it0 = blockIdx.x * TI * tile_stride, px = blockIdx.z;   // first item of the tile (range-relative)
  const int ot0 = blockIdx.x * TI;                                   // its first output slot
  // vectors of the tile: [v0, v1)
  const int v0 = gather ? blockIdx.y * pr.Pq : blockIdx.y * TV;
  const int v1 = gather ? v0 + pr.Pq : pr.B * pr.Pq;
  const int cnt = gather ? item_count[blockIdx.y] : nt;   // items of the row
  const int N = pr.N, D = pr.d;
  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);

  // loader: 4 item-row chunks and BL vector-row chunks per thread and step
  const bf16_t* xsrc[4];
  int aslot[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = tid + 256 * i, r = e / CH, ch = e % CH;
    int item;
    if (gather) {
      // candidates past the count read item 0 (valid memory, never stored)
      const int pos = it0 + r;
      item = pos < cnt ? items[blockIdx.y * item_stride + pos] : 0;
      item = min(max(item, 0), N - 1);
    } else {
      item = min(n0 + it0 + r, N - 1);                // past the tile: a valid row, never stored
    }
    xsrc[i] = X + (static_cast<long>(px) * N + item) * D + 8 * ch;
    aslot[i] = r * CH + dots_swz8(r, ch);
  }
  const bf16_t* qsrc[BL];
  int bslot[BL];
  bool vok[BL];
#pragma unroll
  for (int i = 0; i < BL; ++i) {
    const int e = tid + 256 * i, r = e / CH, ch = e % CH;
    vok[i] = v0 + r < v1;
    qsrc[i] = Q + static_cast<long>(vok[i] ? v0 + r : 0) * D + 8 * ch;
    bslot[i] = r * CH + dots_swz8(r, ch);
  }

  const int c = lane & 31, h = lane >> 5;
  const int wm = wave & 1, wn = wave >> 1;            // item half (64), vector half (TV/2) of the tile
  // candidates: the thresholds of the lane's lists (vector wn TV/2 + 32 jb +
  // c of each block column jb, component px), read now so that the reads
  // complete during the K loop
  uint64_t thr_v[NBV];
  long list_v[NBV];
#pragma unroll
  for (int jb = 0; jb < NBV; ++jb) {
    thr_v[jb] = ~0ull;
    list_v[jb] = 0;
    if (MODE == kDotsToCandidates) {
      const int v = v0 + wn * (TV / 2) + jb * 32 + c;
      if (v < v1) {
        const int b = v / pr.Pq, pq = v - (v / pr.Pq) * pr.Pq;
        list_v[jb] = static_cast<long>(b) * pr.P + pq * pr.Px + px;
        thr_v[jb] = thr[list_v[jb] * thr_stride];
      }
    }
  }

  f32x16_t acc[2][NBV];
  auto zero_acc = [&]() {
#pragma unroll
    for (int ib = 0; ib < 2; ++ib)
#pragma unroll
      for (int jb = 0; jb < NBV; ++jb) acc[ib][jb] = f32x16_t{};
  };

  // every loader slot of a thread holds the same chunk (tid % 8); with d a
  // multiple of 32 only, the upper half of the last K step reads zeros
  const int kch = 8 * (tid % CH);
  uint4 xa[4], qb[BL];
  long xoff = 0;                                      // component offset (max-dot form: px walked here)
  auto load = [&](int k0) {
    const bool kin = k0 + kch < D;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      xa[i] = kin ? *reinterpret_cast<const uint4*>(xsrc[i] + xoff + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < BL; ++i)
      qb[i] = kin && vok[i] ? *reinterpret_cast<const uint4*>(qsrc[i] + k0) : make_uint4(0, 0, 0, 0);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) sA[buf * TI * CH + aslot[i]] = xa[i];
#pragma unroll
    for (int i = 0; i < BL; ++i) sB[buf * TV * CH + bslot[i]] = qb[i];
  };
  const int nk = (D + KS - 1) / KS;
  // max-dot form: every component of the items in turn, keeping the
  // elementwise maximum of the dot tiles
  f32x16_t run[2][NBV];
  const int npx = MODE == kDotsToMaxKeys ? pr.Px : 1;
  for (int cx = 0; cx < npx; ++cx) {
    xoff = MODE == kDotsToMaxKeys ? static_cast<long>(cx) * N * D : 0l;
    zero_acc();
    load(0);
    store(0);
    __syncthreads();
    for (int kk = 0; kk < nk; ++kk) {
      const int cur = kk & 1;
      const bool more = kk + 1 < nk;
      if (more) load(KS * (kk + 1));
#pragma unroll
      for (int kb = 0; kb < KS / 16; ++kb) {             // K blocks of 16
        uint4 bv[NBV];
#pragma unroll
        for (int jb = 0; jb < NBV; ++jb) {
          const int rb = wn * (TV / 2) + jb * 32 + c;    // B row (vector)
          bv[jb] = sB[cur * TV * CH + rb * CH + dots_swz8(rb, 2 * kb + h)];
        }
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
          const int ra = wm * 64 + ib * 32 + c;           // A row (item)
          const uint4 a = sA[cur * TI * CH + ra * CH + dots_swz8(ra, 2 * kb + h)];
#pragma unroll
          for (int jb = 0; jb < NBV; ++jb) acc[ib][jb] = mfma32x16_bf16(a, bv[jb], acc[ib][jb]);
        }
      }
      if (more) store(cur ^ 1);
      __syncthreads();
    }
    if (MODE == kDotsToMaxKeys) {
#pragma unroll
      for (int ib = 0; ib < 2; ++ib)
#pragma unroll
        for (int jb = 0; jb < NBV; ++jb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            run[ib][jb][e] = cx == 0 ? acc[ib][jb][e] : fmaxf(run[ib][jb][e], acc[ib][jb][e]);
    }
  }
  if (MODE == kDotsToMaxKeys) {
#pragma unroll
    for (int ib = 0; ib < 2; ++ib)
#pragma unroll
      for (int jb = 0; jb < NBV; ++jb) acc[ib][jb] = run[ib][jb];
  }

  if constexpr (MODE == kDotsToCandidates) {
    // Straight from the accumulators: lane (c, h) of block (ib, jb) holds
    // list jb's scores of items wm 64 + 32 ib + 8 j + 4 h + i (j, i < 4).
    // A key reaches th iff its score beats th's, or ties it with an index
    // that keeps the key at or above th: the float compare decides almost
    // every item, and the key is formed only for the kept ones.  The two
    // lanes of a list (h = 0, 1) reserve their slots with one atomic add.
#pragma unroll
    for (int jb = 0; jb < NBV; ++jb) {
      const uint64_t th = thr_v[jb];
      const float ts = key_score(th);
      auto kept = [&](int ib, int e) {
        const int i = it0 + wm * 64 + ib * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
        const float v = acc[ib][jb][e];
        return i < cnt && v >= ts && (v > ts || make_key(v, n0 + i) >= th);
      };
      uint32_t n = 0;
#pragma unroll
      for (int ib = 0; ib < 2; ++ib)
#pragma unroll
        for (int e = 0; e < 16; ++e) n += kept(ib, e) ? 1u : 0u;
      const uint32_t n_other = static_cast<uint32_t>(__shfl_xor(static_cast<int>(n), 32, 64));
      if (__ballot(n > 0) == 0ull) continue;               // no lane keeps a key (wave-uniform)
      uint32_t base = 0;
      if (h == 0 && n + n_other > 0) base = atomicAdd(counts + list_v[jb], n + n_other);
      const uint32_t base0 = static_cast<uint32_t>(__shfl_xor(static_cast<int>(base), 32, 64));
      uint32_t pos = h == 0 ? base : base0 + n_other;
      uint64_t* dst = keys + list_v[jb] * key_stride;
      if (n > 0) {
#pragma unroll
        for (int ib = 0; ib < 2; ++ib)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kept(ib, e)) {
              const int i = it0 + wm * 64 + ib * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
              dst[pos++] = make_key(acc[ib][jb][e], n0 + i);
            }
      }
    }
    return;
  }

  // The loop ended with a barrier: the staging area is free.  Each 64-row
  // half of the tile goes through LDS (rows padded to TR floats) so that
  // every global store instruction writes a contiguous run of one row.
  float* sT = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int hv = 0; hv < HALVES; ++hv) {
    if (hv > 0) __syncthreads();                       // the previous half has been written out
#pragma unroll
    for (int jb = 0; jb < NBV; ++jb) {
      const int row = wn * (TV / 2) + jb * 32 - 64 * hv;   // first tile row of block jb, in this half
      if (row < 0 || row >= 64) continue;                  // wave-uniform
#pragma unroll
      for (int ib = 0; ib < 2; ++ib)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<float4*>(sT + (row + c) * TR + wm * 64 + ib * 32 + 8 * j + 4 * h) =
              float4{acc[ib][jb][4 * j + 0], acc[ib][jb][4 * j + 1], acc[ib][jb][4 * j + 2], acc[ib][jb][4 * j + 3]};
    }
    __syncthreads();
    const int vh = v0 + 64 * hv;                       // first vector of the half
    if (MODE == kDotsToMaxKeys) {
      // m = max over each query's P_q rows (P_q divides 64, so a query's rows
      // are one run of the half); wave w takes queries w, w+4, ...
      const int nq = 64 / pr.Pq, b0 = vh / pr.Pq;
      for (int qi = wave; qi < nq; qi += 4) {
        const int b = b0 + qi;
        if (b >= pr.B) break;                            // wave-uniform; queries ascend
        uint64_t* dst = keys + static_cast<long>(b) * key_stride;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int i = it0 + 64 * t + lane;
          float m = sT[(qi * pr.Pq) * TR + 64 * t + lane];
          for (int pq = 1; pq < pr.Pq; ++pq) m = fmaxf(m, sT[(qi * pr.Pq + pq) * TR + 64 * t + lane]);
          if (i < cnt) dst[i] = make_key(m, n0 + i);
        }
      }
    } else {
      // each wave writes 16 of the half's vector rows
      for (int rr = 0; rr < 16; ++rr) {
        const int r = wave * 16 + rr;
        const int v = vh + r;
        if (v >= v1) break;                                // rows ascend: the rest are past the end too
        const int b = v / pr.Pq, pq = v - (v / pr.Pq) * pr.Pq;
        const int p = pq * pr.Px + px;
        if (MODE == kDotsToBuffer) {
          // the buffer rows are padded to whole 128-item tiles
          const float2 val = *reinterpret_cast<const float2*>(sT + r * TR + 2 * lane);
          *reinterpret_cast<float2*>(sbuf + p * s_pstride + b * s_bstride + it0 + 2 * lane) = val;
        } else {
          uint64_t* dst = keys + (static_cast<long>(b) * pr.P + p) * key_stride;
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int i = it0 + 64 * t + lane;
            if (i < cnt) dst[ot0 + 64 * t + lane] = make_key(sT[r * TR + 64 * t + lane], n0 + i);
            else if (tile_stride > 1) dst[ot0 + 64 * t + lane] = 0ull;
          }
        }
      }
    }
  }
}

bool dots_mfma_supported(const DevProb& pr) {
  return pr.dtype == MOL_BF16 && pr.d % 32 == 0 && pr.d <= MOL_MAX_D;
}

long dots_buffer_row(int nt) { return (static_cast<long>(nt) + 127) / 128 * 128; }

// 128-vector tiles when there are at least 128 query vectors
static int dots_tv(const DevProb& pr) { return pr.B * pr.Pq >= 128 ? 128 : 64; }

template <int MODE>
static void dots_launch(int tv, dim3 grid, hipStream_t st, const DevProb& pr, int n0, int nt, int tile_stride,
                        const int32_t* items, const int32_t* item_count, long item_stride, float* sbuf,
                        long s_pstride, long s_bstride, uint64_t* keys, long key_stride, const uint64_t* thr,
                        long thr_stride, uint32_t* counts) {
  if (tv == 128)
    hipLaunchKernelGGL((k_dots_mfma<MODE, 128>), grid, dim3(256), 0, st, pr, n0, nt, tile_stride, items,
                       item_count, item_stride, sbuf, s_pstride, s_bstride, keys, key_stride, thr, thr_stride,
                       counts);
  else
    hipLaunchKernelGGL((k_dots_mfma<MODE, 64>), grid, dim3(256), 0, st, pr, n0, nt, tile_stride, items,
                       item_count, item_stride, sbuf, s_pstride, s_bstride, keys, key_stride, thr, thr_stride,
                       counts);
}

hipError_t launch_dots_mfma(const DevProb& pr, int n0, int nt, int mode, float* sbuf, long s_pstride,
                            long s_bstride, uint64_t* keys, long key_stride, hipStream_t st, int tile_stride) {
  if (nt <= 0) return hipSuccess;
  if (tile_stride < 1 || (tile_stride > 1 && mode != kDotsToKeys)) return hipErrorInvalidValue;
  const int tv = dots_tv(pr);
  const int tiles = (nt + 127) / 128;
  const dim3 grid((tiles + tile_stride - 1) / tile_stride, (pr.B * pr.Pq + tv - 1) / tv, pr.Px);
  if (mode == kDotsToBuffer)
    dots_launch<kDotsToBuffer>(tv, grid, st, pr, n0, nt, 1, nullptr, nullptr, 0l, sbuf, s_pstride, s_bstride,
                               nullptr, 0l, nullptr, 0l, nullptr);
  else
    dots_launch<kDotsToKeys>(tv, grid, st, pr, n0, nt, tile_stride, nullptr, nullptr, 0l, nullptr, 0l, 0l, keys,
                             key_stride, nullptr, 0l, nullptr);
  return hipGetLastError();
}

bool dots_maxkeys_supported(const DevProb& pr) { return dots_mfma_supported(pr) && 64 % pr.Pq == 0; }

hipError_t launch_dots_mfma_maxkeys(const DevProb& pr, int n0, int nt, uint64_t* keys, long key_stride,
                                    hipStream_t st) {
  if (nt <= 0) return hipSuccess;
  if (!dots_maxkeys_supported(pr)) return hipErrorInvalidValue;
  const int tv = dots_tv(pr);
  const dim3 grid((nt + 127) / 128, (pr.B * pr.Pq + tv - 1) / tv, 1);
  dots_launch<kDotsToMaxKeys>(tv, grid, st, pr, n0, nt, 1, nullptr, nullptr, 0l, nullptr, 0l, 0l, keys, key_stride,
                              nullptr, 0l, nullptr);
  return hipGetLastError();
}

// keys per row of the keys form: nt (tile_stride 1: exactly the range's
// keys are written), else whole sampled tiles (slots past the range cleared)
long dots_sample_len(int nt, int tile_stride) {
  return tile_stride == 1 ? nt : ((nt + 127) / 128 + tile_stride - 1) / tile_stride * 128l;
}

hipError_t launch_dots_mfma_candidates(const DevProb& pr, int n0, int nt, const uint64_t* thr, long thr_stride,
                                       uint64_t* cand, long cand_stride, uint32_t* counts, hipStream_t st) {
  if (nt <= 0) return hipSuccess;
  const int tv = dots_tv(pr);
  const dim3 grid((nt + 127) / 128, (pr.B * pr.Pq + tv - 1) / tv, pr.Px);
  dots_launch<kDotsToCandidates>(tv, grid, st, pr, n0, nt, 1, nullptr, nullptr, 0l, nullptr, 0l, 0l, cand,
                                 cand_stride, thr, thr_stride, counts);
  return hipGetLastError();
}

hipError_t launch_dots_mfma_gather(const DevProb& pr, const int32_t* items, const int32_t* item_count,
                                   long item_stride, int C, float* sbuf, long s_pstride, long s_bstride,
                                   hipStream_t st) {
  if (C <= 0) return hipSuccess;
  if (pr.Pq > 64) return hipErrorInvalidValue;
  const dim3 grid((C + 127) / 128, pr.B, pr.Px);
  dots_launch<kDotsToBuffer>(64, grid, st, pr, 0, C, 1, items, item_count, item_stride, sbuf, s_pstride, s_bstride,
                             nullptr, 0l, nullptr, 0l, nullptr);
  return hipGetLastError();
}

}  // namespace mol
