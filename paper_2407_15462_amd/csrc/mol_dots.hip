// Component dot products of every query vector with a tile of items on
// gfx950 matrix cores, for the shapes the fused kernels do not cover
// (any P_q, P_x <= 64, d a multiple of 32 up to 1024, bf16): the first step
// of Eq. 1 / Eq. 2 as a plain GEMM, S_px = X_px Q^T per item component px.
//
// Workgroup: 4 waves on a 64-item x 64-vector output tile, each wave one
// 32 x 32 block on 32x32x16 bf16 MFMAs.  The K dimension (d) is walked 32 at
// a time through double-buffered LDS tiles [64 rows][32 K] whose 16-byte
// chunks are XOR-swizzled by row so that a 16-lane group's 16 rows read
// distinct bank slots.  In the result D[item][vector] lane (c = lane % 32,
// h = lane / 32) holds vector c's dot products with items 8 j + 4 h + i
// (j, i < 4): four runs of 4 consecutive items.
//
// Gather form (items != NULL): block row y is query b and the tile's items
// are b's candidates items[b * item_stride + i], i < item_count[b]; the
// vector slots past b's P_q vectors are zero (the matrix core has work to
// spare at rerank sizes).
//
// Outputs, per mode:
//   kDotsToBuffer  s[p][b][i] float32 (p = pq * P_x + px, i = item - n0),
//                  the input of the pair-wise gating kernel;
//   kDotsToKeys    keys[(b * P + p) * key_stride + i], the per-component
//                  lists (TopKDotProduct) before selection.
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f32x16_t mfma32x16_bf16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// physical 16-byte chunk of logical chunk ch in row r (rows of 4 chunks)
__device__ __forceinline__ int dots_swz(int r, int ch) { return ch ^ ((r >> 2) & 3); }

}  // namespace

// Grid: x = 64-item tiles of [n0, n0 + nt), y = 64-vector tiles of the
// B * P_q query vectors, z = item component px.
template <int MODE>
__global__ __launch_bounds__(256) void k_dots_mfma(DevProb pr, int n0, int nt, const int32_t* __restrict__ items,
                                                   const int32_t* __restrict__ item_count, long item_stride,
                                                   float* __restrict__ sbuf, long s_pstride, long s_bstride,
                                                   uint64_t* __restrict__ keys, long key_stride) {
  __shared__ uint4 sA[2][64 * 4];   // items   [row][chunk], 4 KB per buffer
  __shared__ uint4 sB[2][64 * 4];   // vectors [row][chunk]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool gather = items != nullptr;
  const int it0 = blockIdx.x * 64, px = blockIdx.z;
  // vectors of the tile: [v0, v1)
  const int v0 = gather ? blockIdx.y * pr.Pq : blockIdx.y * 64;
  const int v1 = gather ? v0 + pr.Pq : pr.B * pr.Pq;
  const int cnt = gather ? item_count[blockIdx.y] : nt;   // items of the row
  const int N = pr.N, D = pr.d;
  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);

  // loader: thread t moves row t / 4, chunk t % 4 of both tiles
  const int lr = tid >> 2, lc = tid & 3;
  int item;
  if (gather) {
    // candidates past the count read item 0 (valid memory, never stored)
    const int i = it0 + lr;
    item = i < cnt ? items[blockIdx.y * item_stride + i] : 0;
    item = min(max(item, 0), N - 1);
  } else {
    item = min(n0 + it0 + lr, N - 1);                // past the tile: a valid row, never stored
  }
  const bool vok = v0 + lr < v1;
  const bf16_t* xsrc = X + (static_cast<long>(px) * N + item) * D + 8 * lc;
  const bf16_t* qsrc = Q + static_cast<long>(vok ? v0 + lr : 0) * D + 8 * lc;
  const int lslot = lr * 4 + dots_swz(lr, lc);

  const int c = lane & 31, h = lane >> 5;
  const int wm = wave & 1, wn = wave >> 1;            // item half, vector half of the tile
  const int ra = wm * 32 + c, rb = wn * 32 + c;       // A row (item), B row (vector)
  f32x16_t acc = f32x16_t{};

  uint4 xa = *reinterpret_cast<const uint4*>(xsrc);
  uint4 qb = vok ? *reinterpret_cast<const uint4*>(qsrc) : make_uint4(0, 0, 0, 0);
  sA[0][lslot] = xa;
  sB[0][lslot] = qb;
  __syncthreads();
  const int nk = D / 32;
  for (int kk = 0; kk < nk; ++kk) {
    const int cur = kk & 1;
    const bool more = kk + 1 < nk;
    if (more) {
      xa = *reinterpret_cast<const uint4*>(xsrc + 32 * (kk + 1));
      qb = vok ? *reinterpret_cast<const uint4*>(qsrc + 32 * (kk + 1)) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {                  // two K blocks of 16
      const uint4 a = sA[cur][ra * 4 + dots_swz(ra, 2 * kb + h)];
      const uint4 b = sB[cur][rb * 4 + dots_swz(rb, 2 * kb + h)];
      acc = mfma32x16_bf16(a, b, acc);
    }
    if (more) {
      sA[cur ^ 1][lslot] = xa;
      sB[cur ^ 1][lslot] = qb;
    }
    __syncthreads();
  }

  const int v = v0 + rb;
  if (v >= v1) return;
  const int b = v / pr.Pq, pq = v - (v / pr.Pq) * pr.Pq;
  const int p = pq * pr.Px + px;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i0 = it0 + wm * 32 + 8 * j + 4 * h;     // first of 4 consecutive items
    if (MODE == kDotsToBuffer) {
      // the buffer rows are padded to whole 64-item tiles
      float4* dst = reinterpret_cast<float4*>(sbuf + p * s_pstride + b * s_bstride + i0);
      *dst = float4{acc[4 * j + 0], acc[4 * j + 1], acc[4 * j + 2], acc[4 * j + 3]};
    } else {
      uint64_t* dst = keys + (static_cast<long>(b) * pr.P + p) * key_stride;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i0 + i < cnt) dst[i0 + i] = make_key(acc[4 * j + i], n0 + i0 + i);
    }
  }
}

bool dots_mfma_supported(const DevProb& pr) {
  return pr.dtype == MOL_BF16 && pr.d % 32 == 0 && pr.d <= MOL_MAX_D;
}

long dots_buffer_row(int nt) { return (static_cast<long>(nt) + 63) / 64 * 64; }

hipError_t launch_dots_mfma(const DevProb& pr, int n0, int nt, int mode, float* sbuf, long s_pstride,
                            long s_bstride, uint64_t* keys, long key_stride, hipStream_t st) {
  if (nt <= 0) return hipSuccess;
  const int nvec = pr.B * pr.Pq;
  const dim3 grid((nt + 63) / 64, (nvec + 63) / 64, pr.Px);
  if (mode == kDotsToBuffer)
    hipLaunchKernelGGL(k_dots_mfma<kDotsToBuffer>, grid, dim3(256), 0, st, pr, n0, nt, nullptr, nullptr, 0l,
                       sbuf, s_pstride, s_bstride, nullptr, 0l);
  else
    hipLaunchKernelGGL(k_dots_mfma<kDotsToKeys>, grid, dim3(256), 0, st, pr, n0, nt, nullptr, nullptr, 0l,
                       nullptr, 0l, 0l, keys, key_stride);
  return hipGetLastError();
}

hipError_t launch_dots_mfma_gather(const DevProb& pr, const int32_t* items, const int32_t* item_count,
                                   long item_stride, int C, float* sbuf, long s_pstride, long s_bstride,
                                   hipStream_t st) {
  if (C <= 0) return hipSuccess;
  if (pr.Pq > 64) return hipErrorInvalidValue;
  const dim3 grid((C + 63) / 64, pr.B, pr.Px);
  hipLaunchKernelGGL(k_dots_mfma<kDotsToBuffer>, grid, dim3(256), 0, st, pr, 0, C, items, item_count,
                     item_stride, sbuf, s_pstride, s_bstride, nullptr, 0l);
  return hipGetLastError();
}

}  // namespace mol
