// MoL rerank of deduplicated candidates on gfx950 matrix cores
// (Algorithm 2, BruteForceTopKMoL over the candidate set G).
//
// Each wave takes one query and one chunk of its distinct candidate ids and
// walks it 16 items at a time: the items' component embeddings are gathered
// from the component-major corpus one step ahead, by direct global -> LDS
// copies (one 16-byte copy per lane per component and K block) into a
// buffer of the wave (Px d / 32 KB), and read back as MFMA operands at the start of their
// step (their gating logits a_x are prefetched into registers);
// GEMM1 forms the 8 x 16 dot products of the query's components with the
// items' components in rows 2 pq of the 16x16x32 tile (the odd rows are
// zero), which leaves them in the run layout of mol_tile.h, and the shared
// MFMA epilogue evaluates the gating MLP, softmax and phi.  A running
// top-k per wave is merged across chunks afterwards by segmented sorts.
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {
constexpr int kWaves = 4;
constexpr int kTopkRegion = WaveTopk::kList + WaveTopk::kStage;
}  // namespace

template <int PX, int D, int H, bool NEG, bool X2>
__global__ __launch_bounds__(64 * kWaves, 2) void k_mol_rerank(
    DevProb pr, const int32_t* __restrict__ uniq, const int32_t* __restrict__ n_unique, int C,
    int k, int chunk, int nchunks, uint64_t* __restrict__ partial) {
  using Mlp = MolMlp<PX, H, X2>;   // X2: the two-term gating chain
  constexpr int P = 8 * PX, RUN = 2 * PX, KD = D / 32, PT = P / 16;
  __shared__ uint64_t sTop[kWaves * kTopkRegion];
  // the wave's gather buffer: block (px, kk) of 1 KB holds lane i's 16 bytes
  // of component px, K block kk at byte 16 i (a direct global -> LDS copy)
  extern __shared__ __attribute__((aligned(16))) unsigned char sGather[];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int base = lane_base(g, PX);
  const long wid = static_cast<long>(blockIdx.x) * kWaves + wave;
  if (wid >= static_cast<long>(pr.B) * nchunks) return;     // whole wave exits
  const int b = static_cast<int>(wid / nchunks), j = static_cast<int>(wid % nchunks);
  const int nu = n_unique[b];
  const int i0 = j * chunk, i1 = min(nu, i0 + chunk);
  const int N = pr.N;
  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);
  const int32_t* ids = uniq + static_cast<long>(b) * C;

  WaveTopk top;
  top.init(sTop + wave * kTopkRegion, k, lane);
  Mlp mlp;
  mlp.load(pr, c, g);
  // log2(e) (a_q + b2) of query b at the lane's p = base(g) + 4 pt + i
  f32x4_t cbf[PT];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = base + 4 * pt + i;
      cbf[pt][i] = kLog2e * (pr.a_q[static_cast<long>(b) * P + p] + pr.b2[p]);
    }
  // query b's component pq as GEMM1 row 2 pq (odd rows zero)
  uint4 qop[KD];
#pragma unroll
  for (int kk = 0; kk < KD; ++kk)
    qop[kk] = (c & 1) == 0
                  ? *reinterpret_cast<const uint4*>(Q + (static_cast<long>(b) * 8 + (c >> 1)) * D + 32 * kk + 8 * g)
                  : make_uint4(0, 0, 0, 0);

  // Each step's 16 items are gathered one step ahead: the component
  // operands by direct global -> LDS copies into the wave's buffer (read
  // back into registers at the start of the step, after which the next
  // step's copies are issued into it), the item logits a_x into registers.
  unsigned char* gbuf = sGather + __builtin_amdgcn_readfirstlane(wave) * (PX * KD * 1024);
  auto item_at = [&](int pos) { return pos < i1 ? min(max(ids[pos], 0), N - 1) : 0; };   // ids are in range
  float4 axn[PT];
  auto gather = [&](int it) {
#pragma unroll
    for (int px = 0; px < PX; ++px)
#pragma unroll
      for (int kk = 0; kk < KD; ++kk)
        copy16_to_lds(X + (static_cast<long>(px) * N + it) * D + 32 * kk + 8 * g,
                      lds_addr(gbuf + (px * KD + kk) * 1024));
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
      axn[pt] = *reinterpret_cast<const float4*>(pr.a_x + static_cast<long>(it) * P + base + 4 * pt);
  };
  int item_n = item_at(i0 + c);
  if (i0 < i1) gather(item_n);
  int item_nn = item_at(i0 + 16 + c);
  for (int s0 = i0; s0 < i1; s0 += 16) {
    const int pos = s0 + c;
    const bool ok = pos < i1;
    const int item = item_n;
    // this step's copies have landed (only the younger id load may be
    // outstanding); read the operands, then refill the buffer
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(1));
    asm volatile("" ::: "memory");
    uint4 xop[PX][KD];
#pragma unroll
    for (int px = 0; px < PX; ++px)
#pragma unroll
      for (int kk = 0; kk < KD; ++kk)
        xop[px][kk] = *reinterpret_cast<const uint4*>(gbuf + (px * KD + kk) * 1024 + 16 * lane);
    f32x4_t c0[1][PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt)
      c0[0][pt] = f32x4_t{kLog2e * axn[pt].x, kLog2e * axn[pt].y, kLog2e * axn[pt].z, kLog2e * axn[pt].w} + cbf[pt];
    wave_lds_sync();
    if (s0 + 16 < i1) {
      item_n = item_nn;
      gather(item_n);
      item_nn = item_at(s0 + 32 + c);
    }
    f32x4_t acc1[PX];
#pragma unroll
    for (int px = 0; px < PX; ++px) {
      acc1[px] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KD; ++kk) acc1[px] = mfma_bf16(qop[kk], xop[px][kk], acc1[px]);
    }
    // accumulator row 4 g + i with i even is pq = 2 g + i / 2: p = base(g) + (i / 2) PX + px
    float s[1][RUN];
#pragma unroll
    for (int mu = 0; mu < RUN; ++mu) s[0][mu] = acc1[mu % PX][2 * (mu / PX)];
    float phi[1];
    mlp.template phi<1>(s, c0, phi);
    top.offer_score(NEG ? -phi[0] : phi[0], item, g == 0 && ok, lane);
  }
  top.flush(lane);
  uint64_t* dst = partial + (static_cast<long>(b) * nchunks + j) * k;
  for (int i = lane; i < k; i += 64) dst[i] = top.reg[i];
}

// ---------------------------------------------------------------------------
bool rerank_supported(const DevProb& pr, int k) { return fused_supported(pr, k); }

// Candidates per wave: the largest of 4096, 2048, 1024, 512 and 256 that
// still gives at least one round of resident waves (two 4-wave workgroups
// per CU on 256 CUs), so that long lists amortise each wave's operand set-up
// and small batches still fill the chip.  With the candidates in ascending
// id bins (the dedup's output order) and every wave resident at once, the
// waves sweep the corpus together and the several queries that share an
// item gather it close in time (exact_1m: 1.67 ms with 2048, 1.52 ms with
// 4096; 1.88 ms in hash order).
int rerank_chunk(int B, int C) {
  constexpr long kResidentWaves = 2l * kWaves * 256;
  for (int chunk = 4096; chunk > 256; chunk /= 2)
    if (static_cast<long>(B) * ((C + chunk - 1) / chunk) >= kResidentWaves) return chunk;
  return 256;
}

template <int PX, int D, int H, bool NEG, bool X2>
static hipError_t launch_rerank_x(const DevProb& pr, dim3 grid, const int32_t* uniq, const int32_t* n_unique,
                                  int C, int k, int chunk, int nchunks, uint64_t* partial, hipStream_t st) {
  constexpr int kGather = kWaves * PX * (D / 32) * 1024;   // the waves' gather buffers
  auto kern = &k_mol_rerank<PX, D, H, NEG, X2>;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kGather);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, grid, dim3(64 * kWaves), kGather, st, pr, uniq, n_unique, C, k, chunk, nchunks, partial);
  return hipGetLastError();
}

template <int PX, int D, int H, bool NEG>
static hipError_t launch_rerank_one(const DevProb& pr, dim3 grid, const int32_t* uniq, const int32_t* n_unique,
                                    int C, int k, int chunk, int nchunks, uint64_t* partial, hipStream_t st) {
  if (pr.flags & MOL_FLAG_BF16X2_GATING)
    return launch_rerank_x<PX, D, H, NEG, true>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  return launch_rerank_x<PX, D, H, NEG, false>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
}

template <bool NEG>
static hipError_t launch_rerank_t(const DevProb& pr, dim3 grid, const int32_t* uniq, const int32_t* n_unique,
                                  int C, int k, int chunk, int nchunks, uint64_t* partial, hipStream_t st) {
  if (pr.Px == 8 && pr.d == 32)
    return launch_rerank_one<8, 32, 64, NEG>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  if (pr.Px == 8)
    return launch_rerank_one<8, 64, 64, NEG>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  if (pr.d == 128)
    return launch_rerank_one<4, 128, 128, NEG>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  return launch_rerank_one<4, 64, 64, NEG>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
}

hipError_t launch_rerank(const DevProb& pr, const int32_t* uniq, const int32_t* n_unique, int C, int k,
                         bool negate, uint64_t* partial, hipStream_t st) {
  const int chunk = rerank_chunk(pr.B, C);
  const int nchunks = (C + chunk - 1) / chunk;
  const long waves = static_cast<long>(pr.B) * nchunks;
  const dim3 grid(static_cast<unsigned>((waves + kWaves - 1) / kWaves));
  return negate ? launch_rerank_t<true>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st)
                : launch_rerank_t<false>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
}

}  // namespace mol
