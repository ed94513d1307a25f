// MoL rerank of deduplicated candidates on gfx950 matrix cores
// (Algorithm 2, BruteForceTopKMoL over the candidate set G).
//
// Each wave takes one query and one chunk of its distinct candidate ids and
// walks it 16 items at a time: the items' component embeddings and gating
// logits are gathered straight from the component-major corpus into MFMA
// operand registers (one 16-byte load per lane per component and K block),
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

template <int PX, int D, int H, bool NEG>
__global__ __launch_bounds__(64 * kWaves, 2) void k_mol_rerank(
    DevProb pr, const int32_t* __restrict__ uniq, const int32_t* __restrict__ n_unique, int C,
    int k, int chunk, int nchunks, uint64_t* __restrict__ partial) {
  using Mlp = MolMlp<PX, H>;
  constexpr int P = 8 * PX, RUN = 2 * PX, KD = D / 32, PT = P / 16;
  __shared__ uint64_t sTop[kWaves * kTopkRegion];

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

  for (int s0 = i0; s0 < i1; s0 += 16) {
    const int pos = s0 + c;
    const bool ok = pos < i1;
    int item = ok ? ids[pos] : 0;
    item = min(max(item, 0), N - 1);       // ids come from the dedup pass: in range
    // gather the 16 items' components as GEMM1 B operands
    uint4 xop[PX][KD];
#pragma unroll
    for (int px = 0; px < PX; ++px)
#pragma unroll
      for (int kk = 0; kk < KD; ++kk)
        xop[px][kk] = *reinterpret_cast<const uint4*>(X + (static_cast<long>(px) * N + item) * D + 32 * kk + 8 * g);
    f32x4_t c0[1][PT];
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) {
      const float4 a = *reinterpret_cast<const float4*>(pr.a_x + static_cast<long>(item) * P + base + 4 * pt);
      c0[0][pt] = f32x4_t{kLog2e * a.x, kLog2e * a.y, kLog2e * a.z, kLog2e * a.w} + cbf[pt];
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

template <bool NEG>
static void launch_rerank_t(const DevProb& pr, dim3 grid, const int32_t* uniq, const int32_t* n_unique,
                            int C, int k, int chunk, int nchunks, uint64_t* partial, hipStream_t st) {
  if (pr.Px == 8 && pr.d == 32)
    hipLaunchKernelGGL((k_mol_rerank<8, 32, 64, NEG>), grid, dim3(64 * kWaves), 0, st, pr, uniq, n_unique, C,
                       k, chunk, nchunks, partial);
  else if (pr.Px == 8)
    hipLaunchKernelGGL((k_mol_rerank<8, 64, 64, NEG>), grid, dim3(64 * kWaves), 0, st, pr, uniq, n_unique, C,
                       k, chunk, nchunks, partial);
  else if (pr.d == 128)
    hipLaunchKernelGGL((k_mol_rerank<4, 128, 128, NEG>), grid, dim3(64 * kWaves), 0, st, pr, uniq, n_unique,
                       C, k, chunk, nchunks, partial);
  else
    hipLaunchKernelGGL((k_mol_rerank<4, 64, 64, NEG>), grid, dim3(64 * kWaves), 0, st, pr, uniq, n_unique, C,
                       k, chunk, nchunks, partial);
}

hipError_t launch_rerank(const DevProb& pr, const int32_t* uniq, const int32_t* n_unique, int C, int k,
                         bool negate, uint64_t* partial, hipStream_t st) {
  const int chunk = rerank_chunk(pr.B, C);
  const int nchunks = (C + chunk - 1) / chunk;
  const long waves = static_cast<long>(pr.B) * nchunks;
  const dim3 grid(static_cast<unsigned>((waves + kWaves - 1) / kWaves));
  if (negate)
    launch_rerank_t<true>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  else
    launch_rerank_t<false>(pr, grid, uniq, n_unique, C, k, chunk, nchunks, partial, st);
  return hipGetLastError();
}

}  // namespace mol
