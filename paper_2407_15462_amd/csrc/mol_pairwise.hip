// Pair-wise MoL scoring on gfx950 matrix cores over a buffer of component
// dot products: the gating MLP + softmax + weighted sum of Eq. 1 (two-layer
// SiLU gating of Appendix A.3) for the shapes the fused kernels do not
// cover, P = Pq * Px <= 64 and H <= 128, bf16 problems.
//
// Input: s[p * s_pstride + b * s_bstride + i], the float32 dot products of
// the MFMA dots kernel for item i of a contiguous range (or candidate i of
// query b's list).  Each wave scores 16 items of one query per iteration
// with the MFMA gating chain of mol_tile.h, padded to P' = 8 PXV components
// and H' = HV hidden units with zero weights; padded components carry a
// -inf logit, so their softmax weight is exactly zero.
//
// Work split: a workgroup takes up to kPairQB queries and 4 wave ranges of
// `steps` 16-item steps; a wave walks its range step by step and, within a
// step, query by query, so the item-side inputs (a_x rows of the range) are
// read from L2 once per step and hit the L1 for the other queries.
//
// Lane (c = lane % 16, g = lane / 16) holds item c's dot products for the
// run p = base(g) + mu, mu < 2 PXV, of the padded layout.  Modes and
// outputs are those of the one-thread-per-pair kernel (GenMode); the
// max-component mode, which has no gating chain, is left to that kernel.
// PXV = 2 stands for P' = 16: the K = 16 gating chain (MolMlp16), whose lane
// runs are p = 4 g + mu, mu < 4.
#include <type_traits>

#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {
constexpr int kPairQB = 8;         // queries per workgroup
// 16-item steps per wave: enough that a wave runs at least kPairMinIters
// iterations (it builds its MLP operands once, from scattered weight
// reads), more when the launch would exceed one round of resident waves
constexpr int kPairMinIters = 16;
}  // namespace

// BOUNDED: Algorithm 1's second pass (kGenBounded); otherwise phi, negated
// when `neg` is set (kGenPhi, kGenNegPhi).  GATHER: per-query candidate
// lists (items != NULL) rather than a contiguous range.
template <int PXV, int HV, bool BOUNDED, bool GATHER, bool X2>
__global__ __launch_bounds__(256) void k_phi_mfma(
    DevProb pr, bool neg, const float* __restrict__ bound, int n_begin, int n_count, int steps,
    const int32_t* __restrict__ items, const int32_t* __restrict__ item_count, long item_stride,
    const float* __restrict__ sbuf, long s_pstride, long s_bstride,
    float* __restrict__ phi, long phi_stride, uint64_t* __restrict__ keys, long key_stride) {
  // X2: the two-term gating chain
  using Mlp = std::conditional_t<PXV == 2, MolMlp16<HV, X2>, MolMlp<PXV, HV, X2>>;
  constexpr int RUN = Mlp::RUN, PT = Mlp::PT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int P = pr.P;
  const int base = Mlp::base(g);
  const int b0 = blockIdx.y * kPairQB, nq = min(kPairQB, pr.B - b0);

  Mlp mlp;
  mlp.load_padded(pr, c, g);
  // log2(e) b2 of the lane's GEMM3 accumulator slots (p = base + 4 pt + e)
  float b2v[PT][4];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int e = 0; e < 4; ++e) b2v[pt][e] = kLog2e * pr.b2[min(base + 4 * pt + e, P - 1)];
  // a_x and a_q rows read as float4 runs where they are 16-byte aligned
  const bool vec4 = P % 4 == 0 && ((reinterpret_cast<uintptr_t>(pr.a_x) | reinterpret_cast<uintptr_t>(pr.a_q)) & 15) == 0;
  auto load_run = [&](const float* row, float (&out)[PT][4]) {
    if (vec4) {
      // P % 4 == 0: each run of 4 is wholly in range or wholly padding
#pragma unroll
      for (int pt = 0; pt < PT; ++pt) {
        const float4 a = *reinterpret_cast<const float4*>(row + min(base + 4 * pt, P - 4));
        out[pt][0] = a.x;
        out[pt][1] = a.y;
        out[pt][2] = a.z;
        out[pt][3] = a.w;
      }
    } else {
#pragma unroll
      for (int pt = 0; pt < PT; ++pt)
#pragma unroll
        for (int e = 0; e < 4; ++e) out[pt][e] = row[min(base + 4 * pt + e, P - 1)];
    }
  };

  // The wave's iterations: nsteps <= steps steps of 16 items from `first`,
  // nq queries each.  Two stages alternate: the loads of one are issued
  // before the other's gating chain runs.  Loads are unconditional, from
  // clamped in-range addresses (item 0 of the range, the last component; a
  // fetch past the wave's iterations reads those too), and their values are
  // masked only when used: no load sits in a branch that would wait for it,
  // and no stage is copied to another.
  const int first = (blockIdx.x * 4 + wave) * steps * 16;
  const int nsteps = min(steps, max(0, (n_count - first + 15) / 16));
  const int nit = nsteps * nq;
  uint32_t soff[RUN];                                       // element offset of the lane's rows
#pragma unroll
  for (int mu = 0; mu < RUN; ++mu) soff[mu] = static_cast<uint32_t>(min(base + mu, P - 1) * s_pstride);
  struct Stage {
    float s[RUN];       // raw: masked when used
    float ax[PT][4];
    float aq[PT][4];
    long n;
    int i, b, cnt;
    float bnd;
  };
  int ft = 0, fq = 0;   // step and query of the next fetch
  auto fetch = [&](Stage& st) {
    st.b = b0 + fq;
    st.i = first + 16 * ft + c;
    st.cnt = GATHER ? min(item_count[st.b], n_count) : n_count;
    if (BOUNDED) st.bnd = bound[st.b];
    const uint32_t ic = st.i < st.cnt ? st.i : 0;
    const long nl = GATHER ? static_cast<long>(items[st.b * item_stride + ic]) : static_cast<long>(n_begin) + ic;
    st.n = st.i < st.cnt ? nl : 0l;
    const float* sq = sbuf + st.b * s_bstride;
#pragma unroll
    for (int mu = 0; mu < RUN; ++mu) st.s[mu] = sq[soff[mu] + ic];
    load_run(pr.a_x + st.n * P, st.ax);
    load_run(pr.a_q + static_cast<long>(st.b) * P, st.aq);
    if (++fq == nq) {
      fq = 0;
      ++ft;
    }
  };
  auto score = [&](const Stage& st) {
    const int i = st.i, b = st.b;
    const bool live = i < st.cnt;
    float sv[1][RUN];
#pragma unroll
    for (int mu = 0; mu < RUN; ++mu) sv[0][mu] = live && base + mu < P ? st.s[mu] : 0.f;
    bool keep = live;
    if (BOUNDED) {
      float m = -__builtin_inff(), mabs = 0.f;
#pragma unroll
      for (int mu = 0; mu < RUN; ++mu)
        if (base + mu < P) {
          m = fmaxf(m, sv[0][mu]);
          mabs = fmaxf(mabs, fabsf(sv[0][mu]));
        }
      m = max_groups(m);
      mabs = max_groups(mabs);
      keep = keep && !(m + bound_margin(mabs) < st.bnd);   // phi <= m: cannot reach the bound
    }
    float v = 0.f;
    if (!BOUNDED || __any(keep)) {
      // log2(e) (a_x + a_q + b2), the GEMM3 accumulator input
      f32x4_t c0[1][PT];
#pragma unroll
      for (int pt = 0; pt < PT; ++pt)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          c0[0][pt][e] = base + 4 * pt + e < P ? fmaf(kLog2e, st.ax[pt][e] + st.aq[pt][e], b2v[pt][e])
                                               : -__builtin_inff();
      float out[1];
      mlp.template phi<1>(sv, c0, out);
      v = neg ? -out[0] : out[0];
    }
    // one lane per item writes
    if (g == 0 && i < n_count) {
      if (!keep) {
        if (phi && live) phi[b * phi_stride + i] = -__builtin_inff();
        if (keys) keys[b * key_stride + i] = 0;
      } else {
        if (phi) phi[b * phi_stride + i] = v;
        if (keys) keys[b * key_stride + i] = make_key(v, static_cast<int32_t>(st.n));
      }
    }
  };

  Stage sa, sb;
  fetch(sa);
  for (int u = 0; u < nit; u += 2) {
    fetch(sb);
    score(sa);
    if (u + 1 >= nit) break;
    fetch(sa);
    score(sb);
  }
}

bool phi_mfma_supported(const DevProb& pr) {
  return !(pr.flags & MOL_FLAG_F32_GATING) && pr.dtype == MOL_BF16 && pr.P <= 64 && pr.H <= 128;
}

// Waves of one k_phi_mfma instantiation that the device holds at once.
template <int PXV, int HV, bool BOUNDED, bool GATHER, bool X2>
static long pair_resident_waves() {
  static const long waves = [] {
    int dev = 0, ncu = 0, nb = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
      ncu = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_phi_mfma<PXV, HV, BOUNDED, GATHER, X2>, 256, 0) !=
            hipSuccess ||
        nb <= 0)
      nb = 1;
    return static_cast<long>(nb) * 4 * ncu;
  }();
  return waves;
}

// Work split: per_query 16-item steps for each of `groups` query groups of
// up to kPairQB (qb) queries.  Each wave takes `steps` steps: at least
// kPairMinIters iterations, and about one round of resident waves for the
// whole launch (a wave that lives longer amortises its operand set-up), but
// no more than one workgroup of 4 waves needs for the whole range.
template <int PXV, int HV, bool BOUNDED, bool GATHER, bool X2>
static void launch_phi_mfma_x(long per_query, long groups, long qb, const DevProb& pr, bool neg,
                              const float* bound, int n_begin, int n_count, const int32_t* items,
                              const int32_t* item_count, long item_stride, const float* sbuf, long s_pstride,
                              long s_bstride, float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st) {
  const long waves = pair_resident_waves<PXV, HV, BOUNDED, GATHER, X2>();
  long steps = std::max<long>((kPairMinIters + qb - 1) / qb, (per_query * groups + waves - 1) / waves);
  steps = std::max<long>(1, std::min<long>(steps, (per_query + 3) / 4));
  const dim3 grid(static_cast<unsigned>((per_query + 4 * steps - 1) / (4 * steps)), static_cast<unsigned>(groups));
  hipLaunchKernelGGL((k_phi_mfma<PXV, HV, BOUNDED, GATHER, X2>), grid, dim3(256), 0, st, pr, neg, bound, n_begin,
                     n_count, static_cast<int>(steps), items, item_count, item_stride, sbuf, s_pstride, s_bstride,
                     phi, phi_stride, keys, key_stride);
}

// the two-term chain where the problem asks for it (MOL_FLAG_BF16X2_GATING)
template <int PXV, int HV, bool BOUNDED, bool GATHER>
static void launch_phi_mfma_k(long per_query, long groups, long qb, const DevProb& pr, bool neg,
                              const float* bound, int n_begin, int n_count, const int32_t* items,
                              const int32_t* item_count, long item_stride, const float* sbuf, long s_pstride,
                              long s_bstride, float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st) {
  if (pr.flags & MOL_FLAG_BF16X2_GATING)
    launch_phi_mfma_x<PXV, HV, BOUNDED, GATHER, true>(per_query, groups, qb, pr, neg, bound, n_begin, n_count,
                                                      items, item_count, item_stride, sbuf, s_pstride, s_bstride,
                                                      phi, phi_stride, keys, key_stride, st);
  else
    launch_phi_mfma_x<PXV, HV, BOUNDED, GATHER, false>(per_query, groups, qb, pr, neg, bound, n_begin, n_count,
                                                       items, item_count, item_stride, sbuf, s_pstride, s_bstride,
                                                       phi, phi_stride, keys, key_stride, st);
}

template <int PXV, int HV, bool BOUNDED>
static void launch_phi_mfma_m(long per_query, long groups, long qb, const DevProb& pr, bool neg,
                              const float* bound, int n_begin, int n_count, const int32_t* items,
                              const int32_t* item_count, long item_stride, const float* sbuf, long s_pstride,
                              long s_bstride, float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st) {
  if (items)
    launch_phi_mfma_k<PXV, HV, BOUNDED, true>(per_query, groups, qb, pr, neg, bound, n_begin, n_count, items,
                                              item_count, item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride,
                                              keys, key_stride, st);
  else
    launch_phi_mfma_k<PXV, HV, BOUNDED, false>(per_query, groups, qb, pr, neg, bound, n_begin, n_count, items,
                                               item_count, item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride,
                                               keys, key_stride, st);
}

template <int PXV, int HV>
static void launch_phi_mfma_t(long per_query, long groups, long qb, const DevProb& pr, int mode,
                              const float* bound, int n_begin, int n_count, const int32_t* items,
                              const int32_t* item_count, long item_stride, const float* sbuf, long s_pstride,
                              long s_bstride, float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st) {
  if (mode == kGenBounded)
    launch_phi_mfma_m<PXV, HV, true>(per_query, groups, qb, pr, false, bound, n_begin, n_count, items, item_count,
                                     item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
  else
    launch_phi_mfma_m<PXV, HV, false>(per_query, groups, qb, pr, mode == kGenNegPhi, nullptr, n_begin, n_count,
                                      items, item_count, item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride,
                                      keys, key_stride, st);
}

hipError_t launch_phi_mfma(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                           const int32_t* items, const int32_t* item_count, long item_stride,
                           const float* sbuf, long s_pstride, long s_bstride, float* phi, long phi_stride,
                           uint64_t* keys, long key_stride, hipStream_t st) {
  if (n_count <= 0) return hipSuccess;
  if (!phi_mfma_supported(pr) || sbuf == nullptr) return hipErrorInvalidValue;
  // the max-component mode has no gating chain (and may carry no gating
  // input), and the kernel addresses a query's rows with 32-bit element offsets
  if (mode == kGenMaxDot || static_cast<long>(pr.P) * s_pstride >= (1l << 32))
    return launch_phi_generic(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf, s_pstride,
                              s_bstride, phi, phi_stride, keys, key_stride, st);
  const long per_query = (static_cast<long>(n_count) + 15) / 16;   // 16-item steps per query
  const long groups = (pr.B + kPairQB - 1) / kPairQB;
  const long qb = std::min<long>(kPairQB, pr.B);
#define MOL_PHI_MFMA(PXV, HV)                                                                              \
  launch_phi_mfma_t<PXV, HV>(per_query, groups, qb, pr, mode, bound, n_begin, n_count, items, item_count, \
                             item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st)
  if (pr.P <= 16) {
    if (pr.H <= 32) MOL_PHI_MFMA(2, 32);
    else if (pr.H <= 64) MOL_PHI_MFMA(2, 64);
    else MOL_PHI_MFMA(2, 128);
  } else if (pr.P <= 32) {
    if (pr.H <= 32) MOL_PHI_MFMA(4, 32);
    else if (pr.H <= 64) MOL_PHI_MFMA(4, 64);
    else MOL_PHI_MFMA(4, 128);
  } else {
    if (pr.H <= 32) MOL_PHI_MFMA(8, 32);
    else if (pr.H <= 64) MOL_PHI_MFMA(8, 64);
    else MOL_PHI_MFMA(8, 128);
  }
#undef MOL_PHI_MFMA
  return hipGetLastError();
}

}  // namespace mol
