// Fused MoL scoring on gfx950 matrix cores (bf16 embeddings, P_q = 8).
//
// One wave scores 2 queries against 16 items per step.  GEMM1 (bf16
// 16x16x32) forms S[(q, pq)][item] = Q[q][pq] . X[px][item] for every px with
// rows 2 pq + q, so a lane of group g = lane / 16 holds pq in {2 g, 2 g + 1}
// of both queries: each query's 64 dot products are already spread over the
// 64 lanes in the run layout of mol_tile.h, whose chained f16 MFMAs evaluate
// the gating MLP, the softmax and phi (Eq. 1 / Eq. 2 with the SiLU gating MLP
// of Appendix A.3) with no lane exchange and no LDS re-layout.  (The max-dot
// form keeps rows 8 q + pq, so that two lane groups hold one query.)
//
// Epilogues (EPI):
//  - kEpiTopk: a running per-query top-k of phi (Definition 1) kept in LDS
//    with threshold rejection;
//  - kEpiDense: a dense phi store;
//  - kEpiBounded: the same top-k over the items that can reach a per-query
//    bound: phi is a convex combination of the s_p, so phi <= m = max_p s_p,
//    and an item whose m (plus a rounding margin) stays below the bound, or
//    below the running k-th score, cannot be in the result.  Groups of 16
//    items where no item can are skipped before the gating MLP (Algorithm 1's
//    RangeDotProduct + BruteForceTopKMoL in one pass);
//  - kEpiMaxDot: a running top-k of m itself, without the gating MLP
//    (Section 3's max approximation of MoL, a subsection cut from the
//    published text);
//  - kEpiTopkPipe: kEpiTopk as a software-pipelined loop (each step's
//    softmax tail issued with the next step's GEMM1); a step whose softmax
//    sum leaves its safe range flags its workgroup's range, which a second
//    launch of kEpiTopk rescores.
//
// Workgroup: 8 waves (2 per SIMD) = 16 queries sharing an LDS-staged
// stream of 32-item tiles (a three-deep ring) loaded with direct
// global->LDS copies.  The max-dot form stages 16-item tiles, gives each
// wave four queries (32 per workgroup, one workgroup per CU) and takes m
// straight from GEMM1's tiles without splitting the queries.
#include "mol_tile.h"

namespace mol {

using namespace tile;

namespace {

enum FusedEpi { kEpiTopk = 0, kEpiDense = 1, kEpiBounded = 2, kEpiMaxDot = 3, kEpiTopkPipe = 4 };

constexpr int kWaves = 8;
constexpr int kQueriesPerWG = 2 * kWaves;   // the gating forms
// queries per wave: two in the gating forms; four in the max-dot form, whose
// step is GEMM1 alone: each LDS read of the X tile then feeds two GEMM1s (the
// 64 KB of top-k lists leave one workgroup per CU; at exact_1m 9.5 ms against
// 9.8 ms for two queries per wave and two workgroups per CU)
template <bool AX>
constexpr int queries_per_wave() { return AX ? 2 : 4; }
// items per LDS stage: two 16-item steps with the gating MLP; one step in
// the max-dot form (no a_x stream)
template <bool AX>
constexpr int tile_items() { return AX ? 32 : 16; }
constexpr int kRing = 3;         // item stages in flight
constexpr int kTopkRegion = WaveTopk::kList + WaveTopk::kStage;

// PX, D, H: shape; AX: the gating inputs (a_x stream, a_q + b2) are needed
template <int PX, int D, int H, bool AX>
struct FusedShape {
  static constexpr int P = 8 * PX;
  static constexpr int TILE = tile_items<AX>();
  static constexpr int RUN = 2 * PX;     // s values per lane per query
  static constexpr int KD = D / 32;      // K blocks of GEMM1
  static constexpr int PT = P / 16;      // output tiles of GEMM3
  static constexpr int XROWCH = D / 8;   // 16-byte chunks per X row
  static constexpr int AROWCH = P / 4;   // 16-byte chunks per a_x row
  static constexpr int XSTAGE = PX * TILE * D * 2;   // bytes of one X stage
  static constexpr int ASTAGE = AX ? TILE * P * 4 : 0;   // bytes of one a_x stage
  static constexpr int LDS_X = kRing * XSTAGE;
  static constexpr int LDS_AX = kRing * ASTAGE;
  static constexpr int LDS_CB = AX ? kQueriesPerWG * P * 4 : 0;   // [query][p] log2(e) (a_q + b2), f32
  static constexpr int QPW = queries_per_wave<AX>();   // queries per wave
  static constexpr int QWG = QPW * kWaves;             // queries per workgroup
  static constexpr int LDS_TOPK = QWG * kTopkRegion * 8;
  static constexpr int LDS_TOTAL = LDS_X + LDS_AX + LDS_CB + LDS_TOPK;
  // 16-byte global->LDS copies per stage, in 1 KB blocks of one wave each
  static constexpr int XBLOCKS = XSTAGE / 1024;
  static constexpr int ABLOCKS = ASTAGE / 1024;
  static_assert(XBLOCKS % kWaves == 0, "X stage must split evenly over the waves");
  // fewest copies any wave issues per stage (a_x blocks may not split evenly)
  static constexpr int LOADS = XBLOCKS / kWaves + ABLOCKS / kWaves;
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

}  // namespace

template <int PX, int D, int H, int EPI, bool X2>
__global__ __launch_bounds__(64 * kWaves, 1) void k_mol_fused(
    DevProb pr, int k, int R, int range_len, int G, int n_begin, int n_end,
    const float* __restrict__ bound, uint64_t* __restrict__ partial, float* __restrict__ phi_out,
    long phi_stride, int* __restrict__ redo) {
  constexpr bool DENSE = EPI == kEpiDense;
  constexpr bool MLP = EPI != kEpiMaxDot;
  // software-pipelined top-k scan
  constexpr bool PIPE = EPI == kEpiTopkPipe;
  using S = FusedShape<PX, D, H, MLP>;
  // X2: the two-term chain (plain loop only: top-k, dense and bounded forms)
  static_assert(!X2 || EPI == kEpiTopk || EPI == kEpiDense || EPI == kEpiBounded, "two-term forms");
  using Mlp = MolMlp<PX, H, X2>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* sX = smem;
  unsigned char* sAx = smem + S::LDS_X;
  float* sCb = reinterpret_cast<float*>(smem + S::LDS_X + S::LDS_AX);
  uint64_t* sTop = reinterpret_cast<uint64_t*>(smem + S::LDS_X + S::LDS_AX + S::LDS_CB);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int c = lane & 15, g = lane >> 4;
  const int base = lane_base(g, PX);
  // second launch after the pipelined scan: only the workgroups whose
  // range it flagged run (uniform per workgroup, before any barrier)
  if (EPI == kEpiTopk && redo) {
    int any = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) any |= redo[blockIdx.x * kWaves + w];
    if (!any) return;
  }
  int r, qg;
  wg_coords(blockIdx.x, R, G, r, qg);
  const int qwg = qg * S::QWG;            // first query of the workgroup
  const int qwv = qwg + S::QPW * wave;    // first of this wave's QPW queries
  const int nr0 = n_begin + r * range_len;
  const int nr1 = min(n_end, nr0 + range_len);
  const int ntiles = nr1 > nr0 ? (nr1 - nr0 + S::TILE - 1) / S::TILE : 0;
  const int N = pr.N;
  constexpr int P = S::P;

  const bf16_t* X = static_cast<const bf16_t*>(pr.X);
  const bf16_t* Q = static_cast<const bf16_t*>(pr.Q);

  // ---- stage tile t into LDS buffer buf with direct global->LDS copies ----
  // X stage layout [px][item][16-byte chunk ^ (item % XROWCH)], a_x stage
  // [item][16-byte chunk ^ (item % AROWCH)].  Lane i of a copy writes LDS
  // bytes 16 i of its 1 KB block, so the global side picks the chunk that
  // belongs there.  Items past the end are clamped to N-1 (valid memory,
  // masked later).
  auto stage = [&](int t, int buf) {
    const int n0 = nr0 + S::TILE * t;
#pragma unroll
    for (int cp = 0; cp < S::XBLOCKS / kWaves; ++cp) {
      const int blk = wave + kWaves * cp;
      const int pos = blk * 64 + lane;
      const int px = pos / (S::TILE * S::XROWCH);
      const int rem = pos % (S::TILE * S::XROWCH);
      const int n = rem / S::XROWCH, phys = rem % S::XROWCH;
      const int cc = phys ^ (n % S::XROWCH);
      const int item = min(n0 + n, N - 1);
      const bf16_t* src = X + (static_cast<long>(px) * N + item) * D + 8 * cc;
      unsigned char* dst = sX + buf * S::XSTAGE + blk * 1024;
      copy16_to_lds(src, lds_addr(dst));
    }
    for (int blk = wave; MLP && blk < S::ABLOCKS; blk += kWaves) {
      const int pos = blk * 64 + lane;
      const int n = pos / S::AROWCH, phys = pos % S::AROWCH;
      const int cc = phys ^ (n % S::AROWCH);
      const int item = min(n0 + n, N - 1);
      const float* src = pr.a_x + static_cast<long>(item) * P + 4 * cc;
      unsigned char* dst = sAx + buf * S::ASTAGE + blk * 1024;
      copy16_to_lds(src, lds_addr(dst));
    }
  };
  for (int t = 0; t < kRing - 1 && t < ntiles; ++t) stage(t, t);

  // ---- per-workgroup constants ----
  // log2(e) (a_q + b2) per query of the workgroup, [query][p]
  if (MLP)
    for (int i = tid; i < kQueriesPerWG * P; i += 64 * kWaves) {
      const int qi = i / P, p = i % P, b = qwg + qi;
      sCb[i] = b < pr.B ? kLog2e * (pr.a_q[static_cast<long>(b) * P + p] + pr.b2[p]) : 0.f;
    }
  WaveTopk top[S::QPW];
  if (!DENSE) {
#pragma unroll
    for (int qb = 0; qb < S::QPW; ++qb) top[qb].init(sTop + (S::QPW * wave + qb) * kTopkRegion, k, lane);
  }
  // per-query bound of the bounded epilogue (queries past B: +inf, skipped)
  float qbound[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
    qbound[qb] = EPI == kEpiBounded && qwv + qb < pr.B ? bound[qwv + qb] : __builtin_inff();
  Mlp mlp;
  if (MLP) mlp.load(pr, c, g);
  // Q as GEMM1 A operands: row c = 2 pq + q (gating forms) or 8 q + pq
  // (max-dot form, queries 2 h and 2 h + 1 in set h), K slot 8g+e <-> d =
  // 32 kk + 8 g + e
  uint4 qop[S::QPW / 2][S::KD];
#pragma unroll
  for (int h = 0; h < S::QPW / 2; ++h) {
    const int b = MLP ? qwv + (c & 1) : qwv + 2 * h + (c >> 3), pq = MLP ? c >> 1 : c & 7;
#pragma unroll
    for (int kk = 0; kk < S::KD; ++kk)
      qop[h][kk] = b < pr.B
                       ? *reinterpret_cast<const uint4*>(Q + (static_cast<long>(b) * 8 + pq) * D + 32 * kk + 8 * g)
                       : make_uint4(0, 0, 0, 0);
  }

  // stage 0 complete; later stages' copies may still be in flight
  if (ntiles >= kRing - 1) ring_barrier<(kRing - 2) * S::LOADS>();
  else ring_barrier<0>();

  if constexpr (PIPE) {
    // Software-pipelined top-k scan.  Each step's chain is split
    // in two: stage A (both queries' GEMM2 -> SiLU -> GEMM3 and query 0's
    // softmax sums) and stage B (query 1's softmax sums and the sums over an
    // item's four lanes).  Stage B of step s is issued in one scheduling
    // region with the LDS reads and GEMM1 of step s + 1, so that GEMM1's
    // matrix instructions run under the wave's own vector work; then step s
    // is finished (reciprocal, top-k offers) and stage A of step s + 1
    // follows.  The arithmetic of every pair is that of phi2_interleaved.
    //
    // Ring discipline: one barrier per stage, in the step that is about to
    // read the next stage.  A stage is last read in the first step of its
    // own tile (the second step's reads are issued one step earlier), so past
    // the barrier of tile t's second step every wave is done with tile t - 1
    // and its buffer is refilled right away.
    auto x_reads = [&](int t, int st, uint4(&xb)[PX][S::KD]) {
      const unsigned char* xs = sX + (t % kRing) * S::XSTAGE;
      const int n = 16 * st + c;
#pragma unroll
      for (int px = 0; px < PX; ++px) {
        const unsigned char* row = xs + (px * S::TILE + n) * (D * 2);
#pragma unroll
        for (int kk = 0; kk < S::KD; ++kk) {
          const int phys = (4 * kk + g) ^ (n % S::XROWCH);
          xb[px][kk] = *reinterpret_cast<const uint4*>(row + 16 * phys);
        }
      }
    };
    auto ax_reads = [&](int t, int st, float4(&axv)[S::PT]) {
      const unsigned char* as = sAx + (t % kRing) * S::ASTAGE;
      const int n = 16 * st + c;
#pragma unroll
      for (int q4 = 0; q4 < S::PT; ++q4) {
        const int phys = (base / 4 + q4) ^ (n % S::AROWCH);
        axv[q4] = *reinterpret_cast<const float4*>(as + n * (P * 4) + 16 * phys);
      }
    };
    // GEMM1: accumulator row 4 g + i is pq = 2 g + i / 2 of query i % 2
    auto gemm1 = [&](const uint4(&xb)[PX][S::KD], float(&s2)[2][S::RUN]) {
      f32x4_t acc1[PX];
#pragma unroll
      for (int px = 0; px < PX; ++px) {
        acc1[px] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < S::KD; ++kk) acc1[px] = mfma_bf16(qop[0][kk], xb[px][kk], acc1[px]);
      }
#pragma unroll
      for (int mu = 0; mu < S::RUN; ++mu) {
        s2[0][mu] = acc1[mu % PX][2 * (mu / PX)];
        s2[1][mu] = acc1[mu % PX][2 * (mu / PX) + 1];
      }
    };
    // GEMM3 accumulator inputs of both queries: log2(e) a_x + log2(e) (a_q + b2)
    auto gate_bias2 = [&](const float4(&axv)[S::PT], f32x4_t(&c0)[2][S::PT]) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt) {
          const float4 cb = *reinterpret_cast<const float4*>(sCb + (2 * wave + qb) * P + base + 4 * pt);
          c0[qb][pt] = f32x4_t{fmaf(axv[pt].x, kLog2e, cb.x), fmaf(axv[pt].y, kLog2e, cb.y),
                               fmaf(axv[pt].z, kLog2e, cb.z), fmaf(axv[pt].w, kLog2e, cb.w)};
        }
    };
    bool redo_wave = false;
    f32x4_t lg1[S::PT];     // query 1's logits of the step in flight
    float s1[S::RUN];       // query 1's dot products of the step in flight
    float den0 = 0.f, num0 = 0.f;
    if (ntiles > 0) {
      uint4 xb[PX][S::KD];
      float4 axv[S::PT];
      float s2[2][S::RUN];
      f32x4_t c0[2][S::PT];
      x_reads(0, 0, xb);
      ax_reads(0, 0, axv);
      gemm1(xb, s2);
      gate_bias2(axv, c0);
      mlp.template phi2_stage_a<5>(s2, c0, lg1, den0, num0);
#pragma unroll
      for (int mu = 0; mu < S::RUN; ++mu) s1[mu] = s2[1][mu];
    }
    for (int t = 0; t < ntiles; ++t) {
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int item = nr0 + S::TILE * t + 16 * st + c;
        const bool item_ok = item < nr1;
        const bool has_next = st == 0 || t + 1 < ntiles;
        if (st == 1 && t + 1 < ntiles) {
          ring_barrier<0>();
          if (t + 2 < ntiles) stage(t + 2, (t + 2) % kRing);
        }
        // the next step's X reads and GEMM1 with this step's stage B (past
        // the last step the current step's stage is read again, unused)
        const int tn = st == 0 ? t : (has_next ? t + 1 : t), stn = st == 0 ? 1 : (has_next ? 0 : 1);
        float s2n[2][S::RUN];
        float Dn, Nm;
        __builtin_amdgcn_sched_barrier(0);
        {
          uint4 xb[PX][S::KD];
          x_reads(tn, stn, xb);
          gemm1(xb, s2n);
        }
        mlp.phi2_stage_b(lg1, s1, den0, num0, Dn, Nm);
        {
          constexpr int kMfma = 0x008, kValu = 0x002 | 0x400, kDsRead = 0x100;
          // the X reads, then some of stage B's vector instructions while
          // they land, then the MFMAs each followed by vector instructions
          // (A/B: H = 64, exact_1m, 0 / 8 / 16 / 20 / 24 leading and two per
          // MFMA: 38.4 / 38.2 / 38.0 / 37.7 / 38.2 ms; H = 128, hybrid_8m,
          // whose stage B is shorter (P = 32): 20 and two per MFMA 86.9 ms,
          // 16 and one 86.1, none 88.8 without pipelining)
          constexpr int kLead = H > 64 ? 16 : 20, kPer = H > 64 ? 1 : 2;
          __builtin_amdgcn_sched_group_barrier(kDsRead, PX * S::KD, 0);
          __builtin_amdgcn_sched_group_barrier(kValu, kLead, 0);
#pragma unroll
          for (int i = 0; i < PX * S::KD; ++i) {
            __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kValu, kPer, 0);
          }
        }
        // the next step's dot products are read after the branches below
        mfma_drain();
        // the next step's a_x reads go out before the offers, which then
        // cover their LDS latency
        float4 axv[S::PT];
        ax_reads(tn, stn, axv);
        // finish this step.  A sum outside [2^-60, 2^60] (logits far from
        // zero) marks the wave: its workgroup's range is then scored again by
        // the non-pipelined scan, which subtracts the row maximum (this
        // launch's lists of that range are overwritten)
        const float v = Nm * __builtin_amdgcn_rcpf(Dn);
        redo_wave |= !__all(Dn >= 0x1p-60f && Dn <= 0x1p60f);
        // one ballot decides whether either query has a candidate
        {
          const bool m0 = g == 0 && item_ok && v >= top[0].theta_score;
          const bool m1 = g == 2 && item_ok && v >= top[1].theta_score;
          if (__ballot(m0 || m1)) {
            top[0].offer(m0 ? make_key(v, item) : 0ull, lane);
            top[1].offer(m1 ? make_key(v, item) : 0ull, lane);
          }
        }
        if (has_next) {
          f32x4_t c0[2][S::PT];
          gate_bias2(axv, c0);   // 2 PT LDS reads of a_q + b2
          mlp.template phi2_stage_a<5, 2 * S::PT>(s2n, c0, lg1, den0, num0);
        }
        // unconditional (past the last step s1 is dead): a copy under
        // has_next cost 32 register moves per two steps
#pragma unroll
        for (int mu = 0; mu < S::RUN; ++mu) s1[mu] = s2n[1][mu];
      }
    }
    if (lane == 0) redo[blockIdx.x * kWaves + wave] = redo_wave ? 1 : 0;
  } else {
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t % kRing;
    const unsigned char* xs = sX + buf * S::XSTAGE;
    const unsigned char* as = sAx + buf * S::ASTAGE;

#pragma unroll
    for (int st = 0; st < S::TILE / 16; ++st) {
      const int n = 16 * st + c;            // item within the stage
      const int item = nr0 + S::TILE * t + n;
      const bool item_ok = item < nr1;

      // LDS operands of the step, all issued before the first MFMA so that
      // one LDS round trip is exposed per step: the X tile (GEMM1 B
      // operands) and a_x
      uint4 xb[PX][S::KD];
#pragma unroll
      for (int px = 0; px < PX; ++px) {
        const unsigned char* row = xs + (px * S::TILE + n) * (D * 2);
#pragma unroll
        for (int kk = 0; kk < S::KD; ++kk) {
          const int phys = (4 * kk + g) ^ (n % S::XROWCH);
          xb[px][kk] = *reinterpret_cast<const uint4*>(row + 16 * phys);
        }
      }
      float4 axv[S::PT];
#pragma unroll
      for (int q4 = 0; q4 < S::PT; ++q4) {
        const int phys = (base / 4 + q4) ^ (n % S::AROWCH);
        axv[q4] = MLP ? *reinterpret_cast<const float4*>(as + n * (P * 4) + 16 * phys)
                      : float4{0.f, 0.f, 0.f, 0.f};
      }
      __builtin_amdgcn_sched_barrier(0);

      // GEMM1: the wave's queries (set h: two of them) x 16 items x all px
      __builtin_amdgcn_s_setprio(1);
      f32x4_t acc1[PX], acc2[PX];
#pragma unroll
      for (int px = 0; px < PX; ++px) {
        acc1[px] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        acc2[px] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < S::KD; ++kk) {
          acc1[px] = mfma_bf16(qop[0][kk], xb[px][kk], acc1[px]);
          if constexpr (S::QPW == 4) acc2[px] = mfma_bf16(qop[S::QPW / 2 - 1][kk], xb[px][kk], acc2[px]);
        }
      }
      mfma_priority_end();
      // the two queries' runs: s2[q][mu] holds p = base(g) + mu
      float s2[2][S::RUN];
      float mrow[2] = {0.f, 0.f};
      if constexpr (EPI == kEpiMaxDot) {
        // no split: lane group g holds query 2 h + g / 2's rows pq = 4 (g % 2)
        // .. + 3 for every px, so the maximum over its 4 PX values and the
        // other group of the query (one permlane16 swap) is m, valid in the
        // lanes of rows 2 q and 2 q + 1 as the offers expect
#pragma unroll
        for (int h = 0; h < S::QPW / 2; ++h) {
          const f32x4_t(&acc)[PX] = h == 0 ? acc1 : acc2;
          float mx = acc[0][0];
#pragma unroll
          for (int px = 0; px < PX; ++px)
#pragma unroll
            for (int e = 0; e < 4; ++e) mx = fmaxf(mx, acc[px][e]);
          const uint32_t u = __float_as_uint(mx);
          auto sw = __builtin_amdgcn_permlane16_swap(u, u, false, false);
          mrow[h] = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        }
      } else {
        // accumulator row 4 g + i is pq = 2 g + i / 2 of query i % 2, i.e.
        // p = base(g) + (i / 2) PX + px
#pragma unroll
        for (int mu = 0; mu < S::RUN; ++mu) {
          s2[0][mu] = acc1[mu % PX][2 * (mu / PX)];
          s2[1][mu] = acc1[mu % PX][2 * (mu / PX) + 1];
        }
      }
      float phi[S::QPW];
      bool offer[S::QPW];
      bool need[2] = {true, true};   // bounded form: the query's chain runs
#pragma unroll
      for (int qb = 0; qb < S::QPW; ++qb) offer[qb] = item_ok;
      // GEMM3 accumulator input of query qb: log2(e) a_x (the item's, from
      // the stage) + log2(e) (a_q + b2) (the query's), at the lane's
      // p = base(g) + 4 pt + i
      auto gate_bias = [&](int qb, f32x4_t(&c0)[S::PT]) {
#pragma unroll
        for (int pt = 0; pt < S::PT; ++pt) {
          const float4 cb = *reinterpret_cast<const float4*>(sCb + (2 * wave + qb) * P + base + 4 * pt);
          c0[pt] = f32x4_t{fmaf(axv[pt].x, kLog2e, cb.x), fmaf(axv[pt].y, kLog2e, cb.y),
                           fmaf(axv[pt].z, kLog2e, cb.z), fmaf(axv[pt].w, kLog2e, cb.w)};
        }
      };
      if constexpr (EPI == kEpiTopk || EPI == kEpiDense) {
        // both queries' MLP chains in one call: interleaved by hand where the
        // matrix chains are short against the SiLU work (H <= 64), else
        // left to the compiler with raised priority around each chain
        if constexpr (X2) {
          // the two-term chains one query after the other, each with its own
          // gate inputs: both at once spilled 3-12 VGPRs (exact_1m_skewed
          // top-k 60.3 ms against 54.4 ms this way)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            float sq[1][S::RUN];
#pragma unroll
            for (int mu = 0; mu < S::RUN; ++mu) sq[0][mu] = s2[qb][mu];
            f32x4_t c0[1][S::PT];
            gate_bias(qb, c0[0]);
            float pq[1];
            mlp.template phi<1>(sq, c0, pq);
            phi[qb] = pq[0];
            __builtin_amdgcn_sched_barrier(0);
          }
        } else {
          f32x4_t c0[2][S::PT];
          gate_bias(0, c0[0]);
          gate_bias(1, c0[1]);
          if constexpr (H <= 64) mlp.template phi2_interleaved<5>(s2, c0, phi);
          else mlp.template phi<2>(s2, c0, phi);
        }
      }
#pragma unroll
      for (int qb = 0; qb < 2 && (EPI == kEpiBounded || EPI == kEpiMaxDot); ++qb) {
        if constexpr (EPI == kEpiMaxDot) {
          phi[qb] = mrow[0];
          phi[qb + 2] = mrow[1];
          continue;
        }
        if constexpr (EPI == kEpiBounded) {
          // m = max_p s_p of the lane's item
          float m = s2[qb][0];
#pragma unroll
          for (int mu = 1; mu < S::RUN; ++mu) m = fmaxf(m, s2[qb][mu]);
          m = max_groups(m);
          const float floor = fmaxf(qbound[qb], top[qb].theta_score);
          // |m| <= max_p |s_p|: passing with the margin of |m| is passing
          bool pass = m + bound_margin(fabsf(m)) >= floor;
          if (!__all(pass || !item_ok)) {
            // the margin of max_p |s_p| decides the rest
            float mabs = fabsf(s2[qb][0]);
#pragma unroll
            for (int mu = 1; mu < S::RUN; ++mu) mabs = fmaxf(mabs, fabsf(s2[qb][mu]));
            mabs = max_groups(mabs);
            pass = m + bound_margin(mabs) >= floor;
          }
          offer[qb] = item_ok && pass;
          phi[qb] = -__builtin_inff();
          need[qb] = __any(offer[qb]);   // some item of the group can qualify
        }
      }
      if constexpr (EPI == kEpiBounded) {
        if (need[0] && need[1] && !X2) {
          // both chains run: as one two-query call (the same arithmetic; the
          // two-term form takes the per-query calls below, whose registers fit)
          f32x4_t c0[2][S::PT];
          gate_bias(0, c0[0]);
          gate_bias(1, c0[1]);
          if constexpr (H <= 64 && !X2) mlp.template phi2_interleaved<5>(s2, c0, phi);
          else mlp.template phi<2>(s2, c0, phi);
        } else {
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            if (!need[qb]) continue;
            float sq[1][S::RUN];
#pragma unroll
            for (int mu = 0; mu < S::RUN; ++mu) sq[0][mu] = s2[qb][mu];
            f32x4_t c0[1][S::PT];
            gate_bias(qb, c0[0]);
            float pq[1];
            mlp.template phi<1>(sq, c0, pq);
            phi[qb] = pq[0];
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
      // phi[qb] is valid in the lanes of rows 2 (qb % 2) and 2 (qb % 2) + 1
      // (the two-query chain and the max-dot sets leave each query's result
      // there; the other forms in every lane)
#pragma unroll
      for (int qb = 0; qb < S::QPW; ++qb) {
        const int b = qwv + qb;
        if constexpr (DENSE) {
          if (g == 2 * qb && item_ok && b < pr.B) phi_out[b * phi_stride + (item - n_begin)] = phi[qb];
        } else {
          top[qb].offer_score(phi[qb], item, g == 2 * (qb % 2) && offer[qb], lane);
        }
      }
    }
    // refill the buffer read in iteration t-1, then wait for stage t+1
    if (t + kRing - 1 < ntiles) {
      stage(t + kRing - 1, (t + kRing - 1) % kRing);
      ring_barrier<(kRing - 2) * S::LOADS>();
    } else {
      ring_barrier<0>();
    }
  }
  }

  if constexpr (!DENSE) {
#pragma unroll
    for (int qb = 0; qb < S::QPW; ++qb) {
      top[qb].flush(lane);
      const int b = qwv + qb;
      if (b < pr.B) {
        uint64_t* dst = partial + (static_cast<long>(b) * R + r) * k;
        for (int i = lane; i < k; i += 64) dst[i] = top[qb].reg[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
static bool fused_shape(const DevProb& pr, bool mlp) {
  if (pr.dtype != MOL_BF16 || pr.Pq != 8) return false;
  if (pr.Px == 8 && (pr.d == 64 || pr.d == 32)) return !mlp || pr.H == 64;
  if (pr.Px == 4 && pr.d == 64) return !mlp || pr.H == 64;
  if (pr.Px == 4 && pr.d == 128) return !mlp || pr.H == 128;
  return false;
}

bool fused_supported(const DevProb& pr, int k) {
  return !(pr.flags & MOL_FLAG_F32_GATING) && fused_shape(pr, true) && k <= WaveTopk::kList;
}
bool fused_maxdot_supported(const DevProb& pr, int k) {
  return fused_shape(pr, false) && k <= WaveTopk::kList;
}

void fused_grid(const DevProb& pr, int n_count, int& R, int& range_len, int& G, bool maxdot) {
  const int qwg = queries_per_wave<false>() * kWaves;   // max-dot form
  G = maxdot ? (pr.B + qwg - 1) / qwg : (pr.B + kQueriesPerWG - 1) / kQueriesPerWG;
  // about one workgroup per CU
  R = std::max(1, 256 / G);
  // ranges of at least 128 items (4 tiles): small corpora still fill the chip
  const int max_r = std::max(1, n_count / 128);
  R = std::min(R, max_r);
  range_len = (n_count + R - 1) / R;
  range_len = (range_len + 31) / 32 * 32;   // whole stages of either form
  R = (n_count + range_len - 1) / range_len;
}

template <int PX, int D, int H, int EPI, bool X2>
static hipError_t launch_fused_x(const DevProb& pr, int k, int R, int range_len, int G, int n_begin,
                                 int n_end, const float* bound, uint64_t* partial, float* phi,
                                 long phi_stride, int* redo, hipStream_t st) {
  using S = FusedShape<PX, D, H, EPI != kEpiMaxDot>;
  auto kern = &k_mol_fused<PX, D, H, EPI, X2>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, S::LDS_TOTAL);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(R * G), dim3(64 * kWaves), S::LDS_TOTAL, st, pr, k, R, range_len,
                     G, n_begin, n_end, bound, partial, phi, phi_stride, redo);
  return hipGetLastError();
}

// the two-term chain where the problem asks for it (MOL_FLAG_BF16X2_GATING)
template <int PX, int D, int H, int EPI>
static hipError_t launch_fused_t(const DevProb& pr, int k, int R, int range_len, int G, int n_begin,
                                 int n_end, const float* bound, uint64_t* partial, float* phi,
                                 long phi_stride, int* redo, hipStream_t st) {
  if constexpr (EPI == kEpiTopk || EPI == kEpiDense || EPI == kEpiBounded) {
    if (pr.flags & MOL_FLAG_BF16X2_GATING)
      return launch_fused_x<PX, D, H, EPI, true>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                                 phi_stride, redo, st);
  }
  return launch_fused_x<PX, D, H, EPI, false>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                              phi_stride, redo, st);
}

template <int EPI>
static hipError_t launch_fused_d(const DevProb& pr, int k, int R, int range_len, int G, int n_begin,
                                 int n_end, const float* bound, uint64_t* partial, float* phi,
                                 long phi_stride, int* redo, hipStream_t st) {
  // the max-dot epilogue has no gating MLP: one instantiation per (Px, d)
  if (pr.Px == 8 && pr.d == 32)
    return launch_fused_t<8, 32, 64, EPI>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                          phi_stride, redo, st);
  if (pr.Px == 8)
    return launch_fused_t<8, 64, 64, EPI>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                          phi_stride, redo, st);
  if (pr.d == 128)
    return launch_fused_t<4, 128, 128, EPI>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                            phi_stride, redo, st);
  return launch_fused_t<4, 64, 64, EPI>(pr, k, R, range_len, G, n_begin, n_end, bound, partial, phi,
                                        phi_stride, redo, st);
}

long fused_redo_flags(int R, int G) { return static_cast<long>(R) * G * kWaves; }

hipError_t launch_fused_topk(const DevProb& pr, int k, int R, int range_len, int G,
                             const float* bound, uint64_t* partial, int* redo, hipStream_t st) {
  if (bound)
    return launch_fused_d<kEpiBounded>(pr, k, R, range_len, G, 0, pr.N, bound, partial, nullptr, 0, nullptr,
                                       st);
  if (redo && !(pr.flags & MOL_FLAG_BF16X2_GATING)) {
    // pipelined scan, then the plain scan over the ranges it flagged
    hipError_t e = launch_fused_d<kEpiTopkPipe>(pr, k, R, range_len, G, 0, pr.N, nullptr, partial, nullptr, 0,
                                                redo, st);
    if (e != hipSuccess) return e;
    return launch_fused_d<kEpiTopk>(pr, k, R, range_len, G, 0, pr.N, nullptr, partial, nullptr, 0, redo, st);
  }
  return launch_fused_d<kEpiTopk>(pr, k, R, range_len, G, 0, pr.N, nullptr, partial, nullptr, 0, nullptr, st);
}

hipError_t launch_fused_maxdot(const DevProb& pr, int k, int R, int range_len, int G,
                               uint64_t* partial, hipStream_t st) {
  return launch_fused_d<kEpiMaxDot>(pr, k, R, range_len, G, 0, pr.N, nullptr, partial, nullptr, 0, nullptr,
                                    st);
}

hipError_t launch_fused_dense(const DevProb& pr, int n_begin, int n_count, float* phi,
                              hipStream_t st) {
  int R, range_len, G;
  fused_grid(pr, n_count, R, range_len, G, false);
  return launch_fused_d<kEpiDense>(pr, 1, R, range_len, G, n_begin, n_begin + n_count, nullptr, nullptr,
                                   phi, n_count, nullptr, st);
}

}  // namespace mol
