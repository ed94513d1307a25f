// Generic gfx950 kernels of the MoL library: one thread per (query, item)
// pair, float32 arithmetic, any supported shape and both storage types.
// They serve the float32 problems and every shape the MFMA kernels do not
// cover, and provide the selection machinery (segmented bitonic top-k,
// key decoding), the candidate deduplication of the approximate path and
// the TopKAvg materialisation.
#include "mol_kernels.h"

namespace mol {

// ---------------------------------------------------------------------------
// MoL score of one (query, item) pair, float32 (Eq. 1 with the two-layer
// SiLU gating MLP of Appendix A.3).  Gating weights live in LDS as float32,
// rows padded with zeros to PMAX so that a row is read as aligned 16-byte
// vectors (every lane reads the same address: one broadcast per read):
// sW1 [H][PMAX] = W1, sW2t [H][PMAX] = W2 transposed, sb1 [H],
// sc [PMAX] = a_q[b] + b2.
// ---------------------------------------------------------------------------
template <typename T, int PMAX>
__device__ __forceinline__ void pair_dots(const DevProb& pr, int b, long n, float (&s)[PMAX]) {
  const T* Qb = static_cast<const T*>(pr.Q) + static_cast<long>(b) * pr.Pq * pr.d;
  const T* Xn = static_cast<const T*>(pr.X) + n * pr.d;
  const long xstride = static_cast<long>(pr.N) * pr.d;
#pragma unroll
  for (int p = 0; p < PMAX; ++p) {
    s[p] = 0.f;
    if (p < pr.P) {
      const int pq = p / pr.Px, px = p - (p / pr.Px) * pr.Px;
      const T* q = Qb + pq * pr.d;
      const T* x = Xn + px * xstride;
      float acc = 0.f;
      for (int t = 0; t < pr.d; ++t) acc = fmaf(to_f32(q[t]), to_f32(x[t]), acc);
      s[p] = acc;
    }
  }
}

template <int PMAX>
__device__ __forceinline__ float pair_phi(const DevProb& pr, long n, const float (&s)[PMAX],
                                          const float* sW1, const float* sW2t,
                                          const float* sb1, const float* sc) {
  constexpr float kLog2e = 1.4426950408889634f;
  const int P = pr.P, H = pr.H;
  float l[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) l[p] = (p < P) ? sc[p] + pr.a_x[n * P + p] : 0.f;
  for (int j = 0; j < H; ++j) {
    const float* w1 = sW1 + j * PMAX;
    const float* w2 = sW2t + j * PMAX;
    float u = sb1[j];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) u = fmaf(w1[p], s[p], u);   // padded slots are zero
    // SiLU: u sigma(u), sigma(u) = 1 / (1 + e^-u)
    const float h = u * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-kLog2e * u));
#pragma unroll
    for (int p = 0; p < PMAX; ++p) l[p] = fmaf(w2[p], h, l[p]);
  }
  float m = l[0];
#pragma unroll
  for (int p = 1; p < PMAX; ++p)
    if (p < P) m = fmaxf(m, l[p]);
  float den = 0.f, num = 0.f;
#pragma unroll
  for (int p = 0; p < PMAX; ++p) {
    if (p < P) {
      const float w = __builtin_amdgcn_exp2f(kLog2e * (l[p] - m));
      den += w;
      num = fmaf(w, s[p], num);
    }
  }
  return num * __builtin_amdgcn_rcpf(den);
}

// Grid: x over items (256 per block), y over queries.  Items are either the
// contiguous range n_begin .. n_begin+n_count-1 or, when `items` is given,
// items[b*item_stride + i] for i < item_count[b].  Writes a score (float32)
// and/or sort keys; key slots past a query's item count are cleared to 0
// (empty).  The score is, by `mode`:
//   kGenPhi      phi;
//   kGenBounded  phi, for items whose m = max_p s_p plus the rounding
//                margin reaches bound[b] (phi <= m: Algorithm 1's range
//                condition); other items get an empty key;
//   kGenMaxDot   m itself (no gating MLP);
//   kGenNegPhi   -phi (the smallest phi as the top-1 of the negated keys).
template <typename T, int PMAX>
__global__ __launch_bounds__(256) void k_phi_generic(
    DevProb pr, int mode, const float* __restrict__ bound, int n_begin, int n_count,
    const int32_t* __restrict__ items, const int32_t* __restrict__ item_count, long item_stride,
    const float* __restrict__ sbuf, long s_pstride, long s_bstride,
    float* __restrict__ phi, long phi_stride, uint64_t* __restrict__ keys, long key_stride) {
  extern __shared__ float smem[];
  const int P = pr.P, H = pr.H;
  float* sW1 = smem;
  float* sW2t = sW1 + H * PMAX;
  float* sb1 = sW2t + H * PMAX;
  float* sc = sb1 + H;
  const int b = blockIdx.y;
  if (mode != kGenMaxDot) {
    for (int i = threadIdx.x; i < H * PMAX; i += blockDim.x) {
      const int j = i / PMAX, p = i - (i / PMAX) * PMAX;
      sW1[i] = p < P ? to_f32(static_cast<const T*>(pr.W1)[j * P + p]) : 0.f;
      sW2t[i] = p < P ? to_f32(static_cast<const T*>(pr.W2)[p * H + j]) : 0.f;
    }
    for (int i = threadIdx.x; i < H; i += blockDim.x) sb1[i] = pr.b1[i];
    for (int i = threadIdx.x; i < PMAX; i += blockDim.x)
      sc[i] = i < P ? pr.a_q[static_cast<long>(b) * P + i] + pr.b2[i] : 0.f;
  }
  __syncthreads();

  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_count) return;
  const int cnt = items ? item_count[b] : n_count;
  if (i >= cnt) {
    if (keys) keys[b * key_stride + i] = 0;
    return;
  }
  const long n = items ? static_cast<long>(items[b * item_stride + i]) : static_cast<long>(n_begin) + i;
  float s[PMAX];
  if (sbuf) {   // dot products formed by the MFMA kernel
#pragma unroll
    for (int p = 0; p < PMAX; ++p) s[p] = p < P ? sbuf[p * s_pstride + b * s_bstride + i] : 0.f;
  } else {
    pair_dots<T, PMAX>(pr, b, n, s);
  }
  float v;
  if (mode == kGenBounded || mode == kGenMaxDot) {
    float m = s[0], mabs = fabsf(s[0]);
#pragma unroll
    for (int p = 1; p < PMAX; ++p)
      if (p < P) {
        m = fmaxf(m, s[p]);
        mabs = fmaxf(mabs, fabsf(s[p]));
      }
    if (mode == kGenMaxDot) {
      v = m;
    } else if (m + 0x1p-12f * (1.f + mabs) < bound[b]) {   // phi <= m: cannot reach the bound
      if (phi) phi[b * phi_stride + i] = -__builtin_inff();
      if (keys) keys[b * key_stride + i] = 0;
      return;
    } else {
      v = pair_phi<PMAX>(pr, n, s, sW1, sW2t, sb1, sc);
    }
  } else {
    v = pair_phi<PMAX>(pr, n, s, sW1, sW2t, sb1, sc);
    if (mode == kGenNegPhi) v = -v;
  }
  if (phi) phi[b * phi_stride + i] = v;
  if (keys) keys[b * key_stride + i] = make_key(v, static_cast<int32_t>(n));
}

// Per-component dot products as sort keys, rows r = b * P + p
// (TopKDotProduct for every component).  Grid: x over items, y over queries.
template <typename T, int PMAX>
__global__ __launch_bounds__(256) void k_dots_generic(DevProb pr, int n_begin, int n_count,
                                                      uint64_t* __restrict__ keys, long key_stride) {
  const int b = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_count) return;
  const long n = static_cast<long>(n_begin) + i;
  float s[PMAX];
  pair_dots<T, PMAX>(pr, b, n, s);
#pragma unroll
  for (int p = 0; p < PMAX; ++p)
    if (p < pr.P) keys[(static_cast<long>(b) * pr.P + p) * key_stride + i] = make_key(s[p], static_cast<int32_t>(n));
}

// ---------------------------------------------------------------------------
// Segmented top-k: block (seg, row) takes keys in[row][seg*S .. seg*S+S)
// into LDS (missing slots are empty keys) and writes the k largest, sorted
// descending, to out[row][seg*k ..].  With C the power of two >= k (at
// least 64): runs of C keys are bitonic-sorted in alternating directions,
// then rounds halve the keys, each keeping, of two adjacent runs (one
// descending, one ascending), the elementwise maximum (a bitonic sequence
// holding the C largest of the pair) and bitonic-merging it, until one
// descending run of C remains.  Where C >= S this is a full bitonic sort.
// Empty keys sort last and never reach the result, so the segment's
// nonzero keys are packed to the front first and the network runs over the
// smallest power of two (at least C) that holds them.
// ---------------------------------------------------------------------------
template <int S, int NT>
__global__ __launch_bounds__(NT) void k_segment_topk(const uint64_t* __restrict__ in, long in_stride,
                                                     int L, int k, uint64_t* __restrict__ out,
                                                     long out_stride, const uint32_t* __restrict__ gate) {
  static_assert(NT % 64 == 0, "whole waves");
  __shared__ uint64_t sk[S];
  __shared__ int s_nz;
  if (gate && *gate == 0u) return;             // whole workgroup: a path that is not taken
  const long row = blockIdx.y;
  const long base = static_cast<long>(blockIdx.x) * S;
  const uint64_t* src = in + row * in_stride + base;
  const int len = static_cast<int>(min(static_cast<long>(S), static_cast<long>(L) - base));
  const int lane = threadIdx.x & 63;
  if (threadIdx.x == 0) s_nz = 0;
  __syncthreads();
  // nonzero keys to the front (in any order: the network sorts them), one
  // LDS atomic per wave and pass
  for (int t0 = 0; t0 < S; t0 += NT) {
    const int t = t0 + static_cast<int>(threadIdx.x);
    const uint64_t key = t < len ? src[t] : 0ull;
    const uint64_t m = __ballot(key != 0ull);
    int at = 0;
    if (lane == 0 && m != 0ull) at = atomicAdd(&s_nz, __popcll(m));
    at = __shfl(at, 0);
    if (key != 0ull) sk[at + __popcll(m & ((1ull << lane) - 1ull))] = key;
  }
  __syncthreads();
  const int nz = s_nz;
  int C = 64;
  while (C < k && C < S) C <<= 1;
  int n0 = C;                                  // keys the network runs over: <= S
  while (n0 < nz) n0 <<= 1;
  for (int t = nz + static_cast<int>(threadIdx.x); t < n0; t += NT) sk[t] = 0ull;
  __syncthreads();
  // one compare-exchange stage over the first n keys: pairs at distance
  // stride, direction alternating every dirspan keys
  auto stage = [&](int n, int stride, int dirspan) {
    for (int i = threadIdx.x; i < n / 2; i += NT) {
      const int lo = 2 * i - (i & (stride - 1));
      const int hi = lo + stride;
      const bool desc = (lo & dirspan) == 0;
      const uint64_t a = sk[lo], c = sk[hi];
      if ((a < c) == desc) {
        sk[lo] = c;
        sk[hi] = a;
      }
    }
    __syncthreads();
  };
  // runs of C keys, sorted descending / ascending in turn
  for (int size = 2; size <= C; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) stage(n0, stride, size);
  for (int n = n0; n > C; n >>= 1) {
    // run pair (2m, 2m+1) -> run m: the elementwise maximum, kept in
    // registers until every thread has read its pair
    uint64_t keep[S / (2 * NT) > 0 ? S / (2 * NT) : 1];
    int cnt = 0;
    for (int t = threadIdx.x; t < n / 2; t += NT, ++cnt) {
      const int m = t / C, i = t - m * C;
      const uint64_t a = sk[2 * m * C + i], c = sk[(2 * m + 1) * C + i];
      keep[cnt] = a > c ? a : c;
    }
    __syncthreads();
    cnt = 0;
    for (int t = threadIdx.x; t < n / 2; t += NT, ++cnt) sk[t] = keep[cnt];
    __syncthreads();
    // merge each bitonic run; the last one (n / 2 == C) descending
    for (int stride = C >> 1; stride > 0; stride >>= 1) stage(n / 2, stride, C);
  }
  uint64_t* dst = out + row * out_stride + static_cast<long>(blockIdx.x) * k;
  for (int t = threadIdx.x; t < k; t += NT) dst[t] = sk[t];
}

__global__ void k_decode_keys(const uint64_t* __restrict__ keys, long key_stride, int rows, int k,
                              float* __restrict__ score, int32_t* __restrict__ idx,
                              const uint32_t* __restrict__ gate) {
  if (gate && *gate == 0u) return;
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(rows) * k) return;
  const long r = i / k, j = i - (i / k) * k;
  const uint64_t key = keys[r * key_stride + j];
  if (score) score[i] = key_score(key);
  if (idx) idx[i] = key_item(key);
}

__global__ void k_fill_u64(uint64_t* __restrict__ p, long n, uint64_t v) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Copy rows of k keys into a strided destination (the running top-k list is
// appended to the next tile's keys).
__global__ void k_copy_rows(const uint64_t* __restrict__ src, long src_stride, int rows, int k,
                            uint64_t* __restrict__ dst, long dst_stride) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<long>(rows) * k) return;
  const long r = i / k, j = i - (i / k) * k;
  dst[r * dst_stride + j] = src[r * src_stride + j];
}

// ---------------------------------------------------------------------------
// Candidate union + dedup (the deduplicated set G of Algorithm 2): one block
// per query inserts its C candidate ids into an LDS open-addressing hash set
// (linear probing, capacity a power of two >= 1.5 C) and counts each new id
// in one of kDedupBins bins of consecutive ids (id >> bin_shift); the ids are
// then written bin by bin (a counting sort: ascending bins, arbitrary order
// inside a bin), so that the rerank walks every query's candidates from the
// front of the corpus to its end and concurrent waves gather nearby items.
// Ids outside [0, N) are empty slots.
// ---------------------------------------------------------------------------
constexpr int kDedupBins = 1024;
__global__ __launch_bounds__(1024) void k_dedup(const int32_t* __restrict__ cand, int C,
                                                const int32_t* __restrict__ cand2, int C2, int N,
                                                int cap_log2, int bin_shift, int32_t* __restrict__ uniq,
                                                int32_t* __restrict__ n_unique) {
  extern __shared__ int32_t table[];     // cap slots, then kDedupBins bin counters
  __shared__ int count;
  __shared__ int wsum[1024 / 64];
  const int cap = 1 << cap_log2;
  int32_t* bins = table + cap;
  const long b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < cap; i += blockDim.x) table[i] = -1;
  for (int i = tid; i < kDedupBins; i += blockDim.x) bins[i] = 0;
  if (tid == 0) count = 0;
  __syncthreads();
  const int CT = C + C2;                 // both sets; uniq rows hold CT slots
  for (int i = tid; i < CT; i += blockDim.x) {
    const int32_t id = i < C ? cand[b * C + i] : cand2[b * C2 + (i - C)];
    if (id < 0 || id >= N) continue;
    uint32_t h = (static_cast<uint32_t>(id) * 0x9E3779B1u) >> (32 - cap_log2);
    for (int probe = 0; probe < cap; ++probe) {
      const int32_t prev = atomicCAS(&table[h], -1, id);
      if (prev == -1) {
        atomicAdd(&count, 1);
        atomicAdd(&bins[id >> bin_shift], 1);
        break;
      }
      if (prev == id) break;
      h = (h + 1) & (cap - 1);
    }
  }
  __syncthreads();
  // exclusive prefix sum of the bin counts (blockDim.x == kDedupBins)
  const int v = bins[tid];
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  bins[tid] = before + incl - v;
  __syncthreads();
  for (int s = tid; s < cap; s += blockDim.x) {
    const int32_t id = table[s];
    if (id >= 0) uniq[b * CT + atomicAdd(&bins[id >> bin_shift], 1)] = id;
  }
  if (tid == 0) n_unique[b] = count;
}

// ---------------------------------------------------------------------------
// Theorem 2 certificate: one thread per query, a max over P list entries.
// ---------------------------------------------------------------------------
__global__ void k_gap_bound(int B, int P, int m, const float* __restrict__ dots, int k,
                            const float* __restrict__ scores, float* out_S, float* out_SK,
                            float* out_bound, float* out_looser) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  float S = -__builtin_inff(), Sk = -__builtin_inff();
  for (int p = 0; p < P; ++p) {
    const float* row = dots + (static_cast<long>(b) * P + p) * m;
    S = fmaxf(S, row[m - 1]);
    Sk = fmaxf(Sk, row[m - 2]);
  }
  const float SK = scores[static_cast<long>(b) * k + (k - 1)];
  if (out_S) out_S[b] = S;
  if (out_SK) out_SK[b] = SK;
  if (out_bound) out_bound[b] = S - SK;
  if (out_looser) out_looser[b] = Sk - SK;
}

// ---------------------------------------------------------------------------
// Theorem 3 certificate of the combined candidates: one workgroup per query.
// The TopKAvg ids A_b go into an LDS hash set; for every component list
// (descending, m entries) the first entry at position >= kprime whose id is
// outside A_b is the largest s_p over items outside (X_{kprime,p} U A_b),
// since the list's first kprime entries are X_{kprime,p} itself.  S' is the
// maximum over p; -inf when some list runs out before finding one (cannot
// happen when m > kprime + k_avg).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gap_bound_combined(int P, int m, const float* __restrict__ dots,
                                                            const int32_t* __restrict__ ids, int kprime,
                                                            const int32_t* __restrict__ avg_ids, int k_avg,
                                                            int cap_log2, int k, const float* __restrict__ scores,
                                                            float* out_S, float* out_SK, float* out_bound) {
  extern __shared__ int32_t set[];
  __shared__ float s_best[4];
  const int cap = 1 << cap_log2;
  const long b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < cap; i += 256) set[i] = -1;
  __syncthreads();
  for (int i = tid; i < k_avg; i += 256) {
    const int32_t id = avg_ids[b * k_avg + i];
    if (id < 0) continue;
    uint32_t h = (static_cast<uint32_t>(id) * 0x9E3779B1u) >> (32 - cap_log2);
    for (int probe = 0; probe < cap; ++probe) {
      const int32_t prev = atomicCAS(&set[h], -1, id);
      if (prev == -1 || prev == id) break;
      h = (h + 1) & (cap - 1);
    }
  }
  __syncthreads();
  auto in_set = [&](int32_t id) {
    uint32_t h = (static_cast<uint32_t>(id) * 0x9E3779B1u) >> (32 - cap_log2);
    for (int probe = 0; probe < cap; ++probe) {
      const int32_t v = set[h];
      if (v == id) return true;
      if (v == -1) return false;
      h = (h + 1) & (cap - 1);
    }
    return false;
  };
  float best = -__builtin_inff();
  for (int p = wave; p < P; p += 4) {              // one wave per list
    const long row = (b * P + p) * static_cast<long>(m);
    for (int base = kprime; base < m; base += 64) {
      const int pos = base + lane;
      const bool outside = pos < m && !in_set(ids[row + pos]);
      const uint64_t hit = __ballot(outside);
      if (hit) {
        const int first = __ffsll(static_cast<long long>(hit)) - 1;
        best = fmaxf(best, dots[row + base + first]);
        break;
      }
    }
  }
  if (lane == 0) s_best[wave] = best;
  __syncthreads();
  if (tid == 0) {
    const float S = fmaxf(fmaxf(s_best[0], s_best[1]), fmaxf(s_best[2], s_best[3]));
    const float SK = scores[b * k + (k - 1)];
    if (out_S) out_S[b] = S;
    if (out_SK) out_SK[b] = SK;
    if (out_bound) out_bound[b] = S - SK;
  }
}

hipError_t launch_gap_bound_combined(int B, int P, int m, const float* dots, const int32_t* ids, int kprime,
                                     const int32_t* avg_ids, int k_avg, int k, const float* scores,
                                     float* out_S, float* out_SK, float* out_bound, hipStream_t st) {
  const int cap_log2 = dedup_cap_log2(k_avg);
  const size_t smem = sizeof(int32_t) << cap_log2;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gap_bound_combined),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_gap_bound_combined, dim3(B), dim3(256), smem, st, P, m, dots, ids, kprime, avg_ids,
                     k_avg, cap_log2, k, scores, out_S, out_SK, out_bound);
  return hipGetLastError();
}

// bound[b] = sign * scores[b][col] (Algorithm 1's threshold from the rerank
// output over G).
__global__ void k_pick_bound(const float* __restrict__ scores, int stride, int col, float sign, int B,
                             float* __restrict__ bound) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) bound[b] = sign * scores[static_cast<long>(b) * stride + col];
}

hipError_t launch_pick_bound(const float* scores, int stride, int col, float sign, int B, float* bound,
                             hipStream_t st) {
  hipLaunchKernelGGL(k_pick_bound, dim3((B + 255) / 256), dim3(256), 0, st, scores, stride, col, sign, B,
                     bound);
  return hipGetLastError();
}

hipError_t launch_gap_bound(int B, int P, int m, const float* dots, int k, const float* scores,
                            float* out_S, float* out_SK, float* out_bound, float* out_looser,
                            hipStream_t st) {
  hipLaunchKernelGGL(k_gap_bound, dim3((B + 255) / 256), dim3(256), 0, st, B, P, m, dots, k, scores,
                     out_S, out_SK, out_bound, out_looser);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// TopKAvg materialisation: out[m][t] = round(sum_c in[c*sc + m*sm + t]),
// summed in float64, rounded once (nearest-even).
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_avg_embed(const T* __restrict__ in, long sc, long sm, int ncomp, long M, int d,
                            T* __restrict__ out) {
  const long i = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= M * d) return;
  const long m = i / d, t = i - (i / d) * d;
  double acc = 0.0;
  for (int c = 0; c < ncomp; ++c) acc += static_cast<double>(to_f32(in[c * sc + m * sm + t]));
  if constexpr (sizeof(T) == 2)
    out[i] = f64_to_bf16_rne(acc);
  else
    out[i] = static_cast<float>(acc);
}

// ---------------------------------------------------------------------------
// Host-side launchers.
// ---------------------------------------------------------------------------
static size_t phi_smem_bytes(const DevProb& pr, int pmax) {
  return sizeof(float) * (2 * static_cast<size_t>(pr.H) * pmax + pr.H + pmax);
}

template <typename T, int PMAX>
static hipError_t launch_phi_t(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                               const int32_t* items, const int32_t* item_count, long item_stride,
                               const float* sbuf, long s_pstride, long s_bstride,
                               float* phi, long phi_stride, uint64_t* keys, long key_stride,
                               hipStream_t st) {
  const size_t smem = mode == kGenMaxDot ? 0 : phi_smem_bytes(pr, PMAX);
  if (smem > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_phi_generic<T, PMAX>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       static_cast<int>(smem));
    if (e != hipSuccess) return e;
  }
  dim3 grid((n_count + 255) / 256, pr.B);
  hipLaunchKernelGGL((k_phi_generic<T, PMAX>), grid, dim3(256), smem, st, pr, mode, bound, n_begin,
                     n_count, items, item_count, item_stride, sbuf, s_pstride, s_bstride, phi, phi_stride,
                     keys, key_stride);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_phi_p(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                               const int32_t* items, const int32_t* item_count, long item_stride,
                               const float* sbuf, long s_pstride, long s_bstride,
                               float* phi, long phi_stride, uint64_t* keys, long key_stride,
                               hipStream_t st) {
  if (pr.P <= 4)
    return launch_phi_t<T, 4>(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf,
                              s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
  if (pr.P <= 16)
    return launch_phi_t<T, 16>(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf,
                               s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
  return launch_phi_t<T, 64>(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf,
                             s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
}

hipError_t launch_phi_generic(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                              const int32_t* items, const int32_t* item_count, long item_stride,
                              const float* sbuf, long s_pstride, long s_bstride,
                              float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st) {
  if (n_count <= 0) return hipSuccess;
  if (pr.dtype == MOL_BF16)
    return launch_phi_p<bf16_t>(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf,
                                s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
  return launch_phi_p<float>(pr, mode, bound, n_begin, n_count, items, item_count, item_stride, sbuf,
                             s_pstride, s_bstride, phi, phi_stride, keys, key_stride, st);
}

template <typename T>
static hipError_t launch_dots_t(const DevProb& pr, int n_begin, int n_count, uint64_t* keys,
                                long key_stride, hipStream_t st) {
  dim3 grid((n_count + 255) / 256, pr.B);
  if (pr.P <= 4)
    hipLaunchKernelGGL((k_dots_generic<T, 4>), grid, dim3(256), 0, st, pr, n_begin, n_count, keys, key_stride);
  else if (pr.P <= 16)
    hipLaunchKernelGGL((k_dots_generic<T, 16>), grid, dim3(256), 0, st, pr, n_begin, n_count, keys, key_stride);
  else
    hipLaunchKernelGGL((k_dots_generic<T, 64>), grid, dim3(256), 0, st, pr, n_begin, n_count, keys, key_stride);
  return hipGetLastError();
}

hipError_t launch_dots_generic(const DevProb& pr, int n_begin, int n_count, uint64_t* keys,
                               long key_stride, hipStream_t st) {
  if (n_count <= 0) return hipSuccess;
  if (pr.dtype == MOL_BF16) return launch_dots_t<bf16_t>(pr, n_begin, n_count, keys, key_stride, st);
  return launch_dots_t<float>(pr, n_begin, n_count, keys, key_stride, st);
}

int segment_size_for(int L, int k) {
  // One segment when it fits, else the largest segment (always >= 4k so
  // every pass shrinks the rows).
  if (L <= 256 && k <= 256) return 256;
  if (L <= 512 && k <= 512) return 512;
  if (L <= 1024 && k <= 1024) return 1024;
  return 4096;
}

hipError_t launch_segment_topk(const uint64_t* in, long in_stride, int rows, int L, int k,
                               uint64_t* out, long out_stride, hipStream_t st, const uint32_t* gate) {
  const int S = segment_size_for(L, k);
  dim3 grid((L + S - 1) / S, rows);
  if (S == 256)
    hipLaunchKernelGGL((k_segment_topk<256, 128>), grid, dim3(128), 0, st, in, in_stride, L, k, out, out_stride,
                       gate);
  else if (S == 512)
    hipLaunchKernelGGL((k_segment_topk<512, 256>), grid, dim3(256), 0, st, in, in_stride, L, k, out, out_stride,
                       gate);
  else if (S == 1024)
    hipLaunchKernelGGL((k_segment_topk<1024, 512>), grid, dim3(512), 0, st, in, in_stride, L, k, out, out_stride,
                       gate);
  else
    hipLaunchKernelGGL((k_segment_topk<4096, 1024>), grid, dim3(1024), 0, st, in, in_stride, L, k, out,
                       out_stride, gate);
  return hipGetLastError();
}

hipError_t launch_decode(const uint64_t* keys, long key_stride, int rows, int k, float* score,
                         int32_t* idx, hipStream_t st, const uint32_t* gate) {
  const long n = static_cast<long>(rows) * k;
  hipLaunchKernelGGL(k_decode_keys, dim3((n + 255) / 256), dim3(256), 0, st, keys, key_stride, rows, k, score, idx,
                     gate);
  return hipGetLastError();
}

hipError_t launch_fill(uint64_t* p, long n, uint64_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_u64, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const uint64_t* src, long src_stride, int rows, int k, uint64_t* dst,
                            long dst_stride, hipStream_t st) {
  const long n = static_cast<long>(rows) * k;
  hipLaunchKernelGGL(k_copy_rows, dim3((n + 255) / 256), dim3(256), 0, st, src, src_stride, rows, k, dst, dst_stride);
  return hipGetLastError();
}

int dedup_cap_log2(int C) {
  int lg = 1;
  while ((1 << lg) < C + C / 2) ++lg;
  return lg;
}

hipError_t launch_dedup(const int32_t* cand, int C, const int32_t* cand2, int C2, int B, int N,
                        int32_t* uniq, int32_t* n_unique, hipStream_t st) {
  const int lg = dedup_cap_log2(C + C2);
  const size_t smem = (sizeof(int32_t) << lg) + sizeof(int32_t) * kDedupBins;
  int bin_shift = 0;                     // (N - 1) >> bin_shift < kDedupBins
  while (((static_cast<long>(N) - 1) >> bin_shift) >= kDedupBins) ++bin_shift;
  if (smem > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_dedup),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       static_cast<int>(smem));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_dedup, dim3(B), dim3(kDedupBins), smem, st, cand, C, cand2, C2, N, lg, bin_shift, uniq,
                     n_unique);
  return hipGetLastError();
}

hipError_t launch_avg_embed(const DevProb& pr, void* q_avg, void* x_avg, hipStream_t st) {
  const long nq = static_cast<long>(pr.B) * pr.d, nx = static_cast<long>(pr.N) * pr.d;
  if (pr.dtype == MOL_BF16) {
    if (q_avg)
      hipLaunchKernelGGL((k_avg_embed<bf16_t>), dim3((nq + 255) / 256), dim3(256), 0, st,
                         static_cast<const bf16_t*>(pr.Q), static_cast<long>(pr.d),
                         static_cast<long>(pr.Pq) * pr.d, pr.Pq, static_cast<long>(pr.B), pr.d,
                         static_cast<bf16_t*>(q_avg));
    if (x_avg)
      hipLaunchKernelGGL((k_avg_embed<bf16_t>), dim3((nx + 255) / 256), dim3(256), 0, st,
                         static_cast<const bf16_t*>(pr.X), static_cast<long>(pr.N) * pr.d,
                         static_cast<long>(pr.d), pr.Px, static_cast<long>(pr.N), pr.d,
                         static_cast<bf16_t*>(x_avg));
  } else {
    if (q_avg)
      hipLaunchKernelGGL((k_avg_embed<float>), dim3((nq + 255) / 256), dim3(256), 0, st,
                         static_cast<const float*>(pr.Q), static_cast<long>(pr.d),
                         static_cast<long>(pr.Pq) * pr.d, pr.Pq, static_cast<long>(pr.B), pr.d,
                         static_cast<float*>(q_avg));
    if (x_avg)
      hipLaunchKernelGGL((k_avg_embed<float>), dim3((nx + 255) / 256), dim3(256), 0, st,
                         static_cast<const float*>(pr.X), static_cast<long>(pr.N) * pr.d,
                         static_cast<long>(pr.d), pr.Px, static_cast<long>(pr.N), pr.d,
                         static_cast<float*>(x_avg));
  }
  return hipGetLastError();
}

}  // namespace mol
