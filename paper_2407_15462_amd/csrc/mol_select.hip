// Exact top-k of long rows of 64-bit sort keys by radix selection
// (Definition 1's selection step for rows too long, or k too large, for the
// segmented sorts): one workgroup per row, or per chunk of a row when the
// rows are few (the chunks' top-k lists are then selected again).
//
// Keys of a row are distinct (the low word carries the item index) except
// empty slots (key 0), which never count.  The k-th largest key T is found
// digit by digit, 8 bits at a time from the top: a 256-bin histogram of the
// keys that share the digits found so far locates the bin holding the k-th
// key.  Once the keys sharing the prefix fit in LDS they are gathered there
// and the remaining digits read LDS only.  Every key >= T (exactly k of
// them, or all nonzero keys when the row has fewer) is then gathered,
// bitonic-sorted in LDS and written out, padded with empty keys.
#include "mol_kernels.h"

namespace mol {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelCap = 8192;     // keys held in LDS: candidates, then the sorted output

__device__ __forceinline__ uint32_t digit_of(uint64_t key, int shift) {
  return static_cast<uint32_t>(key >> shift) & 255u;
}
// key agrees with prefix on every digit above `shift`
__device__ __forceinline__ bool has_prefix(uint64_t key, uint64_t prefix, int shift) {
  return shift >= 56 || (key >> (shift + 8)) == (prefix >> (shift + 8));
}

}  // namespace

__global__ __launch_bounds__(kSelThreads) void k_radix_topk(const uint64_t* __restrict__ in, long in_stride,
                                                            long L_all, int k, uint64_t* __restrict__ out,
                                                            long out_stride, const uint32_t* __restrict__ row_len,
                                                            int chunks, long chunk_len,
                                                            const uint32_t* __restrict__ gate) {
  __shared__ uint64_t buf[kSelCap];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_bin, s_above, s_nz, s_count;
  if (gate && *gate == 0u) return;             // whole workgroup: a path that is not taken
  const int tid = threadIdx.x, lane = tid & 63;
  // workgroup = (row, chunk j): keys [j chunk_len, (j + 1) chunk_len) of the row
  const long row = blockIdx.x / chunks, j = blockIdx.x - (blockIdx.x / chunks) * chunks;
  const long Lrow = row_len ? min(L_all, static_cast<long>(row_len[row])) : L_all;
  const uint64_t* src = in + row * in_stride + j * chunk_len;
  const long L = max(0l, min(chunk_len, Lrow - j * chunk_len));

  // f(key) for every key of the range (keys past its end read as empty):
  // eight loads per thread are issued before any is used, so a pass over
  // global memory keeps that many in flight instead of one
  auto for_keys = [&](auto&& f) {
    constexpr int U = 8;
    for (long i0 = tid; i0 < L; i0 += static_cast<long>(U) * kSelThreads) {
      uint64_t kv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const long i = i0 + static_cast<long>(u) * kSelThreads;
        kv[u] = i < L ? src[i] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) f(kv[u]);
    }
  };

  uint64_t prefix = 0;
  uint32_t kk = static_cast<uint32_t>(k);   // rank of T among the keys sharing the prefix
  bool in_lds = false;
  uint32_t n_lds = 0;
  bool all_nonzero = false;                  // fewer than k keys: take every nonzero key
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0u;
    __syncthreads();
    if (in_lds) {
      for (uint32_t i = tid; i < n_lds; i += kSelThreads) {
        const uint64_t key = buf[i];
        if (has_prefix(key, prefix, shift)) atomicAdd(&hist[digit_of(key, shift)], 1u);
      }
    } else {
      for_keys([&](uint64_t key) {
        if (key != 0 && has_prefix(key, prefix, shift)) atomicAdd(&hist[digit_of(key, shift)], 1u);
      });
    }
    __syncthreads();
    // wave 0: bins in descending order, 4 per lane (lane 0 holds 255..252);
    // an inclusive scan of the lane sums finds the bin holding rank kk
    if (tid < 64) {
      uint32_t h[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        h[j] = hist[255 - 4 * lane - j];
        sum += h[j];
      }
      uint32_t incl = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      const uint32_t total = __shfl(incl, 63, 64);
      const uint64_t hit = __ballot(incl >= kk);
      if (lane == 0) s_nz = total;
      if (hit) {
        const int first = __ffsll(static_cast<long long>(hit)) - 1;
        if (lane == first) {
          uint32_t above = incl - sum;
          int bin = 255 - 4 * lane;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (above + h[j] >= kk) {
              bin = 255 - 4 * lane - j;
              break;
            }
            above += h[j];
          }
          s_bin = static_cast<uint32_t>(bin);
          s_above = above;
        }
      }
    }
    __syncthreads();
    if (shift == 56 && s_nz <= static_cast<uint32_t>(k)) {   // at most k nonzero keys in the row
      all_nonzero = true;
      break;
    }
    const uint32_t bin = s_bin, above = s_above;
    const uint32_t inbin = hist[bin];
    kk -= above;
    prefix |= static_cast<uint64_t>(bin) << shift;
    __syncthreads();
    // gather the keys sharing the new prefix into LDS once they fit
    if (!in_lds && shift > 0 && inbin <= static_cast<uint32_t>(kSelCap)) {
      if (tid == 0) s_count = 0u;
      __syncthreads();
      for_keys([&](uint64_t key) {
        if (key != 0 && has_prefix(key, prefix, shift - 8)) {
          const uint32_t pos = atomicAdd(&s_count, 1u);
          if (pos < static_cast<uint32_t>(kSelCap)) buf[pos] = key;   // (inbin of them: always)
        }
      });
      __syncthreads();
      n_lds = min(s_count, static_cast<uint32_t>(kSelCap));
      in_lds = true;
    }
  }
  // T = prefix: the k-th largest key.  Gather every key >= T.
  const uint64_t T = all_nonzero ? 1ull : prefix;
  __syncthreads();
  if (tid == 0) s_count = 0u;
  __syncthreads();
  for_keys([&](uint64_t key) {
    if (key >= T && key != 0) {
      const uint32_t pos = atomicAdd(&s_count, 1u);
      if (pos < static_cast<uint32_t>(kSelCap)) buf[pos] = key;   // (at most k of them: always)
    }
  });
  __syncthreads();
  const uint32_t n = min(s_count, static_cast<uint32_t>(kSelCap));   // == min(k, nonzero keys)
  int S = 64;
  while (S < static_cast<int>(n)) S <<= 1;
  for (int i = static_cast<int>(n) + tid; i < S; i += kSelThreads) buf[i] = 0ull;
  __syncthreads();
  for (int size = 2; size <= S; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < S / 2; i += kSelThreads) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const uint64_t a = buf[lo], c = buf[hi];
        if ((a < c) == desc) {
          buf[lo] = c;
          buf[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  uint64_t* dst = out + static_cast<long>(blockIdx.x) * out_stride;
  for (int i = tid; i < k; i += kSelThreads) dst[i] = i < static_cast<int>(n) ? buf[i] : 0ull;
}

hipError_t launch_radix_topk(const uint64_t* in, long in_stride, int rows, long L, int k, uint64_t* out,
                             long out_stride, hipStream_t st, const uint32_t* row_len, const uint32_t* gate) {
  if (k > kSelCap) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_radix_topk, dim3(rows), dim3(kSelThreads), 0, st, in, in_stride, L, k, out, out_stride,
                     row_len, 1, L, gate);
  return hipGetLastError();
}

hipError_t launch_radix_topk_chunks(const uint64_t* in, long in_stride, int rows, long L, int k, int chunks,
                                    long chunk_len, uint64_t* out, hipStream_t st, const uint32_t* gate) {
  if (k > kSelCap || chunks < 1 || static_cast<long>(chunks) * chunk_len < L) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_radix_topk, dim3(rows * chunks), dim3(kSelThreads), 0, st, in, in_stride, L, k, out,
                     static_cast<long>(k), nullptr, chunks, chunk_len, gate);
  return hipGetLastError();
}

}  // namespace mol
