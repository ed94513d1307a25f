// Issue-rate probe of the fused scan's per-step instruction mix (see
// include/mol_probe.h).  Every instruction is written as inline asm on
// registers the probe owns: four independent MFMA accumulator chains (each
// chain's next MFMA is four MFMAs later) and eight independent vector
// registers, so nothing waits on a result inside the loop.  Results are only
// summed into `sink` after the loop (their values are meaningless).
#include <hip/hip_runtime.h>

#include "mol_probe.h"

namespace {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kGroups = 48;        // MFMAs per wave-step

struct Regs {
  uint4 ld[2];     // LDS read results (never read in the loop)
  uint32_t sc;     // scalar counter
  f32x4_t acc[4];
  float x[8];      // transcendental inputs (never written in the loop)
  float t[8];      // transcendental results (never read in the loop)
  float a[8];      // plain ALU chains, read by the conversions
  unsigned pk;
  f16x8_t A, Bm;
};

template <int I>
__device__ __forceinline__ void mfma(Regs& r) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(r.acc[I & 3]) : "v"(r.A), "v"(r.Bm));
}
template <int I>
__device__ __forceinline__ void trans(Regs& r) {
  asm volatile("v_exp_f32 %0, %1" : "+v"(r.t[I & 7]) : "v"(r.x[I & 7]));
}
template <int I>
__device__ __forceinline__ void plain(Regs& r) {
  asm volatile("v_add_f32 %0, 1.0, %0" : "+v"(r.a[I & 7]));
}
template <int I>
__device__ __forceinline__ void cvt(Regs& r) {
  asm volatile("v_cvt_pk_f16_f32 %0, %1, %2" : "+v"(r.pk) : "v"(r.a[(I + 4) & 7]), "v"(r.a[(I + 5) & 7]));
}

// the vector share of group G: 2 transcendental (3 in group 0), 4 plain
// (5 in 14 of the 48 groups) and a conversion in two groups of three:
// 97 / 206 / 32 per step, the fused scan's counts (SQ_INSTS_VALU_TRANS_F32
// and SQ_INSTS_VALU less the MFMAs, per wave-step of k_mol_fused)
template <int G>
__device__ __forceinline__ void vector_share(Regs& r) {
  trans<2 * G>(r);
  plain<5 * G>(r);
  plain<5 * G + 1>(r);
  trans<2 * G + 1>(r);
  plain<5 * G + 2>(r);
  plain<5 * G + 3>(r);
  if ((G * 14) % 48 < 14) plain<5 * G + 4>(r);
  if (G == 0) trans<101>(r);
  if (G % 3 != 2) cvt<G>(r);
}

// the rest of the fused scan's per-step stream (counters: 28.5 LDS and 39
// scalar instructions per wave-step; its listing's nops: two 11-slot MFMA
// drains and about 25 more nops of 2.8 slots on average per step): in group
// G, an LDS read of 16 bytes per lane in 28 of the 48 groups, a scalar
// multiply in 39, a three-slot s_nop in 25 and an 11-slot drain in two
template <int G>
__device__ __forceinline__ void rest_share(Regs& r, uint32_t lds_off) {
  if constexpr ((G * 28) % 48 < 28) {
    asm volatile("ds_read_b128 %0, %1" : "=v"(r.ld[G & 1]) : "v"(lds_off));
  }
  // s_mul_i32 leaves SCC alone; the clobber keeps the compiler from relying
  // on it across the statement regardless
  if constexpr ((G * 39) % 48 < 39) asm volatile("s_mul_i32 %0, %0, 3" : "+s"(r.sc) : : "scc");
  if constexpr ((G * 25) % 48 < 25) asm volatile("s_nop 2");
  if constexpr (G == 0 || G == 24) asm volatile("s_nop 7\n\ts_nop 2");
}

template <int PATTERN, int G>
__device__ __forceinline__ void groups(Regs& r, uint32_t lds_off = 0) {
  if constexpr (G < kGroups) {
    if constexpr (PATTERN == 4) {
      mfma<G>(r);
      vector_share<G>(r);
      rest_share<G>(r, lds_off);
    } else if constexpr (PATTERN == 0) {
      mfma<G>(r);
      vector_share<G>(r);
    } else if constexpr (PATTERN == 1) {
      vector_share<G>(r);
    } else if constexpr (PATTERN == 2) {
      mfma<G>(r);
    }
    groups<PATTERN, G + 1>(r, lds_off);
  }
}
template <int G>
__device__ __forceinline__ void mfmas_only(Regs& r) {
  if constexpr (G < kGroups) {
    mfma<G>(r);
    mfmas_only<G + 1>(r);
  }
}

template <int PATTERN>
__global__ __launch_bounds__(256) void k_issue_probe(float* __restrict__ sink, int iters) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[256 * 16];
  for (int i = threadIdx.x; i < 256 * 16; i += blockDim.x) lds[i] = static_cast<unsigned char>(i);
  __syncthreads();
  // each lane reads its own 16 bytes of its wave's 1 KB (in bounds: 4 waves x 1 KB)
  const uint32_t lds_off =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) void*)(lds))) +
      16u * threadIdx.x;
  Regs r;
  r.ld[0] = r.ld[1] = make_uint4(0, 0, 0, 0);
  r.sc = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) r.acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    r.a[i] = 1e-3f * static_cast<float>(threadIdx.x + i);
    r.x[i] = r.a[i] - 0.5f;
    r.t[i] = 0.f;
    r.A[i] = static_cast<_Float16>(1e-3f * i);
    r.Bm[i] = static_cast<_Float16>(1.f - 1e-3f * i);
  }
  r.pk = 0u;
  for (int it = 0; it < iters; ++it) {
    if constexpr (PATTERN == 3) {
      mfmas_only<0>(r);
      groups<1, 0>(r);
    } else {
      groups<PATTERN, 0>(r, lds_off);
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // drain the matrix pipe before reading its registers (the asm above is
  // opaque to the compiler's hazard padding)
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7");
  float s = static_cast<float>((r.pk ^ r.ld[0].x ^ r.ld[1].y ^ r.sc) & 0xffu);
#pragma unroll
  for (int i = 0; i < 8; ++i) s += r.a[i] + r.t[i];
#pragma unroll
  for (int i = 0; i < 4; ++i) s += r.acc[i][0];
  sink[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

extern "C" int mol_probe_issue_mix(int pattern, int waves_per_simd, int iters, float* sink, void* stream) {
  if (waves_per_simd < 1 || waves_per_simd > 8 || iters < 1 || pattern < 0 || pattern > 4 || !sink) return -1;
  const dim3 grid(256 * waves_per_simd), block(256);
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (pattern) {
    case 0: hipLaunchKernelGGL(k_issue_probe<0>, grid, block, 0, st, sink, iters); break;
    case 1: hipLaunchKernelGGL(k_issue_probe<1>, grid, block, 0, st, sink, iters); break;
    case 2: hipLaunchKernelGGL(k_issue_probe<2>, grid, block, 0, st, sink, iters); break;
    case 4: hipLaunchKernelGGL(k_issue_probe<4>, grid, block, 0, st, sink, iters); break;
    case 3: hipLaunchKernelGGL(k_issue_probe<3>, grid, block, 0, st, sink, iters); break;
    default: return -1;
  }
  return static_cast<int>(hipGetLastError());
}
