// Host-side launchers of the gfx950 kernels (all asynchronous on `st`).
#pragma once

#include "mol_device.h"

namespace mol {

// Generic (one thread per pair, float32 arithmetic) kernels.
// Score of the pair-wise kernel: phi; phi restricted to items whose
// max_p s_p can reach bound[b]; max_p s_p; -phi.
enum GenMode { kGenPhi = 0, kGenBounded = 1, kGenMaxDot = 2, kGenNegPhi = 3 };
// sbuf: NULL, or the component dot products of items n_begin + i laid out
// as sbuf[p * s_pstride + b * s_bstride + i] (contiguous ranges only).
hipError_t launch_phi_generic(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                              const int32_t* items, const int32_t* item_count, long item_stride,
                              const float* sbuf, long s_pstride, long s_bstride,
                              float* phi, long phi_stride, uint64_t* keys, long key_stride,
                              hipStream_t st);
hipError_t launch_dots_generic(const DevProb& pr, int n_begin, int n_count, uint64_t* keys,
                               long key_stride, hipStream_t st);

// Component dot products on MFMA for the generic shapes (bf16, d % 32 == 0):
// into a buffer s[p][b][i] (row stride dots_buffer_row(nt) floats, p stride
// B * that) for the pair-wise gating kernel, or into per-component sort keys.
// tile_stride > 1 (keys only): every tile_stride-th 128-item tile, keys
// stored compactly, dots_sample_len(nt, tile_stride) slots per row (the
// slots past the range cleared to 0); tile_stride 1 writes nt keys.
// Candidates: the keys of list (b, p) at or above thr[(b * P + p) *
// thr_stride] appended to its row of `cand` (which must hold nt keys),
// counts[b * P + p] advanced (the counts start at zero).
enum DotsMode { kDotsToBuffer = 0, kDotsToKeys = 1, kDotsToCandidates = 2, kDotsToMaxKeys = 3 };
// max_p s_p of every (query, item) as sort keys [B][key_stride] (P_q divides 64)
bool dots_maxkeys_supported(const DevProb& pr);
hipError_t launch_dots_mfma_maxkeys(const DevProb& pr, int n0, int nt, uint64_t* keys, long key_stride,
                                    hipStream_t st);
bool dots_mfma_supported(const DevProb& pr);
long dots_buffer_row(int nt);
long dots_sample_len(int nt, int tile_stride);
hipError_t launch_dots_mfma(const DevProb& pr, int n0, int nt, int mode, float* sbuf, long s_pstride,
                            long s_bstride, uint64_t* keys, long key_stride, hipStream_t st,
                            int tile_stride = 1);
hipError_t launch_dots_mfma_candidates(const DevProb& pr, int n0, int nt, const uint64_t* thr, long thr_stride,
                                       uint64_t* cand, long cand_stride, uint32_t* counts, hipStream_t st);
// the same into the buffer for per-query candidate lists (items [B][item_stride],
// item_count [B], at most C per query): s[p][b][i] of candidate i
hipError_t launch_dots_mfma_gather(const DevProb& pr, const int32_t* items, const int32_t* item_count,
                                   long item_stride, int C, float* sbuf, long s_pstride, long s_bstride,
                                   hipStream_t st);

// Pair-wise gating on MFMA over the dots buffer (bf16, P <= 64, H <= 128):
// the same modes, arguments and outputs as launch_phi_generic with sbuf set.
bool phi_mfma_supported(const DevProb& pr);
hipError_t launch_phi_mfma(const DevProb& pr, int mode, const float* bound, int n_begin, int n_count,
                           const int32_t* items, const int32_t* item_count, long item_stride,
                           const float* sbuf, long s_pstride, long s_bstride, float* phi, long phi_stride,
                           uint64_t* keys, long key_stride, hipStream_t st);

// Selection machinery over 64-bit sort keys.  gate: NULL, or a device flag
// read at the start of every workgroup; the launch does nothing while it is
// zero (the second of two alternative paths, chosen on the device).
int segment_size_for(int L, int k);
// Rows of L keys -> their top k (k <= 8192) by radix selection, one
// workgroup per row (keys of a row distinct apart from empty ones).
// row_len: NULL, or per-row key counts (row r reads min(row_len[r], L) keys).
hipError_t launch_radix_topk(const uint64_t* in, long in_stride, int rows, long L, int k, uint64_t* out,
                             long out_stride, hipStream_t st, const uint32_t* row_len = nullptr,
                             const uint32_t* gate = nullptr);
// The same per chunk of chunk_len keys (chunks * chunk_len >= L): row r's
// chunk j's top k at out[(r * chunks + j) * k], so a row's chunk lists are
// one contiguous run of chunks * k keys.
hipError_t launch_radix_topk_chunks(const uint64_t* in, long in_stride, int rows, long L, int k, int chunks,
                                    long chunk_len, uint64_t* out, hipStream_t st, const uint32_t* gate = nullptr);
hipError_t launch_segment_topk(const uint64_t* in, long in_stride, int rows, int L, int k,
                               uint64_t* out, long out_stride, hipStream_t st, const uint32_t* gate = nullptr);
hipError_t launch_decode(const uint64_t* keys, long key_stride, int rows, int k, float* score,
                         int32_t* idx, hipStream_t st, const uint32_t* gate = nullptr);
hipError_t launch_fill(uint64_t* p, long n, uint64_t v, hipStream_t st);
hipError_t launch_copy_rows(const uint64_t* src, long src_stride, int rows, int k, uint64_t* dst,
                            long dst_stride, hipStream_t st);

// Approximate path helpers.
int dedup_cap_log2(int C);
hipError_t launch_dedup(const int32_t* cand, int C, const int32_t* cand2, int C2, int B, int N,
                        int32_t* uniq, int32_t* n_unique, hipStream_t st);
hipError_t launch_gap_bound(int B, int P, int m, const float* dots, int k, const float* scores,
                            float* out_S, float* out_SK, float* out_bound, float* out_looser,
                            hipStream_t st);
hipError_t launch_gap_bound_combined(int B, int P, int m, const float* dots, const int32_t* ids, int kprime,
                                     const int32_t* avg_ids, int k_avg, int k, const float* scores,
                                     float* out_S, float* out_SK, float* out_bound, hipStream_t st);
hipError_t launch_avg_embed(const DevProb& pr, void* q_avg, void* x_avg, hipStream_t st);
hipError_t launch_pick_bound(const float* scores, int stride, int col, float sign, int B, float* bound,
                             hipStream_t st);

}  // namespace mol

namespace mol {

// Fused MFMA scoring (bf16, Pq = 8; (Px, d, H) in {(8,32,64), (8,64,64), (4,64,64),
// (4,128,128)}).
bool fused_supported(const DevProb& pr, int k);
// max-component-dot epilogue: the same shapes with H ignored
bool fused_maxdot_supported(const DevProb& pr, int k);
void fused_grid(const DevProb& pr, int n_count, int& R, int& range_len, int& G, bool maxdot);
// bound: NULL, or [B] floats: only items with max_p s_p (plus the rounding
// margin) at or above bound[b] are ranked for query b.  redo: NULL, or
// fused_redo_flags(R, G) ints of workspace; with it (and no bound) the
// software-pipelined scan runs, whose workgroups flag a
// range where a softmax sum left its safe range, and a second launch
// rescores only the flagged ranges.
long fused_redo_flags(int R, int G);
hipError_t launch_fused_topk(const DevProb& pr, int k, int R, int range_len, int G,
                             const float* bound, uint64_t* partial, int* redo, hipStream_t st);
hipError_t launch_fused_maxdot(const DevProb& pr, int k, int R, int range_len, int G,
                               uint64_t* partial, hipStream_t st);
hipError_t launch_fused_dense(const DevProb& pr, int n_begin, int n_count, float* phi,
                              hipStream_t st);

}  // namespace mol

namespace mol {

// Per-component top-k' with MFMA dots: a bucket-maximum scan, a per-list
// starting threshold, and a threshold scan with staged merges
// (bf16, d in {32, 64, 128}, k' <= 1024).
struct PerEmbdGrid {
  struct Scan {
    int R = 0, range_len = 0, G = 0;   // item ranges, items per range, vector groups
  };
  Scan s1, s2;                         // bucket scan, threshold scan
  int bucket_tiles = 0, nbk = 0;       // 32-item tiles per bucket, buckets per range
  bool pruned = false;                 // the pruned second pass (else the threshold scan)
  int key_cap = 0;                     // pruned pass: keys per list buffer
  int vec_wg_pruned = 0, CH = 0;       // pruned pass: vectors per workgroup, chunks per bucket group
  int groups = 0;                      // bucket groups Px * s1.R * nbk
};
// Device buffers of the per-component path (rows = B * Pq * Px lists).
struct PerEmbdBufs {
  float* bmax = nullptr;      // [Px][s1.R][nbk][B*Pq] bucket maxima
  float* thr = nullptr;       // [rows] starting thresholds
  float* thr_t = nullptr;     // [Px][B*Pq]: the same, component-major
  uint64_t* lists = nullptr;  // [rows][s2.R][KL] keys (threshold scan)
  uint64_t* stg = nullptr;    // [rows][s2.R][stage_cap] keys (threshold scan)
  int* hot_v = nullptr;       // [groups][B*Pq] (pruned pass)
  int* hot_n = nullptr;       // [groups]
  int* work = nullptr;        // [groups * CH]
  uint32_t* ctl = nullptr;    // [rows] key counts, then the overflow flag, then the work-list length
  uint64_t* keys = nullptr;   // [rows][key_cap]
};
bool per_embd_supported(const DevProb& pr, int kp);
int per_embd_list_cap(int kp);
int per_embd_stage_cap(int kp);
void per_embd_grid(const DevProb& pr, int kp, PerEmbdGrid& g);
// the scans (and, for the pruned form, its work list and pass); the lists
// are then finished by launch_per_embd_select (pruned form) and, gated on
// ctl[rows] (every list when it is set; always without the pruned form),
// by the segmented reduction of `lists`
hipError_t launch_per_embd(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b, hipStream_t st);
hipError_t launch_per_embd_select(const DevProb& pr, int kp, const PerEmbdGrid& g, const PerEmbdBufs& b,
                                  float* out_dot, int32_t* out_idx, hipStream_t st);

}  // namespace mol

namespace mol {

// Fused MFMA rerank of deduplicated candidates (same shapes as the fused scorer).
bool rerank_supported(const DevProb& pr, int k);
int rerank_chunk(int B, int C);
// negate: rank by -phi (the smallest scores first)
hipError_t launch_rerank(const DevProb& pr, const int32_t* uniq, const int32_t* n_unique, int C, int k,
                         bool negate, uint64_t* partial, hipStream_t st);

}  // namespace mol
