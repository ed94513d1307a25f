// Host side of the C ABI declared in include/mol.h: argument validation,
// workspace planning and kernel sequencing on the caller's stream.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "mol_kernels.h"

using namespace mol;

namespace {

thread_local std::string g_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(MOL_EHIP, "%s: %s", where, hipGetErrorString(e));
}

#define MOL_TRY_HIP(expr, where)               \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

// ---------------------------------------------------------------------------
// Kernel timing: while enabled, event pairs recorded on the caller's stream
// around each entry point's main kernel; read (and recycled) by
// mol_timing_read.
constexpr int kTimedOps = 7;                  // mol_op codes 0..6

struct EvPair {
  hipEvent_t a = nullptr, b = nullptr;
};

struct TimingLog {
  std::mutex mu;
  bool on = false;
  std::vector<EvPair> rec[kTimedOps];
  std::vector<EvPair> spare;
};

TimingLog& timing_log() {
  static TimingLog t;
  return t;
}

EvPair timing_start(hipStream_t st) {
  TimingLog& t = timing_log();
  std::lock_guard<std::mutex> g(t.mu);
  EvPair p;
  if (!t.on) return p;
  if (!t.spare.empty()) {
    p = t.spare.back();
    t.spare.pop_back();
  } else {
    if (hipEventCreate(&p.a) != hipSuccess) return EvPair{};
    if (hipEventCreate(&p.b) != hipSuccess) {
      (void)hipEventDestroy(p.a);
      return EvPair{};
    }
  }
  if (hipEventRecord(p.a, st) != hipSuccess) {
    t.spare.push_back(p);
    return EvPair{};
  }
  return p;
}

void timing_stop(int op, const EvPair& p, hipStream_t st, bool launched) {
  if (!p.a) return;
  TimingLog& t = timing_log();
  const bool ok = launched && hipEventRecord(p.b, st) == hipSuccess;
  std::lock_guard<std::mutex> g(t.mu);
  (ok ? t.rec[op] : t.spare).push_back(p);
}

// Launch `expr` (a hipError_t expression) between the events of `op`
// (op < 0: not recorded).
#define MOL_TIMED_LAUNCH(op, st, expr, where)              \
  do {                                                     \
    const EvPair tp_ = (op) >= 0 ? timing_start(st) : EvPair{}; \
    const hipError_t te_ = (expr);                         \
    timing_stop((op), tp_, (st), te_ == hipSuccess);       \
    MOL_TRY_HIP(te_, where);                               \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Shape / pointer validation shared by every entry point.
int check_problem(const mol_problem* p, bool gating) {
  if (!p) return fail(MOL_EINVAL, "prob is NULL");
  if (p->B < 1 || p->N < 1 || p->Pq < 1 || p->Px < 1 || p->d < 1)
    return fail(MOL_EINVAL, "sizes must be positive (B=%d N=%d Pq=%d Px=%d d=%d)", p->B, p->N,
                p->Pq, p->Px, p->d);
  if (gating && p->H < 1) return fail(MOL_EINVAL, "H must be positive (H=%d)", p->H);
  if (p->B > MOL_MAX_B) return fail(MOL_EUNSUPPORTED, "B = %d exceeds %d", p->B, MOL_MAX_B);
  if (p->dtype != MOL_F32 && p->dtype != MOL_BF16)
    return fail(MOL_EUNSUPPORTED, "dtype %d is not MOL_F32 or MOL_BF16", p->dtype);
  if (p->flags & ~(MOL_FLAG_F32_GATING | MOL_FLAG_BF16X2_GATING))
    return fail(MOL_EINVAL, "unknown flag bits 0x%x", p->flags);
  if (p->Pq > MOL_MAX_P || p->Px > MOL_MAX_P || p->Pq * p->Px > MOL_MAX_P)
    return fail(MOL_EUNSUPPORTED, "P = Pq*Px = %d*%d exceeds %d", p->Pq, p->Px, MOL_MAX_P);
  if (p->d > MOL_MAX_D) return fail(MOL_EUNSUPPORTED, "d = %d exceeds %d", p->d, MOL_MAX_D);
  if (gating && p->H > MOL_MAX_H) return fail(MOL_EUNSUPPORTED, "H = %d exceeds %d", p->H, MOL_MAX_H);
  if (!p->Q || !p->X) return fail(MOL_EINVAL, "Q or X is NULL");
  if (gating && (!p->a_q || !p->a_x || !p->W1 || !p->b1 || !p->W2 || !p->b2))
    return fail(MOL_EINVAL, "a gating pointer (a_q, a_x, W1, b1, W2, b2) is NULL");
  return MOL_OK;
}

DevProb dev_prob(const mol_problem* p) {
  DevProb d;
  d.B = p->B; d.N = p->N; d.Pq = p->Pq; d.Px = p->Px; d.P = p->Pq * p->Px;
  d.d = p->d; d.H = p->H; d.dtype = p->dtype; d.flags = p->flags;
  d.Q = p->Q; d.X = p->X; d.a_q = p->a_q; d.a_x = p->a_x;
  d.W1 = p->W1; d.b1 = p->b1; d.W2 = p->W2; d.b2 = p->b2;
  return d;
}

// ---------------------------------------------------------------------------
// Streaming top-k over tiles of items (generic path).  For every row the
// keys of one tile plus the running top-k are reduced by repeated segmented
// sorts until k remain.
// ---------------------------------------------------------------------------
// rows longer than this are reduced by radix selection, shorter ones by
// segmented sorts
constexpr long kRadixRowMin = 1l << 15;
constexpr long kRadixChunk = 1l << 14;   // keys per workgroup of the chunked first pass
constexpr int kRadixFewRows = 128;       // rows below which long rows are chunked

struct StreamPlan {
  int rows = 0, k = 0, T = 0;
  long strideA = 0, strideB = 0;
  long sRow = 0;                   // dot buffer: floats per (p, b) row (0: no buffer)
  size_t offRun = 0, offA = 0, offB = 0, offS = 0, bytes = 0;
};

// dots_P, dots_B: when nonzero, a buffer of the tile's component dot
// products [dots_P][dots_B][T] is planned too (the MFMA dots kernel feeds
// the pair-wise kernel through it), and the tile is sized to keep it under
// 512 MB.
StreamPlan plan_stream(int rows, int N, int k, int dots_P = 0, int dots_B = 0) {
  StreamPlan s;
  s.rows = rows;
  s.k = k;
  const long budget = 512l << 20;  // bytes of tile keys
  long T = budget / (8l * rows);
  if (dots_P > 0) T = std::min(T, (512l << 20) / (4l * dots_P * dots_B));
  T = std::max(1024l, std::min(T, static_cast<long>(N)));
  T = (T + 255) / 256 * 256;
  s.T = static_cast<int>(T);
  const long L0 = T + k;
  const int S0 = segment_size_for(static_cast<int>(L0), k);
  s.strideA = L0;
  s.strideB = std::max<long>((L0 + S0 - 1) / S0 * k, k);
  size_t off = 0;
  s.offRun = off; off = align_up(off + 8ul * rows * k);
  s.offA = off;   off = align_up(off + 8ul * rows * s.strideA);
  s.offB = off;   off = align_up(off + 8ul * rows * s.strideB);
  if (dots_P > 0) {
    s.sRow = dots_buffer_row(s.T);
    s.offS = off;  off = align_up(off + 4ul * dots_P * dots_B * s.sRow);
  }
  s.bytes = off;
  return s;
}

// Plan of the tile-streamed pair-wise path of a MoL-scored selection: with
// the MFMA dots kernel where the shape allows.
StreamPlan plan_pairwise(const DevProb& pr, int k) {
  return dots_mfma_supported(pr) ? plan_stream(pr.B, pr.N, k, pr.P, pr.B) : plan_stream(pr.B, pr.N, k);
}

// Score one tile of the pair-wise path into keys A (mode: GenMode).
hipError_t pairwise_tile(const DevProb& pr, const StreamPlan& s, char* w, int mode, const float* bound,
                         int n0, int nt, uint64_t* A, long strideA, hipStream_t st) {
  if (s.sRow == 0)
    return launch_phi_generic(pr, mode, bound, n0, nt, nullptr, nullptr, 0, nullptr, 0, 0, nullptr, 0, A,
                              strideA, st);
  float* sbuf = reinterpret_cast<float*>(w + s.offS);
  const long pstride = s.sRow * pr.B;
  hipError_t e = launch_dots_mfma(pr, n0, nt, kDotsToBuffer, sbuf, pstride, s.sRow, nullptr, 0, st);
  if (e != hipSuccess) return e;
  return (phi_mfma_supported(pr) ? launch_phi_mfma : launch_phi_generic)(
      pr, mode, bound, n0, nt, nullptr, nullptr, 0, sbuf, pstride, s.sRow, nullptr, 0, A, strideA, st);
}

// Reduce rows of `len` keys held in buffer A (stride strideA) to the top k,
// written to `out` (stride out_stride).  Uses A and B as ping-pong buffers.
// gate: NULL, or a device flag; every launch does nothing while it is zero.
int reduce_rows(const StreamPlan& s, char* ws, long len, uint64_t* out, long out_stride,
                hipStream_t st, const uint32_t* gate = nullptr) {
  uint64_t* bufs[2] = {reinterpret_cast<uint64_t*>(ws + s.offA), reinterpret_cast<uint64_t*>(ws + s.offB)};
  long strides[2] = {s.strideA, s.strideB};
  int cur = 0;
  // few long rows: a radix selection per 16K-key chunk first (more
  // workgroups), then the rows of chunk lists are reduced as below.  The
  // chunk lists fit the second buffer: chunks * k <= ceil(len / 4096) * k.
  if (len > 2 * kRadixChunk && s.rows < kRadixFewRows && s.k <= 1024) {
    const int chunks = static_cast<int>((len + kRadixChunk - 1) / kRadixChunk);
    if (static_cast<long>(chunks) * s.k > strides[1]) return fail(MOL_EHIP, "internal: chunk lists too long");
    MOL_TRY_HIP(launch_radix_topk_chunks(bufs[0], strides[0], s.rows, len, s.k, chunks, kRadixChunk, bufs[1], st,
                                         gate),
                "radix top-k per chunk");
    // (rows of chunks * k keys at stride chunks * k)
    strides[1] = static_cast<long>(chunks) * s.k;
    len = strides[1];
    cur = 1;
  }
  // long rows or large k: one radix selection per row
  if (s.k > 1024 || len > kRadixRowMin) {
    MOL_TRY_HIP(launch_radix_topk(bufs[cur], strides[cur], s.rows, len, s.k, out, out_stride, st, nullptr, gate),
                "radix top-k");
    return MOL_OK;
  }
  for (;;) {
    const int S = segment_size_for(static_cast<int>(len), s.k);
    const long nseg = (len + S - 1) / S;
    if (nseg == 1) {
      MOL_TRY_HIP(launch_segment_topk(bufs[cur], strides[cur], s.rows, static_cast<int>(len), s.k,
                                      out, out_stride, st, gate), "segment top-k");
      return MOL_OK;
    }
    const int nxt = 1 - cur;
    if (nseg * s.k > strides[nxt]) return fail(MOL_EHIP, "internal: top-k buffer too small");
    MOL_TRY_HIP(launch_segment_topk(bufs[cur], strides[cur], s.rows, static_cast<int>(len), s.k,
                                    bufs[nxt], strides[nxt], st, gate), "segment top-k");
    len = nseg * s.k;
    cur = nxt;
  }
}

// Tile-by-tile exact selection; `score_tile` writes keys of items
// [n0, n0+nt) into A (row stride strideA).
template <typename F>
int stream_topk(const StreamPlan& s, int N, char* ws, F score_tile, float* out_score,
                int32_t* out_idx, hipStream_t st) {
  uint64_t* run = reinterpret_cast<uint64_t*>(ws + s.offRun);
  uint64_t* A = reinterpret_cast<uint64_t*>(ws + s.offA);
  MOL_TRY_HIP(launch_fill(run, static_cast<long>(s.rows) * s.k, 0ull, st), "fill");
  for (long n0 = 0; n0 < N; n0 += s.T) {
    const int nt = static_cast<int>(std::min<long>(s.T, N - n0));
    MOL_TRY_HIP(score_tile(static_cast<int>(n0), nt, A, s.strideA), "score tile");
    MOL_TRY_HIP(launch_copy_rows(run, s.k, s.rows, s.k, A + nt, s.strideA, st), "copy rows");
    int rc = reduce_rows(s, ws, nt + s.k, run, s.k, st);
    if (rc != MOL_OK) return rc;
  }
  MOL_TRY_HIP(launch_decode(run, s.k, s.rows, s.k, out_score, out_idx, st), "decode");
  return MOL_OK;
}

// Rerank workspace: uniq [B][C], n_unique [B], key rows A/B, final keys,
// and on the generic path with MFMA dots the candidates' dot products.
struct RerankPlan {
  StreamPlan s;
  long sRow = 0;
  size_t offUniq = 0, offNu = 0, offFinal = 0, offS = 0, bytes = 0;
};

RerankPlan plan_rerank(const DevProb& pr, int C, int k) {
  const int B = pr.B;
  RerankPlan r;
  StreamPlan& s = r.s;
  s.rows = B;
  s.k = k;
  s.T = C;
  // generic path: keys of every candidate; fused path: per-chunk top-k lists
  long L0 = C;
  if (rerank_supported(pr, k)) {
    const int chunk = rerank_chunk(B, C);
    L0 = static_cast<long>((C + chunk - 1) / chunk) * k;
  }
  const int S0 = segment_size_for(static_cast<int>(L0), k);
  s.strideA = std::max<long>(L0, k);
  s.strideB = std::max<long>((L0 + S0 - 1) / S0 * k, k);
  size_t off = 0;
  s.offA = off;   off = align_up(off + 8ul * B * s.strideA);
  s.offB = off;   off = align_up(off + 8ul * B * s.strideB);
  r.offFinal = off; off = align_up(off + 8ul * B * k);
  r.offUniq = off;  off = align_up(off + 4ul * B * C);
  r.offNu = off;    off = align_up(off + 4ul * B);
  if (!rerank_supported(pr, k) && dots_mfma_supported(pr)) {
    r.sRow = dots_buffer_row(C);
    r.offS = off;   off = align_up(off + 4ul * pr.P * B * r.sRow);
  }
  r.bytes = off;
  return r;
}

// Exact top-k through the fused kernel: partial lists [B][R][k] are reduced
// to [B][k] by segmented sorts.
struct FusedExactPlan {
  StreamPlan s;  // offA = partial lists (stride R*k), offB = ping-pong
  int R = 0, range_len = 0, G = 0;
  size_t offFinal = 0, offRedo = 0, bytes = 0;
};

FusedExactPlan plan_fused_exact(const DevProb& pr, int k, bool maxdot = false) {
  FusedExactPlan f;
  fused_grid(pr, pr.N, f.R, f.range_len, f.G, maxdot);
  StreamPlan& s = f.s;
  s.rows = pr.B;
  s.k = k;
  const long L0 = static_cast<long>(f.R) * k;
  const int S0 = segment_size_for(static_cast<int>(L0), k);
  s.strideA = L0;
  s.strideB = std::max<long>((L0 + S0 - 1) / S0 * k, k);
  size_t off = 0;
  s.offA = off;     off = align_up(off + 8ul * pr.B * s.strideA);
  s.offB = off;     off = align_up(off + 8ul * pr.B * s.strideB);
  f.offFinal = off; off = align_up(off + 8ul * pr.B * k);
  f.offRedo = off;  off = align_up(off + 4ul * fused_redo_flags(f.R, f.G));
  f.bytes = off;
  return f;
}

// Per-component top-k' through the MFMA kernel: lists [P*B rows][R][KL]
// are reduced to [rows][k'] by segmented sorts.
struct PerEmbdPlan {
  StreamPlan s;
  PerEmbdGrid g;
  int KL = 0;
  size_t offFinal = 0, offStg = 0, offBmax = 0, offThr = 0, offThrT = 0;
  size_t offCtl = 0, offKeys = 0, offHotV = 0, offHotN = 0, offWork = 0, bytes = 0;
};

PerEmbdPlan plan_per_embd(const DevProb& pr, int kp) {
  PerEmbdPlan f;
  per_embd_grid(pr, kp, f.g);
  f.KL = per_embd_list_cap(kp);
  StreamPlan& s = f.s;
  s.rows = pr.B * pr.P;
  s.k = kp;
  const long L0 = static_cast<long>(f.g.s2.R) * f.KL;
  const int S0 = segment_size_for(static_cast<int>(L0), kp);
  s.strideA = L0;
  s.strideB = std::max<long>((L0 + S0 - 1) / S0 * kp, kp);
  size_t off = 0;
  s.offA = off;     off = align_up(off + 8ul * s.rows * s.strideA);
  s.offB = off;     off = align_up(off + 8ul * s.rows * s.strideB);
  f.offFinal = off; off = align_up(off + 8ul * s.rows * kp);
  f.offStg = off;   off = align_up(off + 8ul * s.rows * f.g.s2.R * per_embd_stage_cap(kp));
  f.offBmax = off;  off = align_up(off + 4ul * s.rows * f.g.s1.R * f.g.nbk);
  f.offThr = off;   off = align_up(off + 4ul * s.rows);
  f.offThrT = off;  off = align_up(off + 4ul * s.rows);
  if (f.g.pruned) {
    const size_t nvec = static_cast<size_t>(pr.B) * pr.Pq;
    f.offCtl = off;   off = align_up(off + 4ul * (s.rows + 2) + 4);       // counts, flag, work-list length
    f.offKeys = off;  off = align_up(off + 8ul * s.rows * f.g.key_cap);
    f.offHotV = off;  off = align_up(off + 4ul * f.g.groups * nvec);
    f.offHotN = off;  off = align_up(off + 4ul * f.g.groups);
    f.offWork = off;  off = align_up(off + 4ul * f.g.groups * f.g.CH);
  }
  f.bytes = off;
  return f;
}

PerEmbdBufs per_embd_bufs(const PerEmbdPlan& f, char* w) {
  PerEmbdBufs b;
  b.lists = reinterpret_cast<uint64_t*>(w + f.s.offA);
  b.stg = reinterpret_cast<uint64_t*>(w + f.offStg);
  b.bmax = reinterpret_cast<float*>(w + f.offBmax);
  b.thr = reinterpret_cast<float*>(w + f.offThr);
  b.thr_t = reinterpret_cast<float*>(w + f.offThrT);
  if (f.g.pruned) {
    b.ctl = reinterpret_cast<uint32_t*>(w + f.offCtl);
    b.keys = reinterpret_cast<uint64_t*>(w + f.offKeys);
    b.hot_v = reinterpret_cast<int*>(w + f.offHotV);
    b.hot_n = reinterpret_cast<int*>(w + f.offHotN);
    b.work = reinterpret_cast<int*>(w + f.offWork);
  }
  return b;
}

// Per-component top-k' for the shapes without the fused per-component
// kernels, when the dots run on MFMA: a threshold from a sample, then one
// pass that keeps only the keys reaching it.  The k'-th largest key of any
// subset of a list is at most the list's k'-th largest key, so every key of
// the list's top k' reaches the sample's k'-th key and the selection over
// the kept keys is exact.  The kept-key rows hold every item, so nothing can
// overflow; a sample with fewer than k' keys gives threshold 0 (keep all).
struct ThreshPlan {
  int rows = 0, tile_stride = 1;
  long ns = 0;   // sample slots per row
  size_t offCnt = 0, offSmp = 0, offTk = 0, offCand = 0, offFin = 0, bytes = 0;
};
constexpr int kThreshMinN = 1 << 14;               // shorter rows: the streamed path
constexpr size_t kThreshMaxCand = size_t(2) << 30;  // kept-key rows, bytes

bool use_thresh_per_embd(const DevProb& pr, int kp) {
  return !per_embd_supported(pr, kp) && dots_mfma_supported(pr) && pr.N >= kThreshMinN &&
         8ul * pr.B * pr.P * pr.N <= kThreshMaxCand;
}

ThreshPlan plan_thresh(const DevProb& pr, int kp) {
  ThreshPlan t;
  t.rows = pr.B * pr.P;
  // a 1/8 sample where it still holds 16 k' items per list
  t.tile_stride = static_cast<int>(std::max<long>(1, std::min<long>(8, pr.N / (16l * kp))));
  t.ns = dots_sample_len(pr.N, t.tile_stride);
  size_t off = 0;
  t.offCnt = off;  off = align_up(off + 4ul * t.rows);
  t.offSmp = off;  off = align_up(off + 8ul * t.rows * t.ns);
  t.offTk = off;   off = align_up(off + 8ul * t.rows * kp);
  t.offCand = off; off = align_up(off + 8ul * t.rows * pr.N);
  t.offFin = off;  off = align_up(off + 8ul * t.rows * kp);
  t.bytes = off;
  return t;
}

size_t per_embd_ws_bytes(const DevProb& pr, int kp) {
  if (per_embd_supported(pr, kp)) return plan_per_embd(pr, kp).bytes;
  if (use_thresh_per_embd(pr, kp)) return plan_thresh(pr, kp).bytes;
  return plan_stream(pr.B * pr.P, pr.N, kp).bytes;
}

size_t exact_ws_bytes(const DevProb& pr, int k) {
  return fused_supported(pr, k) ? plan_fused_exact(pr, k).bytes : plan_pairwise(pr, k).bytes;
}

size_t maxdot_ws_bytes(const DevProb& pr, int k) {
  if (fused_maxdot_supported(pr, k)) return plan_fused_exact(pr, k, true).bytes;
  return dots_maxkeys_supported(pr) ? plan_stream(pr.B, pr.N, k).bytes : plan_pairwise(pr, k).bytes;
}

// Algorithm 1 workspace: per-component lists, the rerank output over G,
// the bound, and one region shared by the three phases (they run in order
// on one stream).
struct TwoPassPlan {
  size_t offDots = 0, offIdx = 0, offScore = 0, offRidx = 0, offBound = 0, offWork = 0, bytes = 0;
};

TwoPassPlan plan_two_pass(const DevProb& pr, int k) {
  TwoPassPlan t;
  const size_t lists = static_cast<size_t>(pr.B) * pr.P * k;
  size_t off = 0;
  t.offDots = off;  off = align_up(off + 4 * lists);
  t.offIdx = off;   off = align_up(off + 4 * lists);
  t.offScore = off; off = align_up(off + 4ul * pr.B * k);
  t.offRidx = off;  off = align_up(off + 4ul * pr.B * k);
  t.offBound = off; off = align_up(off + 4ul * pr.B);
  t.offWork = off;
  const size_t work = std::max({per_embd_ws_bytes(pr, k), plan_rerank(pr, pr.P * k, k).bytes,
                                exact_ws_bytes(pr, k)});
  t.bytes = off + align_up(work);
  return t;
}

int check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return MOL_OK;
  if (!ws) return fail(MOL_EINVAL, "workspace is NULL (need %zu bytes)", need);
  if (reinterpret_cast<uintptr_t>(ws) % kAlign)
    return fail(MOL_EINVAL, "workspace must be %zu-byte aligned", kAlign);
  if (have < need) return fail(MOL_EWORKSPACE, "workspace has %zu bytes, needs %zu", have, need);
  return MOL_OK;
}

int check_k(int32_t k, int32_t N, const char* name) {
  if (k < 1 || k > MOL_MAX_K) return fail(MOL_EINVAL, "%s = %d outside [1, %d]", name, k, MOL_MAX_K);
  if (k > N) return fail(MOL_EINVAL, "%s = %d exceeds N = %d", name, k, N);
  return MOL_OK;
}

// Algorithm 1 reranks the P k candidates of the first pass
int check_two_pass_k(const mol_problem* prob, int32_t k) {
  int rc;
  if ((rc = check_k(k, prob->N, "k"))) return rc;
  const long C = static_cast<long>(prob->Pq) * prob->Px * k;
  if (C > MOL_MAX_C) return fail(MOL_EINVAL, "P * k = %ld candidates exceed %d", C, MOL_MAX_C);
  return MOL_OK;
}

// ---------------------------------------------------------------------------
// Entry-point bodies (arguments already validated, workspace checked).
// timed_op: mol_op code under which the main kernel is timed, -1 for none.
// ---------------------------------------------------------------------------

// Exact MoL top-k over the corpus; with `bound` ([B] floats) only the items
// whose max_p s_p can reach bound[b] are ranked.
int run_exact(const DevProb& pr, int k, const float* bound, float* out_score, int32_t* out_idx,
              char* w, int timed_op, hipStream_t st) {
  int rc;
  if (fused_supported(pr, k)) {
    const FusedExactPlan f = plan_fused_exact(pr, k);
    uint64_t* partial = reinterpret_cast<uint64_t*>(w + f.s.offA);
    uint64_t* fin = reinterpret_cast<uint64_t*>(w + f.offFinal);
    int* redo = reinterpret_cast<int*>(w + f.offRedo);
    MOL_TIMED_LAUNCH(timed_op, st, launch_fused_topk(pr, k, f.R, f.range_len, f.G, bound, partial, redo, st),
                     "fused MoL top-k");
    if ((rc = reduce_rows(f.s, w, static_cast<long>(f.R) * k, fin, k, st))) return rc;
    MOL_TRY_HIP(launch_decode(fin, k, pr.B, k, out_score, out_idx, st), "decode");
    return MOL_OK;
  }
  const StreamPlan s = plan_pairwise(pr, k);
  const int mode = bound ? kGenBounded : kGenPhi;
  auto tile = [&](int n0, int nt, uint64_t* A, long strideA) {
    return pairwise_tile(pr, s, w, mode, bound, n0, nt, A, strideA, st);
  };
  return stream_topk(s, pr.N, w, tile, out_score, out_idx, st);
}

// Top-k by the largest component dot product max_p s_p.
int run_maxdot(const DevProb& pr, int k, float* out_score, int32_t* out_idx, char* w, int timed_op,
               hipStream_t st) {
  int rc;
  if (fused_maxdot_supported(pr, k)) {
    const FusedExactPlan f = plan_fused_exact(pr, k, true);
    uint64_t* partial = reinterpret_cast<uint64_t*>(w + f.s.offA);
    uint64_t* fin = reinterpret_cast<uint64_t*>(w + f.offFinal);
    MOL_TIMED_LAUNCH(timed_op, st, launch_fused_maxdot(pr, k, f.R, f.range_len, f.G, partial, st),
                     "fused max-dot top-k");
    if ((rc = reduce_rows(f.s, w, static_cast<long>(f.R) * k, fin, k, st))) return rc;
    MOL_TRY_HIP(launch_decode(fin, k, pr.B, k, out_score, out_idx, st), "decode");
    return MOL_OK;
  }
  if (dots_maxkeys_supported(pr)) {
    // max-component keys straight from the dots GEMM (no dots buffer)
    const StreamPlan s = plan_stream(pr.B, pr.N, k);
    auto tile = [&](int n0, int nt, uint64_t* A, long strideA) {
      return launch_dots_mfma_maxkeys(pr, n0, nt, A, strideA, st);
    };
    return stream_topk(s, pr.N, w, tile, out_score, out_idx, st);
  }
  const StreamPlan s = plan_pairwise(pr, k);
  auto tile = [&](int n0, int nt, uint64_t* A, long strideA) {
    return pairwise_tile(pr, s, w, kGenMaxDot, nullptr, n0, nt, A, strideA, st);
  };
  return stream_topk(s, pr.N, w, tile, out_score, out_idx, st);
}

int run_per_embd(const DevProb& pr, int kprime, float* out_dot, int32_t* out_idx, char* w, int timed_op,
                 hipStream_t st) {
  int rc;
  const int rows = pr.B * pr.P;
  if (per_embd_supported(pr, kprime)) {
    const PerEmbdPlan f = plan_per_embd(pr, kprime);
    const PerEmbdBufs b = per_embd_bufs(f, w);
    uint64_t* fin = reinterpret_cast<uint64_t*>(w + f.offFinal);
    MOL_TIMED_LAUNCH(timed_op, st, launch_per_embd(pr, kprime, f.g, b, st), "per-component top-k'");
    // pruned form: a sort per list, then the threshold scan's lists are
    // reduced only if some list overflowed its key buffer (flag ctl[rows])
    const uint32_t* gate = nullptr;
    if (f.g.pruned) {
      MOL_TRY_HIP(launch_per_embd_select(pr, kprime, f.g, b, out_dot, out_idx, st), "per-component select");
      gate = b.ctl + rows;
    }
    if ((rc = reduce_rows(f.s, w, static_cast<long>(f.g.s2.R) * f.KL, fin, kprime, st, gate))) return rc;
    MOL_TRY_HIP(launch_decode(fin, kprime, rows, kprime, out_dot, out_idx, st, gate), "decode");
    return MOL_OK;
  }
  if (use_thresh_per_embd(pr, kprime)) {
    const ThreshPlan t = plan_thresh(pr, kprime);
    uint32_t* counts = reinterpret_cast<uint32_t*>(w + t.offCnt);
    uint64_t* smp = reinterpret_cast<uint64_t*>(w + t.offSmp);
    uint64_t* tk = reinterpret_cast<uint64_t*>(w + t.offTk);
    uint64_t* cand = reinterpret_cast<uint64_t*>(w + t.offCand);
    uint64_t* fin = reinterpret_cast<uint64_t*>(w + t.offFin);
    MOL_TRY_HIP(launch_fill(reinterpret_cast<uint64_t*>(counts), (rows + 1) / 2, 0ull, st), "clear counts");
    MOL_TRY_HIP(launch_dots_mfma(pr, 0, pr.N, kDotsToKeys, nullptr, 0, 0, smp, t.ns, st, t.tile_stride),
                "sample dots");
    MOL_TRY_HIP(launch_radix_topk(smp, t.ns, rows, t.ns, kprime, tk, kprime, st), "sample top-k'");
    MOL_TRY_HIP(launch_dots_mfma_candidates(pr, 0, pr.N, tk + (kprime - 1), kprime, cand, pr.N, counts, st),
                "thresholded dots");
    MOL_TRY_HIP(launch_radix_topk(cand, pr.N, rows, pr.N, kprime, fin, kprime, st, counts), "top-k'");
    MOL_TRY_HIP(launch_decode(fin, kprime, rows, kprime, out_dot, out_idx, st), "decode");
    return MOL_OK;
  }
  const StreamPlan s = plan_stream(rows, pr.N, kprime);
  const bool gemm = dots_mfma_supported(pr);
  auto tile = [&](int n0, int nt, uint64_t* A, long strideA) {
    return gemm ? launch_dots_mfma(pr, n0, nt, kDotsToKeys, nullptr, 0, 0, A, strideA, st)
                : launch_dots_generic(pr, n0, nt, A, strideA, st);
  };
  return stream_topk(s, pr.N, w, tile, out_dot, out_idx, st);
}

// Union + dedup of two candidate sets, then MoL top-k over the distinct ids
// (by -phi when `negate`: the smallest scores first).
int run_rerank(const DevProb& pr, const int32_t* cand, int C, const int32_t* cand2, int C2, int k,
               bool negate, float* out_score, int32_t* out_idx, int32_t* out_n_unique, char* w,
               int timed_op, hipStream_t st) {
  int rc;
  const int CT = C + C2;
  const RerankPlan r = plan_rerank(pr, CT, k);
  int32_t* uniq = reinterpret_cast<int32_t*>(w + r.offUniq);
  int32_t* nu = reinterpret_cast<int32_t*>(w + r.offNu);
  uint64_t* A = reinterpret_cast<uint64_t*>(w + r.s.offA);
  uint64_t* fin = reinterpret_cast<uint64_t*>(w + r.offFinal);
  MOL_TRY_HIP(launch_dedup(cand, C, cand2, C2, pr.B, pr.N, uniq, nu, st), "dedup");
  if (rerank_supported(pr, k)) {
    const int chunk = rerank_chunk(pr.B, CT);
    const long L0 = static_cast<long>((CT + chunk - 1) / chunk) * k;
    MOL_TIMED_LAUNCH(timed_op, st, launch_rerank(pr, uniq, nu, CT, k, negate, A, st), "fused rerank");
    if ((rc = reduce_rows(r.s, w, L0, fin, k, st))) return rc;
  } else {
    // candidates' dot products on MFMA where the shape allows, then the
    // pair-wise gating kernel
    float* sbuf = r.sRow ? reinterpret_cast<float*>(w + r.offS) : nullptr;
    const long pstride = r.sRow * pr.B;
    if (sbuf)
      MOL_TRY_HIP(launch_dots_mfma_gather(pr, uniq, nu, CT, CT, sbuf, pstride, r.sRow, st), "rerank dots");
    MOL_TIMED_LAUNCH(timed_op, st,
                     (sbuf && phi_mfma_supported(pr) ? launch_phi_mfma : launch_phi_generic)(
                         pr, negate ? kGenNegPhi : kGenPhi, nullptr, 0, CT, uniq, nu, CT, sbuf, pstride,
                         r.sRow, nullptr, 0, A, r.s.strideA, st),
                     "rerank score");
    if ((rc = reduce_rows(r.s, w, CT, fin, k, st))) return rc;
  }
  MOL_TRY_HIP(launch_decode(fin, k, pr.B, k, out_score, out_idx, st), "decode");
  if (out_n_unique)
    MOL_TRY_HIP(hipMemcpyAsync(out_n_unique, nu, sizeof(int32_t) * pr.B, hipMemcpyDeviceToDevice, st),
                "copy n_unique");
  return MOL_OK;
}

// Algorithm 1: G = union over p of TopKDotProduct(k); the bound from the
// MoL scores over G; then the exact top-k over the items whose max_p s_p
// reaches the bound (RangeDotProduct + BruteForceTopKMoL in one pass).
int run_two_pass(const DevProb& pr, int k, int mode, float* out_score, int32_t* out_idx,
                 float* out_bound, char* w, hipStream_t st) {
  int rc;
  const TwoPassPlan t = plan_two_pass(pr, k);
  float* dots = reinterpret_cast<float*>(w + t.offDots);
  int32_t* ids = reinterpret_cast<int32_t*>(w + t.offIdx);
  float* rscore = reinterpret_cast<float*>(w + t.offScore);
  int32_t* ridx = reinterpret_cast<int32_t*>(w + t.offRidx);
  float* bound = reinterpret_cast<float*>(w + t.offBound);
  char* work = w + t.offWork;
  if ((rc = run_per_embd(pr, k, dots, ids, work, -1, st))) return rc;
  const bool smallest = mode == MOL_TWO_PASS_MIN;
  const int kk = smallest ? 1 : k;
  if ((rc = run_rerank(pr, ids, pr.P * k, nullptr, 0, kk, smallest, rscore, ridx, nullptr, work, -1, st)))
    return rc;
  // MIN: bound = min over G of phi = -(top-1 of -phi); KTH: the k-th largest
  MOL_TRY_HIP(launch_pick_bound(rscore, kk, kk - 1, smallest ? -1.f : 1.f, pr.B, bound, st), "bound");
  if ((rc = run_exact(pr, k, bound, out_score, out_idx, work, -1, st))) return rc;
  if (out_bound)
    MOL_TRY_HIP(hipMemcpyAsync(out_bound, bound, sizeof(float) * pr.B, hipMemcpyDeviceToDevice, st),
                "copy bound");
  return MOL_OK;
}

// ---------------------------------------------------------------------------
// Library-owned scratch of mol_topk_exact_noalloc: a file-scope device
// array of MOL_NOALLOC_SCRATCH_BYTES, one copy per GPU, held until the
// process ends.  In host code `scratch` only names the symbol; its device
// address on each GPU comes from hipGetSymbolAddress (taken once per
// device, with that device current) and is the only handle host code
// passes on.  Calls that overlap on one GPU share the array and race.
static __device__ __align__(256) unsigned char scratch[MOL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

struct ScratchTable {
  std::mutex mu;
  void* ptr[kMaxDevices] = {};
};

ScratchTable& scratch_table() {
  static ScratchTable t;
  return t;
}

// Device address of the scratch array on the current device (nullptr and a
// recorded error on failure).
void* scratch_ptr() {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    hip_fail(e, "hipGetDevice");
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    fail(MOL_EUNSUPPORTED, "device %d beyond the %d the scratch table holds", dev, kMaxDevices);
    return nullptr;
  }
  ScratchTable& t = scratch_table();
  std::lock_guard<std::mutex> g(t.mu);
  if (!t.ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
      return nullptr;
    }
    t.ptr[dev] = p;
  }
  return t.ptr[dev];
}

}  // namespace

extern "C" {

const char* mol_last_error(void) { return g_err.c_str(); }

const char* mol_status_str(int status) {
  switch (status) {
    case MOL_OK: return "MOL_OK";
    case MOL_EINVAL: return "MOL_EINVAL: invalid argument";
    case MOL_EUNSUPPORTED: return "MOL_EUNSUPPORTED: shape or dtype not supported";
    case MOL_EWORKSPACE: return "MOL_EWORKSPACE: workspace too small";
    case MOL_EHIP: return "MOL_EHIP: HIP runtime error";
    default: return "unknown mol_status";
  }
}

int mol_workspace_size(const mol_problem* prob, int op, int32_t k, int32_t kprime, int32_t C,
                       size_t* bytes) {
  if (!bytes) return fail(MOL_EINVAL, "bytes is NULL");
  int rc;
  switch (op) {
    case MOL_OP_SCORE:
      if ((rc = check_problem(prob, true))) return rc;
      *bytes = 0;
      return MOL_OK;
    case MOL_OP_TOPK_EXACT:
      if ((rc = check_problem(prob, true))) return rc;
      if ((rc = check_k(k, prob->N, "k"))) return rc;
      *bytes = exact_ws_bytes(dev_prob(prob), k);
      return MOL_OK;
    case MOL_OP_TOPK_PER_EMBD:
      if ((rc = check_problem(prob, false))) return rc;
      if ((rc = check_k(kprime, prob->N, "kprime"))) return rc;
      *bytes = per_embd_ws_bytes(dev_prob(prob), kprime);
      return MOL_OK;
    case MOL_OP_RERANK:
      if ((rc = check_problem(prob, true))) return rc;
      if (k < 1 || k > MOL_MAX_K) return fail(MOL_EINVAL, "k = %d outside [1, %d]", k, MOL_MAX_K);
      if (C < 1 || C > MOL_MAX_C) return fail(MOL_EINVAL, "C = %d outside [1, %d]", C, MOL_MAX_C);
      *bytes = plan_rerank(dev_prob(prob), C, k).bytes;
      return MOL_OK;
    case MOL_OP_TOPK_MAXDOT:
      if ((rc = check_problem(prob, false))) return rc;
      if ((rc = check_k(k, prob->N, "k"))) return rc;
      *bytes = maxdot_ws_bytes(dev_prob(prob), k);
      return MOL_OK;
    case MOL_OP_TOPK_BOUNDED:
      if ((rc = check_problem(prob, true))) return rc;
      if ((rc = check_k(k, prob->N, "k"))) return rc;
      *bytes = exact_ws_bytes(dev_prob(prob), k);
      return MOL_OK;
    case MOL_OP_TOPK_TWO_PASS:
      if ((rc = check_problem(prob, true))) return rc;
      if ((rc = check_two_pass_k(prob, k))) return rc;
      *bytes = plan_two_pass(dev_prob(prob), k).bytes;
      return MOL_OK;
    default:
      return fail(MOL_EINVAL, "unknown op %d", op);
  }
}

int mol_score(const mol_problem* prob, int32_t n_begin, int32_t n_count, float* phi, void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if (n_begin < 0 || n_count < 0 || static_cast<long>(n_begin) + n_count > prob->N)
    return fail(MOL_EINVAL, "item range [%d, %d+%d) outside [0, %d)", n_begin, n_begin, n_count, prob->N);
  if (n_count == 0) return MOL_OK;
  if (!phi) return fail(MOL_EINVAL, "phi is NULL");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const DevProb pr = dev_prob(prob);
  if (fused_supported(pr, 1)) {
    MOL_TIMED_LAUNCH(MOL_OP_SCORE, st, launch_fused_dense(pr, n_begin, n_count, phi, st), "mol_score (fused)");
    return MOL_OK;
  }
  MOL_TIMED_LAUNCH(MOL_OP_SCORE, st,
                   launch_phi_generic(pr, kGenPhi, nullptr, n_begin, n_count, nullptr, nullptr, 0, nullptr, 0,
                                      0, phi, n_count, nullptr, 0, st),
                   "mol_score");
  return MOL_OK;
}

int mol_topk_exact(const mol_problem* prob, int32_t k, float* out_score, int32_t* out_idx, void* ws,
                   size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if ((rc = check_k(k, prob->N, "k"))) return rc;
  if (!out_score || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, exact_ws_bytes(pr, k)))) return rc;
  return run_exact(pr, k, nullptr, out_score, out_idx, static_cast<char*>(ws), MOL_OP_TOPK_EXACT,
                   static_cast<hipStream_t>(stream));
}

int mol_topk_exact_noalloc(const mol_problem* prob, int32_t k, float* out_score, int32_t* out_idx,
                           void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if ((rc = check_k(k, prob->N, "k"))) return rc;
  if (!out_score || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  const size_t need = exact_ws_bytes(pr, k);
  if (need > MOL_NOALLOC_SCRATCH_BYTES)
    return fail(MOL_EWORKSPACE, "this problem needs %zu bytes of scratch; the library holds %zu "
                "(use mol_topk_exact with a workspace)", need, static_cast<size_t>(MOL_NOALLOC_SCRATCH_BYTES));
  char* w = static_cast<char*>(scratch_ptr());
  if (!w) return MOL_EHIP;
  return run_exact(pr, k, nullptr, out_score, out_idx, w, MOL_OP_TOPK_EXACT, static_cast<hipStream_t>(stream));
}

int mol_topk_exact_bounded(const mol_problem* prob, int32_t k, const float* bound, float* out_score,
                           int32_t* out_idx, void* ws, size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if ((rc = check_k(k, prob->N, "k"))) return rc;
  if (!bound) return fail(MOL_EINVAL, "bound is NULL");
  if (!out_score || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, exact_ws_bytes(pr, k)))) return rc;
  return run_exact(pr, k, bound, out_score, out_idx, static_cast<char*>(ws), MOL_OP_TOPK_BOUNDED,
                   static_cast<hipStream_t>(stream));
}

int mol_topk_maxdot(const mol_problem* prob, int32_t k, float* out_score, int32_t* out_idx, void* ws,
                    size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, false))) return rc;
  if ((rc = check_k(k, prob->N, "k"))) return rc;
  if (!out_score || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, maxdot_ws_bytes(pr, k)))) return rc;
  return run_maxdot(pr, k, out_score, out_idx, static_cast<char*>(ws), MOL_OP_TOPK_MAXDOT,
                    static_cast<hipStream_t>(stream));
}

int mol_topk_two_pass(const mol_problem* prob, int32_t k, int32_t mode, float* out_score, int32_t* out_idx,
                      float* out_bound, void* ws, size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if ((rc = check_two_pass_k(prob, k))) return rc;
  if (mode != MOL_TWO_PASS_MIN && mode != MOL_TWO_PASS_KTH)
    return fail(MOL_EINVAL, "mode = %d is not MOL_TWO_PASS_MIN or MOL_TWO_PASS_KTH", mode);
  if (!out_score || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, plan_two_pass(pr, k).bytes))) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const EvPair tp = timing_start(st);
  rc = run_two_pass(pr, k, mode, out_score, out_idx, out_bound, static_cast<char*>(ws), st);
  timing_stop(MOL_OP_TOPK_TWO_PASS, tp, st, rc == MOL_OK);
  return rc;
}

int mol_topk_per_embd(const mol_problem* prob, int32_t kprime, float* out_dot, int32_t* out_idx,
                      void* ws, size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, false))) return rc;
  if ((rc = check_k(kprime, prob->N, "kprime"))) return rc;
  if (!out_dot || !out_idx) return fail(MOL_EINVAL, "output pointer is NULL");
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, per_embd_ws_bytes(pr, kprime)))) return rc;
  return run_per_embd(pr, kprime, out_dot, out_idx, static_cast<char*>(ws), MOL_OP_TOPK_PER_EMBD,
                      static_cast<hipStream_t>(stream));
}

int mol_rerank(const mol_problem* prob, const int32_t* cand, int32_t C, const int32_t* cand2, int32_t C2,
               int32_t k, float* out_score, int32_t* out_idx, int32_t* out_n_unique, void* ws,
               size_t ws_bytes, void* stream) {
  int rc;
  if ((rc = check_problem(prob, true))) return rc;
  if (k < 1 || k > MOL_MAX_K) return fail(MOL_EINVAL, "k = %d outside [1, %d]", k, MOL_MAX_K);
  if (C < 1 || C2 < 0 || static_cast<long>(C) + C2 > MOL_MAX_C)
    return fail(MOL_EINVAL, "C = %d, C2 = %d: need C >= 1, C2 >= 0, C + C2 <= %d", C, C2, MOL_MAX_C);
  if (!cand || !out_score || !out_idx) return fail(MOL_EINVAL, "cand or output pointer is NULL");
  if (C2 > 0 && !cand2) return fail(MOL_EINVAL, "cand2 is NULL with C2 = %d", C2);
  const DevProb pr = dev_prob(prob);
  if ((rc = check_ws(ws, ws_bytes, plan_rerank(pr, C + C2, k).bytes))) return rc;
  return run_rerank(pr, cand, C, cand2, C2, k, false, out_score, out_idx, out_n_unique, static_cast<char*>(ws),
                    MOL_OP_RERANK, static_cast<hipStream_t>(stream));
}

int mol_avg_embed(const mol_problem* prob, void* q_avg, void* x_avg, void* stream) {
  int rc;
  if ((rc = check_problem(prob, false))) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  MOL_TRY_HIP(launch_avg_embed(dev_prob(prob), q_avg, x_avg, st), "avg embed");
  return MOL_OK;
}

int mol_gap_bound(int32_t B, int32_t P, int32_t m, const float* dots, int32_t k, const float* scores,
                  float* out_S, float* out_SK, float* out_bound, float* out_looser, void* stream) {
  if (B < 1 || P < 1 || P > MOL_MAX_P) return fail(MOL_EINVAL, "B = %d, P = %d: need B >= 1, 1 <= P <= %d", B, P, MOL_MAX_P);
  if (m < 2) return fail(MOL_EINVAL, "m = %d: the lists need at least 2 entries", m);
  if (k < 1 || k > MOL_MAX_K) return fail(MOL_EINVAL, "k = %d outside [1, %d]", k, MOL_MAX_K);
  if (!dots || !scores) return fail(MOL_EINVAL, "dots or scores is NULL");
  MOL_TRY_HIP(launch_gap_bound(B, P, m, dots, k, scores, out_S, out_SK, out_bound, out_looser,
                               static_cast<hipStream_t>(stream)), "gap bound");
  return MOL_OK;
}

int mol_gap_bound_combined(int32_t B, int32_t P, int32_t m, const float* dots, const int32_t* ids,
                           int32_t kprime, const int32_t* avg_ids, int32_t k_avg, int32_t k,
                           const float* scores, float* out_S, float* out_SK, float* out_bound, void* stream) {
  if (B < 1 || P < 1 || P > MOL_MAX_P) return fail(MOL_EINVAL, "B = %d, P = %d: need B >= 1, 1 <= P <= %d", B, P, MOL_MAX_P);
  if (kprime < 1 || k_avg < 0 || k_avg > MOL_MAX_K)
    return fail(MOL_EINVAL, "kprime = %d, k_avg = %d: need kprime >= 1, 0 <= k_avg <= %d", kprime, k_avg, MOL_MAX_K);
  if (static_cast<long>(m) <= static_cast<long>(kprime) + k_avg)
    return fail(MOL_EINVAL, "m = %d: the lists need more than kprime + k_avg = %d entries", m, kprime + k_avg);
  if (k < 1 || k > MOL_MAX_K) return fail(MOL_EINVAL, "k = %d outside [1, %d]", k, MOL_MAX_K);
  if (!dots || !ids || !scores) return fail(MOL_EINVAL, "dots, ids or scores is NULL");
  if (k_avg > 0 && !avg_ids) return fail(MOL_EINVAL, "avg_ids is NULL with k_avg = %d", k_avg);
  MOL_TRY_HIP(launch_gap_bound_combined(B, P, m, dots, ids, kprime, avg_ids, k_avg, k, scores, out_S, out_SK,
                                        out_bound, static_cast<hipStream_t>(stream)),
              "combined gap bound");
  return MOL_OK;
}

int mol_timing_enable(int on) {
  TimingLog& t = timing_log();
  std::lock_guard<std::mutex> g(t.mu);
  t.on = on != 0;
  return MOL_OK;
}

int mol_timing_read(int op, double* total_ms, int32_t* launches) {
  if (op < 0 || op >= kTimedOps) return fail(MOL_EINVAL, "unknown op %d", op);
  if (!total_ms || !launches) return fail(MOL_EINVAL, "output pointer is NULL");
  TimingLog& t = timing_log();
  std::lock_guard<std::mutex> g(t.mu);
  double sum = 0.0;
  int32_t n = 0;
  hipError_t err = hipSuccess;
  for (const EvPair& p : t.rec[op]) {
    float ms = 0.f;
    if (err == hipSuccess) err = hipEventSynchronize(p.b);
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, p.a, p.b);
    sum += ms;
    ++n;
    t.spare.push_back(p);
  }
  t.rec[op].clear();
  if (err != hipSuccess) return hip_fail(err, "mol_timing_read");
  *total_ms = sum;
  *launches = n;
  return MOL_OK;
}

}  // extern "C"
