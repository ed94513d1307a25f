/*
 * mol.h -- C ABI of the MI355X (gfx950) Mixture-of-Logits retrieval library.
 *
 * Problem (paper: "Retrieval with Learned Similarities", Section 2 Eq. 1-2,
 * Section 3 Definition 1, Algorithm 2, Appendix A.3):
 *
 *   s_p(q,x)  = < f_pq(q), g_px(x) >,            p = pq * Px + px, P = Pq * Px
 *   u_j       = b1[j] + sum_p W1[j][p] s_p        (j < H)
 *   l_p       = a_q[q][p] + a_x[x][p] + b2[p] + sum_j W2[p][j] SiLU(u_j)
 *   pi        = softmax_p(l)                      (sum_p pi_p = 1)
 *   phi(q,x)  = sum_p pi_p s_p
 *
 * Memory: every array pointer below is a DEVICE pointer owned by the caller.
 * The library allocates no device memory, keeps no pointer after a call
 * returns, and holds no global state other than a per-thread last-error
 * string, the optional kernel-timing records (mol_timing_enable) and the
 * static device scratch array of mol_topk_exact_noalloc.
 * Calls are asynchronous on `stream` (a hipStream_t passed as void*,
 * NULL = the null stream); outputs are valid once the caller has
 * synchronised that stream.  Calls on different streams may run
 * concurrently as long as their outputs and workspaces do not overlap.
 *
 * Layouts (row-major, densely packed, element types by `dtype`):
 *   Q   [B][Pq][d]   query component embeddings            (dtype)
 *   X   [Px][N][d]   item component embeddings, component-major (dtype)
 *   a_q [B][P]  a_x [N][P]  b1 [H]  b2 [P]                 (float32)
 *   W1  [H][P]  W2  [P][H]                                 (dtype)
 * Embeddings are used as given: Eq. 2's L2 normalisation is a
 * precomputation and is never redone by the library.  Inputs must be finite.
 *
 * Ordering: every top-k output row is sorted by score descending, ties
 * broken by item index ascending.  Where a row has fewer than k valid items
 * (mol_rerank, mol_topk_exact_bounded) it is padded with index -1 and score
 * -INFINITY.
 *
 * Errors: each entry point validates all arguments on the host before it
 * launches anything.  On error it returns a nonzero mol_status, launches
 * nothing, leaves outputs untouched, and records a message retrievable with
 * mol_last_error() on the calling thread.  MOL_EHIP reports a HIP runtime
 * failure at launch time (the message carries the HIP error string).
 */
#ifndef MOL_H_
#define MOL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOL_OK = 0,
  MOL_EINVAL = 1,        /* null pointer, size out of range, bad k          */
  MOL_EUNSUPPORTED = 2,  /* shape or dtype outside the kernel set           */
  MOL_EWORKSPACE = 3,    /* workspace smaller than mol_workspace_size says  */
  MOL_EHIP = 4           /* HIP runtime error on launch                     */
} mol_status;

typedef enum { MOL_F32 = 0, MOL_BF16 = 1 } mol_dtype;

/* Operation codes for mol_workspace_size. */
typedef enum {
  MOL_OP_SCORE = 0,
  MOL_OP_TOPK_EXACT = 1,
  MOL_OP_TOPK_PER_EMBD = 2,
  MOL_OP_RERANK = 3,
  MOL_OP_TOPK_MAXDOT = 4,
  MOL_OP_TOPK_BOUNDED = 5,
  MOL_OP_TOPK_TWO_PASS = 6
} mol_op;

/* Threshold of the two-pass exact algorithm (mol_topk_two_pass). */
typedef enum {
  MOL_TWO_PASS_MIN = 0,  /* Algorithm 1: smallest MoL score over G           */
  MOL_TWO_PASS_KTH = 1   /* k-th largest MoL score over G (tighter)          */
} mol_two_pass_mode;

/* Problem flags (mol_problem.flags). */
#define MOL_FLAG_F32_GATING 1u     /* gating MLP in float32 (see mol_problem)        */
#define MOL_FLAG_BF16X2_GATING 2u  /* gating MLP on two-term bf16 operands (ditto)    */

/* Limits of the kernel set. */
#define MOL_MAX_B 65535   /* queries per call                                */
#define MOL_MAX_P 64      /* Pq * Px                                        */
#define MOL_MAX_H 256     /* gating MLP hidden width                         */
#define MOL_MAX_D 1024    /* component embedding width                       */
#define MOL_MAX_K 8192    /* k of every top-k output                         */
#define MOL_MAX_C 16384   /* candidates per query handed to mol_rerank       */

/* One retrieval problem: shapes, storage type and device pointers (the
 * notation table of Section 2; gating parameters per Appendix A.3).
 * Pointers not used by an entry point may be NULL (see each function).
 *
 * Precision of the gating MLP.  By default the bf16 fused kernels evaluate
 * it on matrix cores with float16 operands: s, -log2(e) W1 and the hidden
 * activations are rounded to float16 (W2 is exact), accumulation is
 * float32.  The resulting error in phi grows with the scale of W1 and W2:
 * measured against float64 on the exact_1m data recipe, its largest value
 * over 16 x 4096 pairs is 2.2e-6 for entries of standard deviation 0.1,
 * 7.8e-6 for 0.2, 2.0e-5 for 0.3 and 1.5e-4 for 0.5.  The fused path is
 * meant for gating weights with entries of RMS up to 0.3.  Beyond that,
 * set one of two flags:
 *  - MOL_FLAG_BF16X2_GATING: the fused kernels take W1 and W2 exactly (bf16)
 *    and carry -log2(e) s and the hidden activations as two bf16 terms each
 *    (hi + lo, about 16 significant bits), with float32 accumulation: twice
 *    the matrix work of the chain's two gating products.  Its error on the
 *    same recipe: 4.3e-6 for entries of standard deviation 0.5, 7.6e-6 to
 *    2.0e-5 for 1.0, but up to 7.0e-5 for 2.0, so it is meant for entries
 *    of RMS up to 1.  bf16 shapes without a fused kernel take the same
 *    two-term chain in the pair-wise kernel (P <= 64, H <= 128), others
 *    the float32 path below.
 *  - MOL_FLAG_F32_GATING: the gating MLP, softmax and phi run in float32 in
 *    the pair-wise kernel (component dots still on matrix cores, exact
 *    products, float32 sums), more than ten times slower than the fused
 *    path, with no limit on the weights.  It takes precedence when both
 *    flags are set.
 * float32 problems always take the float32 path. */
typedef struct mol_problem {
  int32_t B;      /* number of queries                                      */
  int32_t N;      /* number of items                                        */
  int32_t Pq;     /* query components                                       */
  int32_t Px;     /* item components                                        */
  int32_t d;      /* component embedding width d_P                          */
  int32_t H;      /* gating MLP hidden width                                */
  int32_t dtype;  /* mol_dtype of Q, X, W1, W2                              */
  const void *Q;
  const void *X;
  const float *a_q;
  const float *a_x;
  const void *W1;
  const float *b1;
  const void *W2;
  const float *b2;
  uint32_t flags; /* MOL_FLAG_* bits; 0 for the defaults                    */
} mol_problem;

/* Bytes of workspace an entry point needs for this problem (k, kprime and C
 * as they will be passed; ignored where irrelevant).  Writes *bytes.
 * Returns MOL_OK or the validation error the entry point would return. */
int mol_workspace_size(const mol_problem *prob, int op, int32_t k,
                       int32_t kprime, int32_t C, size_t *bytes);

/* Dense MoL scores (Eq. 1 with the Appendix A.3 gating) of every query
 * against items n_begin .. n_begin + n_count - 1:
 *   phi[b][i] = phi(q_b, x_{n_begin + i}),   phi is float32 [B][n_count].
 * Needs every problem pointer.  n_count == 0 is a no-op.  No workspace. */
int mol_score(const mol_problem *prob, int32_t n_begin, int32_t n_count,
              float *phi, void *stream);

/* Exact top-k with MoL (Definition 1; the paper's brute-force baseline):
 * for every query, the k items of the whole corpus with the largest phi.
 * out_score float32 [B][k], out_idx int32 [B][k].  1 <= k <= min(N, 8192).
 * Needs every problem pointer and mol_workspace_size(MOL_OP_TOPK_EXACT)
 * bytes of workspace (any alignment of 256 bytes or more). */
int mol_topk_exact(const mol_problem *prob, int32_t k, float *out_score,
                   int32_t *out_idx, void *ws, size_t ws_bytes, void *stream);

/* Bytes of device scratch the library itself holds on each GPU for
 * mol_topk_exact_noalloc. */
#define MOL_NOALLOC_SCRATCH_BYTES (16u << 20)

/* mol_topk_exact without a workspace argument and without allocating, for
 * callers that cannot allocate device memory at call time (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same computation, outputs, ordering and limits as mol_topk_exact; the
 * workspace mol_topk_exact would take (mol_workspace_size with
 * MOL_OP_TOPK_EXACT) must be at most MOL_NOALLOC_SCRATCH_BYTES, which
 * covers the fused shapes at up to 1024 queries and k <= 128 (e.g. B = 1024,
 * N = 2^20, P = 8 x 8, d = 64: 4.7 MiB); larger needs return
 * MOL_EWORKSPACE and launch nothing.  The scratch is a static device array
 * of the library, one per GPU, kept until the process ends and located on
 * each device's first call.  Every call on a GPU uses that GPU's one array:
 * calls that overlap on the same GPU (two streams, two threads) race and
 * must be serialised by the caller.  The kernels write every scratch byte
 * they read, so no clearing is needed between calls.  Nothing is allocated,
 * freed or synchronised. */
int mol_topk_exact_noalloc(const mol_problem *prob, int32_t k, float *out_score,
                           int32_t *out_idx, void *stream);

/* Exact top-k with MoL among the items that can reach a per-query bound
 * (Algorithm 1's RangeDotProduct followed by BruteForceTopKMoL, in one pass
 * over the corpus).  phi is a convex combination of the s_p, so
 * phi(q, x) <= m(q, x) = max_p s_p(q, x); for query b only items with
 * m + margin >= bound[b] are scored and ranked, margin = 2^-12 (1 +
 * max_p |s_p|) covering float32 rounding of phi.  Whenever bound[b] is at
 * most the k-th largest phi over the corpus the result equals
 * mol_topk_exact's, bit for bit; with a higher bound it is the top-k of the
 * qualifying items (padded with -INFINITY / -1).  bound float32 [B], device.
 * Groups of items that cannot qualify (nor beat the running k-th score)
 * skip the gating MLP, which is where the time goes.  Same outputs, limits
 * and workspace as mol_topk_exact (mol_workspace_size(MOL_OP_TOPK_BOUNDED)). */
int mol_topk_exact_bounded(const mol_problem *prob, int32_t k,
                           const float *bound, float *out_score,
                           int32_t *out_idx, void *ws, size_t ws_bytes,
                           void *stream);

/* Two-pass exact top-k (Algorithm 1, Section 3.1):
 *   1. G = union over p of TopKDotProduct(f_p(q), X_p) with K = k items each
 *      (mol_topk_per_embd with kprime = k);
 *   2. the bound: mode MOL_TWO_PASS_MIN, the smallest MoL score over G (the
 *      algorithm as given); MOL_TWO_PASS_KTH, the k-th largest MoL score
 *      over G (G holds k items scoring at least that much, so it is also at
 *      most the corpus-wide k-th score: the same result, fewer items pass);
 *   3. the exact top-k over the items with max_p s_p >= bound
 *      (mol_topk_exact_bounded).
 * out_score float32 [B][k], out_idx int32 [B][k]: equal to mol_topk_exact's
 * output.  out_bound float32 [B] (may be NULL): the bound used per query.
 * 1 <= k <= min(N, 8192) and P k <= 16384.  Needs every problem pointer and
 * mol_workspace_size(MOL_OP_TOPK_TWO_PASS) bytes of workspace. */
int mol_topk_two_pass(const mol_problem *prob, int32_t k, int32_t mode,
                      float *out_score, int32_t *out_idx, float *out_bound,
                      void *ws, size_t ws_bytes, void *stream);

/* Max-component top-k (Section 3's "max approximation of MoL", a
 * subsection the published text cuts): for every query, the k
 * items with the largest m(q, x) = max_p s_p(q, x).  Since phi <= m, it is
 * also the candidate generator whose k-th score bounds Algorithm 1's range.
 * out_score float32 [B][k] (the m values), out_idx int32 [B][k].
 * 1 <= k <= min(N, 8192).  Reads only Q and X (gating pointers may be NULL,
 * H is ignored).  Workspace: mol_workspace_size(MOL_OP_TOPK_MAXDOT). */
int mol_topk_maxdot(const mol_problem *prob, int32_t k, float *out_score,
                    int32_t *out_idx, void *ws, size_t ws_bytes, void *stream);

/* TopKPerEmbedding stage 1 (Algorithm 2, TopKDotProduct for every
 * component): for every query b and component p = pq * Px + px, the k'
 * items with the largest s_p = <f_pq(q_b), g_px(x)>.
 * out_dot float32 [B][P][k'], out_idx int32 [B][P][k'].
 * 1 <= kprime <= min(N, 8192).  Reads only Q and X (a_q, a_x, W1, b1, W2,
 * b2 may be NULL; H is ignored).  TopKAvg (Section 3.2) is this call on the
 * averaged problem: Pq = Px = 1, Q = q', X = x' from mol_avg_embed. */
int mol_topk_per_embd(const mol_problem *prob, int32_t kprime, float *out_dot,
                      int32_t *out_idx, void *ws, size_t ws_bytes,
                      void *stream);

/* Candidate union, deduplication and MoL rerank (Algorithm 2: the union G
 * of the candidate sets, deduplicated, then BruteForceTopKMoL over G).
 * cand int32 [B][C] and cand2 int32 [B][C2]: two candidate sets per query
 * (e.g. TopKPerEmbedding's [B][P][k'] ids and TopKAvg's [B][k_avg]); cand2
 * may be NULL when C2 == 0.  Duplicates are allowed; an id outside [0, N)
 * (e.g. -1) marks an empty slot and is skipped.  For each query the
 * distinct ids of both sets are scored with full MoL and the top-k kept.
 * out_score float32 [B][k], out_idx int32 [B][k] (padded with -INFINITY /
 * -1 when a query has fewer than k distinct ids), out_n_unique int32 [B]
 * (may be NULL).  C >= 1, C2 >= 0, C + C2 <= 16384, 1 <= k <= 8192.
 * Needs every problem pointer; mol_workspace_size takes C + C2 as C. */
int mol_rerank(const mol_problem *prob, const int32_t *cand, int32_t C,
               const int32_t *cand2, int32_t C2, int32_t k, float *out_score,
               int32_t *out_idx, int32_t *out_n_unique, void *ws,
               size_t ws_bytes, void *stream);

/* TopKAvg materialisation (Section 3.2, Algorithm 2 TopKAvg):
 *   q_avg[b][t] = round( sum_pq Q[b][pq][t] ),  [B][d]
 *   x_avg[n][t] = round( sum_px X[px][n][t] ),  [N][d]
 * each sum formed exactly (float64) and rounded once to dtype, nearest-even.
 * The averaged dot product's 1/P factor does not change any ranking and is
 * left out.  Either output pointer may be NULL to skip it.  No workspace. */
int mol_avg_embed(const mol_problem *prob, void *q_avg, void *x_avg,
                  void *stream);

/* Gap certificate of TopKPerEmbedding (Theorem 2, Definition 2).
 * dots float32 [B][P][m]: per-component lists sorted descending, as written
 * by mol_topk_per_embd with kprime = m (m >= 2); scores float32 [B][k]: the
 * MoL top-k (descending, as written by mol_rerank) over candidates that
 * include at least the first m - 1 ids of every list.  Writes, per query b:
 *   out_S[b]      = max_p dots[b][p][m - 1]   (the largest m-th dot product:
 *                   no item outside the candidates has a larger MoL score)
 *   out_SK[b]     = scores[b][k - 1]          (the k-th retrieved MoL score)
 *   out_bound[b]  = out_S[b] - out_SK[b]      (>= the gap of Definition 2)
 *   out_looser[b] = max_p dots[b][p][m - 2] - out_SK[b]
 * (the looser bound of Theorem 2).  Any output pointer may be NULL.  Pure
 * device reduction, no workspace.  1 <= k <= 8192, P <= 64. */
int mol_gap_bound(int32_t B, int32_t P, int32_t m, const float *dots,
                  int32_t k, const float *scores, float *out_S, float *out_SK,
                  float *out_bound, float *out_looser, void *stream);

/* Gap certificate of the combined heuristic (Theorem 3).
 * dots float32 [B][P][m], ids int32 [B][P][m]: per-component lists sorted
 * descending (mol_topk_per_embd with kprime = m), m > kprime + k_avg;
 * avg_ids int32 [B][k_avg]: the TopKAvg ids (negative = empty slot; may be
 * NULL when k_avg == 0); scores float32 [B][k]: the MoL top-k (descending)
 * over candidates that include the first kprime ids of every list and all
 * of avg_ids.  Writes, per query b:
 *   out_S[b]     = S', the largest s_p over items outside the union of the
 *                  first kprime ids of list p and avg_ids, maximised over p
 *                  (no item outside the candidates has a larger MoL score)
 *   out_SK[b]    = scores[b][k - 1]
 *   out_bound[b] = out_S[b] - out_SK[b]   (>= the gap of Definition 2)
 * With k_avg == 0 it is Theorem 2's bound.  Any output may be NULL.  Pure
 * device work, no workspace.  P <= 64, kprime >= 1, 0 <= k_avg <= 8192,
 * 1 <= k <= 8192. */
int mol_gap_bound_combined(int32_t B, int32_t P, int32_t m, const float *dots,
                           const int32_t *ids, int32_t kprime,
                           const int32_t *avg_ids, int32_t k_avg, int32_t k,
                           const float *scores, float *out_S, float *out_SK,
                           float *out_bound, void *stream);

/* Kernel timing, a diagnostic for throughput measurements.
 * mol_timing_enable(1) makes every later call record a pair of HIP events on
 * its stream around its main kernel: the fused scoring kernel of mol_score,
 * the scoring + per-range top-k scan of mol_topk_exact (and of
 * mol_topk_exact_bounded, mol_topk_maxdot), the whole sequence of
 * mol_topk_two_pass, the two
 * per-component scans (with the threshold selection between them) of
 * mol_topk_per_embd and the candidate scoring of mol_rerank
 * (validation, merges of partial lists and decoding are outside the pair).
 * mol_timing_enable(0) stops recording; records already taken stay.
 * mol_timing_read(op, &ms, &n) waits for the recorded events of operation
 * `op` (a mol_op code), writes their summed duration in milliseconds and
 * their count, and clears them.  Process-wide and thread-safe; events are
 * created on first use and reused, never freed; every recorded stream must
 * belong to the device that is current when reading.  Returns MOL_EINVAL
 * for an unknown op or NULL output, MOL_EHIP if an event wait fails. */
int mol_timing_enable(int on);
int mol_timing_read(int op, double *total_ms, int32_t *launches);

/* Static description of a status code. */
const char *mol_status_str(int status);

/* Message of the last failing call on this thread ("" if none). */
const char *mol_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MOL_H_ */
