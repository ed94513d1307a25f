"""Plain FP64 CPU oracle for Mixture-of-Logits (MoL) retrieval.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module; only the test suite, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the GPU library.

What it computes (all arithmetic in float64, on inputs decoded exactly from
the stored bfloat16 / float32 arrays):

* component dot products  s_p = <f_pq(q), g_px(x)>,  p = pq * P_x + px
  (Section 2, Eq. 1 and its outer-product form Eq. 2; the embeddings arrive
  already L2-normalised, since Eq. 2's normalisation can be precomputed);
* gating weights pi = softmax_p(l), with gating logits
  l = a_q[q] + a_x[x] + b2 + W2 SiLU(W1 s + b1)  (Appendix A.3: a two-layer
  SiLU MLP over the P dot products, plus per-query and per-item gating
  logits);
* phi(q, x) = sum_p pi_p s_p  (Eq. 1), with sum_p pi_p = 1;
* exact top-K (Definition 1) by sorting all items on (phi desc, index asc);
* the approximate path of Algorithm 2: TopKPerEmbedding (top-K' per
  component by dot product, union, dedup), TopKAvg (top-K by the dot product
  of the summed query and item components, Section 3.2), their combination,
  and the MoL rerank of the deduplicated candidates;
* Algorithm 1 (exact two-pass top-K, with its second pass also available on
  its own for a given threshold), the max approximation of MoL (top-K by
  max_p s_p, a subsection of Section 3 cut from the published text),
  Definition 2 (gap of an approximate top-K) and the gap bounds of
  Theorems 2 and 3.

Parity status: every function here is pinned by the CPU tests against the
paper's worked example (Appendix B), closed forms or brute force, except the
recall figures reported on synthetic data ("parity unpinned": the paper has no
values for these distributions).
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

CHUNK = 1 << 16  # items scored per block (bounds the float64 temporaries)


# --------------------------------------------------------------------------
# Storage formats
# --------------------------------------------------------------------------
def decode(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of a stored array ("bf16" = uint16 bit patterns)."""
    if dtype == "bf16":
        a = np.ascontiguousarray(arr, dtype=np.uint16)
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage type, round-to-nearest-even.

    bf16 keeps 8 significant bits and float32's exponent range; the result
    is returned as uint16 bit patterns.  Values are assumed finite and below
    the bf16 overflow threshold.
    """
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype != "bf16":
        raise ValueError(f"unknown dtype {dtype!r}")
    _, e = np.frexp(x)                      # x = m 2^e, 0.5 <= |m| < 1
    ulp = np.ldexp(1.0, np.maximum(e - 8, -133))   # 8 significant bits; subnormal floor
    r = np.round(x / ulp) * ulp              # np.round: ties to even
    r = np.where(x == 0, 0.0 * x, r)         # keep signed zero
    return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


class Problem:
    """One MoL retrieval problem held on the host.

    Arrays follow the library's layouts: Q [B][Pq][d], X [Px][N][d]
    (component-major), a_q [B][P], a_x [N][P], W1 [H][P], b1 [H], W2 [P][H],
    b2 [P].  Q, X, W1, W2 are in the storage dtype; the rest float32.
    X is decoded block by block, so very large corpora fit in host memory.
    """

    def __init__(self, Q, X, a_q, a_x, W1, b1, W2, b2, dtype: str):
        self.dtype = dtype
        self.Qraw = np.asarray(Q)
        self.X = np.asarray(X)
        self.Px, self.N, self.d = self.X.shape
        B, self.Pq, d2 = self.Qraw.shape
        if d2 != self.d:
            raise ValueError("Q and X disagree on d")
        self.B = B
        self.P = self.Pq * self.Px
        self.Q = decode(self.Qraw, dtype)
        self.a_q = np.asarray(a_q, dtype=np.float64).reshape(B, self.P)
        self.a_x = np.asarray(a_x, dtype=np.float32).reshape(self.N, self.P)
        self.W1 = decode(W1, dtype).reshape(-1, self.P)
        self.H = self.W1.shape[0]
        self.b1 = np.asarray(b1, dtype=np.float64).reshape(self.H)
        self.W2 = decode(W2, dtype).reshape(self.P, self.H)
        self.b2 = np.asarray(b2, dtype=np.float64).reshape(self.P)
        for name in ("Q", "a_q", "W1", "b1", "W2", "b2"):
            if not np.all(np.isfinite(getattr(self, name))):
                raise ValueError(f"non-finite values in {name}")

    @classmethod
    def from_arrays(cls, arrays: Dict[str, object]) -> "Problem":
        return cls(arrays["Q"], arrays["X"], arrays["a_q"], arrays["a_x"],
                   arrays["W1"], arrays["b1"], arrays["W2"], arrays["b2"],
                   arrays["dtype"])

    def items(self, idx) -> np.ndarray:
        """Decoded item components [Px][len(idx)][d] for items ``idx``
        (a slice or an index array)."""
        return decode(self.X[:, idx, :], self.dtype)


# --------------------------------------------------------------------------
# MoL score: Eq. 1 / Eq. 2 with the gating MLP of Appendix A.3
# --------------------------------------------------------------------------
def component_dots(q: np.ndarray, xs: np.ndarray) -> np.ndarray:
    """s[n, p] = <f_pq(q), g_px(x_n)> for p = pq * Px + px.

    q: [Pq][d] one query's components; xs: [Px][n][d] item components.
    """
    Pq = q.shape[0]
    Px, n, _ = xs.shape
    s = np.empty((n, Pq, Px), dtype=np.float64)
    for px in range(Px):
        s[:, :, px] = xs[px] @ q.T          # [n][Pq]
    return s.reshape(n, Pq * Px)


def silu(u: np.ndarray) -> np.ndarray:
    """SiLU(u) = u * sigmoid(u)."""
    with np.errstate(over="ignore"):
        return u / (1.0 + np.exp(-u))


def gating_logits(prob: Problem, b: int, items, s: np.ndarray) -> np.ndarray:
    """l[n, p] = a_q[b,p] + a_x[n,p] + b2[p] + sum_j W2[p,j] SiLU(u_j),
    u_j = b1[j] + sum_p W1[j,p] s[n,p]."""
    u = s @ prob.W1.T + prob.b1                         # [n][H]
    h = silu(u)
    ax = prob.a_x[items].astype(np.float64)             # [n][P]
    return prob.a_q[b] + ax + prob.b2 + h @ prob.W2.T


def softmax(l: np.ndarray) -> np.ndarray:
    """Softmax over the last axis, with the maximum subtracted first."""
    z = np.exp(l - l.max(axis=-1, keepdims=True))
    return z / z.sum(axis=-1, keepdims=True)


def mol_terms(prob: Problem, b: int, items) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(s, pi, phi) for query b against ``items`` (slice or index array)."""
    s = component_dots(prob.Q[b], prob.items(items))
    pi = softmax(gating_logits(prob, b, items, s))
    phi = (pi * s).sum(axis=-1)
    return s, pi, phi


def mol_scores(prob: Problem, queries: Sequence[int], n_begin: int = 0,
               n_count: Optional[int] = None) -> np.ndarray:
    """phi[len(queries)][n_count] for items n_begin .. n_begin+n_count-1."""
    n_count = prob.N - n_begin if n_count is None else n_count
    out = np.empty((len(queries), n_count), dtype=np.float64)
    for c0 in range(n_begin, n_begin + n_count, CHUNK):
        c1 = min(c0 + CHUNK, n_begin + n_count)
        xs = prob.items(slice(c0, c1))
        for i, b in enumerate(queries):
            s = component_dots(prob.Q[b], xs)
            pi = softmax(gating_logits(prob, b, slice(c0, c1), s))
            out[i, c0 - n_begin:c1 - n_begin] = (pi * s).sum(axis=-1)
    return out


# --------------------------------------------------------------------------
# Top-K selection (Definition 1): order by (score desc, index asc)
# --------------------------------------------------------------------------
def topk_desc(values: np.ndarray, k: int, ids: Optional[np.ndarray] = None
              ) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k of ``values`` ordered by (value desc, id asc).

    Returns (values, ids) of length min(k, n).  ``ids`` defaults to
    positions.  Exact: every element tied with the k-th value is considered
    before the id tie-break is applied.
    """
    values = np.asarray(values, dtype=np.float64)
    n = values.shape[0]
    ids = np.arange(n, dtype=np.int64) if ids is None else np.asarray(ids, dtype=np.int64)
    k = min(k, n)
    if k <= 0:
        return values[:0], ids[:0]
    if k < n:
        kth = np.partition(values, n - k)[n - k]          # k-th largest
        cand = np.nonzero(values >= kth)[0]
    else:
        cand = np.arange(n)
    order = np.lexsort((ids[cand], -values[cand]))[:k]
    sel = cand[order]
    return values[sel], ids[sel]


def kth_largest(values: np.ndarray, k: int) -> float:
    """k-th largest value counted with multiplicity (1-based); -inf if k > n."""
    n = values.shape[0]
    if k > n:
        return -math.inf
    return float(np.partition(values, n - k)[n - k])


def exact_topk(prob: Problem, queries: Sequence[int], k: int
               ) -> Tuple[np.ndarray, np.ndarray]:
    """Brute-force MoL top-k (Definition 1) for each query in ``queries``:
    phi for all N items, then sort.  Returns ([nq][k] scores, [nq][k] ids)."""
    phi = mol_scores(prob, queries)
    out_s = np.empty((len(queries), k))
    out_i = np.empty((len(queries), k), dtype=np.int64)
    for i in range(len(queries)):
        out_s[i], out_i[i] = topk_desc(phi[i], k)
    return out_s, out_i


# --------------------------------------------------------------------------
# Approximate retrieval (Algorithm 2, Section 3.2)
# --------------------------------------------------------------------------
def all_dots(prob: Problem, b: int) -> np.ndarray:
    """s[N][P] for query b over the whole corpus."""
    s = np.empty((prob.N, prob.P), dtype=np.float64)
    for c0 in range(0, prob.N, CHUNK):
        c1 = min(c0 + CHUNK, prob.N)
        s[c0:c1] = component_dots(prob.Q[b], prob.items(slice(c0, c1)))
    return s


def topk_per_embedding(prob: Problem, b: int, kprime: int
                       ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """TopKPerEmbedding stage 1 for query b: for each component p, the top-k'
    items by s_p (TopKDotProduct).  Returns (dots [P][k'], ids [P][k'],
    kth [P] = k'-th largest s_p, next [P] = (k'+1)-th largest s_p)."""
    s = all_dots(prob, b)
    P = prob.P
    dots = np.empty((P, kprime))
    ids = np.empty((P, kprime), dtype=np.int64)
    kth = np.empty(P)
    nxt = np.empty(P)
    for p in range(P):
        dots[p], ids[p] = topk_desc(s[:, p], kprime)
        kth[p] = kth_largest(s[:, p], kprime)
        nxt[p] = kth_largest(s[:, p], kprime + 1)
    return dots, ids, kth, nxt


def averaged_embeddings(prob: Problem) -> Tuple[np.ndarray, np.ndarray]:
    """TopKAvg's materialised embeddings (Section 3.2): q' = sum_pq f_pq(q),
    x' = sum_px g_px(x), each summed in float64 and rounded to the storage
    type.  The 1/P factor of the averaged dot product is a positive constant
    and does not change the ranking, so it is left out.
    Returns (q' [B][d], x' [N][d]) in the storage format."""
    qbar = round_to_storage(prob.Q.sum(axis=1), prob.dtype)
    xbar = np.empty((prob.N, prob.d), dtype=np.uint16 if prob.dtype == "bf16" else np.float32)
    for c0 in range(0, prob.N, CHUNK):
        c1 = min(c0 + CHUNK, prob.N)
        xbar[c0:c1] = round_to_storage(prob.items(slice(c0, c1)).sum(axis=0), prob.dtype)
    return qbar, xbar


def averaged_problem(prob: Problem) -> Problem:
    """The P = 1 problem whose only component is (q', x'); gating inputs are
    zero (a single component always has weight 1)."""
    qbar, xbar = averaged_embeddings(prob)
    one = np.zeros((1, 1), dtype=np.float32)
    return Problem(qbar[:, None, :], xbar[None, :, :],
                   np.zeros((prob.B, 1), np.float32), np.zeros((prob.N, 1), np.float32),
                   round_to_storage(one, prob.dtype), np.zeros(1, np.float32),
                   round_to_storage(one, prob.dtype), np.zeros(1, np.float32), prob.dtype)


def topk_avg(prob: Problem, b: int, k: int, avg: Optional[Problem] = None
             ) -> Tuple[np.ndarray, np.ndarray]:
    """TopKAvg: top-k items by <q', x'>.  Returns (dots [k], ids [k])."""
    avg = averaged_problem(prob) if avg is None else avg
    d, i, _, _ = topk_per_embedding(avg, b, k)
    return d[0], i[0]


def union_dedup(cands: Iterable[np.ndarray]) -> np.ndarray:
    """Deduplicated union of candidate id lists (Algorithm 2's G), ascending;
    negative ids mark empty slots and are dropped."""
    allc = np.concatenate([np.asarray(c, dtype=np.int64).ravel() for c in cands])
    return np.unique(allc[allc >= 0])


def rerank(prob: Problem, b: int, cand: np.ndarray, k: int
           ) -> Tuple[np.ndarray, np.ndarray, int]:
    """BruteForceTopKMoL over a candidate set: dedup ``cand``, score the
    unique ids with full MoL, keep the top-k.  Pads with (-inf, -1) when
    fewer than k unique candidates exist.  Returns (scores, ids, n_unique)."""
    uniq = union_dedup([cand])
    _, _, phi = mol_terms(prob, b, uniq)
    s, i = topk_desc(phi, k, ids=uniq)
    out_s = np.full(k, -np.inf)
    out_i = np.full(k, -1, dtype=np.int64)
    out_s[:len(s)], out_i[:len(i)] = s, i
    return out_s, out_i, len(uniq)


def approx_topk(prob: Problem, b: int, k: int, kprime: int, k_avg: int = 0,
                avg: Optional[Problem] = None) -> Dict[str, object]:
    """Algorithm 2, ApproxTopK: candidates from TopKPerEmbedding(k') (and,
    when k_avg > 0, TopKAvg(k_avg): the combined heuristic), deduplicated,
    then reranked with MoL to the top-k."""
    dots, ids, kth, nxt = topk_per_embedding(prob, b, kprime) if kprime > 0 else (
        None, np.empty((0, 0), np.int64), None, None)
    lists = [ids]
    avg_ids = np.empty(0, np.int64)
    if k_avg > 0:
        _, avg_ids = topk_avg(prob, b, k_avg, avg)
        lists.append(avg_ids)
    cand = np.concatenate([l.ravel() for l in lists])
    scores, out_ids, n_unique = rerank(prob, b, cand, k)
    return dict(scores=scores, ids=out_ids, n_unique=n_unique, cand=cand,
                per_embd_dots=dots, per_embd_ids=ids, kth=kth, next=nxt,
                avg_ids=avg_ids)


# --------------------------------------------------------------------------
# Cross-checks: Algorithm 1, Definition 2, Theorems 2 and 3
# --------------------------------------------------------------------------
def two_pass_threshold(prob: Problem, b: int, k: int, threshold: str = "min") -> float:
    """Algorithm 1's first pass: G = union over p of the top-k items by s_p
    (TopKDotProduct); the threshold is the smallest MoL score over G
    ("min", the algorithm as given) or the k-th largest MoL score over G
    ("kth": G holds k items scoring at least that much, so the corpus-wide
    k-th score is no smaller and the second pass stays exact)."""
    s = all_dots(prob, b)
    G = union_dedup([topk_desc(s[:, p], k)[1] for p in range(prob.P)])
    _, _, phiG = mol_terms(prob, b, G)
    if threshold == "min":
        return float(phiG.min())
    if threshold == "kth":
        return kth_largest(phiG, k)
    raise ValueError(threshold)


def exact_topk_bounded(prob: Problem, b: int, k: int, bound: float
                       ) -> Tuple[np.ndarray, np.ndarray]:
    """Algorithm 1's second pass: G' holds every item whose dot product
    reaches ``bound`` for some component (RangeDotProduct over all p); the
    result is the brute-force MoL top-k over G', padded with (-inf, -1) when
    G' has fewer than k items."""
    s = all_dots(prob, b)
    G2 = np.nonzero((s >= bound).any(axis=1))[0]
    out_s = np.full(k, -np.inf)
    out_i = np.full(k, -1, dtype=np.int64)
    if G2.size:
        _, _, phi2 = mol_terms(prob, b, G2)
        v, i = topk_desc(phi2, k, ids=G2)
        out_s[:len(v)], out_i[:len(i)] = v, i
    return out_s, out_i


def exact_two_pass(prob: Problem, b: int, k: int, threshold: str = "min"
                   ) -> Tuple[np.ndarray, np.ndarray]:
    """Algorithm 1: top-k per component by dot product gives G; S_min is the
    smallest MoL score over G (or, with threshold="kth", the k-th largest);
    G' holds every item whose dot product reaches it for some component;
    brute-force MoL top-k over G'."""
    return exact_topk_bounded(prob, b, k, two_pass_threshold(prob, b, k, threshold))


def max_dot_topk(prob: Problem, b: int, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Max approximation of MoL (a subsection of Section 3 that the published
    text cuts): each item is scored by the largest of its component dot
    products, m = max_p s_p, and the top-k items by m are returned as
    (m values [k], ids [k])."""
    return topk_desc(all_dots(prob, b).max(axis=1), k)


def gap(phi_all: np.ndarray, approx_ids: np.ndarray, k: int) -> float:
    """Definition 2: S_delta = max phi over exact top-k items missing from the
    approximate result minus min phi over the approximate result (-inf when
    nothing is missed)."""
    _, exact_ids = topk_desc(phi_all, k)
    missed = np.setdiff1d(exact_ids, approx_ids)
    if missed.size == 0:
        return -math.inf
    return float(phi_all[missed].max() - phi_all[approx_ids].min())


def gap_bound_per_embd(prob: Problem, b: int, k: int, kprime: int) -> Dict[str, float]:
    """Theorem 2 for TopKPerEmbedding(k'): S = max over p of the (k'+1)-th
    largest s_p; S_K = k-th largest MoL score among the candidates; the gap
    is at most S - S_K.  The looser bound replaces S by the largest k'-th
    retrieved dot product."""
    _, ids, kth, nxt = topk_per_embedding(prob, b, kprime)
    cand = union_dedup([ids])
    _, _, phi = mol_terms(prob, b, cand)
    S_K = kth_largest(phi, k)
    S = float(nxt.max())
    return dict(S=S, S_K=S_K, bound=S - S_K, looser=float(kth.max()) - S_K)


def gap_bound_combined(prob: Problem, b: int, k: int, kprime: int, k_avg: int,
                       avg: Optional[Problem] = None) -> Dict[str, float]:
    """Theorem 3: with X'_K the TopKAvg result, S' = max over p of the largest
    s_p among items outside (X_{k',p} union X'_K); the gap is at most
    S' - S_K, S_K being the k-th largest MoL score among the candidates."""
    s = all_dots(prob, b)
    _, avg_ids = topk_avg(prob, b, k_avg, avg)
    lists = [topk_desc(s[:, p], kprime)[1] for p in range(prob.P)]
    cand = union_dedup(lists + [avg_ids])
    _, _, phi = mol_terms(prob, b, cand)
    S_K = kth_largest(phi, k)
    S_prime = -math.inf
    for p in range(prob.P):
        keep = np.ones(prob.N, dtype=bool)
        keep[lists[p]] = False
        keep[avg_ids] = False
        if keep.any():
            S_prime = max(S_prime, float(s[keep, p].max()))
    return dict(S=S_prime, S_K=S_K, bound=S_prime - S_K)


# --------------------------------------------------------------------------
# Parity helpers
# --------------------------------------------------------------------------
def valid_topk(oracle_scores_all: np.ndarray, got_ids: np.ndarray, k: int,
               tau: float) -> Tuple[bool, str]:
    """tau rule for a returned top-k id set G against exact scores of every
    item: |G| = k, ids distinct, every item scoring >= t + tau is in G and
    every member scores > t - tau, t being the exact k-th score.  When the
    exact k-th to (k+1)-th gap is at least tau this is set equality."""
    got = np.asarray(got_ids, dtype=np.int64)
    if got.shape[0] != k or len(np.unique(got)) != k:
        return False, "size or duplicates"
    if got.min() < 0 or got.max() >= oracle_scores_all.shape[0]:
        return False, "id out of range"
    t = kth_largest(oracle_scores_all, k)
    must = np.nonzero(oracle_scores_all >= t + tau)[0]
    missing = np.setdiff1d(must, got)
    if missing.size:
        return False, f"missing ids {missing[:5].tolist()}"
    low = got[oracle_scores_all[got] <= t - tau]
    if low.size:
        return False, f"ids below threshold {low[:5].tolist()}"
    return True, "ok"
