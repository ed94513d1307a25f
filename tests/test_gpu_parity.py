"""GPU parity: every entry point of the C ABI against the FP64 oracle on the
same seeded inputs (MI355X only)."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import mol_oracle as mo
from paper_2407_15462_amd import mol
from parity_helpers import (TAU, assert_dedup_set, check_scores, check_topk_row, cuda_inputs, log,
                            oracle_problem, recall)

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


def _cases_small():
    # sizes the oracle finishes in seconds, spanning several tiles with a
    # ragged tail
    return [
        ("tiny_exact_f32", W["tiny_exact_f32"]),
        ("exact_32k_ragged", W["exact_32k"].scaled(B=37, N=5003, clusters=64)),
        ("exact_1m_shape_ragged", W["exact_1m"].scaled(B=20, N=4099, clusters=64)),
        ("hybrid_8m_shape_ragged", W["hybrid_8m"].scaled(B=9, N=3001, clusters=64)),
        # bf16 with P_q = 4: served by the generic kernels
        ("bf16_pq4_generic", dataclasses.replace(W["exact_32k"], Pq=4, B=11, N=2100, clusters=16)),
        # the paper's top-K benchmark shapes at 32 queries: d = 32 (fused),
        # d = 128 with P = 8 x 4 (fused), d = 768 with P = 4 x 4 (generic)
        ("paper_books_shape", W["paper_books"].scaled(N=5003, clusters=64)),
        ("paper_ml20m_shape", W["paper_ml20m"].scaled(N=3001, clusters=32)),
        ("paper_nq320k_shape", W["paper_nq320k"].scaled(N=2011, clusters=16)),
    ]


@pytest.mark.parametrize("name,spec", _cases_small(), ids=[c[0] for c in _cases_small()])
def test_score_matches_oracle(name, spec):
    log(f"[score] {name} B={spec.B} N={spec.N} P={spec.P} d={spec.d} H={spec.H} {spec.dtype}")
    inp = cuda_inputs(spec, seed=11)
    prob = mol.Problem.from_inputs(inp)
    phi = mol.score(prob)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want)
    # a sub-range of items
    phi2 = mol.score(prob, n_begin=1001, n_count=777)
    torch.cuda.synchronize()
    check_scores(phi2.cpu().numpy(), want[:, 1001:1778])


@pytest.mark.parametrize("name,spec", _cases_small(), ids=[c[0] for c in _cases_small()])
def test_topk_exact_matches_oracle(name, spec):
    k = min(spec.k, 100)
    log(f"[topk_exact] {name} B={spec.B} N={spec.N} k={k}")
    inp = cuda_inputs(spec, seed=12)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, k)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], k, f"{name} query {b}")


@pytest.mark.parametrize("k", [1, 128, 129, 500])
def test_topk_exact_k_boundaries(k):
    """k = 1 and k = 128 stay on the fused kernel's running lists; k = 129
    and 500 take the pair-wise path (MFMA dots + pair-wise gating kernel)."""
    spec = W["exact_1m"].scaled(B=6, N=4099, clusters=32)
    log(f"[topk_exact] k={k} B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=19)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, k)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], k, f"k_boundary k={k} query {b}")


def test_topk_exact_full_32k_workload():
    spec = W["exact_32k"]
    log(f"[topk_exact] exact_32k full B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=0)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, spec.k)
    torch.cuda.synchronize()
    queries = list(range(0, spec.B, 97))
    want = mo.mol_scores(oracle_problem(inp), queries)
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for r, b in enumerate(queries):
        check_topk_row(want[r], i[b], s[b], spec.k, f"exact_32k query {b}")


def test_topk_exact_k_equals_n_and_single_query():
    spec = W["exact_32k"].scaled(B=1, N=300, clusters=8)
    inp = cuda_inputs(spec, seed=13)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, 300)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), [0])[0]
    check_topk_row(want, i.cpu().numpy()[0], s.cpu().numpy()[0], 300, "k=N")


def test_duplicate_items_tie_to_lower_index():
    spec = W["exact_32k"].scaled(B=3, N=2000, clusters=8)
    inp = cuda_inputs(spec, seed=14)
    # item 1500 becomes an exact copy of item 17 (embeddings and logits)
    inp.X[:, 1500] = inp.X[:, 17]
    inp.a_x[1500] = inp.a_x[17]
    # make them the best item for query 0: copy query 0 from item 17 and give
    # the matching components (px == pq mod Px) a large item gating logit
    inp.Q[0] = inp.X[torch.arange(spec.Pq, device="cuda") % spec.Px, 17]
    for pq in range(spec.Pq):
        inp.a_x[[17, 1500], pq * spec.Px + pq % spec.Px] = 4.0
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, 10)
    phi = mol.score(prob)
    torch.cuda.synchronize()
    row = i.cpu().numpy()[0].tolist()
    assert 17 in row and 1500 in row
    assert row.index(17) + 1 == row.index(1500)
    assert phi[0, 17].item() == phi[0, 1500].item()


@pytest.mark.parametrize("name,spec,kp", [
    ("small_p32", W["exact_32k"].scaled(B=5, N=5003, clusters=32), 128),
    ("small_p64", W["exact_1m"].scaled(B=3, N=4099, clusters=32), 128),
    ("small_d128", W["hybrid_8m"].scaled(B=3, N=3001, clusters=32), 256),
    ("small_p64_k600", W["exact_1m"].scaled(B=2, N=9001, clusters=32), 600),
    ("small_d128_k1024", W["hybrid_8m"].scaled(B=2, N=12003, clusters=32), 1024),
    ("f32", W["tiny_exact_f32"].scaled(B=4, N=2000), 50),
    ("books_d32_k5", W["paper_books"].scaled(B=3, N=9001, clusters=32), 5),
    ("books_d32_k200", W["paper_books"].scaled(B=3, N=9001, clusters=32), 200),
    ("nq_d768_generic", W["paper_nq320k"].scaled(B=3, N=3001, clusters=16), 50),
    # long rows of the generic shapes: sampled threshold, then the kept keys
    ("nq_d768_thresh", W["paper_nq320k"].scaled(B=3, N=20011, clusters=16), 50),
    ("nq_d768_thresh_k1000", W["paper_nq320k"].scaled(B=2, N=16411, clusters=16), 1000),
    ("pq4_d64_thresh", dataclasses.replace(W["exact_32k"], Pq=4, B=4, N=33001, clusters=32), 100),
    # the smallest rows that take the sampled threshold, one query, k' at the limit
    ("nq_d768_thresh_kmax", W["paper_nq320k"].scaled(B=1, N=16384, clusters=16), 8192),
])
def test_topk_per_embd_matches_oracle(name, spec, kp):
    log(f"[per_embd] {name} B={spec.B} N={spec.N} P={spec.P} k'={kp}")
    inp = cuda_inputs(spec, seed=15)
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    for b in range(spec.B):
        s = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s[:, p], ids[b, p], dots[b, p], kp, f"{name} b={b} p={p}")


def test_topk_per_embd_adversarial_order_and_ties():
    """Lists whose best items are contiguous (one block of identical items)
    or all tied (a zero query vector): the bucket-maximum threshold is then
    loose, staging overflows and the merge path runs; ties resolve to the
    lowest item indices."""
    spec = W["exact_1m"].scaled(B=3, N=12000, clusters=32)
    kp = 128
    inp = cuda_inputs(spec, seed=21)
    blk0, blk1 = 2000, 5000
    inp.X[0, blk0:blk1, :] = inp.Q[1, 0, :]          # list (b=1, pq=0, px=0): a tied block on top
    inp.Q[2, 3, :] = 0                                # lists (b=2, pq=3, *): every dot is 0
    log(f"[per_embd adversarial] B={spec.B} N={spec.N} k'={kp}")
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    Px = spec.Px
    assert ids[1, 0].tolist() == list(range(blk0, blk0 + kp))
    assert np.all(dots[1, 0] == dots[1, 0, 0])
    for px in range(Px):
        p = 3 * Px + px
        assert ids[2, p].tolist() == list(range(kp)), f"zero query, component {p}"
        assert np.all(dots[2, p] == 0.0)
    op = oracle_problem(inp)
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"adversarial b={b} p={p}")


@pytest.mark.parametrize("name,spec,kp", [
    # more than 256 query vectors: the bucket scan, the per-bucket hot-vector
    # lists and the pruned pass (lists of up to 256 keys)
    ("pruned_p64", W["exact_1m"].scaled(B=40, N=20011, clusters=64), 128),
    ("pruned_p64_k37", W["exact_1m"].scaled(B=36, N=9001, clusters=32), 37),
    ("pruned_d128", W["hybrid_8m"].scaled(B=40, N=40009, clusters=64), 256),
    ("pruned_d32", W["paper_books"].scaled(B=40, N=30011, clusters=32), 100),
])
def test_pruned_per_embd_matches_oracle(name, spec, kp):
    log(f"[per_embd pruned] {name} B={spec.B} N={spec.N} P={spec.P} k'={kp}")
    inp = cuda_inputs(spec, seed=25)
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    for b in range(spec.B):
        s = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s[:, p], ids[b, p], dots[b, p], kp, f"{name} b={b} p={p}")


def test_pruned_per_embd_overflow_and_ties():
    """More than 256 query vectors with a tied block of 3000 identical items
    on top of one list and an all-zero query vector: those lists receive far
    more keys than their buffers hold, the device flag routes every list
    through the threshold scan, and ties resolve to the lowest indices."""
    spec = W["exact_1m"].scaled(B=40, N=24000, clusters=32)
    kp = 128
    inp = cuda_inputs(spec, seed=26)
    blk0, blk1 = 2000, 5000
    inp.X[0, blk0:blk1, :] = inp.Q[1, 0, :]
    inp.Q[2, 3, :] = 0
    log(f"[per_embd pruned overflow] B={spec.B} N={spec.N} k'={kp}")
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    Px = spec.Px
    assert ids[1, 0].tolist() == list(range(blk0, blk0 + kp))
    assert np.all(dots[1, 0] == dots[1, 0, 0])
    for px in range(Px):
        p = 3 * Px + px
        assert ids[2, p].tolist() == list(range(kp)), f"zero query, component {p}"
        assert np.all(dots[2, p] == 0.0)
    op = oracle_problem(inp)
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"pruned overflow b={b} p={p}")


def test_pruned_per_embd_dense_bucket():
    """60 distinct near-copies of one query vector placed in consecutive
    items: two or three buckets then hold about half of that list's top k',
    so its lanes find far more hits in one work item than their LDS slots
    keep and append the rest with one atomic each.  The list's keys (the 60,
    about one per other hot bucket and a few collisions: near 210) stay below
    its buffer's 256, so the pruned result stands (no fallback)."""
    spec = W["exact_1m"].scaled(B=40, N=24000, clusters=32)
    kp = 128
    inp = cuda_inputs(spec, seed=27)
    g = torch.Generator(device="cpu").manual_seed(27)
    n0, n1 = 6000, 6060
    base = inp.Q[1, 0, :].float().cpu()
    noise = torch.randn((n1 - n0, base.numel()), generator=g) * 0.05
    near = base[None, :] + noise
    near = near / near.norm(dim=1, keepdim=True)
    inp.X[0, n0:n1, :] = near.to(inp.X.dtype).to(inp.X.device)
    log(f"[per_embd pruned dense bucket] B={spec.B} N={spec.N} k'={kp}")
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    # list (query 1, component 0) ranks the planted block first
    assert set(range(n0, n1)) <= set(ids[1, 0].tolist())
    op = oracle_problem(inp)
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"pruned dense bucket b={b} p={p}")


def test_thresholded_per_embd_adversarial_order_and_ties():
    """Generic-shape lists (d = 768) long enough for the sampled threshold:
    a tied block on top that lies wholly in tiles the sample skips (every
    8th 128-item tile is sampled), and all-tied lists (a zero query vector).
    The threshold then keeps many keys, and ties resolve to the lowest
    item indices."""
    spec = W["paper_nq320k"].scaled(B=3, N=17000, clusters=16)
    kp = 50
    inp = cuda_inputs(spec, seed=22)
    blk0, blk1 = 128, 1024                            # tiles 1..7: none sampled
    inp.X[0, blk0:blk1, :] = inp.Q[1, 0, :]
    inp.Q[2, 3, :] = 0
    log(f"[per_embd thresholded adversarial] B={spec.B} N={spec.N} k'={kp}")
    prob = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(prob, kp)
    torch.cuda.synchronize()
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    Px = spec.Px
    assert ids[1, 0].tolist() == list(range(blk0, blk0 + kp))
    assert np.all(dots[1, 0] == dots[1, 0, 0])
    for px in range(Px):
        p = 3 * Px + px
        assert ids[2, p].tolist() == list(range(kp)), f"zero query, component {p}"
        assert np.all(dots[2, p] == 0.0)
    op = oracle_problem(inp)
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"thresholded b={b} p={p}")


def test_avg_embed_bit_exact_and_topk_avg():
    spec = W["hybrid_8m"].scaled(B=6, N=5000, clusters=32)
    inp = cuda_inputs(spec, seed=16)
    prob = mol.Problem.from_inputs(inp)
    q, x = mol.avg_embed(prob)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    qbar, xbar = mo.averaged_embeddings(op)
    assert np.array_equal(q.view(torch.int16).cpu().numpy().view(np.uint16), qbar)
    assert np.array_equal(x.view(torch.int16).cpu().numpy().view(np.uint16), xbar)
    avg = mol.averaged_problem(prob, q, x)
    oavg = mo.averaged_problem(op)
    # TopKAvg list sizes up to the k_avg = 1024 of the 8M-item workload
    for kp in (300, 1024):
        dots, ids = mol.topk_per_embd(avg, kp)
        torch.cuda.synchronize()
        for b in range(spec.B):
            s = mo.all_dots(oavg, b)[:, 0]
            check_topk_row(s, ids.cpu().numpy()[b, 0], dots.cpu().numpy()[b, 0], kp, f"avg k'={kp} b={b}")


def test_combined_candidates_rerank():
    """CombTopK: the union of per-component top-k' and TopKAvg top-k_avg ids,
    deduplicated across both sets and reranked with full MoL."""
    spec = W["hybrid_8m"].scaled(B=4, N=6007, clusters=32)
    kp, kavg, k = 32, 200, 100
    inp = cuda_inputs(spec, seed=23)
    prob = mol.Problem.from_inputs(inp)
    _, pe_ids = mol.topk_per_embd(mol.Problem(inp.Q, inp.X), kp)
    q, x = mol.avg_embed(prob)
    _, avg_ids = mol.topk_per_embd(mol.averaged_problem(prob, q, x), kavg)
    cand, cand2 = pe_ids.view(spec.B, -1), avg_ids.view(spec.B, -1)
    rs, ri, nu = mol.rerank(prob, cand, k, cand2=cand2)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    cand_np, cand2_np = cand.cpu().numpy(), cand2.cpu().numpy()
    rs, ri, nu = rs.cpu().numpy(), ri.cpu().numpy(), nu.cpu().numpy()
    for b in range(spec.B):
        uniq = mo.union_dedup([cand_np[b], cand2_np[b]])
        assert nu[b] == len(uniq), f"b={b}: {nu[b]} unique on the GPU, {len(uniq)} in the union"
        _, _, phi = mo.mol_terms(op, b, uniq)
        full = np.full(spec.N, -np.inf)
        full[uniq] = phi
        check_topk_row(full, ri[b], rs[b], k, f"comb b={b}")


def test_gap_certificate_theorem2():
    """Theorem 2: with per-component lists of k'+1 entries, S = the largest
    (k'+1)-th dot product bounds every non-candidate's MoL score, so
    S - S_K bounds the gap (Definition 2) of the reranked top-k."""
    spec = W["exact_1m"].scaled(B=4, N=6007, clusters=16)
    kp, k = 24, 20
    inp = cuda_inputs(spec, seed=29)
    prob = mol.Problem.from_inputs(inp)
    dots, ids = mol.topk_per_embd(mol.Problem(inp.Q, inp.X), kp + 1)
    cand = ids.view(spec.B, -1)
    rs, ri, nu = mol.rerank(prob, cand, k)
    S, SK, bound, looser = mol.gap_bound(dots, rs)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    cand_np, ri = cand.cpu().numpy(), ri.cpu().numpy()
    S, SK, bound, looser = (t.cpu().numpy() for t in (S, SK, bound, looser))
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        S_oracle = max(mo.kth_largest(s_all[:, p], kp + 1) for p in range(spec.P))
        assert abs(S[b] - S_oracle) <= TAU
        uniq = mo.union_dedup([cand_np[b]])
        _, _, phi_c = mo.mol_terms(op, b, uniq)
        assert abs(SK[b] - mo.kth_largest(phi_c, k)) <= TAU
        assert abs(bound[b] - (S[b] - SK[b])) <= 1e-6 and looser[b] >= bound[b] - 1e-6
        phi_all = mo.mol_scores(op, [b])[0]
        outside = np.setdiff1d(np.arange(spec.N), uniq)
        assert phi_all[outside].max() <= S_oracle + 1e-12      # the theorem's premise
        g = mo.gap(phi_all, ri[b], k)
        assert g <= bound[b] + TAU, f"b={b}: gap {g} above the bound {bound[b]}"
        log(f"[gap] b={b} S={S[b]:.5f} S_K={SK[b]:.5f} bound={bound[b]:.5f} gap={g:.5f}")


def test_gap_certificate_theorem3_combined():
    """Theorem 3: S' = the largest s_p over items outside (X_{k',p} U X'_K)
    bounds every non-candidate's MoL score, so S' - S_K bounds the gap of the
    combined heuristic.  S' is checked against a brute force over all items
    with the GPU's own candidate sets."""
    spec = W["hybrid_8m"].scaled(B=4, N=6007, clusters=16)
    kp, kavg, k = 16, 40, 20
    inp = cuda_inputs(spec, seed=30)
    prob = mol.Problem.from_inputs(inp)
    m = kp + kavg + 1
    dots, ids = mol.topk_per_embd(mol.Problem(inp.Q, inp.X), m)
    q, x = mol.avg_embed(prob)
    _, avg_ids = mol.topk_per_embd(mol.averaged_problem(prob, q, x), kavg)
    avg_ids = avg_ids.view(spec.B, kavg)
    cand = ids[:, :, :kp].contiguous().view(spec.B, -1)
    rs, ri, nu = mol.rerank(prob, cand, k, cand2=avg_ids)
    S, SK, bound = mol.gap_bound_combined(dots, ids, kp, avg_ids, rs)
    # with no averaged candidates it is Theorem 2's bound from (k'+1)-th values
    S2, _, _ = mol.gap_bound_combined(dots, ids, kp, None, rs)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    ids_np, avg_np, cand_np = ids.cpu().numpy(), avg_ids.cpu().numpy(), cand.cpu().numpy()
    dots_np, ri = dots.cpu().numpy(), ri.cpu().numpy()
    S, SK, bound, S2 = (t.cpu().numpy() for t in (S, SK, bound, S2))
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        S_want = -np.inf
        for p in range(spec.P):
            keep = np.ones(spec.N, dtype=bool)
            keep[ids_np[b, p, :kp]] = False
            keep[avg_np[b]] = False
            S_want = max(S_want, s_all[keep, p].max())
        assert abs(S[b] - S_want) <= TAU, f"b={b}: S' {S[b]} vs brute force {S_want}"
        assert S2[b] == dots_np[b, :, kp].max()
        uniq = mo.union_dedup([cand_np[b], avg_np[b]])
        _, _, phi_c = mo.mol_terms(op, b, uniq)
        assert abs(SK[b] - mo.kth_largest(phi_c, k)) <= TAU
        phi_all = mo.mol_scores(op, [b])[0]
        outside = np.setdiff1d(np.arange(spec.N), uniq)
        assert phi_all[outside].max() <= S_want + 1e-12      # the theorem's premise
        g = mo.gap(phi_all, ri[b], k)
        assert g <= bound[b] + TAU, f"b={b}: gap {g} above the bound {bound[b]}"
        log(f"[gap3] b={b} S'={S[b]:.5f} S_K={SK[b]:.5f} bound={bound[b]:.5f} gap={g:.5f}")


@pytest.mark.parametrize("C,k", [(700, 100), (64, 100), (4096, 100)])
def test_rerank_matches_oracle(C, k):
    spec = W["exact_1m"].scaled(B=7, N=3000, clusters=32)
    log(f"[rerank] C={C} k={k}")
    inp = cuda_inputs(spec, seed=17)
    prob = mol.Problem.from_inputs(inp)
    g = torch.Generator(device="cuda").manual_seed(5)
    cand = torch.randint(-1, spec.N, (spec.B, C), device="cuda", generator=g, dtype=torch.int32)
    cand[1] = 42                      # every slot the same id
    cand[2, : C // 2] = -1            # half empty
    cand[3, 0] = spec.N + 5           # out of range: treated as empty
    s, i, nu = mol.rerank(prob, cand, k)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    cand_np = cand.cpu().numpy().astype(np.int64)
    cand_np[cand_np >= spec.N] = -1
    s, i, nu = s.cpu().numpy(), i.cpu().numpy(), nu.cpu().numpy()
    for b in range(spec.B):
        uniq = mo.union_dedup([cand_np[b]])
        assert nu[b] == len(uniq), f"n_unique query {b}: {nu[b]} vs {len(uniq)}"
        _, _, phi = mo.mol_terms(op, b, uniq)
        kk = min(k, len(uniq))
        full = np.full(spec.N, -np.inf)
        full[uniq] = phi
        check_topk_row(full, i[b, :kk], s[b, :kk], kk, f"rerank query {b}")
        assert np.all(i[b, kk:] == -1) and np.all(np.isneginf(s[b, kk:]))


@pytest.mark.parametrize("C,C2,N", [(700, 0, 3000), (4096, 0, 3000), (1000, 300, 3000),
                                     (900, 0, 700), (1500, 200, 1025)])
def test_dedup_union_is_exact_set(C, C2, N):
    """Algorithm 2's deduplicated set G, checked as a set: mol_rerank with
    k = C + C2 returns every distinct candidate of a query (the rest padded),
    so the id set must equal the union computed by the oracle, integer for
    integer -- a dedup that dropped one id and kept another twice, or emitted
    a wrong id, fails here even where counts and the top-k agree.  The dedup
    writes ids bin by bin (1024 bins of consecutive ids): N = 700 puts one id
    in a bin, N = 1025 two per bin but one in the last."""
    spec = W["exact_1m"].scaled(B=7, N=N, clusters=32)
    k = C + C2
    log(f"[dedup set] C={C} C2={C2} N={N} k={k}")
    inp = cuda_inputs(spec, seed=27)
    prob = mol.Problem.from_inputs(inp)
    g = torch.Generator(device="cuda").manual_seed(9)
    cand = torch.randint(-1, spec.N, (spec.B, C), device="cuda", generator=g, dtype=torch.int32)
    cand[1] = 42                      # every slot the same id
    cand[2, : C // 2] = -1            # half empty
    cand[3, 0] = spec.N + 5           # out of range: treated as empty
    cand[4, C // 3:] = cand[4, : C - C // 3].clone()   # long runs of repeats
    cand2 = None
    if C2:
        cand2 = torch.randint(-1, spec.N, (spec.B, C2), device="cuda", generator=g, dtype=torch.int32)
        cand2[5] = cand[5, :C2]       # the second set repeats the first
        cand2[6] = -1                 # the second set empty
    s, i, nu = mol.rerank(prob, cand, k, cand2=cand2)
    torch.cuda.synchronize()
    cand_np = cand.cpu().numpy().astype(np.int64)
    cand_np[cand_np >= spec.N] = -1
    sets = [cand_np]
    if C2:
        c2 = cand2.cpu().numpy().astype(np.int64)
        c2[c2 >= spec.N] = -1
        sets.append(c2)
    i, nu = i.cpu().numpy(), nu.cpu().numpy()
    for b in range(spec.B):
        want = mo.union_dedup([c[b] for c in sets])
        assert_dedup_set(i[b], int(nu[b]), want, f"dedup C={C} C2={C2} query {b}")


@pytest.mark.parametrize("name,spec,C", [
    ("books_d32", W["paper_books"].scaled(B=5, N=4001, clusters=32), 1000),
    ("nq_d768_generic", W["paper_nq320k"].scaled(B=5, N=2003, clusters=16), 600),
])
def test_rerank_paper_shapes(name, spec, C):
    k = spec.k
    log(f"[rerank] {name} C={C} k={k}")
    inp = cuda_inputs(spec, seed=18)
    prob = mol.Problem.from_inputs(inp)
    g = torch.Generator(device="cuda").manual_seed(6)
    cand = torch.randint(0, spec.N, (spec.B, C), device="cuda", generator=g, dtype=torch.int32)
    s, i, nu = mol.rerank(prob, cand, k)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    cand_np = cand.cpu().numpy()
    s, i, nu = s.cpu().numpy(), i.cpu().numpy(), nu.cpu().numpy()
    for b in range(spec.B):
        uniq = mo.union_dedup([cand_np[b]])
        assert nu[b] == len(uniq)
        _, _, phi = mo.mol_terms(op, b, uniq)
        full = np.full(spec.N, -np.inf)
        full[uniq] = phi
        check_topk_row(full, i[b], s[b], k, f"rerank_{name} query {b}")


def test_radix_selection_long_rows_large_k_and_ties():
    """Rows longer than the segmented sorts take (70,001 items of a d = 768
    problem with one all-zero query vector: every key of its lists ties on
    the score), and k above 1024 (TopKAvg, exact MoL top-k) go through the
    radix selection."""
    spec = W["paper_nq320k"].scaled(B=2, N=70001, clusters=64)
    inp = cuda_inputs(spec, seed=41)
    inp.Q[1, 2, :] = 0
    log(f"[radix] per-component k'=300 B={spec.B} N={spec.N} d={spec.d}")
    pe = mol.Problem(inp.Q, inp.X)
    dots, ids = mol.topk_per_embd(pe, 300)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], 300, f"radix b={b} p={p}")
    for px in range(spec.Px):
        assert ids[1, 2 * spec.Px + px].tolist() == list(range(300))
    # TopKAvg with k' = 3000 on a d = 32 problem (generic MFMA dots + radix)
    spec2 = W["paper_books"].scaled(B=4, N=20011, clusters=64)
    inp2 = cuda_inputs(spec2, seed=42)
    prob2 = mol.Problem.from_inputs(inp2)
    q, x = mol.avg_embed(prob2)
    d2, i2 = mol.topk_per_embd(mol.averaged_problem(prob2, q, x), 3000)
    # exact MoL top-k with k = 1500 (the pair-wise path)
    s3, i3 = mol.topk_exact(prob2, 1500)
    torch.cuda.synchronize()
    op2 = oracle_problem(inp2)
    oavg = mo.averaged_problem(op2)
    phi = mo.mol_scores(op2, list(range(spec2.B)))
    d2, i2, s3, i3 = d2.cpu().numpy(), i2.cpu().numpy(), s3.cpu().numpy(), i3.cpu().numpy()
    for b in range(spec2.B):
        s = mo.all_dots(oavg, b)[:, 0]
        check_topk_row(s, i2[b, 0], d2[b, 0], 3000, f"radix_avg b={b}")
        check_topk_row(phi[b], i3[b], s3[b], 1500, f"radix_exact b={b}")


def test_radix_chunked_first_pass_few_long_rows():
    """Few rows of more than 32K keys (k <= 1024) are first reduced per
    16K-key chunk by separate workgroups, then per row: exact MoL top-k and
    max-component top-k on a d = 768 shape with 40,001 items, and the
    streamed per-component lists of a float32 problem, one list all-tied."""
    spec = W["paper_nq320k"].scaled(B=3, N=40001, clusters=16)
    inp = cuda_inputs(spec, seed=43)
    log(f"[radix chunks] B={spec.B} N={spec.N} d={spec.d}")
    prob = mol.Problem.from_inputs(inp)
    s1, i1 = mol.topk_exact(prob, 100)
    s2, i2 = mol.topk_exact(prob, 1000)
    ms, mi = mol.topk_maxdot(mol.Problem(inp.Q, inp.X), 1000)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    phi = mo.mol_scores(op, list(range(spec.B)))
    for b in range(spec.B):
        check_topk_row(phi[b], i1[b].cpu().numpy(), s1[b].cpu().numpy(), 100, f"radix_chunks k=100 b={b}")
        check_topk_row(phi[b], i2[b].cpu().numpy(), s2[b].cpu().numpy(), 1000, f"radix_chunks k=1000 b={b}")
        m = mo.all_dots(op, b).max(axis=1)
        check_topk_row(m, mi[b].cpu().numpy(), ms[b].cpu().numpy(), 1000, f"radix_chunks maxdot b={b}")
    spec2 = W["tiny_exact_f32"].scaled(B=2, N=40000)
    inp2 = cuda_inputs(spec2, seed=44)
    inp2.Q[1, 0, :] = 0
    dots, ids = mol.topk_per_embd(mol.Problem(inp2.Q, inp2.X), 50)
    torch.cuda.synchronize()
    op2 = oracle_problem(inp2)
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    for b in range(spec2.B):
        s_all = mo.all_dots(op2, b)
        for p in range(spec2.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], 50, f"radix_chunks f32 b={b} p={p}")
    for px in range(spec2.Px):
        assert ids[1, px].tolist() == list(range(50))


def test_f32_gating_on_skewed_weights_matches_oracle():
    """Gating weights of standard deviation 0.5 (the skewed workload, whose
    largest gating weight per pair averages 0.23) lie outside the fused
    f16-operand chain's range; with MOL_FLAG_F32_GATING the gating MLP,
    softmax and phi run in float32 and mol_score, the exact top-k and the
    rerank meet the 1e-4 bar."""
    spec = W["exact_1m_skewed"].scaled(B=12, N=4099, clusters=64)
    log(f"[f32 gating] skewed B={spec.B} N={spec.N} std={spec.gating_std}")
    inp = cuda_inputs(spec, seed=28)
    prob = mol.Problem.from_inputs(inp, flags=mol.MOL_FLAG_F32_GATING)
    phi = mol.score(prob)
    s, i = mol.topk_exact(prob, 100)
    g = torch.Generator(device="cuda").manual_seed(7)
    cand = torch.randint(-1, spec.N, (spec.B, 700), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, nu = mol.rerank(prob, cand, 100)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    want = mo.mol_scores(op, list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want, what="f32_gating phi")
    s, i = s.cpu().numpy(), i.cpu().numpy()
    rs, ri, nu = rs.cpu().numpy(), ri.cpu().numpy(), nu.cpu().numpy()
    cand_np = cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], 100, f"f32_gating exact query {b}")
        uniq = mo.union_dedup([cand_np[b]])
        full = np.full(spec.N, -np.inf)
        full[uniq] = want[b][uniq]
        check_topk_row(full, ri[b], rs[b], 100, f"f32_gating rerank query {b}")


@pytest.mark.parametrize("wl,std", [("exact_1m", 0.5), ("exact_1m", 1.0), ("exact_32k", 1.0), ("hybrid_8m", 1.0),
                                    ("paper_books", 1.0)])
def test_bf16x2_gating_matches_oracle(wl, std):
    """MOL_FLAG_BF16X2_GATING: every fused shape (P = 8 x 8 at d = 64 and 32,
    8 x 4 at d = 64 and 128) with gating weights of standard deviation 1,
    the top of the two-term chain's stated range and far outside the f16
    chain's, and 0.5 (the skewed workload): mol_score, the exact top-k, the
    bounded pass at the k-th score, Algorithm 1's two passes, the
    allocation-free exact top-k and the rerank meet the 1e-4 bar."""
    spec = dataclasses.replace(W[wl].scaled(B=12, N=4099, clusters=64), gating_std=std)
    log(f"[bf16x2 gating] {wl} std={std} B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=31)
    prob = mol.Problem.from_inputs(inp, flags=mol.MOL_FLAG_BF16X2_GATING)
    phi = mol.score(prob)
    s, i = mol.topk_exact(prob, 100)
    bs, bi = mol.topk_exact_bounded(prob, 100, s[:, 99].contiguous())
    ts, ti, _ = mol.topk_two_pass(prob, 100, mol.MOL_TWO_PASS_KTH)
    ns, ni = torch.empty_like(s), torch.empty_like(i)
    mol.mol_topk_exact_noalloc(prob, 100, ns, ni)
    g = torch.Generator(device="cuda").manual_seed(8)
    cand = torch.randint(-1, spec.N, (spec.B, 700), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, nu = mol.rerank(prob, cand, 100)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want, what=f"bf16x2_{wl}_{std} phi")
    s, i, bs, bi = s.cpu().numpy(), i.cpu().numpy(), bs.cpu().numpy(), bi.cpu().numpy()
    ts, ti, ns, ni = ts.cpu().numpy(), ti.cpu().numpy(), ns.cpu().numpy(), ni.cpu().numpy()
    rs, ri = rs.cpu().numpy(), ri.cpu().numpy()
    cand_np = cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], 100, f"bf16x2_{wl}_{std} exact query {b}")
        check_topk_row(want[b], bi[b], bs[b], 100, f"bf16x2_{wl}_{std} bounded query {b}")
        check_topk_row(want[b], ti[b], ts[b], 100, f"bf16x2_{wl}_{std} two-pass query {b}")
        check_topk_row(want[b], ni[b], ns[b], 100, f"bf16x2_{wl}_{std} no-alloc query {b}")
        uniq = mo.union_dedup([cand_np[b]])
        full = np.full(spec.N, -np.inf)
        full[uniq] = want[b][uniq]
        check_topk_row(full, ri[b], rs[b], 100, f"bf16x2_{wl}_{std} rerank query {b}")


def test_fused_gating_at_the_edge_of_its_range():
    """The fused chain at the edge of its stated range (gating entries of
    standard deviation 0.3) still meets the 1e-4 bar for scores and top-k."""
    spec = dataclasses.replace(W["exact_1m"].scaled(B=12, N=4099, clusters=64), gating_std=0.3)
    log(f"[fused gating] std={spec.gating_std} B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=29)
    prob = mol.Problem.from_inputs(inp)
    phi = mol.score(prob)
    s, i = mol.topk_exact(prob, 100)
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want, what="fused_std0.3 phi")
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], 100, f"fused_std0.3 exact query {b}")


def test_worked_example_through_the_abi():
    """Appendix B's example run through the library: exact top-2 {a, d},
    TopKPerEmbedding(2) candidates {a, b, c}, rerank of those -> {a, b}."""
    from test_oracle_pins import worked_example_problem
    op, names, rows, expect = worked_example_problem()
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    prob = mol.Problem(t(op.Qraw), t(op.X), t(op.a_q.astype(np.float32)), t(op.a_x),
                       t(op.W1.astype(np.float32)), t(op.b1.astype(np.float32)),
                       t(op.W2.astype(np.float32)), t(op.b2.astype(np.float32)))
    s, i = mol.topk_exact(prob, 2)
    dots, ids = mol.topk_per_embd(mol.Problem(prob.tensors[0], prob.tensors[1]), 2)
    cand = ids.reshape(1, -1).contiguous()
    rs, ri, nu = mol.rerank(prob, cand, 2)
    torch.cuda.synchronize()
    assert [names[j] for j in i.cpu().numpy()[0]] == expect["exact top-2"]
    got_cand = sorted(set(ids.cpu().numpy().ravel().tolist()))
    assert [names[j] for j in got_cand] == expect["TopKPerEmbedding(K'=2) candidates"]
    assert nu.item() == 3
    assert [names[j] for j in ri.cpu().numpy()[0]] == ["a", "b"]
    assert abs(rs[0, 1].item() - float(expect["Theorem 2 S_K"][0])) < 1e-6


@pytest.mark.parametrize("name,spec", [
    ("p64_h64", W["exact_1m"].scaled(B=6, N=1200, clusters=16)),       # two-query pipelined chain
    ("p32_h64", W["exact_32k"].scaled(B=6, N=1200, clusters=16)),      # pipelined chain, P_x = 4
    ("p32_h128_d128", W["hybrid_8m"].scaled(B=6, N=1200, clusters=16)),  # two-query chain, H = 128
], ids=lambda v: v if isinstance(v, str) else "")
def test_softmax_redo_far_logits(name, spec):
    """Reading R13: the softmax sums skip the max subtraction only while they
    stay inside [2^-60, 2^60]; items whose base-2 logits all sit near +-72 or
    +-144 (past the float32 range), items with one dominant logit, and whole
    queries shifted by +-45 take the redo with the row maximum subtracted.  Queries 0 and 1 share a wave, so
    one query redoes while the other does not."""
    log(f"[softmax redo] {name} B={spec.B} N={spec.N} P={spec.P} H={spec.H}")
    inp = cuda_inputs(spec, seed=71)
    P = spec.P
    # 2^(log2(e) 100) overflows float32 and 2^(-log2(e) 100) underflows it:
    # without the redo those rows would give inf / inf or 0 / 0
    inp.a_x[0:48] = 50.0
    inp.a_x[48:96] = 100.0
    inp.a_x[96:144] = -50.0
    inp.a_x[144:192] = -100.0
    rows = torch.arange(192, 288, device="cuda")
    inp.a_x[rows, rows % P] = 60.0
    inp.a_q[1] = 45.0
    inp.a_q[4] = -45.0
    prob = mol.Problem.from_inputs(inp)
    k = 50
    phi = mol.score(prob)
    s, i = mol.topk_exact(prob, k)
    bs, bi = mol.topk_exact_bounded(prob, k, s[:, k - 1].contiguous())
    g = torch.Generator(device="cuda").manual_seed(5)
    cand = torch.randint(0, spec.N, (spec.B, 400), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, rn = mol.rerank(prob, cand, k)
    torch.cuda.synchronize()
    assert torch.equal(bi, i) and torch.equal(bs, s), f"{name}: bounded pass differs from brute force"
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want, what="redo_phi")
    s, i, rs, ri, cand = s.cpu().numpy(), i.cpu().numpy(), rs.cpu().numpy(), ri.cpu().numpy(), cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], k, f"redo {name} query {b}")
        uniq = mo.union_dedup([cand[b]])
        full = np.full(spec.N, -np.inf)
        full[uniq] = want[b][uniq]
        check_topk_row(full, ri[b], rs[b], k, f"redo_rerank {name} query {b}")
