"""Parity at full workload sizes: every entry point runs on the whole problem
and sampled outputs are checked against the FP64 oracle one query at a time.

* 1024 queries x 1,048,576 items, P = 8 x 8, d = 64, H = 64 (the launch
  configuration bench.py times): exact top-100; per-component top-128 and
  rerank.
* 256 queries x 8,388,608 items, P = 8 x 4, d = 128, H = 128: exact top-100;
  per-component top-256, TopKAvg top-1024 and the MoL rerank of their union.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import mol_oracle as mo
from paper_2407_15462_amd import mol
from parity_helpers import assert_dedup_set, check_topk_row, log, recall

pytestmark = pytest.mark.gpu

SAMPLE = [0, 517, 1023]


@pytest.fixture(scope="module")
def full():
    spec = synth.WORKLOADS["exact_1m"]
    log(f"[full] generating {spec.name} B={spec.B} N={spec.N}")
    inp = synth.generate(spec, seed=0, device="cuda")
    prob = mol.Problem.from_inputs(inp)
    arrays = synth.to_numpy(inp, queries=SAMPLE)
    op = mo.Problem.from_arrays(arrays)
    return spec, inp, prob, op


def test_exact_top100_full_scale(full):
    spec, inp, prob, op = full
    s, i = mol.topk_exact(prob, spec.k)
    torch.cuda.synchronize()
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for r, b in enumerate(SAMPLE):
        log(f"[full] exact query {b}")
        phi = mo.mol_scores(op, [r])[0]
        check_topk_row(phi, i[b], s[b], spec.k, f"exact_1m query {b}")


def test_two_pass_and_maxdot_full_scale(full):
    """Algorithm 1 (k-th-score threshold) returns the brute-force rows bit for
    bit for every query; the max-component top-k of sampled queries against
    the oracle."""
    spec, inp, prob, op = full
    es, ei = mol.topk_exact(prob, spec.k)
    s, i, bound = mol.topk_two_pass(prob, spec.k, mol.MOL_TWO_PASS_KTH)
    ms, mi = mol.topk_maxdot(mol.Problem(inp.Q, inp.X), spec.k)
    torch.cuda.synchronize()
    assert torch.equal(i, ei) and torch.equal(s, es)
    log(f"[full] two-pass bound {bound.min().item():.4f} .. {bound.max().item():.4f}")
    ms, mi = ms.cpu().numpy(), mi.cpu().numpy()
    for r, b in enumerate(SAMPLE):
        log(f"[full] max-dot query {b}")
        m = mo.all_dots(op, r).max(axis=1)
        check_topk_row(m, mi[b], ms[b], spec.k, f"maxdot_1m query {b}")


def test_per_embd_and_rerank_full_scale(full):
    spec, inp, prob, op = full
    kp = spec.kprime
    dots, ids = mol.topk_per_embd(mol.Problem(inp.Q, inp.X), kp)
    C = spec.P * kp
    cand = ids.view(spec.B, C)
    rs, ri, nu = mol.rerank(prob, cand, spec.k)
    es, ei = mol.topk_exact(prob, spec.k)
    torch.cuda.synchronize()
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    rs, ri, nu = rs.cpu().numpy(), ri.cpu().numpy(), nu.cpu().numpy()
    cand_np = cand.cpu().numpy()
    for r, b in enumerate(SAMPLE):
        log(f"[full] per-component top-{kp} and rerank, query {b}")
        s_all = mo.all_dots(op, r)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"per_embd b={b} p={p}")
        uniq = mo.union_dedup([cand_np[b]])
        assert nu[b] == len(uniq)
        _, _, phi = mo.mol_terms(op, r, uniq)
        full_phi = np.full(spec.N, -np.inf)
        full_phi[uniq] = phi
        check_topk_row(full_phi, ri[b], rs[b], spec.k, f"rerank b={b}")
    rec = recall(ri, ei.cpu().numpy())
    log(f"[full] approx recall@100 vs exact (all {spec.B} queries): {rec:.4f}; "
        f"candidates/query mean {nu.mean():.0f}")
    assert 0.0 < rec <= 1.0
    # the deduplicated union of the sampled queries' full-size candidate rows
    # as an exact set: a rerank with k = C returns all of it
    sub = mol.Problem(inp.Q[SAMPLE].contiguous(), inp.X, inp.a_q[SAMPLE].contiguous(), inp.a_x,
                      inp.W1, inp.b1, inp.W2, inp.b2)
    _, si, snu = mol.rerank(sub, cand[SAMPLE].contiguous(), C)
    torch.cuda.synchronize()
    si, snu = si.cpu().numpy(), snu.cpu().numpy()
    for r, b in enumerate(SAMPLE):
        log(f"[full] deduplicated union of query {b} as a set")
        assert_dedup_set(si[r], int(snu[r]), mo.union_dedup([cand_np[b]]), f"dedup_1m query {b}")


# ---------------------------------------------------------------- 8M items
SAMPLE8 = [0, 255]


@pytest.fixture(scope="module")
def full8m():
    spec = synth.WORKLOADS["hybrid_8m"]
    log(f"[full8m] generating {spec.name} B={spec.B} N={spec.N}")
    inp = synth.generate(spec, seed=0, device="cuda")
    prob = mol.Problem.from_inputs(inp)
    arrays = synth.to_numpy(inp, queries=SAMPLE8)
    op = mo.Problem.from_arrays(arrays)
    return spec, inp, prob, op


def test_exact_top100_8m_items(full8m):
    spec, inp, prob, op = full8m
    s, i = mol.topk_exact(prob, spec.k)
    torch.cuda.synchronize()
    s, i = s.cpu().numpy(), i.cpu().numpy()
    for r, b in enumerate(SAMPLE8):
        log(f"[full8m] exact query {b}")
        phi = mo.mol_scores(op, [r])[0]
        check_topk_row(phi, i[b], s[b], spec.k, f"hybrid_8m query {b}")


def test_hybrid_candidates_and_rerank_8m_items(full8m):
    spec, inp, prob, op = full8m
    kp, kavg = spec.kprime, spec.k_avg
    pe = mol.Problem(inp.Q, inp.X)
    pe_d, pe_i = mol.topk_per_embd(pe, kp)
    q, x = mol.avg_embed(prob)
    avg = mol.averaged_problem(prob, q, x)
    av_d, av_i = mol.topk_per_embd(avg, kavg)
    cand, cand2 = pe_i.view(spec.B, -1), av_i.view(spec.B, -1)
    rs, ri, nu = mol.rerank(prob, cand, spec.k, cand2=cand2)
    es, ei = mol.topk_exact(prob, spec.k)
    torch.cuda.synchronize()
    log("[full8m] averaged embeddings, bit-exact")
    qbar, xbar = mo.averaged_embeddings(op)
    assert np.array_equal(x.view(torch.int16).cpu().numpy().view(np.uint16), xbar)
    assert np.array_equal(q.view(torch.int16).cpu().numpy().view(np.uint16)[SAMPLE8], qbar)
    oavg = mo.averaged_problem(op)
    pe_d, pe_i, av_d, av_i = pe_d.cpu().numpy(), pe_i.cpu().numpy(), av_d.cpu().numpy(), av_i.cpu().numpy()
    cand_np, cand2_np = cand.cpu().numpy(), cand2.cpu().numpy()
    rs, ri, nu = rs.cpu().numpy(), ri.cpu().numpy(), nu.cpu().numpy()
    for r, b in enumerate(SAMPLE8):
        log(f"[full8m] per-component top-{kp}, TopKAvg top-{kavg}, rerank: query {b}")
        s_all = mo.all_dots(op, r)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], pe_i[b, p], pe_d[b, p], kp, f"per_embd b={b} p={p}")
        del s_all
        s_avg = mo.all_dots(oavg, r)[:, 0]
        check_topk_row(s_avg, av_i[b, 0], av_d[b, 0], kavg, f"topk_avg b={b}")
        uniq = mo.union_dedup([cand_np[b], cand2_np[b]])
        assert nu[b] == len(uniq)
        _, _, phi = mo.mol_terms(op, r, uniq)
        full_phi = np.full(spec.N, -np.inf)
        full_phi[uniq] = phi
        check_topk_row(full_phi, ri[b], rs[b], spec.k, f"rerank b={b}")
    rec = recall(ri, ei.cpu().numpy())
    log(f"[full8m] approx recall@100 vs exact (all {spec.B} queries): {rec:.4f}; "
        f"candidates/query mean {nu.mean():.0f}")
    assert 0.0 < rec <= 1.0
