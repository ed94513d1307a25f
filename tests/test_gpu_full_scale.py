"""Parity at full workload size, in the launch configuration bench.py times
(1024 queries x 1,048,576 items, P = 8 x 8, d = 64, H = 64, bf16): every
entry point runs on the whole problem, and sampled outputs are checked
against the FP64 oracle one query at a time."""
import numpy as np
import pytest
import torch

import synth
from oracle import mol_oracle as mo
from paper_2407_15462_amd import mol
from parity_helpers import check_topk_row, log, recall

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
