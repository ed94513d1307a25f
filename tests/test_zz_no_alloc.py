"""The allocation-free exact top-k (mol_topk_exact_noalloc) against
mol_topk_exact with a caller workspace, through the C ABI (MI355X only).

Two calls in a row, the second on a smaller problem, so that the second
reads scratch the first left behind; each must equal the workspace entry
point's output bit for bit (same kernels, same order of work)."""
import ctypes

import numpy as np
import pytest
import torch

import synth
from oracle import mol_oracle as mo
from paper_2407_15462_amd import mol
from parity_helpers import check_topk_row, cuda_inputs, log, oracle_problem

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


def _noalloc(prob, k):
    s = torch.full((prob.B, k), 7.0, dtype=torch.float32, device=prob.device)
    i = torch.full((prob.B, k), -7, dtype=torch.int32, device=prob.device)
    mol.mol_topk_exact_noalloc(prob, k, s, i)
    return s, i


def test_noalloc_equals_workspace_entry_point_twice_shrinking():
    cases = [
        ("exact_1m_shape", W["exact_1m"].scaled(B=40, N=9001, clusters=64), 100),
        ("hybrid_8m_shape", W["hybrid_8m"].scaled(B=9, N=3001, clusters=32), 50),
    ]
    for name, spec, k in cases:
        log(f"[noalloc] {name} B={spec.B} N={spec.N} k={k}")
        inp = cuda_inputs(spec, seed=31)
        prob = mol.Problem.from_inputs(inp)
        ws_s, ws_i = mol.topk_exact(prob, k)
        na_s, na_i = _noalloc(prob, k)
        torch.cuda.synchronize()
        assert torch.equal(na_i, ws_i), f"{name}: ids differ from mol_topk_exact"
        assert torch.equal(na_s, ws_s), f"{name}: scores differ from mol_topk_exact"
        want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
        s, i = na_s.cpu().numpy(), na_i.cpu().numpy()
        for b in range(spec.B):
            check_topk_row(want[b], i[b], s[b], k, f"noalloc {name} query {b}")


def test_noalloc_full_size_then_small():
    """The bench configuration (1024 queries x 2^20 items, P = 8 x 8), then a
    small problem: the scratch holds the large call's partial lists when the
    small one starts."""
    spec = W["exact_1m"]
    log(f"[noalloc] full size B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=0)
    prob = mol.Problem.from_inputs(inp)
    ws_s, ws_i = mol.topk_exact(prob, spec.k)
    na_s, na_i = _noalloc(prob, spec.k)
    torch.cuda.synchronize()
    assert torch.equal(na_i, ws_i) and torch.equal(na_s, ws_s)
    del inp, prob, ws_s, ws_i, na_s, na_i
    small = W["exact_1m"].scaled(B=3, N=2000, clusters=16)
    log(f"[noalloc] then B={small.B} N={small.N}")
    inp = cuda_inputs(small, seed=32)
    prob = mol.Problem.from_inputs(inp)
    ws_s, ws_i = mol.topk_exact(prob, 10)
    na_s, na_i = _noalloc(prob, 10)
    torch.cuda.synchronize()
    assert torch.equal(na_i, ws_i) and torch.equal(na_s, ws_s)
    want = mo.mol_scores(oracle_problem(inp), list(range(small.B)))
    s, i = na_s.cpu().numpy(), na_i.cpu().numpy()
    for b in range(small.B):
        check_topk_row(want[b], i[b], s[b], 10, f"noalloc small query {b}")


def test_noalloc_rejects_problems_beyond_the_scratch():
    """A shape whose workspace exceeds the library's scratch is refused on the
    host with MOL_EWORKSPACE and launches nothing (outputs untouched)."""
    spec = W["exact_1m"].scaled(B=16, N=20000, clusters=16)
    inp = cuda_inputs(spec, seed=33)
    prob = mol.Problem.from_inputs(inp)
    k = 500                                  # beyond the fused lists: the tiled generic path
    need = mol.mol_workspace_size(prob, mol.MOL_OP_TOPK_EXACT, k=k)
    lib = mol.load()
    assert need > 16 << 20
    s = torch.full((spec.B, k), 7.0, dtype=torch.float32, device="cuda")
    i = torch.full((spec.B, k), -7, dtype=torch.int32, device="cuda")
    rc = lib.mol_topk_exact_noalloc(prob.ref, k, s.data_ptr(), i.data_ptr(), None)
    torch.cuda.synchronize()
    assert rc == mol.MOL_EWORKSPACE and b"scratch" in lib.mol_last_error()
    assert bool((s == 7.0).all()) and bool((i == -7).all())
