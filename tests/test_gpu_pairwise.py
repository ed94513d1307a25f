"""GPU parity of the pair-wise path (MFMA dot products into a buffer, then
the gating MLP on matrix cores, zero-padded to 16, 32 or 64 components and
32, 64 or 128 hidden units) on shapes the fused kernels do not take: brute-force
top-k, rerank of candidate lists, the max-component top-k and the bounded
second pass of Algorithm 1, against the FP64 oracle (MI355X only)."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import mol_oracle as mo
from paper_2407_15462_amd import mol
from parity_helpers import check_scores, check_topk_row, cuda_inputs, log, oracle_problem

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["exact_32k"]
# (name, Pq, Px, d, H, side logits): every padded instantiation, ragged P
# and H, d not a multiple of 64, and one H above the MFMA kernel's limit
# (one thread per pair)
SHAPES = [
    ("p12_h32_d64", 3, 4, 64, 32, True),
    ("p8_h128_d64", 2, 4, 64, 128, False),
    ("p16_h48_d96", 4, 4, 96, 48, True),
    ("p32_h64_d64", 4, 8, 64, 64, False),
    ("p24_h100_d128", 2, 12, 128, 100, True),
    ("p32_h128_d64", 2, 16, 64, 128, True),
    ("p48_h64_d64", 6, 8, 64, 64, True),
    ("p64_h32_d32", 4, 16, 32, 32, True),
    ("p64_h128_d64", 8, 8, 64, 128, True),   # P_q = 8 but (P_x, d, H) unfused
    ("p16_h160_d64", 4, 4, 64, 160, True),
]
# (name, B): enough queries for 128-vector tiles of the dots GEMM, with a
# ragged last tile
MANY = [("b40_pq4", 40), ("b33_pq4", 33)]


def _spec(Pq, Px, d, H, side):
    return dataclasses.replace(BASE, name="pairwise", B=6, N=1531, Pq=Pq, Px=Px, d=d, H=H, clusters=16,
                               side_logits=side)


@pytest.mark.parametrize("name,Pq,Px,d,H,side", SHAPES, ids=[s[0] for s in SHAPES])
def test_pairwise_shapes(name, Pq, Px, d, H, side):
    spec = _spec(Pq, Px, d, H, side)
    k = 50
    log(f"[pairwise] {name} B={spec.B} N={spec.N} P={spec.P} d={d} H={H}")
    inp = cuda_inputs(spec, seed=61)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, k)
    g = torch.Generator(device="cuda").manual_seed(9)
    cand = torch.randint(0, spec.N, (spec.B, 333), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, rn = mol.rerank(prob, cand, k)
    ms, mi = mol.topk_maxdot(mol.Problem(inp.Q, inp.X), k)
    bs, bi = mol.topk_exact_bounded(prob, k, s[:, k - 1].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(bi, i) and torch.equal(bs, s), f"{name}: bounded pass differs from brute force"
    op = oracle_problem(inp)
    phi = mo.mol_scores(op, list(range(spec.B)))
    s, i = s.cpu().numpy(), i.cpu().numpy()
    rs, ri, rn = rs.cpu().numpy(), ri.cpu().numpy(), rn.cpu().numpy()
    ms, mi = ms.cpu().numpy(), mi.cpu().numpy()
    cand = cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(phi[b], i[b], s[b], k, f"pairwise {name} query {b}")
        uniq = mo.union_dedup([cand[b]])
        assert rn[b] == len(uniq)
        full = np.full(spec.N, -np.inf)
        full[uniq] = phi[b][uniq]
        check_topk_row(full, ri[b], rs[b], k, f"pairwise_rerank {name} query {b}")
        m = mo.all_dots(op, b).max(axis=1)
        check_topk_row(m, mi[b], ms[b], k, f"pairwise_maxdot {name} query {b}")


@pytest.mark.parametrize("name,B", MANY, ids=[m[0] for m in MANY])
def test_pairwise_many_queries(name, B):
    """The same checks with 132 to 160 query vectors: the dots GEMM takes
    128-vector tiles (the rerank's per-query tiles stay at 64)."""
    spec = dataclasses.replace(_spec(4, 4, 64, 64, True), B=B, N=2131)
    k = 50
    log(f"[pairwise many] {name} B={spec.B} N={spec.N} P={spec.P}")
    inp = cuda_inputs(spec, seed=62)
    prob = mol.Problem.from_inputs(inp)
    s, i = mol.topk_exact(prob, k)
    g = torch.Generator(device="cuda").manual_seed(10)
    cand = torch.randint(0, spec.N, (spec.B, 200), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, rn = mol.rerank(prob, cand, k)
    ms, mi = mol.topk_maxdot(mol.Problem(inp.Q, inp.X), k)
    bs, bi = mol.topk_exact_bounded(prob, k, s[:, k - 1].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(bi, i) and torch.equal(bs, s), f"{name}: bounded pass differs from brute force"
    op = oracle_problem(inp)
    phi = mo.mol_scores(op, list(range(spec.B)))
    s, i = s.cpu().numpy(), i.cpu().numpy()
    rs, ri = rs.cpu().numpy(), ri.cpu().numpy()
    ms, mi = ms.cpu().numpy(), mi.cpu().numpy()
    cand = cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(phi[b], i[b], s[b], k, f"pairwise {name} query {b}")
        uniq = mo.union_dedup([cand[b]])
        full = np.full(spec.N, -np.inf)
        full[uniq] = phi[b][uniq]
        check_topk_row(full, ri[b], rs[b], k, f"pairwise_rerank {name} query {b}")
        m = mo.all_dots(op, b).max(axis=1)
        check_topk_row(m, mi[b], ms[b], k, f"pairwise_maxdot {name} query {b}")


def test_thresholded_lists_many_queries():
    """Per-component lists through the sampled threshold with 136 query
    vectors (128-vector tiles of the sample and kept-key passes); d = 96 has
    no fused per-component kernel."""
    spec = dataclasses.replace(_spec(4, 4, 96, 64, True), B=34, N=16500)
    kp = 20
    log(f"[thresholded many] B={spec.B} N={spec.N} k'={kp}")
    inp = cuda_inputs(spec, seed=63)
    dots, ids = mol.topk_per_embd(mol.Problem(inp.Q, inp.X), kp)
    torch.cuda.synchronize()
    op = oracle_problem(inp)
    dots, ids = dots.cpu().numpy(), ids.cpu().numpy()
    for b in range(spec.B):
        s_all = mo.all_dots(op, b)
        for p in range(spec.P):
            check_topk_row(s_all[:, p], ids[b, p], dots[b, p], kp, f"thresholded_many b={b} p={p}")


def test_pairwise_softmax_redo_far_logits():
    """Reading R13 on the pair-wise gating kernel (P = 12 and 16 padded to
    16): items and queries whose base-2 logits sit far from zero take the
    redo with the row maximum subtracted."""
    for Pq, Px in ((3, 4), (4, 4)):
        spec = dataclasses.replace(_spec(Pq, Px, 64, 64, True), N=1531)
        P = spec.P
        log(f"[pairwise redo] B={spec.B} N={spec.N} P={P}")
        inp = cuda_inputs(spec, seed=72)
        inp.a_x[0:50] = 50.0
        inp.a_x[50:100] = 100.0        # past the float32 range without the redo
        inp.a_x[100:150] = -50.0
        inp.a_x[150:200] = -100.0
        rows = torch.arange(200, 300, device="cuda")
        inp.a_x[rows, rows % P] = 60.0
        inp.a_q[1] = 45.0
        prob = mol.Problem.from_inputs(inp)
        k = 50
        s, i = mol.topk_exact(prob, k)
        torch.cuda.synchronize()
        op = oracle_problem(inp)
        phi = mo.mol_scores(op, list(range(spec.B)))
        s, i = s.cpu().numpy(), i.cpu().numpy()
        for b in range(spec.B):
            check_topk_row(phi[b], i[b], s[b], k, f"pairwise redo P={P} query {b}")


# the two-term gating chain (MOL_FLAG_BF16X2_GATING) on the pair-wise path:
# both MLP forms (P <= 16 and the padded 16x16x32 one), at gating weights of
# standard deviation 1, the top of the flag's stated range
X2_SHAPES = [s for s in SHAPES if s[0] in ("p12_h32_d64", "p16_h48_d96", "p24_h100_d128", "p48_h64_d64",
                                           "p64_h128_d64")]


@pytest.mark.parametrize("name,Pq,Px,d,H,side", X2_SHAPES, ids=[s[0] for s in X2_SHAPES])
def test_pairwise_bf16x2_gating(name, Pq, Px, d, H, side):
    spec = dataclasses.replace(_spec(Pq, Px, d, H, side), gating_std=1.0)
    k = 50
    log(f"[pairwise bf16x2] {name} B={spec.B} N={spec.N} P={spec.P} d={d} H={H} std={spec.gating_std}")
    inp = cuda_inputs(spec, seed=62)
    prob = mol.Problem.from_inputs(inp, flags=mol.MOL_FLAG_BF16X2_GATING)
    phi = mol.score(prob)
    s, i = mol.topk_exact(prob, k)
    g = torch.Generator(device="cuda").manual_seed(10)
    cand = torch.randint(0, spec.N, (spec.B, 333), device="cuda", generator=g, dtype=torch.int32)
    rs, ri, _ = mol.rerank(prob, cand, k)
    bs, bi = mol.topk_exact_bounded(prob, k, s[:, k - 1].contiguous())
    torch.cuda.synchronize()
    want = mo.mol_scores(oracle_problem(inp), list(range(spec.B)))
    check_scores(phi.cpu().numpy(), want, what=f"pairwise_bf16x2 {name} phi")
    s, i, rs, ri = s.cpu().numpy(), i.cpu().numpy(), rs.cpu().numpy(), ri.cpu().numpy()
    bs, bi, cand_np = bs.cpu().numpy(), bi.cpu().numpy(), cand.cpu().numpy()
    for b in range(spec.B):
        check_topk_row(want[b], i[b], s[b], k, f"pairwise_bf16x2 {name} exact query {b}")
        check_topk_row(want[b], bi[b], bs[b], k, f"pairwise_bf16x2 {name} bounded query {b}")
        uniq = mo.union_dedup([cand_np[b]])
        full = np.full(spec.N, -np.inf)
        full[uniq] = want[b][uniq]
        check_topk_row(full, ri[b], rs[b], k, f"pairwise_bf16x2 {name} rerank query {b}")
