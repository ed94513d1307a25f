"""The library's calls can be captured into a HIP graph (no allocation, no
synchronisation, no memset nodes inside): a captured exact + approximate
pass replayed several times, with eager work overwriting the outputs in
between, reproduces the eager outputs bit for bit on every replay
(MI355X only)."""
import pytest
import torch

import synth
from paper_2407_15462_amd import mol
from parity_helpers import cuda_inputs, log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,spec", [
    ("fused_shape", synth.WORKLOADS["exact_1m"].scaled(B=20, N=4099, clusters=32)),
    ("generic_shape", synth.WORKLOADS["paper_nq320k"].scaled(B=8, N=3001, clusters=16)),
])
def test_graph_replay_matches_eager(name, spec):
    log(f"[graph] {name} B={spec.B} N={spec.N}")
    inp = cuda_inputs(spec, seed=51)
    prob = mol.Problem.from_inputs(inp)
    pe = mol.Problem(inp.Q, inp.X)
    k, kp = 50, 16
    B, P = spec.B, spec.P
    ws_ex = mol.workspace(prob, mol.MOL_OP_TOPK_EXACT, k=k)
    ws_pe = mol.workspace(pe, mol.MOL_OP_TOPK_PER_EMBD, kprime=kp)
    ws_rr = mol.workspace(prob, mol.MOL_OP_RERANK, k=k, C=P * kp)
    ex_s = torch.empty((B, k), device="cuda")
    ex_i = torch.empty((B, k), dtype=torch.int32, device="cuda")
    pe_d = torch.empty((B, P, kp), device="cuda")
    pe_i = torch.empty((B, P, kp), dtype=torch.int32, device="cuda")
    rr_s = torch.empty((B, k), device="cuda")
    rr_i = torch.empty((B, k), dtype=torch.int32, device="cuda")
    rr_n = torch.empty((B,), dtype=torch.int32, device="cuda")
    outs = (ex_s, ex_i, pe_d, pe_i, rr_s, rr_i, rr_n)

    def run():
        mol.mol_topk_exact(prob, k, ex_s, ex_i, ws_ex)
        mol.mol_topk_per_embd(pe, kp, pe_d, pe_i, ws_pe)
        mol.mol_rerank(prob, pe_i.view(B, P * kp), P * kp, None, 0, k, rr_s, rr_i, rr_n, ws_rr)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    want = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(4):
        for t in outs:
            t.fill_(-3)                     # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j, (t, w) in enumerate(zip(outs, want)):
            assert torch.equal(t, w), f"{name}: replay {rep}, output {j} differs from the eager run"
