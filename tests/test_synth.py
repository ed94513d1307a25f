"""Seeded input generator: determinism, shapes, layouts (CPU)."""
import numpy as np
import torch

import synth


def test_generator_is_deterministic_and_seed_sensitive():
    w = synth.WORKLOADS["exact_32k"].scaled(B=8, N=3000, clusters=16)
    a = synth.to_numpy(synth.generate(w, seed=3))
    b = synth.to_numpy(synth.generate(w, seed=3))
    c = synth.to_numpy(synth.generate(w, seed=4))
    for f in ("Q", "X", "a_q", "a_x", "W1", "b1", "W2", "b2"):
        assert np.array_equal(a[f], b[f]), f
        assert not np.array_equal(a[f], c[f]), f


def test_shapes_dtypes_and_unit_norm_components():
    for name in ("tiny_exact_f32", "exact_32k"):
        w = synth.WORKLOADS[name].scaled(B=4, N=1000, clusters=8)
        inp = synth.generate(w, seed=0)
        P = w.Pq * w.Px
        assert inp.Q.shape == (4, w.Pq, w.d) and inp.X.shape == (w.Px, 1000, w.d)
        assert inp.a_q.shape == (4, P) and inp.a_x.shape == (1000, P)
        assert inp.W1.shape == (w.H, P) and inp.W2.shape == (P, w.H)
        assert inp.b1.shape == (w.H,) and inp.b2.shape == (P,)
        want = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        assert inp.X.dtype == want and inp.Q.dtype == want and inp.a_x.dtype == torch.float32
        tol = 1e-5 if w.dtype == "f32" else 1e-2
        n = torch.linalg.vector_norm(inp.X.float(), dim=-1)
        assert torch.all((n - 1).abs() < tol)
        n = torch.linalg.vector_norm(inp.Q.float(), dim=-1)
        assert torch.all((n - 1).abs() < tol)


def test_noisy_queries_resemble_their_source_item():
    w = synth.WORKLOADS["exact_32k"].scaled(B=64, N=2000, clusters=16)
    inp = synth.generate(w, seed=1)
    # every query component is close to some item's matching component
    q = inp.Q.float()[:, 0, :]                     # pq = 0 -> px = 0
    x = inp.X.float()[0]
    best = (q @ x.T).max(dim=1).values
    assert torch.all(best > 0.3)
