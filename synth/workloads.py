"""Seeded synthetic Mixture-of-Logits workloads.

The shapes follow the paper's retrieval workloads (Section 4.3, workload
statistics table: P_q = 8 query components, P_x in {4, 8} item components,
d in {64, 128}) and the problem statement of top-K retrieval with MoL
(Section 3, Definition 1).  The real datasets and trained encoders are not
available, so the component embeddings are drawn from seeded distributions:

* ``iid``      every component vector is N(0, I_d), then L2-normalised;
* ``mixture``  each item picks one of C clusters uniformly; every
               (cluster, item component) pair has its own centre drawn from
               N(0, I_d); an item component is its centre plus 0.3 N(0, I_d),
               L2-normalised.  Query b copies a random source item: query
               component pq is item component (pq mod P_x) of the source plus
               ``q_noise`` N(0, I_d), L2-normalised.

Gating parameters (per-query logits a_q, per-item logits a_x, and the
two-layer gating MLP W1, b1, W2, b2) are 0.1 N(0, 1).  For bf16 workloads the
embeddings and the MLP weight matrices are stored in bfloat16 (round to
nearest even); the logits and biases stay float32.

Layouts (all row-major, C-contiguous):

  Q   [B][P_q][d]      query component embeddings
  X   [P_x][N][d]      item component embeddings, component-major
  a_q [B][P]  a_x [N][P]  W1 [H][P]  b1 [H]  W2 [P][H]  b2 [P]
  with p = pq * P_x + px.

Every array is drawn from its own generator, keyed by (seed, workload name,
array name, chunk), so a workload is reproducible on a given device type.
Generation on "cuda" and on "cpu" give different (but each deterministic)
values; callers hand the same arrays to the GPU library and to the oracle.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Dict, Optional

import numpy as np
import torch

_CHUNK = 1 << 20  # items generated per chunk (bounds host/device temporaries)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    Pq: int
    Px: int
    d: int
    H: int
    dtype: str            # "f32" or "bf16": storage type of Q, X, W1, W2
    k: int                # final top-k
    items: str            # "iid" or "mixture"
    clusters: int = 0
    q_noise: float = 0.0
    kprime: int = 0       # per-component top-k' (approximate path)
    k_avg: int = 0        # averaged-embedding top-k (approximate path)
    gating_std: float = 0.1   # standard deviation of a_q, a_x, W1, b1, W2, b2
    side_logits: bool = True  # per-query / per-item gating logits a_q, a_x (else zero)
    note: str = ""

    @property
    def P(self) -> int:
        return self.Pq * self.Px

    def scaled(self, B: Optional[int] = None, N: Optional[int] = None,
               clusters: Optional[int] = None) -> "Workload":
        """Same recipe at a different size (parity tests use smaller ones)."""
        return dataclasses.replace(
            self,
            B=self.B if B is None else B,
            N=self.N if N is None else N,
            clusters=self.clusters if clusters is None else clusters)


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny_exact_f32", B=32, N=4096, Pq=4, Px=4, d=64, H=32,
                 dtype="f32", k=10, items="iid",
                 note="exact MoL top-10 in fp32"),
        Workload("exact_32k", B=1024, N=32768, Pq=8, Px=4, d=64, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=256,
                 q_noise=0.2, note="exact MoL top-100, 32K items"),
        Workload("exact_1m", B=1024, N=1 << 20, Pq=8, Px=8, d=64, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=4096,
                 q_noise=0.2, kprime=128,
                 note="exact MoL top-100 at corpus scale, 1M items"),
        Workload("approx_1m", B=1024, N=1 << 20, Pq=8, Px=8, d=64, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=4096,
                 q_noise=0.2, kprime=128,
                 note="TopKPerEmbd(128) over all 64 components, then rerank"),
        Workload("exact_1m_skewed", B=1024, N=1 << 20, Pq=8, Px=8, d=64, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=4096,
                 q_noise=0.2, kprime=128, gating_std=0.5,
                 note="the 1M-item data with gating parameters of standard "
                      "deviation 0.5: the largest gating weight averages about 0.23"),
        Workload("hybrid_8m", B=256, N=1 << 23, Pq=8, Px=4, d=128, H=128,
                 dtype="bf16", k=100, items="mixture", clusters=16384,
                 q_noise=0.2, kprime=256, k_avg=1024,
                 note="per-component top-256 and averaged top-1024, rerank"),
        # Shapes of the paper's top-K retrieval benchmark (Section 4's workload
        # table: items, P_q x P_x, d_P), measured on batches of 32 queries.
        # The query noise gives a cosine of about 0.53 to the source item at
        # every d (sigma = 1.6 / sqrt(d)).  The hidden width is not stated:
        # H = 128 at d = 128, 64 otherwise.  The question-answering workload
        # gates on the dot products alone (no per-query / per-item logits).
        Workload("paper_ml20m", B=32, N=24186, Pq=8, Px=4, d=128, H=128,
                 dtype="bf16", k=100, items="mixture", clusters=128,
                 q_noise=1.6 / 128 ** 0.5,
                 note="ML-20M shape: 24,186 items, 8 x 4 components, d = 128"),
        Workload("paper_books", B=32, N=674044, Pq=8, Px=8, d=32, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=4096,
                 q_noise=1.6 / 32 ** 0.5,
                 note="Books shape: 674,044 items, 8 x 8 components, d = 32"),
        Workload("paper_nq320k", B=32, N=109739, Pq=4, Px=4, d=768, H=64,
                 dtype="bf16", k=100, items="mixture", clusters=512,
                 q_noise=1.6 / 768 ** 0.5, side_logits=False,
                 note="NQ320K shape: 109,739 items, 4 x 4 components, d = 768"),
    ]
}

# Method rows of the paper's top-K table for each of its workloads:
# ("per_embd", N), ("avg", N), ("comb", N1, N2).
PAPER_METHODS = {
    "paper_ml20m": [("per_embd", 5), ("per_embd", 10), ("per_embd", 50), ("per_embd", 100),
                    ("avg", 200), ("avg", 500), ("comb", 5, 200)],
    "paper_books": [("per_embd", 5), ("per_embd", 50), ("per_embd", 100), ("per_embd", 200),
                    ("avg", 200), ("avg", 500), ("avg", 1000), ("avg", 2000), ("avg", 4000),
                    ("avg", 8000), ("comb", 5, 200), ("comb", 50, 500), ("comb", 100, 1000),
                    ("comb", 200, 2000)],
    "paper_nq320k": [("per_embd", 5), ("per_embd", 10), ("per_embd", 50), ("avg", 100),
                     ("comb", 5, 100)],
}

# The 1M-item approximate workload reuses the exact one's data.
_DATA_ALIAS = {"approx_1m": "exact_1m", "exact_1m_skewed": "exact_1m"}


@dataclasses.dataclass
class MolInputs:
    """Device tensors of one workload instance (see module docstring)."""
    spec: Workload
    Q: torch.Tensor
    X: torch.Tensor
    a_q: torch.Tensor
    a_x: torch.Tensor
    W1: torch.Tensor
    b1: torch.Tensor
    W2: torch.Tensor
    b2: torch.Tensor

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.spec.dtype == "bf16" else torch.float32


def _generator(device: str, *key) -> torch.Generator:
    h = hashlib.sha256(repr(key).encode()).digest()
    g = torch.Generator(device=device)
    g.manual_seed(int.from_bytes(h[:8], "little") & ((1 << 63) - 1))
    return g


def _unit(v: torch.Tensor) -> torch.Tensor:
    return v / torch.linalg.vector_norm(v, dim=-1, keepdim=True)


def generate(spec: Workload, seed: int = 0, device: str = "cpu") -> MolInputs:
    """Draw one seeded instance of ``spec`` on ``device``."""
    name = _DATA_ALIAS.get(spec.name, spec.name)
    store = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    B, N, Pq, Px, d, H, P = spec.B, spec.N, spec.Pq, spec.Px, spec.d, spec.H, spec.P
    key = (seed, name, B, N)

    def randn(shape, *k):
        return torch.randn(shape, generator=_generator(device, *key, *k),
                           device=device, dtype=torch.float32)

    X = torch.empty((Px, N, d), dtype=store, device=device)
    a_x = torch.empty((N, P), dtype=torch.float32, device=device)
    if spec.items == "mixture":
        C = max(1, spec.clusters)
        centres = randn((C, Px, d), "centres")
    for c0 in range(0, N, _CHUNK):
        n = min(_CHUNK, N - c0)
        z = randn((n, Px, d), "items", c0)
        if spec.items == "mixture":
            cid = torch.randint(0, C, (n,), device=device,
                                generator=_generator(device, *key, "cluster", c0))
            z = centres[cid] + 0.3 * z
        X[:, c0:c0 + n, :] = _unit(z).to(store).permute(1, 0, 2)
        a_x[c0:c0 + n] = (spec.gating_std if spec.side_logits else 0.0) * randn((n, P), "a_x", c0)

    if spec.items == "mixture":
        src = torch.randint(0, N, (B,), device=device,
                            generator=_generator(device, *key, "qsrc"))
        base = torch.stack([X[pq % Px, src, :].float() for pq in range(Pq)], dim=1)
        Q = _unit(base + spec.q_noise * randn((B, Pq, d), "qnoise")).to(store)
    else:
        Q = _unit(randn((B, Pq, d), "queries")).to(store)

    sd = spec.gating_std
    sd_side = sd if spec.side_logits else 0.0
    return MolInputs(
        spec=spec, Q=Q.contiguous(), X=X,
        a_q=(sd_side * randn((B, P), "a_q")).contiguous(),
        a_x=a_x,
        W1=(sd * randn((H, P), "W1")).to(store).contiguous(),
        b1=(sd * randn((H,), "b1")).contiguous(),
        W2=(sd * randn((P, H), "W2")).to(store).contiguous(),
        b2=(sd * randn((P,), "b2")).contiguous(),
    )


def _np(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def to_numpy(inp: MolInputs, queries=None, fields=None) -> Dict[str, object]:
    """Host copies for the oracle: bf16 tensors become their uint16 bit
    patterns, float32 tensors stay float32.  ``queries`` selects a subset of
    query rows (Q and a_q) for sampled checks."""
    fields = fields or ("Q", "X", "a_q", "a_x", "W1", "b1", "W2", "b2")
    out: Dict[str, object] = {"dtype": inp.spec.dtype, "Pq": inp.spec.Pq,
                              "Px": inp.spec.Px}
    for f in fields:
        t = getattr(inp, f)
        if queries is not None and f in ("Q", "a_q"):
            t = t[torch.as_tensor(queries, device=t.device, dtype=torch.long)]
        out[f] = _np(t)
    return out
