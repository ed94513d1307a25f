"""MI355X-native Mixture-of-Logits retrieval (gfx950 HIP kernels behind a C ABI).

The compute path lives in libmol.so (paper_2407_15462_amd/csrc, declared in
include/mol.h); this package is its Python binding.
"""
from . import mol
from .mol import (MolError, Problem, avg_embed, averaged_problem, rerank, score,
                  topk_exact, topk_per_embd)

__all__ = ["mol", "MolError", "Problem", "score", "topk_exact", "topk_per_embd", "rerank",
           "avg_embed", "averaged_problem"]
