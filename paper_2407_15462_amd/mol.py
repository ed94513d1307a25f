"""ctypes binding of the MoL C ABI (include/mol.h).

Argument marshalling only: every step of the retrieval path runs in the HIP
kernels of libmol.so.  torch provides device memory and streams.  The
functions carry the C names; the lower-case helpers at the bottom allocate
outputs and workspace with torch and call them.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmol.so")

MOL_OK, MOL_EINVAL, MOL_EUNSUPPORTED, MOL_EWORKSPACE, MOL_EHIP = range(5)
MOL_F32, MOL_BF16 = 0, 1
(MOL_OP_SCORE, MOL_OP_TOPK_EXACT, MOL_OP_TOPK_PER_EMBD, MOL_OP_RERANK, MOL_OP_TOPK_MAXDOT,
 MOL_OP_TOPK_BOUNDED, MOL_OP_TOPK_TWO_PASS) = range(7)
MOL_TWO_PASS_MIN, MOL_TWO_PASS_KTH = 0, 1
MOL_FLAG_F32_GATING = 1
MOL_FLAG_BF16X2_GATING = 2

EXPORTS = ("mol_workspace_size", "mol_score", "mol_topk_exact", "mol_topk_exact_noalloc", "mol_topk_exact_bounded",
           "mol_topk_two_pass", "mol_topk_maxdot", "mol_topk_per_embd",
           "mol_rerank", "mol_avg_embed", "mol_gap_bound", "mol_gap_bound_combined",
           "mol_timing_enable", "mol_timing_read",
           "mol_status_str", "mol_last_error")


class MolError(RuntimeError):
    """A nonzero mol_status from the library."""

    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class MolProblemC(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("Pq", ctypes.c_int32),
                ("Px", ctypes.c_int32), ("d", ctypes.c_int32), ("H", ctypes.c_int32),
                ("dtype", ctypes.c_int32),
                ("Q", ctypes.c_void_p), ("X", ctypes.c_void_p),
                ("a_q", ctypes.c_void_p), ("a_x", ctypes.c_void_p),
                ("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
                ("W2", ctypes.c_void_p), ("b2", ctypes.c_void_p), ("flags", ctypes.c_uint32)]


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmol.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2407_15462_amd.build` (there is no fallback)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(MolProblemC)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sig = {
        "mol_workspace_size": [P, ctypes.c_int, i32, i32, i32, ctypes.POINTER(sz)],
        "mol_score": [P, i32, i32, vp, vp],
        "mol_topk_exact": [P, i32, vp, vp, vp, sz, vp],
        "mol_topk_exact_noalloc": [P, i32, vp, vp, vp],
        "mol_topk_exact_bounded": [P, i32, vp, vp, vp, vp, sz, vp],
        "mol_topk_two_pass": [P, i32, i32, vp, vp, vp, vp, sz, vp],
        "mol_topk_maxdot": [P, i32, vp, vp, vp, sz, vp],
        "mol_topk_per_embd": [P, i32, vp, vp, vp, sz, vp],
        "mol_rerank": [P, vp, i32, vp, i32, i32, vp, vp, vp, vp, sz, vp],
        "mol_avg_embed": [P, vp, vp, vp],
        "mol_gap_bound": [i32, i32, i32, vp, i32, vp, vp, vp, vp, vp, vp],
        "mol_gap_bound_combined": [i32, i32, i32, vp, vp, i32, vp, i32, i32, vp, vp, vp, vp, vp],
        "mol_timing_enable": [ctypes.c_int],
        "mol_timing_read": [ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.mol_status_str.argtypes = [ctypes.c_int]
    lib.mol_status_str.restype = ctypes.c_char_p
    lib.mol_last_error.argtypes = []
    lib.mol_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != MOL_OK:
        lib = load()
        raise MolError(status, f"{lib.mol_status_str(status).decode()}: "
                               f"{lib.mol_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors handed to the MoL library must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


class Problem:
    """A mol_problem built from torch tensors (kept alive by this object).

    Q [B][Pq][d], X [Px][N][d] in bfloat16 or float32; a_q [B][P], a_x [N][P],
    b1 [H], b2 [P] float32; W1 [H][P], W2 [P][H] in the embedding dtype.
    Gating tensors may be None for mol_topk_per_embd.
    """

    def __init__(self, Q, X, a_q=None, a_x=None, W1=None, b1=None, W2=None, b2=None, flags: int = 0):
        self.tensors = (Q, X, a_q, a_x, W1, b1, W2, b2)
        if Q.dtype == torch.bfloat16:
            dtype = MOL_BF16
        elif Q.dtype == torch.float32:
            dtype = MOL_F32
        else:
            raise ValueError(f"unsupported embedding dtype {Q.dtype}")
        B, Pq, d = Q.shape
        Px, N, d2 = X.shape
        H = W1.shape[0] if W1 is not None else 1
        self.c = MolProblemC(B, N, Pq, Px, d if d == d2 else -1, H, dtype,
                             _ptr(Q), _ptr(X), _ptr(a_q), _ptr(a_x), _ptr(W1), _ptr(b1),
                             _ptr(W2), _ptr(b2), flags)
        self.B, self.N, self.Pq, self.Px, self.d, self.H = B, N, Pq, Px, d, H
        self.P = Pq * Px
        self.device = Q.device

    @classmethod
    def from_inputs(cls, inp, flags: int = 0) -> "Problem":
        return cls(inp.Q, inp.X, inp.a_q, inp.a_x, inp.W1, inp.b1, inp.W2, inp.b2, flags)

    @property
    def ref(self):
        return ctypes.byref(self.c)


# ---------------------------------------------------------------- C entry points
def mol_workspace_size(prob: Problem, op: int, k: int = 0, kprime: int = 0, C: int = 0) -> int:
    out = ctypes.c_size_t(0)
    _check(load().mol_workspace_size(prob.ref, op, k, kprime, C, ctypes.byref(out)))
    return out.value


def mol_score(prob: Problem, n_begin: int, n_count: int, phi: torch.Tensor, stream=None) -> None:
    _check(load().mol_score(prob.ref, n_begin, n_count, _ptr(phi), _stream(stream)))


def mol_topk_exact(prob: Problem, k: int, out_score, out_idx, ws, stream=None) -> None:
    _check(load().mol_topk_exact(prob.ref, k, _ptr(out_score), _ptr(out_idx), _ptr(ws),
                                 ws.numel() if ws is not None else 0, _stream(stream)))


def mol_topk_exact_noalloc(prob: Problem, k: int, out_score, out_idx, stream=None) -> None:
    _check(load().mol_topk_exact_noalloc(prob.ref, k, _ptr(out_score), _ptr(out_idx), _stream(stream)))


def mol_topk_exact_bounded(prob: Problem, k: int, bound, out_score, out_idx, ws, stream=None) -> None:
    _check(load().mol_topk_exact_bounded(prob.ref, k, _ptr(bound), _ptr(out_score), _ptr(out_idx),
                                         _ptr(ws), ws.numel() if ws is not None else 0,
                                         _stream(stream)))


def mol_topk_two_pass(prob: Problem, k: int, mode: int, out_score, out_idx, out_bound, ws,
                      stream=None) -> None:
    _check(load().mol_topk_two_pass(prob.ref, k, mode, _ptr(out_score), _ptr(out_idx),
                                    _ptr(out_bound), _ptr(ws), ws.numel() if ws is not None else 0,
                                    _stream(stream)))


def mol_topk_maxdot(prob: Problem, k: int, out_score, out_idx, ws, stream=None) -> None:
    _check(load().mol_topk_maxdot(prob.ref, k, _ptr(out_score), _ptr(out_idx), _ptr(ws),
                                  ws.numel() if ws is not None else 0, _stream(stream)))


def mol_topk_per_embd(prob: Problem, kprime: int, out_dot, out_idx, ws, stream=None) -> None:
    _check(load().mol_topk_per_embd(prob.ref, kprime, _ptr(out_dot), _ptr(out_idx), _ptr(ws),
                                    ws.numel() if ws is not None else 0, _stream(stream)))


def mol_rerank(prob: Problem, cand, C: int, cand2, C2: int, k: int, out_score, out_idx,
               out_n_unique, ws, stream=None) -> None:
    _check(load().mol_rerank(prob.ref, _ptr(cand), C, _ptr(cand2), C2, k, _ptr(out_score),
                             _ptr(out_idx), _ptr(out_n_unique), _ptr(ws),
                             ws.numel() if ws is not None else 0, _stream(stream)))


def mol_avg_embed(prob: Problem, q_avg, x_avg, stream=None) -> None:
    _check(load().mol_avg_embed(prob.ref, _ptr(q_avg), _ptr(x_avg), _stream(stream)))


def mol_gap_bound(B: int, P: int, m: int, dots, k: int, scores, out_S, out_SK, out_bound,
                  out_looser, stream=None) -> None:
    _check(load().mol_gap_bound(B, P, m, _ptr(dots), k, _ptr(scores), _ptr(out_S), _ptr(out_SK),
                                _ptr(out_bound), _ptr(out_looser), _stream(stream)))


def mol_gap_bound_combined(B: int, P: int, m: int, dots, ids, kprime: int, avg_ids, k_avg: int, k: int,
                           scores, out_S, out_SK, out_bound, stream=None) -> None:
    _check(load().mol_gap_bound_combined(B, P, m, _ptr(dots), _ptr(ids), kprime, _ptr(avg_ids), k_avg, k,
                                         _ptr(scores), _ptr(out_S), _ptr(out_SK), _ptr(out_bound),
                                         _stream(stream)))


def mol_timing_enable(on: bool) -> None:
    _check(load().mol_timing_enable(1 if on else 0))


def mol_timing_read(op: int) -> Tuple[float, int]:
    """(summed milliseconds, launch count) of the main kernel of ``op`` since
    the last read; waits for the recorded events."""
    ms, n = ctypes.c_double(0.0), ctypes.c_int32(0)
    _check(load().mol_timing_read(op, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ------------------------------------------------- torch-allocating conveniences
def workspace(prob: Problem, op: int, k: int = 0, kprime: int = 0, C: int = 0) -> torch.Tensor:
    """A uint8 device buffer of the size the library asks for (>= 1 byte)."""
    n = mol_workspace_size(prob, op, k, kprime, C)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=prob.device)


def score(prob: Problem, n_begin: int = 0, n_count: Optional[int] = None, stream=None):
    n_count = prob.N - n_begin if n_count is None else n_count
    phi = torch.empty((prob.B, n_count), dtype=torch.float32, device=prob.device)
    mol_score(prob, n_begin, n_count, phi, stream)
    return phi


def topk_exact(prob: Problem, k: int, ws=None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    ws = workspace(prob, MOL_OP_TOPK_EXACT, k=k) if ws is None else ws
    s = torch.empty((prob.B, k), dtype=torch.float32, device=prob.device)
    i = torch.empty((prob.B, k), dtype=torch.int32, device=prob.device)
    mol_topk_exact(prob, k, s, i, ws, stream)
    return s, i


def _topk_out(prob: Problem, k: int):
    return (torch.empty((prob.B, k), dtype=torch.float32, device=prob.device),
            torch.empty((prob.B, k), dtype=torch.int32, device=prob.device))


def topk_exact_bounded(prob: Problem, k: int, bound: torch.Tensor, ws=None, stream=None):
    """Exact top-k among items whose max component dot can reach bound[b]."""
    ws = workspace(prob, MOL_OP_TOPK_BOUNDED, k=k) if ws is None else ws
    s, i = _topk_out(prob, k)
    mol_topk_exact_bounded(prob, k, bound, s, i, ws, stream)
    return s, i


def topk_two_pass(prob: Problem, k: int, mode: int = MOL_TWO_PASS_MIN, ws=None, stream=None):
    """Algorithm 1: (scores, ids, bound used per query)."""
    ws = workspace(prob, MOL_OP_TOPK_TWO_PASS, k=k) if ws is None else ws
    s, i = _topk_out(prob, k)
    bound = torch.empty((prob.B,), dtype=torch.float32, device=prob.device)
    mol_topk_two_pass(prob, k, mode, s, i, bound, ws, stream)
    return s, i, bound


def topk_maxdot(prob: Problem, k: int, ws=None, stream=None):
    """Top-k by max_p s_p: (max dots, ids)."""
    ws = workspace(prob, MOL_OP_TOPK_MAXDOT, k=k) if ws is None else ws
    s, i = _topk_out(prob, k)
    mol_topk_maxdot(prob, k, s, i, ws, stream)
    return s, i


def topk_per_embd(prob: Problem, kprime: int, ws=None, stream=None):
    ws = workspace(prob, MOL_OP_TOPK_PER_EMBD, kprime=kprime) if ws is None else ws
    s = torch.empty((prob.B, prob.P, kprime), dtype=torch.float32, device=prob.device)
    i = torch.empty((prob.B, prob.P, kprime), dtype=torch.int32, device=prob.device)
    mol_topk_per_embd(prob, kprime, s, i, ws, stream)
    return s, i


def rerank(prob: Problem, cand: torch.Tensor, k: int, ws=None, stream=None,
           cand2: Optional[torch.Tensor] = None):
    """Union of the candidate rows of cand [B][C] (and cand2 [B][C2]),
    deduplicated and reranked with full MoL: (scores, ids, n_unique)."""
    C = cand.shape[1]
    C2 = 0 if cand2 is None else cand2.shape[1]
    ws = workspace(prob, MOL_OP_RERANK, k=k, C=C + C2) if ws is None else ws
    s = torch.empty((prob.B, k), dtype=torch.float32, device=prob.device)
    i = torch.empty((prob.B, k), dtype=torch.int32, device=prob.device)
    nu = torch.empty((prob.B,), dtype=torch.int32, device=prob.device)
    mol_rerank(prob, cand, C, cand2, C2, k, s, i, nu, ws, stream)
    return s, i, nu


def gap_bound(dots: torch.Tensor, scores: torch.Tensor, stream=None):
    """Theorem 2 certificate from per-component lists dots [B][P][m] and the
    reranked scores [B][k]: (S, S_K, bound, looser), each float32 [B]."""
    B, P, m = dots.shape
    k = scores.shape[1]
    outs = [torch.empty((B,), dtype=torch.float32, device=dots.device) for _ in range(4)]
    mol_gap_bound(B, P, m, dots, k, scores, *outs, stream=stream)
    return tuple(outs)


def gap_bound_combined(dots: torch.Tensor, ids: torch.Tensor, kprime: int, avg_ids, scores: torch.Tensor,
                       stream=None):
    """Theorem 3 certificate from per-component lists dots / ids [B][P][m]
    (m > kprime + k_avg), the TopKAvg ids [B][k_avg] (or None) and the
    reranked scores [B][k]: (S', S_K, bound), each float32 [B]."""
    B, P, m = dots.shape
    k = scores.shape[1]
    k_avg = 0 if avg_ids is None else avg_ids.shape[-1]
    outs = [torch.empty((B,), dtype=torch.float32, device=dots.device) for _ in range(3)]
    mol_gap_bound_combined(B, P, m, dots, ids, kprime, avg_ids, k_avg, k, scores, *outs, stream=stream)
    return tuple(outs)


def avg_embed(prob: Problem, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    dt = torch.bfloat16 if prob.c.dtype == MOL_BF16 else torch.float32
    q = torch.empty((prob.B, prob.d), dtype=dt, device=prob.device)
    x = torch.empty((prob.N, prob.d), dtype=dt, device=prob.device)
    mol_avg_embed(prob, q, x, stream)
    return q, x


def averaged_problem(prob: Problem, q_avg: torch.Tensor, x_avg: torch.Tensor) -> Problem:
    """The P = 1 problem TopKAvg runs on (Q = q', X = x')."""
    return Problem(q_avg.view(prob.B, 1, prob.d), x_avg.view(1, prob.N, prob.d))
