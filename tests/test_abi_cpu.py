"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments on the host before launching anything (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2407_15462_amd import mol

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mol.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mol_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = mol.load()
    names = declared_functions()
    assert set(names) == set(mol.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_probe_library_exports_its_declared_function():
    # the measurement aid of include/mol_probe.h, built next to libmol.so
    path = os.path.join(ROOT, "paper_2407_15462_amd", "libmol_probe.so")
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "mol_probe.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(mol_[a-z_]+)\s*\(", text)))
    assert names == ["mol_probe_issue_mix"]
    lib = ctypes.CDLL(path)
    for n in names:
        assert hasattr(lib, n), n
    # arguments are checked before any launch: nothing runs without a GPU
    f = lib.mol_probe_issue_mix
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    assert f(0, 0, 10, 256, None) == -1
    assert f(7, 1, 10, 256, None) == -1
    assert f(5, 1, 10, 256, None) == -1
    assert f(0, 1, 0, 256, None) == -1
    assert f(0, 1, 10, None, None) == -1


def _problem(**kw):
    # Non-null dummy pointers: validation must reject before any launch.
    fake = 256
    c = mol.MolProblemC(4, 100, 2, 2, 64, 16, mol.MOL_BF16, fake, fake, fake, fake, fake, fake,
                        fake, fake)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def _ws(c, op, k=0, kp=0, C=0):
    lib = mol.load()
    out = ctypes.c_size_t(0)
    rc = lib.mol_workspace_size(ctypes.byref(c), op, k, kp, C, ctypes.byref(out))
    return rc, out.value


def test_status_strings_and_last_error():
    lib = mol.load()
    assert lib.mol_status_str(0) == b"MOL_OK"
    assert b"workspace" in lib.mol_status_str(3)
    rc, _ = _ws(_problem(B=0), mol.MOL_OP_TOPK_EXACT, k=5)
    assert rc == mol.MOL_EINVAL and b"B=0" in lib.mol_last_error()


@pytest.mark.parametrize("field,value,status", [
    ("B", 0, mol.MOL_EINVAL), ("N", -1, mol.MOL_EINVAL), ("d", 0, mol.MOL_EINVAL),
    ("H", 0, mol.MOL_EINVAL), ("Pq", 40, mol.MOL_EUNSUPPORTED), ("d", 4096, mol.MOL_EUNSUPPORTED),
    ("H", 1000, mol.MOL_EUNSUPPORTED), ("dtype", 7, mol.MOL_EUNSUPPORTED),
    ("Q", None, mol.MOL_EINVAL), ("a_x", None, mol.MOL_EINVAL), ("W2", None, mol.MOL_EINVAL),
    ("B", 65536, mol.MOL_EUNSUPPORTED),
])
def test_problem_validation(field, value, status):
    rc, _ = _ws(_problem(**{field: value}), mol.MOL_OP_TOPK_EXACT, k=5)
    assert rc == status


def test_k_and_C_limits():
    c = _problem()
    assert _ws(c, mol.MOL_OP_TOPK_EXACT, k=0)[0] == mol.MOL_EINVAL
    assert _ws(c, mol.MOL_OP_TOPK_EXACT, k=101)[0] == mol.MOL_EINVAL      # k > N
    assert _ws(c, mol.MOL_OP_TOPK_PER_EMBD, kp=2000)[0] == mol.MOL_EINVAL
    assert _ws(c, mol.MOL_OP_RERANK, k=5, C=0)[0] == mol.MOL_EINVAL
    assert _ws(c, mol.MOL_OP_RERANK, k=5, C=20000)[0] == mol.MOL_EINVAL
    assert _ws(c, 9)[0] == mol.MOL_EINVAL
    rc, n = _ws(c, mol.MOL_OP_TOPK_EXACT, k=10)
    assert rc == mol.MOL_OK and n > 0 and n % 256 == 0
    rc, n = _ws(c, mol.MOL_OP_SCORE)
    assert rc == mol.MOL_OK and n == 0
    # per-embedding top-k' needs no gating tensors
    rc, _ = _ws(_problem(a_q=None, a_x=None, W1=None, b1=None, W2=None, b2=None, H=0),
                mol.MOL_OP_TOPK_PER_EMBD, kp=10)
    assert rc == mol.MOL_OK


def test_entry_points_reject_before_launch():
    lib = mol.load()
    c = _problem()
    ws = ctypes.c_void_p(256)
    # workspace too small -> MOL_EWORKSPACE, nothing launched
    rc = lib.mol_topk_exact(ctypes.byref(c), 10, 256, 256, ws, 16, None)
    assert rc == mol.MOL_EWORKSPACE
    # misaligned workspace
    rc = lib.mol_topk_exact(ctypes.byref(c), 10, 256, 256, ctypes.c_void_p(257), 1 << 40, None)
    assert rc == mol.MOL_EINVAL
    rc = lib.mol_score(ctypes.byref(c), 90, 20, 256, None)        # range past N
    assert rc == mol.MOL_EINVAL
    assert lib.mol_score(ctypes.byref(c), 0, 0, None, None) == mol.MOL_OK   # empty range
    rc = lib.mol_rerank(ctypes.byref(c), None, 8, None, 0, 5, 256, 256, None, ws, 1 << 40, None)
    assert rc == mol.MOL_EINVAL
    # second candidate set: NULL with C2 > 0, negative C2, total above the limit
    cand = ctypes.c_void_p(256)
    assert lib.mol_rerank(ctypes.byref(c), cand, 8, None, 4, 5, 256, 256, None, ws, 1 << 40,
                          None) == mol.MOL_EINVAL
    assert lib.mol_rerank(ctypes.byref(c), cand, 8, cand, -1, 5, 256, 256, None, ws, 1 << 40,
                          None) == mol.MOL_EINVAL
    assert lib.mol_rerank(ctypes.byref(c), cand, 16000, cand, 1000, 5, 256, 256, None, ws,
                          1 << 40, None) == mol.MOL_EINVAL
    assert lib.mol_topk_exact(None, 10, 256, 256, ws, 1 << 40, None) == mol.MOL_EINVAL


def test_timing_records_are_empty_and_validated():
    lib = mol.load()
    ms, n = ctypes.c_double(-1.0), ctypes.c_int32(-1)
    assert lib.mol_timing_enable(0) == mol.MOL_OK
    assert lib.mol_timing_read(mol.MOL_OP_TOPK_EXACT, ctypes.byref(ms), ctypes.byref(n)) == mol.MOL_OK
    assert (ms.value, n.value) == (0.0, 0)
    assert lib.mol_timing_read(7, ctypes.byref(ms), ctypes.byref(n)) == mol.MOL_EINVAL
    assert lib.mol_timing_read(-1, ctypes.byref(ms), ctypes.byref(n)) == mol.MOL_EINVAL
    assert lib.mol_timing_read(0, None, ctypes.byref(n)) == mol.MOL_EINVAL
    # a call rejected before launch records nothing
    c = _problem()
    assert lib.mol_timing_enable(1) == mol.MOL_OK
    assert lib.mol_topk_exact(ctypes.byref(c), 10, 256, 256, ctypes.c_void_p(256), 16, None) \
        == mol.MOL_EWORKSPACE
    assert lib.mol_timing_enable(0) == mol.MOL_OK
    assert lib.mol_timing_read(mol.MOL_OP_TOPK_EXACT, ctypes.byref(ms), ctypes.byref(n)) == mol.MOL_OK
    assert n.value == 0


def test_gap_bound_validation():
    lib = mol.load()
    p = ctypes.c_void_p(256)
    assert lib.mol_gap_bound(0, 8, 5, p, 10, p, None, None, None, None, None) == mol.MOL_EINVAL
    assert lib.mol_gap_bound(4, 65, 5, p, 10, p, None, None, None, None, None) == mol.MOL_EINVAL
    assert lib.mol_gap_bound(4, 8, 1, p, 10, p, None, None, None, None, None) == mol.MOL_EINVAL
    assert lib.mol_gap_bound(4, 8, 5, p, 0, p, None, None, None, None, None) == mol.MOL_EINVAL
    assert lib.mol_gap_bound(4, 8, 5, None, 10, p, None, None, None, None, None) == mol.MOL_EINVAL


def test_two_pass_bounded_and_maxdot_validation():
    """Algorithm 1 / bounded / max-dot entry points reject bad arguments
    before launching anything."""
    lib = mol.load()
    c = _problem(N=100000)
    ws = ctypes.c_void_p(256)
    big = 1 << 40
    # workspace sizes exist for the new operations
    for op, k in ((mol.MOL_OP_TOPK_MAXDOT, 10), (mol.MOL_OP_TOPK_BOUNDED, 10),
                  (mol.MOL_OP_TOPK_TWO_PASS, 10)):
        rc, n = _ws(c, op, k=k)
        assert rc == mol.MOL_OK and n > 0, op
    # the two-pass algorithm reranks P k candidates: at most 16384
    wide = _problem(N=100000, Pq=8, Px=8)
    assert _ws(wide, mol.MOL_OP_TOPK_TWO_PASS, k=256)[0] == mol.MOL_OK
    assert _ws(wide, mol.MOL_OP_TOPK_TWO_PASS, k=257)[0] == mol.MOL_EINVAL
    assert lib.mol_topk_two_pass(ctypes.byref(wide), 257, 0, 256, 256, None, ws, big, None) \
        == mol.MOL_EINVAL
    assert lib.mol_topk_two_pass(ctypes.byref(c), 10, 2, 256, 256, None, ws, big, None) \
        == mol.MOL_EINVAL
    assert lib.mol_topk_two_pass(ctypes.byref(c), 10, mol.MOL_TWO_PASS_KTH, None, 256, None, ws,
                                 big, None) == mol.MOL_EINVAL
    assert lib.mol_topk_two_pass(ctypes.byref(c), 10, mol.MOL_TWO_PASS_MIN, 256, 256, None, ws, 16,
                                 None) == mol.MOL_EWORKSPACE
    assert lib.mol_topk_two_pass(ctypes.byref(_problem(a_q=None)), 10, 0, 256, 256, None, ws, big,
                                 None) == mol.MOL_EINVAL
    # bounded: the bound array is required; k within [1, min(N, 8192)]
    assert lib.mol_topk_exact_bounded(ctypes.byref(c), 10, None, 256, 256, ws, big, None) \
        == mol.MOL_EINVAL
    assert lib.mol_topk_exact_bounded(ctypes.byref(c), 0, 256, 256, 256, ws, big, None) \
        == mol.MOL_EINVAL
    assert lib.mol_topk_exact_bounded(ctypes.byref(c), 10, 256, 256, 256, ws, 16, None) \
        == mol.MOL_EWORKSPACE
    # max-dot reads only Q and X: gating pointers may be NULL, H is ignored
    bare = _problem(N=100000, a_q=None, a_x=None, W1=None, b1=None, W2=None, b2=None, H=0)
    rc, n = _ws(bare, mol.MOL_OP_TOPK_MAXDOT, k=10)
    assert rc == mol.MOL_OK and n > 0
    assert lib.mol_topk_maxdot(ctypes.byref(bare), 10, 256, 256, ws, 16, None) == mol.MOL_EWORKSPACE
    assert lib.mol_topk_maxdot(ctypes.byref(bare), 100001, 256, 256, ws, big, None) == mol.MOL_EINVAL
    assert lib.mol_topk_maxdot(ctypes.byref(bare), 10, None, 256, ws, big, None) == mol.MOL_EINVAL


def test_combined_gap_bound_validation():
    lib = mol.load()
    ok = (4, 8, 40, 256, 256, 10, 256, 20, 5, 256, None, None, None, None)
    args = list(ok)
    # lists must hold more than kprime + k_avg entries
    args[2] = 30
    assert lib.mol_gap_bound_combined(*args) == mol.MOL_EINVAL
    args = list(ok)
    args[6] = None                     # avg_ids NULL with k_avg > 0
    assert lib.mol_gap_bound_combined(*args) == mol.MOL_EINVAL
    args = list(ok)
    args[1] = 65                       # P > 64
    assert lib.mol_gap_bound_combined(*args) == mol.MOL_EINVAL
    args = list(ok)
    args[8] = 0                        # k < 1
    assert lib.mol_gap_bound_combined(*args) == mol.MOL_EINVAL
    args = list(ok)
    args[3] = None                     # dots NULL
    assert lib.mol_gap_bound_combined(*args) == mol.MOL_EINVAL


def test_noalloc_entry_point_validates_on_the_host():
    """mol_topk_exact_noalloc rejects bad arguments, and problems whose
    workspace would exceed the library's static scratch, before touching the
    GPU."""
    lib = mol.load()
    c = _problem(B=4, N=1000, Pq=8, Px=8, d=64, H=64)
    assert lib.mol_topk_exact_noalloc(ctypes.byref(c), 10, None, 256, None) == mol.MOL_EINVAL
    assert lib.mol_topk_exact_noalloc(ctypes.byref(c), 0, 256, 256, None) == mol.MOL_EINVAL
    assert lib.mol_topk_exact_noalloc(None, 10, 256, 256, None) == mol.MOL_EINVAL
    big = _problem(B=65535, N=1 << 20, Pq=8, Px=8, d=64, H=64)
    rc, need = _ws(big, mol.MOL_OP_TOPK_EXACT, k=100)
    assert rc == mol.MOL_OK and need > 16 << 20
    assert lib.mol_topk_exact_noalloc(ctypes.byref(big), 100, 256, 256, None) == mol.MOL_EWORKSPACE
    assert b"scratch" in lib.mol_last_error()


def test_unknown_problem_flags_are_rejected():
    lib = mol.load()
    c = _problem()
    c.flags = 0x6
    rc, _ = _ws(c, mol.MOL_OP_TOPK_EXACT, k=5)
    assert rc == mol.MOL_EINVAL and b"flag" in lib.mol_last_error()
    for flags in (mol.MOL_FLAG_F32_GATING, mol.MOL_FLAG_BF16X2_GATING,
                  mol.MOL_FLAG_F32_GATING | mol.MOL_FLAG_BF16X2_GATING):
        c.flags = flags
        rc, _ = _ws(c, mol.MOL_OP_TOPK_EXACT, k=5)
        assert rc == mol.MOL_OK
