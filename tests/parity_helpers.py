"""Shared helpers for the GPU-vs-oracle parity tests."""
from __future__ import annotations

import sys

import numpy as np
import torch

import synth
from oracle import mol_oracle as mo

TAU = 1e-4          # score tolerance and tie window (absolute)
MAX_ERR = {}        # largest |gpu - oracle| seen per check label (reported at session end)


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_problem(inp: synth.MolInputs) -> mo.Problem:
    return mo.Problem.from_arrays(synth.to_numpy(inp))


def check_scores(got: np.ndarray, want: np.ndarray, tol: float = TAU, what: str = "phi") -> None:
    err = np.abs(got.astype(np.float64) - want)
    if err.size == 0:
        return
    i = np.unravel_index(np.argmax(err), err.shape)
    label = what.split(" ")[0]
    MAX_ERR[label] = max(MAX_ERR.get(label, 0.0), float(err.max()))
    assert err.max() <= tol, f"{what}: max |err| {err.max():.3e} at {i} (got {got[i]}, want {want[i]})"


def check_topk_row(scores_all: np.ndarray, got_ids: np.ndarray, got_scores: np.ndarray, k: int,
                   what: str) -> None:
    """tau rule on ids, plus returned scores within TAU of the exact ones and
    returned order (score desc, id asc)."""
    ok, msg = mo.valid_topk(scores_all, got_ids, k, TAU)
    assert ok, f"{what}: {msg}"
    check_scores(got_scores, scores_all[got_ids], what=f"{what} scores")
    s = got_scores.astype(np.float64)
    for j in range(k - 1):
        assert s[j] > s[j + 1] or (s[j] == s[j + 1] and got_ids[j] < got_ids[j + 1]), \
            f"{what}: order broken at rank {j}"


def assert_dedup_set(ids_row, n_unique, want, what):
    """The deduplicated union G as an exact integer set: the first n_unique
    slots hold distinct ids equal to the oracle's union, the rest is padding."""
    got = np.asarray(ids_row[:n_unique], dtype=np.int64)
    assert n_unique == len(want), f"{what}: {n_unique} unique ids, {len(want)} in the union"
    assert len(np.unique(got)) == n_unique, f"{what}: duplicate ids in the deduplicated set"
    assert np.array_equal(np.sort(got), want), \
        f"{what}: id set differs from the union ({np.setdiff1d(want, got)[:5]} missing, " \
        f"{np.setdiff1d(got, want)[:5]} extra)"
    assert np.all(ids_row[n_unique:] == -1), f"{what}: padding past the unique ids"


def recall(got_ids: np.ndarray, exact_ids: np.ndarray) -> float:
    hits = sum(len(set(g.tolist()) & set(e.tolist())) for g, e in zip(got_ids, exact_ids))
    return hits / exact_ids.size


def cuda_inputs(spec: synth.Workload, seed: int = 0) -> synth.MolInputs:
    return synth.generate(spec, seed=seed, device="cuda")
