"""Seeded synthetic inputs for Mixture-of-Logits retrieval.

This package only draws random numbers and lays them out; it holds none of
the scoring or retrieval arithmetic.  Both the GPU library (through its
Python binding) and the CPU oracle consume what it produces.
"""
from .workloads import PAPER_METHODS, WORKLOADS, Workload, MolInputs, generate, to_numpy

__all__ = ["PAPER_METHODS", "WORKLOADS", "Workload", "MolInputs", "generate", "to_numpy"]
