"""Throughput benchmark of the MoL retrieval hot path on one MI355X.

One step = one pass of the whole path over one batch of the workload.
Default workload exact_1m (B = 1024 queries, N = 1,048,576 items,
P_q = P_x = 8, d = 64, H = 64, bf16):
  exact:  mol_topk_exact (fused MoL scoring + top-100 selection)
  approx: mol_topk_per_embd (top-128 per component, all 64 components)
          + mol_rerank (union, dedup, MoL rerank to top-100)
With --workload hybrid_8m (B = 256, N = 8,388,608, P = 8 x 4, d = 128,
H = 128) the approximate path also runs TopKAvg (mol_avg_embed of the
queries + mol_topk_per_embd top-1024 on the averaged embeddings, whose item
side is precomputed outside the timed region) and reranks the union of both
candidate sets.
With --workload paper_ml20m / paper_books / paper_nq320k (the item counts,
component counts and widths of the paper's top-K benchmark, 32 queries per
call) it times each method row of the paper's table instead -- brute force,
TopKPerEmbd(N), TopKAvg(N), CombTopK(N1, N2) -- plus the two-pass exact
algorithm and the max-component heuristic: mean, standard deviation and
median of the call latency over --steps warm runs (HIP events on the
stream), the mean latency of the same calls captured once into a HIP graph
and replayed, and recall@100 against the brute-force result.
Inputs are synthetic, seeded, and resident in HBM before timing starts.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoL top-100 queries/sec at N=1M (exact + approx); recall@100 vs exact; % MFMA peak"
PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA
F32_GATING_STD = 0.3           # largest gating-entry RMS the fused f16 chain is stated for (include/mol.h)
X2_GATING_STD = 1.0            # largest the fused two-term bf16 chain is stated for (include/mol.h)
PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2407_15462_amd", "csrc")
# sources of the fused exact scan kernel: a traffic figure measured on other
# sources is stale and is not reported
FUSED_SOURCES = ("mol_fused.hip", "mol_tile.h", "mol_device.h")
TRAFFIC_FILE = "traffic_k_mol_fused_{workload}.txt"
COUNTER_FILE = "counters_k_mol_fused_{workload}.txt"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="exact_1m")
    ap.add_argument("--paths", default="exact,approx")
    ap.add_argument("--cpu-baseline-queries", type=int, default=None,
                    help="oracle queries timed for cpu_baseline (default: about 10-20 s of work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extras", default="hybrid_8m,exact_1m_skewed",
                    help="other workloads summarised as extra keys of the exact_1m line "
                         "(comma list; empty for none)")
    ap.add_argument("--extra-steps", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--issue-probe", action="store_true",
                    help="only time the issue-rate probe of the fused scan's per-step instruction "
                         "mix (libmol_probe.so) at 1-4 waves per SIMD and print the implied floor")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (the "
                         "reference dispatch that scales FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def source_digest(names=FUSED_SOURCES) -> str:
    """sha256 of the kernel sources with comments and whitespace removed, so
    that only a change of the code itself marks a measurement as stale."""
    import hashlib
    import re
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def profile_values(name: str):
    """key: value lines of a committed profile summary of the fused exact
    scan, or None when it is missing or was taken on other kernel sources."""
    path = os.path.join(PROFILES, name)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    return kv if kv.get("source_sha256") == source_digest() else None


def measured_traffic(workload: str):
    """HBM bytes per launch of the fused exact scan (FETCH_SIZE + WRITE_SIZE
    counters, copy-calibrated), or None."""
    kv = profile_values(TRAFFIC_FILE.format(workload=workload))
    try:
        return float(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def measured_counters(workload: str):
    """Matrix-core and vector-ALU occupancy of the fused exact scan from its
    committed counter summary (SQ_VALU_MFMA_BUSY_CYCLES, SQ_ACTIVE_INST_VALU,
    SQ_VALU_MFMA_COEXEC_CYCLES, GRBM_GUI_ACTIVE), or None."""
    kv = profile_values(COUNTER_FILE.format(workload=workload))
    if not kv:
        return None
    keys = ("mfma_busy_frac", "valu_active_frac", "mfma_valu_coexec_frac", "simd_busy_frac",
            "gpu_clock_ghz", "valu_insts_per_mfma", "trans_insts_per_mfma")
    try:
        return {k: float(kv[k]) for k in keys}
    except (KeyError, ValueError):
        return None


def measured_issue_floor(workload: str):
    """The issue-rate floor of the fused scan's instruction stream at its two
    waves per SIMD (bench.py --issue-probe, summarised in profiles/), reported
    while the kernel's counter summary -- whose per-step counts the probe
    issues -- still matches the sources; else None."""
    if measured_counters(workload) is None:
        return None
    path = os.path.join(PROFILES, f"issue_floor_k_mol_fused_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    try:
        return {"waves_per_simd": int(kv["kernel_waves_per_simd"]),
                "mix_floor_ms": float(kv["mix_floor_ms_w2"]), "mix_frac_max": float(kv["mix_frac_max_w2"]),
                "full_stream_floor_ms": float(kv["full_stream_floor_ms_w2"]),
                "full_stream_frac_max": float(kv["full_stream_frac_max_w2"])}
    except (KeyError, ValueError):
        return None


def copy_calibration():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for i in range(3):
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"# copy {i}: {n} bytes", file=sys.stderr, flush=True)
    print(json.dumps({"copy_bytes": n, "dispatches": 3}), flush=True)


def issue_probe(iters=2000):
    """Time the probe kernel of include/mol_probe.h: the fused scan's
    per-step instruction mix (48 MFMA, 97 transcendental, 206 plain vector
    instructions, 32 pack conversions per wave-step) issued with no
    dependencies, no memory traffic and no barriers, at 1-4 waves per SIMD.
    Prints ns per wave-step per SIMD and the floor it implies for the fused
    exact scan at exact_1m (1024 x 2^20 pairs = 32768 wave-steps per SIMD)."""
    import ctypes

    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2407_15462_amd", "libmol_probe.so"))
    lib.mol_probe_issue_mix.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    names = {0: "mix_interleaved", 1: "vector_only", 2: "mfma_only", 3: "mix_phased", 4: "full_stream"}
    stream = torch.cuda.current_stream()
    out = {}
    for w in (1, 2, 3, 4):
        sink = torch.empty(256 * w * 256, dtype=torch.float32, device="cuda")
        for p, name in names.items():
            for n_it in (iters // 10, iters):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                rc = lib.mol_probe_issue_mix(p, w, n_it, ctypes.c_void_p(sink.data_ptr()),
                                             ctypes.c_void_p(stream.cuda_stream))
                e1.record()
                if rc != 0:
                    raise RuntimeError(f"mol_probe_issue_mix failed ({rc})")
            torch.cuda.synchronize()
            ns = e0.elapsed_time(e1) * 1e6 / (w * iters)
            out[f"{name}_w{w}_ns_per_wave_step"] = ns
            print(f"# issue probe {name} waves/SIMD={w}: {ns:.1f} ns per wave-step", file=sys.stderr, flush=True)
    steps_per_simd = (1024 // 2) * (1 << 20) // 16 // 1024
    flops = 1024 * (1 << 20) * (2 * 64 * 64 + 4 * 64 * 64)
    for w in (1, 2, 3, 4):
        best = min(out[f"mix_interleaved_w{w}_ns_per_wave_step"], out[f"mix_phased_w{w}_ns_per_wave_step"])
        ms = best * steps_per_simd / 1e6
        out[f"exact_1m_floor_ms_w{w}"] = ms
        out[f"exact_1m_frac_max_w{w}"] = flops / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS
        full = out[f"full_stream_w{w}_ns_per_wave_step"] * steps_per_simd / 1e6
        out[f"exact_1m_full_stream_floor_ms_w{w}"] = full
        out[f"exact_1m_full_stream_frac_max_w{w}"] = flops / (full / 1e3) / 1e12 / PEAK_BF16_TFLOPS
    print(json.dumps({"issue_probe": out, "iters": iters,
                      "mix_per_wave_step": {"mfma_16x16x32": 48, "transcendental": 97, "plain_valu": 206,
                                            "cvt_pk_f16_f32": 32},
                      "wave_steps_per_simd_exact_1m": steps_per_simd}), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the retrieval path has no multi-GPU mode "
              "(corpus sharding is a design note only)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.issue_probe:
        issue_probe()
        return
    import torch

    import synth
    from paper_2407_15462_amd import mol

    spec = synth.WORKLOADS[args.workload]
    if spec.name in synth.PAPER_METHODS:
        paper_table(spec, args)
        return
    paths = [p for p in args.paths.split(",") if p]
    out, inp = run_workload(spec, args.steps, args.warmup, paths, args.seed)
    ms_step = out.pop("_ms_step")
    line = {
        "metric": METRIC,
        "value": spec.B / (ms_step / 1e3),
        "unit": "queries/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": spec.dtype, "data": "synthetic",
        "config": {"workload": spec.name, "B": spec.B, "N": spec.N, "Pq": spec.Pq, "Px": spec.Px,
                   "d": spec.d, "H": spec.H, "k": spec.k,
                   "kprime": (spec.kprime or 128) if "approx" in paths else None, "paths": paths},
    }
    line.update(out)
    if not args.no_cpu_baseline:
        nq = args.cpu_baseline_queries or max(1, (16 << 20) // spec.N)
        line["cpu_baseline"] = cpu_baseline(inp, spec, nq, max(1, nq // 8))
    del inp
    extras = [e for e in args.extras.split(",") if e and e != spec.name] if spec.name == "exact_1m" else []
    for name in extras:
        import torch
        torch.cuda.empty_cache()
        x_spec = synth.WORKLOADS[name]
        x_out, x_inp = run_workload(x_spec, args.extra_steps, 1, ["exact", "approx"], args.seed)
        x_ms = x_out.pop("_ms_step")
        summary = {"config": {"B": x_spec.B, "N": x_spec.N, "Pq": x_spec.Pq, "Px": x_spec.Px, "d": x_spec.d,
                              "H": x_spec.H, "k": x_spec.k, "kprime": x_spec.kprime, "k_avg": x_spec.k_avg or None,
                              "gating_std": x_spec.gating_std},
                   "steps": args.extra_steps, "ms_per_step": x_ms, "queries_per_s": x_spec.B / (x_ms / 1e3)}
        ex, ap_, rf = x_out.get("exact", {}), x_out.get("approx", {}), x_out.get("roofline", {})
        summary.update({
            "exact_ms": ex.get("ms"), "exact_kernel_ms": ex.get("kernel_ms"), "exact_path": ex.get("path"),
            "fused_frac": rf.get("frac"), "fused_traffic": rf.get("traffic"),
            "approx_ms": ap_.get("ms"), "per_embd_ms": ap_.get("ms_per_embd"),
            "topk_avg_ms": ap_.get("ms_topk_avg"), "rerank_ms": ap_.get("ms_rerank"),
            "recall_at_100_vs_exact": ap_.get("recall_at_100_vs_exact"),
            "candidates_per_query_mean": ap_.get("candidates_per_query_mean")})
        line[name] = summary
        print(f"# extra {name}: {x_ms:.1f} ms/step, recall {summary['recall_at_100_vs_exact']}",
              file=sys.stderr, flush=True)
        del x_inp
    print(json.dumps(line), flush=True)


def run_workload(spec, steps, warmup, paths, seed):
    """Time `steps` steps (after `warmup`) of the exact and / or approximate
    path on one workload.  Returns (result keys, the inputs)."""
    import statistics

    import torch

    import synth
    from paper_2407_15462_amd import mol

    dev = "cuda"
    t0 = time.time()
    inp = synth.generate(spec, seed=seed, device=dev)
    torch.cuda.synchronize()
    print(f"# generated {spec.name} in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    # gating weights beyond the fused f16 chain's stated range (entries of RMS
    # up to 0.3, include/mol.h) take the two-term bf16 chain (up to 1), and
    # beyond that the library's float32 gating path
    gating = ("f16" if spec.gating_std <= F32_GATING_STD else
              "bf16x2" if spec.gating_std <= X2_GATING_STD else "f32")
    flags = {"f16": 0, "bf16x2": mol.MOL_FLAG_BF16X2_GATING, "f32": mol.MOL_FLAG_F32_GATING}[gating]
    prob = mol.Problem.from_inputs(inp, flags)
    B, N, P, d, H, k = spec.B, spec.N, spec.P, spec.d, spec.H, spec.k
    kprime = spec.kprime or 128

    # outputs and workspaces allocated once, outside the timed region
    ws_exact = mol.workspace(prob, mol.MOL_OP_TOPK_EXACT, k=k)
    ex_s = torch.empty((B, k), dtype=torch.float32, device=dev)
    ex_i = torch.empty((B, k), dtype=torch.int32, device=dev)
    pe_prob = mol.Problem(inp.Q, inp.X)
    C = P * kprime
    k_avg = spec.k_avg
    if "approx" in paths:
        ws_pe = mol.workspace(pe_prob, mol.MOL_OP_TOPK_PER_EMBD, kprime=kprime)
        pe_d = torch.empty((B, P, kprime), dtype=torch.float32, device=dev)
        pe_i = torch.empty((B, P, kprime), dtype=torch.int32, device=dev)
        if k_avg:
            # item side of TopKAvg: precomputed once (preprocessing, untimed)
            x_avg = torch.empty((N, d), dtype=inp.Q.dtype, device=dev)
            q_avg = torch.empty((B, d), dtype=inp.Q.dtype, device=dev)
            mol.mol_avg_embed(pe_prob, None, x_avg)
            avg_prob = mol.averaged_problem(pe_prob, q_avg, x_avg)
            ws_av = mol.workspace(avg_prob, mol.MOL_OP_TOPK_PER_EMBD, kprime=k_avg)
            av_d = torch.empty((B, 1, k_avg), dtype=torch.float32, device=dev)
            av_i = torch.empty((B, 1, k_avg), dtype=torch.int32, device=dev)
        ws_rr = mol.workspace(prob, mol.MOL_OP_RERANK, k=k, C=C + k_avg)
        rr_s = torch.empty((B, k), dtype=torch.float32, device=dev)
        rr_i = torch.empty((B, k), dtype=torch.int32, device=dev)
        rr_n = torch.empty((B,), dtype=torch.int32, device=dev)

    ev = lambda: torch.cuda.Event(enable_timing=True)
    seg = {p: [] for p in ("exact", "per_embd", "topk_avg", "rerank")}

    def step(record):
        if "exact" in paths:
            e0, e1 = ev(), ev()
            e0.record()
            mol.mol_topk_exact(prob, k, ex_s, ex_i, ws_exact)
            e1.record()
            if record:
                seg["exact"].append((e0, e1))
        if "approx" in paths:
            e0, e1, e2, e3 = ev(), ev(), ev(), ev()
            e0.record()
            mol.mol_topk_per_embd(pe_prob, kprime, pe_d, pe_i, ws_pe)
            e1.record()
            if k_avg:
                mol.mol_avg_embed(pe_prob, q_avg, None)
                mol.mol_topk_per_embd(avg_prob, k_avg, av_d, av_i, ws_av)
            e2.record()
            mol.mol_rerank(prob, pe_i.view(B, C), C, av_i.view(B, k_avg) if k_avg else None, k_avg, k,
                           rr_s, rr_i, rr_n, ws_rr)
            e3.record()
            if record:
                seg["per_embd"].append((e0, e1))
                seg["topk_avg"].append((e1, e2))
                seg["rerank"].append((e2, e3))

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    timed_ops = (mol.MOL_OP_TOPK_EXACT, mol.MOL_OP_TOPK_PER_EMBD, mol.MOL_OP_RERANK)
    for op in timed_ops:
        mol.mol_timing_read(op)             # drop anything recorded before
    mol.mol_timing_enable(True)
    t_start = time.perf_counter()
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    mol.mol_timing_enable(False)
    ms_step = 1e3 * wall / steps
    seg_ms = {p: [a.elapsed_time(b) for a, b in v] for p, v in seg.items()}
    ms = {p: (statistics.fmean(v) if v else None) for p, v in seg_ms.items()}

    def spread(v):
        return {"median": statistics.median(v), "std": statistics.stdev(v) if len(v) > 1 else 0.0}
    kern = {}          # main-kernel milliseconds per launch
    kern_step = {}     # main-kernel milliseconds per step (all launches of the op)
    for op in timed_ops:
        tot, n = mol.mol_timing_read(op)
        kern[op] = tot / n if n else None
        kern_step[op] = tot / steps if n else None

    flops_pair = 2 * P * d + 4 * P * H
    out = {"_ms_step": ms_step}
    if ms["exact"]:
        t = ms["exact"] / 1e3
        # the float32 gating path times no single main kernel: its event time stands in
        tk = (kern[mol.MOL_OP_TOPK_EXACT] if kern[mol.MOL_OP_TOPK_EXACT] is not None else ms["exact"]) / 1e3
        # the dots-only share of the work (2 P d of the 2 P d + 4 P H flop)
        out["exact"] = {"ms": ms["exact"], "ms_spread": spread(seg_ms["exact"]), "kernel_ms": tk * 1e3,
                        "queries_per_s": B / t,
                        "items_scored_per_s": B * N / t,
                        "mfma_frac_dots_only": B * N * 2.0 * P * d / tk / 1e12 / PEAK_BF16_TFLOPS}
        # algorithmic work of one launch: every (query, item) pair once,
        # 2 P d flops of component dots + 4 P H of the gating MLP
        ach = B * N * flops_pair / tk / 1e12
        traffic = measured_traffic(spec.name)
        out["exact"]["path"] = {"f16": "fused", "bf16x2": "fused, two-term bf16 gating",
                                "f32": "float32 gating (pair-wise)"}[gating]
        if gating == "f16":
            out["roofline"] = {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                               "unit": "TFLOP/s", "frac": ach / PEAK_BF16_TFLOPS, "traffic": traffic,
                               "kernel": "k_mol_fused (MoL scoring + per-range top-k scan)",
                               "flops_per_launch": B * N * flops_pair,
                               "counters": measured_counters(spec.name),
                               "issue_floor": measured_issue_floor(spec.name)}
    if ms["per_embd"]:
        t = (ms["per_embd"] + ms["topk_avg"] + ms["rerank"]) / 1e3
        recall = None
        if "exact" in paths:
            ex = ex_i.cpu()
            got = rr_i.cpu()
            hits = sum(len(set(a.tolist()) & set(b.tolist())) for a, b in zip(got, ex))
            recall = hits / ex.numel()
        # both scans of every per-component (and TopKAvg) list, per step
        tpe = kern_step[mol.MOL_OP_TOPK_PER_EMBD] / 1e3
        pe_flops = 2.0 * B * P * N * d + (2.0 * B * N * d if k_avg else 0.0)
        # rerank: every unique candidate's P_x d bf16 components and P
        # float32 item logits gathered once
        uniq_total = float(rr_n.float().sum().item())
        trr = (kern[mol.MOL_OP_RERANK] if kern[mol.MOL_OP_RERANK] is not None else ms["rerank"]) / 1e3
        approx_ms = [a + b + c for a, b, c in zip(seg_ms["per_embd"], seg_ms["topk_avg"], seg_ms["rerank"])]
        out["approx"] = {"ms": statistics.fmean(approx_ms), "ms_spread": spread(approx_ms),
                         "ms_per_embd": ms["per_embd"], "ms_topk_avg": ms["topk_avg"] if k_avg else None,
                         "k_avg": k_avg or None, "ms_rerank": ms["rerank"],
                         "kernel_ms_per_embd_per_step": tpe * 1e3,
                         "kernel_ms_rerank": kern[mol.MOL_OP_RERANK],
                         "per_embd_mfma_frac": pe_flops / tpe / 1e12 / PEAK_BF16_TFLOPS,
                         "reranked_pairs_per_s": uniq_total / trr,
                         "rerank_gather_hbm_frac": uniq_total * (spec.Px * d * 2 + P * 4) / trr / 1e9
                         / PEAK_HBM_GBS,
                         "queries_per_s": B / t,
                         "recall_at_100_vs_exact": recall,
                         "candidates_per_query_mean": uniq_total / B}

    return out, inp


def paper_table(spec, args):
    """Latency of every method row of the paper's top-K table on a synthetic
    instance of one of its workload shapes (32 queries per call)."""
    import statistics

    import torch

    import synth
    from paper_2407_15462_amd import mol

    dev = "cuda"
    inp = synth.generate(spec, seed=args.seed, device=dev)
    prob = mol.Problem.from_inputs(inp)
    pe_prob = mol.Problem(inp.Q, inp.X)
    B, N, P, d, k = spec.B, spec.N, spec.P, spec.d, spec.k
    # item side of TopKAvg: materialised once, untimed (preprocessing)
    x_avg = torch.empty((N, d), dtype=inp.Q.dtype, device=dev)
    q_avg = torch.empty((B, d), dtype=inp.Q.dtype, device=dev)
    mol.mol_avg_embed(pe_prob, None, x_avg)
    avg_prob = mol.averaged_problem(pe_prob, q_avg, x_avg)

    def out2(n):
        return (torch.empty((B, n), dtype=torch.float32, device=dev),
                torch.empty((B, n), dtype=torch.int32, device=dev))

    ex_s, ex_i = out2(k)
    ws_ex = mol.workspace(prob, mol.MOL_OP_TOPK_EXACT, k=k)
    rr_s, rr_i = out2(k)
    rr_n = torch.empty((B,), dtype=torch.int32, device=dev)

    def method(row):
        """(label, callable running the whole method) or (label, reason)"""
        kind = row[0]
        n1 = row[1] if kind in ("per_embd", "comb") else 0
        n2 = row[1] if kind == "avg" else (row[2] if kind == "comb" else 0)
        label = {"per_embd": f"TopKPerEmbd({n1})", "avg": f"TopKAvg({n2})",
                 "comb": f"CombTopK{n1}_{n2}"}[kind]
        try:
            C = P * n1
            if n1:
                ws_pe = mol.workspace(pe_prob, mol.MOL_OP_TOPK_PER_EMBD, kprime=n1)
                pe_d = torch.empty((B, P, n1), dtype=torch.float32, device=dev)
                pe_i = torch.empty((B, P, n1), dtype=torch.int32, device=dev)
            if n2:
                ws_av = mol.workspace(avg_prob, mol.MOL_OP_TOPK_PER_EMBD, kprime=n2)
                av_d = torch.empty((B, 1, n2), dtype=torch.float32, device=dev)
                av_i = torch.empty((B, 1, n2), dtype=torch.int32, device=dev)
            ws_rr = mol.workspace(prob, mol.MOL_OP_RERANK, k=k, C=C + n2)
        except mol.MolError as e:
            return label, str(e)

        def run():
            if n1:
                mol.mol_topk_per_embd(pe_prob, n1, pe_d, pe_i, ws_pe)
            if n2:
                mol.mol_avg_embed(pe_prob, q_avg, None)
                mol.mol_topk_per_embd(avg_prob, n2, av_d, av_i, ws_av)
            first = pe_i.view(B, C) if n1 else av_i.view(B, n2)
            second = av_i.view(B, n2) if (n1 and n2) else None
            mol.mol_rerank(prob, first, C if n1 else n2, second, n2 if (n1 and n2) else 0, k,
                           rr_s, rr_i, rr_n, ws_rr)
        return label, run

    rows = [("BruteForce", lambda: mol.mol_topk_exact(prob, k, ex_s, ex_i, ws_ex))]
    for r in synth.PAPER_METHODS[spec.name]:
        rows.append(method(r))
    ws_tp = mol.workspace(prob, mol.MOL_OP_TOPK_TWO_PASS, k=k)
    tp_s, tp_i = out2(k)
    rows.append(("TwoPassExact(k-th bound)",
                 lambda: mol.mol_topk_two_pass(prob, k, mol.MOL_TWO_PASS_KTH, tp_s, tp_i, None, ws_tp)))
    mx_n = min(1024, 10 * k)
    ws_mx = mol.workspace(pe_prob, mol.MOL_OP_TOPK_MAXDOT, k=mx_n)
    ws_mr = mol.workspace(prob, mol.MOL_OP_RERANK, k=k, C=mx_n)
    mx_s, mx_i = out2(mx_n)

    def maxdot_rerank():
        mol.mol_topk_maxdot(pe_prob, mx_n, mx_s, mx_i, ws_mx)
        mol.mol_rerank(prob, mx_i, mx_n, None, 0, k, rr_s, rr_i, rr_n, ws_mr)
    rows.append((f"MaxTopK({mx_n})", maxdot_rerank))

    def timed(run):
        times = []
        for _ in range(args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run()
            e1.record()
            times.append((e0, e1))
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in times]

    def graph_latency(fn, outs):
        """The method captured once into a HIP graph and replayed: mean
        latency over --steps replays.  Every replay of a first batch is
        checked against the eager outputs, with the outputs overwritten by
        eager work in between."""
        want = [t.clone() for t in outs]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        for _ in range(3):
            for t in outs:
                t.fill_(-7)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for t, w in zip(outs, want):
                if not torch.equal(t, w):
                    raise RuntimeError("graph replay differs from the eager result")
        ms = timed(g.replay)
        return statistics.fmean(ms)

    # brute force first: its result is the recall reference of every row
    results = []
    exact_ids = None
    for label, fn in rows:
        if not callable(fn):
            results.append({"method": label, "supported": False, "reason": fn})
            continue
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ms = timed(fn)
        outs = ((ex_s, ex_i) if label == "BruteForce" else (tp_s, tp_i) if label.startswith("TwoPass")
                else (rr_s, rr_i))
        got = outs[1].cpu()
        if exact_ids is None:
            exact_ids = got.clone()
        hits = sum(len(set(a.tolist()) & set(b.tolist())) for a, b in zip(got, exact_ids))
        mean = statistics.fmean(ms)
        try:
            graph_ms = graph_latency(fn, outs)
        except RuntimeError as e:          # capture refused or replay mismatch: report, go on
            graph_ms = None
            print(f"# {label}: no graph latency ({e})", file=sys.stderr, flush=True)
        results.append({"method": label, "latency_ms": mean,
                        "latency_std_ms": statistics.stdev(ms) if len(ms) > 1 else 0.0,
                        "latency_median_ms": statistics.median(ms),
                        "graph_latency_ms": graph_ms,
                        "queries_per_s": B / (mean / 1e3),
                        "recall_at_100_vs_exact": hits / exact_ids.numel(),
                        "candidates_per_query_mean": None if label in ("BruteForce",) or
                        label.startswith("TwoPass") else float(rr_n.float().mean().item())})
        print(f"# {label}: {mean:.3f} ms (graph replay {graph_ms})", file=sys.stderr, flush=True)
    bf = results[0]["latency_ms"]
    print(json.dumps({
        "metric": "MoL top-100 latency per batch of 32 queries, paper top-K table shapes",
        "value": bf, "unit": "ms (brute force)", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "higher_is_better": False, "vs_baseline": None,
        "dtype": spec.dtype, "data": "synthetic",
        "config": {"workload": spec.name, "B": B, "N": N, "Pq": spec.Pq, "Px": spec.Px, "d": d,
                   "H": spec.H, "k": k},
        "methods": results}), flush=True)


def cpu_model_name():
    """The host CPU's full model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        r = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10)
        for line in r.stdout.splitlines():
            if line.strip().lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# host threads given to the oracle: the CPU share of one GPU on the benchmark
# hosts (16), or fewer where the machine has fewer
CPU_THREAD_CAP = 16


def cpu_baseline(inp, spec, nq, nq_single=1):
    """The FP64 oracle, as it stands, on a bounded sample of the same
    workload: exact MoL top-k for the first ``nq`` queries over all N items
    with the BLAS pool at the host's thread share, and for the first
    ``nq_single`` queries with one thread."""
    from threadpoolctl import threadpool_info, threadpool_limits

    import synth
    from oracle import mol_oracle as mo

    threads = min(CPU_THREAD_CAP, os.cpu_count() or 1)
    arrays = synth.to_numpy(inp, queries=list(range(max(nq, nq_single))))
    op = mo.Problem.from_arrays(arrays)

    def timed(n, limit):
        with threadpool_limits(limits=limit):
            used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
            t0 = time.perf_counter()
            mo.exact_topk(op, list(range(n)), spec.k)
            return time.perf_counter() - t0, used

    dt, used = timed(nq, threads)
    dt1, _ = timed(nq_single, 1)
    return {"value": nq / dt, "unit": "queries/s", "cores": used, "kind": "oracle",
            "sample": f"exact top-{spec.k} for {nq} of {spec.B} queries over all "
                      f"{spec.N} items (FP64 NumPy, BLAS threads={used}); single-thread leg: "
                      f"the first {nq_single} of them",
            "seconds": dt, "threads": used,
            "thread_cap": f"{CPU_THREAD_CAP} (the host CPU share of one GPU)",
            "single_thread_queries_per_s": nq_single / dt1, "single_thread_seconds": dt1,
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model_name()}


if __name__ == "__main__":
    main()
