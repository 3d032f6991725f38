"""Throughput of the MoE-potential training step on one MI355X.

One step = the whole hot path on one batch: neighbour list, geometry and
basis, routing, forward to the energy, force backward, double backward of
the force loss and final backward to every weight gradient.  Inputs are
seeded synthetic batches resident in HBM before the timed region.

Prints ONE JSON line on stdout (details on stderr).  After the warm-up, a
few untimed steps record HIP events around every kernel family (the
per-family table); the timed steps then record events around the dominant
family only, whose average launch time gives the roofline figure.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload irregular]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3e12      # dense fp32 matrix peak of MI355X, FLOP/s
PEAK_HBM = 8.0e12              # HBM3E bandwidth, B/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(b, budget_s: float, seed: int = 0):
    """The float64 oracle, untuned, timed on a bounded sample of the batch: its structures
    in a seeded random order, each one full training step of its own (energy, forces and
    the second-order weight gradient; per structure, the work of a batch step is the same up
    to the loss normalisation), until budget_s seconds of oracle time have passed."""
    import numpy as np
    from oracle.model import training_step
    from paper_2604_15821_amd.synth import subset
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = os.cpu_count()
    order = np.random.default_rng(seed).permutation(b.n_struct)
    atoms, done, dt = 0, 0, 0.0
    for s in order:
        sb = subset(b, [int(s)])
        t0 = time.perf_counter()
        training_step(sb)
        dt += time.perf_counter() - t0
        atoms += sb.n_atoms
        done += 1
        if dt >= budget_s:
            break
    cores = min(aff, blas) if blas else aff
    return {"value": atoms / dt, "unit": "atoms/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} of the batch's {b.n_struct} structures in seeded random order ({atoms} atoms), "
                      f"one full training step each, {dt:.1f} s of oracle time; float64 NumPy, BLAS threads "
                      f"{blas}, affinity {aff}"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # defaults: about a minute of timed work on the full-size batch (6.2 s per step)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="irregular",
                    help="synthetic batch (default: the 512-structure irregular batch, the largest that fits "
                         "one GPU; 'shard' is the 256 x 128-atom per-device share of the billion-scale model)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="oracle time spent on the CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown-steps", type=int, default=None,
                    help="untimed steps with every kernel family's events, for the per-family table "
                         "(default: 3, or 1 when a step takes over a second)")
    ap.add_argument("--workspace-mib", type=int, default=0,
                    help="cap janus_step's workspace (the batch is then processed in chunks of whole structures)")
    ap.add_argument("--serial", action="store_true",
                    help="one stream only (by default the expert weight gradients run on a second stream, "
                         "beside the memory-bound edge and atom kernels)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="one elementwise copy kernel over this many MiB before the run (calibrates HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this library has no multi-GPU path",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2604_15821_amd import janus
    from paper_2604_15821_amd.counters import measured_traffic
    from paper_2604_15821_amd.synth import WORKLOADS, make_batch

    if args.copy_mib > 0:
        # one elementwise kernel that reads and writes copy_mib MiB each
        src = torch.ones(args.copy_mib << 18, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        log(f"calibration copy: {args.copy_mib} MiB read + {args.copy_mib} MiB written")
        del src, dst

    wl = WORKLOADS[args.workload]
    m = wl.model
    b = make_batch(args.workload)
    d = janus.upload(b, "cuda:0")
    ctx = janus.Context(m)
    ctx.set_concurrency(not args.serial)
    if args.workspace_mib:
        ctx.set_workspace_limit(args.workspace_mib << 20)
    nl = ctx.build_edges(d["pos"], d["cell"], d["offsets"])
    Ne = nl.n_edges
    N, S = b.n_atoms, b.n_struct
    out = (torch.empty(1, device="cuda:0"), torch.empty(S, device="cuda:0"), torch.empty(N, 3, device="cuda:0"),
           torch.empty_like(d["W"]))
    # with a stress weight the step also returns the stress and trains on it
    stress = dict(S_ref=d["S_ref"], stress=torch.empty(S, 3, 3, device="cuda:0")) if m.w_S else {}
    if m.n_tasks:
        stress["labels"] = d["labels"]

    def step():
        ne = ctx.build_edges_into(d["pos"], d["cell"], d["offsets"], nl)
        assert ne == Ne
        ctx.step(d["pos"], d["cell"], d["species"], d["offsets"], nl, d["W"], d["E_ref"], d["F_ref"], out=out,
                 **stress)

    log(f"workload {args.workload}: {S} structures, {N} atoms, {Ne} edges, d={m.d} h={m.d_hidden} "
        f"E={m.n_experts} k={m.top_k} T={m.n_blocks}")
    tw = time.perf_counter()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    warm_s = (time.perf_counter() - tw) / max(args.warmup, 1)

    # per-family breakdown from a few untimed steps with every family's events, on one
    # stream, so that each family's rate describes its kernels alone
    nb = args.breakdown_steps if args.breakdown_steps is not None else (1 if warm_s > 1.0 else 3)
    ctx.set_concurrency(False)
    ctx.profile(True)
    for _ in range(nb):
        step()
    torch.cuda.synchronize()
    breakdown = ctx.profile_read()
    ctx.profile(False)
    ctx.set_concurrency(not args.serial)
    # the dominant family (most time) is the one timed inside the timed region
    dom = max(breakdown, key=lambda n: breakdown[n]["ms"])

    ctx.profile(True, families=[dom])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = ctx.profile_read()
    ctx.profile(False)
    Nt = ctx.last_triplets()
    ms = (t1 - t0) * 1e3 / args.steps
    log(f"{ms:.3f} ms/step, loss {float(out[0].cpu()[0]):.6g}, {ctx.last_chunks()} chunk(s)")

    kernels = {}
    for name, r in breakdown.items():
        per = r["ms"] / max(r["launches"], 1)
        e = {"launches_per_step": r["launches"] / nb, "ms_per_step": r["ms"] / nb,
             "avg_launch_ms": per}
        if r["flops"] > 0:
            e["tflops"] = r["flops"] / (r["ms"] * 1e-3) / 1e12
            e["mfma_frac"] = e["tflops"] * 1e12 / PEAK_FP32_MFMA
        if r["bytes"] > 0:
            e["gbs"] = r["bytes"] / (r["ms"] * 1e-3) / 1e9
            e["hbm_frac"] = e["gbs"] * 1e9 / PEAK_HBM
        kernels[name] = e
        log(f"  {name:13s} {r['ms'] / nb:8.3f} ms/step  {r['launches'] / nb:6.1f} launches  "
            + (f"{e.get('tflops', 0):7.2f} TFLOP/s " if 'tflops' in e else "")
            + (f"{e.get('gbs', 0):8.1f} GB/s" if 'gbs' in e else ""))

    if m.n_heads and "attention" in kernels:
        # Algorithmic attention work: per ordered (query, key) pair of a neighbourhood and
        # head, the distinct contractions over the head's d / H columns in the four passes
        # (forward q.k and p v; force backward q.k, p w k, p k and t q; tangent q.k, qh.k,
        # q.kh, pz v, p v, p vh; final backward q.k, qh.k, q.kh, zb k, zhb kh, zb q, zhb qh):
        # 19 of 2 d / H flops.
        deg = torch.diff(nl.rowptr.to(torch.int64)).double()
        attn_flops = 19.0 * 2.0 * (m.d // m.n_heads) * m.n_heads * m.n_blocks * float((deg * deg).sum())
        e = kernels["attention"]
        e["flops_per_step"] = attn_flops
        e["tflops"] = attn_flops / (e["ms_per_step"] * 1e-3) / 1e12
        e["mfma_frac"] = e["tflops"] * 1e12 / PEAK_FP32_MFMA
        log(f"  attention     {e['tflops']:.2f} TFLOP/s of algorithmic contractions, "
            f"{e['mfma_frac']:.3f} of the fp32 matrix peak")

    # roofline of the dominant family, from its events inside the timed region
    r = prof[dom]
    if r["flops"] > 0:
        ach = r["flops"] / r["launches"] / (r["ms"] / r["launches"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": ach, "peak": PEAK_FP32_MFMA / 1e12, "unit": "TFLOP/s",
                "frac": ach * 1e12 / PEAK_FP32_MFMA, "traffic": measured_traffic(args.workload, dom),
                "flops_per_launch": r["flops"] / r["launches"], "avg_launch_ms": r["ms"] / r["launches"]}
    else:
        ach = r["bytes"] / r["launches"] / (r["ms"] / r["launches"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": ach, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": ach * 1e9 / PEAK_HBM, "traffic": measured_traffic(args.workload, dom),
                "bytes_per_launch": r["bytes"] / r["launches"], "avg_launch_ms": r["ms"] / r["launches"]}

    res = {
        "metric": "atoms/s per training step (E+F+2nd-order dL/dW) on 1 MI355X"
        + (" with the stress term" if m.w_S else ""),
        "value": N / (ms * 1e-3),
        "unit": "atoms/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "structures": S, "atoms": N, "edges": Ne, "d": m.d,
                   "d_hidden": m.d_hidden, "experts": m.n_experts, "top_k": m.top_k, "blocks": m.n_blocks,
                   "n_rbf": m.n_rbf, "r_cut": m.r_cut, "parallelism": "none",
                   "streams": 1 if args.serial else 2,
                   **({"workspace_mib": args.workspace_mib} if args.workspace_mib else {}),
                   **({"atom_moe": {"experts": m.n_experts_f, "top_k": m.top_k_f, "d_hidden": m.d_hidden_f}}
                      if m.atom_moe else {}),
                   **({"stress_weight": m.w_S} if m.w_S else {}),
                   **({"robust_loss": {"huber_delta": m.huber_delta, "tau": m.robust_tau}} if m.robust else {}),
                   **({"attention_heads": m.n_heads} if m.n_heads else {}),
                   **({"router": "species pair + linear layer on the edge token"} if m.route_feat else {}),
                   **({"tasks": m.n_tasks, "charges": m.n_charges, "spins": m.n_spins} if m.n_tasks else {})},
        "edges_per_s": Ne / (ms * 1e-3),
        "triplets": Nt,
        "triplets_per_s": Nt / (ms * 1e-3),
        "expert_gemm_flops_per_step": 24.0 * m.top_k * m.d * m.d_hidden * Ne * m.n_blocks
        + (24.0 * m.top_k_f * m.d * m.d_hidden_f * N * m.n_blocks if m.atom_moe else 0.0),
        "roofline": roof,
        "kernels": kernels,
        "kernels_note": "per-family rates from untimed steps on one stream; the roofline's kernel is timed "
                        "inside the timed region",
    }
    ctx.close()
    del d, nl, out
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(b, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
