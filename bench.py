#!/usr/bin/env python3
"""Benchmark of the TreeSpark draft-tree step on one MI355X.

Workload (the batched-serving case at V=151936): 64 requests, D=16, r=64,
bf16 inputs, K=8, T=0.7, per-request theta drawn from {0.02, 0.05, 0.1, 0.2},
synthetic inputs (see paper_2609_22098_amd/synth.py).  One step is one pass of
the whole hot path over that batch:
  1. ts_expand over the 2048-parent serving frontier (2 parents at every depth
     of every request): conditional logits on MFMA, log-sum-exp, top-k,
     k draws without replacement (sequential sampler by default), child
     scoring;
  2. ts_build_tree: best-first trees for the 64 requests under their theta
     (waves on the device; the trees come back to the host and stay on the
     device);
  3. ts_tree_mask: the trees' attention masks and position ids for the
     target's verification pass, from the device copy of the trees;
  4. ts_verify: recursive-rejection verification of those trees at T=0.7.
value = node evaluations (frontier parents + tree-building parents) per
second over the step.  The roofline object covers the dominant kernel (the
streaming pass of ts_expand), timed with HIP events on its own stream, against
the roofline that binds it (HBM bytes or VALU issue slots; the other one is
reported as roofline_other).

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "parent-conditioned node evals/sec at V=151936 + achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
# VALU issue peak: 256 CUs x 4 SIMDs x 32 fp32 lanes per cycle x 2.4 GHz (the
# 157.3 TFLOP/s fp32 vector figure counts an FMA as two); transcendentals
# (v_exp_f32, v_log_f32) issue at a quarter of that rate.
VALU_PEAK_TOPS = 256 * 4 * 32 * 2.4e9 / 1e12
TRANS_WEIGHT = 4
KERNEL_SOURCES = ("paper_2609_22098_amd/csrc/expand_kernels.hpp",
                  "paper_2609_22098_amd/csrc/device_common.hpp")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "expand_eval_serving_traffic.json")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (same process-wide runtime)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            rc = self.hip.hipEventCreate(ctypes.byref(h))
            assert rc == 0, f"hipEventCreate failed ({rc})"
            self.ev[i] = h

    def address(self, i):
        """Address of handle i, i.e. of an array of consecutive hipEvent_t."""
        return ctypes.addressof(self.ev) + i * ctypes.sizeof(ctypes.c_void_p)

    def elapsed_ms(self, a, b):
        t = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(t), self.ev[a], self.ev[b])
        assert rc == 0, f"hipEventElapsedTime failed ({rc})"
        return t.value

    def close(self):
        """Destroy the events while the runtime is up (nothing is left for exit-time teardown)."""
        for i in range(len(self.ev)):
            if self.ev[i]:
                rc = self.hip.hipEventDestroy(self.ev[i])
                assert rc == 0, f"hipEventDestroy failed ({rc})"
                self.ev[i] = None


def copy_calibration(gib, args_out=""):
    """A plain device copy of known size, for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = int(gib * (1 << 30))
    a = torch.ones(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    rec = {"copy_bytes": n, "launches": 3}
    if args_out:
        os.makedirs(args_out, exist_ok=True)
        with open(os.path.join(args_out, "copy.json"), "w") as f:
            json.dump(rec, f)
    print(json.dumps(rec))


EVAL_KERNEL = "expand_eval_lds_kernel"
EVAL_FRONTIER = "expand_eval_lds_kernel<2, 2,"  # rank 64 (KS = 2), two parent blocks per wave


def _counter_per_dispatch(run_dir, counter, name_part):
    """Per-dispatch totals of one counter (summed over its hardware instances) for the
    kernels whose name contains name_part, from a rocprofv3 --pmc csv directory, as
    (grid size, value) pairs."""
    import csv
    import glob
    tot, grid = {}, {}
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for row in csv.DictReader(fh):
                if row["Counter_Name"] != counter or name_part not in row["Kernel_Name"]:
                    continue
                key = (f, row["Dispatch_Id"])
                tot[key] = tot.get(key, 0.0) + float(row["Counter_Value"])
                grid[key] = int(row["Grid_Size"])
    return [(grid[k], v) for k, v in tot.items()]


def _largest_grid(pairs):
    g = max(p[0] for p in pairs)
    return [v for gk, v in pairs if gk == g]


def write_traffic(root, T, sampler):
    """HBM bytes per launch of the streaming pass from FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for a plain copy of known size."""
    with open(os.path.join(root, "copy_fetch", "copy.json")) as f:
        copy_bytes = json.load(f)["copy_bytes"]
    scale = {}
    for counter, sub in (("FETCH_SIZE", "copy_fetch"), ("WRITE_SIZE", "copy_write")):
        vals = _counter_per_dispatch(os.path.join(root, sub), counter, "")
        kib = max(v for _, v in vals)  # the copy is by far the largest dispatch of its run
        scale[counter] = copy_bytes / (kib * 1024.0)
    # the serving frontier's launch: two parent blocks per wave (the tree waves'
    # launches take one, and their upper-bound grids can be larger), rank 64
    fetch = _largest_grid(_counter_per_dispatch(os.path.join(root, "fetch"), "FETCH_SIZE", EVAL_FRONTIER))
    write = _largest_grid(_counter_per_dispatch(os.path.join(root, "write"), "WRITE_SIZE", EVAL_FRONTIER))
    fb = float(np.mean(fetch)) * 1024.0 * scale["FETCH_SIZE"]
    wb = float(np.mean(write)) * 1024.0 * scale["WRITE_SIZE"]
    rec = {"kernel": EVAL_KERNEL, "T": T, "sampler": sampler, "kernel_source_hash": kernel_source_hash(),
           "fetch_kib_per_dispatch": float(np.mean(fetch)), "write_kib_per_dispatch": float(np.mean(write)),
           "dispatches": [len(fetch), len(write)], "copy_bytes": copy_bytes,
           "copy_scale": scale, "fetch_bytes": fb, "write_bytes": wb, "bytes_per_launch": fb + wb}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def cpu_baseline(dr, fr, K, T, seed, seconds, sampler):
    from oracle import oracle
    om = oracle.Model(dr.U32, dr.E32, dr.W2_32)
    n, t0 = 0, time.perf_counter()
    while True:
        oracle.eval_node(om, int(fr["request"][n]), int(fr["token"][n]), int(fr["depth"][n]),
                         int(fr["path"][n]), T, seed, K, want_z=False, sampler=sampler)
        n += 1
        el = time.perf_counter() - t0
        if (el >= seconds and n >= 4) or n == len(fr["token"]):
            break
    return {"value": n / el, "unit": "node-evals/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of the 2048 frontier parents at T={T} (full-vocabulary fp64 "
                      f"evaluation with {sampler} draws, one thread), {el:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--expand-only", action="store_true", help="time only ts_expand (profiling runs)")
    ap.add_argument("--T", type=float, default=0.7, help="temperature (the workload uses 0.7)")
    ap.add_argument("--sampler", default="sequential", choices=("sequential", "gumbel"),
                    help="realisation of the sibling draws at T > 0")
    ap.add_argument("--copy-gib", type=float, default=0.0, help="run only the copy calibration")
    ap.add_argument("--copy-out", default="", help="directory for the copy calibration record")
    ap.add_argument("--traffic-from", default="",
                    help="directory holding the four FETCH_SIZE / WRITE_SIZE counter runs "
                         "(fetch, write, copy_fetch, copy_write); writes the traffic file and exits")
    args = ap.parse_args()
    if args.traffic_from:
        write_traffic(args.traffic_from, args.T, args.sampler)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the draft-tree step runs on "
              f"a single GPU (how it would shard is described in the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_22098_amd import binding, synth
    binding.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_gib > 0:
        copy_calibration(args.copy_gib, args.copy_out)
        return

    w = synth.WORKLOADS[3]
    T, K, N, seed = args.T, w["K"], w["N"], 0
    log("generating the 64-request V=151936 workload")
    dr = synth.make_workload_drafter(3, seed=0)
    fr = synth.make_frontier(dr, per_depth=w["frontier_per_depth"], seed=0)
    anchors, thetas, _ = synth.make_controls(dr.R, dr.V, w["theta"], seed=0)
    P = len(fr["token"])
    dd = binding.drafter_from_host(dr)
    # a second copy of U: alternate steps read different 311 MB buffers, so the
    # 256 MB Infinity Cache cannot serve one step's U from the previous step
    dd2 = binding.DeviceDrafter(dd.U.clone(), dd.E, dd.W2)
    drafters = (dd, dd2)
    parents = binding.parents_to_device(fr["token"], fr["depth"], fr["request"], fr["log_surv"], fr["path"])
    sampler = args.sampler
    outs = binding.expand(dd, parents, P, K, T, seed, sampler=sampler)
    ws_e = outs.pop("_workspace")
    ws_b = torch.empty(binding.build_tree_workspace_size(dd, N, K, T), dtype=torch.uint8, device="cuda")
    ws_v = torch.empty(max(1, binding.verify_workspace_size(dd, N + 1, T)), dtype=torch.uint8, device="cuda")
    tree = binding.build_tree(dd, anchors, thetas, N, K, T, seed, workspace=ws_b, sampler=sampler)
    # target logits for the trees: row i = U[q][min(depth_i, D-1)] + N(0, 1) noise
    tgt = torch.zeros((dr.R, N + 1, dr.V), dtype=torch.bfloat16, device="cuda")
    for q in range(dr.R):
        n1 = int(tree.n[q]) + 1
        s, _ = synth.make_target_rows(dr, q, tree.depth[q, :n1], w["target_sigma"], seed=0)
        tgt[q, :n1] = torch.from_numpy(s).view(torch.bfloat16).cuda()
    tree_evals = int(tree.evals.sum())
    log(f"frontier P={P}; natural trees: sizes {int(tree.n.min())}..{int(tree.n.max())}, "
        f"{tree_evals} evaluations")

    # the trees also stay on the device, where ts_tree_mask reads them
    dtree = binding.DeviceTree(dr.R, N + 1)
    W = binding.lib().ts_tree_mask_words(N + 1)
    mask_out = (torch.empty((dr.R, N + 1, W), dtype=torch.int32, device="cuda"),
                torch.empty((dr.R, N + 1), dtype=torch.int32, device="cuda"))
    nsteps = args.steps + args.warmup
    ev = HipEvents(3 * nsteps)
    # a serving loop holds its stream and output buffers across rounds
    stream = torch.cuda.current_stream()
    vout = (np.zeros((dr.R, binding.TS_MAX_D), np.int32), np.zeros(dr.R, np.int32), np.zeros(dr.R, np.int32))

    def step(i):
        d = drafters[i % 2]
        binding.expand(d, parents, P, K, T, seed, outputs=outs, workspace=ws_e, events=ev.address(3 * i),
                       sampler=sampler, stream=stream)
        if args.expand_only:
            return
        binding.build_tree(d, anchors, thetas, N, K, T, seed, workspace=ws_b, tree=tree, sampler=sampler,
                           device_tree=dtree, stream=stream)
        binding.tree_mask(dtree.parent, dtree.n, N + 1, out=mask_out, stream=stream)
        binding.verify(d, tree, tgt, T, seed, workspace=ws_v, stream=stream, out=vout)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.warmup, nsteps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    eval_ms = np.array([ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(args.warmup, nsteps)])
    merge_ms = np.array([ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(args.warmup, nsteps)])
    assert int(outs["diag"].sum().item()) == 0

    # phase breakdown from a few extra synchronised steps (outside the timed region)
    phases = {}
    if not args.expand_only:
        tb = tv = te = 0.0
        for i in range(3):
            torch.cuda.synchronize(); a = time.perf_counter()
            binding.expand(dd, parents, P, K, T, seed, outputs=outs, workspace=ws_e, sampler=sampler)
            torch.cuda.synchronize(); b = time.perf_counter()
            binding.build_tree(dd, anchors, thetas, N, K, T, seed, workspace=ws_b, tree=tree, sampler=sampler,
                               device_tree=dtree)
            binding.tree_mask(dtree.parent, dtree.n, N + 1, out=mask_out)
            torch.cuda.synchronize()
            c = time.perf_counter()
            binding.verify(dd, tree, tgt, T, seed, workspace=ws_v)
            torch.cuda.synchronize(); e = time.perf_counter()
            te += b - a; tb += c - b; tv += e - c
        phases = {"expand": te / 3e-3, "build_tree_and_mask": tb / 3e-3, "verify": tv / 3e-3}

    # algorithmic bytes of the streaming pass: U rows touched once, W2 once, E rows
    rows = len(set(zip(fr["request"].tolist(), fr["depth"].tolist())))
    alg_bytes = rows * dr.V * 2 + dr.V * dr.r * 2 + P * dr.r * 2
    eval_s = float(eval_ms.mean()) / 1e3
    achieved = alg_bytes / eval_s / 1e9
    # algorithmic VALU work per (parent, token) element, in full-rate issue
    # slots: a running max, and per temperature one FMA (scale and shift), one
    # exp2 (TRANS_WEIGHT slots) and one add; two temperatures when T != 0, 1
    n_temps = 2 if (T > 0 and T != 1.0) else 1
    slots_per_elem = 1 + n_temps * (2 + TRANS_WEIGHT)
    alg_ops = slots_per_elem * P * dr.V
    achieved_ops = alg_ops / eval_s / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if (tr.get("kernel_source_hash") == kernel_source_hash() and abs(tr.get("T", -1) - T) < 1e-9
                and tr.get("sampler") == args.sampler):
            traffic = tr.get("bytes_per_launch")
    evals_step = P + (0 if args.expand_only else tree_evals)
    result = {
        "metric": METRIC,
        "value": evals_step / (ms_step / 1e3),
        "unit": "node-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w["name"].replace("-T0.7", f"-T{T:g}") + (": ts_expand over the 2048-parent frontier" if args.expand_only else
                                            ": 2048-parent ts_expand + best-first trees + tree masks + "
                                            f"T={T:g} verification"),
                   "V": dr.V, "D": dr.D, "r": dr.r, "requests": dr.R, "frontier_parents": P, "K": K,
                   "T": T, "N": N, "sampler": sampler,
                   "tree_evals_per_step": 0 if args.expand_only else tree_evals},
        "roofline": None,
        "expand_ms": {"eval": float(eval_ms.mean()), "merge": float(merge_ms.mean()),
                      "eval_p10": float(np.percentile(eval_ms, 10)), "eval_p90": float(np.percentile(eval_ms, 90))},
        "expand_node_evals_per_s": P / ((eval_ms.mean() + merge_ms.mean()) / 1e3),
        "phases_ms": phases,
    }
    kernel = EVAL_KERNEL + " (streaming pass of ts_expand)"
    hbm = {"bound": "hbm", "kernel": kernel, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "alg_bytes_per_launch": alg_bytes,
           "avg_launch_ms": float(eval_ms.mean())}
    alu = {"bound": "alu", "kernel": kernel, "achieved": achieved_ops, "peak": VALU_PEAK_TOPS,
           "unit": "T VALU slots/s", "frac": achieved_ops / VALU_PEAK_TOPS, "traffic": traffic,
           "alg_slots_per_launch": alg_ops, "slots_per_element": slots_per_elem,
           "avg_launch_ms": float(eval_ms.mean())}
    # the binding roofline is the one with the longer floor, i.e. the larger fraction
    result["roofline"] = alu if alu["frac"] > hbm["frac"] else hbm
    result["roofline_other"] = hbm if alu["frac"] > hbm["frac"] else alu
    # release every HIP object this process made before exit: the events, the library's pinned
    # staging buffer and events (the GPU work is finished)
    torch.cuda.synchronize()
    ev.close()
    binding.release_thread_state()
    if not args.no_cpu:
        log("timing the CPU oracle")
        result["cpu_baseline"] = cpu_baseline(dr, fr, K, T, seed, args.cpu_seconds, sampler)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
