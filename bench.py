#!/usr/bin/env python3
"""Benchmark of the TreeSpark draft-tree step on one MI355X.

Headline workload (the batched-serving case at V=151936): 64 requests, D=16,
r=64, bf16 inputs, K=8, T=0.7, per-request theta drawn from {0.02, 0.05, 0.1,
0.2}, synthetic inputs (paper_2609_22098_amd/synth.py).  One step is one pass
of the whole hot path over that batch:
  1. ts_expand over the 2048-parent serving frontier (2 parents at every depth
     of every request): conditional logits on MFMA, log-sum-exp, top-k, k
     draws without replacement (sequential sampler by default), child scoring;
  2. ts_build_tree: best-first trees for the 64 requests under their theta
     (waves on the device; the trees come back to the host and stay on the
     device);
  3. ts_tree_mask: the trees' attention masks and position ids for the
     target's verification pass, from the device copy of the trees;
  4. ts_verify: recursive-rejection verification of those trees at T=0.7.
value = node evaluations (frontier parents + tree-building parents) per second
over the step.  roofline: the dominant kernel (the streaming pass of
ts_expand), timed with HIP events on its stream over the timed steps, against
the HBM peak (algorithmic bytes per launch / mean launch time); the same
launches against the VALU issue peak are in roofline_alu.

configs: the other workloads' measured units (expansion, tree building,
verification; the high-load chain's per-wave cost) and the serving frontier
at T=0 and with the Gumbel sampler, each expansion with its own HBM fraction.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu] [--no-configs]
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "parent-conditioned node evals/sec at V=151936 + achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
# VALU issue peak for unpacked fp32 instructions: 256 CUs x 4 SIMDs x 16 lanes
# per cycle x 2.4 GHz (a wave64 instruction every 4 cycles; the 157.3 TFLOP/s
# fp32 vector figure needs packed FMAs, 2 per lane, counted as 2 FLOP each).
# Transcendentals (v_exp_f32, v_log_f32) take two issue slots (the counters of
# the streaming pass give 4 cycles per plain and 8 per transcendental wave64
# instruction).
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
TRANS_WEIGHT = 2
KERNEL_SOURCES = ("paper_2609_22098_amd/csrc/expand_kernels.hpp",
                  "paper_2609_22098_amd/csrc/device_common.hpp",
                  # its translation unit and the build's per-unit compiler flags
                  "paper_2609_22098_amd/csrc/expand_eval_bf16_ks2.hip",
                  "__graft_entry__.py")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "expand_eval_serving_counters.json")
EVAL_KERNEL = "expand_eval_lds_kernel"
EVAL_FRONTIER = "expand_eval_lds_kernel<2, 2,"  # rank 64 (KS = 2), two parent blocks per wave


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence (hip_runtime_api.h)


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (same process-wide runtime).  They
    only time kernels (the device is synchronised before they are read), so they are created
    without the system-scope fence: a fenced event between two dependent kernels holds the
    second back by ~5.7 us on MI355X (cache write-back and invalidation)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            rc = self.hip.hipEventCreateWithFlags(ctypes.byref(h), HIP_EVENT_DISABLE_SYSTEM_FENCE)
            assert rc == 0, f"hipEventCreateWithFlags failed ({rc})"
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


def stats_ms(a):
    a = np.asarray(a, dtype=np.float64)
    return {"mean": float(a.mean()), "median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "n": int(a.size)}


def host_cpu():
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count()


# ---------------------------------------------------------------- counters

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


def _frontier_mean(run_dir, counter):
    """Mean of a counter over the serving frontier's launches: two parent blocks per wave, rank
    64 (the tree waves' launches take one), the largest grid of that instantiation."""
    pairs = _counter_per_dispatch(run_dir, counter, EVAL_FRONTIER)
    g = max(p[0] for p in pairs)
    vals = [v for gk, v in pairs if gk == g]
    return float(np.mean(vals)), len(vals)


def write_counters(root, T, sampler):
    """Counters of the serving frontier's streaming pass from rocprofv3 --pmc runs under root:
    fetch (FETCH_SIZE), write (WRITE_SIZE), copy_fetch / copy_write (the same counters for a plain
    copy of known size, which scales them), valu (SQ_INSTS_VALU, SQ_INSTS_VALU_TRANS_F32,
    SQ_INSTS_MFMA), busy (SQ_VALU_MFMA_BUSY_CYCLES, SQ_BUSY_CU_CYCLES)."""
    with open(os.path.join(root, "copy_fetch", "copy.json")) as f:
        copy_bytes = json.load(f)["copy_bytes"]
    scale = {}
    for counter, sub in (("FETCH_SIZE", "copy_fetch"), ("WRITE_SIZE", "copy_write")):
        vals = _counter_per_dispatch(os.path.join(root, sub), counter, "")
        kib = max(v for _, v in vals)  # the copy is by far the largest dispatch of its run
        scale[counter] = copy_bytes / (kib * 1024.0)
    fetch, nf = _frontier_mean(os.path.join(root, "fetch"), "FETCH_SIZE")
    write, nw = _frontier_mean(os.path.join(root, "write"), "WRITE_SIZE")
    fb = fetch * 1024.0 * scale["FETCH_SIZE"]
    wb = write * 1024.0 * scale["WRITE_SIZE"]
    rec = {"kernel": EVAL_KERNEL, "T": T, "sampler": sampler, "kernel_source_hash": kernel_source_hash(),
           "fetch_kib_per_dispatch": fetch, "write_kib_per_dispatch": write, "dispatches": [nf, nw],
           "copy_bytes": copy_bytes, "copy_scale": scale, "fetch_bytes": fb, "write_bytes": wb,
           "bytes_per_launch": fb + wb}
    if os.path.isdir(os.path.join(root, "valu")):
        for c in ("SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_MFMA", "SQ_WAVES"):
            rec[c] = _frontier_mean(os.path.join(root, "valu"), c)[0]
    if os.path.isdir(os.path.join(root, "busy")):
        mb = _frontier_mean(os.path.join(root, "busy"), "SQ_VALU_MFMA_BUSY_CYCLES")[0]
        cb = _frontier_mean(os.path.join(root, "busy"), "SQ_BUSY_CU_CYCLES")[0]
        rec["SQ_VALU_MFMA_BUSY_CYCLES"], rec["SQ_BUSY_CU_CYCLES"] = mb, cb
        # the MFMA busy cycles are summed over the SIMDs (16 cycles per 16x16x32 bf16
        # MFMA), the busy cycles over the CUs: four SIMDs per CU
        rec["mfma_busy"] = mb / (4.0 * cb) if cb > 0 else None
    with open(COUNTERS_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def load_counters(T, sampler):
    """The counters record if it was taken on the current streaming-pass sources, else None."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    with open(COUNTERS_FILE) as f:
        rec = json.load(f)
    if (rec.get("kernel_source_hash") == kernel_source_hash() and abs(rec.get("T", -1) - T) < 1e-9
            and rec.get("sampler") == sampler):
        return rec
    return None


# ---------------------------------------------------------------- measurement helpers

def alg_bytes(dr, fr):
    """Algorithmic bytes of one streaming pass: the U rows the frontier touches (once), W2 once,
    the parents' E rows."""
    rows = len(set(zip(fr["request"].tolist(), fr["depth"].tolist())))
    esz = 2 if dr.dtype == "bf16" else 4
    return rows * dr.V * esz + dr.V * dr.r * esz + len(fr["token"]) * dr.r * esz


def copies_for(bytes_per_launch, floor=600e6):
    """Input copies to rotate so that consecutive launches cannot be served from the 256 MB
    Infinity Cache: at least floor bytes between two uses of one copy."""
    return max(2, int(np.ceil(floor / max(bytes_per_launch, 1.0))))


def drafter_copies(binding, dd, n):
    out = [dd]
    for _ in range(n - 1):
        out.append(binding.DeviceDrafter(dd.U.clone(), dd.E.clone(), dd.W2.clone()))
    return out


def time_expand(binding, drafters, parents, P, K, T, seed, sampler, reps, warmup, stream):
    """HIP-event durations (ms) of the streaming pass and the merge over reps launches, rotating
    the drafter copies."""
    import torch
    outs = binding.expand(drafters[0], parents, P, K, T, seed, sampler=sampler, stream=stream)
    ws = outs.pop("_workspace")
    ev = HipEvents(3 * (reps + warmup))
    for i in range(reps + warmup):
        binding.expand(drafters[i % len(drafters)], parents, P, K, T, seed, outputs=outs, workspace=ws,
                       events=ev.address(3 * i), sampler=sampler, stream=stream)
    torch.cuda.synchronize()
    ev_ms = [ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(warmup, reps + warmup)]
    mg_ms = [ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(warmup, reps + warmup)]
    diag = int(outs["diag"].sum().item())
    ev.close()
    assert diag == 0, "recomputed candidate runs differ from the streaming pass"
    return ev_ms, mg_ms


def expand_record(dr, fr, ev_ms, mg_ms):
    ab = alg_bytes(dr, fr)
    e, m = stats_ms(ev_ms), stats_ms(mg_ms)
    P = len(fr["token"])
    gbs = ab / (e["mean"] / 1e3) / 1e9
    return {"parents": P, "streaming_pass_ms": e, "merge_ms": m,
            "node_evals_per_s": P / ((e["mean"] + m["mean"]) / 1e3),
            "hbm": {"achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                    "alg_bytes_per_launch": ab}}


def wall_ms(fn, reps, warmup=3):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t = []
    for _ in range(reps):
        a = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        t.append((time.perf_counter() - a) * 1e3)
    return stats_ms(t)


def target_for(binding, synth, dr, tree, sigma, seed=0):
    """Target logits for a tree (row i = U[q][min(depth_i, D-1)] + N(0, sigma^2)), device."""
    import torch
    R, cap = tree.R, tree.cap
    tgt = torch.zeros((R, cap, dr.V), dtype=torch.bfloat16, device="cuda")
    for q in range(R):
        n1 = int(tree.n[q]) + 1
        s, _ = synth.make_target_rows(dr, q, tree.depth[q, :n1], sigma, seed=seed)
        tgt[q, :n1] = torch.from_numpy(s).view(torch.bfloat16).cuda()
    return tgt


# ---------------------------------------------------------------- the other workloads

def single_request_config(binding, synth, i, T, sampler, stream):
    """Workloads 1 and 2: one request; ts_expand on the constructed frontier, the whole tree
    build (fixed budget), and its verification."""
    w = synth.WORKLOADS[i]
    dr = synth.make_workload_drafter(i, seed=0)
    fr = synth.make_frontier(dr, per_depth=w["frontier_per_depth"], seed=0)
    dd = binding.drafter_from_host(dr)
    drafters = drafter_copies(binding, dd, copies_for(alg_bytes(dr, fr)))
    P = len(fr["token"])
    parents = binding.parents_to_device(fr["token"], fr["depth"], fr["request"], fr["log_surv"], fr["path"])
    K, N = w["K"], w["N"]
    ev_ms, mg_ms = time_expand(binding, drafters, parents, P, K, T, 0, sampler, 100, 10, stream)
    rec = {"workload": w["name"], "T": T, "sampler": sampler if T > 0 else None, "K": K, "N": N,
           "expand": expand_record(dr, fr, ev_ms, mg_ms), "input_copies_rotated": len(drafters)}
    anchors, _, _ = synth.make_controls(1, dr.V, 0.0, seed=0)
    thetas = np.zeros(1, np.float32)
    ws_b = binding.torch_empty_bytes(binding.build_tree_workspace_size(dd, N, K, T))
    tree = binding.build_tree(dd, anchors, thetas, N, K, T, 0, workspace=ws_b, sampler=sampler)
    evals = int(tree.evals.sum())
    bt = wall_ms(lambda: binding.build_tree(dd, anchors, thetas, N, K, T, 0, workspace=ws_b, tree=tree,
                                            sampler=sampler, stream=stream), 20)
    tgt = target_for(binding, synth, dr, tree, w["target_sigma"])
    ws_v = binding.torch_empty_bytes(binding.verify_workspace_size(dd, N + 1, T))
    out = (np.zeros((1, binding.TS_MAX_D), np.int32), np.zeros(1, np.int32), np.zeros(1, np.int32))
    vt = wall_ms(lambda: binding.verify(dd, tree, tgt, T, 0, workspace=ws_v, stream=stream, out=out), 20)
    rec["build_tree"] = {"ms": bt, "tree_nodes": int(tree.n[0]), "evaluations": evals,
                         "node_evals_per_s": evals / (bt["median"] / 1e3)}
    rec["verify"] = {"ms": vt, "accepted_length": int(out[1][0])}
    rec["round_ms"] = bt["median"] + vt["median"]
    return rec


def chain_config(binding, synth, stream):
    """Workload 4: 256 requests, r=128.  One expansion wave (one parent per request at one depth,
    the depth rotating over launches) at T=0 and T=1; the chain (K=1, theta=0, N=D: 16 sequential
    waves of 256 parents) and the natural trees of the theta sweep, at T=0 and T=1."""
    import torch
    w = synth.WORKLOADS[4]
    dr = synth.make_workload_drafter(4, seed=0)
    dd = binding.drafter_from_host(dr)
    R, D, V = dr.R, dr.D, dr.V
    rng = np.random.default_rng(5)
    fr = {"token": rng.integers(0, V, R).astype(np.int32), "depth": np.zeros(R, np.int32),
          "request": np.arange(R, dtype=np.int32), "log_surv": np.zeros(R, np.float32),
          "path": np.zeros(R, np.uint64)}
    ab = alg_bytes(dr, fr)
    # rotate the depth (different U rows) and copies of E and W2
    ncopy = copies_for(dr.V * dr.r * 4)
    ew = [(dd.E, dd.W2)] + [(dd.E.clone(), dd.W2.clone()) for _ in range(ncopy - 1)]
    drafters = [binding.DeviceDrafter(dd.U, e, w2) for e, w2 in ew]
    parents = []
    for d in range(D):
        f = dict(fr)
        f["depth"] = np.full(R, d, np.int32)
        parents.append(binding.parents_to_device(f["token"], f["depth"], f["request"], f["log_surv"], f["path"]))
    rec = {"workload": w["name"], "K": w["K"], "N": w["N"], "waves": {}, "chain": {}, "natural_trees": {}}
    for T in (0.0, 1.0):
        outs = binding.expand(drafters[0], parents[0], R, w["K"], T, 0, sampler="sequential", stream=stream)
        ws = outs.pop("_workspace")
        n, warm = 64, 8
        ev = HipEvents(3 * (n + warm))
        for i in range(n + warm):
            binding.expand(drafters[i % len(drafters)], parents[i % D], R, w["K"], T, 0, outputs=outs,
                           workspace=ws, events=ev.address(3 * i), sampler="sequential", stream=stream)
        torch.cuda.synchronize()
        ev_ms = [ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(warm, n + warm)]
        mg_ms = [ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(warm, n + warm)]
        ev.close()
        rec["waves"][f"T{T:g}"] = expand_record(dr, fr, ev_ms, mg_ms)
        anchors, thetas, _ = synth.make_controls(R, V, w["theta"], seed=0)
        # the chain: K = 1, no stop, one node per depth
        ws_c = binding.torch_empty_bytes(binding.build_tree_workspace_size(dd, D, 1, T))
        zero = np.zeros(R, np.float32)
        ch = binding.build_tree(dd, anchors, zero, D, 1, T, 0, workspace=ws_c, sampler="sequential")
        ct = wall_ms(lambda: binding.build_tree(dd, anchors, zero, D, 1, T, 0, workspace=ws_c, tree=ch,
                                                sampler="sequential", stream=stream), 10)
        rec["chain"][f"T{T:g}"] = {"ms": ct, "waves": D, "ms_per_wave": ct["median"] / D,
                                   "evaluations": int(ch.evals.sum()),
                                   "node_evals_per_s": int(ch.evals.sum()) / (ct["median"] / 1e3)}
        ws_n = binding.torch_empty_bytes(binding.build_tree_workspace_size(dd, w["N"], w["K"], T))
        nt = binding.build_tree(dd, anchors, thetas, w["N"], w["K"], T, 0, workspace=ws_n, sampler="sequential")
        tt = wall_ms(lambda: binding.build_tree(dd, anchors, thetas, w["N"], w["K"], T, 0, workspace=ws_n,
                                                tree=nt, sampler="sequential", stream=stream), 10)
        sizes = nt.n.astype(int)
        rec["natural_trees"][f"T{T:g}"] = {
            "ms": tt, "evaluations": int(nt.evals.sum()), "tree_nodes_total": int(sizes.sum()),
            "tree_nodes_low_theta_quarter": float(sizes[: R // 4].mean()),
            "tree_nodes_high_theta_quarter": float(sizes[-R // 4:].mean()),
            "node_evals_per_s": int(nt.evals.sum()) / (tt["median"] / 1e3)}
    rec["waves_alg_bytes_note"] = "per wave: 256 U rows (one depth) + W2 + 256 E rows"
    return rec


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
    model, nproc = host_cpu()
    return {"value": n / el, "unit": "node-evals/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of the 2048 frontier parents at T={T} (full-vocabulary fp64 "
                      f"evaluation with {sampler} draws, one thread), {el:.1f} s",
            "cpu_model": model, "nproc": nproc}


# ---------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads")
    ap.add_argument("--expand-only", action="store_true", help="time only ts_expand (profiling runs)")
    ap.add_argument("--T", type=float, default=0.7, help="temperature (the workload uses 0.7)")
    ap.add_argument("--sampler", default="sequential", choices=("sequential", "gumbel"),
                    help="realisation of the sibling draws at T > 0")
    ap.add_argument("--copy-gib", type=float, default=0.0, help="run only the copy calibration")
    ap.add_argument("--copy-out", default="", help="directory for the copy calibration record")
    ap.add_argument("--only", default="", choices=("", "serving_T0", "serving_gumbel", "single_v128256_T0",
                                                      "single_v151936_r256_T1", "chain_256req"),
                    help="run only this entry of configs and print its record (profiling runs)")
    ap.add_argument("--counters-from", default="",
                    help="directory holding the rocprofv3 --pmc runs (fetch, write, copy_fetch, "
                         "copy_write, valu, busy); writes the counters record and exits")
    args = ap.parse_args()
    if args.counters_from:
        write_counters(args.counters_from, args.T, args.sampler)
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

    stream = torch.cuda.current_stream()
    if args.only in ("single_v128256_T0", "single_v151936_r256_T1", "chain_256req"):
        if args.only == "single_v128256_T0":
            rec = single_request_config(binding, synth, 1, 0.0, "sequential", stream)
        elif args.only == "single_v151936_r256_T1":
            rec = single_request_config(binding, synth, 2, 1.0, "gumbel", stream)
        else:
            rec = chain_config(binding, synth, stream)
        torch.cuda.synchronize()
        binding.release_thread_state()
        print(json.dumps({args.only: rec}), flush=True)
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
    if args.only in ("serving_T0", "serving_gumbel"):
        Tx, sx = (0.0, sampler) if args.only == "serving_T0" else (T, "gumbel")
        e, m = time_expand(binding, drafters, parents, P, K, Tx, seed, sx, 100, 10, stream)
        torch.cuda.synchronize()
        binding.release_thread_state()
        print(json.dumps({args.only: expand_record(dr, fr, e, m)}), flush=True)
        return
    # a serving loop holds its stream and output buffers across rounds
    outs = binding.expand(dd, parents, P, K, T, seed, sampler=sampler, stream=stream)
    ws_e = outs.pop("_workspace")
    ws_b = binding.torch_empty_bytes(binding.build_tree_workspace_size(dd, N, K, T))
    ws_v = binding.torch_empty_bytes(binding.verify_workspace_size(dd, N + 1, T))
    tree = binding.build_tree(dd, anchors, thetas, N, K, T, seed, workspace=ws_b, sampler=sampler)
    tgt = target_for(binding, synth, dr, tree, w["target_sigma"])
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
    vout = (np.zeros((dr.R, binding.TS_MAX_D), np.int32), np.zeros(dr.R, np.int32), np.zeros(dr.R, np.int32))

    # The pass and the merge are timed with events on every other step: each
    # event is a stream marker that holds the next kernel back (~3.4 us per
    # step for the three), and 100 of 200 timed launches are enough for the
    # mean, median and percentiles.
    def timed_step(i):
        return (i - args.warmup) % 2 == 0  # the first timed step always has them

    def step(i):
        d = drafters[i % 2]
        binding.expand(d, parents, P, K, T, seed, outputs=outs, workspace=ws_e,
                       events=ev.address(3 * i) if timed_step(i) else None, sampler=sampler, stream=stream)
        if args.expand_only:
            return
        binding.build_tree(d, anchors, thetas, N, K, T, seed, workspace=ws_b, tree=tree, sampler=sampler,
                           device_tree=dtree, stream=stream)
        binding.tree_mask(dtree.parent, dtree.n, N + 1, out=mask_out, stream=stream)
        binding.verify(d, tree, tgt, T, seed, workspace=ws_v, stream=stream, out=vout)

    log(f"timing {args.steps} steps after {args.warmup} warm-up steps")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.warmup, nsteps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    eval_ms = [ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(args.warmup, nsteps) if timed_step(i)]
    merge_ms = [ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(args.warmup, nsteps) if timed_step(i)]
    assert int(outs["diag"].sum().item()) == 0
    ev.close()

    # phase breakdown from extra synchronised steps (outside the timed region):
    # the median of 20 per phase, each phase starting on an idle GPU
    phases = {}
    if not args.expand_only:
        pt = {"expand": [], "build_tree_and_mask": [], "verify": []}
        for i in range(20):
            d = drafters[i % 2]
            torch.cuda.synchronize(); a = time.perf_counter()
            binding.expand(d, parents, P, K, T, seed, outputs=outs, workspace=ws_e, sampler=sampler,
                           stream=stream)
            torch.cuda.synchronize(); b = time.perf_counter()
            binding.build_tree(d, anchors, thetas, N, K, T, seed, workspace=ws_b, tree=tree, sampler=sampler,
                               device_tree=dtree, stream=stream)
            binding.tree_mask(dtree.parent, dtree.n, N + 1, out=mask_out, stream=stream)
            torch.cuda.synchronize()
            c = time.perf_counter()
            binding.verify(d, tree, tgt, T, seed, workspace=ws_v, stream=stream, out=vout)
            torch.cuda.synchronize(); e = time.perf_counter()
            pt["expand"].append(b - a); pt["build_tree_and_mask"].append(c - b); pt["verify"].append(e - c)
        phases = {k: float(np.median(v)) * 1e3 for k, v in pt.items()}

    ab = alg_bytes(dr, fr)
    es = stats_ms(eval_ms)
    eval_s = es["mean"] / 1e3
    achieved = ab / eval_s / 1e9
    # algorithmic VALU work per (parent, token) element, in issue slots of one
    # unpacked instruction: a running max, and per temperature one FMA (scale
    # and shift), one exp2 (TRANS_WEIGHT slots) and one add; two temperatures
    # when T != 0, 1
    n_temps = 2 if (T > 0 and T != 1.0) else 1
    slots_per_elem = 1 + n_temps * (2 + TRANS_WEIGHT)
    alg_ops = slots_per_elem * P * dr.V
    achieved_ops = alg_ops / eval_s / 1e12
    ctr = load_counters(T, sampler)
    evals_step = P + (0 if args.expand_only else tree_evals)
    kernel = EVAL_KERNEL + " (streaming pass of ts_expand)"
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
        "config": {"workload": w["name"].replace("-T0.7", f"-T{T:g}") + (
                       ": ts_expand over the 2048-parent frontier" if args.expand_only else
                       ": 2048-parent ts_expand + best-first trees + tree masks + "
                       f"T={T:g} verification"),
                   "V": dr.V, "D": dr.D, "r": dr.r, "requests": dr.R, "frontier_parents": P, "K": K,
                   "T": T, "N": N, "sampler": sampler,
                   "tree_evals_per_step": 0 if args.expand_only else tree_evals},
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": ctr["bytes_per_launch"] if ctr else None,
                     "alg_bytes_per_launch": ab, "launch_ms": es},
        "roofline_alu": {"bound": "alu", "kernel": kernel, "achieved": achieved_ops, "peak": VALU_PEAK_TOPS,
                         "unit": "T VALU slots/s", "frac": achieved_ops / VALU_PEAK_TOPS,
                         "alg_slots_per_launch": alg_ops, "slots_per_element": slots_per_elem},
        "mfma_busy": ctr.get("mfma_busy") if ctr else None,
        "counters": ({k: ctr[k] for k in ("SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_MFMA")
                      if k in ctr} if ctr else None),
        "merge_ms": stats_ms(merge_ms),
        "expand_node_evals_per_s": P / ((es["mean"] + float(np.mean(merge_ms))) / 1e3),
        "phases_ms": phases,
    }
    if ctr and "SQ_INSTS_VALU" in ctr:
        result["counters"]["valu_instructions_per_element"] = ctr["SQ_INSTS_VALU"] * 64 / (P * dr.V)

    if not args.no_configs and not args.expand_only:
        cfg = {}
        log("serving frontier at T=0 and with Gumbel draws")
        ev0, mg0 = time_expand(binding, drafters, parents, P, K, 0.0, seed, sampler, 100, 10, stream)
        cfg["serving_T0"] = expand_record(dr, fr, ev0, mg0)
        evg, mgg = time_expand(binding, drafters, parents, P, K, T, seed, "gumbel", 50, 5, stream)
        cfg["serving_gumbel"] = expand_record(dr, fr, evg, mgg)
        cfg["serving_gumbel"]["T"] = T
        del dd2, drafters
        torch.cuda.empty_cache()
        log("workload 1 (V=128256, r=64, T=0)")
        cfg["single_v128256_T0"] = single_request_config(binding, synth, 1, 0.0, "sequential", stream)
        log("workload 2 (V=151936, r=256, T=1, Gumbel draws)")
        cfg["single_v151936_r256_T1"] = single_request_config(binding, synth, 2, 1.0, "gumbel", stream)
        torch.cuda.empty_cache()
        log("workload 4 (256 requests, r=128: waves, chains, natural trees)")
        cfg["chain_256req"] = chain_config(binding, synth, stream)
        result["configs"] = cfg

    # release every HIP object this process made before exit: the library's
    # pinned staging buffer and events (the GPU work is finished)
    torch.cuda.synchronize()
    binding.release_thread_state()
    if not args.no_cpu:
        log("timing the CPU oracle")
        result["cpu_baseline"] = cpu_baseline(dr, fr, K, T, seed, args.cpu_seconds, sampler)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
