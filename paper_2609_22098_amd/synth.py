"""Seeded synthetic inputs for the draft-tree step.

This module only draws random inputs: it holds none of the method's
arithmetic.  Both the HIP path and the CPU oracle consume what it returns, so
the two sides always see identical values.

Recipe (numpy PCG64 streams, draws in a fixed order within each stream):
  1. U [q][D][V] of request q comes from its own stream, keyed (seed, q):
     N(0, u_sigma^2) in fp64, depth-major; then, per depth in order, either
     one planted token (uniform over V) that gets +planted, or a fresh random
     permutation pi of the vocabulary where token pi[k-1] gets
     +zipf_scale * k^-zipf_exp.  Requests are drawn in parallel threads
     (independent streams, so the values do not depend on the thread count).
  2. E [V][r] then W2 [V][r] from the stream keyed (seed, 2^32 - 1):
     N(0, ew_sigma^2) in fp64 (E is shared by all requests, as is W2).
  3. Values are rounded fp64 -> fp32 (round to nearest even) and, for bf16
     inputs, fp32 -> bf16 (round to nearest even on the bit pattern).
Target logits, frontiers and per-request controls come from separate streams
(seed offsets below) so that adding them never changes the model tensors.
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field

import numpy as np

# Workloads stand in for the paper's drafter outputs (trained checkpoints and
# evaluation suites are not used); each one names its sizes and distributions.
WORKLOADS = {
    0: dict(name="tiny-v4096-d8-r16-f32", V=4096, D=8, r=16, dtype="f32", R=1, u_sigma=3.0,
            planted=8.0, zipf=None, ew_sigma=0.1, K=4, theta=0.05, N=32, temps=(0.0, 1.0),
            target_sigma=1.0),
    1: dict(name="single-v128256-d16-r64-bf16", V=128256, D=16, r=64, dtype="bf16", R=1,
            u_sigma=2.5, planted=None, zipf=(6.0, 1.1), ew_sigma=0.05, K=8, theta=0.0, N=64,
            temps=(0.0,), target_sigma=1.0, frontier_per_depth=4),
    2: dict(name="single-v151936-d16-r256-bf16-T1", V=151936, D=16, r=256, dtype="bf16", R=1,
            u_sigma=2.5, planted=None, zipf=(6.0, 1.1), ew_sigma=0.05, K=8, theta=0.0, N=128,
            temps=(1.0,), target_sigma=1.5, frontier_per_depth=8),
    3: dict(name="serving-64req-v151936-d16-r64-bf16-T0.7", V=151936, D=16, r=64, dtype="bf16",
            R=64, u_sigma=2.5, planted=None, zipf=(6.0, 1.1), ew_sigma=0.05, K=8,
            theta=("set", 0.02, 0.05, 0.1, 0.2), N=64, temps=(0.7,), target_sigma=1.0,
            frontier_per_depth=2),
    4: dict(name="chain-256req-v151936-d16-r128-bf16", V=151936, D=16, r=128, dtype="bf16", R=256,
            u_sigma=2.5, planted=None, zipf=(6.0, 1.1), ew_sigma=0.05, K=8, theta=("sweep", 0.01, 0.5),
            N=64, temps=(0.0, 1.0), target_sigma=1.0, frontier_per_depth=None),
}

_SEED_TARGET = 1_000_003
_SEED_FRONTIER = 2_000_003
_SEED_CONTROL = 3_000_017


def f32_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest even), returned as uint16 bit patterns."""
    # finite values stay below 0xFF800000 after the rounding increment, so
    # 32-bit arithmetic cannot wrap
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass
class Drafter:
    """Host copies of one synthetic drafter output.

    U, E, W2 hold the device dtype's storage (float32, or uint16 bf16 bit
    patterns); U32, E32, W2_32 hold the same values as float32 for the oracle.
    """
    R: int
    D: int
    V: int
    r: int
    dtype: str
    U: np.ndarray
    E: np.ndarray
    W2: np.ndarray
    U32: np.ndarray = field(repr=False, default=None)
    E32: np.ndarray = field(repr=False, default=None)
    W2_32: np.ndarray = field(repr=False, default=None)


def _store(x64: np.ndarray, dtype: str):
    x32 = x64.astype(np.float32)
    if dtype == "bf16":
        b = f32_to_bf16_bits(x32)
        return b, bf16_bits_to_f32(b)
    return x32, x32


_EW_STREAM = 2**32 - 1  # stream key of E and W2 (request streams use keys below 2^20)


def make_drafter(V, D, r, R=1, dtype="bf16", u_sigma=2.5, planted=None, zipf=(6.0, 1.1),
                 ew_sigma=0.05, seed=0, u_scale=1.0) -> Drafter:
    """Draw U [R][D][V], E [V][r], W2 [V][r] following the recipe in the module docstring.

    u_scale multiplies U after the boosts (a "sharp" variant for deep-tree tests).
    """
    from concurrent.futures import ThreadPoolExecutor
    U = np.empty((R, D, V), dtype=np.uint16 if dtype == "bf16" else np.float32)
    U32 = np.empty((R, D, V), dtype=np.float32)
    ranks = np.arange(1, V + 1, dtype=np.float64)
    boost = zipf[0] * ranks ** (-zipf[1]) if zipf is not None else None

    def request(q):
        rng = np.random.Generator(np.random.PCG64([seed, q]))
        base = rng.standard_normal((D, V)) * u_sigma
        for d in range(D):
            if planted is not None:
                t = rng.integers(0, V)
                base[d, t] += planted
            elif zipf is not None:
                perm = rng.permutation(V)
                base[d, perm] += boost
        base *= u_scale
        U[q], U32[q] = _store(base, dtype)

    workers = max(1, min(R, 16, os.cpu_count() or 1))
    if workers == 1:
        for q in range(R):
            request(q)
    else:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(request, range(R)))
    rng = np.random.Generator(np.random.PCG64([seed, _EW_STREAM]))
    E64 = rng.standard_normal((V, r)) * ew_sigma
    W64 = rng.standard_normal((V, r)) * ew_sigma
    E, E32 = _store(E64, dtype)
    W2, W2_32 = _store(W64, dtype)
    return Drafter(R, D, V, r, dtype, U, E, W2, U32, E32, W2_32)


def make_workload_drafter(i: int, seed: int = 0, R: int | None = None, u_scale: float = 1.0) -> Drafter:
    w = WORKLOADS[i]
    return make_drafter(w["V"], w["D"], w["r"], R=w["R"] if R is None else R, dtype=w["dtype"],
                        u_sigma=w["u_sigma"], planted=w["planted"], zipf=w["zipf"],
                        ew_sigma=w["ew_sigma"], seed=seed, u_scale=u_scale)


def make_target_rows(dr: Drafter, request: int, depths: np.ndarray, sigma: float, seed: int = 0,
                     dtype: str | None = None):
    """Target logits for a tree: row i = U[request][min(depth_i, D-1)] + N(0, sigma^2) noise.

    Returns (storage array [n][V], float32 values [n][V]).  The noise stream is
    keyed by (seed, request) and drawn row by row in node order.
    """
    rng = np.random.Generator(np.random.PCG64([seed + _SEED_TARGET, request]))
    depths = np.asarray(depths)
    rows = np.minimum(depths, dr.D - 1)
    x = dr.U32[request, rows].astype(np.float64) + rng.standard_normal((len(depths), dr.V)) * sigma
    return _store(x, dtype or dr.dtype)


def make_prefix_keyed_target(dr: Drafter, request: int, prefixes, sigma: float, seed: int = 0):
    """Target rows keyed by the token prefix of each node (identical prefixes -> identical rows).

    prefixes: list of tuples of tokens (the root's is the empty tuple).
    """
    out = np.empty((len(prefixes), dr.V), dtype=np.float64)
    for i, pre in enumerate(prefixes):
        key = [seed + _SEED_TARGET, request, len(pre)] + [int(t) for t in pre]
        rng = np.random.Generator(np.random.PCG64(key))
        out[i] = dr.U32[request, min(len(pre), dr.D - 1)] + rng.standard_normal(dr.V) * sigma
    return _store(out, dr.dtype)


def make_frontier(dr: Drafter, per_depth: int, seed: int = 0, requests=None):
    """A constructed frontier: per_depth parents at each depth 0..D-1 of every request.

    Parents are ordered by (request, depth).  Tokens are uniform over V; the
    path id of a depth-d parent has d random 4-bit digits (digits < 8); log S
    is uniform in [-4, 0] (0 at depth 0).
    Returns a dict of arrays: token, depth, request, path (uint64), log_surv (float32).
    """
    rng = np.random.Generator(np.random.PCG64(seed + _SEED_FRONTIER))
    reqs = range(dr.R) if requests is None else requests
    tok, dep, req, path, ls = [], [], [], [], []
    for q in reqs:
        for d in range(dr.D):
            for _ in range(per_depth):
                tok.append(int(rng.integers(0, dr.V)))
                dep.append(d)
                req.append(q)
                digits = rng.integers(0, 8, size=d)
                p = 0
                for lvl, dig in enumerate(digits):
                    p |= int(dig) << (4 * lvl)
                path.append(p)
                ls.append(0.0 if d == 0 else float(rng.uniform(-4.0, 0.0)))
    return dict(token=np.array(tok, np.int32), depth=np.array(dep, np.int32),
                request=np.array(req, np.int32), path=np.array(path, np.uint64),
                log_surv=np.array(ls, np.float32))


def make_controls(R: int, V: int, thetas, seed: int = 0):
    """Per-request anchors (uniform tokens), thetas and 64-bit seeds.

    thetas: a float (same for all), ("set", v1, v2, ...) drawn uniformly per
    request, or ("sweep", lo, hi) geometric from lo to hi over the requests.
    """
    rng = np.random.Generator(np.random.PCG64(seed + _SEED_CONTROL))
    anchors = rng.integers(0, V, size=R).astype(np.int32)
    if np.isscalar(thetas):
        th = np.full(R, float(thetas))
    elif thetas[0] == "set":
        th = rng.choice(np.asarray(thetas[1:], dtype=np.float64), size=R)
    elif thetas[0] == "sweep":
        th = np.geomspace(thetas[1], thetas[2], R)
    else:
        raise ValueError(f"unknown theta spec {thetas!r}")
    seeds = rng.integers(0, 2**63 - 1, size=R, dtype=np.int64).astype(np.uint64)
    return anchors, th.astype(np.float32), seeds
