"""Comparison helpers: GPU results against the oracle, with near-tie accounting.

Parity rules for the outputs of the method:
  - token ids, tree topology and accepted paths are bit-exact wherever the
    oracle's competing scores differ by more than TIE * max(1, |score|);
    positions after the first near-tie are not compared, and near-ties are
    counted;
  - log-probabilities and survival values agree within 1e-5 relative
    (fp32 inputs) or 2e-3 (bf16 inputs), relative to max(1, |x|).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from oracle import oracle as o

TIE = 1e-5


def value_tol(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 2e-3


def close(a, b, tol) -> bool:
    a, b = float(a), float(b)
    if math.isnan(b):
        return math.isnan(a)
    if math.isinf(b):
        return a == b
    return abs(a - b) <= tol * max(1.0, abs(b))


@dataclass
class Tally:
    compared: int = 0        # parents, trees or walks looked at
    near_ties: int = 0       # of those, how many hit a near-tie (compared only up to it)
    units: int = 0           # tree nodes or walk levels that exist on the oracle's side
    units_compared: int = 0  # of those, how many were compared
    max_err: float = 0.0
    failures: list = field(default_factory=list)

    def err(self, a, b):
        a, b = float(a), float(b)
        if math.isfinite(b):
            self.max_err = max(self.max_err, abs(a - b) / max(1.0, abs(b)))

    def check(self, ok, msg):
        if not ok:
            self.failures.append(msg)


def first_tie(vals, upto):
    """Index of the first i < upto with vals[i] - vals[i+1] <= TIE*max(1,|vals[i]|), else upto."""
    for i in range(upto):
        if not np.isfinite(vals[i + 1]):
            continue
        if vals[i] - vals[i + 1] <= TIE * max(1.0, abs(vals[i])):
            return i
    return upto


def first_draw_tie(gaps, K, T):
    """Sequential draws: index of the first draw whose picks came within TIE * max(1, 1/T) of a
    cumulative boundary (relative to the level's total).  A pick compares masses exp(z / T), so an
    fp32 rounding error dz in a logit moves a mass by about dz / T relative; the threshold scales
    with 1/T for that reason."""
    thr = TIE * max(1.0, 1.0 / T)
    for j in range(K):
        if gaps[j] <= thr:
            return j
    return K


def compare_parent(gpu: dict, i: int, ev: o.Eval, log_surv_p: float, T: float, K: int, dtype: str,
                   tally: Tally, a=0.67, b=-0.46, tag="", sampler="gumbel"):
    """Compare ts_expand outputs of parent row i with the oracle evaluation ev."""
    tol = value_tol(dtype)
    tally.compared += 1
    tally.err(gpu["lse0"][i], ev.lse0)
    tally.check(close(gpu["lse0"][i], ev.lse0, tol), f"{tag} lse0 {gpu['lse0'][i]} vs {ev.lse0}")
    # greedy order pi
    t_pi = first_tie(ev.pi_z, K)
    if t_pi < K:
        tally.near_ties += 1
    tally.check(list(gpu["rank_token"][i][:t_pi]) == list(ev.pi[:t_pi]),
                f"{tag} rank tokens {list(gpu['rank_token'][i])} vs {list(ev.pi)} (first tie {t_pi})")
    for j in range(t_pi):
        lq = ev.pi_z[j] - ev.lse0
        tally.err(gpu["rank_log_q0"][i][j], lq)
        tally.check(close(gpu["rank_log_q0"][i][j], lq, tol), f"{tag} rank log q0[{j}]")
    if T == 0:
        upto = t_pi
        for j in range(upto):
            lq = ev.pi_z[j] - ev.lse0
            ls = log_surv_p + o.log_phat(lq, a, b)
            tally.check(gpu["child_token"][i][j] == ev.pi[j], f"{tag} child token {j}")
            for name, want in (("child_log_q0", lq), ("child_log_surv", ls), ("slot_key", ls)):
                tally.err(gpu[name][i][j], want)
                tally.check(close(gpu[name][i][j], want, tol), f"{tag} {name}[{j}] {gpu[name][i][j]} vs {want}")
        return
    tally.err(gpu["lseT"][i], ev.lseT)
    tally.check(close(gpu["lseT"][i], ev.lseT, tol), f"{tag} lseT {gpu['lseT'][i]} vs {ev.lseT}")
    t_sig = first_draw_tie(ev.sigma_g, K, T) if sampler == "sequential" else first_tie(ev.sigma_g, K)
    if t_sig < K:
        tally.near_ties += 1
    tally.check(list(gpu["child_token"][i][:t_sig]) == list(ev.sigma[:t_sig]),
                f"{tag} drawn tokens {list(gpu['child_token'][i])} vs {list(ev.sigma)} (first tie {t_sig})")
    for j in range(t_sig):
        lq = ev.sigma_z[j] - ev.lse0
        lqT = ev.sigma_z[j] / T - ev.lseT
        ls = log_surv_p + o.log_phat(lq, a, b)
        bound = next(k for k in range(K) if ev.pi[k] not in list(ev.sigma[:j]))
        key = log_surv_p + o.log_phat(ev.pi_z[bound] - ev.lse0, a, b)
        for name, want in (("child_log_q0", lq), ("child_log_qT", lqT), ("child_log_surv", ls),
                           ("slot_key", key)):
            tally.err(gpu[name][i][j], want)
            tally.check(close(gpu[name][i][j], want, tol), f"{tag} {name}[{j}] {gpu[name][i][j]} vs {want}")


def tree_compare_limit(ref: o.Tree, theta: float, T: float = 1.0):
    """Number of leading nodes of the oracle tree that no near-tie can change, and the tie count.
    Score gaps of an evaluation (top-k logits, Gumbel keys) use TIE; the picks of sequential
    draws, whose gaps are relative masses, use TIE * max(1, 1/T) (see first_draw_tie)."""
    draw_thr = TIE * max(1.0, 1.0 / T) if T > 0 else TIE
    lt = math.log(theta) if theta > 0 else -math.inf
    limit = ref.n + 1
    ties = 0
    for c in range(1, ref.n + 1):
        tied = False
        if ref.margin[c] <= TIE * max(1.0, abs(ref.key[c])):
            tied = True
        p = ref.parent[c]
        if np.isfinite(ref.eval_gap[p]) and ref.eval_gap[p] <= TIE:
            tied = True
        if np.isfinite(ref.draw_gap[p]) and ref.draw_gap[p] <= draw_thr:
            tied = True
        if math.isfinite(lt) and abs(ref.key[c] - lt) <= TIE * max(1.0, abs(lt)):
            tied = True
        if tied:
            ties += 1
            limit = min(limit, c)
    if math.isfinite(lt) and np.isfinite(ref.stop_key) and abs(ref.stop_key - lt) <= TIE * max(1.0, abs(lt)):
        ties += 1
    return limit, ties


def compare_tree(gpu_tree, q: int, ref: o.Tree, theta: float, dtype: str, tally: Tally, tag="", T=1.0):
    tol = value_tol(dtype)
    limit, ties = tree_compare_limit(ref, theta, T)
    tally.near_ties += ties
    tally.compared += 1
    n = int(gpu_tree.n[q])
    if ties == 0:
        tally.check(n == ref.n, f"{tag} tree size {n} vs {ref.n}")
    upto = min(limit, n + 1, ref.n + 1)
    tally.units += ref.n
    tally.units_compared += max(0, min(limit, ref.n + 1) - 1)
    for name in ("token", "parent", "depth", "rank"):
        g = list(getattr(gpu_tree, name)[q][:upto])
        r = list(getattr(ref, name)[:upto])
        tally.check(g == r, f"{tag} {name} {g} vs {r}")
    tally.check([int(x) for x in gpu_tree.path[q][:upto]] == [int(x) for x in ref.path[:upto]], f"{tag} path")
    for name in ("log_surv", "log_q0", "key"):
        for c in range(1, upto):
            want = getattr(ref, name)[c]
            got = getattr(gpu_tree, name)[q][c]
            tally.err(got, want)
            tally.check(close(got, want, tol), f"{tag} {name}[{c}] {got} vs {want}")
    return upto


def oracle_tree(tree, q: int) -> o.Tree:
    """The oracle's view of request q of a HostTree (for the verification walks)."""
    n1 = int(tree.n[q]) + 1
    return o.Tree(int(tree.n[q]), 0, tree.token[q, :n1].copy(), tree.parent[q, :n1].copy(),
                  tree.depth[q, :n1].copy(), tree.rank[q, :n1].copy(), tree.path[q, :n1].copy(),
                  tree.log_surv[q, :n1].astype(np.float64), tree.log_q0[q, :n1].astype(np.float64),
                  tree.log_qT[q, :n1].astype(np.float64), tree.key[q, :n1].astype(np.float64),
                  np.zeros(n1), np.zeros(n1), np.zeros(n1), float("nan"))


def compare_walk(path, plen, bonus, ref_path, ref_bonus, margins, tally: Tally, tag=""):
    """One verification walk (accepted node ids and bonus token) against the oracle's.
    margins[i] is the oracle's smallest relative margin of the decisions taken at the i-th node
    of its walk.  The nodes accepted before the first level whose margin is <= TIE must be
    identical; without a near-tie the whole walk and the bonus must be.  Returns True if the
    walk was compared whole."""
    levels = len(margins)
    tie = next((i for i, m in enumerate(margins) if m <= TIE), levels)
    tally.compared += 1
    tally.units += levels
    tally.units_compared += tie
    if tie < levels:
        tally.near_ties += 1
        upto = min(tie, len(ref_path))
        tally.check(int(plen) >= upto and list(path[:upto]) == list(ref_path[:upto]),
                    f"{tag} walk {list(path[:plen])} vs {list(ref_path)} (near-tie at level {tie})")
        return False
    tally.check(int(plen) == len(ref_path) and list(path[:plen]) == list(ref_path),
                f"{tag} walk {list(path[:plen])} vs {list(ref_path)}")
    tally.check(int(bonus) == int(ref_bonus), f"{tag} bonus {int(bonus)} vs {int(ref_bonus)}")
    return True


# Near-tie accounting of every parity comparison in this session, written out by conftest.py at
# the end (the parity bar counts and reports near-ties).
RECORDS: list = []


def record(test: str, what: str, tally: Tally):
    RECORDS.append(dict(test=test, what=what, compared=tally.compared, near_ties=tally.near_ties,
                        units=tally.units, units_compared=tally.units_compared,
                        max_rel_err=tally.max_err, failures=len(tally.failures)))
