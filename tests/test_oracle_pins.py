"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: published
known-answer values, closed forms, special cases that reduce to a textbook
routine, brute-force enumeration on tiny inputs, and distributional theorems
(chi-square over >= 1e5 seeds).  Nothing here needs a GPU.
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy import special, stats

from oracle import oracle as o
from paper_2609_22098_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
A, B = 0.67, -0.46


def _tiny_model(V=6, D=3, r=4, seed=0, u_sigma=1.0, ew_sigma=0.6, R=1):
    dr = synth.make_drafter(V, D, r, R=R, dtype="f32", u_sigma=u_sigma, planted=None, zipf=None,
                            ew_sigma=ew_sigma, seed=seed)
    return dr, o.Model(dr.U32, dr.E32, dr.W2_32)


def _golden_calibration():
    vals = {}
    with open(os.path.join(GOLDEN, "calibration.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    return vals


# ---------------------------------------------------------------- randomness

def test_philox_known_answers():
    """Philox4x32-10 reproduces the published known-answer vectors."""
    n = 0
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            w = [int(x, 16) for x in line.split()]
            got = o.philox4x32_10(w[0:4], w[4:6])
            assert list(got) == w[6:10]
            n += 1
    assert n == 3


def test_uniform_counter_layout_and_range():
    """u_token/u_stage read the documented counter words, and u lies strictly in (0, 1)."""
    seed = 0x0123456789ABCDEF
    req, depth, path = 5, 3, 0x321
    for y in (0, 1, 2, 3, 4, 77, 4095):
        ctr = [y >> 2, path & 0xFFFFFFFF, path >> 32, (req << 12) | (depth << 4) | o.TAG_EXPAND]
        w = o.philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32])[y & 3]
        assert o.u_token(seed, req, depth, path, o.TAG_EXPAND, y) == ((int(w) >> 9) + 0.5) / 2**23
    for j in (1, 2, 7):
        ctr = [j, path & 0xFFFFFFFF, path >> 32, (req << 12) | (depth << 4) | o.TAG_ACCEPT]
        w = o.philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32])[0]
        assert o.u_stage(seed, req, depth, path, o.TAG_ACCEPT, j) == ((int(w) >> 9) + 0.5) / 2**23
    us = np.array([o.u_token(7, 0, 0, 0, 1, y) for y in range(20000)])
    assert us.min() > 0.0 and us.max() < 1.0
    # every value is exact in fp32 (24 significant bits), including the extremes
    assert np.all(us.astype(np.float32).astype(np.float64) == us)
    for w in (0, 0xFFFFFFFF, 0x80000000, 0x7FFFFFFF):
        u = ((w >> 9) + 0.5) / 2**23
        assert 0.0 < u < 1.0 and float(np.float32(u)) == u
    # uniformity of the mapped draws
    assert stats.kstest(us, "uniform").pvalue > 1e-3


# ---------------------------------------------------------------- calibration

def test_log_phat_closed_forms():
    """Eq. 3 at points where the logistic map has a closed form."""
    g = _golden_calibration()
    a, b = g["a"], g["b"]
    assert (a, b) == (A, B)
    # q0 = 1/2 -> logit 0 -> p-hat = sigmoid(b)
    assert o.log_phat(math.log(0.5), a, b) == pytest.approx(math.log(special.expit(b)), rel=1e-13)
    # a = 1, b = 0 -> p-hat = q0
    for q in (1e-9, 0.01, 0.3, 0.9, 0.999999):
        assert o.log_phat(math.log(q), 1.0, 0.0) == pytest.approx(math.log(q), rel=1e-10, abs=1e-14)
    # a = 0 -> p-hat = sigmoid(b) for every q0
    assert o.log_phat(math.log(0.01), 0.0, 1.5) == pytest.approx(math.log(special.expit(1.5)), rel=1e-13)
    # general points against the plain formula sigmoid(a*log(q/(1-q)) + b)
    for q in (1e-6, 0.02, 0.2, 0.5, 0.8, 0.99):
        ref = math.log(1.0 / (1.0 + math.exp(-(a * math.log(q / (1.0 - q)) + b))))
        assert o.log_phat(math.log(q), a, b) == pytest.approx(ref, rel=1e-11)
    # q0 = 1 -> p-hat = 1 for a > 0; q0 -> 0 -> -inf
    assert o.log_phat(0.0, a, b) == 0.0
    assert o.log_phat(-math.inf, a, b) == -math.inf
    # monotone in q0 (a > 0)
    lq = np.linspace(-30, -1e-9, 2000)
    vals = np.array([o.log_phat(x, a, b) for x in lq])
    assert np.all(np.diff(vals) >= 0)


def test_cost_accounting_matches_paper():
    """One node evaluation is a |V| x r matvec: 2 r V flops, about 80 MFLOP at the quoted sizes (§5.6)."""
    g = _golden_calibration()
    flops = 2 * g["cost_r"] * g["cost_V"]
    assert abs(flops / 1e6 - g["cost_mflop_approx"]) / g["cost_mflop_approx"] < 0.05


# ---------------------------------------------------------------- node evaluation

def test_eval_rows_normalise():
    """Softmax rows sum to one (Eq. 1), for q0 and for the temperature-scaled qT."""
    dr, m = _tiny_model(V=300, D=4, r=8, seed=3)
    for T in (0.0, 0.5, 1.0, 2.0):
        ev = o.eval_node(m, 0, 17, 2, 0x5, T, 11, 4)
        assert abs(np.exp(ev.z - ev.lse0).sum() - 1.0) < 1e-12
        if T > 0:
            assert abs(np.exp(ev.z / T - ev.lseT).sum() - 1.0) < 1e-12
        else:
            assert math.isnan(ev.lseT)


def test_eval_indexing_with_structured_factors():
    """z[y] = U[q][d][y] + <E[x], W2[y]>: a rank-one construction pins the operands and rows."""
    V, D, r, R = 50, 3, 4, 2
    rng = np.random.default_rng(0)
    U = rng.normal(size=(R, D, V)).astype(np.float32)
    E = np.zeros((V, r), np.float32)
    W2 = np.zeros((V, r), np.float32)
    E[7, 2] = 3.0                      # parent token 7 loads factor 2 only
    E[2, 7 % r] = 100.0                # a transposed lookup would pick this row instead
    W2[:, 2] = np.arange(V) * 0.25     # bias B(7, y) = 3 * 0.25 y
    W2[7, :] = 50.0
    m = o.Model(U, E, W2)
    ev = o.eval_node(m, 1, 7, 2, 0, 0.0, 0, 3)
    expect = U[1, 2].astype(np.float64) + 3.0 * (np.arange(V) * 0.25)
    expect[7] = float(U[1, 2, 7]) + 3.0 * 50.0
    np.testing.assert_allclose(ev.z, expect, rtol=0, atol=1e-9)


def test_marginal_special_case():
    """B == 0 (W2 = 0): every parent at depth d gets top-K of U_d and lse = logsumexp(U_d) (§3.2, marginal tree)."""
    V, D, r = 200, 4, 8
    dr, _ = _tiny_model(V=V, D=D, r=r, seed=5, u_sigma=2.0)
    m = o.Model(dr.U32, dr.E32, np.zeros_like(dr.W2_32))
    K = 5
    for d in range(D):
        row = dr.U32[0, d].astype(np.float64)
        want = np.lexsort((np.arange(V), -row))[:K]
        for tok in (0, 13, 150):
            ev = o.eval_node(m, 0, tok, d, 0, 0.0, 0, K)
            assert list(ev.pi) == list(want)
            assert ev.lse0 == pytest.approx(special.logsumexp(row), rel=1e-14)


def test_gumbel_top_k_low_temperature_limit():
    """As T -> 0 the without-replacement draws become the greedy order (Algorithm 1, T=0 vs T>0)."""
    dr, m = _tiny_model(V=400, D=3, r=8, seed=9, u_sigma=3.0)
    agree = 0
    for tok in range(40):
        ev = o.eval_node(m, 0, tok, 1, 0, 1e-4, 123, 6)
        ties = ev.pi_z[:-1] - ev.pi_z[1:]
        if np.all(ties > 1e-3):
            assert list(ev.sigma) == list(ev.pi)
            agree += 1
    assert agree >= 35


def test_plackett_luce_first_two_draws():
    """Gumbel-top-k realises draws without replacement (§3.3 residual proposal):
    Pr(s1 = x, s2 = y) = q(x) q(y) / (1 - q(x)); chi-square over 1e5 seeds."""
    V, T = 5, 0.8
    dr, m = _tiny_model(V=V, D=2, r=3, seed=21, u_sigma=1.0, ew_sigma=0.5)
    ev0 = o.eval_node(m, 0, 2, 1, 0x3, T, 0, 2)
    q = special.softmax(ev0.z / T)
    expected = np.zeros((V, V))
    for x in range(V):
        for y in range(V):
            if x != y:
                expected[x, y] = q[x] * q[y] / (1.0 - q[x])
    counts = np.zeros((V, V))
    n = 100_000
    for s in range(n):
        ev = o.eval_node(m, 0, 2, 1, 0x3, T, s, 2, want_z=False)
        counts[ev.sigma[0], ev.sigma[1]] += 1
    mask = ~np.eye(V, dtype=bool)
    chi = stats.chisquare(counts[mask], expected[mask] * n)
    assert chi.pvalue > 1e-3
    assert np.all(np.diag(counts) == 0)  # siblings are distinct


def test_sequential_draws_reduce_to_inverse_cdf():
    """Sampler 1 on a one-block vocabulary is textbook inverse-CDF sampling without
    replacement (numpy cumsum + searchsorted with the same Philox words)."""
    rng = np.random.default_rng(5)
    for trial in range(40):
        V = int(rng.integers(2, 65))
        z = rng.normal(size=V) * 2.0
        T = float(rng.choice([0.3, 0.7, 1.0, 2.0]))
        K = int(rng.integers(1, min(V, 16) + 1))
        path, depth, req, seed = int(rng.integers(0, 2**40)), int(rng.integers(0, 16)), int(rng.integers(0, 64)), trial
        got, gap = o.draw_sequential(z, T, seed, req, depth, path, K)
        want = _inverse_cdf_draws(special.softmax(z / T), K, seed, req, depth, path)
        if gap > 1e-9:
            assert list(got) == want, (trial, got, want)


def test_sequential_draws_are_distinct_and_cover_the_vocabulary():
    """Without replacement: K = V draws are a permutation, across segment and block edges."""
    for V, T in [(64, 1.0), (130, 0.5), (4097, 2.0), (8200, 4.0)]:
        z = np.random.default_rng(V).normal(size=V)
        K = min(V, 16)
        got, _ = o.draw_sequential(z, T, 3, 0, 1, 0x21, K)
        assert len(set(got.tolist())) == K and got.min() >= 0 and got.max() < V
    z = np.random.default_rng(1).normal(size=9)
    got, _ = o.draw_sequential(z, 1.0, 7, 0, 0, 0, 9)
    assert sorted(got.tolist()) == list(range(9))


def test_sequential_draws_stop_at_the_support():
    """q_T has no mass on tokens with -inf logits (§3.3): with m finite logits the first m draws
    are those m tokens, in the order inverse-CDF sampling over them alone gives, and every later
    draw is empty (-1), across segment edges."""
    rng = np.random.default_rng(21)
    for V, m, K in [(50, 3, 8), (9000, 5, 12), (9000, 1, 4)]:
        z = np.full(V, -np.inf)
        keep = np.sort(rng.choice(V, m, replace=False))
        z[keep] = rng.normal(size=m) * 2.0
        got, _ = o.draw_sequential(z, 0.7, 4, 1, 2, 0x33, K)
        assert sorted(got[:m].tolist()) == keep.tolist()
        assert np.all(got[m:] == -1)
    # one block: the same words drive inverse-CDF draws over the finite tokens
    z = np.full(40, -np.inf)
    keep = np.array([3, 17, 30])
    z[keep] = [0.5, -1.0, 2.0]
    got, gap = o.draw_sequential(z, 0.9, 9, 0, 1, 0x7, 6)
    q = np.zeros(40)
    q[keep] = special.softmax(z[keep] / 0.9)
    if gap > 1e-9:
        assert list(got[:3]) == _inverse_cdf_draws(q, 3, 9, 0, 1, 0x7)


def test_sequential_draws_low_temperature_limit():
    """As T -> 0 the residual proposal puts all mass on the best unused token: sigma = pi."""
    rng = np.random.default_rng(8)
    z = rng.normal(size=9000) * 3.0
    got, _ = o.draw_sequential(z, 1e-3, 11, 2, 3, 0x5, 8)
    assert list(got) == list(np.lexsort((np.arange(len(z)), -z))[:8])


def test_sequential_draws_follow_plackett_luce_across_segments():
    """Pr(s1 = x, s2 = y) = q(x) q(y) / (1 - q(x)) for draws whose tokens sit in different
    segments and blocks (V = 9000: three segments); chi-square over 40000 seeds."""
    V, T = 9000, 1.0
    heavy = [5, 70, 4100, 4160, 8999]
    z = np.full(V, -6.0)
    z[heavy] = [1.0, 0.6, 0.9, 0.2, 0.5]
    q = special.softmax(z / T)
    cats = heavy + [-1]  # -1: any other token
    qc = np.array([q[h] for h in heavy] + [1.0 - q[heavy].sum()])
    expected = np.zeros((6, 6))
    for i in range(6):
        for k in range(6):
            if i == k and i < 5:
                continue
            # the "other" bucket holds many tokens, so it can follow itself
            expected[i, k] = qc[i] * qc[k] / (1.0 - (qc[i] if i < 5 else 0.0))
    # second draw after "other": its mass loses one light token, negligible at these sizes
    n = 40_000
    counts = np.zeros((6, 6))
    idx = {h: i for i, h in enumerate(heavy)}
    for s in range(n):
        got, _ = o.draw_sequential(z, T, s, 0, 2, 0x7, 2)
        counts[idx.get(int(got[0]), 5), idx.get(int(got[1]), 5)] += 1
    mask = expected > 0
    expected = expected / expected[mask].sum()
    chi = stats.chisquare(counts[mask], expected[mask] * n)
    assert chi.pvalue > 1e-3, chi


# ---------------------------------------------------------------- expansion

def _draw_words(seed, request, depth, path, j):
    """The three words of one sequential draw (tag 4, c0 = j), from the Philox pin."""
    ctr = [j, path & 0xFFFFFFFF, path >> 32, (request << 12) | (depth << 4) | 4]
    w = o.philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32])
    return [((int(x) >> 9) + 0.5) / 2**23 for x in w[:3]]


def _inverse_cdf_draws(q, K, seed, request, depth, path):
    """Textbook inverse-CDF draws without replacement for a vocabulary of one 64-token
    block (segment and block picks are forced): token = searchsorted(cumsum, u * total)."""
    q = np.array(q, dtype=np.float64)
    out = []
    for j in range(1, K + 1):
        u3 = _draw_words(seed, request, depth, path, j)[2]
        c = np.cumsum(q)
        out.append(int(np.searchsorted(c, u3 * c[-1], side="right")))
        q[out[-1]] = 0.0
    return out


def _universe_brute_force(model_arrays, V, D, r, anchor, theta, N, K, T, seed, a=A, b=B,
                          sampler="gumbel", request=0):
    """Enumerate the full K-ary universe of slots with numpy and return the top-N keys >= log theta.
    model_arrays holds this request's U rows as U[0]; request keys the random words."""
    U, E, W2 = model_arrays
    slots = []

    def philox_u(depth, path, tag, y):
        ctr = [y >> 2, path & 0xFFFFFFFF, path >> 32, (request << 12) | (depth << 4) | tag]
        w = o.philox4x32_10(ctr, [seed & 0xFFFFFFFF, seed >> 32])[y & 3]
        return ((int(w) >> 9) + 0.5) / 2**23

    def logphat(lq):
        q = math.exp(lq)
        if q >= 1.0:
            return 0.0
        x = a * (math.log(q) - math.log1p(-q)) + b
        return -math.log1p(math.exp(-x)) if x >= 0 else x - math.log1p(math.exp(x))

    def expand(token, depth, path, logS):
        z = U[0, depth].astype(np.float64) + W2.astype(np.float64) @ E[token].astype(np.float64)
        lse0 = special.logsumexp(z)
        pi = list(np.lexsort((np.arange(V), -z))[:K])
        if T > 0 and sampler == "sequential":
            sigma = _inverse_cdf_draws(special.softmax(z / T), K, seed, request, depth, path)
        elif T > 0:
            g = z / T - np.log(-np.log([philox_u(depth, path, 1, y) for y in range(V)]))
            sigma = list(np.lexsort((np.arange(V), -g))[:K])
        for j in range(1, K + 1):
            if T == 0:
                tok = pi[j - 1]
                key = logS + logphat(z[tok] - lse0)
                lS = key
            else:
                tok = sigma[j - 1]
                bound = next(t for t in pi if t not in sigma[: j - 1])
                key = logS + logphat(z[bound] - lse0)
                lS = logS + logphat(z[tok] - lse0)
            cpath = path | ((j - 1) << (4 * depth))
            slots.append((key, depth + 1, cpath, tok, lS))
            if depth + 1 < D:
                expand(tok, depth + 1, cpath, lS)

    expand(anchor, 0, 0, 0.0)
    slots.sort(key=lambda s: (-s[0], s[1], s[2]))
    lt = math.log(theta) if theta > 0 else -math.inf
    out = []
    for s in slots:
        if len(out) == N or s[0] < lt:
            break
        out.append(s)
    return out


@pytest.mark.parametrize("T,theta,N,K,D,sampler", [(0.0, 0.0, 9, 3, 3, "gumbel"),
                                                    (0.0, 0.08, 20, 2, 4, "gumbel"),
                                                    (1.0, 0.0, 11, 3, 3, "gumbel"),
                                                    (0.7, 0.05, 20, 2, 4, "gumbel"),
                                                    (1.0, 0.0, 11, 3, 3, "sequential"),
                                                    (0.7, 0.05, 20, 2, 4, "sequential")])
def test_expansion_equals_universe_top_n(T, theta, N, K, D, sampler):
    """Best-first expansion (Algorithm 1) returns the top-N slots >= theta of the full K-ary
    universe, in (key desc, depth asc, path asc) order: brute force on a tiny vocabulary."""
    V, r = 7, 3
    dr, m = _tiny_model(V=V, D=D, r=r, seed=31, u_sigma=2.0, ew_sigma=0.8)
    seed = 99
    tree = o.expand_tree(m, 0, 4, theta, N, K, T, seed, sampler=sampler)
    want = _universe_brute_force((dr.U32, dr.E32, dr.W2_32), V, D, r, 4, theta, N, K, T, seed,
                                 sampler=sampler)
    assert tree.n == len(want)
    for i, s in enumerate(want, start=1):
        assert tree.key[i] == pytest.approx(s[0], rel=1e-12, abs=1e-12)
        assert tree.depth[i] == s[1]
        assert int(tree.path[i]) == s[2]
        assert tree.token[i] == s[3]
        assert tree.log_surv[i] == pytest.approx(s[4], rel=1e-12, abs=1e-12)


def test_tree_invariants_and_survival_product():
    """Path survival is the product of p-hat along the path (§3.5); keys are non-increasing in
    creation order; siblings are distinct with contiguous ranks; path ids follow the parent."""
    dr = synth.make_workload_drafter(0, seed=0)
    m = o.Model(dr.U32, dr.E32, dr.W2_32)
    for T in (0.0, 1.0):
        tree = o.expand_tree(m, 0, 11, 0.0, 32, 4, T, 0)
        assert tree.n == 32  # fixed budget is theta = 0
        for c in range(1, tree.n + 1):
            p = tree.parent[c]
            assert tree.depth[c] == tree.depth[p] + 1
            assert int(tree.path[c]) == int(tree.path[p]) | ((tree.rank[c] - 1) << (4 * tree.depth[p]))
            # survival = product of p-hat computed from the emitted log q0 with the plain formula
            s, v = 0.0, c
            while v != 0:
                q = math.exp(tree.log_q0[v])
                s += math.log(special.expit(A * math.log(q / (1 - q)) + B))
                v = tree.parent[v]
            assert tree.log_surv[c] == pytest.approx(s, rel=1e-9, abs=1e-12)
            assert tree.key[c] <= tree.key[c - 1] + 1e-15 or c == 1
            if T == 0:
                assert tree.key[c] == tree.log_surv[c]
        for v in range(tree.n + 1):
            kids = [c for c in range(1, tree.n + 1) if tree.parent[c] == v]
            assert [tree.rank[c] for c in kids] == list(range(1, len(kids) + 1))
            assert len({tree.token[c] for c in kids}) == len(kids)


def test_chain_special_case():
    """K = 1, theta = 0, N = D at T = 0 reproduces the chain x_k = argmax(U_k + B(x_{k-1})) (§3.1, App. C)."""
    dr = synth.make_workload_drafter(0, seed=4)
    m = o.Model(dr.U32, dr.E32, dr.W2_32)
    anchor = 123
    tree = o.expand_tree(m, 0, anchor, 0.0, dr.D, 1, 0.0, 0)
    x = anchor
    chain = []
    for d in range(dr.D):
        z = dr.U32[0, d].astype(np.float64) + dr.W2_32.astype(np.float64) @ dr.E32[x].astype(np.float64)
        x = int(np.argmax(z))
        chain.append(x)
    assert tree.n == dr.D
    assert list(tree.token[1:]) == chain
    assert list(tree.parent[1:]) == list(range(dr.D))


def test_theta_stop_is_strict_and_monotone():
    """Expansion stops at the first popped key below log theta (§3.5); larger theta gives a subtree prefix."""
    dr = synth.make_workload_drafter(0, seed=0)
    m = o.Model(dr.U32, dr.E32, dr.W2_32)
    big = o.expand_tree(m, 0, 11, 0.0, 32, 4, 0.0, 0)
    for theta in (0.2, 0.05, 0.01, 0.002):
        t = o.expand_tree(m, 0, 11, theta, 32, 4, 0.0, 0)
        lt = math.log(theta)
        assert np.all(t.key[1:] >= lt)
        if t.n < 32:
            assert t.stop_key < lt
        assert list(t.token) == list(big.token[: t.n + 1])


# ---------------------------------------------------------------- verification

def test_greedy_verify_equals_greedy_decoding():
    """At T = 0 the accepted tokens are the longest tree prefix of the greedy target path and the
    bonus is the greedy next token (§3.2 item 3, §3.3): checked against direct greedy decoding."""
    V, D = 12, 4
    dr, m = _tiny_model(V=V, D=D, r=4, seed=2, u_sigma=2.0)
    rng = np.random.default_rng(5)
    table = {}

    def row(prefix):
        if prefix not in table:
            table[prefix] = rng.normal(size=V).astype(np.float32) * 2
        return table[prefix]

    for trial in range(60):
        table.clear()
        tree = o.expand_tree(m, 0, trial % V, 0.0, 10, 3, 0.0, 0)
        prefixes = []
        for i in range(tree.n + 1):
            pre, v = [], i
            while v != 0:
                pre.append(int(tree.token[v])); v = tree.parent[v]
            prefixes.append(tuple(reversed(pre)))
        if trial % 3 == 0:  # plant a fully accepted greedy path through the deepest node
            deepest = int(np.argmax(tree.depth))
            for k in range(len(prefixes[deepest]) + 1):
                pre = prefixes[deepest][:k]
                r_ = row(pre).copy()
                if k < len(prefixes[deepest]):
                    r_[prefixes[deepest][k]] = 50.0
                table[pre] = r_
        target = np.stack([row(p) for p in prefixes])
        path, bonus, _ = o.verify_greedy(tree, target)
        # direct greedy decoding against the same target function
        greedy, pre = [], ()
        for _ in range(D + 2):
            g = int(np.argmax(row(pre)))
            greedy.append(g)
            pre = pre + (g,)
        accepted = [int(tree.token[c]) for c in path]
        assert accepted == greedy[: len(accepted)]
        assert bonus == greedy[len(accepted)]
        # longest: no child of the last accepted node carries the next greedy token
        last = path[-1] if len(path) else 0
        kids = [c for c in range(1, tree.n + 1) if tree.parent[c] == last]
        assert greedy[len(accepted)] not in [int(tree.token[c]) for c in kids]
        if trial % 3 == 0:
            assert len(path) == tree.depth[int(np.argmax(tree.depth))]


def test_residual_scalar_form_equals_literal_recursion():
    """p_j = norm(max(p_{j-1} - q_{j-1}, 0)) with q_j = norm(qT * 1[not drawn]) (§3.3) equals the
    two-scalar form max(alpha_j p - beta_j qT, 0) used by the GPU, at every stage the walk can
    reach (a stage is reached only if every earlier stage had ratio < 1)."""
    rng = np.random.default_rng(1)
    for trial in range(200):
        V = int(rng.integers(3, 40))
        p = rng.dirichlet(np.ones(V) * rng.uniform(0.2, 3))
        qT = rng.dirichlet(np.ones(V) * rng.uniform(0.2, 3))
        m = int(rng.integers(1, min(V, 8) + 1))
        x = rng.choice(V, size=m, replace=False)
        ratio, Z, pf = o.residual_stages(p, qT, x)
        alpha, beta, R = 1.0, 0.0, 1.0
        all_rejectable = True
        for j in range(m):
            xj = x[j]
            pj = max(alpha * p[xj] - beta * qT[xj], 0.0)
            assert ratio[j] == pytest.approx(pj / (qT[xj] / R), rel=1e-9, abs=1e-12)
            if ratio[j] >= 1.0:
                # acceptance is certain: later stages are never reached by the walk
                all_rejectable = False
                break
            beta_p = beta + 1.0 / R
            zj = np.maximum(alpha * p - beta_p * qT, 0.0).sum()
            assert Z[j] == pytest.approx(zj, rel=1e-9, abs=1e-13)
            if zj > 0:
                alpha, beta = alpha / zj, beta_p / zj
            R -= qT[xj]
        final = np.maximum(alpha * p - beta * qT, 0.0)
        if all_rejectable and Z[-1] > 0:
            np.testing.assert_allclose(pf, final, rtol=1e-8, atol=1e-12)
    # one stage: Z_1 = TV(p, q)
    p = np.array([0.5, 0.3, 0.2]); q = np.array([0.2, 0.3, 0.5])
    _, Z, _ = o.residual_stages(p, q, np.array([2]))
    assert Z[0] == pytest.approx(0.5 * np.abs(p - q).sum(), rel=1e-14)


def _prefix_rows(V, D, seed, scale):
    rng = np.random.default_rng(seed)
    rows = {}
    for depth in range(D + 1):
        for pre in itertools.product(range(V), repeat=depth):
            rows[pre] = (rng.normal(size=V) * scale).astype(np.float32)
    return rows


def _tree_prefixes(tree):
    prefixes = [()]
    for i in range(1, tree.n + 1):
        prefixes.append(prefixes[tree.parent[i]] + (int(tree.token[i]),))
    return prefixes


def _emitted(tree, path, bonus):
    return [int(tree.token[c]) for c in path] + [bonus]


@pytest.mark.slow
@pytest.mark.parametrize("sampler", ["gumbel", "sequential"])
def test_losslessness_chi_square(sampler):
    """Proposition 1: with sampled trees and recursive rejection the first emitted token follows
    softmax(target_root / T), and the token after an accepted depth-1 child x follows
    softmax(target_x / T); chi-square over 1e5 seeds, for both realisations of the draws."""
    V, D, K, N, T = 6, 3, 3, 7, 1.0
    dr, m = _tiny_model(V=V, D=D, r=3, seed=41, u_sigma=0.8, ew_sigma=0.6)
    rows = _prefix_rows(V, D, 7, 1.0)
    n = 100_000
    first = np.zeros(V)
    second = {}
    for s in range(n):
        tree = o.expand_tree(m, 0, 1, 0.0, N, K, T, s, sampler=sampler)
        target = np.stack([rows[p] for p in _tree_prefixes(tree)])
        path, bonus, _ = o.verify_sample(m, 0, tree, target, T, s)
        em = _emitted(tree, path, bonus)
        first[em[0]] += 1
        if len(path) >= 1:
            second.setdefault(em[0], np.zeros(V))[em[1]] += 1
    p_root = special.softmax(rows[()].astype(np.float64) / T)
    assert stats.chisquare(first, p_root * n).pvalue > 1e-3
    x1 = max(second, key=lambda k: second[k].sum())
    cnt = second[x1]
    p_x1 = special.softmax(rows[(x1,)].astype(np.float64) / T)
    assert cnt.sum() > 5000
    assert stats.chisquare(cnt, p_x1 * cnt.sum()).pvalue > 1e-3


def test_top_k_control_is_rejected():
    """Power check (§3.3 failure mode): deterministic top-k children with the same rejection walk
    are biased; the same chi-square rejects them on a target equal to the drafter."""
    V, D, K, N, T = 6, 2, 3, 3, 1.0
    dr, m = _tiny_model(V=V, D=D, r=3, seed=43, u_sigma=0.3, ew_sigma=0.3)
    root_z = o.eval_node(m, 0, 1, 0, 0, T, 0, 1).z
    n = 20_000
    first = np.zeros(V)
    for s in range(n):
        tree = o.expand_tree(m, 0, 1, 0.0, N, K, T, s, control_topk=True)
        target = np.tile(root_z.astype(np.float32), (tree.n + 1, 1))
        path, bonus, _ = o.verify_sample(m, 0, tree, target, T, s)
        first[_emitted(tree, path, bonus)[0]] += 1
    p_root = special.softmax(root_z / T)
    assert stats.chisquare(first, p_root * n).pvalue < 1e-12


def test_single_child_acceptance_rate():
    """One drawn child: acceptance probability is sum_x min(p(x), q(x)) = 1 - TV(p, q)
    (standard speculative sampling, cited in §3.3); binomial check over 1e5 seeds."""
    V, T = 8, 1.0
    dr, m = _tiny_model(V=V, D=2, r=3, seed=47, u_sigma=1.0, ew_sigma=0.5)
    rng = np.random.default_rng(3)
    root_row = (rng.normal(size=V) * 1.2).astype(np.float32)
    q = special.softmax(o.eval_node(m, 0, 1, 0, 0, T, 0, 1).z / T)
    p = special.softmax(root_row.astype(np.float64) / T)
    want = np.minimum(p, q).sum()
    n = 100_000
    acc = 0
    for s in range(n):
        tree = o.expand_tree(m, 0, 1, 0.0, 1, 1, T, s)
        target = np.stack([root_row, root_row])
        path, _, _ = o.verify_sample(m, 0, tree, target, T, s)
        acc += len(path)
    sd = math.sqrt(want * (1 - want) / n)
    assert abs(acc / n - want) < 5 * sd


# ---------------------------------------------------------------- tree attention mask

@pytest.mark.parametrize("T,sampler", [(0.0, "gumbel"), (1.0, "gumbel"), (0.7, "sequential")])
def test_tree_mask_equals_path_prefix_relation(T, sampler):
    """Bit j of row i is set iff node j's structural path id is a prefix of node i's (j is i
    or an ancestor of i), and pos = offset + depth, on deep oracle trees."""
    dr = synth.make_drafter(300, 8, 16, R=1, dtype="f32", u_sigma=3.0, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.3, seed=21, u_scale=3.0)
    m = o.Model(dr.U32, dr.E32, dr.W2_32)
    tree = o.expand_tree(m, 0, 5, 0.0, 40, 3, T, 4, sampler=sampler)
    assert tree.depth.max() >= 3
    cap = tree.n + 9  # unused rows at the end
    parent = np.full(cap, -1, np.int32)
    parent[: tree.n + 1] = tree.parent
    mask, pos = o.tree_mask(parent, tree.n, cap, offset=100)
    for i in range(cap):
        for j in range(cap):
            bit = (int(mask[i, j >> 5]) >> (j & 31)) & 1
            if i > tree.n or j > tree.n:
                want = 0
            else:
                dj = int(tree.depth[j])
                low = (1 << (4 * dj)) - 1
                want = int(dj <= tree.depth[i] and (int(tree.path[i]) & low) == int(tree.path[j]))
            assert bit == want, (i, j)
        assert pos[i] == (100 + tree.depth[i] if i <= tree.n else -1)


def test_tree_mask_chain_and_star():
    """A chain gives the lower-triangular all-ones mask with pos = offset + i; a star gives
    {0, i} rows with pos = offset + 1 (offset 0 for the anchor)."""
    n = 70
    chain = np.arange(-1, n, dtype=np.int32)
    mask, pos = o.tree_mask(chain, n, n + 1, offset=7)
    dense = np.unpackbits(mask.view(np.uint8), axis=1, bitorder="little")[:, : n + 1]
    assert np.array_equal(dense, np.tril(np.ones((n + 1, n + 1), np.uint8)))
    assert list(pos) == [7 + i for i in range(n + 1)]
    star = np.zeros(n + 1, np.int32)
    star[0] = -1
    mask, pos = o.tree_mask(star, n, n + 1)
    dense = np.unpackbits(mask.view(np.uint8), axis=1, bitorder="little")[:, : n + 1]
    want = np.eye(n + 1, dtype=np.uint8)
    want[:, 0] = 1
    assert np.array_equal(dense, want)
    assert pos[0] == 0 and np.all(pos[1:] == 1)


def test_tree_mask_rejects_a_parent_after_its_child():
    with pytest.raises(ValueError):
        o.tree_mask(np.array([-1, 0, 3, 1], np.int32), 3, 4)


# ---------------------------------------------------------------- global node budget

def _forest_model(R=3, V=7, D=4, r=3, seed=17):
    dr = synth.make_drafter(V, D, r, R=R, dtype="f32", u_sigma=2.0, planted=None, zipf=None,
                            ew_sigma=0.8, seed=seed)
    return dr, o.Model(dr.U32, dr.E32, dr.W2_32)


@pytest.mark.parametrize("T,sampler", [(0.0, "gumbel"), (0.8, "gumbel"), (0.8, "sequential")])
def test_forest_without_budget_equals_independent_trees(T, sampler):
    """With no binding global budget every request's tree is its own Algorithm 1 tree."""
    dr, m = _forest_model()
    anchors, thetas = [1, 4, 6], [0.0, 0.03, 0.1]
    trees = o.expand_forest(m, anchors, thetas, 12, 0, 3, T, 5, sampler=sampler)
    for q in range(3):
        ref = o.expand_tree(m, q, anchors[q], thetas[q], 12, 3, T, 5, sampler=sampler)
        assert trees[q].n == ref.n
        for name in ("token", "parent", "depth", "rank", "path"):
            assert list(getattr(trees[q], name)) == list(getattr(ref, name)), (q, name)
        assert np.allclose(trees[q].log_surv, ref.log_surv, rtol=0, atol=1e-12)


@pytest.mark.parametrize("budget,T", [(5, 0.0), (9, 0.0), (14, 0.7), (30, 1.0)])
def test_forest_equals_global_top_b_of_the_universes(budget, T):
    """Brute force: the budgeted trees are the global top-B slots of the requests' K-ary
    universes, each request limited to its own top-N slots above its theta."""
    R, V, D, r, K, N = 3, 7, 4, 3, 2, 8
    dr, m = _forest_model(R, V, D, r)
    anchors, thetas = [2, 5, 3], [0.0, 0.02, 0.0]
    trees = o.expand_forest(m, anchors, thetas, N, budget, K, T, 11)
    pool = []
    for q in range(R):
        U = dr.U32[q:q + 1]
        slots = _universe_brute_force((U, dr.E32, dr.W2_32), V, D, r, anchors[q], thetas[q], N, K, T, 11,
                                      request=q)
        pool += [(s[0], q, s[1], s[2], s[3]) for s in slots]
    pool.sort(key=lambda s: (-s[0], s[1], s[2], s[3]))
    chosen = pool[:budget]
    for q in range(R):
        mine = [s for s in chosen if s[1] == q]
        assert trees[q].n == len(mine), q
        for i, s in enumerate(mine, start=1):
            assert trees[q].key[i] == pytest.approx(s[0], rel=1e-12, abs=1e-12)
            assert int(trees[q].path[i]) == s[3] and trees[q].token[i] == s[4]


def test_forest_is_a_uniform_price():
    """Section 4: under one marginal price the budget allocation is the theta rule: each budgeted
    tree equals the request's own tree with theta' = max(theta, exp(key of the last node))."""
    dr, m = _forest_model(R=4, V=9, D=5, r=3, seed=23)
    anchors, thetas = [1, 2, 3, 4], [0.0, 0.01, 0.0, 0.05]
    trees = o.expand_forest(m, anchors, thetas, 30, 17, 3, 0.0, 2)
    last = min(t.key[1:t.n + 1].min() for t in trees if t.n > 0)
    assert sum(t.n for t in trees) == 17
    for q in range(4):
        th = max(thetas[q], math.exp(last))
        ref = o.expand_tree(m, q, anchors[q], th, 30, 3, 0.0, 2)
        assert trees[q].n == ref.n and list(trees[q].token) == list(ref.token), q


# ---------------------------------------------------------------- calibration fit (§3.4 Eq. 3)

def test_logit_q0_closed_forms():
    """logit q0 = log(q0 / (1 - q0)): 0 at q0 = 1/2, log 9 at 0.9, -log 999 at 0.001, +inf at 1;
    the two branches of log(1 - q0) meet at q0 = 1/2."""
    lq = np.log(np.array([0.5, 0.9, 0.001, 1.0, 0.5 - 1e-12, 0.5 + 1e-12]))
    got = o.logit_q0(lq)
    assert got[0] == pytest.approx(0.0, abs=1e-15)
    assert got[1] == pytest.approx(math.log(9.0), rel=1e-13)
    assert got[2] == pytest.approx(-math.log(999.0), rel=1e-13)
    assert got[3] == math.inf
    assert abs(got[4]) < 1e-11 and abs(got[5]) < 1e-11


def test_calib_labels_on_a_hand_tree():
    """Root 0; nodes 1, 2 under the root, 3 under 1, 4 under 3, 5 under 2.  The target's greedy
    choices: row 0 -> token of node 1, row 1 -> not the token of node 3, row 3 -> token of node 4,
    row 2 -> token of node 5 (a tie broken toward the smaller id).  Accepted edges: 1, 4, 5;
    ancestors-accepted edges: 1, 2 (root children) and 3 (under the accepted 1)."""
    parent = np.array([-1, 0, 0, 1, 3, 2, -1], np.int32)
    token = np.array([9, 4, 6, 2, 7, 1, -1], np.int32)
    V = 10
    target = np.zeros((7, V))
    target[0, 4] = 3.0             # greedy 4 = token of node 1
    target[1, 5] = 2.0             # greedy 5, node 3 has token 2
    target[3, 7] = 1.0             # greedy 7 = token of node 4
    target[2, 1] = target[2, 8] = 5.0  # tie: smallest id 1 = token of node 5
    y, sel = o.calib_labels(parent, token, 5, target)
    assert list(y) == [-1, 1, 0, 0, 1, 1, -1]
    assert list(sel) == [0, 1, 1, 1, 0, 0, 0]


def test_platt_fit_saturated_closed_form():
    """Two distinct inputs with acceptance frequencies f1, f2: the maximum-likelihood map passes
    through both, a = (logit f1 - logit f2) / (x1 - x2), b = logit f1 - a x1."""
    x1, x2, n1, k1, n2, k2 = 1.5, -0.5, 400, 300, 600, 150
    x = np.r_[np.full(n1, x1), np.full(n2, x2)]
    y = np.r_[np.ones(k1), np.zeros(n1 - k1), np.ones(k2), np.zeros(n2 - k2)]
    lg = lambda f: math.log(f / (1 - f))
    a_ref = (lg(k1 / n1) - lg(k2 / n2)) / (x1 - x2)
    b_ref = lg(k1 / n1) - a_ref * x1
    a, b, _, _ = o.platt_fit(x, y)
    assert a == pytest.approx(a_ref, rel=1e-9) and b == pytest.approx(b_ref, rel=1e-9)


def test_platt_fit_equals_unpenalised_logistic_regression():
    """The fit is the unpenalised logistic regression of y on x (scikit-learn's solver), and the score
    equations sum(p - y) = 0, sum((p - y) x) = 0 hold at it."""
    from sklearn.linear_model import LogisticRegression
    rng = np.random.default_rng(5)
    x = rng.normal(-1.0, 2.5, 20000)
    y = (rng.random(20000) < 1.0 / (1.0 + np.exp(-(0.8 * x + 0.3)))).astype(float)
    a, b, nll, steps = o.platt_fit(x, y)
    m = LogisticRegression(penalty=None, tol=1e-12, max_iter=10000).fit(x[:, None], y)
    assert a == pytest.approx(float(m.coef_[0, 0]), rel=1e-6)
    assert b == pytest.approx(float(m.intercept_[0]), rel=1e-6, abs=1e-8)
    p = 1.0 / (1.0 + np.exp(-(a * x + b)))
    assert abs(np.sum(p - y)) < 1e-7 * len(x) and abs(np.sum((p - y) * x)) < 1e-7 * len(x)
    assert steps < 20 and 0.0 < nll < math.log(2.0)


def test_platt_fit_recovers_the_papers_coefficients():
    """Labels drawn from the paper's map sigma(0.67 logit q0 - 0.46) over 2e5 edges give back
    (0.67, -0.46) within five standard errors (about 0.005 each here)."""
    rng = np.random.default_rng(11)
    x = rng.normal(0.5, 2.0, 200_000)
    y = (rng.random(len(x)) < 1.0 / (1.0 + np.exp(-(0.67 * x - 0.46)))).astype(float)
    a, b, _, _ = o.platt_fit(x, y)
    assert abs(a - 0.67) < 0.025 and abs(b + 0.46) < 0.03
