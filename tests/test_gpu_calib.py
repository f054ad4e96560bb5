"""GPU parity of the calibration utility (ts_calib_labels, ts_calib_fit) against the oracle."""
import math

import numpy as np
import pytest

from oracle import oracle as o
from paper_2609_22098_amd import synth
from helpers import Tally, compare_tree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_22098_amd import binding
    binding.lib()
    return t


def _samples(seed, n, a, b, spread, frac_sel=0.8, n_inf=0):
    rng = np.random.default_rng(seed)
    x = rng.normal(0.3, spread, n).astype(np.float32)
    p = 1.0 / (1.0 + np.exp(-(a * x.astype(np.float64) + b)))
    y = (rng.random(n) < p).astype(np.int32)
    sel = (rng.random(n) < frac_sel).astype(np.int32)
    x[:n_inf] = np.inf  # q0 == 1: left out of the fit
    return x, y, sel


@pytest.mark.parametrize("seed,n,a,b,spread", [(0, 30000, 0.67, -0.46, 2.0), (1, 1000, 1.5, 0.8, 1.0),
                                                (2, 123457, 0.3, -1.2, 3.0), (3, 17, 0.9, 0.1, 2.0)])
def test_calib_fit_matches_oracle(torch, seed, n, a, b, spread):
    """The device fit equals the oracle's Newton fit on the same samples (sel = 1, finite x):
    (a, b) and the mean negative log-likelihood within 2e-6 relative, the same number of steps."""
    from paper_2609_22098_amd import binding
    x, y, sel = _samples(seed, n, a, b, spread, n_inf=3 if n > 100 else 0)
    m = (sel == 1) & np.isfinite(x)
    ra, rb, rnll, rsteps = o.platt_fit(x[m].astype(np.float64), y[m])
    ga, gb, gnll, gsteps = binding.calib_fit(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(),
                                             torch.from_numpy(sel).cuda())
    print(f"n={n}: device a={ga:.6f} b={gb:.6f} nll={gnll:.6f} steps={gsteps}; "
          f"oracle a={ra:.6f} b={rb:.6f} nll={rnll:.6f} steps={rsteps}")
    assert ga == pytest.approx(ra, rel=2e-6, abs=1e-6) and gb == pytest.approx(rb, rel=2e-6, abs=1e-6)
    assert gnll == pytest.approx(rnll, rel=2e-6)
    assert abs(gsteps - rsteps) <= 1


def test_calib_fit_degenerate_inputs(torch):
    """No sample taking part, or a single input value (singular curvature): NaN scalars."""
    from paper_2609_22098_amd import binding
    x = torch.full((50,), 0.5, dtype=torch.float32, device="cuda")
    y = torch.tensor([0, 1] * 25, dtype=torch.int32, device="cuda")
    a, b, nll, steps = binding.calib_fit(x, y, torch.zeros(50, dtype=torch.int32, device="cuda"))
    assert math.isnan(a) and math.isnan(b) and math.isnan(nll)
    a, b, nll, steps = binding.calib_fit(x, y, torch.ones(50, dtype=torch.int32, device="cuda"))
    assert math.isnan(a) and math.isnan(b)


def _oracle_round(dr, anchors, N, K, sigma, seed):
    """Oracle trees at T = 0, their target rows and labels: (trees, target [R][cap][V] float32,
    y [R][cap], sel [R][cap], x [R][cap])."""
    om = o.Model(dr.U32, dr.E32, dr.W2_32)
    cap = N + 1
    R = dr.R
    target = np.zeros((R, cap, dr.V), np.float32)
    ys = np.full((R, cap), -1, np.int32)
    sels = np.zeros((R, cap), np.int32)
    xs = np.full((R, cap), np.nan)
    trees = []
    for q in range(R):
        t = o.expand_tree(om, q, int(anchors[q]), 0.0, N, K, 0.0, seed)
        trees.append(t)
        n1 = t.n + 1
        _, vals = synth.make_target_rows(dr, q, t.depth[:n1], sigma, seed=seed, dtype="f32")
        target[q, :n1] = vals
        parent = np.full(cap, -1, np.int32)
        token = np.full(cap, -1, np.int32)
        parent[:n1] = t.parent
        token[:n1] = t.token
        y, sel = o.calib_labels(parent, token, t.n, target[q])
        ys[q], sels[q] = y, sel
        xs[q, 1:n1] = o.logit_q0(t.log_q0[1:n1].astype(np.float32).astype(np.float64))
    return trees, target, ys, sels, xs


def test_calib_labels_match_oracle(torch):
    """Greedy labels of oracle-built trees (the paper's instrumented round: N=28, K=8, T=0), from
    target rows U-row + N(0, 1): y and sel bit-exact, x within 1e-6 relative."""
    from paper_2609_22098_amd import binding
    dr = synth.make_drafter(3000, 8, 32, R=8, dtype="f32", u_sigma=2.5, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.3, seed=21)
    anchors, _, _ = synth.make_controls(dr.R, dr.V, 0.0, seed=21)
    N, K = 28, 8
    trees, target, ys, sels, xs = _oracle_round(dr, anchors, N, K, 1.0, 5)
    ht = binding.HostTree.empty(dr.R, N + 1)
    for q, t in enumerate(trees):
        n1 = t.n + 1
        ht.n[q] = t.n
        ht.parent[q, :n1] = t.parent
        ht.token[q, :n1] = t.token
        ht.depth[q, :n1] = t.depth
        ht.log_q0[q, :n1] = t.log_q0
    x, y, sel = binding.calib_labels(ht, torch.from_numpy(target).cuda())
    x, y, sel = x.cpu().numpy(), y.cpu().numpy(), sel.cpu().numpy()
    assert np.array_equal(y, ys)
    assert np.array_equal(sel, sels)
    fin = np.isfinite(xs)
    assert np.array_equal(np.isfinite(x), fin)
    assert np.allclose(x[fin], xs[fin], rtol=1e-6, atol=1e-6)
    print(f"labels: {int((ys >= 0).sum())} edges, {int(sels.sum())} ancestors-accepted, "
          f"accepted rate {float(ys[sels == 1].mean()):.3f}")
    assert 0 < sels.sum() < (ys >= 0).sum()


def test_calib_round_end_to_end(torch):
    """A whole calibration round on the device: greedy trees (ts_build_tree), labels, fit.  It is
    compared with the oracle's own round (its trees, labels and fit) on the same inputs, and the fit
    satisfies the score equation: mean prediction = acceptance rate on the fitted edges."""
    from paper_2609_22098_amd import binding
    dr = synth.make_drafter(3000, 8, 32, R=16, dtype="f32", u_sigma=2.5, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.3, seed=22)
    anchors, _, _ = synth.make_controls(dr.R, dr.V, 0.0, seed=22)
    N, K, sigma, seed = 28, 8, 1.0, 6
    _, target, ys, sels, xs = _oracle_round(dr, anchors, N, K, sigma, seed)
    m = (sels == 1) & np.isfinite(xs)
    ra, rb, _, _ = o.platt_fit(xs[m], ys[m])
    dd = binding.drafter_from_host(dr)
    tree = binding.build_tree(dd, anchors, np.zeros(dr.R, np.float32), N, K, 0.0, seed)
    gt = np.zeros((dr.R, N + 1, dr.V), np.float32)
    for q in range(dr.R):
        n1 = int(tree.n[q]) + 1
        _, vals = synth.make_target_rows(dr, q, tree.depth[q, :n1], sigma, seed=seed, dtype="f32")
        gt[q, :n1] = vals
    x, y, sel = binding.calib_labels(tree, torch.from_numpy(gt).cuda())
    ga, gb, gnll, steps = binding.calib_fit(x.reshape(-1), y.reshape(-1), sel.reshape(-1))
    xh, yh, sh = x.cpu().numpy(), y.cpu().numpy(), sel.cpu().numpy()
    mm = (sh == 1) & np.isfinite(xh)
    p = 1.0 / (1.0 + np.exp(-(ga * xh[mm].astype(np.float64) + gb)))
    print(f"round: {int(mm.sum())} fitted edges, device (a, b) = ({ga:.4f}, {gb:.4f}) in {steps} steps, "
          f"oracle ({ra:.4f}, {rb:.4f})")
    assert abs(float(np.mean(p)) - float(np.mean(yh[mm]))) < 1e-4
    # the same trees (up to near-ties of the tree building) give the same labels and fit
    om = o.Model(dr.U32, dr.E32, dr.W2_32)
    tally = Tally()
    for q in range(dr.R):
        ref = o.expand_tree(om, q, int(anchors[q]), 0.0, N, K, 0.0, seed)
        compare_tree(tree, q, ref, 0.0, dr.dtype, tally, tag=f"request {q}", T=0.0)
    assert not tally.failures, tally.failures[:3]
    if tally.near_ties == 0:
        assert np.array_equal(yh, ys) and np.array_equal(sh, sels)
        assert ga == pytest.approx(ra, rel=1e-4) and gb == pytest.approx(rb, rel=1e-4, abs=1e-5)
    else:
        assert abs(ga - ra) < 0.05 and abs(gb - rb) < 0.05
