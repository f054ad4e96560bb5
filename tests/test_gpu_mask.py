"""GPU parity of ts_tree_mask against the oracle: bit-exact masks and position ids."""
import numpy as np
import pytest

from oracle import oracle as o
from paper_2609_22098_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_22098_amd import binding
    binding.lib()
    return t


def _check(torch, parent, n, cap, offsets):
    from paper_2609_22098_amd import binding
    R = len(n)
    dp = torch.from_numpy(np.ascontiguousarray(parent, np.int32)).cuda()
    dn = torch.from_numpy(np.ascontiguousarray(n, np.int32)).cuda()
    doff = torch.from_numpy(np.ascontiguousarray(offsets, np.int32)).cuda()
    mask, pos = binding.tree_mask(dp, dn, cap, doff)
    torch.cuda.synchronize()
    gm = mask.cpu().numpy().view(np.uint32)
    gp = pos.cpu().numpy()
    for q in range(R):
        want_m, want_p = o.tree_mask(parent[q], int(n[q]), cap, int(offsets[q]))
        assert np.array_equal(gm[q], want_m), q
        assert np.array_equal(gp[q], want_p), q


def _random_tree(rng, n, cap, deep):
    parent = np.full(cap, -1, np.int32)
    for i in range(1, n + 1):
        parent[i] = i - 1 if deep and rng.random() < 0.7 else rng.integers(0, i)
    return parent


def test_mask_of_built_trees(torch):
    """The benchmark's natural trees (64 requests, T=0.7) and deep sharp trees."""
    from paper_2609_22098_amd import binding
    w = synth.WORKLOADS[3]
    dr = synth.make_workload_drafter(3, seed=0)
    anchors, thetas, _ = synth.make_controls(dr.R, dr.V, w["theta"], seed=0)
    dd = binding.drafter_from_host(dr)
    tree = binding.build_tree(dd, anchors, thetas, w["N"], w["K"], 0.7, 0, sampler="sequential")
    _check(torch, tree.parent, tree.n, tree.cap, np.arange(dr.R) * 3)
    dr2 = synth.make_drafter(3000, 8, 32, R=6, dtype="bf16", u_sigma=3.0, planted=None, zipf=(6.0, 1.1),
                             ew_sigma=0.3, seed=3, u_scale=3.0)
    dd2 = binding.drafter_from_host(dr2)
    t2 = binding.build_tree(dd2, np.arange(6, dtype=np.int32), np.zeros(6, np.float32), 40, 3, 0.0, 0)
    assert t2.depth.max() >= 3
    _check(torch, t2.parent, t2.n, t2.cap, np.zeros(6, np.int32))


@pytest.mark.parametrize("cap", [1, 31, 32, 33, 65, 1000, 4096])
def test_mask_random_trees_and_edges(torch, cap):
    """Random trees across word boundaries up to the largest cap: chains, bushy trees, a root
    alone, trees that fill every row, and an unused request (n = -1)."""
    rng = np.random.default_rng(cap)
    R = 5
    parent = np.full((R, cap), -1, np.int32)
    n = np.array([cap - 1, (cap - 1) // 2, 0, cap - 1, -1], np.int32)
    for q in range(R):
        if n[q] > 0:
            parent[q] = _random_tree(rng, int(n[q]), cap, deep=(q == 3))
    want_n = np.maximum(n, 0)
    from paper_2609_22098_amd import binding
    dp = torch.from_numpy(parent).cuda()
    dn = torch.from_numpy(n).cuda()
    mask, pos = binding.tree_mask(dp, dn, cap)
    torch.cuda.synchronize()
    gm = mask.cpu().numpy().view(np.uint32)
    gp = pos.cpu().numpy()
    for q in range(R):
        if n[q] < 0:
            assert not gm[q].any() and np.all(gp[q] == -1)
            continue
        want_m, want_p = o.tree_mask(parent[q], int(want_n[q]), cap, 0)
        assert np.array_equal(gm[q], want_m), q
        assert np.array_equal(gp[q], want_p), q
