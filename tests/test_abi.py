"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching a GPU (no compute calls here)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_22098_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x1000  # a non-null address that is never dereferenced


def _declared():
    txt = open(os.path.join(ROOT, "include", "treespark.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const char\*|size_t|int32_t)\s+(ts_\w+)\s*\(", txt, re.M)))


def test_library_exports_every_declared_symbol():
    declared = _declared()
    assert len(declared) == 19
    assert sorted(b.EXPORTED) == declared
    L = b.lib()
    for name in declared:
        assert hasattr(L, name), name
    assert b"gfx950" in L.ts_version()


def test_verify_level_counts_start_at_zero_and_check_pointers():
    L = b.lib()
    x = ctypes.c_int64(-1)
    assert L.ts_verify_level_counts(None, ctypes.byref(x), ctypes.byref(x)) == b.TS_EINVAL
    # no ts_verify call has run on this thread
    assert b.verify_level_counts() == (0, 0, 0)
    assert L.ts_verify_set_mode(2) == b.TS_EINVAL and L.ts_verify_set_mode(-1) == b.TS_EINVAL
    assert L.ts_verify_set_mode(1) == b.TS_OK and L.ts_verify_set_mode(0) == b.TS_OK


def test_release_without_state_touches_no_device():
    # nothing allocated on this thread yet: the release returns without a HIP call
    assert b.lib().ts_release_thread_state() == b.TS_OK


def _drafter(R=1, D=4, V=1000, r=16, dtype=b.TS_F32, null=False):
    return b.Drafter(None if null else FAKE, FAKE, FAKE, R, D, V, r, dtype)


def _expand(d, P=4, k=2, T=0.0, ws_bytes=1 << 30, out=True, parents=FAKE, sampler=0):
    o = b.ExpandOut(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None, None, None) if out else None
    return b.lib().ts_expand(ctypes.byref(d), parents, P, b.Calib(0.67, -0.46), k, T, 0, sampler,
                             ctypes.byref(o) if o else None, FAKE, ws_bytes, None)


def test_expand_rejects_bad_arguments():
    L = b.lib()
    assert _expand(_drafter(null=True)) == b.TS_EINVAL
    assert b"NULL" in L.ts_last_error()
    assert _expand(_drafter(V=0)) == b.TS_EINVAL
    assert _expand(_drafter(V=256 * 4096 + 1)) == b.TS_EUNSUPPORTED
    assert _expand(_drafter(D=17)) == b.TS_EUNSUPPORTED
    assert _expand(_drafter(r=24)) == b.TS_EUNSUPPORTED
    assert _expand(_drafter(r=16, dtype=b.TS_BF16)) == b.TS_EUNSUPPORTED
    assert _expand(_drafter(dtype=7)) == b.TS_EINVAL
    # model tensors must start 16-byte aligned (the kernels read them in 16-byte pieces)
    bad = _drafter()
    bad.W2 = FAKE + 8
    assert _expand(bad) == b.TS_EINVAL
    assert b"aligned" in L.ts_last_error()
    assert _expand(_drafter(), k=0) == b.TS_EINVAL
    assert _expand(_drafter(), k=17) == b.TS_EUNSUPPORTED
    assert _expand(_drafter(V=3), k=4) == b.TS_EINVAL
    assert _expand(_drafter(), T=-1.0) == b.TS_EINVAL
    assert _expand(_drafter(), T=float("inf")) == b.TS_EINVAL
    assert _expand(_drafter(), T=float("nan")) == b.TS_EINVAL
    assert _expand(_drafter(), sampler=2) == b.TS_EINVAL
    assert _expand(_drafter(), sampler=-1) == b.TS_EINVAL
    assert _expand(_drafter(), P=-1) == b.TS_EINVAL
    assert _expand(_drafter(), parents=None) == b.TS_EINVAL
    assert _expand(_drafter(), out=False) == b.TS_EINVAL
    assert _expand(_drafter(), ws_bytes=16) == b.TS_ENOSPACE
    # an empty frontier is valid and launches nothing
    assert _expand(_drafter(), P=0) == b.TS_OK


def test_workspace_sizes_are_monotone_and_positive():
    d = _drafter(V=151936, r=64, dtype=b.TS_BF16, D=16, R=64)
    L = b.lib()
    s0 = L.ts_expand_workspace_size(ctypes.byref(d), 2048, 8, 0.0)
    s1 = L.ts_expand_workspace_size(ctypes.byref(d), 2048, 8, 0.7)
    assert 0 < s0 < s1 < 64 << 20
    assert L.ts_expand_workspace_size(ctypes.byref(d), 0, 8, 0.0) == 0
    assert L.ts_build_tree_workspace_size(ctypes.byref(d), 64, 8, 0.7) > s1
    assert L.ts_verify_workspace_size(ctypes.byref(d), 65, 0.7) >= 64 * 151936 * 4


def test_build_tree_rejects_bad_arguments():
    L = b.lib()
    d = _drafter(R=2)
    tree = b.HostTree.empty(2, 9)
    s = tree.struct()
    anchor = np.array([1, 2], np.int32)
    theta = np.array([0.0, 0.1], np.float32)

    def call(anchor=anchor, theta=theta, N=8, K=2, T=0.0, ws=1 << 30, st=s, sampler=1, dev=None):
        return L.ts_build_tree(ctypes.byref(d), anchor.ctypes.data, theta.ctypes.data, N, 0, K,
                               b.Calib(0.67, -0.46), T, 0, sampler, ctypes.byref(st),
                               ctypes.byref(dev) if dev is not None else None, FAKE, ws, None)

    assert call(anchor=np.array([1, 5000], np.int32)) == b.TS_EINVAL
    assert call(theta=np.array([0.0, -0.1], np.float32)) == b.TS_EINVAL
    assert call(N=9) == b.TS_EINVAL       # cap 9 < N + 1
    assert call(N=-1) == b.TS_EINVAL
    assert call(K=0) == b.TS_EINVAL
    assert call(sampler=5) == b.TS_EINVAL
    assert call(ws=8) == b.TS_ENOSPACE
    bad = b.HostTree.empty(3, 9).struct()
    assert call(st=bad) == b.TS_EINVAL
    # a device tree must match out's R and cap and have every array
    assert call(dev=b.HostTree.empty(2, 10).struct()) == b.TS_EINVAL
    nulls = b.HostTree.empty(2, 9).struct()
    nulls.key = None
    assert call(dev=nulls) == b.TS_EINVAL


def test_verify_rejects_malformed_trees():
    L = b.lib()
    d = _drafter(R=1, D=4, V=100)
    tree = b.HostTree.empty(1, 5)
    tree.n[0] = 2
    tree.token[0, :3] = [1, 2, 3]
    tree.parent[0, :3] = [-1, 0, 0]
    tree.depth[0, :3] = [0, 1, 1]
    path = np.zeros((1, 16), np.int32); plen = np.zeros(1, np.int32); bonus = np.zeros(1, np.int32)

    def call(T=0.0, ws=1 << 30, tdt=b.TS_F32):
        s = tree.struct()
        return L.ts_verify(ctypes.byref(d), ctypes.byref(s), FAKE, tdt, T, 0, path.ctypes.data,
                           plen.ctypes.data, bonus.ctypes.data, FAKE, ws, None)

    tree.parent[0, 2] = 2  # a node cannot be its own parent
    assert call() == b.TS_EINVAL
    tree.parent[0, 2] = 0
    tree.depth[0, 2] = 2   # depth must be the parent's + 1
    assert call() == b.TS_EINVAL
    tree.depth[0, 2] = 1
    tree.token[0, 1] = 100  # token outside [0, V)
    assert call() == b.TS_EINVAL
    tree.token[0, 1] = 2
    assert call(tdt=9) == b.TS_EINVAL
    assert call(T=-0.5) == b.TS_EINVAL
    assert call(ws=4) == b.TS_ENOSPACE


def test_tree_mask_rejects_bad_arguments():
    L = b.lib()
    assert L.ts_tree_mask_words(1) == 1 and L.ts_tree_mask_words(32) == 1 and L.ts_tree_mask_words(33) == 2
    assert L.ts_tree_mask_words(0) == 0
    assert L.ts_tree_mask(FAKE, FAKE, 2, 0, None, FAKE, FAKE, None) == b.TS_EINVAL
    assert L.ts_tree_mask(FAKE, FAKE, 2, 4097, None, FAKE, FAKE, None) == b.TS_EINVAL
    assert L.ts_tree_mask(FAKE, FAKE, -1, 8, None, FAKE, FAKE, None) == b.TS_EINVAL
    assert L.ts_tree_mask(None, FAKE, 2, 8, None, FAKE, FAKE, None) == b.TS_EINVAL
    assert L.ts_tree_mask(FAKE, FAKE, 2, 8, None, None, FAKE, None) == b.TS_EINVAL
    assert L.ts_tree_mask(FAKE, FAKE, 0, 8, None, None, None, None) == b.TS_OK  # nothing to do


def _golden_ladder():
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "ladder.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                bs, T, want = line.split()
                rows.append((int(bs), float(T), want))
    return rows


def test_default_ladder_matches_the_paper():
    """The shipped ladder reproduces the paper's measured cells and its stated T=0 interpolation
    (tests/golden/ladder.txt); the chain sentinel gives K=1, N=block length, theta=0."""
    rungs = b.ladder_default()
    assert len(rungs) == 7
    for bs, T, want in _golden_ladder():
        theta, K, N, chain = b.ladder_lookup(rungs, bs, T, K=8, N=64, block_len=16)
        if want == "chain":
            assert chain and (theta, K, N) == (0.0, 1, 16), (bs, T)
        else:
            assert not chain and K == 8 and N == 64 and abs(theta - float(want)) < 1e-7, (bs, T, theta)


def test_ladder_lookup_rule_and_errors():
    """Nearest tabulated temperature (ties to the lower one), smallest covering bs_max, the widest
    rung above the table; bad arguments are rejected."""
    rungs = [(2, 0.0, 0.1), (10, 0.0, 0.2), (4, 1.0, 0.3), (8, 1.0, -1.0)]
    assert b.ladder_lookup(rungs, 1, 0.2, 4, 9, 5)[0] == pytest.approx(0.1)
    assert b.ladder_lookup(rungs, 3, 0.2, 4, 9, 5)[0] == pytest.approx(0.2)
    assert b.ladder_lookup(rungs, 50, 0.0, 4, 9, 5)[0] == pytest.approx(0.2)   # above the table
    assert b.ladder_lookup(rungs, 3, 0.5, 4, 9, 5)[0] == pytest.approx(0.2)    # tie -> T = 0 rungs
    assert b.ladder_lookup(rungs, 3, 0.8, 4, 9, 5)[0] == pytest.approx(0.3)
    assert b.ladder_lookup(rungs, 6, 2.0, 4, 9, 5) == (0.0, 1, 5, True)
    for args in [(0, 0.0, 4, 9, 5), (1, -1.0, 4, 9, 5), (1, 0.0, 0, 9, 5), (1, 0.0, 4, -1, 5),
                 (1, 0.0, 4, 9, 17), (1, float("nan"), 4, 9, 5)]:
        with pytest.raises(RuntimeError):
            b.ladder_lookup(rungs, *args)
    with pytest.raises(RuntimeError):
        b.ladder_lookup([], 1, 0.0, 4, 9, 5)


def test_calib_entry_points_reject_bad_arguments():
    L = b.lib()
    tree = b.HostTree.empty(2, 5)
    tree.n[:] = [1, 0]
    tree.parent[0, :2] = [-1, 0]
    tree.token[0, :2] = [3, 4]
    s = tree.struct()
    x = y = sel = out = FAKE
    ws = L.ts_calib_labels_workspace_size(2, 5)
    assert ws > 0 and L.ts_calib_labels_workspace_size(0, 5) == 0

    def labels(st=s, dtype=b.TS_F32, V=10, wsb=ws):
        return L.ts_calib_labels(ctypes.byref(st), FAKE, dtype, V, x, y, sel, FAKE, wsb, None)

    assert labels(V=4) == b.TS_EINVAL            # token 4 outside [0, V)
    assert labels(dtype=7) == b.TS_EINVAL
    assert labels(wsb=8) == b.TS_ENOSPACE
    bad = b.HostTree.empty(2, 5)
    bad.n[:] = [2, 0]
    bad.parent[0, :3] = [-1, 0, 2]                # a parent that is not before its child
    assert labels(st=bad.struct()) == b.TS_EINVAL
    assert L.ts_calib_fit(None, y, sel, 4, 10, 1e-9, out, None) == b.TS_EINVAL
    assert L.ts_calib_fit(x, y, sel, -1, 10, 1e-9, out, None) == b.TS_EINVAL
    assert L.ts_calib_fit(x, y, sel, 4, 0, 1e-9, out, None) == b.TS_EINVAL
    assert L.ts_calib_fit(x, y, sel, 4, 10, 0.0, out, None) == b.TS_EINVAL


def test_expand_noalloc_host_checks():
    """ts_expand_noalloc shares ts_expand's argument checks and refuses, before any launch, a
    launch whose plan needs more than its scratch array."""
    L = b.lib()

    def call(d, P=4, k=2, T=0.0, sampler=0, out=True):
        o = b.ExpandOut(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None, None, None) if out else None
        return L.ts_expand_noalloc(ctypes.byref(d), FAKE, P, b.Calib(0.67, -0.46), k, T, 0, sampler,
                                   ctypes.byref(o) if o else None, None)

    assert call(_drafter(null=True)) == b.TS_EINVAL
    assert call(_drafter(), out=False) == b.TS_EINVAL
    assert call(_drafter(), k=0) == b.TS_EINVAL
    assert call(_drafter(), sampler=5) == b.TS_EINVAL
    assert call(_drafter(), P=0) == b.TS_OK  # nothing to do, nothing launched
    # 60000 parents over V = 151936 with sequential draws: the block table alone is ~570 MB
    big = _drafter(V=151936, r=64, dtype=b.TS_BF16)
    assert call(big, P=60000, T=0.7, sampler=1) == b.TS_EUNSUPPORTED
    assert b"scratch" in L.ts_last_error()
