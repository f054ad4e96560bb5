"""GPU parity of ts_expand against the oracle, element by element."""
import numpy as np
import pytest

from oracle import oracle as o
from paper_2609_22098_amd import synth
from helpers import Tally, compare_parent, record

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_22098_amd import binding
    binding.lib()
    return t


def _expand_and_compare(torch, dr, fr, K, T, seed, sample=None, calib=(0.67, -0.46), tag="",
                        sampler="gumbel"):
    from paper_2609_22098_amd import binding
    dd = binding.drafter_from_host(dr)
    P = len(fr["token"])
    parents = binding.parents_to_device(fr["token"], fr["depth"], fr["request"], fr["log_surv"], fr["path"])
    out = binding.expand(dd, parents, P, K, T, seed, calib=calib, sampler=sampler)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items() if not k.startswith("_")}
    assert np.all(g["diag"] == 0), "recomputed candidate runs differ from the streaming pass"
    om = o.Model(dr.U32, dr.E32, dr.W2_32)
    idx = range(P) if sample is None else sample
    tally = Tally()
    for i in idx:
        ev = o.eval_node(om, int(fr["request"][i]), int(fr["token"][i]), int(fr["depth"][i]),
                         int(fr["path"][i]), T, seed, K, want_z=False, sampler=sampler)
        compare_parent(g, i, ev, float(fr["log_surv"][i]), T, K, dr.dtype, tally, a=calib[0], b=calib[1],
                       tag=f"{tag} parent {i}", sampler=sampler)
    print(f"{tag}: compared {tally.compared} parents, near-ties {tally.near_ties}, "
          f"max rel err {tally.max_err:.2e}")
    record(tag, "ts_expand parents", tally)
    assert not tally.failures, tally.failures[:5]
    # a near-tie cuts a parent's comparison short: most parents must be compared whole
    assert tally.compared >= 1 and tally.near_ties <= max(1, tally.compared // 4), (tally.compared, tally.near_ties)
    return g


@pytest.mark.parametrize("T", [0.0, 1.0, 0.6])
def test_tiny_workload_all_parents(torch, T):
    """V=4096, D=8, r=16, fp32 (the tiny oracle workload): every parent of a 3-per-depth frontier."""
    dr = synth.make_workload_drafter(0, seed=0)
    fr = synth.make_frontier(dr, per_depth=3, seed=1)
    _expand_and_compare(torch, dr, fr, 4, T, seed=0, tag=f"tiny T={T}")


@pytest.mark.parametrize("dtype,r,V", [("f32", 16, 1000), ("f32", 32, 4097), ("bf16", 32, 4097),
                                       ("bf16", 64, 100), ("f32", 64, 77), ("bf16", 128, 3000)])
@pytest.mark.parametrize("T", [0.0, 0.8])
def test_ragged_shapes(torch, dtype, r, V, T):
    """Vocabularies that are not multiples of the 16/64-token tiles, tiny vocabularies and a
    ragged parent count (37)."""
    dr = synth.make_drafter(V, 5, r, R=3, dtype=dtype, u_sigma=2.0, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.2, seed=7)
    fr = synth.make_frontier(dr, per_depth=3, seed=2)
    keep = np.arange(37)
    fr = {k: v[keep] for k, v in fr.items()}
    _expand_and_compare(torch, dr, fr, min(5, V), T, seed=3, tag=f"ragged {dtype} r={r} V={V} T={T}")


@pytest.mark.parametrize("dtype,r,V", [("bf16", 64, 30011), ("f32", 32, 5000)])
@pytest.mark.parametrize("T", [0.0, 1.3])
def test_max_siblings(torch, dtype, r, V, T):
    """K = 16 (the library's maximum) with the greedy order and Gumbel draws: the merge's
    threshold then takes the 16th largest recorded run key, and the candidate lists hold 16
    entries; a ragged vocabulary over many chunks and a ragged parent count (45)."""
    dr = synth.make_drafter(V, 6, r, R=3, dtype=dtype, u_sigma=2.0, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.2, seed=13)
    fr = synth.make_frontier(dr, per_depth=3, seed=4)
    fr = {k: v[:45] for k, v in fr.items()}
    _expand_and_compare(torch, dr, fr, 16, T, seed=9, tag=f"K=16 {dtype} r={r} V={V} T={T}")


@pytest.mark.parametrize("T", [0.0, 0.7])
def test_wide_frontier_blocks(torch, T):
    """A frontier of 700 parents (the 4-block-per-wave layout) with shared rows, bf16 r=64."""
    dr = synth.make_drafter(20000, 16, 64, R=22, dtype="bf16", seed=11)
    fr = synth.make_frontier(dr, per_depth=2, seed=3)
    sample = list(range(0, 704, 11))
    _expand_and_compare(torch, dr, fr, 8, T, seed=5, sample=sample, tag=f"wide T={T}")


def test_single_request_v128256_frontier(torch):
    """V=128256, D=16, r=64, bf16, T=0: the whole 64-parent frontier (4 per depth)."""
    dr = synth.make_workload_drafter(1, seed=0)
    fr = synth.make_frontier(dr, per_depth=4, seed=0)
    _expand_and_compare(torch, dr, fr, 8, 0.0, seed=0, tag="v128256")


def test_single_request_v151936_r256_sampling(torch):
    """V=151936, D=16, r=256, bf16, T=1: 128 parents, 24 sampled for the oracle."""
    dr = synth.make_workload_drafter(2, seed=0)
    fr = synth.make_frontier(dr, per_depth=8, seed=0)
    rng = np.random.default_rng(0)
    sample = sorted(rng.choice(128, 24, replace=False))
    _expand_and_compare(torch, dr, fr, 8, 1.0, seed=0, sample=sample, tag="v151936 r256 T=1")


def test_serving_2048_parent_frontier(torch):
    """64 requests, V=151936, r=64, bf16, T=0.7: the 2048-parent frontier timed by the bench,
    in the same launch configuration; 40 sampled parents against the oracle."""
    dr = synth.make_workload_drafter(3, seed=0)
    fr = synth.make_frontier(dr, per_depth=2, seed=0)
    assert len(fr["token"]) == 2048
    rng = np.random.default_rng(1)
    sample = sorted(rng.choice(2048, 40, replace=False))
    _expand_and_compare(torch, dr, fr, 8, 0.7, seed=0, sample=sample, tag="serving T=0.7")
    _expand_and_compare(torch, dr, fr, 8, 0.0, seed=0, sample=sample[:16], tag="serving T=0")


# ---------------------------------------------------------------- sequential draws

@pytest.mark.parametrize("T", [1.0, 0.6])
def test_sequential_tiny_workload_all_parents(torch, T):
    """Sequential draws (one 4096-token segment, 64 blocks), fp32: every parent of a 3-per-depth
    frontier of the tiny workload."""
    dr = synth.make_workload_drafter(0, seed=0)
    fr = synth.make_frontier(dr, per_depth=3, seed=1)
    _expand_and_compare(torch, dr, fr, 4, T, seed=2, tag=f"sequential tiny T={T}", sampler="sequential")


@pytest.mark.parametrize("dtype,r,V", [("f32", 16, 1000), ("f32", 32, 4097), ("bf16", 32, 8193),
                                       ("bf16", 64, 100), ("f32", 64, 77), ("bf16", 128, 12000)])
def test_sequential_ragged_shapes(torch, dtype, r, V):
    """Sequential draws over ragged vocabularies: partial last block and segment, several
    segments, vocabularies smaller than one block; K up to 12 (draws cross blocks and segments)."""
    dr = synth.make_drafter(V, 5, r, R=3, dtype=dtype, u_sigma=1.0, planted=None, zipf=None,
                            ew_sigma=0.2, seed=8)
    fr = synth.make_frontier(dr, per_depth=3, seed=2)
    keep = np.arange(37)
    fr = {k: v[keep] for k, v in fr.items()}
    _expand_and_compare(torch, dr, fr, min(12, V), 1.7, seed=4, tag=f"sequential ragged {dtype} r={r} V={V}",
                        sampler="sequential")


def test_sequential_v151936_r256_T1(torch):
    """V=151936, r=256, bf16, T=1 (one sum serves lse0 and lseT): 24 sampled parents of 128."""
    dr = synth.make_workload_drafter(2, seed=0)
    fr = synth.make_frontier(dr, per_depth=8, seed=0)
    rng = np.random.default_rng(2)
    sample = sorted(rng.choice(128, 24, replace=False))
    _expand_and_compare(torch, dr, fr, 8, 1.0, seed=1, sample=sample, tag="sequential v151936 r256 T=1",
                        sampler="sequential")


def test_sequential_serving_2048_parent_frontier(torch):
    """The benchmark's launch: 64 requests, V=151936 (38 segments), r=64, bf16, T=0.7, 2048
    parents; 48 sampled parents against the oracle."""
    dr = synth.make_workload_drafter(3, seed=0)
    fr = synth.make_frontier(dr, per_depth=2, seed=0)
    rng = np.random.default_rng(3)
    sample = sorted(rng.choice(2048, 48, replace=False))
    _expand_and_compare(torch, dr, fr, 8, 0.7, seed=0, sample=sample, tag="sequential serving T=0.7",
                        sampler="sequential")


def test_sequential_large_vocabulary(torch):
    """V = 170000 (42 segments): the block table stays in the workspace instead of LDS."""
    dr = synth.make_drafter(170000, 3, 32, R=1, dtype="bf16", u_sigma=1.5, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.1, seed=12)
    fr = synth.make_frontier(dr, per_depth=4, seed=6)
    _expand_and_compare(torch, dr, fr, 8, 0.8, seed=5, tag="sequential V=170000", sampler="sequential")


@pytest.mark.parametrize("T", [0.7, 1.0])
def test_sequential_segment_slots(torch, T):
    """V = 300000: 74 segments, more than one per lane, so the segment pick scans several slots per
    lane (and the block table stays in the workspace); 40 parents against the oracle."""
    dr = synth.make_drafter(300000, 3, 32, R=2, dtype="bf16", u_sigma=1.5, planted=None, zipf=(6.0, 1.1),
                            ew_sigma=0.1, seed=13)
    fr = synth.make_frontier(dr, per_depth=7, seed=8)
    assert len(fr["token"]) == 42
    _expand_and_compare(torch, dr, fr, 8, T, seed=6, sample=list(range(40)), tag=f"sequential V=300000 T={T}",
                        sampler="sequential")


@pytest.mark.parametrize("T", [0.02, 0.2])
def test_sequential_low_temperature(torch, T):
    """Low temperatures: the remaining mass after the first draws is tiny next to the drawn
    tokens' mass, so every level renormalises against its own maximum; all parents against the
    oracle across three segments."""
    dr = synth.make_drafter(9000, 4, 32, R=2, dtype="bf16", u_sigma=3.0, planted=None, zipf=None,
                            ew_sigma=0.2, seed=9)
    fr = synth.make_frontier(dr, per_depth=4, seed=5)
    _expand_and_compare(torch, dr, fr, 8, T, seed=3, tag=f"sequential low T={T}", sampler="sequential")


@pytest.mark.parametrize("dtype,r,V", [("f32", 16, 1000), ("bf16", 32, 9000)])
@pytest.mark.parametrize("T,sampler", [(0.0, "sequential"), (0.7, "sequential"), (0.7, "gumbel")])
def test_masked_logits_fewer_than_k(torch, dtype, r, V, T, sampler):
    """Rows of U that are -inf except for 3-5 tokens (masked vocabularies) with k = 8: the
    sequential sampler's draws past the finite tokens are empty (token -1, -inf values), the
    greedy and Gumbel orders continue with -inf tokens by id, all as the oracle gives."""
    dr = synth.make_drafter(V, 3, r, R=2, dtype=dtype, u_sigma=2.0, planted=None, zipf=None,
                            ew_sigma=0.2, seed=14)
    rng = np.random.default_rng(15)
    ninf = np.uint16(0xFF80) if dtype == "bf16" else np.float32(-np.inf)
    for q in range(dr.R):
        for d in range(dr.D):
            keep = rng.choice(V, int(rng.integers(3, 6)), replace=False)
            row = dr.U[q, d].copy()
            dr.U[q, d] = ninf
            dr.U[q, d, keep] = row[keep]
            dr.U32[q, d] = -np.inf
            dr.U32[q, d, keep] = (synth.bf16_bits_to_f32(row[keep]) if dtype == "bf16" else row[keep])
    fr = synth.make_frontier(dr, per_depth=4, seed=3)
    g = _expand_and_compare(torch, dr, fr, 8, T, seed=2, tag=f"masked {dtype} T={T} {sampler}",
                            sampler=sampler)
    if T > 0 and sampler == "sequential":
        empty = g["child_token"] < 0
        assert empty.any() and np.all(np.isneginf(g["child_log_q0"][empty]))
        assert np.all(np.isneginf(g["child_log_surv"][empty])) and np.all(np.isneginf(g["slot_key"][empty]))


def test_deterministic_and_invalid_parents(torch):
    """Two calls give bitwise-identical outputs; a parent with an out-of-range field gets
    token -1 and NaN values without disturbing the others."""
    from paper_2609_22098_amd import binding
    dr = synth.make_drafter(5000, 6, 32, R=2, dtype="bf16", seed=4)
    fr = synth.make_frontier(dr, per_depth=3, seed=4)
    fr["token"][5] = 5000      # out of range
    fr["depth"][9] = 6         # out of range
    fr["request"][11] = -1     # out of range
    dd = binding.drafter_from_host(dr)
    P = len(fr["token"])
    parents = binding.parents_to_device(fr["token"], fr["depth"], fr["request"], fr["log_surv"], fr["path"])
    outs = []
    for _ in range(2):
        out = binding.expand(dd, parents, P, 6, 0.9, 17)
        torch.cuda.synchronize()
        outs.append({k: v.cpu().numpy() for k, v in out.items() if not k.startswith("_")})
    for k in outs[0]:
        assert np.array_equal(outs[0][k].view(np.uint8), outs[1][k].view(np.uint8)), k
    for bad in (5, 9, 11):
        assert np.all(outs[0]["child_token"][bad] == -1)
        assert np.all(np.isnan(outs[0]["child_log_q0"][bad]))
    good = [i for i in range(P) if i not in (5, 9, 11)]
    assert np.all(outs[0]["child_token"][good] >= 0)
    # the valid parents still match the oracle
    fr_ok = {k: v[good] for k, v in fr.items()}
    _expand_and_compare(torch, dr, fr_ok, 6, 0.9, 17, sample=list(range(0, len(good), 4)), tag="valid rows")
