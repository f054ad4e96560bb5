"""ts_expand_noalloc (the expansion in the library's per-GPU scratch array, no workspace, no
allocation in the call) against ts_expand on the same inputs: two calls in a row, the second
with a smaller frontier, both equal to ts_expand's outputs."""
import numpy as np
import pytest

from paper_2609_22098_amd import synth

pytestmark = pytest.mark.gpu

FIELDS = ("child_token", "child_log_q0", "child_log_qT", "child_log_surv", "slot_key", "rank_token",
          "rank_log_q0", "lse0", "lseT", "diag")


def _outputs(torch, P, k):
    i32, f32 = torch.int32, torch.float32
    shapes = dict(child_token=((P, k), i32), child_log_q0=((P, k), f32), child_log_qT=((P, k), f32),
                  child_log_surv=((P, k), f32), slot_key=((P, k), f32), rank_token=((P, k), i32),
                  rank_log_q0=((P, k), f32), lse0=((P,), f32), lseT=((P,), f32), diag=((P,), i32))
    # filled with a pattern, so that an output the call does not write shows up as a difference
    return {n: torch.full(s, -7, dtype=t, device="cuda") for n, (s, t) in shapes.items()}


def test_expand_noalloc_matches_expand():
    import torch
    from paper_2609_22098_amd import binding
    assert torch.cuda.is_available()
    binding.lib()
    dr = synth.make_drafter(151936, 4, 64, R=8, dtype="bf16", seed=11)
    dd = binding.drafter_from_host(dr)
    fr = synth.make_frontier(dr, per_depth=16, seed=11)  # 8 requests x 4 depths x 16 = 512 parents
    P1 = len(fr["token"])
    parents = binding.parents_to_device(fr["token"], fr["depth"], fr["request"], fr["log_surv"], fr["path"])
    k = 8
    # call 1: 512 parents, T = 0.7, sequential draws; call 2: the first 100, T = 1, Gumbel draws
    for P, T, sampler in ((P1, 0.7, "sequential"), (100, 1.0, "gumbel")):
        print(f"noalloc: P={P} T={T} sampler={sampler}", flush=True)
        want = binding.expand(dd, parents, P, k, T, 5, sampler=sampler)
        got = binding.expand_noalloc(dd, parents, P, k, T, 5, _outputs(torch, P, k), sampler=sampler)
        torch.cuda.synchronize()
        for name in FIELDS:
            a, b = got[name].cpu().numpy(), want[name].cpu().numpy()
            assert np.array_equal(a, b, equal_nan=True), (P, T, name)
        assert int(got["diag"].sum()) == 0
