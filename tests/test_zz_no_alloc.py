"""sched_bruteforce_argmin_noalloc (no workspace: the library's fixed per-GPU
array) against sched_bruteforce_argmin with a caller workspace, bit-exact, on
consecutive calls whose inputs shrink: the array keeps the previous call's
contents, which must not leak into the next result."""
import pytest

import paper_2607_22242_amd as S
from workloads import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch


def with_workspace(P, lo, hi):
    return S.sched_bruteforce_argmin(P.handle, lo, hi, S.workspace([P.handle]))


def test_noalloc_matches_the_workspace_entry_point(torch_cuda):
    big = S.Problem.from_instance(synth.load(3))      # 3^19: 65,536 block partials
    small = S.Problem.from_instance(synth.load(1))    # 3^12: a few hundred blocks
    mid = S.Problem.from_instance(synth.load(2))      # 3^16, searched in part
    calls = [(big, 0, big.n_mappings), (small, 0, small.n_mappings),
             (mid, 12345, 2_000_000), (small, 100, 200)]
    for P, lo, hi in calls:
        print(f"noalloc: {P.n} tools [{lo}, {hi})", flush=True)
        got = S.sched_bruteforce_argmin_noalloc(P.handle, lo, hi)
        assert got == with_workspace(P, lo, hi), (P.n, lo, hi)
    # the same twice more, second call smaller than the first
    a = S.sched_bruteforce_argmin_noalloc(mid.handle, 0, mid.n_mappings)
    b = S.sched_bruteforce_argmin_noalloc(small.handle, 0, 1000)
    assert a == with_workspace(mid, 0, mid.n_mappings)
    assert b == with_workspace(small, 0, 1000)


def test_noalloc_rejects_bad_ranges_before_device_work(torch_cuda):
    P = S.Problem.from_instance(synth.load(0))
    for lo, hi in [(5, 5), (0, P.n_mappings + 1)]:
        with pytest.raises(S.SchedError) as e:
            S.sched_bruteforce_argmin_noalloc(P.handle, lo, hi)
        assert "SCHED_E_RANGE" in str(e.value)
