"""The library's sliding-window monitor against the oracle's (host-only)."""
import numpy as np
import pytest

import paper_2607_22242_amd as S


def err(fn, *a):
    with pytest.raises(S.SchedError) as e:
        fn(*a)
    return e.value.name


@pytest.mark.parametrize("window", [1, 2, 3, 5, 16])
def test_monitor_matches_oracle(oracle_mod, window):
    O = oracle_mod
    n = 7
    rng = np.random.default_rng(window)
    lib, ref = S.Monitor(n, window), O.Monitor(n, window)
    profile = [[int(rng.integers(1, 10 ** 6)), int(rng.integers(1, 10 ** 6)),
                int(rng.integers(0, 10 ** 6)), int(rng.integers(0, 10 ** 4)), 100]
               for _ in range(n)]
    for r in range(60):
        modes = [int(x) for x in rng.integers(0, 3, n)]
        lat = [int(x) for x in rng.integers(-1, 2 * 10 ** 6, n)]
        lib.observe(modes, lat)
        ref.observe(modes, lat)
        mean, cnt = lib.averages()
        for v in range(n):
            for m in range(3):
                want = ref.mean(v, m)
                assert cnt[3 * v + m] == len(ref.obs[v][m])
                assert mean[3 * v + m] == (0 if want is None else want)
        assert lib.latencies(profile) == ref.latencies(profile), r


def test_monitor_validation():
    assert err(S.sched_monitor_create, 0, 3) == "SCHED_E_SIZE"
    assert err(S.sched_monitor_create, 41, 3) == "SCHED_E_SIZE"
    assert err(S.sched_monitor_create, 4, 0) == "SCHED_E_SIZE"
    m = S.Monitor(2, 4)
    assert err(m.observe, [0, 3], [1, 1]) == "SCHED_E_VALUE"
    assert err(m.observe, [-1, 0], [1, 1]) == "SCHED_E_VALUE"
    mean, cnt = m.averages()
    assert cnt == [0] * 6 and mean == [0] * 6  # nothing recorded on error
    m.observe([1, 1], [(1 << 62), (1 << 62) + 1])
    m.observe([1, 1], [(1 << 62), (1 << 62)])
    mean, _ = m.averages()
    assert mean[1] == 1 << 62 and mean[4] == (1 << 62) + 1  # 128-bit sum, half up
