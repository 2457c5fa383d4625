"""The seeded instance generator and the committed instance files."""
import json
import os

import pytest

from workloads import synth


@pytest.mark.parametrize("c", [0, 1, 2, 3, 4, 5])
def test_committed_instances_regenerate_exactly(c):
    with open(synth.instance_path(c)) as f:
        assert f.read() == synth.dumps(synth.BUILDERS[c]())


def test_splitmix64_reference_values():
    # First outputs of SplitMix64 seeded with 0 (published test vector of the
    # generator: 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F).
    g = synth.SplitMix64(0)
    assert [g.next_u64() for _ in range(3)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def acyclic(n, edges):
    indeg = [0] * n
    succ = [[] for _ in range(n)]
    for u, v in edges:
        succ[u].append(v)
        indeg[v] += 1
    stack = [v for v in range(n) if indeg[v] == 0]
    seen = 0
    while stack:
        u = stack.pop()
        seen += 1
        for v in succ[u]:
            indeg[v] -= 1
            if indeg[v] == 0:
                stack.append(v)
    return seen == n


def check_tools(tools, mem_lo, mem_hi):
    for g, c, l, x, m in tools:
        assert 1000 <= g <= 1000000
        assert c >= 1
        assert 0 <= l and 0 <= x
        assert mem_lo <= m <= mem_hi


def test_config_shapes():
    c0 = synth.load(0)
    assert c0["n_tools"] == 8 and c0["edges"] == [[v, v + 1] for v in range(7)]
    check_tools(c0["tools"], 512, 24576)
    c1 = synth.load(1)
    assert c1["n_tools"] == 12 and acyclic(12, c1["edges"])
    assert all(u // 4 + 1 == v // 4 for u, v in c1["edges"])
    c2 = synth.load(2)
    assert c2["n_tools"] == 16 and acyclic(16, c2["edges"])
    check_tools(c2["tools"], 4096, 24576)
    assert c2["vram_budget_mib"] == sum(t[4] for t in c2["tools"]) // 4
    c3 = synth.load(3)
    assert c3["n_tools"] == 19 and acyclic(19, c3["edges"])
    assert len({tuple(e) for e in c3["edges"]}) == len(c3["edges"])
    p = c3["pcie_tool"]
    assert c3["tools"][p][3] >= 5 * c3["tools"][p][0]
    for v in c3["neutral_tools"]:
        g, c = c3["tools"][v][:2]
        assert 0.9 * g - 1 <= c <= 1.1 * g + 1
    for c in range(4):
        assert synth.load(c)["contention_q16"] == [65536, 88474, 117965, 157286]


def test_binary_config_shape():
    c5 = synth.load(5)
    assert c5["n_tools"] == 32 and acyclic(32, c5["edges"])
    assert sorted(set(c5["allowed"])) == [1, 3] and c5["allowed"].count(1) == 2
    assert [v for v in range(32) if c5["allowed"][v] == 1] == c5["neutral_tools"]
    assert c5["vram_budget_mib"] == sum(t[4] for t in c5["tools"])
    assert 2 ** c5["allowed"].count(3) == 1 << 30


def test_batch_config_shape():
    b = synth.load(4)
    sc = b["scenarios"]
    assert len(sc) == 13
    for s, inst in enumerate(sc):
        assert inst["n_tools"] == 14 and acyclic(14, inst["edges"])
        assert len(inst["replicas"]) == 64
        if 4 <= s <= 8:
            assert inst["edges"] == []
            assert inst["vram_budget_mib"] == sum(t[4] for t in inst["tools"])
        for rep in inst["replicas"]:
            for (g, c, l, x), base in zip(rep, inst["tools"]):
                assert 0.8 * base[0] - 1 <= g <= 1.2 * base[0] + 1
                assert 0.8 * base[1] - 1 <= c <= 1.2 * base[1] + 1
                assert 0.8 * base[2] - 1 <= l <= 1.2 * base[2] + 1
                assert 0.8 * base[3] - 1 <= x <= 1.2 * base[3] + 1
    assert 13 * 64 * 3 ** 14 == 3979430208


def test_expected_file_matches_instances():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "expected_configs.json")
    with open(path) as f:
        exp = json.load(f)
    for key, entry in exp.items():
        c = int(key[len("config"):])
        assert entry["instance_sha256"] == synth.sha256_of(c)


def test_counted_work_per_mapping():
    """tests/golden/ops_per_mapping.json (tests/golden/count_ops.py, oracle
    only): where every mapping is feasible the count equals the work of a
    complete evaluation; elsewhere it lies below it."""
    import math
    with open(os.path.join(os.path.dirname(__file__), "golden", "ops_per_mapping.json")) as f:
        ops = json.load(f)

    def complete(inst):
        n, e = len(inst["tools"]), len(inst["edges"])
        return n * (3.0 * e / n + 14.0 + 2.0 * math.log2(n)) + 6.0

    for c in (0, 5):
        assert ops[f"config{c}"]["feasible_fraction"] == 1.0
        assert abs(ops[f"config{c}"]["ops_per_mapping"] - complete(synth.load(c))) < 1e-9
    for c in (1, 2, 3):
        rec = ops[f"config{c}"]
        assert 0.3 < rec["feasible_fraction"] < 1.0
        assert 6.0 < rec["ops_per_mapping"] < complete(synth.load(c))
