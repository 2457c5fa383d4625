"""Pins of the CPU oracle against facts it does not compute itself.

Sources of truth, none of which is the oracle:
  * the paper's printed scenarios and oracle mappings (tests/golden);
  * hand-solved tiny instances (N = 1..3) worked out below, one rule each;
  * closed forms: serial chains, all-CPU longest paths, all-gpu_now fan-outs;
  * a Viterbi dynamic programme for chains;
  * a tick-by-tick simulator (time advanced by 1 us) on tiny instances;
  * invariants of every returned schedule (precedence, VRAM, queue order).
"""
import itertools
import json
import os

import pytest

from workloads import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
INF = (1 << 63) - 1
F2 = [65536, 98304]  # 1.0x, 1.5x


def q16(b, f):
    return (b * f + 32768) >> 16


def mk(O, tools, edges, budget, table=F2):
    return O.Problem(tools, edges, table, budget)


# ---------------------------------------------------------------------------
# Hand-solved tiny instances.  Rows are (gpu, cpu, load, xfer, mem).


def test_single_tool_modes_and_tie_break(oracle_mod):
    O = oracle_mod
    # gpu_queue pays load-in: 100 + 50 (tau of Section 2.1).
    P = mk(O, [[100, 300, 50, 0, 10]], [], 16)
    assert [P.eval_index(x) for x in range(3)] == [300, 100, 150]
    assert P.argmin() == (1, 100)
    # A GPU mode whose footprint exceeds the budget is infeasible, both for
    # an immediate start (out of memory) and for a queued one (never fits).
    P = mk(O, [[100, 300, 50, 0, 10]], [], 5)
    assert [P.eval_index(x) for x in range(3)] == [300, INF, INF]
    assert P.argmin() == (0, 300)
    # Equal makespans: the lower index wins.
    P = mk(O, [[100, 100, 50, 0, 10]], [], 16)
    assert [P.eval_index(x) for x in range(3)] == [100, 100, 150]
    assert P.argmin() == (0, 100)


CHAIN2 = [[100, 300, 50, 20, 10], [200, 250, 40, 30, 10]]


def test_chain_of_two_consumer_pays_transfer(oracle_mod):
    O = oracle_mod
    P = mk(O, CHAIN2, [[0, 1]], 16)
    got = [P.eval_index(x) for x in range(9)]
    # idx1 = gpu_now then cpu: 100 + xfer of the consumer (30) + 250 = 380
    # (charging the producer's 20 would give 370).  gpu_now -> gpu_queue
    # (idx7) stays on one device: 100 + 240, no transfer.
    assert got == [550, 380, 430, 530, 300, 350, 570, 340, 390]
    assert P.argmin() == (4, 300)


def test_release_before_acquire(oracle_mod):
    O = oracle_mod
    # Both tools on gpu_now need 10 MiB each with a 16 MiB budget; the
    # second starts exactly when the first finishes, so it must fit.
    P = mk(O, CHAIN2, [[0, 1]], 16)
    assert P.eval_index(4) == 300


def test_two_parallel_tools(oracle_mod):
    O = oracle_mod
    P = mk(O, CHAIN2, [], 16)
    # idx4: both gpu_now at t=0 need 20 > 16 MiB -> out of memory.
    # idx5: tool 1 gpu_now holds 10 MiB, queued tool 0 (10 MiB) waits for
    #       the release at 200, then runs alone: 200 + 150.
    # idx7: tool 0 gpu_now [0,100), queued tool 1 admitted at 100: 100+240.
    assert [P.eval_index(x) for x in range(9)] == [300, 250, 250, 300, INF, 350,
                                                  300, 340, 390]
    P = mk(O, CHAIN2, [], 32)
    # With room for both: idx4 co-starts two gpu_now tools, k=2 -> 1.5x:
    # 150 and 300.  idx5 admits the queued tool beside the immediate one
    # (k=2): 225 and 300.  idx7: 150 and 360.
    assert [P.eval_index(x) for x in range(9)] == [300, 250, 250, 300, 300, 300,
                                                  300, 360, 390]
    assert P.argmin() == (1, 250)


def test_contention_fixed_at_start_counts_costarters(oracle_mod):
    O = oracle_mod
    # Two gpu_now tools co-start: both get k=2 for their whole life:
    # 400*1.5 = 600 (processor sharing would give 450, counting the
    # co-starter only for the later one would give 400).
    P = mk(O, [[400, 5000, 50, 0, 1], [100, 5000, 50, 0, 1]], [], 16)
    assert P.eval_index(4) == 600


def test_queue_is_fifo_on_ready_time_then_index(oracle_mod):
    O = oracle_mod
    tools = [[100, 5000, 50, 0, 10], [200, 5000, 40, 0, 10], [5000, 500, 0, 10, 1]]
    P = mk(O, tools, [[0, 2]], 16)
    # idx 8 = (gpu_queue, gpu_queue, cpu).  Tools 0 and 1 are both ready at 0;
    # tool 0 (lower index) runs [0,150), tool 1 [150,390); tool 2 is ready at
    # 150 + 10 (device change) and runs [160,660).  The other order gives 900.
    assert P.eval_index(8) == 660


def test_queue_admits_into_free_vram_beside_running_tools(oracle_mod):
    O = oracle_mod
    # Tool 0 gpu_now (10 MiB) leaves 6 MiB; queued tool 1 (5 MiB) fits and is
    # admitted at t=0 beside it, so both run with k=2: 400*1.5 = 600.  (A
    # queue that waits for an idle GPU would give 400 + 150 = 550.)
    P = mk(O, [[400, 5000, 50, 0, 10], [100, 5000, 50, 0, 5]], [], 16)
    assert P.eval_index(7) == 600


def test_contention_table_clamps(oracle_mod):
    O = oracle_mod
    # Three co-starting gpu_now tools with a two-level table: k=3 uses 1.5x.
    P = mk(O, [[100, 5000, 50, 0, 1]] * 3, [], 100)
    assert P.eval_index(1 + 3 + 9) == 150


def test_running_queued_tool_holds_vram(oracle_mod):
    O = oracle_mod
    # Tool 0 is queued and admitted at t=0 (10 MiB, runs [0,150)).  Tool 2 is
    # a 50 us CPU task feeding tool 1 (gpu_now, 10 MiB, no transfer cost).
    # At t=50 the running queued tool still holds its 10 MiB: 20 > 16.
    tools = [[100, 5000, 50, 0, 10], [100, 5000, 50, 0, 10], [5000, 50, 0, 0, 1]]
    P = mk(O, tools, [[2, 1]], 16)
    assert P.eval_index(2 + 3 * 1 + 9 * 0) == INF
    # With 20 MiB both fit: tool 1 starts at 50 beside the queued tool (k=2).
    P = mk(O, tools, [[2, 1]], 20)
    assert P.eval_index(2 + 3 * 1) == 50 + 150


def test_cpu_tools_are_not_slowed_and_not_counted(oracle_mod):
    O = oracle_mod
    # A CPU tool running beside one gpu_now tool: the GPU tool sees k=1.
    P = mk(O, [[100, 5000, 50, 0, 1], [100, 70, 50, 0, 1]], [], 100)
    assert P.eval_index(1 + 3 * 0) == 100


def test_rounding_is_half_up(oracle_mod):
    O = oracle_mod
    # 3 * 1.5 = 4.5 -> 5 ; 1 * 1.5 = 1.5 -> 2 ; 5 * 1.5 = 7.5 -> 8
    P = mk(O, [[3, 100, 0, 0, 1], [1, 100, 0, 0, 1]], [], 10)
    ms, s, c = P.schedule([1, 1])
    assert c == [5, 2] and ms == 5
    P = mk(O, [[5, 100, 0, 0, 1], [1, 100, 0, 0, 1]], [], 10, [65536, 98303])
    # 5 * 98303 / 65536 = 7.4998 -> 7
    assert P.schedule([1, 1])[2] == [7, 1]


# ---------------------------------------------------------------------------
# Paper scenarios.


def load_paper():
    with open(os.path.join(GOLDEN, "paper_scenarios.json")) as f:
        return json.load(f)


def paper_problem(O, d, s):
    edges = d["diamond_edges"] if s["topology"] == "diamond" else []
    return O.Problem(s["tools"], edges, d["contention_q16"], s["budget"])


@pytest.mark.parametrize("name", ["S2", "S4", "S5", "S13"])
def test_paper_oracle_mapping_reproduced(oracle_mod, name):
    O = oracle_mod
    d = load_paper()
    s = d["scenarios"][name]
    P = paper_problem(O, d, s)
    bi, bm = P.argmin(threads=1)
    assert O.modes_of(bi, 4) == s["paper_oracle"], name


def test_paper_s5_and_s13_makespans(oracle_mod):
    O = oracle_mod
    d = load_paper()
    P5 = paper_problem(O, d, d["scenarios"]["S5"])
    # S5 oracle: A, B, D on gpu_now co-start (k=3, 1.8x); C on CPU for 739 ms
    # hides behind them: A = round(370000 * 117965 / 2^16) = 666001 < 739000.
    assert P5.argmin() == (31, 739000)
    assert q16(370000, 117965) == 666001
    # All-GPU (k=4, 2.4x) is slower: ocr_x2 = round(370000*157286/2^16).
    assert P5.eval_index(40) == q16(370000, 157286) == 887998
    P13 = paper_problem(O, d, d["scenarios"]["S13"])
    # S13 oracle: A, C gpu_now (1044 MiB, k=2) ; B queued, admitted when C
    # releases 417 MiB at round(136000*1.35); D on CPU.
    c_end = q16(136000, 88474)
    assert c_end == 183601
    assert P13.argmin() == (16, c_end + q16(153000 + 245000, 88474))
    assert P13.argmin()[1] == 720903


def test_paper_known_divergences(oracle_mod):
    """S1 and S3: fixed-at-start contention disagrees with the measurement.

    S1: llama_1b (447 ms) co-starting with sentiment (7 ms) is charged 1.35x
    for its whole run, so putting sentiment on the GPU looks worse here than
    on the paper's hardware.  S3: web_search is 128 ms on GPU vs 127 ms on CPU,
    a 1 ms, noise-level difference.
    """
    O = oracle_mod
    d = load_paper()
    for name, idx, ms in [("S1", 4, 612000), ("S3", 4, 176000)]:
        s = d["scenarios"][name]
        P = paper_problem(O, d, s)
        assert P.argmin() == (idx, ms)
        assert O.modes_of(idx, 4) != s["paper_oracle"]


def test_paper_s13_memory_feasibility(oracle_mod):
    O = oracle_mod
    d = load_paper()
    s = d["scenarios"]["S13"]
    P = paper_problem(O, d, s)
    mem = [t[4] for t in s["tools"]]
    for m in d["s13_memory"]["infeasible"]:
        assert P.eval_index(O.index_of(m)) == INF
    for m in d["s13_memory"]["feasible"]:
        assert P.eval_index(O.index_of(m)) < INF
    for key, total in d["s13_memory"]["gpu_now_sum_at_t0"].items():
        modes = [int(c) for c in key.split(",")]
        ms, start, fin = P.schedule(modes)
        at0 = sum(mem[v] for v in range(4) if modes[v] == 1 and start[v] == 0)
        assert at0 == total
    # Section 4.5 with Table 1 footprints: 656 + 442 = 1098 <= 1100.
    assert 656 + 442 <= s["budget"] < 656 + 486 + 442


def test_paper_s13_whatif_block(oracle_mod):
    """Round-3 what-if block of S13 around the round-2 mapping.

    The model gives every printed probe the paper's feasibility, puts the
    two swaps in the paper's order (C<->B before C<->A) and the single moves
    to CPU above the base, and the winning swap is the brute-force optimum.
    The paper measured D->gpu_queue 435 ms below the base; the model, which
    has no loading overlap, puts it above: a recorded divergence.
    """
    O = oracle_mod
    d = load_paper()
    s = d["scenarios"]["S13"]
    w = d["s13_whatif"]
    P = paper_problem(O, d, s)
    mem = [t[4] for t in s["tools"]]
    base = O.index_of(w["base"])
    probes = O.reprobes(P, base)
    assert probes[0]["kind"] == 0 and probes[0]["index"] == base
    by_key = {(p["tool"], p["mode"], p["swap_tool"]): p for p in probes}
    for e in w["printed"]:
        p = by_key[(e["tool"], e["mode"], e.get("swap_tool", -1))]
        assert (p["makespan_us"] < INF) == e["feasible"], e
        if "full" in e:
            assert p["index"] == O.index_of(e["full"])
    # Fan-out: every gpu_now tool starts at 0, so a move is infeasible exactly
    # when the gpu_now footprints exceed the budget.
    for p in probes:
        modes = O.modes_of(p["index"], 4)
        over = sum(mem[v] for v in range(4) if modes[v] == 1) > s["budget"]
        assert (p["makespan_us"] == INF) == over, p
    sw = {e.get("swap_tool"): e for e in w["printed"] if "swap_tool" in e}
    assert (by_key[(2, 1, 1)]["makespan_us"] < by_key[(2, 1, 0)]["makespan_us"]) == \
        (sw[1]["e2e_ms"] < sw[0]["e2e_ms"])
    base_ms = probes[0]["makespan_us"]
    assert by_key[(1, 0, -1)]["makespan_us"] > by_key[(0, 0, -1)]["makespan_us"] > base_ms
    assert by_key[(2, 1, 1)]["index"] == P.argmin()[0] == O.index_of(s["paper_oracle"])
    assert by_key[(3, 2, -1)]["makespan_us"] > base_ms  # divergence, see docstring
    # Both gpu_now moves that overflow (C and D) get one swap per gpu_now tool.
    assert [(p["tool"], p["swap_tool"]) for p in probes if p["kind"] == 2] == \
        [(2, 0), (2, 1), (3, 0), (3, 1)]
    assert len(probes) == 1 + 2 * 4 + 4


@pytest.mark.parametrize("seed", range(6))
def test_reprobe_neighbourhood_by_brute_force(oracle_mod, seed):
    """The probe set equals its definition checked over every mapping: all
    mappings one digit away from the base, plus those two digits away that
    put an overflowing gpu_now move i beside j moved gpu_now -> gpu_queue."""
    O = oracle_mod
    n = 5
    inst = synth.random_instance(9100 + seed, n, "random", tight=True)
    P = O.Problem(inst["tools"], inst["edges"], inst["contention_q16"], inst["vram_budget_mib"])
    allms = P.eval_many(range(3 ** n), threads=1)
    for base in (0, 3 ** n - 1, 121, 40 + 81 * seed % 243, 200):
        b = O.modes_of(base, n)
        probes = O.reprobes(P, base)
        want1, want2 = set(), set()
        for x in range(3 ** n):
            m = O.modes_of(x, n)
            diff = [v for v in range(n) if m[v] != b[v]]
            if len(diff) == 1:
                want1.add(x)
            if len(diff) == 2:
                for i, j in (diff, diff[::-1]):
                    mi = list(b)
                    mi[i] = 1
                    if (m[i] == 1 and b[j] == 1 and m[j] == 2 and
                            allms[O.index_of(mi)] == INF):
                        want2.add(x)
        got1 = [p["index"] for p in probes if p["kind"] == 1]
        got2 = [p["index"] for p in probes if p["kind"] == 2]
        assert sorted(got1) == sorted(want1) and len(got1) == 2 * n
        assert sorted(set(got2)) == sorted(want2) and len(got2) == len(want2)
        for p in probes:
            assert p["makespan_us"] == allms[p["index"]]
        # order: tool ascending, modes ascending, swaps right after their move
        keys = [(p["tool"], p["mode"], p["kind"], p["swap_tool"]) for p in probes[1:]]
        assert keys == sorted(keys)


@pytest.mark.parametrize("name", ["S2", "S4", "S5"])
def test_paper_binary_space_reproduces_table3(oracle_mod, name):
    """S1-S10 decide GPU or CPU per tool (Section 4.1): 2^4 = 16 mappings.
    With every tool restricted to cpu or gpu_now, the oracle picks the
    mapping of Table 3 for S2, S4 and S5."""
    O = oracle_mod
    d = load_paper()
    s = d["scenarios"][name]
    P = paper_problem(O, d, s)
    sp = O.Space([3, 3, 3, 3])
    assert sp.size() == 16
    x, ms = O.masked_argmin(P, sp)
    assert sp.modes(x) == s["paper_oracle"]
    assert ms == P.eval_index(O.index_of(s["paper_oracle"]))


def test_paper_binary_space_neutral_tool(oracle_mod):
    """web_search has no GPU implementation (Table 1).  Restricted to the
    CPU, S3's optimum agrees with Table 3 on every other tool; S1 stays a
    recorded divergence (sentiment, see test_paper_known_divergences)."""
    O = oracle_mod
    d = load_paper()
    s = d["scenarios"]["S3"]
    sp = O.Space([3, 3, 3, 1])
    assert sp.size() == 8
    x, _ = O.masked_argmin(paper_problem(O, d, s), sp)
    assert sp.modes(x)[:3] == s["paper_oracle"][:3] and sp.modes(x)[3] == 0
    s1 = d["scenarios"]["S1"]
    x1, _ = O.masked_argmin(paper_problem(O, d, s1), sp)
    assert sp.modes(x1) != s1["paper_oracle"]


@pytest.mark.parametrize("seed", range(8))
def test_masked_space_by_brute_force(oracle_mod, seed):
    """A restricted space against the full 3^N space: its mappings are the
    allowed ones, its index order is the colexicographic order of the
    per-tool ranks, and its optimum is the first allowed mapping of minimum
    makespan in that order."""
    O = oracle_mod
    n = 2 + seed % 5
    inst = synth.random_instance(9300 + seed, n, ["random", "fanout", "permuted", "chain"][seed % 4],
                                 tight=seed % 2 == 0)
    P = O.Problem(inst["tools"], inst["edges"], inst["contention_q16"], inst["vram_budget_mib"])
    masks = [(seed * 5 + 3 * v) % 7 + 1 for v in range(n)]
    sp = O.Space(masks)
    full = P.eval_many(range(3 ** n), threads=1)
    allowed = []
    for x in range(3 ** n):
        m = O.modes_of(x, n)
        if all((masks[v] >> m[v]) & 1 for v in range(n)):
            ranks = tuple(bin(masks[v] & ((1 << m[v]) - 1)).count("1") for v in range(n))
            allowed.append((ranks[::-1], x))
    allowed.sort()
    assert len(allowed) == sp.size()
    for k, (_, x3) in enumerate(allowed):
        assert int(sp.base3([k])[0]) == x3 and O.index_of(sp.modes(k)) == x3
        assert sp.index(O.modes_of(x3, n)) == k
    ms = [full[x3] for _, x3 in allowed]
    best = min(ms)
    want = (ms.index(best), best) if best != INF else (O.NO_INDEX, INF)
    assert O.masked_argmin(P, sp, chunk=7) == want
    # every mode allowed: the base-3 space itself
    every = O.Space([7] * n)
    assert O.masked_argmin(P, every) == P.argmin(threads=1)


def test_monitor_running_averages_by_hand(oracle_mod):
    """Sliding windows worked out by hand (window 3)."""
    O = oracle_mod
    M = O.Monitor(3, 3)
    rounds = [([1, 0, 2], [10, 1, 1000]),
              ([1, 0, 2], [20, 2, 1400]),
              ([1, 2, 2], [31, 500, -1]),   # tool 2 not observed
              ([1, 0, 0], [40, -1, 77])]
    for modes, lat in rounds:
        M.observe(modes, lat)
    assert M.mean(0, 1) == 30        # last three of 10, 20, 31, 40: 91/3 = 30.33
    assert M.mean(1, 0) == 2         # (1 + 2) / 2 = 1.5, half up
    assert M.mean(1, 2) == 500
    assert M.mean(2, 2) == 1200      # (1000 + 1400) / 2
    assert M.mean(2, 0) == 77
    assert M.mean(0, 0) is None and M.mean(2, 1) is None
    profile = [[300, 900, 50, 7, 1], [100, 9, 40, 3, 1], [250, 60, 30, 5, 1]]
    assert M.latencies(profile) == [
        [30, 900, 50, 7],            # gpu_now average; cpu and load unobserved
        [100, 2, 400, 3],            # load = gpu_queue 500 - gpu 100
        [250, 77, 950, 5],           # load = 1200 - 250 (gpu from the profile)
    ]
    M2 = O.Monitor(1, 2)
    M2.observe([2], [10])
    assert M2.latencies([[300, 9, 50, 0, 1]]) == [[300, 9, 0, 0]]  # queue faster than gpu: 0


# ---------------------------------------------------------------------------
# Closed forms and exact alternative computations.


def chain_closed_form(tools, modes, table):
    """Serial chain: one task at a time, so k = 1 and VRAM never binds."""
    total = 0
    for v, (g, c, l, x, m) in enumerate(tools):
        a = modes[v]
        b = c if a == 0 else (g if a == 1 else g + l)
        total += b if a == 0 else q16(b, table[0])
        if v > 0 and (modes[v - 1] == 0) != (a == 0):
            total += x
    return total


@pytest.mark.parametrize("seed", range(6))
def test_chain_closed_form_all_mappings(oracle_mod, seed):
    O = oracle_mod
    n = 2 + seed % 4
    inst = synth.random_instance(seed, n, "chain")
    inst["vram_budget_mib"] = max(t[4] for t in inst["tools"])
    P = O.Problem.from_instance(inst)
    got = P.eval_many(range(3 ** n), threads=1)
    for x in range(3 ** n):
        want = chain_closed_form(inst["tools"], O.modes_of(x, n), inst["contention_q16"])
        assert got[x] == want, (seed, x)


def viterbi_chain_optimum(tools, table):
    """Min over mappings of a chain: DP over 3 states per position."""
    def cost(v, a):
        g, c, l, x, m = tools[v]
        return c if a == 0 else q16(g if a == 1 else g + l, table[0])
    best = [cost(0, a) for a in range(3)]
    for v in range(1, len(tools)):
        x = tools[v][3]
        best = [min(best[p] + ((x if (p == 0) != (a == 0) else 0)) for p in range(3)) + cost(v, a)
                for a in range(3)]
    return min(best)


def test_config0_chain_optimum_matches_dp(oracle_mod):
    O = oracle_mod
    inst = synth.load(0)
    P = O.Problem.from_instance(inst)
    bi, bm = P.argmin()
    assert bm == viterbi_chain_optimum(inst["tools"], inst["contention_q16"])
    # and the index is the lowest one reaching it
    allv = P.eval_many(range(3 ** 8))
    assert bi == int(next(i for i in range(3 ** 8) if allv[i] == bm))


def longest_path(n, edges, w):
    preds = [[] for _ in range(n)]
    for u, v in edges:
        preds[v].append(u)
    memo = {}

    def fin(v):
        if v not in memo:
            memo[v] = w[v] + max([fin(u) for u in preds[v]] + [0])
        return memo[v]
    return max(fin(v) for v in range(n))


@pytest.mark.parametrize("c", [1, 2, 3])
def test_all_cpu_is_longest_path(oracle_mod, c):
    O = oracle_mod
    inst = synth.load(c)
    P = O.Problem.from_instance(inst)
    n = inst["n_tools"]
    assert P.eval_index(0) == longest_path(n, inst["edges"], [t[1] for t in inst["tools"]])


def test_all_gpu_now_fanout_closed_form(oracle_mod):
    O = oracle_mod
    for seed in range(4):
        inst = synth.random_instance(100 + seed, 5, "fanout", levels=3)
        inst["vram_budget_mib"] = sum(t[4] for t in inst["tools"])
        P = O.Problem.from_instance(inst)
        f = inst["contention_q16"][min(5, 3) - 1]
        want = max(q16(t[0], f) for t in inst["tools"])
        assert P.eval_index(O.index_of([1] * 5)) == want


@pytest.mark.parametrize("seed", range(4))
def test_critical_path_lower_bound_and_all_cpu_upper_bound(oracle_mod, seed):
    O = oracle_mod
    inst = synth.random_instance(200 + seed, 6, "random", tight=(seed % 2 == 1))
    P = O.Problem.from_instance(inst)
    n = 6
    lb = longest_path(n, inst["edges"], [min(t[0], t[1]) for t in inst["tools"]])
    allv = P.eval_many(range(3 ** n), threads=1)
    feas = [v for v in allv if v != INF]
    assert min(feas) >= lb
    assert P.argmin()[1] <= allv[0]


def test_zero_budget_only_all_cpu(oracle_mod):
    O = oracle_mod
    inst = synth.load(1)
    inst = dict(inst, vram_budget_mib=0)
    P = O.Problem.from_instance(inst)
    assert P.argmin() == (0, P.eval_index(0))
    sample = P.eval_many(range(1, 3 ** 7), threads=4)
    assert (sample == INF).all()


def test_range_split_merges(oracle_mod):
    O = oracle_mod
    P = O.Problem.from_instance(synth.load(1))
    total = P.num_mappings()
    full = P.argmin()
    for h in [1, 12345, total // 2, full[0], full[0] + 1, total - 1]:
        a = P.argmin(0, h)
        b = P.argmin(h, total)
        merged = min([a, b], key=lambda r: (r[1], r[0]))
        assert merged == full


def test_empty_range_has_no_result(oracle_mod):
    O = oracle_mod
    P = O.Problem.from_instance(synth.load(0))
    assert P.argmin(5, 5) == ((1 << 64) - 1, INF)


# ---------------------------------------------------------------------------
# Tick-by-tick simulation: time advances by 1 us; at every tick the rules of
# the schedule model are applied in order.  No event list at all.


def tick_simulate(tools, edges, table, budget, modes, horizon=20000):
    n = len(tools)
    preds = [[] for _ in range(n)]
    for u, v in edges:
        if u not in preds[v]:
            preds[v].append(u)
    state = ["wait"] * n
    fin = [0] * n
    on_gpu = [m != 0 for m in modes]
    for t in range(horizon):
        for v in range(n):
            if state[v] == "run" and fin[v] <= t:
                state[v] = "done"
        ready = {}
        for v in range(n):
            if state[v] == "wait" and all(state[u] == "done" for u in preds[v]):
                ready[v] = max([fin[u] + (tools[v][3] if on_gpu[u] != on_gpu[v] else 0)
                                for u in preds[v]] + [0])
        used = sum(tools[v][4] for v in range(n) if state[v] == "run" and on_gpu[v])
        starters = [v for v in sorted(ready) if modes[v] != 2 and ready[v] <= t]
        used += sum(tools[v][4] for v in starters if modes[v] == 1)
        if used > budget:
            return INF
        if not any(state[v] == "run" and modes[v] == 2 for v in range(n)):
            queued = sorted((ready[v], v) for v in ready if modes[v] == 2 and ready[v] <= t)
            if queued and tools[queued[0][1]][4] <= budget - used:
                starters.append(queued[0][1])
        k = sum(1 for v in range(n) if on_gpu[v] and (state[v] == "run" or v in starters))
        f = table[min(k, len(table)) - 1]
        for v in starters:
            g, c, l, x, m = tools[v]
            b = c if modes[v] == 0 else (g if modes[v] == 1 else g + l)
            fin[v] = t + (b if modes[v] == 0 else q16(b, f))
            state[v] = "run"
        if all(s != "wait" for s in state):
            return max(fin)
    return INF


@pytest.mark.parametrize("seed,shape,tight", [
    (0, "random", False), (1, "random", True), (2, "fanout", True),
    (3, "chain", False), (4, "random", True), (5, "fanout", False),
    (6, "random", True), (7, "random", False)])
def test_event_simulation_matches_tick_simulation(oracle_mod, seed, shape, tight):
    O = oracle_mod
    n = 4
    inst = synth.random_instance(300 + seed, n, shape, levels=3, tight=tight,
                                 small_values=True)
    P = O.Problem.from_instance(inst)
    got = P.eval_many(range(3 ** n), threads=1)
    for x in range(3 ** n):
        want = tick_simulate(inst["tools"], inst["edges"], inst["contention_q16"],
                             inst["vram_budget_mib"], O.modes_of(x, n))
        assert got[x] == want, (seed, x)


# Processor sharing (the other reading of Factor A).


def ps_rate(f):
    return ((1 << 33) + f) // (2 * f)  # round(2^32 / f), halves up


def ps_tick_simulate(tools, edges, table, budget, modes, horizon=20000):
    """Processor sharing advanced one microsecond at a time: each tick every
    running GPU task completes ps_rate(F[k]) units of its b * 2^16 units of
    work, and finishes at the first tick where none is left."""
    n = len(tools)
    preds = [[] for _ in range(n)]
    for u, v in edges:
        if u not in preds[v]:
            preds[v].append(u)
    state = ["wait"] * n
    fin = [0] * n
    rem = [0] * n
    on_gpu = [m != 0 for m in modes]
    for t in range(horizon):
        for v in range(n):
            if state[v] == "run" and (rem[v] <= 0 if on_gpu[v] else fin[v] <= t):
                state[v] = "done"
                fin[v] = t
        if all(s == "done" for s in state):
            return max(fin)
        ready = {}
        for v in range(n):
            if state[v] == "wait" and all(state[u] == "done" for u in preds[v]):
                ready[v] = max([fin[u] + (tools[v][3] if on_gpu[u] != on_gpu[v] else 0)
                                for u in preds[v]] + [0])
        used = sum(tools[v][4] for v in range(n) if state[v] == "run" and on_gpu[v])
        starters = [v for v in sorted(ready) if modes[v] != 2 and ready[v] <= t]
        used += sum(tools[v][4] for v in starters if modes[v] == 1)
        if used > budget:
            return INF
        if not any(state[v] == "run" and modes[v] == 2 for v in range(n)):
            queued = sorted((ready[v], v) for v in ready if modes[v] == 2 and ready[v] <= t)
            if queued and tools[queued[0][1]][4] <= budget - used:
                starters.append(queued[0][1])
        for v in starters:
            g, c, l, x, m = tools[v]
            state[v] = "run"
            if modes[v] == 0:
                fin[v] = t + c
            else:
                rem[v] = (g if modes[v] == 1 else g + l) << 16
        k = sum(1 for v in range(n) if on_gpu[v] and state[v] == "run")
        if k:
            w = ps_rate(table[min(k, len(table)) - 1])
            for v in range(n):
                if on_gpu[v] and state[v] == "run":
                    rem[v] -= w
    return INF


def test_ps_hand_cases(oracle_mod):
    O = oracle_mod
    # V4 under processor sharing: t1 ends at 150 (100 at 1.5x) having let t0
    # do 100 of its 400; t0 runs alone for the other 300.
    P = mk(O, [[400, 5000, 50, 0, 1], [100, 5000, 50, 0, 1]], [], 16)
    Ps = O.Problem([[400, 5000, 50, 0, 1], [100, 5000, 50, 0, 1]], [], F2, 16, sharing=True)
    assert P.eval_index(4) == 600 and Ps.eval_index(4) == 450
    # one GPU task at 1.0x: exactly its latency; a lone queued task pays load
    one = O.Problem([[123, 9000, 45, 0, 1]], [], F2, 16, sharing=True)
    assert [one.eval_index(x) for x in range(3)] == [9000, 123, 168]
    assert ps_rate(65536) == 65536 and ps_rate(98304) == 43691


@pytest.mark.parametrize("seed,shape,tight", [
    (0, "random", False), (1, "random", True), (2, "fanout", True),
    (3, "chain", False), (4, "random", True), (5, "fanout", False)])
def test_ps_event_simulation_matches_tick_simulation(oracle_mod, seed, shape, tight):
    O = oracle_mod
    n = 4
    inst = synth.random_instance(700 + seed, n, shape, levels=3, tight=tight,
                                 small_values=True)
    P = O.Problem.from_instance(inst, sharing=True)
    got = P.eval_many(range(3 ** n), threads=1)
    for x in range(3 ** n):
        want = ps_tick_simulate(inst["tools"], inst["edges"], inst["contention_q16"],
                                inst["vram_budget_mib"], O.modes_of(x, n))
        assert got[x] == want, (seed, x)


@pytest.mark.parametrize("seed", range(6))
def test_ps_fanout_against_exact_sharing(oracle_mod, seed):
    """All-gpu_now fan-outs against processor sharing in exact rationals:
    tasks finish in order of work; while k run each advances at 1 / F[k].
    The integer reading stays within one microsecond per event plus the
    rounding of the rates."""
    from fractions import Fraction
    O = oracle_mod
    n = 3 + seed % 4
    inst = synth.random_instance(800 + seed, n, "fanout", levels=4)
    F = inst["contention_q16"]
    P = O.Problem(inst["tools"], [], F, sum(t[4] for t in inst["tools"]), sharing=True)
    work = sorted(t[0] for t in inst["tools"])
    t, done = Fraction(0), 0
    for i, wv in enumerate(work):
        k = n - i
        t += (wv - done) * Fraction(F[min(k, len(F)) - 1], 1 << 16)
        done = wv
    got = P.eval_index(O.index_of([1] * n))
    rel = max(Fraction(1, 2 * ps_rate(f)) for f in F)
    assert abs(got - t) <= n + 1 + t * rel * 2


def test_paper_ps_readings(oracle_mod):
    """Processor sharing picks Table 3's mapping for S1, which the
    fixed-at-start reading misses, but makes all-GPU win S5 (613.8 ms, worked
    out by hand in the exact reading) where the paper offloads C."""
    O = oracle_mod
    d = load_paper()
    sp = O.Space([3, 3, 3, 3])
    s1 = d["scenarios"]["S1"]
    P1 = O.Problem(s1["tools"], d["diamond_edges"], d["contention_q16"], s1["budget"],
                   sharing=True)
    assert sp.modes(O.masked_argmin(P1, sp)[0]) == s1["paper_oracle"]
    s5 = d["scenarios"]["S5"]
    P5 = O.Problem(s5["tools"], [], d["contention_q16"], s5["budget"], sharing=True)
    x, ms = O.masked_argmin(P5, sp)
    assert sp.modes(x) == [1, 1, 1, 1] != s5["paper_oracle"]
    # B ends at 136 * 2.4 = 326.4 ms, D 9 ms of work later at 1.8x (342.6),
    # C 132 ms of work later at 1.35x (520.8), A its last 93 ms alone.
    assert abs(ms - 613800) <= 4


# ---------------------------------------------------------------------------
# Invariants of returned schedules.


def check_schedule(inst, modes, ms, start, fin):
    tools = inst["tools"]
    n = len(tools)
    table = inst["contention_q16"]
    M = inst["vram_budget_mib"]
    gpu = [m != 0 for m in modes]
    preds = [[] for _ in range(n)]
    for u, v in inst["edges"]:
        preds[v].append(u)
    ready = [max([fin[u] + (tools[v][3] if gpu[u] != gpu[v] else 0) for u in preds[v]] + [0])
             for v in range(n)]
    assert ms == max(fin)
    sinks = [v for v in range(n) if not any(u == v for u, _ in inst["edges"])]
    assert ms == max(fin[v] for v in sinks)
    for v in range(n):
        # cpu and gpu_now never wait; queued tools never start early
        if modes[v] != 2:
            assert start[v] == ready[v]
        else:
            assert start[v] >= ready[v]
        running = [u for u in range(n) if gpu[u] and start[u] <= start[v] < fin[u]]
        used = sum(tools[u][4] for u in running)
        assert used <= M
        g, c, l, x, m = tools[v]
        if modes[v] == 0:
            assert fin[v] - start[v] == c
        else:
            k = len(running)
            b = g if modes[v] == 1 else g + l
            assert fin[v] - start[v] == q16(b, table[min(k, len(table)) - 1])
    q = sorted([v for v in range(n) if modes[v] == 2], key=lambda v: start[v])
    for a, b in zip(q, q[1:]):
        assert fin[a] <= start[b]                      # serialized
        assert (ready[a], a) < (ready[b], b)           # FIFO on (r, v)
    for v in q:
        # a queued tool starts when it becomes ready or when something ends
        assert start[v] == ready[v] or any(fin[u] == start[v] for u in range(n))


@pytest.mark.parametrize("seed", range(6))
def test_returned_schedules_are_valid(oracle_mod, seed):
    O = oracle_mod
    n = 5
    inst = synth.random_instance(400 + seed, n, "random", tight=True)
    P = O.Problem.from_instance(inst)
    n_feasible = 0
    for modes in itertools.product(range(3), repeat=n):
        ms, s, c = P.schedule(list(modes))
        if ms == INF:
            continue
        n_feasible += 1
        check_schedule(inst, list(modes), ms, s, c)
    assert n_feasible > 0


def test_relabelling_tools_preserves_makespans_without_queue(oracle_mod):
    O = oracle_mod
    n = 5
    inst = synth.random_instance(500, n, "random", tight=True)
    perm = [3, 0, 4, 1, 2]  # new label of old tool v is perm[v]
    tools2 = [None] * n
    for v in range(n):
        tools2[perm[v]] = inst["tools"][v]
    edges2 = [[perm[u], perm[v]] for u, v in inst["edges"]]
    P1 = O.Problem.from_instance(inst)
    P2 = O.Problem(tools2, edges2, inst["contention_q16"], inst["vram_budget_mib"])
    for modes in itertools.product(range(2), repeat=n):
        m2 = [0] * n
        for v in range(n):
            m2[perm[v]] = modes[v]
        assert P1.schedule(list(modes))[0] == P2.schedule(m2)[0]


def test_step_counts_of_the_work_model(oracle_mod):
    """The oracle's step counts behind the per-mapping work figure
    (tests/golden/count_ops.py): a chain where every mapping is feasible
    reads every edge and starts every tool; an out-of-memory start ends the
    count there.  Hand-built: A and B sources, C after A; footprints 10, 95,
    10 against a budget of 100; B runs long on the GPU."""
    O = oracle_mod
    inst = synth.load(0)
    Q = O.Problem.from_instance(inst)
    e, s, f = Q.count_steps(range(3 ** 8))
    assert (e, s, f) == (7 * 3 ** 8, 8 * 3 ** 8, 3 ** 8)
    tools = [[10, 20, 0, 5, 10], [1000, 2000, 0, 0, 95], [10, 20, 0, 3, 10]]
    P = mk(O, tools, [[0, 2]], 100)
    idx = lambda a, b, c: a + 3 * b + 9 * c  # noqa: E731
    # A and B on gpu_now together: 105 > 100 at t = 0, nothing starts
    assert P.count_steps([idx(1, 1, 0)]) == (0, 0, 0)
    # A on the CPU, B on gpu_now: both start at 0; C becomes ready at
    # 20 + 3 and runs out of VRAM beside B (95 + 10): one edge read, two starts
    assert P.eval_index(idx(0, 1, 1)) == O.INFEASIBLE
    assert P.count_steps([idx(0, 1, 1)]) == (1, 2, 0)
    # the same with C on the CPU: feasible, everything counted
    assert P.count_steps([idx(0, 1, 0)]) == (1, 3, 1)
