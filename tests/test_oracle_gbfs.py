"""Pins for the oracle G-BFS (§4.2, Alg.1) — CPU only, synthetic costs.

The paper exercises G-BFS on a 2-D space with a randomly generated reward
(§4.2, Fig.5c) and states that with ρ = len(g(s)) and unlimited time every
state is visited. The pins below are that invariant, a hand-traced tiny
search, greedy convergence on a unimodal cost, and budget accounting.
"""
import json
import math
import os

import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def test_splitmix64_reference_outputs(orc):
    g = json.load(open(GOLD))["splitmix64_seed0"]
    assert [f"{v:016x}" for v in orc.splitmix64_stream(0, 3)] == g["outputs_hex"]


def test_hand_traced_three_state_search(orc):
    # ξ_m = [(1,4), (2,2), (4,1)] (ranks 0,1,2); N = K = 1. Costs 1, 2, 3.
    # s0 = (4,1) is timed (log [2]); pop it: g = [(2,2)], one pick (2,2) -> timed.
    # pop (2,2): g = [(1,4), (4,1)]; rho = 1; j = 0 + r2 mod 2 with the second
    # SplitMix64 output of seed 0 (…65f4, even) -> pick (1,4) -> timed.
    # pop (1,4): its only neighbour is visited; queue empty -> stop.
    sp = orc.Space(4, 1, 1, (2, 1, 1), "f32", False)
    cost = {0: 1.0, 1: 2.0, 2: 3.0}
    s0 = ((4, 1), (1,), (1,), 0)
    r = orc.gbfs(sp, s0, rho=1, budget=100, seed=0, cost_fn=lambda c, rk: cost[rk])
    assert r["log_ranks"] == [2, 1, 0]
    assert r["best"] == ((1, 4), (1,), (1,), 0) and r["best_cost"] == 1.0
    assert r["timed"] == 3 and r["popped"] == 3
    # a budget of 2 stops right after the second timing
    r = orc.gbfs(sp, s0, rho=1, budget=2, seed=0, cost_fn=lambda c, rk: cost[rk])
    assert r["log_ranks"] == [2, 1] and r["best"] == ((2, 2), (1,), (1,), 0)


def orc_mix(x):
    # one SplitMix64 output with state x: a counter-based random reward
    M = (1 << 64) - 1
    z = (x + 0x9E3779B97F4A7C15) & M
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
    return z ^ (z >> 31)


@pytest.mark.parametrize("mode", [0, 1])
def test_exhaustive_when_rho_is_full_degree(orc, mode):
    # every state of this small space is legitimate, so with rho >= max degree and
    # an unlimited budget Alg.1 visits the whole space (§4.2)
    sp = orc.Space(16, 8, 8, (3, 2, 2), "f32", False, mode=mode)
    allc = sp.enumerate()
    assert all(j for _, j in allc)
    r = orc.gbfs(sp, sp.paper_s0(), rho=64, budget=10 ** 6, seed=7,
                 cost_fn=lambda c, rk: 1.0 + orc_mix(rk ^ 7) / 2.0 ** 64)
    assert r["timed"] == sp.size()
    assert sorted(r["log_ranks"]) == list(range(sp.size()))
    best_rank = min(range(sp.size()), key=lambda rk: 1.0 + orc_mix(rk ^ 7) / 2.0 ** 64)
    assert sp.rank(r["best"]) == best_rank


def test_unimodal_cost_reaches_target(orc):
    sp = orc.Space(32, 16, 16, (4, 3, 3), "bf16", True)
    target = ((2, 2, 2, 4), (2, 2, 4), (2, 2, 4), 32)

    def expo(c):
        return [int(math.log2(v)) for lv in c[:3] for v in lv] + [c[3] // 32]

    te = expo(target)

    def cost(c, rk):
        return 1.0 + sum(abs(a - b) for a, b in zip(expo(c), te))

    assert sp.legit(target)
    r = orc.gbfs(sp, sp.paper_s0(), rho=64, budget=10 ** 6, seed=1, cost_fn=cost)
    assert r["best"] == target and r["best_cost"] == 1.0


def test_budget_is_exact_and_best_is_argmin_of_log(orc):
    sp = orc.Space(1024, 1024, 1024, (4, 4, 4), "f32", False)
    r = orc.gbfs(sp, sp.paper_s0(), rho=5, budget=200, seed=3,
                 cost_fn=lambda c, rk: 1.0 + orc_mix(rk ^ 3) / 2.0 ** 64)
    assert r["timed"] == 200 == len(r["log_ranks"])
    assert len(set(r["log_ranks"])) == 200            # never times a state twice
    i = min(range(200), key=lambda t: (r["log_costs"][t], t))
    assert sp.rank(r["best"]) == r["log_ranks"][i]
    for rk in r["log_ranks"]:
        assert sp.legit(sp.unrank(rk))


def test_infinite_cost_is_counted_not_expanded(orc):
    sp = orc.Space(4, 1, 1, (2, 1, 1), "f32", False)
    cost = {0: 1.0, 1: math.inf, 2: 3.0}
    r = orc.gbfs(sp, ((4, 1), (1,), (1,), 0), rho=5, budget=100, seed=0,
                 cost_fn=lambda c, rk: cost[rk])
    # (2,2) fails: counted and visited but never pushed, so (1,4) is never reached
    assert r["log_ranks"] == [2, 1] and r["best_cost"] == 3.0 and r["popped"] == 1


def test_rejects_illegitimate_start(orc):
    sp = orc.Space(4096, 4096, 4096, (4, 4, 4), "bf16", True)
    with pytest.raises(ValueError):
        orc.gbfs(sp, ((16, 8, 1, 32), (64, 1, 4, 16), (32, 4, 1, 32), 32), 5, 10, 0,
                 lambda c, rk: 1.0)


@pytest.mark.parametrize("search", ["gbfs", "random", "na2c"])
def test_nan_cost_reads_as_a_failed_candidate(orc, search):
    """A cost that is not a number is no measurement: each search follows
    exactly the trajectory it follows when those candidates cost +∞, and
    logs them as +∞."""
    sp = orc.Space(128, 64, 256, (3, 2, 3), "f32", False)
    s0 = sp.paper_s0()

    def cost_with(fail):
        def f(c, r):
            h = (r * 2654435761) % 997
            return fail if h % 4 == 0 else 1.0 + h / 997
        return f

    def run(fail):
        if search == "gbfs":
            return orc.gbfs(sp, s0, 3, 120, 7, cost_with(fail))
        if search == "random":
            return orc.random_search(sp, 120, 7, cost_with(fail))
        return orc.na2c(sp, s0, 120, 7, cost_with(fail))

    a, b = run(float("nan")), run(math.inf)
    assert a["log_ranks"] == b["log_ranks"] and a["log_costs"] == b["log_costs"]
    assert a["best"] == b["best"] and a["best_cost"] == b["best_cost"]
    assert math.inf in a["log_costs"] and not any(math.isnan(v) for v in a["log_costs"])
