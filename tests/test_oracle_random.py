"""Pins of the oracle's equal-budget random search (the §5 baseline).

The draw sequence is pinned to the published SplitMix64 reference outputs
(tests/golden/paper_values.json), the visit set to brute-force enumeration of
small spaces, and the result to the global minimum of a known cost when the
budget covers every legitimate configuration."""
import json
import math
import os

import pytest

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _all_legit_space(orc):
    # 16x16x16, two levels each: every tuple is a 1-wavefront kernel, all legitimate
    sp = orc.Space(16, 16, 16, (2, 2, 2), "f32", False)
    assert all(legit for _, legit in sp.enumerate())
    return sp


def test_first_draws_follow_published_splitmix64(orc):
    sp = _all_legit_space(orc)
    n = sp.size()
    outs = [int(h, 16) for h in GOLDEN["splitmix64_seed0"]["outputs_hex"]]
    expect = []
    for v in outs:
        r = v % n
        if r not in expect:
            expect.append(r)
    res = orc.random_search(sp, len(expect), 0, lambda c, r: 1.0)
    assert res["log_ranks"] == expect
    assert res["popped"] == len(outs) if len(expect) == len(outs) else True


def test_budget_covering_the_space_finds_the_global_minimum(orc):
    sp = _all_legit_space(orc)
    n = sp.size()
    cost = lambda c, r: float((r * 7919) % 1009) + 0.5 * (r % 3)   # noqa: E731
    res = orc.random_search(sp, n, 42, cost)
    assert sorted(res["log_ranks"]) == list(range(n))            # every configuration once
    brute = min(range(n), key=lambda r: (cost(None, r), r))
    best_cost = cost(None, brute)
    assert res["best_cost"] == best_cost
    assert sp.rank(res["best"]) in [r for r in range(n) if cost(None, r) == best_cost]
    # the first minimum in timing order is kept (strict <)
    first = next(r for r in res["log_ranks"] if cost(None, r) == best_cost)
    assert sp.rank(res["best"]) == first


def test_skips_illegitimate_draws_and_respects_the_budget(orc):
    sp = orc.Space(256, 256, 256, (3, 3, 3), "f32", False)
    legit = {sp.rank(c) for c, ok in sp.enumerate() if ok}
    assert 0 < len(legit) < sp.size()
    res = orc.random_search(sp, 40, 7, lambda c, r: 1.0 + r)
    ranks = res["log_ranks"]
    assert len(ranks) == 40 == res["timed"] and len(set(ranks)) == 40
    assert set(ranks) <= legit
    assert res["popped"] >= 40
    assert res["best_cost"] == min(1.0 + r for r in ranks)


def test_one_point_space_exhausts_its_draws(orc):
    sp = orc.Space(1, 1, 1, (4, 4, 4), "f32", False)
    res = orc.random_search(sp, 5, 0, lambda c, r: 2.0)
    assert res["timed"] == 1 and res["popped"] == 64 * 5 + 1024
    assert res["best_cost"] == 2.0


def test_infinite_costs_and_budget_one(orc):
    sp = _all_legit_space(orc)
    res = orc.random_search(sp, 1, 3, lambda c, r: math.inf)
    assert res["timed"] == 1 and math.isinf(res["best_cost"])
    assert sp.rank(res["best"]) == res["log_ranks"][0]
    with pytest.raises(ValueError):
        orc.random_search(sp, 0, 3, lambda c, r: 1.0)
