"""Property tests of the configuration space against the oracle on randomly
drawn spaces (§3.3 Eq.1–4, §4.1 Eq.5–9): extents with odd cofactors, one to
four levels per dimension, both dtypes, with and without the MFMA
coordinate, both neighbour relations. For every drawn space the library and
the oracle agree on |ξ|, and at drawn ranks on unrank, rank, legitimacy and
the neighbour list; a space one side rejects the other rejects too. On
drawn spaces, starts, budgets, seeds and settings, G-BFS (Alg.1), the random
search and N-A2C (Alg.2) time the oracle's sequence of configurations."""
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

ODD = [1, 3, 5, 7, 43]


@st.composite
def extents(draw):
    q = draw(st.sampled_from(ODD))
    e = draw(st.integers(0, 12))
    return q << e


@st.composite
def spaces(draw):
    M, N, K = draw(extents()), draw(extents()), draw(extents())
    d = tuple(draw(st.integers(1, 4)) for _ in range(3))
    dt = draw(st.sampled_from(["f32", "bf16"]))
    mc = draw(st.booleans())
    mode = draw(st.integers(0, 1))
    fracs = draw(st.lists(st.floats(0.0, 1.0, exclude_max=True), min_size=6, max_size=6))
    return (M, N, K, d, dt, mc), mode, fracs


@pytest.fixture(scope="module")
def sides():
    from paper_1909_10616_amd import gemmtune
    import oracle
    gemmtune.lib()
    return gemmtune, oracle


@settings(max_examples=500, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(spaces())
def test_random_spaces_match_oracle(sides, case):
    gt, orc = sides
    args, mode, fracs = case
    try:
        ls = gt.Space(*args, mode=mode)
        lsize = ls.size()
    except Exception:
        ls = None
    try:
        os_ = orc.Space(*args, mode=mode)
        osize = os_.size()
    except Exception:
        os_ = None
    assert (ls is None) == (os_ is None), args
    if ls is None:
        return
    assert lsize == osize
    ranks = {0, lsize - 1} | {int(f * lsize) for f in fracs}
    for r in sorted(ranks):
        c = ls.unrank(r)
        assert c == os_.unrank(r), (args, r)
        assert ls.rank(c) == r == os_.rank(c)
        assert ls.legit(c) == os_.legit(c), (args, c)
        assert ls.neighbours(c) == os_.neighbours(c), (args, mode, c)


def _splitmix_cost(seed, inf_mod):
    """A synthetic cost keyed by rank (after the paper's random-reward
    experiment): 1 + SplitMix64(rank ⊕ seed) / 2^64, and when inf_mod > 0
    +∞ for every rank ≡ 5 and NaN for every rank ≡ 3 (mod inf_mod): two
    ways a candidate fails."""
    M64 = (1 << 64) - 1

    def f(cfg, rank):
        if inf_mod and rank % inf_mod == 5:
            return float("inf")
        if inf_mod and rank % inf_mod == 3:
            return float("nan")
        z = ((rank ^ seed) + 0x9E3779B97F4A7C15) & M64
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
        return 1.0 + (z ^ (z >> 31)) / 2.0 ** 64
    return f


@st.composite
def searches(draw):
    args, mode, fracs = draw(spaces())
    rho = draw(st.integers(1, 8))
    budget = draw(st.integers(1, 300))
    seed = draw(st.integers(0, (1 << 32) - 1))
    inf_mod = draw(st.sampled_from([0, 7, 11]))
    return args, mode, fracs, rho, budget, seed, inf_mod


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(searches())
def test_random_searches_match_oracle(sides, case):
    """G-BFS (Alg.1) from a drawn legitimate start, and the equal-budget
    random search, under synthetic costs with failures: the same ordered
    list of timed ranks, the same s*, cost, count timed and pops."""
    gt, orc = sides
    args, mode, fracs, rho, budget, seed, inf_mod = case
    ls, os_ = gt.Space(*args, mode=mode), orc.Space(*args, mode=mode)
    size = ls.size()
    starts = [ls.unrank(int(f * size)) for f in fracs] + [ls.paper_s0()]
    s0 = next((c for c in starts if ls.legit(c)), None)
    cost = _splitmix_cost(seed, inf_mod)
    if s0 is not None:
        got = gt.tune_gbfs(ls, budget=budget, s0=s0, rho=rho, seed=seed, cost_fn=cost)
        exp = orc.gbfs(os_, s0, rho, budget, seed, cost)
        assert [e["rank"] for e in got["log"]] == exp["log_ranks"], (args, mode, s0, rho, seed)
        assert got["best"] == exp["best"] and got["best_cost"] == exp["best_cost"]
        assert got["timed"] == exp["timed"] and got["popped"] == exp["popped"]
    got = gt.tune_random(ls, budget=budget, seed=seed, cost_fn=cost)
    exp = orc.random_search(os_, budget, seed, cost)
    assert [e["rank"] for e in got["log"]] == exp["log_ranks"], (args, seed)
    assert got["best"] == exp["best"] and got["best_cost"] == exp["best_cost"]
    assert got["timed"] == exp["timed"] and got["popped"] == exp["popped"]


@st.composite
def na2c_runs(draw):
    args, mode, fracs = draw(spaces())
    params = {
        "T": draw(st.integers(1, 5)), "B": draw(st.integers(1, 16)), "H": draw(st.integers(1, 64)),
        "mem": draw(st.integers(1, 512)), "max_walks": draw(st.integers(1, 96)),
        "reward": draw(st.integers(0, 1)), "eps_halving": draw(st.integers(0, 1)),
        "eps": draw(st.floats(0.0, 1.0)), "gamma": draw(st.floats(0.0, 1.0)),
        "lr": draw(st.floats(1e-4, 0.2)), "r_clip": draw(st.floats(0.25, 10.0)),
    }
    budget = draw(st.integers(1, 150))
    seed = draw(st.integers(0, (1 << 32) - 1))
    inf_mod = draw(st.sampled_from([0, 7, 11]))
    return args, mode, fracs, params, budget, seed, inf_mod


@settings(max_examples=80, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(na2c_runs())
def test_random_na2c_runs_match_oracle(sides, case):
    """N-A2C (§4.3, Alg.2) from a drawn legitimate start with drawn settings
    (walk length, batch, hidden width, memory, ε, γ, learning rate, both
    rewards, ε halving) under synthetic costs with failures: the same timed
    ranks and costs, s*, count timed and episodes, bit for bit."""
    gt, orc = sides
    args, mode, fracs, params, budget, seed, inf_mod = case
    ls, os_ = gt.Space(*args, mode=mode), orc.Space(*args, mode=mode)
    size = ls.size()
    starts = [ls.unrank(int(f * size)) for f in fracs] + [ls.paper_s0()]
    s0 = next((c for c in starts if ls.legit(c)), None)
    if s0 is None:
        return
    cost = _splitmix_cost(seed, inf_mod)
    got = gt.tune_na2c(ls, budget, s0=s0, seed=seed, cost_fn=cost, params=params)
    exp = orc.na2c(os_, s0, budget, seed, cost, params)
    assert [e["rank"] for e in got["log"]] == exp["log_ranks"], (args, mode, s0, params, seed)
    assert [e["cost_ms"] for e in got["log"]] == exp["log_costs"]
    assert got["best"] == exp["best"] and got["best_cost"] == exp["best_cost"]
    assert got["timed"] == exp["timed"] and got["popped"] == exp["popped"]
