"""Property tests of the configuration space against the oracle on randomly
drawn spaces (§3.3 Eq.1–4, §4.1 Eq.5–9): extents with odd cofactors, one to
four levels per dimension, both dtypes, with and without the MFMA
coordinate, both neighbour relations. For every drawn space the library and
the oracle agree on |ξ|, and at drawn ranks on unrank, rank, legitimacy and
the neighbour list; a space one side rejects the other rejects too."""
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
