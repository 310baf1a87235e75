"""Pins for the oracle configuration space (Eq.1–4), rank order, legitimacy
(Eq.5) and neighbour relation (Eq.6, Eq.9) — CPU only."""
import itertools
import json
import math
import os

import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def _divisors(D):
    return [v for v in range(1, D + 1) if D % v == 0]


def _brute_tuples(D, d):
    """All ordered d-tuples of positive integers with product D, filtered to
    power-of-two levels with the odd cofactor of D at level 0, sorted."""
    q = D
    while q % 2 == 0:
        q //= 2
    out = []
    for t in itertools.product(_divisors(D), repeat=d):
        if math.prod(t) != D:
            continue
        if t[0] % q or (t[0] // q) & (t[0] // q - 1):
            continue
        if any(v & (v - 1) for v in t[1:]):
            continue
        out.append(t)
    return sorted(out)


@pytest.mark.parametrize("D", [1, 2, 8, 16, 48, 64, 96, 3, 40])
@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_tuples_match_brute_force(orc, D, d):
    assert orc.dim_tuples(D, d) == _brute_tuples(D, d)


@pytest.mark.parametrize("E", range(0, 13))
@pytest.mark.parametrize("d", [1, 2, 3, 4])
def test_tuple_count_closed_form(orc, E, d):
    assert len(orc.dim_tuples(2 ** E, d)) == math.comb(E + d - 1, d - 1)


def test_paper_space_sizes(orc):
    g = json.load(open(GOLD))["space_sizes_d424"]
    for D in (512, 1024, 2048):
        assert orc.Space(D, D, D, d=(4, 2, 4)).size() == g[str(D)]


def test_workload_space_sizes(orc):
    S = orc.Space
    assert S(256, 256, 256, (3, 3, 3)).size() == 91125
    assert S(1024, 1024, 1024, (4, 4, 4)).size() == 23393656
    assert S(2048, 2048, 2048, (4, 4, 4)).size() == 48228544
    assert S(4096, 4096, 4096, (4, 4, 4), "bf16", True).size() == 188392750
    assert S(4096, 11008, 4096, (4, 4, 4), "bf16", True).size() == 68318250
    assert S(64, 4096, 4096, (4, 4, 4), "bf16", True).size() == 34780200


def test_odd_extent_11008(orc):
    # 11008 = 43 * 2^8: 165 tuples with the cofactor at level 0, 660 without that rule
    assert len(orc.dim_tuples(11008, 4)) == 165
    allf = [t for t in itertools.product(_divisors(11008), repeat=4) if math.prod(t) == 11008]
    assert len(allf) == 660


def test_fig4_config_member_and_roundtrip(orc):
    g = json.load(open(GOLD))["fig4_config"]
    sp = orc.Space(g["M"], g["N"], g["K"], d=(2, 2, 2))
    cfg = (tuple(g["m"]), tuple(g["k"]), tuple(g["n"]), 0)
    assert sp.member(cfg)
    assert sp.unrank(sp.rank(cfg)) == cfg


def test_paper_s0_is_last_in_each_dimension(orc):
    sp = orc.Space(1024, 1024, 1024, d=(4, 2, 4))
    s0 = sp.paper_s0()
    assert s0 == ((1024, 1, 1, 1), (1024, 1), (1024, 1, 1, 1), 0)
    assert sp.rank(s0) == sp.size() - 1
    assert sp.unrank(0) == ((1, 1, 1, 1024), (1, 1024), (1, 1, 1, 1024), 0)


@pytest.mark.parametrize("args", [
    (8, 4, 16, (3, 2, 3), "f32", False),
    (12, 8, 4, (2, 3, 2), "bf16", True),
    (16, 16, 16, (4, 1, 2), "bf16", True),
])
def test_rank_is_a_bijection_in_enumeration_order(orc, args):
    M, N, K, d, dt, mc = args
    sp = orc.Space(M, N, K, d, dt, mc)
    allc = sp.enumerate()
    assert len(allc) == sp.size()
    # mixed-radix order: m slowest, then k, n, mfma; each dimension lexicographic
    tm, tk, tn = (orc.dim_tuples(M, d[0]), orc.dim_tuples(K, d[1]), orc.dim_tuples(N, d[2]))
    mf = [16, 32] if mc else [0]
    expect = [(a, b, c, f) for a in tm for b in tk for c in tn for f in mf]
    assert [c for c, _ in allc] == expect
    for r, (c, _) in enumerate(allc):
        assert sp.rank(c) == r
        assert sp.unrank(r) == c


def _is_neighbour_pair(s, t, d, mode, mc):
    """Direct pairwise check of Eq.6 plus the MFMA toggle."""
    diff = [x for x in range(3) if s[x] != t[x]]
    if not diff:
        return mc and s[3] != t[3]
    if len(diff) != 1 or s[3] != t[3]:
        return False
    x = diff[0]
    idx = [i for i in range(d[x]) if s[x][i] != t[x][i]]
    if len(idx) != 2:
        return False
    a, b = idx
    for i, j in ((a, b), (b, a)):
        if t[x][i] == 2 * s[x][i] and 2 * t[x][j] == s[x][j]:
            if mode == 1 or abs(i - j) == 1:
                return True
    return False


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("args", [
    (8, 16, 4, (3, 2, 3), "f32", False),
    (12, 8, 8, (4, 2, 2), "bf16", True),
])
def test_neighbours_brute_force_symmetry(orc, mode, args):
    M, N, K, d, dt, mc = args
    sp = orc.Space(M, N, K, d, dt, mc, mode=mode)
    allc = [c for c, _ in sp.enumerate()]
    nb = {c: [t for t, _ in sp.neighbours(c)] for c in allc}
    for s in allc:
        expect = [t for t in allc if _is_neighbour_pair(s, t, d, mode, mc)]
        assert nb[s] == expect          # both in ascending rank (enumeration) order
        for t in nb[s]:
            assert s in nb[t]           # symmetry


@pytest.mark.parametrize("E,d", [(8, 3), (10, 4), (6, 4), (5, 2), (3, 1)])
def test_edge_count_closed_forms(orc, E, d):
    # per-dimension directed edges: ANY_PAIR d(d-1)C(E+d-2,d-1), ADJACENT 2(d-1)C(E+d-2,d-1)
    D = 2 ** E
    for mode, per in ((1, d * (d - 1)), (0, 2 * (d - 1))):
        sp = orc.Space(D, 1, 1, (d, 1, 1), "f32", False, mode=mode)
        edges = sum(len(sp.neighbours(c)) for c, _ in sp.enumerate())
        expect = per * math.comb(E + d - 2, d - 1) if E >= 1 else 0
        assert edges == expect


def test_degree_of_s0_and_connectivity(orc):
    for mode, deg in ((1, 3), (0, 1)):
        sp = orc.Space(16, 8, 4, (4, 4, 4), "bf16", True, mode=mode)
        s0 = sp.paper_s0()
        nb = sp.neighbours(s0)
        assert len(nb) == 3 * deg + 1   # three dimensions plus the MFMA toggle
        seen, todo = {s0}, [s0]
        while todo:
            s = todo.pop()
            for t, _ in sp.neighbours(s):
                if t not in seen:
                    seen.add(t)
                    todo.append(t)
        assert len(seen) == sp.size()


# --- legitimacy: hand-worked cases of the frozen predicate --------------------

def test_legit_hand_worked(orc):
    sp = orc.Space(4096, 4096, 4096, (4, 4, 4), "bf16", True)
    # paper start state: 1 wave, I=16, TM=TN=1, acc=4, LDS 4 bytes
    assert sp.legit(sp.paper_s0())
    # 256x256x64 tiles, 2x2 waves, 4x4 blocks of 32: acc = 16*16 = 256, LDS 64 KiB
    big = ((16, 2, 4, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32)
    assert sp.legit(big)
    # same with 4x2 waves: W=8 leaves 256 registers, acc+96 = 352 -> illegitimate
    assert not sp.legit(((8, 4, 4, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32))
    # 8x4 = 32 waves -> illegitimate
    assert not sp.legit(((16, 8, 1, 32), (64, 1, 4, 16), (32, 4, 1, 32), 32))
    # LDS: BK = 1024 with 256x256 tiles -> 1 MiB per stage
    assert not sp.legit(((16, 2, 4, 32), (4, 1, 1, 1024), (16, 2, 4, 32), 32))
    # BK = 128: (256*128 + 128*256)*2 = 128 KiB <= 160 KiB
    assert sp.legit(((16, 2, 4, 32), (32, 1, 1, 128), (16, 2, 4, 32), 32))
    # BK = 256: 256 KiB -> illegitimate
    assert not sp.legit(((16, 2, 4, 32), (16, 1, 1, 256), (16, 2, 4, 32), 32))
    # 16 waves: at most 128 registers per lane -> acc <= 32
    assert sp.legit(((64, 4, 1, 16), (64, 1, 4, 16), (64, 4, 1, 16), 16))       # acc 4
    assert sp.legit(((32, 4, 2, 16), (64, 1, 4, 16), (64, 4, 1, 16), 32))       # TM=2 acc 32
    assert not sp.legit(((32, 4, 2, 16), (64, 1, 4, 16), (32, 4, 2, 16), 32))   # acc 64
    # I=16 with 8x8 blocks of 16 per wave: acc = 64*4 = 256 (legit), 16x8 blocks -> 512
    assert sp.legit(((32, 1, 8, 16), (64, 1, 4, 16), (32, 1, 8, 16), 16))
    assert not sp.legit(((16, 1, 16, 16), (64, 1, 4, 16), (32, 1, 8, 16), 16))


def test_legit_fp32_derived_mfma(orc):
    sp = orc.Space(1024, 1024, 1024, (4, 4, 4), "f32", False)
    # blkM=32, blkN=16 -> I=16: TM = 4*2 = 8, TN = 4 -> acc = 32*4 = 128
    assert sp.legit(((8, 1, 4, 32), (64, 1, 4, 4), (16, 1, 4, 16), 0))
    # blkM=blkN=32 -> I=32: TM=TN=4 -> acc=256, W=1
    assert sp.legit(((8, 1, 4, 32), (64, 1, 4, 4), (8, 1, 4, 32), 0))
    # blkM=64, blkN=32 -> I=32: TM = 4*2 = 8, TN = 4 -> acc 512 -> illegitimate
    assert not sp.legit(((4, 1, 4, 64), (64, 1, 4, 4), (8, 1, 4, 32), 0))
    # fp32 LDS: BM=BN=128, BK=128: (128*128*2)*4 = 128 KiB ok; BK=256 -> 256 KiB no
    assert sp.legit(((8, 2, 2, 32), (8, 1, 4, 32), (8, 2, 2, 32), 0))
    assert not sp.legit(((8, 2, 2, 32), (4, 1, 8, 32), (8, 2, 2, 32), 0))


def test_legit_grid_limits(orc):
    # work-items along grid.x = grid_M * grid_N * 64 * waves must stay below 2^32
    sp = orc.Space(65536, 65536, 1, (2, 1, 2), "f32", False)
    assert not sp.legit(((8192, 8), (1,), (8192, 8), 0))       # 2^26 * 64 = 2^32
    assert sp.legit(((8192, 8), (1,), (4096, 16), 0))          # 2^25 * 64 = 2^31
    s3 = orc.Space(65536, 65536, 1, (3, 1, 2), "f32", False)
    assert s3.legit(((4096, 2, 8), (1,), (4096, 16), 0))       # 2^24 * 128 = 2^31
    assert not s3.legit(((8192, 2, 4), (1,), (4096, 16), 0))   # 2^25 * 128 = 2^32
    sk = orc.Space(1, 1, 131072, (1, 4, 1), "f32", False)
    assert not sk.legit(((1,), (1, 131072, 1, 1), (1,), 0))    # kSplit 2^17 > 65535
    assert sk.legit(((1,), (4, 32768, 1, 1), (1,), 0))


def test_legit_whole_launch(orc):
    # the whole dispatch, grid_M * grid_N * kSplit * 64 * waves work-items,
    # stays below 2^32
    sp = orc.Space(4096, 4096, 4096, (4, 4, 4), "bf16", True)
    # paper start state: 2^24 one-wave workgroups = 2^30 work-items
    assert sp.legit(((4096, 1, 1, 1), (4096, 1, 1, 1), (4096, 1, 1, 1), 16))
    # the same grid split two ways along K: 2^31; four ways: 2^32
    assert sp.legit(((4096, 1, 1, 1), (2048, 2, 1, 1), (4096, 1, 1, 1), 16))
    assert not sp.legit(((4096, 1, 1, 1), (1024, 4, 1, 1), (4096, 1, 1, 1), 16))
    # every K element its own workgroup: 2^24 * 4096 * 64 = 2^42
    assert not sp.legit(((4096, 1, 1, 1), (1, 4096, 1, 1), (4096, 1, 1, 1), 16))
    # 2^19 tiles of 8 waves, split 4096 ways: 2^19 * 2^12 * 512 = 2^40
    assert not sp.legit(((512, 2, 1, 4), (1, 4096, 1, 1), (1024, 4, 1, 1), 32))
    # the same tiles without the split: 2^28 work-items
    assert sp.legit(((512, 2, 1, 4), (4096, 1, 1, 1), (1024, 4, 1, 1), 32))
    # 256 tiles of 4 waves split 64 ways: 256 * 64 * 256 = 2^22
    assert sp.legit(((16, 2, 4, 32), (1, 64, 4, 16), (16, 2, 4, 32), 32))
