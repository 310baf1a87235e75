"""The host side of the C ABI on arbitrary argument values: every entry
point that needs no GPU (space size, enumeration, rank, unrank, legitimacy,
neighbours, lowering, the three searches with a synthetic cost) returns 0 or
an error code with a message, and never crashes, whatever the space, the
configuration, the option values or the synthetic costs (NaN, ±∞, negative,
zero). Malformed spaces are rejected by the library and the oracle alike."""
import ctypes
import random

import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

INTS = [-(1 << 62), -7, -1, 0, 1, 2, 3, 4, 5, 7, 8, 16, 31, 32, 33, 64, 96, 128, 4096, 11008,
        1 << 20, 1 << 31, 1 << 62]
COSTS = [float("nan"), float("inf"), -float("inf"), -1.0, 0.0, 5e-324, 1e300, 1.0, 2.0]


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def _rint(rng):
    return rng.choice(INTS) if rng.random() < 0.6 else rng.randint(-3, 5000)


def _garbage_space(gt, rng):
    s = gt.gt_space()
    s.M, s.N, s.K = _rint(rng), _rint(rng), _rint(rng)
    s.d_m, s.d_k, s.d_n = (rng.choice([-1, 0, 1, 2, 3, 4, 5, 100]) for _ in range(3))
    s.dtype = rng.choice([-1, 0, 1, 2, 3, 16, 17, 18, 99])
    s.mfma_coord = rng.choice([-1, 0, 1, 2])
    s.neighbour_mode = rng.choice([-1, 0, 1, 2])
    return s


def _valid_space(gt, rng, emax=12):
    s = gt.gt_space()
    s.M, s.N, s.K = (rng.choice([1, 3, 5, 7]) << rng.randint(0, emax) for _ in range(3))
    s.d_m, s.d_k, s.d_n = (rng.randint(1, 4) for _ in range(3))
    s.dtype = rng.choice([0, 1, 16, 17])
    s.mfma_coord = rng.choice([0, 1])
    s.neighbour_mode = rng.choice([0, 1])
    return s


def _size(gt, sp):
    sz = ctypes.c_uint64()
    rc = gt.lib().gt_space_size(ctypes.byref(sp), ctypes.byref(sz))
    return sz.value if rc == 0 else None


def _config(gt, rng, sp):
    c = gt.gt_config()
    size = _size(gt, sp)
    if size and rng.random() < 0.5:
        # a member, sometimes with one value or the MFMA field spoiled
        assert gt.lib().config_unrank(ctypes.byref(sp), rng.randrange(size), ctypes.byref(c)) == 0
        if rng.random() < 0.5:
            rng.choice([c.m, c.k, c.n])[rng.randrange(gt.MAXD)] = _rint(rng)
        if rng.random() < 0.2:
            c.mfma = rng.choice([-1, 0, 8, 16, 32, 64])
        return c
    c.d_m, c.d_k, c.d_n = (rng.choice([-1, 0, 1, 2, 3, 4, 5, 100]) for _ in range(3))
    for arr in (c.m, c.k, c.n):
        for i in range(gt.MAXD):
            arr[i] = _rint(rng)
    c.mfma = rng.choice([-1, 0, 8, 16, 32, 64])
    return c


def _expect(gt, rc):
    assert isinstance(rc, int)
    if rc != 0:
        assert gt.lib().gt_last_error()   # a message names what was wrong


def test_queries_never_crash_on_arbitrary_arguments(gt):
    L = gt.lib()
    rng = random.Random(1909)
    for _ in range(30000):
        sp = _garbage_space(gt, rng) if rng.random() < 0.5 else _valid_space(gt, rng)
        c = _config(gt, rng, sp)
        f = rng.randrange(7)
        if f == 0:
            rc = L.gt_space_size(ctypes.byref(sp), ctypes.byref(ctypes.c_uint64()))
        elif f == 1:
            rc = L.config_rank(ctypes.byref(sp), ctypes.byref(c), ctypes.byref(ctypes.c_uint64()))
        elif f == 2:
            r = rng.choice([0, 1, 5, (1 << 64) - 1, rng.randrange(1 << 40)])
            rc = L.config_unrank(ctypes.byref(sp), r, ctypes.byref(gt.gt_config()))
        elif f == 3:
            rc = L.config_legit(ctypes.byref(sp), ctypes.byref(c), ctypes.byref(ctypes.c_int()))
        elif f == 4:
            cap = rng.choice([0, 1, 2, 200])
            out = (gt.gt_config * max(cap, 1))()
            rc = L.neighbours(ctypes.byref(sp), ctypes.byref(c), out, cap,
                              ctypes.byref(ctypes.c_int()))
        elif f == 5:
            cnt = rng.choice([0, 1, 7, 64])
            buf = (gt.gt_config * max(cnt, 1))()
            start = rng.choice([0, 3, (1 << 64) - 1, rng.randrange(1 << 30)])
            rc = L.enumerate_configs(ctypes.byref(sp), start, buf, cnt,
                                     ctypes.byref(ctypes.c_uint64()))
        else:
            rc = L.gt_lower(ctypes.byref(c), _rint(rng), _rint(rng), _rint(rng),
                            rng.choice([-1, 0, 1, 2, 16, 17, 99]), ctypes.byref(gt.gt_kernel_info()))
        _expect(gt, rc)


def test_searches_never_crash_on_arbitrary_options_and_costs(gt):
    L = gt.lib()
    rng = random.Random(10616)
    ran = 0
    while ran < 1500:
        sp = _valid_space(gt, rng, emax=9)
        size = _size(gt, sp)
        if not size:
            continue
        ran += 1
        o = gt.gt_tune_opts()
        assert L.gt_tune_opts_init(ctypes.byref(o)) == 0
        s0 = _config(gt, rng, sp)
        if rng.random() < 0.8:
            o.s0 = ctypes.pointer(s0)
        o.rho = rng.choice([-1, 0, 1, 2, 5, 100, 1 << 30])
        o.budget = rng.choice([-1, 0, 1, 2, 17, 200])
        o.seed = rng.randrange(1 << 64)
        o.t_max_s = rng.choice([0.0, -1.0, 1e-9, 0.5, float("nan")])
        o.runs, o.warmup = rng.choice([-1, 0, 1, 10]), rng.choice([-1, 0, 1])
        cap = rng.choice([0, 1, 5, max(o.budget, 0)])
        log = (gt.gt_log_entry * max(cap, 1))()
        if rng.random() < 0.8:
            o.log, o.log_cap = ctypes.cast(log, ctypes.POINTER(gt.gt_log_entry)), cap
        else:
            o.log_cap = rng.choice([0, 5])          # no log buffer with a nonzero capacity
        kind = rng.randrange(3)

        def cost(cptr, rank, ctx, kind=kind):
            if kind == 0:
                return 1.0 + (rank * 2654435761 % 997) / 997
            return rng.choice(COSTS) if kind == 1 else float("nan")

        cb = gt.gt_cost_fn(cost)
        res = gt.gt_tune_result()
        which = rng.randrange(3)
        if which == 0:
            rc = L.tune_gbfs(ctypes.byref(sp), ctypes.byref(o), cb, None, ctypes.byref(res))
        elif which == 1:
            rc = L.tune_random(ctypes.byref(sp), ctypes.byref(o), cb, None, ctypes.byref(res))
        else:
            prm = gt.gt_na2c_params()
            assert L.gt_na2c_params_init(ctypes.byref(prm)) == 0
            if rng.random() < 0.7:
                prm.T = rng.choice([-1, 0, 1, 3, 64, 65])
                prm.B = rng.choice([-1, 0, 1, 8, 70000])
                prm.H = rng.choice([-1, 0, 1, 32, 64, 65])
                prm.mem = rng.choice([-1, 0, 1, 256, 70000])
                prm.max_walks = rng.choice([-1, 0, 1, 64])
                prm.reward = rng.choice([-1, 0, 1, 2])
                prm.eps_halving = rng.choice([-1, 0, 1, 2])
                prm.eps = rng.choice([-0.1, 0.0, 0.8, 1.0, 1.5, float("nan")])
                prm.gamma = rng.choice([-1.0, 0.0, 0.9, 1.0, 2.0, float("nan")])
                prm.lr = rng.choice([-1.0, 0.0, 0.01, 1e6, float("nan"), float("inf")])
                prm.r_clip = rng.choice([-1.0, 0.0, 5.0, float("nan"), float("inf")])
            rc = L.tune_na2c(ctypes.byref(sp), ctypes.byref(o), ctypes.byref(prm), cb, None,
                             ctypes.byref(res))
        _expect(gt, rc)
        if rc == 0:
            assert 0 <= res.timed <= max(o.budget, 0) and res.failed <= res.timed


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(st.tuples(st.integers(-3, 1 << 41), st.integers(-3, 1 << 41), st.integers(-3, 1 << 41)),
       st.tuples(st.integers(-1, 5), st.integers(-1, 5), st.integers(-1, 5)),
       st.sampled_from(["f32", "bf16"]), st.booleans(), st.integers(-1, 2))
def test_malformed_spaces_are_rejected_alike(gt, orc, ext, d, dt, mc, mode):
    def size(mod):
        try:
            return mod.Space(*ext, d, dt, mc, mode=mode).size()
        except Exception:
            return None
    assert size(gt) == size(orc), (ext, d, dt, mc, mode)
