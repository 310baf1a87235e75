"""The host entry points called from several threads at once (ctypes drops
the interpreter lock for the duration of each call): the three searches with
synthetic costs reproduce their single-threaded results exactly, and each
thread reads its own last-error message."""
import threading

import pytest


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


SPACES = [(256, 256, 256, (3, 3, 3), "f32", False), (512, 256, 1024, (4, 4, 4), "bf16", True),
          (96, 80, 48, (4, 3, 4), "bf16", True), (1024, 1024, 1024, (4, 2, 4), "f32", False)]


def _job(gt, i):
    M, N, K, d, dt, mc = SPACES[i % len(SPACES)]
    sp = gt.Space(M, N, K, d, dt, mc, mode=i % 2)
    cost = lambda c, r: 1.0 + ((r * 2654435761 + i) % 997) / 997.0   # noqa: E731
    s0 = sp.paper_s0()
    kind = i % 3
    if kind == 0:
        r = gt.tune_gbfs(sp, 200, s0=s0, rho=3, seed=i, cost_fn=cost)
    elif kind == 1:
        r = gt.tune_random(sp, 200, seed=i, cost_fn=cost)
    else:
        r = gt.tune_na2c(sp, 120, s0=s0, seed=i, cost_fn=cost)
    return [e["rank"] for e in r["log"]], r["best"], r["best_cost"]


def test_concurrent_searches_match_serial(gt):
    jobs = list(range(24))
    serial = {i: _job(gt, i) for i in jobs}
    got, errors = {}, []

    def worker(ids):
        try:
            for i in ids:
                got[i] = _job(gt, i)
        except Exception as e:   # reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(jobs[t::8],)) for t in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert got == serial


def test_last_error_is_per_thread(gt):
    """Each thread provokes a different failure and then reads back its own
    message, while the other threads keep failing in between."""
    out, barrier = {}, threading.Barrier(6)

    def worker(t):
        bad = gt.Space(0, 8, 8, (1, 1, 1), "f32", False) if t % 2 else \
            gt.Space(8, 8, 8, (1, 1, 1), "f32", False, mode=7)
        msgs = set()
        for _ in range(200):
            try:
                bad.size()
            except gt.GemmTuneError as e:
                msgs.add(str(e))
            barrier.wait() if _ == 0 else None
        out[t] = msgs

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(6)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    for t, msgs in out.items():
        assert len(msgs) == 1, msgs
        assert ("extents" in next(iter(msgs))) == bool(t % 2)
