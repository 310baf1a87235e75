"""Pins of the oracle's N-A2C (§4.3, Alg.2) against facts outside its code:
finite-difference gradients of both networks, the softmax's support, the
walk's first steps recomputed from the SplitMix64 definition, the graph
distance of every timed state from the states timed before it, the budget,
uniqueness and s* rules, and convergence on a unimodal landscape."""
import math
from collections import deque

import numpy as np
import pytest


def _space(orc, mode=None, mfma=False):
    mode = orc.ANY_PAIR if mode is None else mode
    return orc.Space(64, 32, 64, (3, 2, 3), "bf16" if mfma else "f32", mfma, mode=mode)


def _available(sp, cfg):
    """Action list in the reading's order and which actions are available."""
    acts = []
    for x, f in enumerate(cfg[:3]):
        d = len(f)
        for i in range(d):
            for j in range(d):
                if i != j and (sp.mode == 1 or abs(i - j) == 1):
                    acts.append((x, i, j, f[j] % 2 == 0))
    if sp.mfma_coord:
        acts.append(("mfma", 0, 0, True))
    return acts


@pytest.mark.parametrize("mfma", [False, True])
def test_gradients_match_finite_differences(orc, mfma):
    sp = _space(orc, mfma=mfma)
    cfg = ((4, 2, 8), (8, 8), (2, 4, 4), 16 if mfma else 0)
    assert sp.member(cfg)
    acts = _available(sp, cfg)
    a = next(k for k, t in enumerate(acts) if t[3])
    base = orc.na2c_probe(sp, cfg, a, seed=3, params={"H": 6})
    rng = np.random.default_rng(0)
    theta = rng.normal(0, 0.5, base["n_actor"])
    phi = rng.normal(0, 0.5, base["n_critic"])
    p0 = orc.na2c_probe(sp, cfg, a, seed=3, params={"H": 6}, actor=theta, critic=phi)
    h = 1e-6
    for k in range(base["n_actor"]):
        tp, tm = theta.copy(), theta.copy()
        tp[k] += h
        tm[k] -= h
        lp = math.log(orc.na2c_probe(sp, cfg, a, 3, {"H": 6}, tp, phi)["pi"][a])
        lm = math.log(orc.na2c_probe(sp, cfg, a, 3, {"H": 6}, tm, phi)["pi"][a])
        assert abs((lp - lm) / (2 * h) - p0["g_actor"][k]) <= 1e-6 * (1 + abs(p0["g_actor"][k])), k
    for k in range(base["n_critic"]):
        cp, cm = phi.copy(), phi.copy()
        cp[k] += h
        cm[k] -= h
        vp = orc.na2c_probe(sp, cfg, a, 3, {"H": 6}, theta, cp)["v"]
        vm = orc.na2c_probe(sp, cfg, a, 3, {"H": 6}, theta, cm)["v"]
        assert abs((vp - vm) / (2 * h) - p0["g_critic"][k]) <= 1e-6 * (1 + abs(p0["g_critic"][k])), k


def test_policy_support_is_the_available_actions(orc):
    sp = _space(orc)
    for cfg in [((64, 1, 1), (64, 1), (32, 1, 1), 0), ((1, 1, 64), (1, 64), (1, 1, 32), 0),
                ((8, 8, 1), (8, 8), (4, 2, 4), 0)]:
        acts = _available(sp, cfg)
        pr = orc.na2c_probe(sp, cfg, next(k for k, t in enumerate(acts) if t[3]), seed=1)
        pi = pr["pi"]
        assert len(pi) == len(acts)
        assert abs(pi.sum() - 1.0) < 1e-12
        for k, t in enumerate(acts):
            assert (pi[k] > 0) == t[3], (cfg, k)


def _splitmix(state):
    state = (state + 0x9E3779B97F4A7C15) & (2 ** 64 - 1)
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & (2 ** 64 - 1)
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & (2 ** 64 - 1)
    return state, z ^ (z >> 31)


def test_random_walk_first_episode_from_the_definition(orc):
    """eps = 0: every step is a uniform pick among the available actions
    (SplitMix64 mod their count, in list order), so the first episode's
    collected states follow from the definition alone."""
    sp = _space(orc)
    s0 = sp.paper_s0()
    prm = {"eps": 0.0, "B": 5, "T": 3}
    res = orc.na2c(sp, s0, 6, 11, lambda c, r: 1.0, prm)
    state = 11
    want, seen = [], {sp.rank(s0)}
    while len(want) < 5:
        s = s0
        for _ in range(3):
            acts = _available(sp, s)
            avail = [t for t in acts if t[3]]
            state, _ = _splitmix(state)    # the ε draw (never below 0)
            state, z2 = _splitmix(state)   # the action draw
            x, i, j, _ = avail[z2 % len(avail)]
            f = [list(t) for t in s[:3]]
            f[x][i] *= 2
            f[x][j] //= 2
            s = (tuple(f[0]), tuple(f[1]), tuple(f[2]), s[3])
            r = sp.rank(s)
            if sp.legit(s) and r not in seen and len(want) < 5:
                want.append(r)
                seen.add(r)
    assert res["log_ranks"][1:6] == want


def _distances(orc, sp, src, limit):
    """Graph distances (neighbour moves) from src, up to `limit`."""
    dist = {sp.rank(src): 0}
    dq = deque([src])
    while dq:
        s = dq.popleft()
        ds = dist[sp.rank(s)]
        if ds == limit:
            continue
        for t, _ in sp.neighbours(s):
            r = sp.rank(t)
            if r not in dist:
                dist[r] = ds + 1
                dq.append(t)
    return dist


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_trajectory_rules(orc, seed):
    """Budget, uniqueness and legitimacy of the timed states, s* = the first
    minimum, and every timed state within T + 8 moves of the best state timed
    before it at some point (its episode's centre; walks grow from T to at
    most T + 8 steps)."""
    sp = _space(orc, mfma=True)
    s0 = sp.paper_s0()
    costs = {}

    def cost(c, r):
        costs.setdefault(r, 1.0 + ((r * 2654435761 + seed) % 997) / 997.0)
        return costs[r]

    T = 3
    res = orc.na2c(sp, s0, 80, seed, cost, {"T": T, "B": 6})
    T += 8  # walks lengthen by up to 8 steps after episodes that collect nothing
    log = res["log_ranks"]
    assert res["timed"] == len(log) <= 80 and len(set(log)) == len(log)
    assert all(sp.legit(sp.unrank(r)) for r in log)
    i = min(range(len(log)), key=lambda t: (res["log_costs"][t], t))
    assert sp.rank(res["best"]) == log[i] and res["best_cost"] == res["log_costs"][i]
    # the centre of an episode is the best state timed before it: one of the
    # running-minimum records of the log
    costs_log = res["log_costs"]
    records, dist = [], {}
    for k in range(1, len(log)):
        j = k - 1
        if not records or costs_log[j] < costs_log[records[-1]]:
            records.append(j)
            dist[j] = _distances(orc, sp, sp.unrank(log[j]), T)
        assert any(dist[j].get(log[k], T + 1) <= T for j in records), k


def test_unimodal_landscape_reaches_the_target(orc):
    sp = orc.Space(256, 256, 256, (3, 2, 3), "f32", False, mode=orc.ANY_PAIR)
    target = ((16, 2, 8), (16, 16), (8, 2, 16), 0)
    assert sp.legit(target)

    def cost(c, r):
        e = [math.log2(v) for t in c[:3] for v in t]
        g = [math.log2(v) for t in target[:3] for v in t]
        return 1.0 + sum(abs(a - b) for a, b in zip(e, g))

    res = orc.na2c(sp, sp.paper_s0(), 600, 5, cost)
    assert res["best"] == target and res["best_cost"] == 1.0


# --- the update the search applies, pinned to finite differences -----------

def _fd_grads(orc, sp, cfg, a, theta, crit, H, h=1e-6):
    """Central differences of log π(a|s) and V(s), from the networks'
    forward outputs only."""
    prm = {"H": H}
    ga = np.zeros_like(theta)
    gc = np.zeros_like(crit)
    for k in range(len(theta)):
        tp, tm = theta.copy(), theta.copy()
        tp[k] += h
        tm[k] -= h
        lp = math.log(orc.na2c_probe(sp, cfg, a, 0, prm, tp, crit)["pi"][a])
        lm = math.log(orc.na2c_probe(sp, cfg, a, 0, prm, tm, crit)["pi"][a])
        ga[k] = (lp - lm) / (2 * h)
    for k in range(len(crit)):
        cp, cm = crit.copy(), crit.copy()
        cp[k] += h
        cm[k] -= h
        vp = orc.na2c_probe(sp, cfg, a, 0, prm, theta, cp)["v"]
        vm = orc.na2c_probe(sp, cfg, a, 0, prm, theta, cm)["v"]
        gc[k] = (vp - vm) / (2 * h)
    return ga, gc


def _fd_update(orc, sp, tr, theta, crit, H, gamma, lr):
    """θ + lr·δ·∇ with δ = r + γV(s') − V(s) and ∇ by finite differences,
    everything at the parameters before the update (§4.3: actor-critic with
    the TD(0) advantage)."""
    s, a, r, s2 = tr
    v_s = orc.na2c_probe(sp, s, a, 0, {"H": H}, theta, crit)["v"]
    v_s2 = orc.na2c_probe(sp, s2, 0, 0, {"H": H}, theta, crit)["v"]
    delta = r + gamma * v_s2 - v_s
    ga, gc = _fd_grads(orc, sp, s, a, theta, crit, H)
    return theta + lr * delta * ga, crit + lr * delta * gc


def _close(got, want, base):
    step = want - base
    err = np.abs((got - base) - step)
    assert np.all(err <= 1e-8 + 1e-5 * np.abs(step)), float(err.max())


def _transitions(orc, sp):
    s = ((4, 2, 8), (8, 8), (2, 4, 4), 16)
    acts = _available(sp, s)
    a = next(k for k, t in enumerate(acts) if t[3] and t[0] == 0)
    x, i, j, _ = acts[a]
    f = [list(t) for t in s[:3]]
    f[x][i] *= 2
    f[x][j] //= 2
    s2 = (tuple(f[0]), tuple(f[1]), tuple(f[2]), s[3])
    b = next(k for k, t in enumerate(acts) if t[0] == "mfma")
    s3 = (s[0], s[1], s[2], 32)
    return (s, a, 0.73, s2), (s, b, 1.9, s3)


def test_applied_update_is_the_actor_critic_step(orc):
    """One transition with hand-set weights: the parameters after the
    oracle's training step equal θ + lr·δ·∇ (gradients by finite
    differences, δ the TD(0) error at the weights before the step). A wrong
    sign, a wrong TD target or gradients taken after the step fail this."""
    sp = _space(orc, mfma=True)
    H = 5
    n = orc.na2c_probe(sp, sp.paper_s0(), 0, 0, {"H": H})
    rng = np.random.default_rng(1)
    theta = rng.normal(0, 0.6, n["n_actor"])
    crit = rng.normal(0, 0.6, n["n_critic"])
    t1, _ = _transitions(orc, sp)
    for gamma, lr in ((0.9, 0.5), (0.0, 0.25)):
        want_a, want_c = _fd_update(orc, sp, t1, theta, crit, H, gamma, lr)
        got_a, got_c = orc.na2c_train(sp, [t1], theta, crit,
                                      {"H": H, "gamma": gamma, "lr": lr})
        _close(got_a, want_a, theta)
        _close(got_c, want_c, crit)


def test_updates_apply_in_memory_order(orc):
    """Two transitions: the second update is taken at the parameters the
    first one left (one pass over the memory, oldest first)."""
    sp = _space(orc, mfma=True)
    H = 4
    n = orc.na2c_probe(sp, sp.paper_s0(), 0, 0, {"H": H})
    rng = np.random.default_rng(2)
    theta = rng.normal(0, 0.6, n["n_actor"])
    crit = rng.normal(0, 0.6, n["n_critic"])
    t1, t2 = _transitions(orc, sp)
    a1, c1 = _fd_update(orc, sp, t1, theta, crit, H, 0.9, 0.4)
    a2, c2 = _fd_update(orc, sp, t2, a1, c1, H, 0.9, 0.4)
    got_a, got_c = orc.na2c_train(sp, [t1, t2], theta, crit, {"H": H, "lr": 0.4})
    _close(got_a, a2, theta)
    _close(got_c, c2, crit)
    rev_a, _ = orc.na2c_train(sp, [t2, t1], theta, crit, {"H": H, "lr": 0.4})
    assert np.abs(rev_a - got_a).max() > 1e-6


def _step(sp, cfg, act):
    x, i, j, _ = act
    if x == "mfma":
        return (cfg[0], cfg[1], cfg[2], 32 if cfg[3] == 16 else 16)
    f = [list(t) for t in cfg[:3]]
    f[x][i] *= 2
    f[x][j] //= 2
    return (tuple(f[0]), tuple(f[1]), tuple(f[2]), cfg[3])


@pytest.mark.parametrize("reward", [0, 1])
def test_stored_transitions_and_rewards(orc, reward):
    """Every transition the search stores is (s, a, r, s') with s' the state
    just timed, s an earlier-timed state and step(s, a) = s'; each timed s'
    stores one per timed neighbour that leads into it; r = 1/cost(s') (§4.1),
    or the clipped log ratio for the variant."""
    sp = _space(orc, mfma=True)
    s0 = sp.paper_s0()

    def cost(c, r):
        return 0.5 + ((r * 40503 + 7) % 101) / 37.0

    res = orc.na2c(sp, s0, 60, 4, cost, {"reward": reward, "B": 4}, trace_cap=100000)
    log = res["log_ranks"]
    pos = {r: k for k, r in enumerate(log)}
    trans = res["transitions"]
    assert len(trans) == res["n_transitions"] > 0
    by_target = {}
    for rs, a, r, rs2 in trans:
        s, s2 = sp.unrank(rs), sp.unrank(rs2)
        acts = _available(sp, s)
        assert acts[a][3] and _step(sp, s, acts[a]) == s2
        assert pos[rs] < pos[rs2]
        c, c2 = cost(s, rs), cost(s2, rs2)
        if reward == 0:
            assert r == 1.0 / c2
        else:
            assert r == max(-5.0, min(5.0, math.log(c / c2)))
        by_target.setdefault(rs2, []).append(rs)
    # one transition per earlier-timed state one move away, for every s'
    # timed after the first
    for k, rs2 in enumerate(log[1:], 1):
        s2 = sp.unrank(rs2)
        want = sorted(pos_r for pos_r in log[:k]
                      if any(_step(sp, sp.unrank(pos_r), t) == s2
                             for t in _available(sp, sp.unrank(pos_r)) if t[3]))
        assert sorted(by_target.get(rs2, [])) == want, k


def test_policy_walk_follows_pi(orc):
    """ε = 1: every walk step draws u from SplitMix64 and takes the first
    available action whose cumulative π exceeds u (π from the initial
    weights: no training happens before the first timing)."""
    sp = _space(orc)
    s0 = sp.paper_s0()
    res = orc.na2c(sp, s0, 5, 9, lambda c, r: 1.0, {"eps": 1.0, "B": 4, "T": 3})
    state = 9
    want, seen = [], {sp.rank(s0)}
    while len(want) < 4:
        s = s0
        for _ in range(3):
            acts = _available(sp, s)
            state, _ = _splitmix(state)    # the ε draw (always below 1)
            state, z = _splitmix(state)
            u = (z >> 11) / float(1 << 53)
            pi = orc.na2c_probe(sp, s, next(k for k, t in enumerate(acts) if t[3]), seed=9)["pi"]
            cdf, pick = 0.0, None
            for k, t in enumerate(acts):
                if not t[3]:
                    continue
                pick = k
                cdf += pi[k]
                if u < cdf:
                    break
            s = _step(sp, s, acts[pick])
            r = sp.rank(s)
            if sp.legit(s) and r not in seen and len(want) < 4:
                want.append(r)
                seen.add(r)
    assert res["log_ranks"][1:5] == want
