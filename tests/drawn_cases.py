"""Seeded draws of whole kernel-family cases: a shape with odd cofactors
(extents q·2^e, q odd, from 1 up to a few thousand), one to four levels per
dimension (Eq.1–4), either input dtype, the MFMA coordinate on some bf16
spaces, A row-major or K-major (the perceptron layout of §5), and one
legitimate configuration (Eq.5). Half the cases draw it uniformly by rank
(which lands on the generic kernel almost always); the other half take a
short random walk over neighbours (Eq.6) from the hand-made 128×128 or 64×64
start on a four-level space whose extents allow it, the region where the
register-staged and direct-load kernels apply.

The CPU kernel model and the GPU parity test take the same list, so every
configuration the GPU runs has first been checked for in-bounds global, LDS
and C accesses on the host. Drawing uses the library's space only (rank,
unrank, legitimacy, lowering); nothing here computes a product.
"""
import os
import random

ODD = (1, 3, 5, 7, 9, 15)
MAX_MACS = 1 << 26          # keeps the fp64 oracle product of every case well under a second
MAX_WORKGROUPS = 1 << 16    # keeps each launch short


def draw_cases(gt, count=96, seed=0x1909_10616, max_macs=MAX_MACS):
    """`count` cases (M, N, K, d, dtype, mfma_coord, a_kmajor, cfg) of at
    most `max_macs` multiply-adds; the list depends on the arguments only."""
    rng = random.Random(seed)
    cases = []
    while len(cases) < count:
        walk = len(cases) % 2 == 1
        if walk:
            M, N = (rng.choice(ODD) << rng.randint(6, 9) for _ in range(2))
            K = rng.choice(ODD) << rng.randint(5, 10)
            d = (4, 4, 4)
        else:
            M, N, K = (rng.choice(ODD) << rng.randint(0, 10) for _ in range(3))
            d = tuple(rng.randint(1, 4) for _ in range(3))
        if M * N * K > max_macs:
            continue
        dt = rng.choice(("f32", "bf16"))
        mc = dt == "bf16" and rng.random() < 0.7
        akm = rng.random() < 0.25
        sp = gt.Space(M, N, K, d, dt, mc, a_kmajor=akm)
        code = gt.dtype_code(dt) | (gt.A_KMAJOR if akm else 0)
        size = sp.size()
        for _ in range(400):
            if walk:
                c = gt.hand_start(M, N, K, d, mc)
                for _ in range(rng.randint(0, 12)):
                    c = rng.choice(sp.neighbours(c))[0]
            else:
                c = sp.unrank(rng.randrange(size))
            if not sp.legit(c):
                continue
            info = gt.lower(c, M, N, K, code)
            if info["grid_x"] * info["grid_y"] > MAX_WORKGROUPS:
                continue
            cases.append((M, N, K, d, dt, mc, akm, c))
            break
    return cases


def cases_with_env_seeds(gt):
    """The committed list, plus 100 cases per seed named in GT_DRAWN_SEEDS
    (e.g. "11-14,21-40") for a wider sweep, of at most GT_DRAWN_MAX_MACS
    multiply-adds each (default 2^26; e.g. 1073741824 for larger shapes)."""
    cases = draw_cases(gt)
    bound = int(os.environ.get("GT_DRAWN_MAX_MACS", MAX_MACS))
    for part in filter(None, os.environ.get("GT_DRAWN_SEEDS", "").split(",")):
        lo, _, hi = part.partition("-")
        for seed in range(int(lo), int(hi or lo) + 1):
            cases += draw_cases(gt, count=100, seed=seed, max_macs=bound)
    return cases


def draw_small_spaces(gt, count=6, seed=0x5EA5C4, max_legit=3000):
    """`count` spaces (M, N, K, d, dtype, mfma_coord, a_kmajor) with odd
    cofactors, small enough that every legitimate configuration can be
    checked on the CPU (at most `max_legit` of them) and a search on the GPU
    stays short, each with a legitimate start state."""
    rng = random.Random(seed)
    out = []
    while len(out) < count:
        M, N = (rng.choice(ODD) << rng.randint(4, 8) for _ in range(2))
        K = rng.choice(ODD) << rng.randint(4, 9)
        if M * N * K > (1 << 24):
            continue
        d = tuple(rng.randint(2, 4) for _ in range(3))
        dt = rng.choice(("f32", "bf16"))
        mc = dt == "bf16" and rng.random() < 0.5
        akm = rng.random() < 0.25
        sp = gt.Space(M, N, K, d, dt, mc, a_kmajor=akm)
        legit = [c for c, j in sp.enumerate() if j]
        if not 50 <= len(legit) <= max_legit:
            continue
        out.append((M, N, K, d, dt, mc, akm))
    return out
