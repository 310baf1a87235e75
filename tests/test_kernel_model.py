"""A CPU model of the fast-path and direct-load GEMM kernels' addressing and
of the direct-load ring schedule, run over seeded samples of the configurations
of the 1024³ and 4096³ bf16 spaces and of the 2048³ fp32 space (A row-major
and K-major) that meet the fast path's shape conditions (plus the known
fastest 4096³ configurations). The same model run over all
98,086 such configurations of the 4096³ space finds no violation.

For each configuration the model takes the launch the library chose
(gt_lower: tile sizes, wavefronts, ring depth, LDS bytes) and checks, lane by
lane, that

* every global load of A and B stays inside its operand, for the first and
  last workgroup, split-K slice and stage (the addresses are affine in
  those indices, so the extremes bound all of them);
* every LDS write (register-staged stores and direct loads) and every LDS
  fragment read stays inside its stage and the launch's LDS allocation;
* every C element written belongs to the workgroup's tile;
* in the direct-load ring, each (stage, load) pair is issued exactly once,
  never for a stage past kLoop, into a slot whose previous stage every
  wavefront has finished reading (a barrier in between), and is complete
  (the vmcnt wait before a barrier) before any wavefront reads the stage;
* the ring slot, its LDS address and the stage origins that the direct-load
  loop carries from stage to stage equal their closed forms.

The model restates the kernels' index formulas; it shares no code with them.
"""
import functools
import itertools
import os
import random

import numpy as np
import pytest


@pytest.fixture(scope="module")
def gt():
    from paper_1909_10616_amd import gemmtune
    if not os.path.exists(gemmtune.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    gemmtune.lib()
    return gemmtune


LDS_MAX = 163840


def swz(q):
    return q ^ (((q >> 3) ^ (q >> 6)) & 7)


def bswz(k, cprb):
    j = k & 3
    return (((j << 2) | (((j ^ (j >> 1)) & 1) << 1)) ^ (((k >> 3) & 1) << 3)) & (cprb - 1)


def a_planes(I, CPR):
    """The plane layout: 16×16 MFMA and stages of two or more chunk-steps."""
    return I == 16 and CPR // 4 >= 2


def a_slot_chunk(s, I, BM, CPR):
    """(row, chunk) of the A tile that direct-load slot s of a stage holds:
    the plane layout (plane s // 4BM, [m][4] swizzled) or the stage-wide
    [m][k] layout."""
    if a_planes(I, CPR):
        lgp = lg(BM) + 2
        q = swz(s & ((1 << lgp) - 1))
        return q >> 2, ((s >> lgp) << 2) + (q & 3)
    q = swz(s)
    return q >> lg(CPR), q & (CPR - 1)


def a_read_slot(I, BM, CPR, row, grp, cs):
    """LDS slot a lane reads for A row `row`, chunk cs·G + grp."""
    G = 64 // I
    if a_planes(I, CPR):
        return cs * (BM << 2) + swz((row << 2) + grp)
    c = cs * G
    j = (c >> 3) if CPR >= 8 else 0
    xa = swz((row << lg(CPR)) + grp + 8 * j) - 8 * j
    return (xa ^ (c & 7)) + (c & ~7)


def fast_slot(idx, rows, I, CPR):
    """LDS slot of chunk idx = row·CPR + chunk of a register-staged tile (A
    [m][k] or B stored [n][k]): the stage-wide layout, swizzled."""
    return swz(idx)


def fast_read_slot(row, grp, c, CPR):
    """LDS slot a lane of the register-staged path reads for row `row`, chunk
    c + grp (c = chunk-step·G), as the kernel computes it: a per-row base for
    the 128-byte line of the chunk-step, then the chunk-step's XOR and line."""
    j = (c >> 3) if CPR >= 8 else 0
    x = swz((row << lg(CPR)) + grp + 8 * j) - 8 * j
    return (x ^ (c & 7)) + (c & ~7)


def lg(v):
    r = v.bit_length() - 1
    assert 1 << r == v
    return r


def levels(cfg):
    m, k, n, mf = cfg

    def mn(f):
        d = len(f)
        return f[0], (f[1] if d >= 3 else 1), (f[2] if d == 4 else 1), (1 if d == 1 else f[-1])

    gM, wM, rM, bM = mn(m)
    gN, wN, rN, bN = mn(n)
    dk = len(k)
    L = dict(gridM=gM, wavesM=wM, repM=rM, blkM=bM, gridN=gN, wavesN=wN, repN=rN, blkN=bN,
             kLoop=k[0], kSplit=k[1] if dk == 4 else 1,
             kSub=k[2] if dk == 4 else (k[1] if dk == 3 else 1), kBlk=1 if dk == 1 else k[-1])
    I = mf if mf in (16, 32) else (32 if bM % 32 == 0 and bN % 32 == 0 else 16)
    L.update(I=I, TM=rM * -(-bM // I), TN=rN * -(-bN // I), W=wM * wN, BM=wM * rM * bM,
             BN=wN * rN * bN, BK=L["kSub"] * L["kBlk"], WM=rM * bM, WN=rN * bN)
    return L


def dl_cap(acc):
    return 8 if acc + 96 <= 256 else 16


def tiles(L):
    return [(0, 0, 0, 0), (L["gridM"] - 1, L["gridN"] - 1, L["kSplit"] - 1, L["kLoop"] - 1)]


def frag_steps(L, CPR, lane):
    """(wavefront, its M and N coordinates, chunk-step parameters) of the
    fragment reads."""
    I = L["I"]
    G = 64 // I
    LGCPR = lg(CPR)
    grp = lane // I
    for w in range(L["W"]):
        wm, wn = w % L["wavesM"], w // L["wavesM"]
        for cs in range(CPR // G):
            c = cs * G
            j = (c >> 3) if CPR >= 8 else 0
            yield w, wm, wn, c, j, LGCPR, grp


def check_c_and_frags(L, CPR, achunks, lane, bt_rows=None, a_slots=True):
    """Fragment reads of the register-staged path (A, and B stored [n][k]
    like A): each lane's slot is in the tile and is the slot its chunk
    (row, chunk-step·G + lane group) was written to."""
    I = L["I"]
    for w, wm, wn, c, j, LGCPR, grp in frag_steps(L, CPR, lane):
        for t in range(L["TM"] if a_slots else 0):
            row = wm * L["WM"] + t * I + lane % I
            idx = fast_read_slot(row, grp, c, CPR)
            assert idx.min() >= 0 and idx.max() < achunks
            assert np.array_equal(idx, fast_slot((row << LGCPR) + c + grp, L["BM"], I, CPR))
        if bt_rows is not None:
            for t in range(L["TN"]):
                row = wn * L["WN"] + t * I + lane % I
                idx = fast_read_slot(row, grp, c, CPR)
                assert idx.min() >= 0 and idx.max() < bt_rows << LGCPR
                assert np.array_equal(idx, fast_slot((row << LGCPR) + c + grp, bt_rows, I, CPR))
    for w in range(L["W"]):
        wm, wn = w % L["wavesM"], w // L["wavesM"]
        for e in range(I * I // 64):
            r = (8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) if I == 32 else (4 * (lane >> 4) + e)
            rows = wm * L["WM"] + np.arange(L["TM"])[:, None] * I + r
            assert rows.max() < L["BM"]
        cols = wn * L["WN"] + np.arange(L["TN"])[:, None] * I + lane % I
        assert cols.max() < L["BN"]


def check_fast(L, info, M, N, K, vec=8, akm=False):
    VEC, LGV = vec, lg(vec)
    I = L["I"]
    CPR = L["BK"] // VEC
    LGCPR = lg(CPR)
    nthr = 64 * L["W"]
    BM, BN = L["BM"], L["BN"]
    achunks = BM << LGCPR
    lgnbn = lg(BN) - LGV
    bblocks = CPR << lgnbn
    stage = achunks + (BN << LGCPR)
    assert (2 if info["dbuf"] else 1) * stage * 16 <= info["lds_bytes"] <= LDS_MAX
    tid = np.arange(nthr)
    prefetch = max(-(-achunks // (nthr * 8)), -(-bblocks // nthr)) == 1
    for gm, gn, z, l in tiles(L):
        kbase = (l * L["kSplit"] + z) * L["BK"]
        a0, b0 = gm * BM * K + kbase, gn * BN + kbase * N
        if akm:
            # A K-major: VEC×VEC blocks of W (K×M), like B's
            lgnbm = lg(BM) - LGV
            ablocks = CPR << lgnbm
            if prefetch:
                nab = min(8 // VEC, -(-ablocks // nthr))
                ab = np.concatenate([np.minimum(tid + i * nthr, ablocks - 1) for i in range(nab)])
            else:
                ab = np.arange(ablocks)
            nm, kb = ab & ((1 << lgnbm) - 1), ab >> lgnbm
            for j in range(VEC):
                addr = gm * BM + (kbase + (kb << LGV) + j) * M + (nm << LGV)
                assert addr.min() >= 0 and addr.max() + VEC <= K * M
                assert fast_slot((((nm << LGV) + j) << LGCPR) + kb, BM, I, CPR).max() < achunks
            # every A chunk of the stage is written, each to its own slot
            dst = np.concatenate([fast_slot((((nm << LGV) + j) << LGCPR) + kb, BM, I, CPR)
                                  for j in range(VEC)])
            assert len(np.unique(dst)) == achunks
        elif prefetch:
            ta = np.minimum(tid, achunks - 1)
            na = min(8, -(-achunks // nthr))
            dst = []
            for i in range(na):
                e = ta + i * nthr
                addr = a0 + (ta >> LGCPR) * K + ((ta & (CPR - 1)) << LGV) + i * (nthr >> LGCPR) * K
                assert addr.min() >= 0 and addr.max() + VEC <= M * K
                # the chunk at addr is row e / CPR, chunk e mod CPR of the tile
                assert np.array_equal(addr, a0 + (e >> LGCPR) * K + ((e & (CPR - 1)) << LGV))
                dst.append(fast_slot(e, BM, I, CPR))
            dst = np.concatenate(dst)
            assert dst.max() < achunks and len(np.unique(dst)) == achunks
        else:
            e = np.arange(achunks)
            addr = a0 + (e >> LGCPR) * K + ((e & (CPR - 1)) << LGV)
            dst = fast_slot(e, BM, I, CPR)
            assert addr.max() + VEC <= M * K and dst.max() < achunks
            assert len(np.unique(dst)) == achunks
        b = np.minimum(tid, bblocks - 1) if prefetch else np.arange(bblocks)
        nb, kb = b & ((1 << lgnbn) - 1), b >> lgnbn
        bdst = []
        for j in range(VEC):
            addr = b0 + ((kb << LGV) + j) * N + (nb << LGV)
            assert addr.min() >= 0 and addr.max() + VEC <= K * N
            bdst.append(fast_slot((((nb << LGV) + j) << LGCPR) + kb, BN, I, CPR))
        bdst = np.concatenate(bdst)
        assert bdst.max() < BN << LGCPR and len(np.unique(bdst)) == BN << LGCPR
    check_c_and_frags(L, CPR, achunks, np.arange(64), bt_rows=BN)


def check_dl(L, info, M, N, K):
    I, TM, TN, W = L["I"], L["TM"], L["TN"], L["W"]
    BM, BN, BK = L["BM"], L["BN"], L["BK"]
    CPR = BK // 8
    LGCPR = lg(CPR)
    G = 64 // I
    NCS = CPR // G
    cprb = BN >> 3
    lgcprb = lg(BN) - 3
    achunks, bchunks = BM << LGCPR, BK * cprb
    stage = achunks + bchunks
    pa, pb = achunks >> 6, bchunks >> 6
    assert pa % W == 0 and pb % W == 0
    ninst = (pa + pb) // W
    na_w = pa // W
    cap = dl_cap(TM * TN * I * I // 64)
    ns = info["ring"]
    assert ninst <= cap and 2 <= ns <= 8
    assert ns * stage * 16 <= info["lds_bytes"] <= LDS_MAX
    lane = np.arange(64)
    # which chunk each A slot holds: every chunk of the stage exactly once
    slots = np.arange(achunks)
    arow, achk = a_slot_chunk(slots, I, BM, CPR)
    assert arow.max() < BM and achk.max() < CPR
    assert len(np.unique(arow * CPR + achk)) == achunks
    held = np.empty(achunks, dtype=np.int64)
    held[slots] = arow * CPR + achk
    for w in range(W):
        for i in range(ninst):
            if i < na_w:
                row, chunk = a_slot_chunk(((w + i * W) << 6) + lane, I, BM, CPR)
                off = (row * K + (chunk << 3)) * 2
                dst = (w + i * W) * 1024
                lim = M * K * 2
            else:
                s = ((w + (i - na_w) * W) << 6) + lane
                k, cs = s >> lgcprb, s & (cprb - 1)
                assert k.max() < BK
                off = (k * N + ((cs ^ bswz(k, cprb)) << 3)) * 2
                dst = (achunks + ((w + (i - na_w) * W) << 6)) * 16
                lim = K * N * 2
            assert off.max() < 2 ** 32
            assert dst + 1024 <= stage * 16
            for gm, gn, z, l in tiles(L):
                kbase = (l * L["kSplit"] + z) * BK
                base = (gm * BM * K + kbase) * 2 if i < na_w else (gn * BN + kbase * N) * 2
                assert base + off.min() >= 0 and base + off.max() + 16 <= lim
    # transposing B reads and A reads
    i16, g16 = lane & 15, lane >> 4
    kgrp = (g16 >> 1) if I == 32 else g16
    ncol0 = (16 * (g16 & 1) if I == 32 else 0) + 4 * (i16 & 3)
    krow_l = kgrp * 8 + (i16 >> 2)
    for w in range(W):
        wm, wn = w % L["wavesM"], w // L["wavesM"]
        for cs in range(NCS):
            for t in range(TN):
                col = wn * L["WN"] + t * I + ncol0
                for hh in range(2):
                    k = cs * G * 8 + krow_l + 4 * hh
                    assert k.max() < BK and col.max() < BN
                    bx = np.array([bswz(int(x), cprb) for x in k])
                    chunk = (col >> 3) ^ bx
                    addr = (k * cprb + chunk) * 16 + (col & 4) * 2
                    assert addr.min() >= 0 and addr.max() + 8 <= bchunks * 16
                    # slot (k, chunk) holds column chunk chunk ^ bswz(k) of row k
                    assert np.array_equal(chunk ^ bx, col >> 3)
            # A: the slot each lane reads holds its row and chunk
            for t in range(L["TM"]):
                row = wm * L["WM"] + t * I + lane % I
                slot = a_read_slot(I, BM, CPR, row, lane // I, cs)
                assert slot.min() >= 0 and slot.max() < achunks
                assert np.array_equal(held[slot], row * CPR + cs * G + lane // I)
    check_c_and_frags(L, CPR, achunks, lane, a_slots=False)
    ring_schedule(TM * TN, NCS, cap, ninst, ns, L["kLoop"])


@functools.lru_cache(maxsize=None)
def ring_schedule(TMTN, NCS, cap, ninst, ns, kLoop):
    """Replays the ring's control flow for one wavefront (all wavefronts run
    the same sequence) and checks issue, release and completion rules."""
    SPOS = NCS * TMTN
    NI = ninst if ninst in (cap, cap // 2) else 0
    NIE = NI or cap
    RR = 1 if NI == cap else ((SPOS // 2) // NI if NI else (SPOS - TMTN // 2) // NIE)
    R = max(RR, 1)
    ev = []

    def dma_at(st, on, pos, open_):
        i = pos // R
        ok = lambda j: (open_ or on) and (NI > 0 or j < ninst)  # noqa: E731
        if pos % R == R - 1 and i < NIE and i * R + R - 1 < SPOS and ok(i):
            ev.append(("dma", st, i))
        if pos == SPOS - 1:
            ev.extend(("dma", st, j) for j in range(SPOS // R, NIE) if ok(j))

    npro = min(ns - 1, kLoop)
    ev.extend(("dma", l, i) for l in range(npro) for i in range(ninst))
    ev += [("wait", (npro - 1) * ninst), ("bar",)]
    if ns - 1 < kLoop:
        for pos in range(TMTN):
            dma_at(ns - 1, True, pos, True)
    ev.append(("read", 0))
    for l in range(kLoop):
        open_ = l + ns < kLoop
        ld = l + ns - 1
        for cs in range(NCS - 1):
            ev.append(("read", l))
            for q in range(TMTN):
                dma_at(ld, open_ or ld < kLoop, TMTN + cs * TMTN + q, open_)
        more = open_ or l + 1 < kLoop
        if more:
            ev += [("wait", min(ns - 2, kLoop - 2 - l) * ninst), ("bar",)]
            if NCS >= 2:
                ev.append(("read", l + 1))
        for q in range(TMTN):
            dma_at(l + ns, open_ or l + ns < kLoop, q, open_)
        if NCS == 1 and more:
            ev.append(("read", l + 1))

    issued, seen, done, ready, last_read, nbar = [], set(), set(), set(), {}, 0
    for e in ev:
        if e[0] == "dma":
            _, st, i = e
            assert st < kLoop and 0 <= i < ninst and (st, i) not in seen
            seen.add((st, i))
            if st >= ns:  # slot st % ns last held stage st - ns
                assert last_read.get(st - ns, nbar) < nbar
            issued.append(st)
        elif e[0] == "wait":
            n_done = len(issued) - max(e[1], 0)
            cnt = {}
            for st in issued[:max(n_done, 0)]:
                cnt[st] = cnt.get(st, 0) + 1
            done |= {st for st, c in cnt.items() if c == ninst}
        elif e[0] == "bar":
            nbar += 1
            ready |= done
        else:
            assert e[1] in ready
            last_read[e[1]] = nbar
    assert len(seen) == kLoop * ninst
    return True


def _tuples(D, d):
    E = lg(D)
    return [tuple(2 ** e for e in es) for es in itertools.product(range(E + 1), repeat=d)
            if sum(es) == E]


def fast_candidates(D, dtype="bf16"):
    """Configurations of the D³ space (d = 4; bf16 with the MFMA coordinate,
    fp32 without) that meet the fast path's shape conditions."""
    T = _tuples(D, 4)
    out = []
    vec, esz = (8, 2) if dtype == "bf16" else (4, 4)
    for mf in ((16, 32) if dtype == "bf16" else (0,)):
        for I in ((mf,) if mf else (16, 32)):
            out += _fast_for(T, I, mf, vec, esz)
    return out


def _fast_for(T, I, mf, vec, esz):
    G = 64 // I
    IK = (16 if I == 32 else 32) if vec == 8 else (2 if I == 32 else 4)
    Ms = [t for t in T if t[3] % I == 0]
    Ks = [k for k in T if k[3] % IK == 0 and (k[2] * k[3]) % (vec * G) == 0
          and (k[2] * k[3]) // vec in (2, 4, 8, 16)]
    out = []
    for m, n in itertools.product(Ms, Ms):
        if not mf and (I == 32) != (m[3] % 32 == 0 and n[3] % 32 == 0):
            continue  # fp32: I is 32 exactly when both blocks are multiples of 32
        W = m[1] * n[1]
        acc = m[2] * (m[3] // I) * n[2] * (n[3] // I) * I * I // 64
        if W > 8 or acc > 256 or acc + 96 > 512 // ((W + 3) // 4):
            continue
        BM, BN = m[1] * m[2] * m[3], n[1] * n[2] * n[3]
        out += [(m, k, n, mf) for k in Ks if (BM + BN) * k[2] * k[3] * esz <= LDS_MAX]
    return out


def _run(gt, cfgs, D, dtype="bf16", akm=False):
    n = {"dl": 0, "fast": 0}
    code = gt.dtype_code(dtype) | (gt.A_KMAJOR if akm else 0)
    for c in cfgs:
        try:
            info = gt.lower(c, D, D, D, code)
        except gt.GemmTuneError:
            continue  # (TM, TN) without an instantiation
        L = levels(c)
        assert (info["BM"], info["BN"], info["BK"], info["waves"]) == (L["BM"], L["BN"], L["BK"], L["W"])
        if info["dl"]:
            assert not akm
            check_dl(L, info, D, D, D)
            n["dl"] += 1
        elif info["fast"]:
            check_fast(L, info, D, D, D, vec=8 if dtype == "bf16" else 4, akm=akm)
            n["fast"] += 1
    return n


def test_model_sample_1024(gt):
    n = _run(gt, random.Random(4).sample(fast_candidates(1024), 3000), 1024)
    assert n["dl"] > 100 and n["fast"] > 100, n


def test_model_sample_4096(gt):
    cands = fast_candidates(4096)
    known = [((16, 2, 4, 32), (128, 1, 1, 32), (16, 4, 2, 32), 16),
             ((16, 2, 8, 16), (128, 1, 1, 32), (16, 4, 1, 64), 16),
             ((16, 2, 4, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32),
             ((16, 4, 2, 32), (64, 1, 4, 16), (16, 2, 4, 32), 32)]
    sample = known + random.Random(5).sample(cands, 3000)
    n = _run(gt, sample, 4096)
    assert n["dl"] > 100 and n["fast"] > 100, n


@pytest.mark.parametrize("akm", [False, True])
def test_model_sample_f32(gt, akm):
    """fp32 register-staged path, A row-major and K-major (2048³)."""
    cands = fast_candidates(2048, "f32")
    n = _run(gt, random.Random(6).sample(cands, min(2000, len(cands))), 2048, "f32", akm)
    assert n["fast"] > 500 and n["dl"] == 0, n


@pytest.mark.parametrize("ns", range(2, 9))
def test_ring_schedule_shapes(ns):
    """The schedule rules over ring depths, load counts and stage counts,
    including kLoop shorter than the ring."""
    for TMTN, NCS in ((1, 1), (2, 2), (4, 1), (8, 4), (16, 2), (32, 1)):
        for cap in (8, 16):
            for ninst in sorted({1, 3, cap // 2, cap}):
                for kLoop in (1, 2, 3, ns - 1, ns, ns + 1, 2 * ns + 3):
                    if kLoop >= 1:
                        ring_schedule(TMTN, NCS, cap, ninst, ns, kLoop)


def test_ring_model_detects_a_missing_wait():
    """The schedule check is not vacuous: boundary waits that leave one more
    stage outstanding than the kernel's are caught."""
    assert _replay_with_wait_slack(4, 2, 8, 8, 3, 6, slack=0)
    with pytest.raises(AssertionError):
        _replay_with_wait_slack(4, 2, 8, 8, 3, 6, slack=1)


def _replay_with_wait_slack(TMTN, NCS, cap, ninst, ns, kLoop, slack):
    """ring_schedule with every boundary wait allowing `slack` more stages
    outstanding than the kernel's."""
    import ast
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(ring_schedule.__wrapped__))
    src = src.replace("min(ns - 2, kLoop - 2 - l) * ninst", f"(min(ns - 2, kLoop - 2 - l) + {slack}) * ninst")
    tree = ast.parse(src)
    tree.body[0].decorator_list = []
    ns_ = {}
    exec(compile(tree, "<ring>", "exec"), globals(), ns_)
    return ns_["ring_schedule"](TMTN, NCS, cap, ninst, ns, kLoop)


@pytest.mark.parametrize("ns", range(2, 9))
def test_ring_carried_state_matches_closed_forms(ns):
    """The direct-load loop carries the ring slot, its LDS byte address and the
    global byte origins of stage l + ns from stage to stage (slot + 1 with a
    wrap, origins + one stage's stride) instead of computing them from l. The
    same recurrences, replayed here, equal the closed forms for every stage:
    slot l mod ns, origin ((l·kSplit + z)·BK) bytes of A and that times N of B,
    the previous slot for stage l + ns − 1 and the next slot for stage l + 1."""
    lds0, stage16, BK, N = 4096, 32768, 32, 4096
    for kLoop in list(range(1, 21)) + [128]:
        for kSplit in (1, 4):
            for z in {0, kSplit - 1}:
                stepA = kSplit * BK * 2
                stepB = stepA * N
                zA = z * BK * 2
                cur, cur_b = 0, lds0
                ga2, gb2 = zA + ns * stepA, zA * N + ns * stepB
                for l in range(kLoop):
                    assert cur == l % ns and cur_b == lds0 + (l % ns) * stage16
                    assert ga2 == ((l + ns) * kSplit + z) * BK * 2
                    assert gb2 == ((l + ns) * kSplit + z) * BK * 2 * N
                    # stage l + ns − 1 (the first chunk-steps' window)
                    prev_b = lds0 + (ns - 1) * stage16 if cur == 0 else cur_b - stage16
                    assert prev_b == lds0 + ((l + ns - 1) % ns) * stage16
                    assert ga2 - stepA == ((l + ns - 1) * kSplit + z) * BK * 2
                    assert gb2 - stepB == ((l + ns - 1) * kSplit + z) * BK * 2 * N
                    # stage l + 1 (the next fragments)
                    nx_b = lds0 if cur + 1 == ns else cur_b + stage16
                    assert nx_b == lds0 + ((l + 1) % ns) * stage16
                    ga2 += stepA
                    gb2 += stepB
                    cur += 1
                    if cur == ns:
                        cur, cur_b = 0, lds0
                    else:
                        cur_b += stage16


# --- the generic path, the split-K fill and the launch as a whole ----------

def max_waves(I, TM, TN):
    acc = TM * TN * I * I // 64
    return 16 if acc + 96 <= 128 else (8 if acc + 96 <= 256 else 4)


def tile_map(nt, gridM, gridN, t):
    """Workgroup id t -> (tile row, tile column): the XCD-aware remap when
    the tile count is a multiple of 8, then groups of 4 tile rows."""
    if nt % 8 == 0:
        t = (t & 7) * (nt >> 3) + (t >> 3)
    per_group = 4 * gridN
    group = t // per_group
    first = group * 4
    gsize = np.minimum(gridM - first, 4)
    r = t - group * per_group
    return first + r % gsize, r // gsize


def check_tile_map(L):
    gM, gN = L["gridM"], L["gridN"]
    nt = gM * gN
    if nt <= 1 << 20:
        gm, gn = tile_map(nt, gM, gN, np.arange(nt, dtype=np.int64))
        assert gm.min() >= 0 and gm.max() < gM and gn.min() >= 0 and gn.max() < gN
        assert len(np.unique(gm * gN + gn)) == nt   # every tile exactly once
    else:
        rng = np.random.default_rng(nt)
        t = np.concatenate([np.arange(64), nt - 1 - np.arange(64), rng.integers(0, nt, 4096)])
        gm, gn = tile_map(nt, gM, gN, t.astype(np.int64))
        assert gm.min() >= 0 and gm.max() < gM and gn.min() >= 0 and gn.max() < gN


def _copy_tile(rows, cols, vec, nthr):
    """(row, column) of every element (or first element of a 16-byte chunk)
    the cooperative tile copy moves, over all threads and iterations."""
    if vec > 1:
        lgcpr = lg(cols) - lg(vec)
        e = np.arange((rows * cols) >> lg(vec))
        return e >> lgcpr, (e & ((1 << lgcpr) - 1)) << lg(vec)
    e = np.arange(rows * cols)
    return e >> lg(cols), e & (cols - 1)


def check_generic(L, info, M, N, K, dtype="bf16", akm=False):
    I, TM, TN, W = L["I"], L["TM"], L["TN"], L["W"]
    BM, BN, BK = L["BM"], L["BN"], L["BK"]
    esz, vec = (2, 8) if dtype == "bf16" else (4, 4)
    nthr = 64 * W
    assert nthr <= 64 * max_waves(I, TM, TN)        # the instantiation's launch bound
    stage = (BM + BN) * BK * esz
    assert info["lds_bytes"] == stage * (2 if info["dbuf"] else 1) <= LDS_MAX
    assert info["grid_x"] == L["gridM"] * L["gridN"] and info["grid_y"] == L["kSplit"]
    assert info["grid_x"] * nthr < 2 ** 32 and info["grid_y"] <= 65535
    assert info["grid_x"] * info["grid_y"] * nthr < 2 ** 32
    check_tile_map(L)
    # vector copies only where the lowering allows them (16-byte aligned rows)
    a_vec = vec if ((BM % vec == 0 and M % vec == 0) if akm else (BK % vec == 0 and K % vec == 0)) else 1
    b_vec = vec if (BN % vec == 0 and N % vec == 0) else 1
    for gm, gn, z, l in tiles(L):
        kbase = (l * L["kSplit"] + z) * BK
        for av in sorted({1, a_vec}):
            if akm:   # BK rows of BM contiguous m from W (K×M)
                r, c = _copy_tile(BK, BM, av, nthr)
                src = gm * BM + (kbase + r) * M + c
                assert src.min() >= 0 and src.max() + av <= K * M
                assert ((r << lg(BM)) + c).max() + av <= BM * BK
            else:
                r, c = _copy_tile(BM, BK, av, nthr)
                src = (gm * BM + r) * K + kbase + c
                assert src.min() >= 0 and src.max() + av <= M * K
                assert ((r << lg(BK)) + c).max() + av <= BM * BK
        for bv in sorted({1, b_vec}):
            r, c = _copy_tile(BK, BN, bv, nthr)
            src = (kbase + r) * N + gn * BN + c
            assert src.min() >= 0 and src.max() + bv <= K * N
            assert ((r << lg(BN)) + c).max() + bv <= BK * BN
    # fragment gathers: rows / columns and k inside the stage when unguarded
    lane = np.arange(64)
    IK = (16 if I == 32 else 32) if dtype == "bf16" else (2 if I == 32 else 4)
    EPL = 8 if dtype == "bf16" else 1
    tpbM = L["blkM"] // I if L["blkM"] >= I else 1
    tpbN = L["blkN"] // I if L["blkN"] >= I else 1
    nkk = -(-L["kBlk"] // IK)
    sr, sk = (1, BM) if akm else (BK, 1)
    # k inside the stage, s·kBlk + kl for the first and last sub-step s and
    # every k-chunk (the index is affine in s), this lane's EPL elements
    subs = np.array(sorted({0, L["kSub"] - 1}))[:, None, None, None]
    kl = (np.arange(nkk)[None, :, None, None] * IK + (lane // I)[None, None, None, :] * EPL
          + np.arange(EPL)[None, None, :, None])
    kin = kl < L["kBlk"]
    kidx = subs * L["kBlk"] + kl
    for w in range(W):
        wm, wn = w % L["wavesM"], w // L["wavesM"]
        for t in range(TM):
            inn = (t % tpbM) * I + lane % I
            row = wm * L["WM"] + (t // tpbM) * L["blkM"] + inn
            ok = inn < L["blkM"]
            assert row[ok].max(initial=0) < BM
            okk = ok & kin
            idx = row * sr + kidx * sk
            assert idx[np.broadcast_to(okk, idx.shape)].max(initial=0) < BM * BK
        for t in range(TN):
            inn = (t % tpbN) * I + lane % I
            col = wn * L["WN"] + (t // tpbN) * L["blkN"] + inn
            ok = inn < L["blkN"]
            assert col[ok].max(initial=0) < BN
            okk = ok & kin
            idx = kidx * BN + col
            assert idx[np.broadcast_to(okk, idx.shape)].max(initial=0) < BK * BN
        # epilogue: guarded (row, column) of every accumulator element
        i = np.arange(TM)[:, None, None]
        e = np.arange(I * I // 64)[None, :, None]
        lr = lane[None, None, :]
        ri = (i % tpbM) * I + ((8 * (e >> 2) + 4 * (lr >> 5) + (e & 3)) if I == 32
                               else (4 * (lr >> 4) + e))
        r = (wm * L["WM"] + (i // tpbM) * L["blkM"] + ri)[:, :, None, :]
        j = np.arange(TN)[:, None]
        ci = (j % tpbN) * I + lane[None, :] % I
        c = (wn * L["WN"] + (j // tpbN) * L["blkN"] + ci)[None, None, :, :]
        ok = (ri < L["blkM"])[:, :, None, :] & (ci < L["blkN"])[None, None, :, :]
        for gm, gn, _, _ in tiles(L):
            g = (gm * BM + r) * N + gn * BN + c
            assert g[ok].max(initial=0) < M * N and g[ok].min(initial=0) >= 0


@functools.lru_cache(maxsize=None)
def check_fill(n):
    """The split-K clear: ≤ 65536 blocks of 256 threads, grid-stride loop;
    thread f = block·256 + tid writes f, f + stride, … below n."""
    blocks = min(-(-n // 256), 65536)
    stride = blocks * 256
    assert stride <= 2 ** 32 and (stride >= n or blocks == 65536)
    first = np.arange(stride, dtype=np.int64)
    # every element of C written exactly once
    assert int(np.maximum(0, -(-(n - first) // stride)).sum()) == n
    return True


def run_models(gt, cfgs, M, N, K, dtype="bf16", akm=False):
    n = {"dl": 0, "fast": 0, "generic": 0}
    code = gt.dtype_code(dtype) | (gt.A_KMAJOR if akm else 0)
    for c in cfgs:
        info = gt.lower(c, M, N, K, code)
        L = levels(c)
        # the launch the library chose is the level mapping's (tile, wavefronts,
        # MFMA size, MFMA tiles per wavefront)
        assert (info["BM"], info["BN"], info["BK"], info["waves"], info["I"], info["TM"],
                info["TN"]) == (L["BM"], L["BN"], L["BK"], L["W"], L["I"], L["TM"], L["TN"]), c
        if info["dl"]:
            check_dl(L, info, M, N, K)
            n["dl"] += 1
        elif info["fast"]:
            check_fast(L, info, M, N, K, vec=8 if dtype == "bf16" else 4, akm=akm)
            n["fast"] += 1
        else:
            check_generic(L, info, M, N, K, dtype, akm)
            n["generic"] += 1
        if L["kSplit"] > 1:
            check_fill(M * N)
    return n


def _draws(size, seed, count):
    """The first `count` ranks the random search draws (SplitMix64 mod |ξ|)."""
    out, st = [], seed
    for _ in range(count):
        st = (st + 0x9E3779B97F4A7C15) & (2 ** 64 - 1)
        z = st
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & (2 ** 64 - 1)
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & (2 ** 64 - 1)
        out.append((z ^ (z >> 31)) % size)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_random_search_candidates_4096(gt, orc, seed):
    """Every configuration the equal-budget random search times on the 4096³
    bf16 space (seeds 0-5, budget 1000; draws are cost-independent) passes
    the kernel models: in-bounds global, LDS and C accesses, the tile map a
    bijection, the launch within the instantiation's bound, and the whole
    dispatch below 2^32 work-items. The draw sequence of every seed also holds
    configurations that meet every other legitimacy clause but launch 2^32 or
    more work-items (up to 2^40): the whole-launch clause rejects those."""
    D = 4096
    sp = gt.Space(D, D, D, (4, 4, 4), "bf16", True)
    timed = []
    gt.tune_random(sp, budget=1000, seed=seed, cost_fn=lambda c, r: (timed.append(c), 1.0)[1])
    assert len(timed) == 1000
    n = run_models(gt, timed, D, D, D)
    assert n["generic"] > 900, n
    osp = orc.Space(D, D, D, (4, 4, 4), "bf16", True)
    oversized = 0
    for r in _draws(sp.size(), seed, 3000):
        c = osp.unrank(r)
        L = levels(c)
        items = L["gridM"] * L["gridN"] * L["kSplit"] * 64 * L["W"]
        if items >= 2 ** 32 and not osp.legit(c):
            oversized += 1
    assert oversized > 0


@pytest.mark.parametrize("space", [(4096, 4096, 4096, "bf16"), (4096, 11008, 4096, "bf16"),
                                   (64, 4096, 4096, "bf16"), (1024, 1024, 1024, "f32")])
def test_model_legitimate_sample(gt, space):
    """A seeded sample of legitimate configurations of four workload spaces,
    every path."""
    M, N, K, dt = space
    sp = gt.Space(M, N, K, (4, 4, 4), dt, dt == "bf16")
    rng = random.Random(M * 7 + N)
    cfgs = []
    while len(cfgs) < 400:
        c = sp.unrank(rng.randrange(sp.size()))
        if sp.legit(c):
            cfgs.append(c)
    n = run_models(gt, cfgs, M, N, K, dt)
    assert n["generic"] > 200, n


def test_model_drawn_cases(gt):
    """Every case of the seeded list the GPU parity test runs (random odd
    shapes, one to four levels, both dtypes and layouts, every path) passes
    the kernel models before any of it reaches a GPU."""
    from drawn_cases import cases_with_env_seeds
    n = {"dl": 0, "fast": 0, "generic": 0}
    for M, N, K, d, dt, mc, akm, cfg in cases_with_env_seeds(gt):
        for k, v in run_models(gt, [cfg], M, N, K, dt, akm).items():
            n[k] += v
    assert n["dl"] >= 5 and n["fast"] >= 10 and n["generic"] >= 40, n


def _wide(K=256, N=256):
    return (256, N, K, ((1, 2, 4, 32), (K // 32, 1, 1, 32) if K > 256 else (8, 1, 1, 32),
                        (N // 256, 4, 2, 32), 16))


@pytest.mark.parametrize("case", [
    # (M, N, K, configuration, direct-load expected, ring offsets would wrap):
    # a 256x256 tile, 32-deep stages
    (*_wide(K=7 << 20), 1, 0), (*_wide(K=1 << 23), 0, 0), (*_wide(K=9 << 20), 0, 1),
    (*_wide(N=15 << 22), 1, 0), (*_wide(N=1 << 26), 0, 0), (*_wide(N=9 << 23), 0, 1),
], ids=["BMxK-below-2^31", "BMxK-at-2^31", "BMxK-offsets-wrap",
        "BKxN-below-2^31", "BKxN-at-2^31", "BKxN-offsets-wrap"])
def test_direct_load_offsets_stay_32_bit(gt, case):
    """The direct-load kernel keeps each lane's global offset from the stage
    origin in 32 bits (bytes below 2^32 while BM·K and BK·N stay below 2^31
    elements). Shapes that large are legitimate (operands of several GiB fit
    in HBM), so lowering leaves the ring for the register-staged kernel,
    whose offsets are 64-bit, from that bound on (one row early: at the bound
    itself the offsets would still fit); beyond it they would wrap."""
    M, N, K, cfg, dl, wraps = case
    sp = gt.Space(M, N, K, (4, 4, 4), "bf16", True)
    assert sp.legit(cfg)
    info = gt.lower(cfg, M, N, K, "bf16")
    assert info["fast"] == 1 and info["dl"] == dl, info
    # the ring's per-lane offsets from the stage origins, over every A and B
    # slot of a stage (the formulas of the direct-load model above)
    L = levels(cfg)
    BM, BN, BK, I = L["BM"], L["BN"], L["BK"], L["I"]
    CPR, cprb = BK // 8, BN >> 3
    row, chunk = a_slot_chunk(np.arange(BM * CPR), I, BM, CPR)
    k = np.arange(BK * cprb) >> (lg(BN) - 3)
    cs = np.arange(BK * cprb) & (cprb - 1)
    bx = np.array([bswz(int(x), cprb) for x in k])
    worst = max(int(((row * K + (chunk << 3)) * 2).max()), int(((k * N + ((cs ^ bx) << 3)) * 2).max()))
    assert (worst >= 2 ** 32) == bool(wraps), worst
    assert not (dl and wraps)


def test_model_every_configuration_of_the_search_spaces(gt):
    """Every legitimate configuration of the small drawn spaces the GPU
    search test tunes over (a search may time any of them, whatever the
    timings), every path, passes the kernel models."""
    from drawn_cases import draw_small_spaces
    n = {"dl": 0, "fast": 0, "generic": 0}
    total = 0
    for M, N, K, d, dt, mc, akm in draw_small_spaces(gt):
        sp = gt.Space(M, N, K, d, dt, mc, a_kmajor=akm)
        legit = [c for c, j in sp.enumerate() if j]
        for k, v in run_models(gt, legit, M, N, K, dt, akm).items():
            n[k] += v
        total += len(legit)
    assert sum(n.values()) == total and n["generic"] > 0 and n["fast"] > 0, n
