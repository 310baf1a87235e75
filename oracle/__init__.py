"""CPU oracle for the tuned-GEMM path — TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It wraps ``oracle.c`` (plain C, fp64,
built with gcc) through ctypes and shares no code with the GPU library:

* ``gemm`` / ``gemm_entries`` — C = A·B by the three-loop definition (§3.2),
  fp64, on the exact widening of the input bytes.
* ``Space`` — the configuration space of Eq.1–4, rank/unrank in the frozen
  canonical order, legitimacy J (Eq.5), neighbours g(s) (Eq.6, Eq.9).
* ``gbfs`` — Alg.1 (§4.2) with a caller-supplied cost function;
  ``random_search`` — the equal-budget baseline (§5); ``na2c`` — Alg.2
  (§4.3), with ``na2c_probe`` / ``na2c_train`` exposing its networks and
  its training step.

The hardware part of J (register, LDS and grid limits) has no value in the
paper to pin it; it is checked by hand-worked cases, by every J=1
configuration launching on the GPU, and in one direction against the
compiled kernels' metadata (whatever J admits fits the kernel it launches);
where exactly J draws its line has nothing outside it to pin to.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32, BF16 = 0, 1
ADJACENT, ANY_PAIR = 0, 1
MAXD = 4


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc into liboracle.so (beside the source)."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
               _SRC, "-o", _LIB + ".tmp", "-lpthread", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Space(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("d", ctypes.c_int32 * 3), ("dtype", ctypes.c_int32),
                ("mfma_coord", ctypes.c_int32), ("mode", ctypes.c_int32)]


class _Config(ctypes.Structure):
    _fields_ = [("f", (ctypes.c_int64 * MAXD) * 3), ("mfma", ctypes.c_int32),
                ("legit", ctypes.c_int32)]


class _GbfsResult(ctypes.Structure):
    _fields_ = [("best", _Config), ("best_cost", ctypes.c_double),
                ("timed", ctypes.c_int64), ("popped", ctypes.c_int64)]


class _Na2cParams(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("B", ctypes.c_int32), ("H", ctypes.c_int32),
                ("mem", ctypes.c_int32), ("max_walks", ctypes.c_int32),
                ("reward", ctypes.c_int32), ("eps_halving", ctypes.c_int32),
                ("eps", ctypes.c_double), ("gamma", ctypes.c_double), ("lr", ctypes.c_double),
                ("r_clip", ctypes.c_double)]


class _Na2cTransition(ctypes.Structure):
    _fields_ = [("s", ctypes.c_uint64), ("s2", ctypes.c_uint64), ("a", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("r", ctypes.c_double)]


# N-A2C settings: T = 3 steps per walk (§5) and the reward r = 1/cost(s')
# of §4.1 (reward=0); the rest are readings. reward=1 (clipped log ratio) and
# eps_halving=1 are variants.
NA2C_DEFAULTS = dict(T=3, B=8, H=32, mem=256, max_walks=64, reward=0, eps_halving=0, eps=0.8,
                     gamma=0.9, lr=0.01, r_clip=5.0)


_COST_FN = ctypes.CFUNCTYPE(ctypes.c_double, ctypes.POINTER(_Config), ctypes.c_uint64,
                            ctypes.c_void_p)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        p, i64, u64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64
        L.oracle_gemm.argtypes = [i64, i64, i64, p, p, ctypes.c_int, p, ctypes.c_int]
        L.oracle_gemm_entries.argtypes = [i64, i64, i64, p, p, ctypes.c_int, i64, p, p, p]
        L.oracle_widen.argtypes = [p, ctypes.c_int, i64, p]
        L.or_dim_tuples.argtypes = [i64, ctypes.c_int, p, i64]
        L.or_dim_tuples.restype = i64
        SP, CF = ctypes.POINTER(_Space), ctypes.POINTER(_Config)
        L.or_space_size.argtypes = [SP, ctypes.POINTER(u64)]
        L.or_rank.argtypes = [SP, CF, ctypes.POINTER(u64)]
        L.or_unrank.argtypes = [SP, u64, CF]
        L.or_member.argtypes = [SP, CF]
        L.or_legit.argtypes = [SP, CF]
        L.or_enumerate.argtypes = [SP, u64, u64, CF]
        L.or_neighbours.argtypes = [SP, CF, CF, ctypes.c_int]
        L.or_splitmix64_next.argtypes = [ctypes.POINTER(u64)]
        L.or_splitmix64_next.restype = u64
        L.or_gbfs.argtypes = [SP, CF, ctypes.c_int, i64, u64, _COST_FN, p,
                              ctypes.POINTER(_GbfsResult), p, p, i64]
        L.or_random_search.argtypes = [SP, i64, u64, _COST_FN, p, ctypes.POINTER(_GbfsResult),
                                       p, p, i64]
        NP = ctypes.POINTER(_Na2cParams)
        L.or_na2c.argtypes = [SP, CF, NP, i64, u64, _COST_FN, p, ctypes.POINTER(_GbfsResult),
                              p, p, i64, p, i64, ctypes.POINTER(i64)]
        L.or_na2c_train.argtypes = [SP, NP, CF, p, p, CF, i64, p, p]
        L.or_na2c_probe.argtypes = [SP, NP, u64, CF, ctypes.c_int, p, p, p, p, p, p,
                                    ctypes.POINTER(i64), ctypes.POINTER(i64)]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(dtype) -> int:
    return {"f32": F32, "bf16": BF16, F32: F32, BF16: BF16}[dtype]


# ---------------------------------------------------------------------------
# GEMM
# ---------------------------------------------------------------------------

def gemm(A_bytes: np.ndarray, B_bytes: np.ndarray, M: int, N: int, K: int, dtype,
         nthreads: int | None = None) -> np.ndarray:
    """fp64 C (M×N) from the raw row-major input bytes (see workloads.raw_bytes)."""
    dt = _dtype_code(dtype)
    esz = 4 if dt == F32 else 2
    A_bytes = np.ascontiguousarray(A_bytes, dtype=np.uint8)
    B_bytes = np.ascontiguousarray(B_bytes, dtype=np.uint8)
    assert A_bytes.size == M * K * esz and B_bytes.size == K * N * esz
    C = np.empty((M, N), dtype=np.float64)
    nt = nthreads or os.cpu_count() or 1
    rc = lib().oracle_gemm(M, N, K, _ptr(A_bytes), _ptr(B_bytes), dt, _ptr(C), nt)
    if rc:
        raise MemoryError("oracle_gemm failed")
    return C


def gemm_tn(W_bytes: np.ndarray, B_bytes: np.ndarray, M: int, N: int, K: int, dtype,
            nthreads: int | None = None) -> np.ndarray:
    """The perceptron product of §5, Y = WᵀX with W (K×M) and X (K×N) given as
    raw row-major bytes: A = Wᵀ element by element (a byte-exact transpose),
    then the plain product."""
    esz = 4 if _dtype_code(dtype) == F32 else 2
    W = np.ascontiguousarray(W_bytes, dtype=np.uint8).reshape(K, M, esz)
    A_bytes = np.ascontiguousarray(W.transpose(1, 0, 2)).reshape(-1)
    return gemm(A_bytes, B_bytes, M, N, K, dtype, nthreads)


def gemm_entries(A_bytes, B_bytes, M, N, K, dtype, rows, cols) -> np.ndarray:
    dt = _dtype_code(dtype)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    out = np.empty(rows.size, dtype=np.float64)
    A_bytes = np.ascontiguousarray(A_bytes, dtype=np.uint8)
    B_bytes = np.ascontiguousarray(B_bytes, dtype=np.uint8)
    rc = lib().oracle_gemm_entries(M, N, K, _ptr(A_bytes), _ptr(B_bytes), dt, rows.size,
                                   _ptr(rows), _ptr(cols), _ptr(out))
    if rc:
        raise IndexError("entry out of range")
    return out


def widen(raw: np.ndarray, dtype) -> np.ndarray:
    dt = _dtype_code(dtype)
    raw = np.ascontiguousarray(raw, dtype=np.uint8)
    n = raw.size // (4 if dt == F32 else 2)
    out = np.empty(n, dtype=np.float64)
    lib().oracle_widen(_ptr(raw), dt, n, _ptr(out))
    return out


# ---------------------------------------------------------------------------
# Configuration space
# ---------------------------------------------------------------------------

def dim_tuples(D: int, d: int) -> list:
    L = lib()
    n = L.or_dim_tuples(D, d, None, 0)
    buf = np.zeros(max(n * d, 1), dtype=np.int64)
    L.or_dim_tuples(D, d, _ptr(buf), n)
    return [tuple(int(v) for v in buf[i * d:(i + 1) * d]) for i in range(n)]


class Space:
    """A configuration space; configs are tuples (m_levels, k_levels, n_levels, mfma)."""

    def __init__(self, M, N, K, d=(4, 4, 4), dtype="f32", mfma_coord=False,
                 mode=ADJACENT):
        self.M, self.N, self.K = int(M), int(N), int(K)
        self.d = tuple(int(x) for x in d)
        self.dtype = _dtype_code(dtype)
        self.mfma_coord = bool(mfma_coord)
        self.mode = int(mode)
        s = _Space()
        s.M, s.N, s.K = self.M, self.N, self.K
        for i in range(3):
            s.d[i] = self.d[i]
        s.dtype, s.mfma_coord, s.mode = self.dtype, int(self.mfma_coord), self.mode
        self._s = s

    # -- conversions --
    def _to_c(self, cfg) -> _Config:
        c = _Config()
        for x in range(3):
            lv = cfg[x]
            assert len(lv) == self.d[x], (cfg, self.d)
            for i, v in enumerate(lv):
                c.f[x][i] = int(v)
        c.mfma = int(cfg[3]) if len(cfg) > 3 else 0
        return c

    def _from_c(self, c: _Config):
        return (tuple(int(c.f[0][i]) for i in range(self.d[0])),
                tuple(int(c.f[1][i]) for i in range(self.d[1])),
                tuple(int(c.f[2][i]) for i in range(self.d[2])),
                int(c.mfma))

    # -- queries --
    def size(self) -> int:
        out = ctypes.c_uint64()
        assert lib().or_space_size(ctypes.byref(self._s), ctypes.byref(out)) == 0
        return int(out.value)

    def rank(self, cfg) -> int:
        out = ctypes.c_uint64()
        rc = lib().or_rank(ctypes.byref(self._s), ctypes.byref(self._to_c(cfg)),
                           ctypes.byref(out))
        if rc:
            raise ValueError(f"not a member: {cfg}")
        return int(out.value)

    def unrank(self, r: int):
        c = _Config()
        if lib().or_unrank(ctypes.byref(self._s), int(r), ctypes.byref(c)):
            raise IndexError(r)
        return self._from_c(c)

    def member(self, cfg) -> bool:
        return bool(lib().or_member(ctypes.byref(self._s), ctypes.byref(self._to_c(cfg))))

    def legit(self, cfg) -> bool:
        return bool(lib().or_legit(ctypes.byref(self._s), ctypes.byref(self._to_c(cfg))))

    def enumerate(self, start: int = 0, count: int | None = None):
        """List of (cfg, J) for ranks [start, start+count)."""
        if count is None:
            count = self.size() - start
        arr = (_Config * max(count, 1))()
        rc = lib().or_enumerate(ctypes.byref(self._s), start, count, arr)
        assert rc == 0
        return [(self._from_c(arr[i]), bool(arr[i].legit)) for i in range(count)]

    def enumerate_raw(self, start: int, count: int) -> np.ndarray:
        """Raw config records as a numpy structured view (for bulk comparisons)."""
        arr = (_Config * max(count, 1))()
        assert lib().or_enumerate(ctypes.byref(self._s), start, count, arr) == 0
        return np.frombuffer(arr, dtype=np.uint8).reshape(max(count, 1), ctypes.sizeof(_Config))[:count]

    def neighbours(self, cfg):
        """g(s) in ascending rank: list of (cfg, J)."""
        out = (_Config * (3 * MAXD * MAXD + 1))()
        n = lib().or_neighbours(ctypes.byref(self._s), ctypes.byref(self._to_c(cfg)), out,
                                3 * MAXD * MAXD + 1)
        if n < 0:
            raise ValueError(f"not a member: {cfg}")
        return [(self._from_c(out[i]), bool(out[i].legit)) for i in range(n)]

    def paper_s0(self):
        """The paper's start state: [D,1,…,1] per dimension (§5), MFMA 16."""
        return (tuple([self.M] + [1] * (self.d[0] - 1)),
                tuple([self.K] + [1] * (self.d[1] - 1)),
                tuple([self.N] + [1] * (self.d[2] - 1)),
                16 if self.mfma_coord else 0)


def splitmix64_stream(seed: int, n: int) -> list:
    st = ctypes.c_uint64(seed)
    return [int(lib().or_splitmix64_next(ctypes.byref(st))) for _ in range(n)]


def gbfs(space: Space, s0, rho: int, budget: int, seed: int, cost_fn):
    """Run Alg.1. ``cost_fn(cfg, rank) -> float``. Returns a dict with the best
    configuration, its cost, the count timed, the pops, and the timing log."""
    log_r = np.zeros(budget, dtype=np.uint64)
    log_c = np.zeros(budget, dtype=np.float64)

    def _cb(cptr, rank, _ctx):
        return float(cost_fn(space._from_c(cptr.contents), int(rank)))

    cb = _COST_FN(_cb)
    res = _GbfsResult()
    rc = lib().or_gbfs(ctypes.byref(space._s), ctypes.byref(space._to_c(s0)), int(rho),
                       int(budget), int(seed), cb, None, ctypes.byref(res), _ptr(log_r),
                       _ptr(log_c), budget)
    if rc:
        raise ValueError("or_gbfs: bad argument (illegitimate s0, budget < 1 or rho < 1)")
    n = int(res.timed)
    return {"best": space._from_c(res.best), "best_cost": float(res.best_cost),
            "timed": n, "popped": int(res.popped),
            "log_ranks": [int(v) for v in log_r[:n]], "log_costs": [float(v) for v in log_c[:n]]}


def random_search(space: Space, budget: int, seed: int, cost_fn):
    """Equal-budget random search (§5 baseline): uniform draws by SplitMix64,
    illegitimate and repeated draws skipped. Same result dict as gbfs();
    ``popped`` counts the draws."""
    log_r = np.zeros(budget, dtype=np.uint64)
    log_c = np.zeros(budget, dtype=np.float64)

    def _cb(cptr, rank, _ctx):
        return float(cost_fn(space._from_c(cptr.contents), int(rank)))

    cb = _COST_FN(_cb)
    res = _GbfsResult()
    rc = lib().or_random_search(ctypes.byref(space._s), int(budget), int(seed), cb, None,
                                ctypes.byref(res), _ptr(log_r), _ptr(log_c), budget)
    if rc:
        raise ValueError("or_random_search: bad argument (budget < 1)")
    n = int(res.timed)
    return {"best": space._from_c(res.best), "best_cost": float(res.best_cost),
            "timed": n, "popped": int(res.popped),
            "log_ranks": [int(v) for v in log_r[:n]], "log_costs": [float(v) for v in log_c[:n]]}


def _na2c_params(params=None) -> _Na2cParams:
    v = dict(NA2C_DEFAULTS)
    v.update(params or {})
    return _Na2cParams(**v)


def na2c(space: Space, s0, budget: int, seed: int, cost_fn, params=None, trace_cap: int = 0):
    """N-A2C (§4.3, Alg.2) with the oracle's readings; ``params`` overrides
    NA2C_DEFAULTS. Same result dict as gbfs(); ``popped`` counts episodes.
    With trace_cap > 0, ``transitions`` lists the first trace_cap transitions
    stored into the memory as (rank s, action, r, rank s'), and
    ``n_transitions`` their total count."""
    log_r = np.zeros(budget, dtype=np.uint64)
    log_c = np.zeros(budget, dtype=np.float64)

    def _cb(cptr, rank, _ctx):
        return float(cost_fn(space._from_c(cptr.contents), int(rank)))

    cb = _COST_FN(_cb)
    res = _GbfsResult()
    prm = _na2c_params(params)
    tr = (_Na2cTransition * max(1, trace_cap))()
    n_tr = ctypes.c_int64(0)
    rc = lib().or_na2c(ctypes.byref(space._s), ctypes.byref(space._to_c(s0)), ctypes.byref(prm),
                       int(budget), int(seed), cb, None, ctypes.byref(res), _ptr(log_r),
                       _ptr(log_c), budget, ctypes.cast(tr, ctypes.c_void_p) if trace_cap else None,
                       int(trace_cap), ctypes.byref(n_tr))
    if rc:
        raise ValueError("or_na2c: bad argument")
    n = int(res.timed)
    out = {"best": space._from_c(res.best), "best_cost": float(res.best_cost),
           "timed": n, "popped": int(res.popped),
           "log_ranks": [int(v) for v in log_r[:n]], "log_costs": [float(v) for v in log_c[:n]]}
    if trace_cap:
        k = min(trace_cap, n_tr.value)
        out["transitions"] = [(int(t.s), int(t.a), float(t.r), int(t.s2)) for t in tr[:k]]
        out["n_transitions"] = n_tr.value
    return out


def na2c_train(space: Space, transitions, actor, critic, params=None):
    """The oracle's N-A2C training step applied to caller-given flattened
    parameters (the layout of na2c_probe) for transitions
    [(s, a, r, s'), …] in order; returns the updated (actor, critic)."""
    prm = _na2c_params(params)
    n = len(transitions)
    S = (_Config * max(1, n))(*[space._to_c(t[0]) for t in transitions])
    S2 = (_Config * max(1, n))(*[space._to_c(t[3]) for t in transitions])
    a = np.array([t[1] for t in transitions] or [0], dtype=np.int32)
    r = np.array([t[2] for t in transitions] or [0.0], dtype=np.float64)
    th_a = np.array(actor, dtype=np.float64)
    th_c = np.array(critic, dtype=np.float64)
    rc = lib().or_na2c_train(ctypes.byref(space._s), ctypes.byref(prm), S, _ptr(a), _ptr(r), S2,
                             n, _ptr(th_a), _ptr(th_c))
    if rc:
        raise ValueError("or_na2c_train: bad argument")
    return th_a, th_c


def na2c_probe(space: Space, cfg, a: int, seed: int = 0, params=None, actor=None, critic=None):
    """π(·|s), V(s), ∇θ log π(a|s) and ∇θ V(s) of the N-A2C networks, at the
    initial weights of ``seed`` or at the given flattened parameters."""
    prm = _na2c_params(params)
    na, nc = ctypes.c_int64(), ctypes.c_int64()
    assert lib().or_na2c_probe(ctypes.byref(space._s), ctypes.byref(prm), int(seed), None, 0,
                               None, None, None, None, None, None, ctypes.byref(na),
                               ctypes.byref(nc)) == 0
    A = sum(d * (d - 1) if space.mode == ANY_PAIR else 2 * (d - 1) for d in space.d)
    A += 1 if space.mfma_coord else 0
    pi = np.zeros(64)
    v = np.zeros(1)
    ga, gc = np.zeros(na.value), np.zeros(nc.value)
    ap = None if actor is None else np.ascontiguousarray(actor, dtype=np.float64)
    cp = None if critic is None else np.ascontiguousarray(critic, dtype=np.float64)
    rc = lib().or_na2c_probe(ctypes.byref(space._s), ctypes.byref(prm), int(seed),
                             ctypes.byref(space._to_c(cfg)), int(a),
                             None if ap is None else _ptr(ap), None if cp is None else _ptr(cp),
                             _ptr(pi), _ptr(v), _ptr(ga), _ptr(gc), None, None)
    assert rc == 0
    return {"pi": pi[:A], "v": float(v[0]), "g_actor": ga, "g_critic": gc,
            "n_actor": na.value, "n_critic": nc.value}
