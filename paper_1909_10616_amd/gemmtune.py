"""ctypes binding of libgemmtune (include/gemmtune.h), same names as the C ABI.

Argument marshalling only: every step runs in the library. PyTorch supplies
device memory (``tensor.data_ptr()``) and the stream
(``torch.cuda.current_stream().cuda_stream``). Configurations are tuples
``(m_levels, k_levels, n_levels, mfma)``, dimension order m, k, n.

There is no fallback: if the library is not built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import math
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "libgemmtune.so")
MAXD = 4

F32, BF16 = 0, 1
A_KMAJOR = 16  # dtype flag: A passed as its K×M transpose W, C = WᵀB
ADJACENT, ANY_PAIR = 0, 1
STATUS = {0: "ok", 1: "early-abort", 2: "launch-failure", 3: "mismatch"}
STOP = {0: "budget", 1: "queue-empty", 2: "time-limit", 3: "draws-exhausted"}


class GemmTuneError(RuntimeError):
    pass


class gt_space(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("d_m", ctypes.c_int32), ("d_k", ctypes.c_int32), ("d_n", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("mfma_coord", ctypes.c_int32),
                ("neighbour_mode", ctypes.c_int32)]


class gt_config(ctypes.Structure):
    _fields_ = [("d_m", ctypes.c_int32), ("d_k", ctypes.c_int32), ("d_n", ctypes.c_int32),
                ("mfma", ctypes.c_int32),
                ("m", ctypes.c_int64 * MAXD), ("k", ctypes.c_int64 * MAXD),
                ("n", ctypes.c_int64 * MAXD),
                ("legit", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class gt_kernel_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("I", "IK", "TM", "TN", "fast", "dl", "ring", "waves", "BM", "BN", "BK", "dbuf",
                 "acc_regs", "lds_bytes")] + [("grid_x", ctypes.c_int64), ("grid_y", ctypes.c_int64)]


class gt_log_entry(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_uint64), ("cost_ms", ctypes.c_double),
                ("first_ms", ctypes.c_double), ("rel_err", ctypes.c_double),
                ("status", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("median_ms", ctypes.c_double), ("min_ms", ctypes.c_double),
                ("stdev_ms", ctypes.c_double)]


gt_cost_fn = ctypes.CFUNCTYPE(ctypes.c_double, ctypes.POINTER(gt_config), ctypes.c_uint64,
                              ctypes.c_void_p)


class gt_tune_opts(ctypes.Structure):
    _fields_ = [("s0", ctypes.POINTER(gt_config)), ("rho", ctypes.c_int32),
                ("runs", ctypes.c_int32), ("warmup", ctypes.c_int32), ("check", ctypes.c_int32),
                ("budget", ctypes.c_int64), ("t_max_s", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("max_run_ms", ctypes.c_double),
                ("abort_factor", ctypes.c_double),
                ("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("C", ctypes.c_void_p),
                ("c_ref", ctypes.c_void_p), ("stream", ctypes.c_void_p),
                ("log", ctypes.POINTER(gt_log_entry)), ("log_cap", ctypes.c_int64),
                ("progress_s", ctypes.c_double), ("trace_fd", ctypes.c_int32),
                ("reserved2", ctypes.c_int32)]


class gt_na2c_params(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("B", ctypes.c_int32), ("H", ctypes.c_int32),
                ("mem", ctypes.c_int32), ("max_walks", ctypes.c_int32),
                ("reward", ctypes.c_int32), ("eps_halving", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("eps", ctypes.c_double),
                ("gamma", ctypes.c_double), ("lr", ctypes.c_double), ("r_clip", ctypes.c_double)]


class gt_tune_result(ctypes.Structure):
    _fields_ = [("best", gt_config), ("best_rank", ctypes.c_uint64),
                ("best_cost", ctypes.c_double), ("timed", ctypes.c_int64),
                ("popped", ctypes.c_int64), ("skipped_illegit", ctypes.c_int64),
                ("skipped_visited", ctypes.c_int64), ("failed", ctypes.c_int64),
                ("wall_s", ctypes.c_double), ("stop_reason", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("eval_s", ctypes.c_double),
                ("device_s", ctypes.c_double)]


EXPORTS = ("gt_space_size", "enumerate_configs", "config_rank", "config_unrank", "config_legit",
           "neighbours", "gemm_run", "gt_measure", "gt_reference_gemm", "gt_compare",
           "gt_lower", "gt_tune_opts_init", "tune_gbfs", "tune_random", "gt_na2c_params_init",
           "tune_na2c", "gt_shutdown", "gt_compare_noalloc", "gt_last_error")

_lib = None


def lib():
    """Load libgemmtune.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise GemmTuneError(f"{LIB_PATH} is missing: build it with "
                            "`python -c 'import __graft_entry__ as g; g.build()'`")
    # One HIP runtime per process: PyTorch ships its own copy and asks for it
    # by a name without the soname's version, so with the library loaded first
    # the loader would map the system runtime and PyTorch's side by side, and
    # the second would find no GPU. With PyTorch loaded first, the library's
    # libamdhip64.so.7 resolves to the copy already mapped.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, i64, u64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int
    SP, CF = ctypes.POINTER(gt_space), ctypes.POINTER(gt_config)
    L.gt_space_size.argtypes = [SP, ctypes.POINTER(u64)]
    L.enumerate_configs.argtypes = [SP, u64, CF, u64, ctypes.POINTER(u64)]
    L.config_rank.argtypes = [SP, CF, ctypes.POINTER(u64)]
    L.config_unrank.argtypes = [SP, u64, CF]
    L.config_legit.argtypes = [SP, CF, ctypes.POINTER(i32)]
    L.neighbours.argtypes = [SP, CF, CF, i32, ctypes.POINTER(i32)]
    L.gemm_run.argtypes = [CF, P, P, P, i64, i64, i64, i32, P]
    L.gt_measure.argtypes = [CF, P, P, P, i64, i64, i64, i32, P, i32, i32, ctypes.c_double,
                             ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                             ctypes.POINTER(i32)]
    L.gt_reference_gemm.argtypes = [P, P, P, i64, i64, i64, i32, P]
    L.gt_compare.argtypes = [P, P, i64, P, ctypes.POINTER(ctypes.c_double)]
    L.gt_lower.argtypes = [CF, i64, i64, i64, i32, ctypes.POINTER(gt_kernel_info)]
    L.gt_tune_opts_init.argtypes = [ctypes.POINTER(gt_tune_opts)]
    L.tune_gbfs.argtypes = [SP, ctypes.POINTER(gt_tune_opts), gt_cost_fn, P,
                            ctypes.POINTER(gt_tune_result)]
    L.tune_random.argtypes = [SP, ctypes.POINTER(gt_tune_opts), gt_cost_fn, P,
                              ctypes.POINTER(gt_tune_result)]
    L.gt_na2c_params_init.argtypes = [ctypes.POINTER(gt_na2c_params)]
    L.tune_na2c.argtypes = [SP, ctypes.POINTER(gt_tune_opts), ctypes.POINTER(gt_na2c_params),
                            gt_cost_fn, P, ctypes.POINTER(gt_tune_result)]
    L.gt_shutdown.argtypes = []
    L.gt_compare_noalloc.argtypes = [P, P, i64, P, ctypes.POINTER(ctypes.c_double)]
    L.gt_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name != "gt_last_error":
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int, what: str):
    if rc != 0:
        msg = lib().gt_last_error().decode(errors="replace")
        raise GemmTuneError(f"{what} failed ({rc}): {msg}")


def dtype_code(dtype) -> int:
    if isinstance(dtype, int):
        return dtype
    s = str(dtype)
    if s in ("f32", "torch.float32", "float32"):
        return F32
    if s in ("bf16", "torch.bfloat16", "bfloat16"):
        return BF16
    raise ValueError(f"unsupported dtype {dtype!r}")


def to_c(cfg) -> gt_config:
    c = gt_config()
    m, k, n = cfg[0], cfg[1], cfg[2]
    c.d_m, c.d_k, c.d_n = len(m), len(k), len(n)
    for arr, vals in ((c.m, m), (c.k, k), (c.n, n)):
        for i, v in enumerate(vals):
            arr[i] = int(v)
    c.mfma = int(cfg[3]) if len(cfg) > 3 else 0
    return c


def from_c(c: gt_config):
    return (tuple(int(c.m[i]) for i in range(c.d_m)), tuple(int(c.k[i]) for i in range(c.d_k)),
            tuple(int(c.n[i]) for i in range(c.d_n)), int(c.mfma))


class Space:
    """Configuration space ξ (§3.3 Eq.1–4) with the C-ABI's queries.
    a_kmajor: the problem's A is passed as W = Aᵀ (K×M), C = WᵀB (§5)."""

    def __init__(self, M, N, K, d=(4, 4, 4), dtype="f32", mfma_coord=False,
                 mode=ADJACENT, a_kmajor=False):
        self.M, self.N, self.K = int(M), int(N), int(K)
        self.d = tuple(int(x) for x in d)
        self.dtype = dtype_code(dtype) | (A_KMAJOR if a_kmajor else 0)
        self.a_kmajor = bool(self.dtype & A_KMAJOR)
        self.mfma_coord = bool(mfma_coord)
        self.mode = int(mode)
        s = gt_space()
        s.M, s.N, s.K = self.M, self.N, self.K
        s.d_m, s.d_k, s.d_n = self.d
        s.dtype, s.mfma_coord, s.neighbour_mode = self.dtype, int(self.mfma_coord), self.mode
        self.c = s

    def size(self) -> int:
        out = ctypes.c_uint64()
        _check(lib().gt_space_size(ctypes.byref(self.c), ctypes.byref(out)), "gt_space_size")
        return int(out.value)

    def enumerate_raw(self, start: int, count: int):
        buf = (gt_config * max(count, 1))()
        n = ctypes.c_uint64()
        _check(lib().enumerate_configs(ctypes.byref(self.c), start, buf, count, ctypes.byref(n)),
               "enumerate_configs")
        return buf, int(n.value)

    def enumerate(self, start: int = 0, count: int | None = None):
        if count is None:
            count = self.size() - start
        buf, n = self.enumerate_raw(start, count)
        return [(from_c(buf[i]), bool(buf[i].legit)) for i in range(n)]

    def rank(self, cfg) -> int:
        out = ctypes.c_uint64()
        _check(lib().config_rank(ctypes.byref(self.c), ctypes.byref(to_c(cfg)), ctypes.byref(out)),
               "config_rank")
        return int(out.value)

    def unrank(self, r: int):
        c = gt_config()
        _check(lib().config_unrank(ctypes.byref(self.c), int(r), ctypes.byref(c)), "config_unrank")
        return from_c(c)

    def legit(self, cfg) -> bool:
        J = ctypes.c_int()
        _check(lib().config_legit(ctypes.byref(self.c), ctypes.byref(to_c(cfg)), ctypes.byref(J)),
               "config_legit")
        return bool(J.value)

    def neighbours(self, cfg):
        cap = 3 * MAXD * (MAXD - 1) + 1
        out = (gt_config * cap)()
        n = ctypes.c_int()
        _check(lib().neighbours(ctypes.byref(self.c), ctypes.byref(to_c(cfg)), out, cap,
                                ctypes.byref(n)), "neighbours")
        return [(from_c(out[i]), bool(out[i].legit)) for i in range(n.value)]

    def paper_s0(self):
        """[D,1,…,1] per dimension (§5's start state), MFMA 16."""
        return (tuple([self.M] + [1] * (self.d[0] - 1)), tuple([self.K] + [1] * (self.d[1] - 1)),
                tuple([self.N] + [1] * (self.d[2] - 1)), 16 if self.mfma_coord else 0)


def lower(cfg, M, N, K, dtype) -> dict:
    info = gt_kernel_info()
    _check(lib().gt_lower(ctypes.byref(to_c(cfg)), M, N, K, dtype_code(dtype), ctypes.byref(info)),
           "gt_lower")
    return {name: getattr(info, name) for name, _ in gt_kernel_info._fields_}


# ---------------------------------------------------------------------------
# GPU entry points (torch tensors for memory and stream)
# ---------------------------------------------------------------------------

def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _operands(A, B, C, a_kmajor=False):
    """(M, N, K, dtype code) of C = A·B, or of C = AᵀB when a_kmajor (A is
    then the K×M array W)."""
    import torch
    for t, name in ((A, "A"), (B, "B"), (C, "C")):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous GPU tensor")
    if A.dtype != B.dtype or A.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("A and B must both be float32 or both bfloat16")
    if C.dtype != torch.float32:
        raise ValueError("C must be float32")
    K, M = A.shape if a_kmajor else A.shape[::-1]
    K2, N = B.shape
    if K2 != K or tuple(C.shape) != (M, N):
        raise ValueError(f"shape mismatch A{tuple(A.shape)} B{tuple(B.shape)} C{tuple(C.shape)}")
    return M, N, K, dtype_code(A.dtype) | (A_KMAJOR if a_kmajor else 0)


def gemm_run(cfg, A, B, C, stream=None, a_kmajor=False):
    M, N, K, dt = _operands(A, B, C, a_kmajor)
    _check(lib().gemm_run(ctypes.byref(to_c(cfg)), A.data_ptr(), B.data_ptr(), C.data_ptr(), M, N,
                          K, dt, _stream(stream)), "gemm_run")
    return C


def gt_measure(cfg, A, B, C, warmup=1, runs=10, abort_ms=0.0, stream=None,
               a_kmajor=False) -> dict:
    M, N, K, dt = _operands(A, B, C, a_kmajor)
    mean, first, ab = ctypes.c_double(), ctypes.c_double(), ctypes.c_int()
    _check(lib().gt_measure(ctypes.byref(to_c(cfg)), A.data_ptr(), B.data_ptr(), C.data_ptr(), M,
                            N, K, dt, _stream(stream), warmup, runs, abort_ms, ctypes.byref(mean),
                            ctypes.byref(first), ctypes.byref(ab)), "gt_measure")
    return {"mean_ms": mean.value, "first_ms": first.value, "aborted": bool(ab.value)}


def gt_reference_gemm(A, B, C, stream=None, a_kmajor=False):
    M, N, K, dt = _operands(A, B, C, a_kmajor)
    _check(lib().gt_reference_gemm(A.data_ptr(), B.data_ptr(), C.data_ptr(), M, N, K, dt,
                                   _stream(stream)), "gt_reference_gemm")
    return C


def gt_compare_noalloc(C, R, stream=None) -> float:
    """gt_compare without any device allocation (the result words live in a
    static device array of the library)."""
    assert C.numel() == R.numel() and C.is_cuda and R.is_cuda
    rel = ctypes.c_double()
    _check(lib().gt_compare_noalloc(C.data_ptr(), R.data_ptr(), C.numel(), _stream(stream),
                                    ctypes.byref(rel)), "gt_compare_noalloc")
    return rel.value


def gt_shutdown():
    """Release the device memory the library keeps between calls."""
    _check(lib().gt_shutdown(), "gt_shutdown")


def gt_compare(C, R, stream=None) -> float:
    assert C.numel() == R.numel() and C.is_cuda and R.is_cuda
    rel = ctypes.c_double()
    _check(lib().gt_compare(C.data_ptr(), R.data_ptr(), C.numel(), _stream(stream),
                            ctypes.byref(rel)), "gt_compare")
    return rel.value


def _tune(entry, space: Space, budget: int, s0, rho, seed, runs, warmup, check, t_max_s,
          max_run_ms, abort_factor, A, B, C, c_ref, cost_fn, stream, progress_s=0.0,
          na2c=None, trace_fd=-1) -> dict:
    L = lib()
    o = gt_tune_opts()
    _check(L.gt_tune_opts_init(ctypes.byref(o)), "gt_tune_opts_init")
    s0c = to_c(s0) if s0 is not None else None
    if s0c is not None:
        o.s0 = ctypes.pointer(s0c)
    o.rho, o.runs, o.warmup, o.check = rho, runs, warmup, int(check)
    o.budget, o.t_max_s, o.seed = budget, t_max_s, seed
    o.max_run_ms, o.abort_factor = max_run_ms, abort_factor
    o.progress_s = progress_s
    o.trace_fd = int(trace_fd)
    log = (gt_log_entry * budget)()
    o.log = ctypes.cast(log, ctypes.POINTER(gt_log_entry))
    o.log_cap = budget
    cb = gt_cost_fn()  # NULL
    keep = None
    if cost_fn is not None:
        def _cb(cptr, rank, _ctx):
            return float(cost_fn(from_c(cptr.contents), int(rank)))
        keep = cb = gt_cost_fn(_cb)
    else:
        M, N, K, dt = _operands(A, B, C, space.a_kmajor)
        if (M, N, K, dt) != (space.M, space.N, space.K, space.dtype):
            raise ValueError("operands do not match the space")
        o.A, o.B, o.C = A.data_ptr(), B.data_ptr(), C.data_ptr()
        if c_ref is not None:
            import torch
            # the library writes M·N fp32 values through c_ref
            if not (c_ref.is_cuda and c_ref.device == C.device and c_ref.is_contiguous()
                    and c_ref.dtype == torch.float32 and c_ref.numel() == M * N):
                raise ValueError("c_ref must be a contiguous float32 tensor of M·N elements on "
                                 "C's device")
        o.c_ref = c_ref.data_ptr() if c_ref is not None else None
        o.stream = _stream(stream)
    res = gt_tune_result()
    if entry == "tune_na2c":
        prm = gt_na2c_params()
        _check(L.gt_na2c_params_init(ctypes.byref(prm)), "gt_na2c_params_init")
        for k, v in (na2c or {}).items():
            setattr(prm, k, v)
        rc = L.tune_na2c(ctypes.byref(space.c), ctypes.byref(o), ctypes.byref(prm), cb, None,
                         ctypes.byref(res))
    else:
        rc = getattr(L, entry)(ctypes.byref(space.c), ctypes.byref(o), cb, None, ctypes.byref(res))
    _check(rc, entry)
    del keep
    n = int(res.timed)
    entries = [{"rank": int(log[i].rank), "cost_ms": log[i].cost_ms, "first_ms": log[i].first_ms,
                "median_ms": log[i].median_ms, "min_ms": log[i].min_ms,
                "stdev_ms": log[i].stdev_ms, "rel_err": log[i].rel_err,
                "status": STATUS.get(log[i].status, str(log[i].status))}
               for i in range(min(n, budget))]
    return {"best": from_c(res.best), "best_rank": int(res.best_rank),
            "best_cost": res.best_cost, "timed": n, "popped": int(res.popped),
            "skipped_illegit": int(res.skipped_illegit),
            "skipped_visited": int(res.skipped_visited), "failed": int(res.failed),
            "wall_s": res.wall_s, "eval_s": res.eval_s, "device_s": res.device_s,
            "stop_reason": ("neighbourhood-exhausted" if entry == "tune_na2c" and res.stop_reason == 1
                            else STOP.get(res.stop_reason, "?")),
            "log": entries}


def tune_gbfs(space: Space, budget: int, s0=None, rho: int = 5, seed: int = 0, runs: int = 10,
              warmup: int = 1, check: bool = True, t_max_s: float = 0.0,
              max_run_ms: float = 250.0, abort_factor: float = 50.0, A=None, B=None, C=None,
              c_ref=None, cost_fn=None, stream=None, progress_s: float = 0.0,
              trace_fd: int = -1) -> dict:
    """Run G-BFS (Alg.1). With ``cost_fn(cfg, rank) -> float`` the costs are
    synthetic (no GPU); otherwise A, B, C are GPU tensors and every candidate
    is timed with ``gemm_run`` on the stream (A is W, K×M, when the space has
    a_kmajor). progress_s > 0: a progress line on stderr at most that often;
    trace_fd >= 0: each candidate is named on that file descriptor before it
    is launched."""
    return _tune("tune_gbfs", space, budget, s0, rho, seed, runs, warmup, check, t_max_s,
                 max_run_ms, abort_factor, A, B, C, c_ref, cost_fn, stream, progress_s,
                 trace_fd=trace_fd)


def tune_random(space: Space, budget: int, seed: int = 0, runs: int = 10, warmup: int = 1,
                check: bool = True, t_max_s: float = 0.0, max_run_ms: float = 250.0,
                abort_factor: float = 50.0, A=None, B=None, C=None, c_ref=None, cost_fn=None,
                stream=None, progress_s: float = 0.0, trace_fd: int = -1) -> dict:
    """Equal-budget random search (§5 baseline); same timing and result as
    tune_gbfs, ``popped`` counts the draws."""
    return _tune("tune_random", space, budget, None, 1, seed, runs, warmup, check, t_max_s,
                 max_run_ms, abort_factor, A, B, C, c_ref, cost_fn, stream, progress_s,
                 trace_fd=trace_fd)


def tune_na2c(space: Space, budget: int, s0=None, seed: int = 0, runs: int = 10,
              warmup: int = 1, check: bool = True, t_max_s: float = 0.0,
              max_run_ms: float = 250.0, abort_factor: float = 50.0, A=None, B=None, C=None,
              c_ref=None, cost_fn=None, stream=None, progress_s: float = 0.0,
              params=None, trace_fd: int = -1) -> dict:
    """N-A2C (§4.3, Alg.2); timing, log and result as tune_gbfs (``popped``
    counts episodes). ``params``: overrides of gt_na2c_params (T, B, H, mem,
    max_walks, reward, eps_halving, eps, gamma, lr, r_clip)."""
    return _tune("tune_na2c", space, budget, s0, 1, seed, runs, warmup, check, t_max_s,
                 max_run_ms, abort_factor, A, B, C, c_ref, cost_fn, stream, progress_s,
                 na2c=params, trace_fd=trace_fd)


def tflops(M, N, K, ms) -> float:
    """2·M·N·K floating-point operations per run (one multiply-add = 2 flops)."""
    return 2.0 * M * N * K / (ms * 1e-3) / 1e12 if ms > 0 and math.isfinite(ms) else 0.0


def report(M, N, K, dtype, ms, timed, space_size, peak_tflops) -> dict:
    """The figures a search is reported by (§5 reports the share of the space
    explored): TFLOP/s of the best configuration (2·M·N·K per run), its share
    of the dtype's dense MFMA peak in %, the configurations timed as a
    percentage of the whole space |ξ| (illegitimate states included), and the
    HBM rate at the algorithmic bytes — A and B read once, C (fp32) written
    once."""
    esz = 2 if dtype_code(dtype) & ~A_KMAJOR == BF16 else 4
    alg_bytes = (M * K + K * N) * esz + M * N * 4
    tf = tflops(M, N, K, ms)
    return {"tflops": tf, "pct_of_peak": 100.0 * tf / peak_tflops,
            "fraction_of_space_pct": 100.0 * timed / space_size,
            "algorithmic_bytes": alg_bytes,
            "hbm_gbs": alg_bytes / (ms * 1e-3) / 1e9 if ms > 0 and math.isfinite(ms) else 0.0}


def hand_start(M: int, N: int, K: int, d, mfma_coord: bool):
    """A hand-crafted start state (§4.2 allows one) with a 32-deep K stage
    and 2×2 wavefronts of 32-wide MFMA blocks: 128×128 workgroup tiles (2×2
    blocks per wavefront) where 128 divides M and N, else 64×64 tiles (one
    block per wavefront), for the level layout (4, 4, 4); 64×64 tiles for
    (3, 3, 3). From the 128×128 start G-BFS reached the 256×256×32 tile
    family on 4096×11008×4096 for each of three seeds, from the 64×64 start
    for two of three (one ended 20 % slower); at 4096³ both reach it."""
    if tuple(d) == (4, 4, 4):
        if M % 128 == 0 and N % 128 == 0:
            m, n = (M // 128, 2, 2, 32), (N // 128, 2, 2, 32)
        else:
            m = (M // 64, 2, 1, 32) if M >= 64 else (1, 1, 1, M)
            n = (N // 64, 2, 1, 32)
        k = (K // 32, 1, 2, 16)
        return (m, k, n, 32 if mfma_coord else 0)
    if tuple(d) == (3, 3, 3):
        return ((M // 64, 2, 32), (K // 32, 2, 16), (N // 64, 2, 32), 0)
    raise ValueError("no hand-crafted start for this level layout")


def fmt_cfg(c) -> str:
    return "m{}k{}n{}mfma{}".format(list(c[0]), list(c[1]), list(c[2]), c[3])
