// Lowering of a configuration to a kernel launch, the GEMM entry point, the
// cost measurement the search uses (§4.2 "test" a configuration on the
// hardware; §5: cost is the mean of 10 runs), and the reference/compare
// helpers.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "aux_kernels.h"
#include "gemm_kernel.hpp"
#include "internal.h"
#include "runtime.h"

namespace gt {

namespace {

int ilog2(int64_t v) {
  int e = 0;
  while ((int64_t{1} << e) < v) ++e;
  return e;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return GT_EHIP;
}

}  // namespace

int lower(const gt_config& c, int64_t M, int64_t N, int64_t K, int dtype, const void* A,
          const void* B, void* C, Lowered* out) {
  gt_space sp{};
  sp.M = M;
  sp.N = N;
  sp.K = K;
  sp.d_m = c.d_m;
  sp.d_k = c.d_k;
  sp.d_n = c.d_n;
  sp.dtype = dtype;
  sp.mfma_coord = c.mfma != 0 ? 1 : 0;
  sp.neighbour_mode = GT_ADJACENT;
  Space s;
  if (int rc = make_space(&sp, &s)) return rc;
  if (!is_member(s, c)) {
    set_error("configuration does not factor M, K, N (or bad MFMA value)");
    return GT_EDIMS;
  }
  if (!legit_of(s, c)) {
    set_error("configuration is not legitimate (J = 0)");
    return GT_EILLEGIT;
  }
  Levels& L = out->L;
  const int dt = s.dtype;          // without the layout flag
  const bool akm = s.a_kmajor;     // A given K-major (K×M)
  levels_of(c, dt, &L);
  const int vec = dt == GT_BF16 ? 8 : 4;
  const int G = 64 / L.I;
  const int64_t cpr = L.BK / vec;  // 16-byte chunks per LDS row
  const bool cpr_ok = L.BK % vec == 0 && (cpr == 2 || cpr == 4 || cpr == 8 || cpr == 16);
  // (a K-major A needs 16-byte m chunks, M % vec; its fast path is fp32 only)
  const bool fast = L.blkM % L.I == 0 && L.blkN % L.I == 0 && L.kBlk % L.IK == 0 &&
                    L.BK % (vec * G) == 0 && cpr_ok && L.BN % vec == 0 && K % vec == 0 &&
                    N % vec == 0 && L.W <= 8 && aligned16(A) && aligned16(B) &&
                    (!akm || (dt == GT_F32 && L.BM % vec == 0 && M % vec == 0));
  const int64_t stage_bytes = (L.BM * L.BK + L.BK * L.BN) * L.elem;
  const bool dbuf = L.kLoop >= 2 && 2 * stage_bytes <= kLdsMax;
  // bf16 fast path with direct global->LDS loads into a ring of ns stages:
  // whole 64-slot load instructions, an even split over the wavefronts, at
  // most dl_inst_cap(acc) instructions per wavefront and stage, 32-bit
  // element offsets
  const int64_t achunks = L.BM * L.BK / 8, bchunks = L.BK * L.BN / 8;
  const int64_t dl_inst = (achunks + bchunks) / 64;
  const int64_t ns = std::min<int64_t>(8, kLdsMax / std::max<int64_t>(stage_bytes, 1));
  const bool dl = fast && dt == GT_BF16 && !akm && achunks % (64 * L.W) == 0 &&
                  bchunks % (64 * L.W) == 0 && dl_inst / L.W <= dl_inst_cap(L.acc) && ns >= 2 &&
                  L.BM * K < (int64_t{1} << 31) && L.BK * N < (int64_t{1} << 31);

  KArgs& a = out->args;
  std::memset(&a, 0, sizeof(a));
  a.A = A;
  a.B = B;
  a.C = static_cast<float*>(C);
  a.M = M;
  a.N = N;
  a.K = K;
  a.gridM = static_cast<int32_t>(L.gridM);
  a.gridN = static_cast<int32_t>(L.gridN);
  a.wavesM = static_cast<int32_t>(L.wavesM);
  a.wavesN = static_cast<int32_t>(L.wavesN);
  a.blkM = static_cast<int32_t>(L.blkM);
  a.blkN = static_cast<int32_t>(L.blkN);
  a.lgTpbM = L.blkM >= L.I ? ilog2(L.blkM / L.I) : 0;
  a.lgTpbN = L.blkN >= L.I ? ilog2(L.blkN / L.I) : 0;
  a.kLoop = static_cast<int32_t>(L.kLoop);
  a.kSplit = static_cast<int32_t>(L.kSplit);
  a.kSub = static_cast<int32_t>(L.kSub);
  a.kBlk = static_cast<int32_t>(L.kBlk);
  a.BM = static_cast<int32_t>(L.BM);
  a.BN = static_cast<int32_t>(L.BN);
  a.BK = static_cast<int32_t>(L.BK);
  a.WM = static_cast<int32_t>(L.repM * L.blkM);
  a.WN = static_cast<int32_t>(L.repN * L.blkN);
  a.lgBK = ilog2(L.BK);
  a.lgBN = ilog2(L.BN);
  a.dbuf = dbuf ? 1 : 0;
  a.atomic = L.kSplit > 1 ? 1 : 0;
  a.remap = (L.gridM * L.gridN) % 8 == 0 ? 1 : 0;
  a.aVec = (akm ? (L.BM % vec == 0 && M % vec == 0) : (L.BK % vec == 0 && K % vec == 0)) &&
                   aligned16(A)
               ? vec
               : 1;
  a.aKM = akm ? 1 : 0;
  a.lgBM = ilog2(L.BM);
  a.bVec = (L.BN % vec == 0 && N % vec == 0 && aligned16(B)) ? vec : 1;
  a.dl = dl ? 1 : 0;
  a.ns = dl ? static_cast<int32_t>(ns) : 0;

  out->grid = dim3(static_cast<unsigned>(L.gridM * L.gridN), static_cast<unsigned>(L.kSplit), 1);
  out->block = dim3(static_cast<unsigned>(64 * L.W), 1, 1);
  out->lds = static_cast<size_t>(stage_bytes * (dl ? ns : (dbuf ? 2 : 1)));
  out->fast = fast;
  out->fn = find_gemm_kernel(dt, L.I, fast ? static_cast<int>(cpr) : 0,
                             static_cast<int>(L.TM), static_cast<int>(L.TN), fast && akm);
  if (!out->fn) {
    set_error("no kernel instantiation for this MFMA tile shape");
    return GT_ENOKERNEL;
  }
  return GT_OK;
}

int launch_lowered(const Lowered& lw, hipStream_t s) {
  if (lw.args.atomic) {
    hipError_t e = launch_fill_zero(lw.args.C, lw.args.M * lw.args.N, s);
    if (e != hipSuccess) return hip_fail(e, "clearing C for split-K");
  }
  hipError_t e = lw.fn(lw.args, lw.grid, lw.block, lw.lds, s);
  if (e != hipSuccess) return hip_fail(e, "GEMM launch");
  return GT_OK;
}

namespace {
std::mutex g_cmp_mu;
unsigned* g_cmp_buf[64] = {};  // per device, 2 words, kept until process exit
}  // namespace

int compare_into(const void* C, const void* R, int64_t n, unsigned* buf, hipStream_t s,
                 double* rel) {
  hipError_t e =
      launch_compare(static_cast<const float*>(C), static_cast<const float*>(R), n, buf, s);
  if (e != hipSuccess) return hip_fail(e, "compare launch");
  unsigned host[2];
  e = hipMemcpyAsync(host, buf, sizeof(host), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (compare result)");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize (compare)");
  float md, mr;
  std::memcpy(&md, &host[0], 4);
  std::memcpy(&mr, &host[1], 4);
  if (std::isnan(md))
    *rel = NAN;
  else if (mr == 0.0f)
    *rel = md == 0.0f ? 0.0 : INFINITY;
  else
    *rel = static_cast<double>(md) / static_cast<double>(mr);
  return GT_OK;
}

int compare_on_gpu(const void* C, const void* R, int64_t n, hipStream_t s, double* rel) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) {
    set_error("device index out of range");
    return GT_EINVAL;
  }
  // The device's 2-word result buffer is held from its clear to the copy
  // back: comparisons from several threads (any streams) take turns, and
  // gt_shutdown cannot free the buffer under one in flight.
  std::lock_guard<std::mutex> lk(g_cmp_mu);
  if (!g_cmp_buf[dev]) {
    e = hipMalloc(&g_cmp_buf[dev], 2 * sizeof(unsigned));
    if (e != hipSuccess) return hip_fail(e, "hipMalloc (compare result)");
  }
  return compare_into(C, R, n, g_cmp_buf[dev], s, rel);
}

namespace {
std::mutex g_time_mu[64];    // per device: one timing at a time
std::mutex g_time_mu_other;  // devices beyond 64, or none current
}  // namespace

int measure(const gt_config& c, const void* A, const void* B, void* C, int64_t M, int64_t N,
            int64_t K, int dtype, hipStream_t s, int warmup, int runs, double abort_ms,
            double* mean_ms, double* first_ms, int* aborted, RunStats* stats) {
  Lowered lw;
  if (int rc = lower(c, M, N, K, dtype, A, B, C, &lw)) return rc;
  // Timings on one device take turns (searches in several threads, gt_measure):
  // each holds the device from its first launch until its last has finished,
  // so concurrent callers do not inflate each other's costs.
  int tdev = -1;
  const bool tdev_ok = hipGetDevice(&tdev) == hipSuccess && tdev >= 0 && tdev < 64;
  std::lock_guard<std::mutex> timing(tdev_ok ? g_time_mu[tdev] : g_time_mu_other);
  if (warmup < 1) warmup = 1;
  if (runs < 1) runs = 1;
  // events: [0], [1] around the first warm-up launch; [2 + r] before timed
  // run r and [2 + runs] after the last, so each run has its own duration
  std::vector<hipEvent_t> ev(static_cast<size_t>(runs) + 3, nullptr);
  auto destroy = [&]() {
    for (auto& x : ev)
      if (x) (void)hipEventDestroy(x);
  };
  for (auto& x : ev) {
    hipError_t e = hipEventCreate(&x);
    if (e != hipSuccess) {
      x = nullptr;
      destroy();
      return hip_fail(e, "hipEventCreate");
    }
  }
  int rc = GT_OK;
  float first = 0.0f, total = 0.0f;
  *aborted = 0;
  hipError_t e;
  // first warm-up launch, timed on its own for the early-abort rule
  if ((e = hipEventRecord(ev[0], s)) != hipSuccess) {
    destroy();
    return hip_fail(e, "hipEventRecord");
  }
  if ((rc = launch_lowered(lw, s)) != GT_OK) {
    (void)hipStreamSynchronize(s);
    destroy();
    return rc;
  }
  if ((e = hipEventRecord(ev[1], s)) != hipSuccess || (e = hipEventSynchronize(ev[1])) != hipSuccess ||
      (e = hipEventElapsedTime(&first, ev[0], ev[1])) != hipSuccess) {
    (void)hipStreamSynchronize(s);
    destroy();
    return hip_fail(e, "warm-up run");
  }
  *first_ms = first;
  if (abort_ms > 0.0 && first > abort_ms) {
    *aborted = 1;
    *mean_ms = first;
    if (stats) *stats = RunStats{first, first, 0.0};
    destroy();
    return GT_OK;
  }
  for (int w = 1; w < warmup; ++w)
    if ((rc = launch_lowered(lw, s)) != GT_OK) {
      (void)hipStreamSynchronize(s);
      destroy();
      return rc;
    }
  if ((e = hipEventRecord(ev[2], s)) != hipSuccess) {
    (void)hipStreamSynchronize(s);
    destroy();
    return hip_fail(e, "hipEventRecord");
  }
  for (int r = 0; r < runs; ++r) {
    if ((rc = launch_lowered(lw, s)) != GT_OK) {
      (void)hipStreamSynchronize(s);
      destroy();
      return rc;
    }
    if ((e = hipEventRecord(ev[3 + r], s)) != hipSuccess) {
      (void)hipStreamSynchronize(s);
      destroy();
      return hip_fail(e, "hipEventRecord");
    }
  }
  if ((e = hipEventSynchronize(ev[2 + runs])) != hipSuccess ||
      (e = hipEventElapsedTime(&total, ev[2], ev[2 + runs])) != hipSuccess) {
    destroy();
    return hip_fail(e, "timed runs");
  }
  *mean_ms = static_cast<double>(total) / runs;
  if (stats) {
    std::vector<double> d(static_cast<size_t>(runs));
    for (int r = 0; r < runs; ++r) {
      float ms = 0.0f;
      if ((e = hipEventElapsedTime(&ms, ev[2 + r], ev[3 + r])) != hipSuccess) {
        destroy();
        return hip_fail(e, "hipEventElapsedTime");
      }
      d[r] = ms;
    }
    double var = 0.0;
    for (double x : d) var += (x - *mean_ms) * (x - *mean_ms);
    std::sort(d.begin(), d.end());
    stats->median_ms = runs % 2 ? d[runs / 2] : 0.5 * (d[runs / 2 - 1] + d[runs / 2]);
    stats->min_ms = d[0];
    stats->stdev_ms = runs > 1 ? std::sqrt(var / (runs - 1)) : 0.0;
  }
  destroy();
  return GT_OK;
}

}  // namespace gt

extern "C" {

int gemm_run(const gt_config* cfg, const void* A, const void* B, void* C, int64_t M, int64_t N,
             int64_t K, int dtype, void* stream) {
  if (!cfg || !A || !B || !C) {
    gt::set_error("gemm_run: null argument");
    return GT_EINVAL;
  }
  gt::Lowered lw;
  if (int rc = gt::lower(*cfg, M, N, K, dtype, A, B, C, &lw)) return rc;
  return gt::launch_lowered(lw, static_cast<hipStream_t>(stream));
}

int gt_measure(const gt_config* cfg, const void* A, const void* B, void* C, int64_t M, int64_t N,
               int64_t K, int dtype, void* stream, int warmup, int runs, double abort_ms,
               double* mean_ms, double* first_ms, int* aborted) {
  if (!cfg || !A || !B || !C || !mean_ms || !first_ms || !aborted) {
    gt::set_error("gt_measure: null argument");
    return GT_EINVAL;
  }
  return gt::measure(*cfg, A, B, C, M, N, K, dtype, static_cast<hipStream_t>(stream), warmup, runs,
                     abort_ms, mean_ms, first_ms, aborted, nullptr);
}

int gt_reference_gemm(const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
                      int dtype, void* stream) {
  const int base = dtype & ~GT_A_KMAJOR;
  if (!A || !B || !C || M < 1 || N < 1 || K < 1 || (base != GT_F32 && base != GT_BF16)) {
    gt::set_error("gt_reference_gemm: bad argument");
    return GT_EINVAL;
  }
  hipError_t e = gt::launch_reference(A, B, static_cast<float*>(C), M, N, K, dtype,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    gt::set_error(std::string("reference launch: ") + hipGetErrorString(e));
    return GT_EHIP;
  }
  return GT_OK;
}

int gt_compare(const void* C, const void* R, int64_t n, void* stream, double* rel) {
  if (!C || !R || !rel || n < 1) {
    gt::set_error("gt_compare: bad argument");
    return GT_EINVAL;
  }
  return gt::compare_on_gpu(C, R, n, static_cast<hipStream_t>(stream), rel);
}

int gt_shutdown(void) {
  std::lock_guard<std::mutex> lk(gt::g_cmp_mu);
  int cur = -1;
  const bool have_cur = hipGetDevice(&cur) == hipSuccess;
  int rc = GT_OK;
  for (int d = 0; d < 64; ++d) {
    if (!gt::g_cmp_buf[d]) continue;
    hipError_t e = hipSetDevice(d);
    if (e == hipSuccess) e = hipFree(gt::g_cmp_buf[d]);
    if (e != hipSuccess && rc == GT_OK) rc = gt::hip_fail(e, "gt_shutdown: hipFree (compare result)");
    gt::g_cmp_buf[d] = nullptr;
  }
  if (have_cur) (void)hipSetDevice(cur);
  return rc;
}

int gt_lower(const gt_config* cfg, int64_t M, int64_t N, int64_t K, int dtype,
             gt_kernel_info* info) {
  if (!cfg || !info) {
    gt::set_error("gt_lower: null argument");
    return GT_EINVAL;
  }
  // alignment-independent view: assume 16-byte aligned operands
  gt::Lowered lw;
  static const uint4 dummy[1] = {};
  if (int rc = gt::lower(*cfg, M, N, K, dtype, dummy, dummy, nullptr, &lw)) return rc;
  info->I = lw.L.I;
  info->IK = lw.L.IK;
  info->TM = static_cast<int32_t>(lw.L.TM);
  info->TN = static_cast<int32_t>(lw.L.TN);
  info->fast = lw.fast ? 1 : 0;
  info->dl = lw.args.dl;
  info->ring = lw.args.ns;
  info->waves = static_cast<int32_t>(lw.L.W);
  info->BM = lw.args.BM;
  info->BN = lw.args.BN;
  info->BK = lw.args.BK;
  info->dbuf = lw.args.dbuf;
  info->acc_regs = static_cast<int32_t>(lw.L.acc);
  info->lds_bytes = static_cast<int32_t>(lw.lds);
  info->grid_x = lw.grid.x;
  info->grid_y = lw.grid.y;
  return GT_OK;
}

}  // extern "C"
