// Greedy Best-First Search over the configuration space (§4.2, Alg.1), and
// the equal-budget random search the paper's tuners are measured against
// (§5).
//
// G-BFS: the queue is ordered by increasing (cost, rank); S_v is a hash set
// of ranks. Each pop takes ρ neighbours of g(s) by a partial Fisher–Yates
// shuffle driven by SplitMix64 (Steele, Lea & Flood 2014), then times every
// pick that is legitimate and unvisited. A configuration counts toward the
// budget when it is timed; a failed or mismatching run costs +inf, is
// counted and visited, and is never pushed.
//
// Random search: ranks drawn uniformly (SplitMix64 mod |ξ|), illegitimate
// and repeated draws skipped without cost, at most 64·budget + 1024 draws.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <queue>
#include <string>
#include <unordered_set>
#include <utility>
#include <vector>

#include "internal.h"
#include "runtime.h"

namespace gt {
namespace {

uint64_t splitmix64(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct GpuCtx {
  const gt_tune_opts* o;
  int64_t M, N, K;
  int dtype;
  void* c_ref;
  double tol;
  hipStream_t s;
  hipError_t fatal = hipSuccess;  // device error that outlives the failed call
};

std::string describe(const gt_config& c) {
  std::string r = "((";
  auto tup = [&r](const int64_t* v, int d) {
    for (int i = 0; i < d; ++i) r += (i ? "," : "") + std::to_string(v[i]);
  };
  tup(c.m, c.d_m);
  r += "),(";
  tup(c.k, c.d_k);
  r += "),(";
  tup(c.n, c.d_n);
  r += ")," + std::to_string(c.mfma) + ")";
  return r;
}

// Times one configuration on the GPU; fills the log record; returns the cost.
double gpu_cost(GpuCtx& g, const gt_config& c, double cost_min, gt_log_entry* rec) {
  double abort_ms = g.o->max_run_ms;
  if (g.o->abort_factor > 0.0 && std::isfinite(cost_min))
    abort_ms = std::min(abort_ms > 0.0 ? abort_ms : INFINITY, g.o->abort_factor * cost_min);
  double mean = 0.0, first = 0.0;
  int aborted = 0;
  const int rc = measure(c, g.o->A, g.o->B, g.o->C, g.M, g.N, g.K, g.dtype, g.s, g.o->warmup,
                         g.o->runs, abort_ms, &mean, &first, &aborted);
  rec->first_ms = first;
  rec->rel_err = NAN;
  if (rc != GT_OK) {
    // A failed launch (no kernel, bad shape) leaves the device usable; a
    // fault in a kernel does not, and every later call would fail too.
    const hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) g.fatal = e;
    rec->status = 2;
    rec->cost_ms = INFINITY;
    return INFINITY;
  }
  if (g.o->check) {
    double rel = NAN;
    if (compare_on_gpu(g.o->C, g.c_ref, g.M * g.N, g.s, &rel) != GT_OK) {
      const hipError_t e = hipDeviceSynchronize();
      if (e != hipSuccess) g.fatal = e;
    }
    if (g.fatal != hipSuccess || !(rel <= g.tol)) {
      rec->status = 3;
      rec->rel_err = rel;
      rec->cost_ms = INFINITY;
      return INFINITY;
    }
    rec->rel_err = rel;
  }
  rec->status = aborted ? 1 : 0;
  rec->cost_ms = mean;
  return mean;
}

}  // namespace
}  // namespace gt

extern "C" {

int gt_tune_opts_init(gt_tune_opts* o) {
  if (!o) {
    gt::set_error("gt_tune_opts_init: null");
    return GT_EINVAL;
  }
  std::memset(o, 0, sizeof(*o));
  o->rho = 5;
  o->runs = 10;
  o->warmup = 1;
  o->check = 1;
  o->budget = 1000;
  o->max_run_ms = 250.0;
  o->abort_factor = 50.0;
  return GT_OK;
}

}  // extern "C"

namespace gt {
namespace {

// What both searches share: the space, the timing (callback or GPU, with the
// reference product computed once), the log and the result counters.
struct Tuner {
  Space s;
  const gt_tune_opts* o = nullptr;
  gt_cost_fn cost = nullptr;
  void* ctx = nullptr;
  gt_tune_result* out = nullptr;
  GpuCtx g{};
  void* owned_ref = nullptr;
  double cost_min = INFINITY;
  double last_progress = 0.0;
  const char* who = "";
  std::chrono::steady_clock::time_point t0 = std::chrono::steady_clock::now();

  ~Tuner() {
    if (owned_ref) (void)hipFree(owned_ref);
  }

  int init(const gt_space* sp, const gt_tune_opts* opts, gt_cost_fn cb, void* cb_ctx,
           gt_tune_result* res, const char* who) {
    if (int rc = make_space(sp, &s)) return rc;
    if (!opts || !res) {
      set_error(std::string(who) + ": null options or result");
      return GT_EINVAL;
    }
    if (opts->budget < 1 || opts->rho < 1) {
      set_error(std::string(who) + ": budget and rho must be >= 1");
      return GT_EINVAL;
    }
    o = opts;
    this->who = who;
    cost = cb;
    ctx = cb_ctx;
    out = res;
    std::memset(out, 0, sizeof(*out));
    return GT_OK;
  }

  // GPU mode: operands, tolerance, and the reference product (once).
  int prepare_gpu(const gt_space* sp, const char* who) {
    if (cost) return GT_OK;
    if (!o->A || !o->B || !o->C) {
      set_error(std::string(who) + ": GPU mode needs A, B and C");
      return GT_EINVAL;
    }
    g.o = o;
    g.M = sp->M;
    g.N = sp->N;
    g.K = sp->K;
    g.dtype = sp->dtype;
    g.s = static_cast<hipStream_t>(o->stream);
    g.tol = (sp->dtype & ~GT_A_KMAJOR) == GT_F32 ? 1e-5 * std::sqrt(static_cast<double>(sp->K))
                                                   : 2e-3;
    g.c_ref = o->c_ref;
    if (o->check) {
      if (!g.c_ref) {
        hipError_t e = hipMalloc(&owned_ref, static_cast<size_t>(sp->M * sp->N) * sizeof(float));
        if (e != hipSuccess) {
          owned_ref = nullptr;
          set_error(std::string(who) + ": hipMalloc reference: " + hipGetErrorString(e));
          return GT_EHIP;
        }
        g.c_ref = owned_ref;
      }
      int rc = gt_reference_gemm(o->A, o->B, g.c_ref, sp->M, sp->N, sp->K, sp->dtype, o->stream);
      if (rc == GT_OK && hipStreamSynchronize(g.s) != hipSuccess) rc = GT_EHIP;
      if (rc != GT_OK) return rc;
    }
    return GT_OK;
  }

  double elapsed() const {
    return std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  }

  // Times one configuration, logs it, counts it; returns its cost.
  double time_one(const gt_config& c, uint64_t rank) {
    gt_log_entry rec{};
    rec.rank = rank;
    double v;
    if (cost) {
      v = cost(&c, rank, ctx);
      rec.cost_ms = v;
      rec.first_ms = v;
      rec.rel_err = NAN;
      rec.status = std::isinf(v) ? 2 : 0;
    } else {
      v = gpu_cost(g, c, cost_min, &rec);
    }
    if (o->log && out->timed < o->log_cap) o->log[out->timed] = rec;
    ++out->timed;
    if (std::isinf(v)) ++out->failed;
    if (o->progress_s > 0.0) {
      const double t = elapsed();
      if (t - last_progress >= o->progress_s) {
        last_progress = t;
        std::fprintf(stderr, "[gemmtune] %s: %lld of %lld timed, best %.4f ms, %.1f s\n", who,
                     static_cast<long long>(out->timed), static_cast<long long>(o->budget),
                     std::min(cost_min, v), t);
        std::fflush(stderr);
      }
    }
    return v;
  }

  // After a device error that outlives its call: the result so far, and
  // GT_EHIP with the configuration that was being timed.
  bool fatal() const { return g.fatal != hipSuccess; }
  int fail_fatal(const char* who, const gt_config& c, uint64_t best) {
    finish(best);
    set_error(std::string(who) + ": device error while timing " + describe(c) + ": " +
              hipGetErrorString(g.fatal));
    return GT_EHIP;
  }

  void finish(uint64_t best) {
    unrank_into(s, best, &out->best);
    out->best_rank = best;
    out->best_cost = cost_min;
    out->wall_s = elapsed();
  }
};

}  // namespace
}  // namespace gt

extern "C" {

int tune_gbfs(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
              gt_tune_result* out) {
  using namespace gt;
  Tuner t;
  if (int rc = t.init(sp, o, cost, ctx, out, "tune_gbfs")) return rc;
  const Space& s = t.s;

  // start state: caller's, or [D,1,...,1] per dimension with MFMA 16
  gt_config s0{};
  if (o->s0) {
    s0 = *o->s0;
  } else {
    s0.d_m = s.dim[0].d;
    s0.d_k = s.dim[1].d;
    s0.d_n = s.dim[2].d;
    s0.m[0] = sp->M;
    s0.k[0] = sp->K;
    s0.n[0] = sp->N;
    for (int i = 1; i < s0.d_m; ++i) s0.m[i] = 1;
    for (int i = 1; i < s0.d_k; ++i) s0.k[i] = 1;
    for (int i = 1; i < s0.d_n; ++i) s0.n[i] = 1;
    s0.mfma = s.mfma_coord ? 16 : 0;
  }
  if (!is_member(s, s0)) {
    set_error("tune_gbfs: s0 is not a member of the space");
    return GT_EDIMS;
  }
  if (!legit_of(s, s0)) {
    set_error("tune_gbfs: s0 is not legitimate");
    return GT_EILLEGIT;
  }
  if (int rc = t.prepare_gpu(sp, "tune_gbfs")) return rc;

  using Item = std::pair<double, uint64_t>;  // (cost, rank), smallest first
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> q;
  std::unordered_set<uint64_t> visited;
  uint64_t rng = o->seed;

  const uint64_t r0 = rank_of(s, s0);
  const double c0 = t.time_one(s0, r0);
  visited.insert(r0);
  t.cost_min = c0;
  uint64_t best = r0;
  if (t.fatal()) return t.fail_fatal("tune_gbfs", s0, best);
  if (!std::isinf(c0)) q.push({c0, r0});

  out->stop_reason = 1;
  gt_config g_s[kMaxNeighbours];
  while (true) {
    if (out->timed >= o->budget) {
      out->stop_reason = 0;
      break;
    }
    if (q.empty()) {
      out->stop_reason = 1;
      break;
    }
    if (o->t_max_s > 0.0 && t.elapsed() >= o->t_max_s) {
      out->stop_reason = 2;
      break;
    }
    const Item top = q.top();
    q.pop();
    ++out->popped;
    gt_config cur;
    unrank_into(s, top.second, &cur);
    const int n = neighbour_list(s, cur, g_s);
    const int take = o->rho < n ? o->rho : n;
    for (int i = 0; i < take; ++i) {
      const int j = i + static_cast<int>(splitmix64(&rng) % static_cast<uint64_t>(n - i));
      std::swap(g_s[i], g_s[j]);
    }
    for (int i = 0; i < take && out->timed < o->budget; ++i) {
      if (!g_s[i].legit) {
        ++out->skipped_illegit;
        continue;
      }
      const uint64_t r = rank_of(s, g_s[i]);
      if (visited.count(r)) {
        ++out->skipped_visited;
        continue;
      }
      const double v = t.time_one(g_s[i], r);
      if (t.fatal()) return t.fail_fatal("tune_gbfs", g_s[i], best);
      visited.insert(r);
      if (!std::isinf(v)) q.push({v, r});
      if (v < t.cost_min) {
        t.cost_min = v;
        best = r;
      }
    }
  }
  if (out->timed >= o->budget) out->stop_reason = 0;
  t.finish(best);
  return GT_OK;
}

int tune_random(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
                gt_tune_result* out) {
  using namespace gt;
  Tuner t;
  if (int rc = t.init(sp, o, cost, ctx, out, "tune_random")) return rc;
  if (int rc = t.prepare_gpu(sp, "tune_random")) return rc;
  const Space& s = t.s;
  std::unordered_set<uint64_t> visited;
  uint64_t rng = o->seed;
  const int64_t max_draws = 64 * o->budget + 1024;
  uint64_t best = 0;
  bool have = false;
  out->stop_reason = 3;
  while (true) {
    if (out->timed >= o->budget) {
      out->stop_reason = 0;
      break;
    }
    if (out->popped >= max_draws) {
      out->stop_reason = 3;
      break;
    }
    if (o->t_max_s > 0.0 && t.elapsed() >= o->t_max_s) {
      out->stop_reason = 2;
      break;
    }
    const uint64_t r = splitmix64(&rng) % s.size;
    ++out->popped;
    gt_config c;
    unrank_into(s, r, &c);
    if (!c.legit) {
      ++out->skipped_illegit;
      continue;
    }
    if (visited.count(r)) {
      ++out->skipped_visited;
      continue;
    }
    visited.insert(r);
    const double v = t.time_one(c, r);
    if (t.fatal()) return t.fail_fatal("tune_random", c, best);
    if (!have || v < t.cost_min) {
      t.cost_min = v;
      best = r;
      have = true;
    }
  }
  t.finish(best);
  return GT_OK;
}

}  // extern "C"
