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
//
// N-A2C (§4.3, Alg.2): episodes of T-step walks from a centre (the best state
// so far) collect B unvisited legitimate states, chosen ε-greedily between a
// small actor network's policy and uniform actions; the collected states are
// timed, and every transition into a timed state from an already-timed
// neighbour trains the actor and a critic (one SGD pass over a FIFO memory
// after every timing). The arithmetic is written in a fixed order (no
// contraction of multiply-adds) so that a run is reproducible bit for bit.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <exception>
#include <new>
#include <queue>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <utility>
#include <vector>

#include <unistd.h>

#include "internal.h"
#include "runtime.h"

#pragma clang fp contract(off)

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
  RunStats st{NAN, NAN, NAN};
  const int rc = measure(c, g.o->A, g.o->B, g.o->C, g.M, g.N, g.K, g.dtype, g.s, g.o->warmup,
                         g.o->runs, abort_ms, &mean, &first, &aborted, &st);
  rec->first_ms = first;
  rec->median_ms = st.median_ms;
  rec->min_ms = st.min_ms;
  rec->stdev_ms = st.stdev_ms;
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
  o->trace_fd = -1;
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
           gt_tune_result* res, const char* caller) {
    if (int rc = make_space(sp, &s)) return rc;
    if (!opts || !res) {
      set_error(std::string(caller) + ": null options or result");
      return GT_EINVAL;
    }
    if (opts->budget < 1 || opts->rho < 1) {
      set_error(std::string(caller) + ": budget and rho must be >= 1");
      return GT_EINVAL;
    }
    o = opts;
    who = caller;
    cost = cb;
    ctx = cb_ctx;
    out = res;
    std::memset(out, 0, sizeof(*out));
    return GT_OK;
  }

  // GPU mode: operands, tolerance, and the reference product (once).
  int prepare_gpu(const gt_space* sp) {
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
    if (o->trace_fd >= 0) {
      // on record before any launch: unbuffered, one write per line
      const std::string line = std::string("[gemmtune] ") + who + " timing #" +
                               std::to_string(out->timed) + " rank " + std::to_string(rank) + " " +
                               describe(c) + "\n";
      (void)!::write(o->trace_fd, line.data(), line.size());
    }
    gt_log_entry rec{};
    rec.rank = rank;
    double v;
    const auto te = std::chrono::steady_clock::now();
    if (cost) {
      v = cost(&c, rank, ctx);
      if (std::isnan(v)) v = INFINITY;  // no number, no measurement: a failed candidate
      rec.cost_ms = v;
      rec.first_ms = v;
      rec.rel_err = NAN;
      rec.median_ms = rec.min_ms = v;
      rec.stdev_ms = 0.0;
      rec.status = std::isinf(v) ? 2 : 0;
    } else {
      v = gpu_cost(g, c, cost_min, &rec);
      // device time of the launches: the first warm-up, then the rest at the
      // timed mean (an early abort stops after the first)
      if (std::isfinite(rec.first_ms)) out->device_s += rec.first_ms * 1e-3;
      if (rec.status != 1 && std::isfinite(rec.cost_ms))
        out->device_s += (o->runs + std::max(o->warmup, 1) - 1) * rec.cost_ms * 1e-3;
    }
    out->eval_s += std::chrono::duration<double>(std::chrono::steady_clock::now() - te).count();
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
  int fail_fatal(const gt_config& c, uint64_t best) {
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

static int tune_gbfs_impl(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
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
  if (int rc = t.prepare_gpu(sp)) return rc;

  using Item = std::pair<double, uint64_t>;  // (cost, rank), smallest first
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> q;
  std::unordered_set<uint64_t> visited;
  uint64_t rng = o->seed;

  const uint64_t r0 = rank_of(s, s0);
  const double c0 = t.time_one(s0, r0);
  visited.insert(r0);
  t.cost_min = c0;
  uint64_t best = r0;
  if (t.fatal()) return t.fail_fatal(s0, best);
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
      if (t.fatal()) return t.fail_fatal(g_s[i], best);
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

static int tune_random_impl(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
                            gt_tune_result* out) {
  using namespace gt;
  Tuner t;
  if (int rc = t.init(sp, o, cost, ctx, out, "tune_random")) return rc;
  if (int rc = t.prepare_gpu(sp)) return rc;
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
    if (t.fatal()) return t.fail_fatal(c, best);
    if (!have || v < t.cost_min) {
      t.cost_min = v;
      best = r;
      have = true;
    }
  }
  t.finish(best);
  return GT_OK;
}


int gt_na2c_params_init(gt_na2c_params* p) {
  if (!p) {
    gt::set_error("gt_na2c_params_init: null");
    return GT_EINVAL;
  }
  std::memset(p, 0, sizeof(*p));
  p->T = 3;
  p->B = 8;
  p->H = 32;
  p->mem = 256;
  p->max_walks = 64;
  p->eps = 0.8;
  p->gamma = 0.9;
  p->lr = 0.01;
  p->r_clip = 5.0;
  return GT_OK;
}

}  // extern "C"

namespace gt {
namespace {

// The fixed action list of N-A2C: per dimension (m, k, n) the ordered level
// pairs (i, j) the neighbour mode allows — ×2 at level i, ÷2 at level j —
// then the MFMA toggle when the space has that coordinate.
struct Move {
  int dim, up, down;
  bool toggle;
};

class Agent {
 public:
  Agent(const Space& s, const gt_na2c_params& p, uint64_t seed) : s_(s), H_(p.H) {
    for (int x = 0; x < 3; ++x)
      for (int i = 0; i < s.dim[x].d; ++i)
        for (int j = 0; j < s.dim[x].d; ++j)
          if (i != j && (s.mode == GT_ANY_PAIR || i - j == 1 || j - i == 1))
            moves_.push_back({x, i, j, false});
    if (s.mfma_coord) moves_.push_back({0, 0, 0, true});
    A_ = static_cast<int>(moves_.size());
    F_ = s.dim[0].d + s.dim[1].d + s.dim[2].d + (s.mfma_coord ? 1 : 0);
    W1_.assign(H_ * F_, 0.0);
    b1_.assign(H_, 0.0);
    W2_.assign(A_ * H_, 0.0);
    b2_.assign(A_, 0.0);
    U1_.assign(H_ * F_, 0.0);
    c1_.assign(H_, 0.0);
    u2_.assign(H_, 0.0);
    uint64_t ws = seed ^ 0xA2C0A2C0A2C0A2C0ull;
    const double bF = 1.0 / std::sqrt(static_cast<double>(F_));
    const double bH = 1.0 / std::sqrt(static_cast<double>(H_));
    for (double& w : W1_) w = (2.0 * uniform(&ws) - 1.0) * bF;
    for (double& w : W2_) w = (2.0 * uniform(&ws) - 1.0) * bH;
    for (double& w : U1_) w = (2.0 * uniform(&ws) - 1.0) * bF;
    for (double& w : u2_) w = (2.0 * uniform(&ws) - 1.0) * bH;
  }

  static double uniform(uint64_t* st) {
    return static_cast<double>(splitmix64(st) >> 11) * (1.0 / 9007199254740992.0);
  }

  int actions() const { return A_; }
  int features() const { return F_; }

  static int64_t* lv(gt_config& c, int x) { return x == 0 ? c.m : (x == 1 ? c.k : c.n); }
  static const int64_t* lv(const gt_config& c, int x) { return x == 0 ? c.m : (x == 1 ? c.k : c.n); }

  bool available(const gt_config& c, int a) const {
    const Move& m = moves_[a];
    return m.toggle || lv(c, m.dim)[m.down] % 2 == 0;
  }
  gt_config step(const gt_config& c, int a) const {
    gt_config t = c;
    const Move& m = moves_[a];
    if (m.toggle) {
      t.mfma = c.mfma == 16 ? 32 : 16;
    } else {
      lv(t, m.dim)[m.up] = lv(c, m.dim)[m.up] * 2;
      lv(t, m.dim)[m.down] = lv(c, m.dim)[m.down] / 2;
    }
    return t;
  }
  int inverse(int a) const {
    const Move& m = moves_[a];
    if (m.toggle) return a;
    for (int b = 0; b < A_; ++b)
      if (!moves_[b].toggle && moves_[b].dim == m.dim && moves_[b].up == m.down &&
          moves_[b].down == m.up)
        return b;
    return -1;
  }
  void features(const gt_config& c, double* phi) const {
    int k = 0;
    for (int x = 0; x < 3; ++x) {
      const Dim& dm = s_.dim[x];
      for (int i = 0; i < dm.d; ++i) {
        int64_t v = i == 0 ? lv(c, x)[0] / dm.q : lv(c, x)[i];
        int e = 0;
        while (v > 1) {
          v >>= 1;
          ++e;
        }
        phi[k++] = dm.E ? static_cast<double>(e) / static_cast<double>(dm.E) : 0.0;
      }
    }
    if (s_.mfma_coord) phi[k++] = c.mfma == 32 ? 1.0 : 0.0;
  }

  // π over the available actions (0 elsewhere); h = hidden activations.
  void policy(const double* phi, const char* avail, double* h, double* pi) const {
    for (int k = 0; k < H_; ++k) {
      double z = b1_[k];
      for (int f = 0; f < F_; ++f) z += W1_[k * F_ + f] * phi[f];
      h[k] = std::tanh(z);
    }
    double zmax = -INFINITY;
    for (int a = 0; a < A_; ++a) {
      pi[a] = 0.0;
      if (!avail[a]) continue;
      double z = b2_[a];
      for (int k = 0; k < H_; ++k) z += W2_[a * H_ + k] * h[k];
      pi[a] = z;
      if (z > zmax) zmax = z;
    }
    double sum = 0.0;
    for (int a = 0; a < A_; ++a)
      if (avail[a]) {
        pi[a] = std::exp(pi[a] - zmax);
        sum += pi[a];
      }
    for (int a = 0; a < A_; ++a)
      if (avail[a]) pi[a] /= sum;
  }

  double value(const double* phi, double* g) const {
    double v = c2_;
    for (int k = 0; k < H_; ++k) {
      double z = c1_[k];
      for (int f = 0; f < F_; ++f) z += U1_[k * F_ + f] * phi[f];
      g[k] = std::tanh(z);
      v += u2_[k] * g[k];
    }
    return v;
  }

  struct Transition {
    double phi[3 * GT_MAXD + 1], phi2[3 * GT_MAXD + 1];
    char avail[kMaxNeighbours];
    int a;
    double r;
  };

  // TD(0) advantage δ = r + γV(s') − V(s); every parameter θ moves by
  // (lr·δ)·∂/∂θ, with ∂/∂θ of V(s) for the critic and of log π(a|s) for the
  // actor, all taken at the weights before this update.
  void train(const Transition& t, double gamma, double lr) {
    double g[64], g2[64], h[64], dh[64], pi[kMaxNeighbours];
    const double v2 = value(t.phi2, g2);
    const double v = value(t.phi, g);
    const double delta = t.r + gamma * v2 - v;
    const double step = lr * delta;
    for (int k = 0; k < H_; ++k) {
      const double back = u2_[k] * (1.0 - g[k] * g[k]);
      for (int f = 0; f < F_; ++f) U1_[k * F_ + f] += step * (back * t.phi[f]);
      c1_[k] += step * back;
    }
    for (int k = 0; k < H_; ++k) u2_[k] += step * g[k];
    c2_ += step;
    policy(t.phi, t.avail, h, pi);
    for (int k = 0; k < H_; ++k) {
      double acc = 0.0;
      for (int b = 0; b < A_; ++b)
        if (t.avail[b]) acc += ((b == t.a ? 1.0 : 0.0) - pi[b]) * W2_[b * H_ + k];
      dh[k] = acc * (1.0 - h[k] * h[k]);
    }
    for (int b = 0; b < A_; ++b) {
      if (!t.avail[b]) continue;
      const double e = (b == t.a ? 1.0 : 0.0) - pi[b];
      for (int k = 0; k < H_; ++k) W2_[b * H_ + k] += step * (e * h[k]);
      b2_[b] += step * e;
    }
    for (int k = 0; k < H_; ++k) {
      for (int f = 0; f < F_; ++f) W1_[k * F_ + f] += step * (dh[k] * t.phi[f]);
      b1_[k] += step * dh[k];
    }
  }

 private:
  const Space& s_;
  int H_, A_ = 0, F_ = 0;
  std::vector<Move> moves_;
  std::vector<double> W1_, b1_, W2_, b2_, U1_, c1_, u2_;
  double c2_ = 0.0;
};

// r(s, a) for a transition into s' (cost `after`) from s (cost `before`):
// §4.1's 1/cost(s') (a failed s', cost +inf, earns 0), or with log_ratio the
// variant log(cost(s)/cost(s')) clipped to ±clip.
double reward(bool log_ratio, double before, double after, double clip) {
  if (!log_ratio) return 1.0 / after;
  if (std::isinf(after)) return std::isinf(before) ? 0.0 : -clip;
  if (std::isinf(before)) return clip;
  return std::min(clip, std::max(-clip, std::log(before / after)));
}

}  // namespace
}  // namespace gt

extern "C" {

static int tune_na2c_impl(const gt_space* sp, const gt_tune_opts* o, const gt_na2c_params* params,
                          gt_cost_fn cost, void* ctx, gt_tune_result* out) {
  using namespace gt;
  Tuner t;
  if (int rc = t.init(sp, o, cost, ctx, out, "tune_na2c")) return rc;
  gt_na2c_params p;
  gt_na2c_params_init(&p);
  if (params) p = *params;
  if (p.T < 1 || p.T > 64 || p.B < 1 || p.B > 65536 || p.H < 1 || p.H > 64 || p.mem < 1 ||
      p.mem > 65536 || p.max_walks < 1 || p.max_walks > (1 << 20) ||
      !(p.eps >= 0.0 && p.eps <= 1.0) || !(p.lr >= 0.0) || !(p.r_clip > 0.0) ||
      (p.reward != 0 && p.reward != 1) || (p.eps_halving != 0 && p.eps_halving != 1)) {
    set_error("tune_na2c: parameters out of range (1 <= T <= 64; 1 <= B, mem <= 65536; "
              "1 <= max_walks <= 2^20; 1 <= H <= 64; 0 <= eps <= 1; lr >= 0; r_clip > 0; "
              "reward and eps_halving 0 or 1)");
    return GT_EINVAL;
  }
  const Space& s = t.s;
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
  if (!is_member(s, s0) || !legit_of(s, s0)) {
    set_error("tune_na2c: s0 is not a legitimate member of the space");
    return is_member(s, s0) ? GT_EILLEGIT : GT_EDIMS;
  }
  if (int rc = t.prepare_gpu(sp)) return rc;

  Agent agent(s, p, o->seed);
  const int A = agent.actions();
  std::unordered_map<uint64_t, double> hv;  // H_v: rank → cost
  std::vector<Agent::Transition> mem;       // M, FIFO
  size_t mem_head = 0;
  uint64_t rng = o->seed;

  const uint64_t r0 = rank_of(s, s0);
  const double c0 = t.time_one(s0, r0);
  hv[r0] = c0;
  t.cost_min = c0;
  uint64_t best = r0;
  if (t.fatal()) return t.fail_fatal(s0, best);
  gt_config centre = s0;

  out->stop_reason = 1;
  std::vector<gt_config> coll;
  std::vector<uint64_t> coll_r;
  double phi[3 * GT_MAXD + 1], h[64], pi[kMaxNeighbours];
  char avail[kMaxNeighbours];
  int walk = p.T;        // walk length: grows by one after an episode that collects nothing
  double eps_now = p.eps;  // share of policy steps (halves after such an episode: variant)
  while (true) {
    if (out->timed >= o->budget) {
      out->stop_reason = 0;
      break;
    }
    if (o->t_max_s > 0.0 && t.elapsed() >= o->t_max_s) {
      out->stop_reason = 2;
      break;
    }
    // collect B unvisited legitimate states by walks from the centre
    coll.clear();
    coll_r.clear();
    for (int w = 0; w < p.max_walks && static_cast<int>(coll.size()) < p.B; ++w) {
      gt_config cur = centre;
      for (int step = 0; step < walk; ++step) {
        int navail = 0;
        for (int a = 0; a < A; ++a) navail += (avail[a] = agent.available(cur, a) ? 1 : 0);
        if (navail == 0) break;  // no move leaves cur: the walk ends, nothing drawn
        int act = -1;
        if (Agent::uniform(&rng) < eps_now) {
          agent.features(cur, phi);
          agent.policy(phi, avail, h, pi);
          const double u = Agent::uniform(&rng);
          double cum = 0.0;
          for (int b = 0; b < A; ++b) {
            if (!avail[b]) continue;
            act = b;
            cum += pi[b];
            if (u < cum) break;
          }
        } else {
          int k = static_cast<int>(splitmix64(&rng) % static_cast<uint64_t>(navail));
          for (int b = 0; b < A && act < 0; ++b)
            if (avail[b] && k-- == 0) act = b;
        }
        const gt_config nxt = agent.step(cur, act);
        if (legit_of(s, nxt)) {
          const uint64_t r = rank_of(s, nxt);
          bool dup = hv.count(r) != 0;
          for (uint64_t q : coll_r) dup = dup || q == r;
          if (!dup && static_cast<int>(coll.size()) < p.B) {
            coll.push_back(nxt);
            coll_r.push_back(r);
          }
        }
        cur = nxt;
      }
    }
    ++out->popped;
    if (coll.empty()) {
      // nothing new within `walk` steps of the centre: look one step further
      // (the exploration step may grow, §4.3), up to T + 8, then stop; the
      // eps_halving variant also halves the share of policy steps
      if (walk >= p.T + 8) {
        out->stop_reason = 1;
        break;
      }
      ++walk;
      if (p.eps_halving) eps_now *= 0.5;
      continue;
    }
    for (size_t b = 0; b < coll.size() && out->timed < o->budget; ++b) {
      const double c = t.time_one(coll[b], coll_r[b]);
      if (t.fatal()) return t.fail_fatal(coll[b], best);
      if (c < t.cost_min) {
        t.cost_min = c;
        best = coll_r[b];
        centre = coll[b];
        walk = p.T;  // a new centre: back to T-step walks and the full ε
        eps_now = p.eps;
      }
      hv[coll_r[b]] = c;
      // every (s, a) with step(s, a) = s' and s already timed
      for (int bb = 0; bb < A; ++bb) {
        if (!agent.available(coll[b], bb)) continue;
        const gt_config prev = agent.step(coll[b], bb);
        if (!is_member(s, prev)) continue;
        const auto it = hv.find(rank_of(s, prev));
        if (it == hv.end()) continue;
        Agent::Transition tr{};
        agent.features(prev, tr.phi);
        agent.features(coll[b], tr.phi2);
        for (int a = 0; a < A; ++a) tr.avail[a] = agent.available(prev, a) ? 1 : 0;
        tr.a = agent.inverse(bb);
        tr.r = reward(p.reward == 1, it->second, c, p.r_clip);
        if (mem.size() < static_cast<size_t>(p.mem)) {
          mem.push_back(tr);
        } else {
          mem[mem_head] = tr;
          mem_head = (mem_head + 1) % mem.size();
        }
      }
      for (size_t k = 0; k < mem.size(); ++k)
        agent.train(mem[(mem_head + k) % mem.size()], p.gamma, p.lr);
    }
  }
  if (out->timed >= o->budget) out->stop_reason = 0;
  t.finish(best);
  return GT_OK;
}


}  // extern "C"

namespace {
// The searches allocate host memory as they go (queue, visited set, memory of
// transitions); no C++ exception crosses the C ABI.
template <class F>
int guarded(const char* who, F f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    gt::set_error(std::string(who) + ": out of host memory");
  } catch (const std::exception& e) {
    gt::set_error(std::string(who) + ": " + e.what());
  }
  return GT_EINVAL;
}
}  // namespace

extern "C" {

int tune_gbfs(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
              gt_tune_result* out) {
  return guarded("tune_gbfs", [&] { return tune_gbfs_impl(sp, o, cost, ctx, out); });
}

int tune_random(const gt_space* sp, const gt_tune_opts* o, gt_cost_fn cost, void* ctx,
                gt_tune_result* out) {
  return guarded("tune_random", [&] { return tune_random_impl(sp, o, cost, ctx, out); });
}

int tune_na2c(const gt_space* sp, const gt_tune_opts* o, const gt_na2c_params* params,
              gt_cost_fn cost, void* ctx, gt_tune_result* out) {
  return guarded("tune_na2c", [&] { return tune_na2c_impl(sp, o, params, cost, ctx, out); });
}

}  // extern "C"
