// Configuration space of the tiled GEMM (§3.3 Eq.1–4), the state legitimacy
// bit J (§4.1 Eq.5 and its footnote) and the neighbour relation (§4.1 Eq.6,
// Eq.7, Eq.9). Pure host code.
//
// Within a dimension the tuples are ordered lexicographically on their
// exponents (e_0, …, e_{d−1}), Σ e_i = E; rank and unrank count weak
// compositions directly instead of materialising the list.
#include <algorithm>
#include <cstring>
#include <exception>
#include <mutex>
#include <thread>
#include <vector>

#include "internal.h"

namespace gt {

namespace {

thread_local std::string g_error;

// C(n, k) for the small arguments used here (n ≤ 64 + 3).
uint64_t binom(int64_t n, int64_t k) {
  if (k < 0 || n < 0 || k > n) return 0;
  if (k > n - k) k = n - k;
  uint64_t r = 1;
  for (int64_t i = 1; i <= k; ++i) r = r * static_cast<uint64_t>(n - k + i) / static_cast<uint64_t>(i);
  return r;
}

// Weak compositions of s into p ≥ 1 parts.
uint64_t weak(int64_t s, int p) {
  if (s < 0) return 0;
  if (p == 1) return 1;
  return binom(s + p - 1, p - 1);
}

int ilog2(int64_t v) {
  int e = 0;
  while ((int64_t{1} << e) < v) ++e;
  return e;
}

bool pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

// Exponents of a member tuple of dimension x (e_0 excludes the odd cofactor).
void exponents(const Dim& dm, const int64_t* f, int* e) {
  e[0] = ilog2(f[0] / dm.q);
  for (int i = 1; i < dm.d; ++i) e[i] = ilog2(f[i]);
}

uint64_t dim_rank(const Dim& dm, const int64_t* f) {
  int e[GT_MAXD];
  exponents(dm, f, e);
  uint64_t r = 0;
  int64_t rem = dm.E;
  for (int i = 0; i + 1 < dm.d; ++i) {
    for (int v = 0; v < e[i]; ++v) r += weak(rem - v, dm.d - i - 1);
    rem -= e[i];
  }
  return r;
}

void dim_unrank(const Dim& dm, uint64_t r, int64_t* f) {
  int64_t rem = dm.E;
  for (int i = 0; i < dm.d; ++i) {
    int v = 0;
    if (i + 1 < dm.d) {
      for (;; ++v) {
        const uint64_t w = weak(rem - v, dm.d - i - 1);
        if (r < w) break;
        r -= w;
      }
    } else {
      v = static_cast<int>(rem);
    }
    f[i] = (int64_t{1} << v) * (i == 0 ? dm.q : 1);
    rem -= v;
  }
  for (int i = dm.d; i < GT_MAXD; ++i) f[i] = 0;
}

const int64_t* dim_factors(const gt_config& c, int x) {
  return x == 0 ? c.m : (x == 1 ? c.k : c.n);
}
int64_t* dim_factors(gt_config& c, int x) { return x == 0 ? c.m : (x == 1 ? c.k : c.n); }

}  // namespace

void set_error(const std::string& msg) { g_error = msg; }
const std::string& last_error() { return g_error; }

int make_space(const gt_space* sp, Space* s) {
  if (!sp || !s) {
    set_error("null space");
    return GT_EINVAL;
  }
  const int64_t ext[3] = {sp->M, sp->K, sp->N};
  const int32_t d[3] = {sp->d_m, sp->d_k, sp->d_n};
  const int base = sp->dtype & ~GT_A_KMAJOR;
  if (base != GT_F32 && base != GT_BF16) {
    set_error("space: dtype must be GT_F32 or GT_BF16 (optionally | GT_A_KMAJOR)");
    return GT_EINVAL;
  }
  if (sp->mfma_coord != 0 && sp->mfma_coord != 1) {
    set_error("space: mfma_coord must be 0 or 1");
    return GT_EINVAL;
  }
  if (sp->neighbour_mode != GT_ADJACENT && sp->neighbour_mode != GT_ANY_PAIR) {
    set_error("space: bad neighbour_mode");
    return GT_EINVAL;
  }
  s->size = 1;
  for (int x = 0; x < 3; ++x) {
    if (ext[x] < 1 || ext[x] > (int64_t{1} << 40) || d[x] < 1 || d[x] > GT_MAXD) {
      set_error("space: extents must be in [1, 2^40] and level counts in [1, 4]");
      return GT_EINVAL;
    }
    Dim& dm = s->dim[x];
    dm.D = ext[x];
    dm.q = ext[x];
    dm.E = 0;
    while (dm.q % 2 == 0) {
      dm.q /= 2;
      ++dm.E;
    }
    dm.d = d[x];
    dm.count = binom(dm.E + dm.d - 1, dm.d - 1);
    s->size *= dm.count;
    s->ext[x] = ext[x];
  }
  s->n_mfma = sp->mfma_coord ? 2 : 1;
  s->size *= s->n_mfma;
  s->dtype = base;
  s->a_kmajor = (sp->dtype & GT_A_KMAJOR) != 0;
  s->mfma_coord = sp->mfma_coord;
  s->mode = sp->neighbour_mode;
  return GT_OK;
}

bool is_member(const Space& s, const gt_config& c) {
  const int32_t cd[3] = {c.d_m, c.d_k, c.d_n};
  for (int x = 0; x < 3; ++x) {
    const Dim& dm = s.dim[x];
    if (cd[x] != dm.d) return false;
    const int64_t* f = dim_factors(c, x);
    int64_t prod = 1;
    for (int i = 0; i < dm.d; ++i) {
      const int64_t v = f[i];
      if (v <= 0) return false;
      if (i == 0) {
        if (v % dm.q != 0 || !pow2(v / dm.q)) return false;
      } else if (!pow2(v)) {
        return false;
      }
      if (v > dm.D / prod) return false;
      prod *= v;
    }
    if (prod != dm.D) return false;
  }
  if (s.mfma_coord) return c.mfma == 16 || c.mfma == 32;
  return c.mfma == 0;
}

uint64_t rank_of(const Space& s, const gt_config& c) {
  uint64_t r = 0;
  for (int x = 0; x < 3; ++x) r = r * s.dim[x].count + dim_rank(s.dim[x], dim_factors(c, x));
  return r * s.n_mfma + (s.mfma_coord && c.mfma == 32 ? 1 : 0);
}

void unrank_into(const Space& s, uint64_t rank, gt_config* c) {
  std::memset(c, 0, sizeof(*c));
  c->d_m = s.dim[0].d;
  c->d_k = s.dim[1].d;
  c->d_n = s.dim[2].d;
  const uint64_t im = rank % s.n_mfma;
  rank /= s.n_mfma;
  uint64_t r[3];
  for (int x = 2; x >= 0; --x) {
    r[x] = rank % s.dim[x].count;
    rank /= s.dim[x].count;
  }
  for (int x = 0; x < 3; ++x) dim_unrank(s.dim[x], r[x], dim_factors(*c, x));
  c->mfma = s.mfma_coord ? (im ? 32 : 16) : 0;
  c->legit = legit_of(s, *c);
}

void levels_of(const gt_config& c, int dtype, Levels* L) {
  auto mn = [](const int64_t* f, int d, int64_t* g, int64_t* w, int64_t* r, int64_t* b) {
    *g = f[0];
    *w = d >= 3 ? f[1] : 1;
    *r = d == 4 ? f[2] : 1;
    *b = d == 1 ? 1 : f[d - 1];
  };
  mn(c.m, c.d_m, &L->gridM, &L->wavesM, &L->repM, &L->blkM);
  mn(c.n, c.d_n, &L->gridN, &L->wavesN, &L->repN, &L->blkN);
  L->kLoop = c.k[0];
  L->kSplit = c.d_k == 4 ? c.k[1] : 1;
  L->kSub = c.d_k == 4 ? c.k[2] : (c.d_k == 3 ? c.k[1] : 1);
  L->kBlk = c.d_k == 1 ? 1 : c.k[c.d_k - 1];
  if (c.mfma == 16 || c.mfma == 32)
    L->I = c.mfma;
  else
    L->I = (L->blkM % 32 == 0 && L->blkN % 32 == 0) ? 32 : 16;
  if (dtype == GT_BF16)
    L->IK = L->I == 32 ? 16 : 32;
  else
    L->IK = L->I == 32 ? 2 : 4;
  L->TM = L->repM * ((L->blkM + L->I - 1) / L->I);
  L->TN = L->repN * ((L->blkN + L->I - 1) / L->I);
  L->acc = L->TM * L->TN * L->I * L->I / 64;
  L->W = L->wavesM * L->wavesN;
  L->BM = L->wavesM * L->repM * L->blkM;
  L->BN = L->wavesN * L->repN * L->blkN;
  L->BK = L->kSub * L->kBlk;
  L->elem = dtype == GT_BF16 ? 2 : 4;
}

namespace {
// The hardware clauses of J (a member's levels).
int legit_levels(const Levels& L) {
  if (L.W > 16) return 0;
  if (L.acc > 256) return 0;
  const int64_t simd_share = (L.W + 3) / 4;
  if (L.acc + 96 > 512 / simd_share) return 0;
  if ((L.BM * L.BK + L.BK * L.BN) * L.elem > kLdsMax) return 0;
  // a dispatch packet holds at most 2^32 - 1 work-items per grid dimension
  if (L.gridM * L.gridN * 64 * L.W > int64_t{4294967295}) return 0;
  if (L.kSplit > 65535) return 0;
  // and the launch as a whole stays below 2^32 work-items, so that no 32-bit
  // count over the whole dispatch can wrap (this also bounds the split-K
  // partial sums, M·N·kSplit atomics, and the launches a search can time)
  if (L.gridM * L.gridN * L.kSplit * 64 * L.W > int64_t{4294967295}) return 0;
  return 1;
}
}  // namespace

int legit_of(const Space& s, const gt_config& c) {
  if (!is_member(s, c)) return 0;
  Levels L;
  levels_of(c, s.dtype, &L);
  return legit_levels(L);
}

// Configurations of ranks [start, start + n) in canonical order: each
// dimension's tuples are unranked once into a table, then an odometer over
// (m, k, n, mfma) fills the records; J from the levels (members by
// construction). Large requests are split over threads.
void enumerate_range(const Space& s, uint64_t start, uint64_t n, gt_config* out) {
  std::vector<int64_t> tab[3];
  for (int x = 0; x < 3; ++x) {
    tab[x].resize(s.dim[x].count * GT_MAXD);
    for (uint64_t r = 0; r < s.dim[x].count; ++r) dim_unrank(s.dim[x], r, &tab[x][r * GT_MAXD]);
  }
  auto part = [&](uint64_t first, uint64_t count) {
    uint64_t rank = first;
    uint64_t im = rank % s.n_mfma;
    rank /= s.n_mfma;
    uint64_t r[3];
    for (int x = 2; x >= 0; --x) {
      r[x] = rank % s.dim[x].count;
      rank /= s.dim[x].count;
    }
    gt_config c;
    std::memset(&c, 0, sizeof(c));
    c.d_m = s.dim[0].d;
    c.d_k = s.dim[1].d;
    c.d_n = s.dim[2].d;
    Levels L;
    for (uint64_t i = 0; i < count; ++i) {
      for (int x = 0; x < 3; ++x)
        std::memcpy(dim_factors(c, x), &tab[x][r[x] * GT_MAXD], GT_MAXD * sizeof(int64_t));
      c.mfma = s.mfma_coord ? (im ? 32 : 16) : 0;
      levels_of(c, s.dtype, &L);
      c.legit = legit_levels(L);
      out[first - start + i] = c;
      if (++im < s.n_mfma) continue;
      im = 0;
      for (int x = 2; x >= 0; --x) {
        if (++r[x] < s.dim[x].count) break;
        r[x] = 0;
      }
    }
  };
  const uint64_t per = uint64_t{1} << 20;
  const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
  const unsigned nt = static_cast<unsigned>(std::min<uint64_t>(std::min(hw, 16u), (n + per - 1) / per));
  if (nt <= 1) {
    part(start, n);
    return;
  }
  std::vector<std::thread> th;
  const uint64_t chunk = (n + nt - 1) / nt;
  uint64_t done = 0;  // records [0, done) are owned by started threads
  try {
    th.reserve(nt);
    for (unsigned t = 0; t < nt; ++t) {
      const uint64_t a = t * chunk;
      if (a >= n) break;
      th.emplace_back(part, start + a, std::min(chunk, n - a));
      done = std::min(n, a + chunk);
    }
  } catch (const std::exception&) {
    // no more threads: this thread fills the rest
  }
  if (done < n) part(start + done, n - done);
  for (auto& t : th) t.join();
}

int neighbour_list(const Space& s, const gt_config& c, gt_config* out) {
  struct Item {
    uint64_t rank;
    gt_config cfg;
  };
  Item items[kMaxNeighbours];
  int n = 0;
  for (int x = 0; x < 3; ++x) {
    const int d = s.dim[x].d;
    const int64_t* f = dim_factors(c, x);
    for (int i = 0; i < d; ++i) {
      for (int j = 0; j < d; ++j) {
        if (i == j) continue;
        if (s.mode == GT_ADJACENT && (i - j != 1 && j - i != 1)) continue;
        if (f[j] % 2 != 0) continue;  // f_j / 2 must stay a positive integer
        gt_config t = c;
        dim_factors(t, x)[i] *= 2;
        dim_factors(t, x)[j] /= 2;
        items[n].cfg = t;
        items[n].rank = rank_of(s, t);
        ++n;
      }
    }
  }
  if (s.mfma_coord) {
    gt_config t = c;
    t.mfma = c.mfma == 16 ? 32 : 16;
    items[n].cfg = t;
    items[n].rank = rank_of(s, t);
    ++n;
  }
  std::sort(items, items + n, [](const Item& a, const Item& b) { return a.rank < b.rank; });
  for (int i = 0; i < n; ++i) {
    out[i] = items[i].cfg;
    out[i].legit = legit_of(s, out[i]);
  }
  return n;
}

}  // namespace gt

using gt::set_error;

extern "C" {

const char* gt_last_error(void) { return gt::last_error().c_str(); }

int gt_space_size(const gt_space* sp, uint64_t* size) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!size) {
    set_error("gt_space_size: null output");
    return GT_EINVAL;
  }
  *size = s.size;
  return GT_OK;
}

int enumerate_configs(const gt_space* sp, uint64_t start_rank, gt_config* out, uint64_t cap,
                      uint64_t* n_out) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!n_out || (cap && !out)) {
    set_error("enumerate_configs: null output");
    return GT_EINVAL;
  }
  if (start_rank > s.size) {
    set_error("enumerate_configs: start_rank beyond the space");
    return GT_EINVAL;
  }
  const uint64_t n = std::min<uint64_t>(cap, s.size - start_rank);
  if (n) gt::enumerate_range(s, start_rank, n, out);
  *n_out = n;
  return GT_OK;
}

int config_rank(const gt_space* sp, const gt_config* cfg, uint64_t* rank) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!cfg || !rank) {
    set_error("config_rank: null argument");
    return GT_EINVAL;
  }
  if (!gt::is_member(s, *cfg)) {
    set_error("config_rank: configuration is not a member of the space");
    return GT_EDIMS;
  }
  *rank = gt::rank_of(s, *cfg);
  return GT_OK;
}

int config_unrank(const gt_space* sp, uint64_t rank, gt_config* cfg) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!cfg || rank >= s.size) {
    set_error("config_unrank: null output or rank out of range");
    return GT_EINVAL;
  }
  gt::unrank_into(s, rank, cfg);
  return GT_OK;
}

int config_legit(const gt_space* sp, const gt_config* cfg, int* J) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!cfg || !J) {
    set_error("config_legit: null argument");
    return GT_EINVAL;
  }
  *J = gt::legit_of(s, *cfg);
  return GT_OK;
}

int neighbours(const gt_space* sp, const gt_config* cfg, gt_config* out, int cap, int* n_out) {
  gt::Space s;
  if (int rc = gt::make_space(sp, &s)) return rc;
  if (!cfg || !n_out || (cap > 0 && !out)) {
    set_error("neighbours: null argument");
    return GT_EINVAL;
  }
  if (!gt::is_member(s, *cfg)) {
    set_error("neighbours: configuration is not a member of the space");
    return GT_EDIMS;
  }
  gt_config tmp[gt::kMaxNeighbours];
  const int n = gt::neighbour_list(s, *cfg, tmp);
  *n_out = n;
  if (n > cap) {
    set_error("neighbours: output buffer too small");
    return GT_ESMALL;
  }
  for (int i = 0; i < n; ++i) out[i] = tmp[i];
  return GT_OK;
}

}  // extern "C"
