/*
 * oracle.c — plain, slow, obviously correct CPU reference.
 * TEST INFRASTRUCTURE ONLY (see oracle.h). Shares nothing with the GPU library.
 */
#include "oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Inputs: exact widening of the bytes the GPU receives.                     */
/* ------------------------------------------------------------------------ */

static double widen_one(const void* base, int dtype, int64_t idx) {
  if (dtype == OR_F32) {
    float f;
    memcpy(&f, (const char*)base + 4 * idx, 4);
    return (double)f;
  }
  /* bf16: the 16 bits are the top half of an IEEE-754 binary32 value. */
  uint16_t h;
  memcpy(&h, (const char*)base + 2 * idx, 2);
  uint32_t bits = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

int oracle_widen(const void* src, int dtype, int64_t n, double* dst) {
  for (int64_t i = 0; i < n; ++i) dst[i] = widen_one(src, dtype, i);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* GEMM (§3.2): C[i][j] = sum over l = 0..K-1, ascending, of A[i][l]*B[l][j]. */
/* ------------------------------------------------------------------------ */

typedef struct {
  int64_t M, N, K;
  const double* A;
  const double* B;
  double* C;
  int64_t r0, r1;
} gemm_job;

static void* gemm_rows(void* p) {
  gemm_job* j = (gemm_job*)p;
  for (int64_t i = j->r0; i < j->r1; ++i) {
    double* c = j->C + i * j->N;
    for (int64_t col = 0; col < j->N; ++col) c[col] = 0.0;
    for (int64_t l = 0; l < j->K; ++l) {
      const double a = j->A[i * j->K + l];
      const double* b = j->B + l * j->N;
      for (int64_t col = 0; col < j->N; ++col) c[col] += a * b[col];
    }
  }
  return NULL;
}

int oracle_gemm(int64_t M, int64_t N, int64_t K, const void* A, const void* B,
                int dtype, double* C, int nthreads) {
  double* a = (double*)malloc(sizeof(double) * (size_t)(M * K));
  double* b = (double*)malloc(sizeof(double) * (size_t)(K * N));
  if ((M * K > 0 && !a) || (K * N > 0 && !b)) {
    free(a);
    free(b);
    return -1;
  }
  oracle_widen(A, dtype, M * K, a);
  oracle_widen(B, dtype, K * N, b);
  if (nthreads < 1) nthreads = 1;
  if (nthreads > M) nthreads = (int)(M > 0 ? M : 1);
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  gemm_job* jobs = (gemm_job*)malloc(sizeof(gemm_job) * (size_t)nthreads);
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].M = M;
    jobs[t].N = N;
    jobs[t].K = K;
    jobs[t].A = a;
    jobs[t].B = b;
    jobs[t].C = C;
    jobs[t].r0 = M * t / nthreads;
    jobs[t].r1 = M * (t + 1) / nthreads;
    pthread_create(&th[t], NULL, gemm_rows, &jobs[t]);
  }
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  free(th);
  free(jobs);
  free(a);
  free(b);
  return 0;
}

int oracle_gemm_entries(int64_t M, int64_t N, int64_t K, const void* A,
                        const void* B, int dtype, int64_t n,
                        const int64_t* rows, const int64_t* cols, double* out) {
  for (int64_t t = 0; t < n; ++t) {
    const int64_t i = rows[t], j = cols[t];
    if (i < 0 || i >= M || j < 0 || j >= N) return -1;
    double s = 0.0;
    for (int64_t l = 0; l < K; ++l)
      s += widen_one(A, dtype, i * K + l) * widen_one(B, dtype, l * N + j);
    out[t] = s;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Configuration space (Eq.1–4), in the frozen canonical order.             */
/* ------------------------------------------------------------------------ */

static int64_t odd_part(int64_t D) {
  while (D > 0 && D % 2 == 0) D /= 2;
  return D;
}

static int is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

/* Is v an allowed value at this level? Level 0 carries the odd cofactor q. */
static int level_value_ok(int64_t v, int level, int64_t q) {
  if (v <= 0) return 0;
  if (level == 0) return v % q == 0 && is_pow2(v / q);
  return is_pow2(v);
}

/* Depth-first generation, smallest value first at every level, which yields
 * the tuples in lexicographic order of (f_0, f_1, ...). */
static void gen_tuples(int64_t rem, int level, int d, int64_t q, int64_t* cur,
                       int64_t* out, int64_t cap, int64_t* cnt) {
  if (level == d - 1) {
    if (!level_value_ok(rem, level, q)) return;
    cur[level] = rem;
    if (out && *cnt < cap)
      for (int i = 0; i < d; ++i) out[*cnt * d + i] = cur[i];
    ++*cnt;
    return;
  }
  for (int64_t f = (level == 0 ? q : 1); f <= rem; f *= 2) {
    if (rem % f != 0) break;
    cur[level] = f;
    gen_tuples(rem / f, level + 1, d, q, cur, out, cap, cnt);
  }
}

int64_t or_dim_tuples(int64_t D, int d, int64_t* out, int64_t cap) {
  if (D < 1 || d < 1 || d > OR_MAXD) return -1;
  int64_t cur[OR_MAXD];
  int64_t cnt = 0;
  gen_tuples(D, 0, d, odd_part(D), cur, out, cap, &cnt);
  return cnt;
}

static int64_t sp_ext(const or_space* sp, int x) {
  return x == 0 ? sp->M : (x == 1 ? sp->K : sp->N);
}

/* the domain of a space: extents 1..2^40, 1..4 levels, a known dtype,
 * a 0/1 MFMA coordinate flag and one of the two neighbour relations */
static int sp_ok(const or_space* sp) {
  if (!sp) return 0;
  for (int x = 0; x < 3; ++x)
    if (sp->d[x] < 1 || sp->d[x] > OR_MAXD || sp_ext(sp, x) < 1 ||
        sp_ext(sp, x) > ((int64_t)1 << 40))
      return 0;
  return (sp->dtype == OR_F32 || sp->dtype == OR_BF16) &&
         (sp->mfma_coord == 0 || sp->mfma_coord == 1) &&
         (sp->mode == OR_ADJACENT || sp->mode == OR_ANY_PAIR);
}

/* Per-dimension tuple tables, built fresh for each call (plain, not fast). */
typedef struct {
  int64_t n[3];
  int64_t* t[3];
} tables;

static int build_tables(const or_space* sp, tables* tb) {
  for (int x = 0; x < 3; ++x) {
    int64_t c = or_dim_tuples(sp_ext(sp, x), sp->d[x], NULL, 0);
    tb->n[x] = c;
    tb->t[x] = (int64_t*)malloc(sizeof(int64_t) * (size_t)(c * sp->d[x]));
    or_dim_tuples(sp_ext(sp, x), sp->d[x], tb->t[x], c);
  }
  return 0;
}

static void free_tables(tables* tb) {
  for (int x = 0; x < 3; ++x) free(tb->t[x]);
}

static int64_t find_tuple(const tables* tb, int x, int d, const int64_t* f) {
  for (int64_t r = 0; r < tb->n[x]; ++r) {
    int eq = 1;
    for (int i = 0; i < d; ++i)
      if (tb->t[x][r * d + i] != f[i]) eq = 0;
    if (eq) return r;
  }
  return -1;
}

int or_space_size(const or_space* sp, uint64_t* size) {
  if (!sp_ok(sp)) return -1;
  uint64_t s = 1;
  for (int x = 0; x < 3; ++x)
    s *= (uint64_t)or_dim_tuples(sp_ext(sp, x), sp->d[x], NULL, 0);
  if (sp->mfma_coord) s *= 2;
  *size = s;
  return 0;
}

static int rank_with(const or_space* sp, const tables* tb, const or_config* c,
                     uint64_t* rank) {
  int64_t r[3];
  for (int x = 0; x < 3; ++x) {
    r[x] = find_tuple(tb, x, sp->d[x], c->f[x]);
    if (r[x] < 0) return -1;
  }
  uint64_t nm = 1, im = 0;
  if (sp->mfma_coord) {
    if (c->mfma != 16 && c->mfma != 32) return -1;
    nm = 2;
    im = c->mfma == 32 ? 1 : 0;
  } else if (c->mfma != 0) {
    return -1;
  }
  /* order m, k, n, mfma: m slowest */
  *rank = (((uint64_t)r[0] * (uint64_t)tb->n[1] + (uint64_t)r[1]) *
               (uint64_t)tb->n[2] +
           (uint64_t)r[2]) *
              nm +
          im;
  return 0;
}

static void unrank_with(const or_space* sp, const tables* tb, uint64_t rank,
                        or_config* c) {
  memset(c, 0, sizeof(*c));
  uint64_t nm = sp->mfma_coord ? 2 : 1;
  uint64_t im = rank % nm;
  rank /= nm;
  uint64_t rn = rank % (uint64_t)tb->n[2];
  rank /= (uint64_t)tb->n[2];
  uint64_t rk = rank % (uint64_t)tb->n[1];
  uint64_t rm = rank / (uint64_t)tb->n[1];
  const uint64_t r[3] = {rm, rk, rn};
  for (int x = 0; x < 3; ++x)
    for (int i = 0; i < sp->d[x]; ++i)
      c->f[x][i] = tb->t[x][r[x] * (uint64_t)sp->d[x] + (uint64_t)i];
  c->mfma = sp->mfma_coord ? (im ? 32 : 16) : 0;
}

int or_rank(const or_space* sp, const or_config* c, uint64_t* rank) {
  if (!sp_ok(sp) || !c) return -1;
  tables tb;
  build_tables(sp, &tb);
  int rc = rank_with(sp, &tb, c, rank);
  free_tables(&tb);
  return rc;
}

int or_unrank(const or_space* sp, uint64_t rank, or_config* c) {
  uint64_t size;
  if (or_space_size(sp, &size) || rank >= size || !c) return -1;
  tables tb;
  build_tables(sp, &tb);
  unrank_with(sp, &tb, rank, c);
  free_tables(&tb);
  c->legit = or_legit(sp, c);
  return 0;
}

int or_member(const or_space* sp, const or_config* c) {
  if (!sp_ok(sp) || !c) return 0;
  for (int x = 0; x < 3; ++x) {
    const int64_t D = sp_ext(sp, x), q = odd_part(D);
    int64_t prod = 1;
    for (int i = 0; i < sp->d[x]; ++i) {
      if (!level_value_ok(c->f[x][i], i, q)) return 0;
      prod *= c->f[x][i];
      if (prod > D) return 0;
    }
    if (prod != D) return 0;
  }
  if (sp->mfma_coord) return c->mfma == 16 || c->mfma == 32;
  return c->mfma == 0;
}

/* ------------------------------------------------------------------------ */
/* Legitimacy J (Eq.5 and its footnote): membership plus the frozen          */
/* hardware predicate. Level → hardware mapping:                             */
/*   M, N: d=4 [grid, waves, rep, blk]; d=3 [grid, waves, blk];              */
/*         d=2 [grid, blk]; d=1 [grid].                                      */
/*   K:    d=4 [kLoop, kSplit, kSub, kBlk]; d=3 [kLoop, kSub, kBlk];         */
/*         d=2 [kLoop, kBlk]; d=1 [kLoop].                                   */
/* ------------------------------------------------------------------------ */

static void mn_levels(const int64_t* f, int d, int64_t* grid, int64_t* waves,
                      int64_t* rep, int64_t* blk) {
  *grid = f[0];
  *waves = 1;
  *rep = 1;
  *blk = 1;
  if (d == 2) {
    *blk = f[1];
  } else if (d == 3) {
    *waves = f[1];
    *blk = f[2];
  } else if (d == 4) {
    *waves = f[1];
    *rep = f[2];
    *blk = f[3];
  }
}

static void k_levels(const int64_t* f, int d, int64_t* loop, int64_t* split,
                     int64_t* sub, int64_t* blk) {
  *loop = f[0];
  *split = 1;
  *sub = 1;
  *blk = 1;
  if (d == 2) {
    *blk = f[1];
  } else if (d == 3) {
    *sub = f[1];
    *blk = f[2];
  } else if (d == 4) {
    *split = f[1];
    *sub = f[2];
    *blk = f[3];
  }
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int or_legit(const or_space* sp, const or_config* c) {
  if (!or_member(sp, c)) return 0;
  int64_t gM, wM, rM, bM, gN, wN, rN, bN, kL, kS, kU, kB;
  mn_levels(c->f[0], sp->d[0], &gM, &wM, &rM, &bM);
  mn_levels(c->f[2], sp->d[2], &gN, &wN, &rN, &bN);
  k_levels(c->f[1], sp->d[1], &kL, &kS, &kU, &kB);
  int64_t I;
  if (sp->mfma_coord)
    I = c->mfma;
  else
    I = (bM % 32 == 0 && bN % 32 == 0) ? 32 : 16;
  const int64_t TM = rM * ceil_div(bM, I);
  const int64_t TN = rN * ceil_div(bN, I);
  const int64_t acc = TM * TN * I * I / 64;
  const int64_t W = wM * wN;
  if (W > 16) return 0;
  if (acc > 256) return 0;
  if (acc + 96 > 512 / ceil_div(W, 4)) return 0;
  const int64_t BM = wM * rM * bM, BN = wN * rN * bN, BK = kU * kB;
  const int64_t elem = sp->dtype == OR_F32 ? 4 : 2;
  if ((BM * BK + BK * BN) * elem > 163840) return 0;
  if (gM * gN * 64 * W > 4294967295LL) return 0; /* work-items per dispatch dimension */
  if (kS > 65535) return 0;
  /* work-items of the whole dispatch (grid.x · grid.y · threads per group) */
  const int64_t items = gM * gN * kS * 64 * W;
  if (items > 4294967295LL) return 0;
  return 1;
}

int or_enumerate(const or_space* sp, uint64_t start, uint64_t count,
                 or_config* out) {
  uint64_t size;
  if (or_space_size(sp, &size) || start > size || count > size - start)
    return -1;
  tables tb;
  build_tables(sp, &tb);
  for (uint64_t i = 0; i < count; ++i) {
    unrank_with(sp, &tb, start + i, &out[i]);
    out[i].legit = or_legit(sp, &out[i]);
  }
  free_tables(&tb);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Actions (Eq.6), step (Eq.7), neighbours g(s) (Eq.9).                      */
/* ------------------------------------------------------------------------ */

int or_neighbours(const or_space* sp, const or_config* s, or_config* out,
                  int cap) {
  if (!or_member(sp, s)) return -1;
  tables tb;
  build_tables(sp, &tb);
  or_config buf[3 * OR_MAXD * OR_MAXD + 1];
  uint64_t rk[3 * OR_MAXD * OR_MAXD + 1];
  int n = 0;
  for (int x = 0; x < 3; ++x) {
    const int d = sp->d[x];
    for (int i = 0; i < d; ++i) {
      for (int j = 0; j < d; ++j) {
        if (i == j) continue;
        if (sp->mode == OR_ADJACENT && abs(i - j) != 1) continue;
        if (s->f[x][j] % 2 != 0) continue; /* s_x[j]/2 not a positive integer */
        or_config t = *s;
        t.f[x][i] = s->f[x][i] * 2;
        t.f[x][j] = s->f[x][j] / 2;
        if (!or_member(sp, &t)) continue;
        buf[n++] = t;
      }
    }
  }
  if (sp->mfma_coord) {
    or_config t = *s;
    t.mfma = s->mfma == 16 ? 32 : 16;
    buf[n++] = t;
  }
  for (int a = 0; a < n; ++a) rank_with(sp, &tb, &buf[a], &rk[a]);
  /* insertion sort by rank */
  for (int a = 1; a < n; ++a) {
    for (int b = a; b > 0 && rk[b - 1] > rk[b]; --b) {
      uint64_t tr = rk[b];
      rk[b] = rk[b - 1];
      rk[b - 1] = tr;
      or_config tc = buf[b];
      buf[b] = buf[b - 1];
      buf[b - 1] = tc;
    }
  }
  free_tables(&tb);
  if (n > cap) return -1;
  for (int a = 0; a < n; ++a) {
    out[a] = buf[a];
    out[a].legit = or_legit(sp, &out[a]);
  }
  return n;
}

/* ------------------------------------------------------------------------ */
/* SplitMix64 (Steele, Lea & Flood, OOPSLA 2014).                             */
/* ------------------------------------------------------------------------ */

uint64_t or_splitmix64_next(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* ------------------------------------------------------------------------ */
/* G-BFS (§4.2, Alg.1).                                                      */
/* ------------------------------------------------------------------------ */

/* cost(s) of one candidate (§4.2: its measured run time). A value that is
 * not a number is no measurement: the candidate counts as failed, +∞, as a
 * launch that fails does. */
static double measured(or_cost_fn cost, or_config* c, uint64_t rank, void* ctx) {
  const double v = cost(c, rank, ctx);
  return isnan(v) ? INFINITY : v;
}

int or_gbfs(const or_space* sp, const or_config* s0, int rho, int64_t budget,
            uint64_t seed, or_cost_fn cost, void* ctx, or_gbfs_result* res,
            uint64_t* log_ranks, double* log_costs, int64_t log_cap) {
  uint64_t size;
  if (or_space_size(sp, &size) || !s0 || !cost || !res) return -1;
  if (budget < 1 || rho < 1 || !or_legit(sp, s0)) return -1;
  tables tb;
  build_tables(sp, &tb);

  /* priority queue: unsorted arrays, minimum found by a full scan */
  double* qc = (double*)malloc(sizeof(double) * (size_t)(budget + 1));
  uint64_t* qr = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(budget + 1));
  int64_t qn = 0;
  /* visited list S_v: one bit per rank */
  unsigned char* vis = (unsigned char*)calloc((size_t)(size / 8 + 1), 1);
  uint64_t rng = seed;
  int64_t timed = 0, popped = 0;

  uint64_t r0;
  rank_with(sp, &tb, s0, &r0);
  or_config s0c = *s0;
  double c0 = measured(cost, &s0c, r0, ctx);
  if (timed < log_cap) {
    log_ranks[timed] = r0;
    log_costs[timed] = c0;
  }
  ++timed;
  vis[r0 / 8] |= (unsigned char)(1u << (r0 % 8));
  double cost_min = c0;
  uint64_t best = r0;
  if (!isinf(c0)) {
    qc[qn] = c0;
    qr[qn] = r0;
    ++qn;
  }

  while (qn > 0 && timed < budget) {
    /* pop the minimum (cost, rank) */
    int64_t m = 0;
    for (int64_t i = 1; i < qn; ++i)
      if (qc[i] < qc[m] || (qc[i] == qc[m] && qr[i] < qr[m])) m = i;
    const uint64_t rs = qr[m];
    qc[m] = qc[qn - 1];
    qr[m] = qr[qn - 1];
    --qn;
    ++popped;

    or_config s;
    unrank_with(sp, &tb, rs, &s);
    or_config g[3 * OR_MAXD * OR_MAXD + 1];
    const int n = or_neighbours(sp, &s, g, 3 * OR_MAXD * OR_MAXD + 1);
    const int take = rho < n ? rho : n;
    /* partial Fisher–Yates: the first `take` entries become the picks */
    for (int i = 0; i < take; ++i) {
      const int j = i + (int)(or_splitmix64_next(&rng) % (uint64_t)(n - i));
      or_config t = g[i];
      g[i] = g[j];
      g[j] = t;
    }
    for (int i = 0; i < take && timed < budget; ++i) {
      uint64_t r;
      rank_with(sp, &tb, &g[i], &r);
      if (!g[i].legit) continue;
      if (vis[r / 8] & (1u << (r % 8))) continue;
      const double c = measured(cost, &g[i], r, ctx);
      if (timed < log_cap) {
        log_ranks[timed] = r;
        log_costs[timed] = c;
      }
      ++timed;
      vis[r / 8] |= (unsigned char)(1u << (r % 8));
      if (!isinf(c)) {
        qc[qn] = c;
        qr[qn] = r;
        ++qn;
      }
      if (c < cost_min) {
        cost_min = c;
        best = r;
      }
    }
  }
  unrank_with(sp, &tb, best, &res->best);
  res->best.legit = or_legit(sp, &res->best);
  res->best_cost = cost_min;
  res->timed = timed;
  res->popped = popped;
  free(qc);
  free(qr);
  free(vis);
  free_tables(&tb);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Random search at an equal budget (§5 baseline).                          */
/* ------------------------------------------------------------------------ */

int or_random_search(const or_space* sp, int64_t budget, uint64_t seed, or_cost_fn cost,
                     void* ctx, or_gbfs_result* res, uint64_t* log_ranks, double* log_costs,
                     int64_t log_cap) {
  uint64_t size;
  if (or_space_size(sp, &size) || !cost || !res || budget < 1) return -1;
  tables tb;
  build_tables(sp, &tb);
  unsigned char* vis = (unsigned char*)calloc((size_t)(size / 8 + 1), 1);
  uint64_t rng = seed;
  int64_t timed = 0, draws = 0;
  const int64_t max_draws = 64 * budget + 1024;
  double cost_min = INFINITY;
  uint64_t best = 0;
  int have = 0;
  while (timed < budget && draws < max_draws) {
    const uint64_t r = or_splitmix64_next(&rng) % size;
    ++draws;
    or_config c;
    unrank_with(sp, &tb, r, &c);
    if (!or_legit(sp, &c)) continue;
    if (vis[r / 8] & (1u << (r % 8))) continue;
    vis[r / 8] |= (unsigned char)(1u << (r % 8));
    const double v = measured(cost, &c, r, ctx);
    if (timed < log_cap) {
      log_ranks[timed] = r;
      log_costs[timed] = v;
    }
    ++timed;
    if (!have || v < cost_min) {
      cost_min = v;
      best = r;
      have = 1;
    }
  }
  unrank_with(sp, &tb, best, &res->best);
  res->best.legit = or_legit(sp, &res->best);
  res->best_cost = cost_min;
  res->timed = timed;
  res->popped = draws;
  free(vis);
  free_tables(&tb);
  return 0;
}
/* ------------------------------------------------------------------------ */
/* N-A2C (§4.3, Alg.2).                                                      */
/*                                                                          */
/* The two networks are kept as flat parameter vectors,                     */
/*   actor  θa = [W1 (H×F) | b1 (H) | W2 (A×H) | b2 (A)],                   */
/*   critic θc = [U1 (H×F) | c1 (H) | u2 (H)   | c2],                       */
/* each one hidden tanh layer over the state features φ(s); the actor ends  */
/* in a softmax over the actions available in s, the critic in one linear   */
/* unit V(s). One training transition (s, a, r, s') takes the TD(0) error   */
/* δ = r + γ·V(s') − V(s) and the gradients ∇θa log π(a|s) and ∇θc V(s) at  */
/* the current parameters, then moves both vectors by (lr·δ)·∇.            */
/* ------------------------------------------------------------------------ */

#define NA_MAXF (3 * OR_MAXD + 1)
#define NA_MAXA (3 * OR_MAXD * (OR_MAXD - 1) + 1)
#define NA_MAXH 64

typedef struct {
  int F, A, H;        /* features, actions, hidden units */
  int n_actor, n_critic;
  int mv_x[NA_MAXA];  /* dimension of action a (m, k, n = 0, 1, 2; 3 = MFMA toggle) */
  int mv_up[NA_MAXA]; /* level whose factor doubles */
  int mv_dn[NA_MAXA]; /* level whose factor halves */
  int E[3];           /* power-of-two exponent of each extent */
  int64_t q[3];       /* odd cofactor of each extent */
} na_shape;

/* offsets inside θa and θc */
#define OFF_W1(z) 0
#define OFF_B1(z) ((z)->H * (z)->F)
#define OFF_W2(z) (OFF_B1(z) + (z)->H)
#define OFF_B2(z) (OFF_W2(z) + (z)->A * (z)->H)
#define OFF_U1(z) 0
#define OFF_C1(z) ((z)->H * (z)->F)
#define OFF_U2(z) (OFF_C1(z) + (z)->H)
#define OFF_C2(z) (OFF_U2(z) + (z)->H)

static int exp2_of(int64_t v) {
  int e = 0;
  for (; v > 1; v /= 2) ++e;
  return e;
}

/* Action list 𝒜 (Eq.6): per dimension every ordered level pair the mode
 * allows, then the MFMA toggle when the space has that coordinate. */
static void na_shape_of(const or_space* sp, int H, na_shape* z) {
  memset(z, 0, sizeof(*z));
  for (int x = 0; x < 3; ++x)
    for (int up = 0; up < sp->d[x]; ++up)
      for (int dn = 0; dn < sp->d[x]; ++dn) {
        const int adjacent = up - dn == 1 || dn - up == 1;
        if (up == dn || (sp->mode == OR_ADJACENT && !adjacent)) continue;
        z->mv_x[z->A] = x;
        z->mv_up[z->A] = up;
        z->mv_dn[z->A] = dn;
        z->A++;
      }
  if (sp->mfma_coord) {
    z->mv_x[z->A] = 3;
    z->A++;
  }
  z->F = sp->d[0] + sp->d[1] + sp->d[2] + (sp->mfma_coord ? 1 : 0);
  z->H = H;
  z->n_actor = H * z->F + H + z->A * H + z->A;
  z->n_critic = H * z->F + H + H + 1;
  const int64_t ext[3] = {sp->M, sp->K, sp->N};
  for (int x = 0; x < 3; ++x) {
    z->q[x] = odd_part(ext[x]);
    z->E[x] = exp2_of(ext[x] / z->q[x]);
  }
}

/* φ(s): each level's exponent as a share of its dimension's E (level 0
 * without the odd cofactor), then 1 for MFMA 32. */
static void na_phi(const or_space* sp, const na_shape* z, const or_config* s, double* phi) {
  int f = 0;
  for (int x = 0; x < 3; ++x)
    for (int lvl = 0; lvl < sp->d[x]; ++lvl) {
      const int64_t v = lvl == 0 ? s->f[x][0] / z->q[x] : s->f[x][lvl];
      phi[f++] = z->E[x] == 0 ? 0.0 : (double)exp2_of(v) / (double)z->E[x];
    }
  if (sp->mfma_coord) phi[f++] = s->mfma == 32 ? 1.0 : 0.0;
}

/* a is available in s when the halved factor is even (the result stays a
 * positive integer, Eq.6); the toggle always is. */
static int na_ok(const na_shape* z, const or_config* s, int a) {
  if (z->mv_x[a] == 3) return 1;
  return s->f[z->mv_x[a]][z->mv_dn[a]] % 2 == 0;
}

static void na_ok_all(const na_shape* z, const or_config* s, int* ok) {
  for (int a = 0; a < z->A; ++a) ok[a] = na_ok(z, s, a);
}

/* s' = step(s, a), Eq.7 */
static or_config na_move(const na_shape* z, const or_config* s, int a) {
  or_config t = *s;
  if (z->mv_x[a] == 3) {
    t.mfma = s->mfma == 16 ? 32 : 16;
  } else {
    t.f[z->mv_x[a]][z->mv_up[a]] *= 2;
    t.f[z->mv_x[a]][z->mv_dn[a]] /= 2;
  }
  return t;
}

/* the action leading back: same dimension, the two levels swapped */
static int na_back(const na_shape* z, int a) {
  if (z->mv_x[a] == 3) return a;
  for (int b = 0; b < z->A; ++b)
    if (z->mv_x[b] == z->mv_x[a] && z->mv_up[b] == z->mv_dn[a] && z->mv_dn[b] == z->mv_up[a])
      return b;
  return -1;
}

/* y[o] = tanh(b[o] + Σ_i W[o][i]·x[i]) */
static void tanh_layer(const double* W, const double* b, int n_out, int n_in, const double* x,
                       double* y) {
  for (int o = 0; o < n_out; ++o) {
    double acc = b[o];
    for (int i = 0; i < n_in; ++i) acc += W[o * n_in + i] * x[i];
    y[o] = tanh(acc);
  }
}

/* π(·|s) with hidden activations h; π = 0 on unavailable actions */
static void actor_pi(const na_shape* z, const double* th, const double* phi, const int* ok,
                     double* h, double* pi) {
  tanh_layer(th + OFF_W1(z), th + OFF_B1(z), z->H, z->F, phi, h);
  const double* W2 = th + OFF_W2(z);
  const double* b2 = th + OFF_B2(z);
  double top = -INFINITY;
  for (int a = 0; a < z->A; ++a) {
    pi[a] = 0.0;
    if (!ok[a]) continue;
    double logit = b2[a];
    for (int k = 0; k < z->H; ++k) logit += W2[a * z->H + k] * h[k];
    pi[a] = logit;
    if (logit > top) top = logit;
  }
  double norm = 0.0;
  for (int a = 0; a < z->A; ++a)
    if (ok[a]) {
      pi[a] = exp(pi[a] - top);
      norm += pi[a];
    }
  for (int a = 0; a < z->A; ++a)
    if (ok[a]) pi[a] /= norm;
}

/* V(s) with hidden activations g */
static double critic_v(const na_shape* z, const double* th, const double* phi, double* g) {
  tanh_layer(th + OFF_U1(z), th + OFF_C1(z), z->H, z->F, phi, g);
  const double* u2 = th + OFF_U2(z);
  double v = th[OFF_C2(z)];
  for (int k = 0; k < z->H; ++k) v += u2[k] * g[k];
  return v;
}

/* ∇θa log π(a|s). With e_b = [b = a] − π_b over the available b:
 * ∂/∂b2_b = e_b, ∂/∂W2_bk = e_b·h_k, ∂/∂b1_k = (Σ_b e_b·W2_bk)(1 − h_k²),
 * ∂/∂W1_kf = ∂/∂b1_k · φ_f. */
static void actor_grad(const na_shape* z, const double* th, const double* phi, const int* ok,
                       int a, double* grad) {
  double h[NA_MAXH], pi[NA_MAXA], e[NA_MAXA];
  actor_pi(z, th, phi, ok, h, pi);
  for (int b = 0; b < z->A; ++b) e[b] = ok[b] ? (b == a ? 1.0 : 0.0) - pi[b] : 0.0;
  const double* W2 = th + OFF_W2(z);
  for (int k = 0; k < z->H; ++k) {
    double back = 0.0;
    for (int b = 0; b < z->A; ++b)
      if (ok[b]) back += e[b] * W2[b * z->H + k];
    const double dz = back * (1.0 - h[k] * h[k]);
    for (int f = 0; f < z->F; ++f) grad[OFF_W1(z) + k * z->F + f] = dz * phi[f];
    grad[OFF_B1(z) + k] = dz;
  }
  for (int b = 0; b < z->A; ++b) {
    for (int k = 0; k < z->H; ++k) grad[OFF_W2(z) + b * z->H + k] = e[b] * h[k];
    grad[OFF_B2(z) + b] = e[b];
  }
}

/* ∇θc V(s): ∂/∂c2 = 1, ∂/∂u2_k = g_k, ∂/∂c1_k = u2_k(1 − g_k²),
 * ∂/∂U1_kf = ∂/∂c1_k · φ_f. */
static void critic_grad(const na_shape* z, const double* th, const double* phi, double* grad) {
  double g[NA_MAXH];
  critic_v(z, th, phi, g);
  const double* u2 = th + OFF_U2(z);
  for (int k = 0; k < z->H; ++k) {
    const double dz = u2[k] * (1.0 - g[k] * g[k]);
    for (int f = 0; f < z->F; ++f) grad[OFF_U1(z) + k * z->F + f] = dz * phi[f];
    grad[OFF_C1(z) + k] = dz;
    grad[OFF_U2(z) + k] = g[k];
  }
  grad[OFF_C2(z)] = 1.0;
}

typedef struct { /* a transition (s, a, r, s') as the networks see it */
  double phi[NA_MAXF], phi2[NA_MAXF];
  int ok[NA_MAXA];
  int a;
  double r;
} na_sample;

/* One advantage actor-critic update on one transition. */
static void td_update(const na_shape* z, double* tha, double* thc, const na_sample* t,
                      double gamma, double lr) {
  double g[NA_MAXH], ga[NA_MAXH * NA_MAXF + NA_MAXH + NA_MAXA * NA_MAXH + NA_MAXA];
  double gc[NA_MAXH * NA_MAXF + 2 * NA_MAXH + 1];
  const double v_next = critic_v(z, thc, t->phi2, g);
  const double v_now = critic_v(z, thc, t->phi, g);
  const double delta = t->r + gamma * v_next - v_now;
  actor_grad(z, tha, t->phi, t->ok, t->a, ga);
  critic_grad(z, thc, t->phi, gc);
  const double step = lr * delta;
  for (int k = 0; k < z->n_critic; ++k) thc[k] += step * gc[k];
  for (int k = 0; k < z->n_actor; ++k) tha[k] += step * ga[k];
}

/* Initial parameters: U(−1/√fan_in, 1/√fan_in) from SplitMix64(seed ^
 * 0xA2C0A2C0A2C0A2C0), drawn in the order W1, W2, U1, u2; biases 0. */
static double unit_draw(uint64_t* st) {
  return (double)(or_splitmix64_next(st) >> 11) * (1.0 / 9007199254740992.0);
}

static void na_init_params(const na_shape* z, uint64_t seed, double* tha, double* thc) {
  memset(tha, 0, sizeof(double) * (size_t)z->n_actor);
  memset(thc, 0, sizeof(double) * (size_t)z->n_critic);
  uint64_t st = seed ^ 0xA2C0A2C0A2C0A2C0ULL;
  const double lim_f = 1.0 / sqrt((double)z->F), lim_h = 1.0 / sqrt((double)z->H);
  for (int k = 0; k < z->H * z->F; ++k) tha[OFF_W1(z) + k] = (2.0 * unit_draw(&st) - 1.0) * lim_f;
  for (int k = 0; k < z->A * z->H; ++k) tha[OFF_W2(z) + k] = (2.0 * unit_draw(&st) - 1.0) * lim_h;
  for (int k = 0; k < z->H * z->F; ++k) thc[OFF_U1(z) + k] = (2.0 * unit_draw(&st) - 1.0) * lim_f;
  for (int k = 0; k < z->H; ++k) thc[OFF_U2(z) + k] = (2.0 * unit_draw(&st) - 1.0) * lim_h;
}

/* r(s, a) of a transition into s'. Default (§4.1): 1/cost(s'), so a failed
 * s' (cost +∞) earns 0. Variant: log(cost(s)/cost(s')) clipped to ±clip. */
static double na_r(int mode, double cost_s, double cost_s2, double clip) {
  if (mode == 0) return 1.0 / cost_s2;
  if (isinf(cost_s2)) return isinf(cost_s) ? 0.0 : -clip;
  if (isinf(cost_s)) return clip;
  const double r = log(cost_s / cost_s2);
  return r > clip ? clip : (r < -clip ? -clip : r);
}

/* H_v: rank → cost, open addressing */
typedef struct {
  uint64_t* key;
  double* cost;
  unsigned char* full;
  uint64_t cap;
} na_table;

static uint64_t na_find(const na_table* t, uint64_t r) {
  uint64_t i = (r * 0x9E3779B97F4A7C15ULL) % t->cap;
  while (t->full[i] && t->key[i] != r) i = (i + 1) % t->cap;
  return i;
}

static int params_bad(const or_na2c_params* p) {
  return p->T < 1 || p->B < 1 || p->H < 1 || p->H > NA_MAXH || p->mem < 1 || p->max_walks < 1 ||
         (p->reward != 0 && p->reward != 1) || (p->eps_halving != 0 && p->eps_halving != 1);
}

/* a ∈ 𝒜 drawn for one walk step in s: with probability ε from π(·|s)
 * (inverse CDF over the available actions in list order), else uniformly
 * among the available ones; -1, drawing nothing, when no action is
 * available in s (the walk ends there) */
static int na_pick(const or_space* sp, const na_shape* z, const double* tha, const or_config* s,
                   double eps, uint64_t* rng) {
  int ok[NA_MAXA];
  na_ok_all(z, s, ok);
  int n_ok = 0;
  for (int b = 0; b < z->A; ++b) n_ok += ok[b];
  if (n_ok == 0) return -1;
  if (unit_draw(rng) < eps) {
    double phi[NA_MAXF], h[NA_MAXH], pi[NA_MAXA];
    na_phi(sp, z, s, phi);
    actor_pi(z, tha, phi, ok, h, pi);
    const double u = unit_draw(rng);
    int pick = -1;
    double cdf = 0.0;
    for (int b = 0; b < z->A; ++b) {
      if (!ok[b]) continue;
      pick = b; /* the last available action if rounding leaves u ≥ Σπ */
      cdf += pi[b];
      if (u < cdf) break;
    }
    return pick;
  }
  uint64_t k = or_splitmix64_next(rng) % (uint64_t)n_ok;
  for (int b = 0; b < z->A; ++b)
    if (ok[b] && k-- == 0) return b;
  return -1;
}

int or_na2c(const or_space* sp, const or_config* s0, const or_na2c_params* prm,
            int64_t budget, uint64_t seed, or_cost_fn cost, void* ctx, or_gbfs_result* res,
            uint64_t* log_ranks, double* log_costs, int64_t log_cap,
            or_na2c_transition* trace, int64_t trace_cap, int64_t* trace_n) {
  uint64_t size;
  if (or_space_size(sp, &size) || !s0 || !prm || !cost || !res) return -1;
  if (budget < 1 || params_bad(prm) || !or_legit(sp, s0)) return -1;
  tables tb;
  build_tables(sp, &tb);
  na_shape z;
  na_shape_of(sp, prm->H, &z);
  double* tha = (double*)malloc(sizeof(double) * (size_t)z.n_actor);
  double* thc = (double*)malloc(sizeof(double) * (size_t)z.n_critic);
  na_table hv;
  hv.cap = (uint64_t)budget * 4 + 17;
  hv.key = (uint64_t*)calloc(hv.cap, sizeof(uint64_t));
  hv.cost = (double*)calloc(hv.cap, sizeof(double));
  hv.full = (unsigned char*)calloc(hv.cap, 1);
  na_sample* M = (na_sample*)calloc((size_t)prm->mem, sizeof(na_sample));
  or_config* batch = (or_config*)calloc((size_t)prm->B, sizeof(or_config));
  uint64_t* batch_r = (uint64_t*)calloc((size_t)prm->B, sizeof(uint64_t));
  if (!tha || !thc || !hv.key || !hv.cost || !hv.full || !M || !batch || !batch_r) {
    free(tha), free(thc), free(hv.key), free(hv.cost), free(hv.full), free(M), free(batch),
        free(batch_r);
    free_tables(&tb);
    return -1;
  }
  na_init_params(&z, seed, tha, thc);
  int64_t m_len = 0, m_old = 0; /* FIFO 𝓜: m_len entries from m_old */
  int64_t n_trace = 0;
  uint64_t rng = seed;
  int64_t timed = 0, episodes = 0;

  /* s0 is timed first and is the first centre */
  uint64_t r0;
  rank_with(sp, &tb, s0, &r0);
  or_config first = *s0;
  const double c0 = measured(cost, &first, r0, ctx);
  if (timed < log_cap) log_ranks[timed] = r0, log_costs[timed] = c0;
  ++timed;
  uint64_t slot = na_find(&hv, r0);
  hv.full[slot] = 1, hv.key[slot] = r0, hv.cost[slot] = c0;
  double cost_min = c0;
  uint64_t best = r0;
  or_config centre = *s0;

  int walk = prm->T;    /* 𝒯: grows by one after an episode that collects nothing */
  double eps = prm->eps; /* halves with such an episode when eps_halving is set */
  while (timed < budget) {
    /* B_collect: walks of `walk` steps from the centre until B states that
     * are legitimate, not in H_v and not yet collected are found */
    int nb = 0;
    for (int w = 0; w < prm->max_walks && nb < prm->B; ++w) {
      or_config s = centre;
      for (int t = 0; t < walk; ++t) {
        const int a = na_pick(sp, &z, tha, &s, eps, &rng);
        if (a < 0) break; /* a dead end: no move leaves s */
        const or_config s2 = na_move(&z, &s, a);
        if (or_legit(sp, &s2) && nb < prm->B) {
          uint64_t r2;
          rank_with(sp, &tb, &s2, &r2);
          int seen = hv.full[na_find(&hv, r2)];
          for (int b = 0; b < nb; ++b) seen = seen || batch_r[b] == r2;
          if (!seen) batch[nb] = s2, batch_r[nb] = r2, ++nb;
        }
        s = s2;
      }
    }
    ++episodes;
    if (nb == 0) {
      if (walk >= prm->T + 8) break;
      ++walk;
      if (prm->eps_halving) eps *= 0.5;
      continue;
    }
    for (int b = 0; b < nb && timed < budget; ++b) {
      or_config sb = batch[b];
      const double c = measured(cost, &sb, batch_r[b], ctx);
      if (timed < log_cap) log_ranks[timed] = batch_r[b], log_costs[timed] = c;
      ++timed;
      if (c < cost_min) { /* new s*: the next episode walks from it */
        cost_min = c;
        best = batch_r[b];
        centre = batch[b];
        walk = prm->T;
        eps = prm->eps;
      }
      slot = na_find(&hv, batch_r[b]);
      hv.full[slot] = 1, hv.key[slot] = batch_r[b], hv.cost[slot] = c;
      /* 𝓜 gains (s, a, r, s') for every timed s with step(s, a) = s':
       * s = step(s', a') over the available a', and a leads back */
      for (int ap = 0; ap < z.A; ++ap) {
        if (!na_ok(&z, &batch[b], ap)) continue;
        const or_config s = na_move(&z, &batch[b], ap);
        if (!or_member(sp, &s)) continue;
        uint64_t rs;
        rank_with(sp, &tb, &s, &rs);
        const uint64_t ps = na_find(&hv, rs);
        if (!hv.full[ps]) continue;
        na_sample smp;
        memset(&smp, 0, sizeof(smp));
        na_phi(sp, &z, &s, smp.phi);
        na_phi(sp, &z, &batch[b], smp.phi2);
        na_ok_all(&z, &s, smp.ok);
        smp.a = na_back(&z, ap);
        smp.r = na_r(prm->reward, hv.cost[ps], c, prm->r_clip);
        if (trace && n_trace < trace_cap) {
          trace[n_trace].s = rs;
          trace[n_trace].s2 = batch_r[b];
          trace[n_trace].a = smp.a;
          trace[n_trace].pad = 0;
          trace[n_trace].r = smp.r;
        }
        ++n_trace;
        if (m_len < prm->mem) {
          M[(m_old + m_len) % prm->mem] = smp;
          ++m_len;
        } else { /* full: the oldest entry is replaced */
          M[m_old] = smp;
          m_old = (m_old + 1) % prm->mem;
        }
      }
      /* train on 𝓜, oldest transition first */
      for (int64_t k = 0; k < m_len; ++k)
        td_update(&z, tha, thc, &M[(m_old + k) % prm->mem], prm->gamma, prm->lr);
    }
  }
  unrank_with(sp, &tb, best, &res->best);
  res->best.legit = or_legit(sp, &res->best);
  res->best_cost = cost_min;
  res->timed = timed;
  res->popped = episodes;
  if (trace_n) *trace_n = n_trace;
  free(tha), free(thc), free(hv.key), free(hv.cost), free(hv.full), free(M), free(batch),
      free(batch_r);
  free_tables(&tb);
  return 0;
}

int or_na2c_probe(const or_space* sp, const or_na2c_params* prm, uint64_t seed,
                  const or_config* s, int a, const double* actor_params,
                  const double* critic_params, double* pi, double* v,
                  double* g_actor, double* g_critic, int64_t* n_actor, int64_t* n_critic) {
  uint64_t size;
  if (or_space_size(sp, &size) || !prm || prm->H < 1 || prm->H > NA_MAXH) return -1;
  na_shape z;
  na_shape_of(sp, prm->H, &z);
  if (n_actor) *n_actor = z.n_actor;
  if (n_critic) *n_critic = z.n_critic;
  if (!s || !pi || !v || !g_actor || !g_critic || a < 0 || a >= z.A) return 0;
  double* tha = (double*)malloc(sizeof(double) * (size_t)z.n_actor);
  double* thc = (double*)malloc(sizeof(double) * (size_t)z.n_critic);
  if (!tha || !thc) {
    free(tha), free(thc);
    return -1;
  }
  na_init_params(&z, seed, tha, thc);
  if (actor_params) memcpy(tha, actor_params, sizeof(double) * (size_t)z.n_actor);
  if (critic_params) memcpy(thc, critic_params, sizeof(double) * (size_t)z.n_critic);
  double phi[NA_MAXF], h[NA_MAXH], g[NA_MAXH];
  int ok[NA_MAXA];
  na_phi(sp, &z, s, phi);
  na_ok_all(&z, s, ok);
  actor_pi(&z, tha, phi, ok, h, pi);
  *v = critic_v(&z, thc, phi, g);
  actor_grad(&z, tha, phi, ok, a, g_actor);
  critic_grad(&z, thc, phi, g_critic);
  free(tha), free(thc);
  return 0;
}

int or_na2c_train(const or_space* sp, const or_na2c_params* prm, const or_config* s,
                  const int* a, const double* r, const or_config* s2, int64_t n,
                  double* actor_params, double* critic_params) {
  uint64_t size;
  if (or_space_size(sp, &size) || !prm || prm->H < 1 || prm->H > NA_MAXH || n < 0 ||
      (n > 0 && (!s || !a || !r || !s2)) || !actor_params || !critic_params)
    return -1;
  na_shape z;
  na_shape_of(sp, prm->H, &z);
  for (int64_t t = 0; t < n; ++t) {
    na_sample smp;
    memset(&smp, 0, sizeof(smp));
    if (a[t] < 0 || a[t] >= z.A || !na_ok(&z, &s[t], a[t])) return -1;
    na_phi(sp, &z, &s[t], smp.phi);
    na_phi(sp, &z, &s2[t], smp.phi2);
    na_ok_all(&z, &s[t], smp.ok);
    smp.a = a[t];
    smp.r = r[t];
    td_update(&z, actor_params, critic_params, &smp, prm->gamma, prm->lr);
  }
  return 0;
}
