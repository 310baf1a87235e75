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

static int sp_ok(const or_space* sp) {
  if (!sp) return 0;
  for (int x = 0; x < 3; ++x)
    if (sp->d[x] < 1 || sp->d[x] > OR_MAXD || sp_ext(sp, x) < 1) return 0;
  return 1;
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
  double c0 = cost(&s0c, r0, ctx);
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
      const double c = cost(&g[i], r, ctx);
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
    const double v = cost(&c, r, ctx);
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
/* ------------------------------------------------------------------------ */

typedef struct { /* one action of the fixed list: f[x][i] *= 2, f[x][j] /= 2, or the toggle */
  int x, i, j, toggle;
} na_action;

typedef struct {
  int F, A, H;
  na_action act[3 * OR_MAXD * OR_MAXD + 1];
  int E[3];
  int64_t q[3];
  /* actor */
  double *W1, *b1, *W2, *b2;
  /* critic */
  double *U1, *c1, *u2, c2;
} na_net;

static void na_actions(const or_space* sp, na_net* n) {
  n->A = 0;
  for (int x = 0; x < 3; ++x)
    for (int i = 0; i < sp->d[x]; ++i)
      for (int j = 0; j < sp->d[x]; ++j) {
        if (i == j) continue;
        if (sp->mode == OR_ADJACENT && abs(i - j) != 1) continue;
        na_action a = {x, i, j, 0};
        n->act[n->A++] = a;
      }
  if (sp->mfma_coord) {
    na_action a = {0, 0, 0, 1};
    n->act[n->A++] = a;
  }
}

static int na_log2(int64_t v) {
  int e = 0;
  while (v > 1) {
    v >>= 1;
    ++e;
  }
  return e;
}

/* φ(s): exponent share of every level (level 0 without the odd cofactor),
 * then the MFMA bit. */
static void na_features(const or_space* sp, const na_net* n, const or_config* s, double* phi) {
  int k = 0;
  for (int x = 0; x < 3; ++x)
    for (int i = 0; i < sp->d[x]; ++i) {
      const int64_t v = i == 0 ? s->f[x][0] / n->q[x] : s->f[x][i];
      phi[k++] = n->E[x] ? (double)na_log2(v) / (double)n->E[x] : 0.0;
    }
  if (sp->mfma_coord) phi[k++] = s->mfma == 32 ? 1.0 : 0.0;
}

static int na_available(const na_net* n, const or_config* s, int a) {
  const na_action* ac = &n->act[a];
  if (ac->toggle) return 1;
  return s->f[ac->x][ac->j] % 2 == 0;
}

static or_config na_step(const na_net* n, const or_config* s, int a) {
  or_config t = *s;
  const na_action* ac = &n->act[a];
  if (ac->toggle) {
    t.mfma = s->mfma == 16 ? 32 : 16;
  } else {
    t.f[ac->x][ac->i] = s->f[ac->x][ac->i] * 2;
    t.f[ac->x][ac->j] = s->f[ac->x][ac->j] / 2;
  }
  return t;
}

/* the action that undoes a (from step(s, a) back to s) */
static int na_inverse(const na_net* n, int a) {
  const na_action* ac = &n->act[a];
  if (ac->toggle) return a;
  for (int b = 0; b < n->A; ++b)
    if (!n->act[b].toggle && n->act[b].x == ac->x && n->act[b].i == ac->j && n->act[b].j == ac->i)
      return b;
  return -1;
}

static double na_uniform(uint64_t* st) {
  return (double)(or_splitmix64_next(st) >> 11) * (1.0 / 9007199254740992.0);
}

static int na_alloc(const or_space* sp, const or_na2c_params* prm, uint64_t seed, na_net* n) {
  memset(n, 0, sizeof(*n));
  na_actions(sp, n);
  n->F = sp->d[0] + sp->d[1] + sp->d[2] + (sp->mfma_coord ? 1 : 0);
  n->H = prm->H;
  const int64_t ext[3] = {sp->M, sp->K, sp->N};
  for (int x = 0; x < 3; ++x) {
    n->q[x] = odd_part(ext[x]);
    n->E[x] = na_log2(ext[x] / n->q[x]);
  }
  const int F = n->F, A = n->A, H = n->H;
  n->W1 = (double*)calloc((size_t)(H * F), sizeof(double));
  n->b1 = (double*)calloc((size_t)H, sizeof(double));
  n->W2 = (double*)calloc((size_t)(A * H), sizeof(double));
  n->b2 = (double*)calloc((size_t)A, sizeof(double));
  n->U1 = (double*)calloc((size_t)(H * F), sizeof(double));
  n->c1 = (double*)calloc((size_t)H, sizeof(double));
  n->u2 = (double*)calloc((size_t)H, sizeof(double));
  if (!n->W1 || !n->b1 || !n->W2 || !n->b2 || !n->U1 || !n->c1 || !n->u2) return -1;
  /* weights U(−1/√fan_in, 1/√fan_in) in the order W1, W2, U1, u2; biases 0 */
  uint64_t ws = seed ^ 0xA2C0A2C0A2C0A2C0ULL;
  const double bF = 1.0 / sqrt((double)F), bH = 1.0 / sqrt((double)H);
  for (int k = 0; k < H * F; ++k) n->W1[k] = (2.0 * na_uniform(&ws) - 1.0) * bF;
  for (int k = 0; k < A * H; ++k) n->W2[k] = (2.0 * na_uniform(&ws) - 1.0) * bH;
  for (int k = 0; k < H * F; ++k) n->U1[k] = (2.0 * na_uniform(&ws) - 1.0) * bF;
  for (int k = 0; k < H; ++k) n->u2[k] = (2.0 * na_uniform(&ws) - 1.0) * bH;
  n->c2 = 0.0;
  return 0;
}

static void na_free(na_net* n) {
  free(n->W1);
  free(n->b1);
  free(n->W2);
  free(n->b2);
  free(n->U1);
  free(n->c1);
  free(n->u2);
}

/* actor forward: hidden h[H], π over the available actions (0 elsewhere) */
static void na_actor(const na_net* n, const double* phi, const int* avail, double* h,
                     double* pi) {
  for (int k = 0; k < n->H; ++k) {
    double z = n->b1[k];
    for (int f = 0; f < n->F; ++f) z += n->W1[k * n->F + f] * phi[f];
    h[k] = tanh(z);
  }
  double zmax = -INFINITY;
  for (int a = 0; a < n->A; ++a) {
    if (!avail[a]) {
      pi[a] = 0.0;
      continue;
    }
    double z = n->b2[a];
    for (int k = 0; k < n->H; ++k) z += n->W2[a * n->H + k] * h[k];
    pi[a] = z;
    if (z > zmax) zmax = z;
  }
  double sum = 0.0;
  for (int a = 0; a < n->A; ++a)
    if (avail[a]) {
      pi[a] = exp(pi[a] - zmax);
      sum += pi[a];
    }
  for (int a = 0; a < n->A; ++a)
    if (avail[a]) pi[a] /= sum;
}

static double na_critic(const na_net* n, const double* phi, double* g) {
  double v = n->c2;
  for (int k = 0; k < n->H; ++k) {
    double z = n->c1[k];
    for (int f = 0; f < n->F; ++f) z += n->U1[k * n->F + f] * phi[f];
    g[k] = tanh(z);
    v += n->u2[k] * g[k];
  }
  return v;
}

typedef struct {
  double phi[3 * OR_MAXD + 1], phi2[3 * OR_MAXD + 1];
  int avail[3 * OR_MAXD * OR_MAXD + 1];
  int a;
  double r;
} na_trans;

/* one transition: δ from the current critic, then the critic's and the
 * actor's updates (both with gradients at the pre-update weights) */
static void na_train_one(na_net* n, const na_trans* t, double gamma, double lr, double* h,
                         double* g, double* pi, double* dh) {
  double g2[64];
  const double v2 = na_critic(n, t->phi2, g2);
  const double v = na_critic(n, t->phi, g);
  const double delta = t->r + gamma * v2 - v;
  /* critic: θ += lr·δ·∂V(s)/∂θ */
  for (int k = 0; k < n->H; ++k) {
    const double back = n->u2[k] * (1.0 - g[k] * g[k]);
    for (int f = 0; f < n->F; ++f) n->U1[k * n->F + f] += lr * delta * back * t->phi[f];
    n->c1[k] += lr * delta * back;
  }
  for (int k = 0; k < n->H; ++k) n->u2[k] += lr * delta * g[k];
  n->c2 += lr * delta;
  /* actor: θ += lr·δ·∇ log π(a|s) */
  na_actor(n, t->phi, t->avail, h, pi);
  for (int k = 0; k < n->H; ++k) {
    double s = 0.0;
    for (int b = 0; b < n->A; ++b) {
      if (!t->avail[b]) continue;
      const double e = (b == t->a ? 1.0 : 0.0) - pi[b];
      s += e * n->W2[b * n->H + k];
    }
    dh[k] = s * (1.0 - h[k] * h[k]);
  }
  for (int b = 0; b < n->A; ++b) {
    if (!t->avail[b]) continue;
    const double e = (b == t->a ? 1.0 : 0.0) - pi[b];
    for (int k = 0; k < n->H; ++k) n->W2[b * n->H + k] += lr * delta * e * h[k];
    n->b2[b] += lr * delta * e;
  }
  for (int k = 0; k < n->H; ++k) {
    for (int f = 0; f < n->F; ++f) n->W1[k * n->F + f] += lr * delta * dh[k] * t->phi[f];
    n->b1[k] += lr * delta * dh[k];
  }
}

/* visited hashtable H_v: rank → cost (open addressing) */
typedef struct {
  uint64_t* key;
  double* val;
  unsigned char* used;
  uint64_t cap;
} na_map;

static uint64_t na_slot(const na_map* m, uint64_t r) {
  uint64_t h = (r * 0x9E3779B97F4A7C15ULL) % m->cap;
  while (m->used[h] && m->key[h] != r) h = (h + 1) % m->cap;
  return h;
}

static double na_reward(double cs, double cs2, double clip) {
  if (isinf(cs2)) return isinf(cs) ? 0.0 : -clip;
  if (isinf(cs)) return clip;
  double r = log(cs / cs2);
  if (r > clip) r = clip;
  if (r < -clip) r = -clip;
  return r;
}

int or_na2c(const or_space* sp, const or_config* s0, const or_na2c_params* prm,
            int64_t budget, uint64_t seed, or_cost_fn cost, void* ctx, or_gbfs_result* res,
            uint64_t* log_ranks, double* log_costs, int64_t log_cap) {
  uint64_t size;
  if (or_space_size(sp, &size) || !s0 || !prm || !cost || !res) return -1;
  if (budget < 1 || prm->T < 1 || prm->B < 1 || prm->H < 1 || prm->H > 64 || prm->mem < 1 ||
      prm->max_walks < 1 || !or_legit(sp, s0))
    return -1;
  tables tb;
  build_tables(sp, &tb);
  na_net n;
  if (na_alloc(sp, prm, seed, &n)) return -1;
  na_map hv;
  hv.cap = (uint64_t)budget * 4 + 17;
  hv.key = (uint64_t*)calloc(hv.cap, sizeof(uint64_t));
  hv.val = (double*)calloc(hv.cap, sizeof(double));
  hv.used = (unsigned char*)calloc(hv.cap, 1);
  na_trans* mem = (na_trans*)calloc((size_t)prm->mem, sizeof(na_trans));
  or_config* coll = (or_config*)calloc((size_t)prm->B, sizeof(or_config));
  uint64_t* coll_r = (uint64_t*)calloc((size_t)prm->B, sizeof(uint64_t));
  double h[64], g[64], dh[64], pi[3 * OR_MAXD * OR_MAXD + 1];
  int64_t mem_n = 0, mem_head = 0; /* FIFO: oldest at mem_head */
  uint64_t rng = seed;
  int64_t timed = 0, episodes = 0;

  uint64_t r0;
  rank_with(sp, &tb, s0, &r0);
  or_config c0cfg = *s0;
  const double c0 = cost(&c0cfg, r0, ctx);
  if (timed < log_cap) {
    log_ranks[timed] = r0;
    log_costs[timed] = c0;
  }
  ++timed;
  {
    const uint64_t sl = na_slot(&hv, r0);
    hv.used[sl] = 1;
    hv.key[sl] = r0;
    hv.val[sl] = c0;
  }
  double cost_min = c0;
  uint64_t best = r0;
  or_config center = *s0;

  int steps = prm->T;      /* walk length; grows while episodes collect nothing */
  double eps_cur = prm->eps; /* share of policy steps; halves with each such episode */
  while (timed < budget) {
    /* collect B unvisited legitimate states by walks of `steps` steps from
     * the centre */
    int nb = 0;
    for (int w = 0; w < prm->max_walks && nb < prm->B; ++w) {
      or_config s = center;
      for (int t = 0; t < steps; ++t) {
        double phi[3 * OR_MAXD + 1];
        int avail[3 * OR_MAXD * OR_MAXD + 1], navail = 0;
        for (int a = 0; a < n.A; ++a) {
          avail[a] = na_available(&n, &s, a);
          navail += avail[a];
        }
        int a = -1;
        if (na_uniform(&rng) < eps_cur) {
          na_features(sp, &n, &s, phi);
          na_actor(&n, phi, avail, h, pi);
          const double u = na_uniform(&rng);
          double cum = 0.0;
          for (int b = 0; b < n.A; ++b) {
            if (!avail[b]) continue;
            a = b; /* the last available action if rounding leaves u ≥ Σπ */
            cum += pi[b];
            if (u < cum) break;
          }
        } else {
          int k = (int)(or_splitmix64_next(&rng) % (uint64_t)navail);
          for (int b = 0; b < n.A; ++b)
            if (avail[b] && k-- == 0) {
              a = b;
              break;
            }
        }
        const or_config s2 = na_step(&n, &s, a);
        if (or_legit(sp, &s2)) {
          uint64_t r2;
          rank_with(sp, &tb, &s2, &r2);
          int dup = hv.used[na_slot(&hv, r2)];
          for (int b = 0; b < nb && !dup; ++b) dup = coll_r[b] == r2;
          if (!dup && nb < prm->B) {
            coll[nb] = s2;
            coll_r[nb] = r2;
            ++nb;
          }
        }
        s = s2;
      }
    }
    ++episodes;
    if (nb == 0) {
      /* nothing new within `steps` of the centre: walk one step further
       * (§4.3 lets the exploration step grow) and halve the share of policy
       * steps, up to T + 8 */
      if (steps >= prm->T + 8) break;
      ++steps;
      eps_cur *= 0.5;
      continue;
    }
    for (int b = 0; b < nb && timed < budget; ++b) {
      or_config sc = coll[b];
      const double c = cost(&sc, coll_r[b], ctx);
      if (timed < log_cap) {
        log_ranks[timed] = coll_r[b];
        log_costs[timed] = c;
      }
      ++timed;
      if (c < cost_min) {
        cost_min = c;
        best = coll_r[b];
        center = coll[b];
        steps = prm->T; /* a new centre: back to T-step walks and ε */
        eps_cur = prm->eps;
      }
      const uint64_t sl = na_slot(&hv, coll_r[b]);
      hv.used[sl] = 1;
      hv.key[sl] = coll_r[b];
      hv.val[sl] = c;
      /* every (s, a) with step(s, a) = s' and s already timed */
      for (int bb = 0; bb < n.A; ++bb) {
        if (!na_available(&n, &coll[b], bb)) continue;
        const or_config p = na_step(&n, &coll[b], bb);
        if (!or_member(sp, &p)) continue;
        uint64_t rp;
        rank_with(sp, &tb, &p, &rp);
        const uint64_t ps = na_slot(&hv, rp);
        if (!hv.used[ps]) continue;
        na_trans tr;
        memset(&tr, 0, sizeof(tr));
        na_features(sp, &n, &p, tr.phi);
        na_features(sp, &n, &coll[b], tr.phi2);
        for (int a = 0; a < n.A; ++a) tr.avail[a] = na_available(&n, &p, a);
        tr.a = na_inverse(&n, bb);
        tr.r = na_reward(hv.val[ps], c, prm->r_clip);
        if (mem_n < prm->mem) {
          mem[(mem_head + mem_n) % prm->mem] = tr;
          ++mem_n;
        } else {
          mem[mem_head] = tr;
          mem_head = (mem_head + 1) % prm->mem;
        }
      }
      /* one pass over M, oldest first */
      for (int64_t k = 0; k < mem_n; ++k)
        na_train_one(&n, &mem[(mem_head + k) % prm->mem], prm->gamma, prm->lr, h, g, pi, dh);
    }
  }
  unrank_with(sp, &tb, best, &res->best);
  res->best.legit = or_legit(sp, &res->best);
  res->best_cost = cost_min;
  res->timed = timed;
  res->popped = episodes;
  free(hv.key);
  free(hv.val);
  free(hv.used);
  free(mem);
  free(coll);
  free(coll_r);
  na_free(&n);
  free_tables(&tb);
  return 0;
}

int or_na2c_probe(const or_space* sp, const or_na2c_params* prm, uint64_t seed,
                  const or_config* s, int a, const double* actor_params,
                  const double* critic_params, double* pi, double* v,
                  double* g_actor, double* g_critic, int64_t* n_actor, int64_t* n_critic) {
  uint64_t size;
  if (or_space_size(sp, &size) || !prm || prm->H < 1 || prm->H > 64) return -1;
  na_net n;
  if (na_alloc(sp, prm, seed, &n)) return -1;
  const int F = n.F, A = n.A, H = n.H;
  const int64_t na = (int64_t)H * F + H + (int64_t)A * H + A, nc = (int64_t)H * F + H + H + 1;
  if (n_actor) *n_actor = na;
  if (n_critic) *n_critic = nc;
  if (!s || !pi || !v || !g_actor || !g_critic || a < 0 || a >= A) {
    na_free(&n);
    return 0;
  }
  if (actor_params) {
    int64_t k = 0;
    for (int t = 0; t < H * F; ++t) n.W1[t] = actor_params[k++];
    for (int t = 0; t < H; ++t) n.b1[t] = actor_params[k++];
    for (int t = 0; t < A * H; ++t) n.W2[t] = actor_params[k++];
    for (int t = 0; t < A; ++t) n.b2[t] = actor_params[k++];
  }
  if (critic_params) {
    int64_t k = 0;
    for (int t = 0; t < H * F; ++t) n.U1[t] = critic_params[k++];
    for (int t = 0; t < H; ++t) n.c1[t] = critic_params[k++];
    for (int t = 0; t < H; ++t) n.u2[t] = critic_params[k++];
    n.c2 = critic_params[k++];
  }
  double phi[3 * OR_MAXD + 1], h[64], g[64];
  int avail[3 * OR_MAXD * OR_MAXD + 1];
  na_features(sp, &n, s, phi);
  for (int b = 0; b < A; ++b) avail[b] = na_available(&n, s, b);
  na_actor(&n, phi, avail, h, pi);
  *v = na_critic(&n, phi, g);
  /* ∇ log π(a|s): the update direction na_train_one applies (δ = 1, lr = 1) */
  int64_t k = 0;
  double dh[64];
  for (int q = 0; q < H; ++q) {
    double sacc = 0.0;
    for (int b = 0; b < A; ++b) {
      if (!avail[b]) continue;
      sacc += ((b == a ? 1.0 : 0.0) - pi[b]) * n.W2[b * H + q];
    }
    dh[q] = sacc * (1.0 - h[q] * h[q]);
  }
  for (int q = 0; q < H; ++q)
    for (int f = 0; f < F; ++f) g_actor[k++] = dh[q] * phi[f];
  for (int q = 0; q < H; ++q) g_actor[k++] = dh[q];
  for (int b = 0; b < A; ++b)
    for (int q = 0; q < H; ++q)
      g_actor[k++] = avail[b] ? ((b == a ? 1.0 : 0.0) - pi[b]) * h[q] : 0.0;
  for (int b = 0; b < A; ++b) g_actor[k++] = avail[b] ? (b == a ? 1.0 : 0.0) - pi[b] : 0.0;
  k = 0;
  for (int q = 0; q < H; ++q)
    for (int f = 0; f < F; ++f) g_critic[k++] = n.u2[q] * (1.0 - g[q] * g[q]) * phi[f];
  for (int q = 0; q < H; ++q) g_critic[k++] = n.u2[q] * (1.0 - g[q] * g[q]);
  for (int q = 0; q < H; ++q) g_critic[k++] = g[q];
  g_critic[k++] = 1.0;
  na_free(&n);
  return 0;
}
