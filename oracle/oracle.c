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
