/*
 * oracle.h — plain CPU reference for the tuned-GEMM path.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. It shares no code,
 * header or helper with the GPU library; everything here is written from the
 * paper and from the frozen definitions of the configuration space.
 *
 *   - oracle_gemm*: C = A·B in fp64 by the plain three-loop definition (§3.2),
 *     on the exact fp64 widening of the fp32 or bf16 input bytes.
 *   - or_*: the configuration space of Eq.1–4 (power-of-two factors, odd
 *     cofactor at level 0), the state legitimacy bit J of Eq.5, the action set
 *     of Eq.6 / neighbour list of Eq.9, the G-BFS of Alg.1 (§4.2), the
 *     equal-budget random search (§5) and N-A2C (§4.3, Alg.2) with its
 *     training step exposed for pinning (or_na2c_probe, or_na2c_train).
 *
 * Parity pins: see tests/test_oracle_*.py. The legitimacy predicate beyond
 * membership (the hardware constraints) has no paper value: it is pinned by
 * hand-worked cases, by every J=1 configuration launching on the GPU, and in
 * one direction by the compiled kernels themselves (every configuration it
 * admits fits the register allocation, largest workgroup and LDS that the
 * gfx950 code objects record); where exactly it draws the line is a design
 * choice with nothing outside to pin it to.
 */
#ifndef GEMM_ORACLE_H
#define GEMM_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OR_F32 = 0, OR_BF16 = 1 };
enum { OR_ADJACENT = 0, OR_ANY_PAIR = 1 };
#define OR_MAXD 4

typedef struct {
  int64_t M, N, K;
  int32_t d[3];        /* levels per dimension, order m, k, n */
  int32_t dtype;       /* OR_F32 / OR_BF16 */
  int32_t mfma_coord;  /* 1: MFMA size {16,32} is a coordinate */
  int32_t mode;        /* OR_ADJACENT / OR_ANY_PAIR */
} or_space;

typedef struct {
  int64_t f[3][OR_MAXD]; /* f[0]: m levels, f[1]: k levels, f[2]: n levels */
  int32_t mfma;          /* 16/32 with the coordinate, 0 without */
  int32_t legit;         /* J, filled by the functions that return configs */
} or_config;

/* fp64 GEMM, C (M×N, row-major doubles) = A (M×K) · B (K×N), row-major input
 * bytes of the given dtype. Threads over row blocks. Returns 0. */
int oracle_gemm(int64_t M, int64_t N, int64_t K, const void* A, const void* B,
                int dtype, double* C, int nthreads);
/* C*[rows[t]][cols[t]] for t < n (sampled entries at any size). */
int oracle_gemm_entries(int64_t M, int64_t N, int64_t K, const void* A,
                        const void* B, int dtype, int64_t n,
                        const int64_t* rows, const int64_t* cols, double* out);
/* Exact widening of input bytes to fp64 (n elements). */
int oracle_widen(const void* src, int dtype, int64_t n, double* dst);

/* Tuples of one dimension in canonical (lexicographic) order; returns the
 * count, writes count*d values when out != NULL and count <= cap. */
int64_t or_dim_tuples(int64_t D, int d, int64_t* out, int64_t cap);
int or_space_size(const or_space* sp, uint64_t* size);
int or_rank(const or_space* sp, const or_config* c, uint64_t* rank);
int or_unrank(const or_space* sp, uint64_t rank, or_config* c);
int or_member(const or_space* sp, const or_config* c);
int or_legit(const or_space* sp, const or_config* c);
/* Configurations with ranks [start, start+count) written to out. */
int or_enumerate(const or_space* sp, uint64_t start, uint64_t count,
                 or_config* out);
/* Neighbour list g(s) (Eq.9) in ascending rank; returns the count or -1 if
 * cap is too small. Each entry carries its J. */
int or_neighbours(const or_space* sp, const or_config* s, or_config* out,
                  int cap);

uint64_t or_splitmix64_next(uint64_t* state);

/* cost of a candidate; +∞ marks a failure, and a NaN is taken as +∞ */
typedef double (*or_cost_fn)(const or_config* c, uint64_t rank, void* ctx);
typedef struct {
  or_config best;
  double best_cost;
  int64_t timed;
  int64_t popped;
} or_gbfs_result;
/* G-BFS, Alg.1. log_ranks/log_costs (cap log_cap) receive every timed
 * configuration in timing order. Returns 0, or -1 on a bad argument
 * (s0 illegitimate, budget < 1, rho < 1). */
int or_gbfs(const or_space* sp, const or_config* s0, int rho, int64_t budget,
            uint64_t seed, or_cost_fn cost, void* ctx, or_gbfs_result* res,
            uint64_t* log_ranks, double* log_costs, int64_t log_cap);

/* Random search at an equal budget (the baseline the paper's tuners are
 * compared with, §5): ranks are drawn uniformly, r = splitmix64(seed) mod |ξ|;
 * illegitimate and already-timed draws are skipped (no budget), every other
 * draw is timed until `budget` configurations have been timed or
 * 64·budget + 1024 draws were made; the best is the first minimum cost.
 * res->popped holds the number of draws. Returns 0, or -1 on a bad argument
 * (budget < 1). When nothing was timed, res->best is the configuration of
 * rank 0 and res->best_cost is +inf. */
int or_random_search(const or_space* sp, int64_t budget, uint64_t seed, or_cost_fn cost,
                     void* ctx, or_gbfs_result* res, uint64_t* log_ranks, double* log_costs,
                     int64_t log_cap);

/* N-A2C (§4.3, Alg.2) with the readings listed with the library's
 * implementation: action list (per dimension, ordered level pairs the mode
 * allows, then the MFMA toggle), features e_i/E per level (+ MFMA bit),
 * one-hidden-layer tanh actor (softmax over the available actions) and critic,
 * ε = probability of following π, T-step walks from the current centre until
 * B unvisited legitimate states are collected (at most max_walks walks; an
 * episode that collects nothing lengthens the walks by one step, up to T + 8
 * steps, then the search stops; with eps_halving it also halves ε; a new best
 * resets both), each timed state storing every transition from an
 * already-timed neighbour into the FIFO memory M, and one SGD pass over M
 * after every timing (critic: semi-gradient TD(0); actor: δ·∇log π).
 * Reward: reward = 0 gives §4.1's r(s, a) = 1/cost(s'); reward = 1 the
 * variant log(cost(s)/cost(s')) clipped to ±r_clip. Randomness:
 * SplitMix64(seed) for the walk, SplitMix64(seed ^ 0xA2C0A2C0A2C0A2C0) for
 * the initial weights. res->popped holds the number of episodes. trace
 * (optional, trace_cap entries) receives every transition stored into M, in
 * storing order; *trace_n their total count. Returns 0, or -1 on a bad
 * argument. */
typedef struct {
  int32_t T, B, H, mem, max_walks;
  int32_t reward;       /* 0: 1/cost(s') (§4.1); 1: clipped log ratio */
  int32_t eps_halving;  /* 1: halve ε after an episode that collects nothing */
  double eps, gamma, lr, r_clip;
} or_na2c_params;
typedef struct {
  uint64_t s, s2;  /* ranks of s and s' = step(s, a) */
  int32_t a, pad;
  double r;        /* r(s, a) */
} or_na2c_transition;
int or_na2c(const or_space* sp, const or_config* s0, const or_na2c_params* prm,
            int64_t budget, uint64_t seed, or_cost_fn cost, void* ctx, or_gbfs_result* res,
            uint64_t* log_ranks, double* log_costs, int64_t log_cap,
            or_na2c_transition* trace, int64_t trace_cap, int64_t* trace_n);
/* The actor's and critic's outputs and gradients at one state, for the
 * weights of or_na2c's initialisation or for the given flattened parameters
 * (for gradient checks): pi[A], v, and the flattened gradients of
 * log π(a|s) (actor) and V(s) (critic) with respect to every parameter, in
 * the order W1, b1, W2, b2 (actor) and U1, c1, u2, c2 (critic). Returns the
 * parameter counts through n_actor and n_critic when the buffers are NULL. */
int or_na2c_probe(const or_space* sp, const or_na2c_params* prm, uint64_t seed,
                  const or_config* s, int a, const double* actor_params,
                  const double* critic_params, double* pi, double* v,
                  double* g_actor, double* g_critic, int64_t* n_actor, int64_t* n_critic);
/* The training step or_na2c applies, on caller-given parameters (in/out, the
 * probe's layout): transitions t = 0 … n−1 (s[t], a[t], r[t], s2[t]) in
 * order, each one TD(0) actor-critic update with prm->gamma and prm->lr.
 * Returns 0, or -1 on a bad argument (a[t] not available in s[t]). */
int or_na2c_train(const or_space* sp, const or_na2c_params* prm, const or_config* s,
                  const int* a, const double* r, const or_config* s2, int64_t n,
                  double* actor_params, double* critic_params);

#ifdef __cplusplus
}
#endif
#endif
