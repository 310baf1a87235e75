/*
 * gemmtune.h — C ABI of libgemmtune: a tiling-parameterised GEMM kernel
 * family for AMD Instinct MI355X (gfx950) and the Greedy Best-First Search
 * (G-BFS) that tunes its configuration on the GPU.
 *
 * Paper: Compiler-Level Matrix Multiplication Optimization for Deep Learning
 * (arxiv 1909.10616).
 *
 * Conventions for every entry point:
 *   - Return value: GT_OK (0) or a negative gt_status; gt_last_error() gives a
 *     thread-local message for the last failure on the calling thread.
 *   - The caller owns every buffer passed in (host and device). The library
 *     owns (a) one 2-word device buffer per GPU for the output comparison
 *     (gt_compare and the searches' checks), allocated on its first use on
 *     that GPU and kept until gt_shutdown(), and (b) the M·N fp32 reference
 *     product of a search whose caller passes no c_ref (freed before the
 *     search returns). Kernel attributes (the dynamic LDS limit) are set once
 *     per kernel and GPU and hold no memory.
 *   - Space functions (gt_space_size … neighbours) are pure host code, need no
 *     GPU and are thread-safe.
 *   - gemm_run, gt_measure, gt_reference_gemm, gt_compare and the searches may
 *     be called from several host threads at once: each works on the caller's
 *     buffers and stream, and the comparisons take the per-GPU result buffer
 *     in turn. Timings (gt_measure, each candidate of a search) take turns
 *     per GPU, so concurrent searches do not inflate each other's costs
 *     (other work on the GPU is not held back). The exception is
 *     gt_compare_noalloc, whose calls on one GPU share one scratch array and
 *     must not overlap.
 *   - Dimension order is m, k, n everywhere, as in the paper's configuration
 *     (§3.3 Eq.1) and state (§4.1 Eq.5).
 */
#ifndef GEMMTUNE_H
#define GEMMTUNE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GT_MAXD 4

typedef enum {
  GT_OK = 0,
  GT_EINVAL = -1,      /* invalid argument (null pointer, bad enum, bad size) */
  GT_EDIMS = -2,       /* configuration products do not match M, N, K */
  GT_EILLEGIT = -3,    /* configuration is not legitimate (J = 0) */
  GT_EHIP = -4,        /* a HIP runtime call failed */
  GT_ENOKERNEL = -5,   /* no kernel instantiation for this configuration */
  GT_ETIMEOUT = -6,    /* reserved, not returned: a search always times s0
                          before it checks its time limit */
  GT_ESMALL = -7       /* output buffer too small; *n_out holds the count */
} gt_status;

typedef enum { GT_F32 = 0, GT_BF16 = 1 } gt_dtype;

/* Operand-layout flag OR-ed into every `dtype` argument (and gt_space.dtype):
 * A is passed as W = Aᵀ, a K×M row-major array (element (m, k) at
 * A[k·M + m]), so that the product is C = WᵀB — the perceptron layer
 * Y = WᵀX of §5 with W ∈ R^(k×m), X ∈ R^(k×n). Without the flag A is M×K
 * row-major. B and C are unaffected. */
#define GT_A_KMAJOR 16
typedef enum { GT_ADJACENT = 0, GT_ANY_PAIR = 1 } gt_neighbour_mode;

/* Configuration space ξ = ξ_m × ξ_k × ξ_n (§3.3 Eq.1–4).
 * Each extent D = q·2^E (q odd) is split into d ordered factors, level 0
 * outermost: level 0 holds q·2^e0, levels ≥ 1 hold powers of two.
 * mfma_coord = 1 adds the MFMA instruction size {16, 32} as a coordinate.
 * neighbour_mode: GT_ADJACENT moves a factor of 2 between adjacent levels;
 * GT_ANY_PAIR between any two levels (§4.1 Eq.6 as printed). */
typedef struct gt_space {
  int64_t M, N, K;         /* 1..2^40; a space outside these ranges is GT_EINVAL */
  int32_t d_m, d_k, d_n;   /* 1..GT_MAXD */
  int32_t dtype;           /* gt_dtype of A and B (| GT_A_KMAJOR); C is fp32 */
  int32_t mfma_coord;      /* 0 or 1 */
  int32_t neighbour_mode;  /* gt_neighbour_mode */
} gt_space;

/* One configuration / state s = [s_m, s_k, s_n, J] (§4.1 Eq.5).
 * Level meaning (outermost first):
 *   M, N   d=4 [grid, waves, rep, blk]  d=3 [grid, waves, blk]
 *          d=2 [grid, blk]               d=1 [grid]
 *   K      d=4 [kLoop, kSplit, kSub, kBlk]  d=3 [kLoop, kSub, kBlk]
 *          d=2 [kLoop, kBlk]                d=1 [kLoop]
 * grid = workgroups along the dimension, waves = wavefronts per workgroup
 * along it, rep = MFMA blocks per wavefront, blk = block extent; kLoop =
 * sequential LDS stages, kSplit = workgroups along K, kSub = sub-steps per
 * stage, kBlk = K elements per sub-step. Unused entries are 0. */
typedef struct gt_config {
  int32_t d_m, d_k, d_n;   /* level counts of the space it belongs to */
  int32_t mfma;            /* 16 or 32 with the coordinate; 0 = derived */
  int64_t m[GT_MAXD];
  int64_t k[GT_MAXD];
  int64_t n[GT_MAXD];
  int32_t legit;           /* J, written by the functions that return configs */
  int32_t reserved;
} gt_config;

/* |ξ| = Π_x C(E_x + d_x − 1, d_x − 1) · (2 if mfma_coord). */
int gt_space_size(const gt_space* sp, uint64_t* size);

/* Configurations of ranks [start_rank, start_rank + n) in canonical order
 * (m slowest, then k, n, MFMA 16 before 32; each dimension lexicographic on
 * its factors), n = min(cap, |ξ| − start_rank). out: caller-owned, cap
 * entries. Each entry carries J. */
int enumerate_configs(const gt_space* sp, uint64_t start_rank, gt_config* out,
                      uint64_t cap, uint64_t* n_out);

/* Rank ↔ configuration bijection with [0, |ξ|). */
int config_rank(const gt_space* sp, const gt_config* cfg, uint64_t* rank);
int config_unrank(const gt_space* sp, uint64_t rank, gt_config* cfg);

/* Legitimacy J (§4.1 Eq.5 and its footnote): membership in ξ plus the
 * hardware predicate — waves ≤ 16; accumulator registers
 * acc = TM·TN·I²/64 ≤ 256 and acc + 96 ≤ 512/⌈waves/4⌉; LDS stage
 * (BM·BK + BK·BN)·sizeof(in) ≤ 163840 B; grid_M·grid_N·64·waves ≤ 2^32 − 1;
 * kSplit ≤ 65535; the whole launch grid_M·grid_N·kSplit·64·waves ≤ 2^32 − 1
 * work-items. A non-member gives *J = 0 and GT_OK. */
int config_legit(const gt_space* sp, const gt_config* cfg, int* J);

/* Neighbour list g(s) = [step(s, a) for a in A] (§4.1 Eq.6, Eq.7, Eq.9) in
 * ascending rank, illegitimate entries included with legit = 0 (Alg.1
 * filters them). out: caller-owned, cap entries; too small → GT_ESMALL with
 * the needed count in *n_out. */
int neighbours(const gt_space* sp, const gt_config* s, gt_config* out, int cap,
               int* n_out);

/* C = A·B on the GPU with the kernel the configuration lowers to (§3.2, the
 * operator being tuned). A: M×K row-major (K×M with GT_A_KMAJOR in dtype),
 * B: K×N row-major (dtype), C: M×N row-major fp32, all device pointers.
 * stream: hipStream_t (NULL = default). Asynchronous; C is overwritten. The
 * configuration's products must equal M, K, N and it must be legitimate in
 * the space (M, N, K, cfg->d_*, dtype, mfma_coord = cfg->mfma != 0). With a
 * K split (the second K level above 1) two kernels go on the stream: one
 * clears C, then every slice adds its partial product with fp32 atomics, so
 * the order of those adds, and the last bits of C, can differ from launch to
 * launch (results on exactly representable inputs do not). Those are the
 * GPU's own float atomics, which act on ordinary device memory
 * (hipMalloc, torch CUDA tensors): C must not be fine-grained or
 * host-mapped memory (hipMallocManaged, hipHostMalloc) for such
 * configurations. Errors: GT_EINVAL (null pointer, unknown dtype or a space
 * make_space refuses), GT_EDIMS (products differ from M, K, N), GT_EILLEGIT
 * (J = 0), GT_ENOKERNEL, GT_EHIP (launch failure); nothing is launched
 * unless the result is GT_OK or GT_EHIP. */
int gemm_run(const gt_config* cfg, const void* A, const void* B, void* C,
             int64_t M, int64_t N, int64_t K, int dtype, void* stream);

/* Cost of one configuration as the search measures it (§4.2 "test", §5 mean
 * of 10 runs): `warmup` launches (the first one timed on its own), then
 * `runs` back-to-back launches between two HIP events; *mean_ms = elapsed /
 * runs. If the first warm-up launch exceeds abort_ms (> 0), timing stops
 * there, *mean_ms = its time and *aborted = 1. Synchronises the stream.
 * Timings on one GPU take turns (see the conventions). Errors: those of
 * gemm_run, plus GT_EINVAL for a null output pointer. */
int gt_measure(const gt_config* cfg, const void* A, const void* B, void* C,
               int64_t M, int64_t N, int64_t K, int dtype, void* stream,
               int warmup, int runs, double abort_ms, double* mean_ms,
               double* first_ms, int* aborted);

/* Plain (non-MFMA, one thread per output, any M and N) GPU product in fp32,
 * used by the search as the reference its candidates are checked against.
 * Same operands and layouts as gemm_run (dtype may carry GT_A_KMAJOR); C is
 * caller-owned M·N fp32. Asynchronous. Errors: GT_EINVAL (null pointer,
 * M, N or K below 1, unknown dtype), GT_EHIP (launch failure). */
int gt_reference_gemm(const void* A, const void* B, void* C, int64_t M,
                      int64_t N, int64_t K, int dtype, void* stream);

/* Normwise relative difference max|C − R| / max|R| of two fp32 device
 * arrays of n elements, computed on the GPU (0 when both are all zero, +inf
 * when only R is, NaN when a difference is NaN). Synchronises the stream.
 * Errors: GT_EINVAL (null pointer, n < 1), GT_EHIP. */
int gt_compare(const void* C, const void* R, int64_t n, void* stream,
               double* rel);

/* gt_compare for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same result, with the two result words held in a static 256-byte
 * device array of the library (one copy per GPU, kept until the process
 * ends) instead of the buffer gt_compare allocates on first use. No
 * hipMalloc, hipFree or other allocating call is made; n is not limited (the
 * kernels reduce any n into the two words). Calls that overlap on one GPU
 * race on that array; each call clears it before use. Synchronises the
 * stream. GT_EINVAL for null pointers or n < 1, GT_EHIP for a HIP failure. */
int gt_compare_noalloc(const void* C, const void* R, int64_t n, void* stream,
                       double* rel);

/* How a configuration lowers (for reports and tests): the kernel path, tile
 * and launch gemm_run would use for cfg at M×N×K. Errors: those of gemm_run
 * before its launch (GT_EINVAL, GT_EDIMS, GT_EILLEGIT, GT_ENOKERNEL). */
typedef struct gt_kernel_info {
  int32_t I, IK;             /* MFMA instruction size and its K */
  int32_t TM, TN;            /* MFMA tiles per wavefront */
  int32_t fast;              /* 1: vectorised swizzled-LDS path */
  int32_t dl;                /* 1: fast path with direct global->LDS loads */
  int32_t ring;              /* LDS ring stages of the direct-load path */
  int32_t waves;             /* wavefronts per workgroup */
  int32_t BM, BN, BK;        /* workgroup tile and LDS stage depth */
  int32_t dbuf;              /* LDS double buffering */
  int32_t acc_regs;          /* accumulator registers per lane */
  int32_t lds_bytes;         /* dynamic LDS per workgroup */
  int64_t grid_x, grid_y;    /* launch grid (tiles, K splits) */
} gt_kernel_info;
int gt_lower(const gt_config* cfg, int64_t M, int64_t N, int64_t K, int dtype,
             gt_kernel_info* info);

/* ---- G-BFS (§4.2, Alg.1) ---------------------------------------------- */

/* Per-timed-configuration log record. status: 0 ok, 1 early abort,
 * 2 launch failure (cost +inf), 3 output mismatch (cost +inf). cost_ms is
 * the mean of the timed runs (§5); median, minimum and sample standard
 * deviation of the individual runs beside it (an early abort: the warm-up
 * time, deviation 0; a callback cost: the cost itself). */
typedef struct gt_log_entry {
  uint64_t rank;
  double cost_ms;
  double first_ms;
  double rel_err;
  int32_t status;
  int32_t reserved;
  double median_ms;
  double min_ms;
  double stdev_ms;
} gt_log_entry;

/* Synthetic cost (the CPU "fake backend"): returns the cost of cfg, +inf for
 * a failure. A NaN is taken as +inf (logged as such, counted in `failed`). */
typedef double (*gt_cost_fn)(const gt_config* cfg, uint64_t rank, void* ctx);

typedef struct gt_tune_opts {
  const gt_config* s0;   /* NULL: the paper's start state [D,1,…,1], MFMA 16 */
  int32_t rho;           /* neighbours sampled per pop (ρ); default 5 */
  int32_t runs;          /* timed runs per configuration; default 10 */
  int32_t warmup;        /* untimed-for-cost warm-up launches; default 1 */
  int32_t check;         /* 1: compare every timed output with the reference */
  int64_t budget;        /* configurations timed, s0 included; ≥ 1 */
  double t_max_s;        /* search time limit in seconds; 0 = none */
  uint64_t seed;         /* SplitMix64 seed of the ρ-sampling */
  double max_run_ms;     /* early abort when the warm-up exceeds this; 250 */
  double abort_factor;   /* … or exceeds abort_factor · cost_min; 50 */
  /* GPU mode (cost callback NULL): device buffers and stream. */
  const void* A;
  const void* B;
  void* C;
  void* c_ref;           /* M·N fp32 scratch for the reference; NULL: allocated */
  void* stream;
  gt_log_entry* log;     /* optional, caller-owned, log_cap entries */
  int64_t log_cap;
  double progress_s;     /* > 0: a progress line on stderr at most this often */
  int32_t trace_fd;      /* ≥ 0: before timing a candidate, one line naming it
                            (index, rank, factors) is written to this file
                            descriptor with write(2), so that the candidate
                            in flight is on record if the process dies; -1 none */
  int32_t reserved2;
} gt_tune_opts;

typedef struct gt_tune_result {
  gt_config best;        /* s* */
  uint64_t best_rank;
  double best_cost;      /* cost_min (ms in GPU mode) */
  int64_t timed;         /* configurations timed (≤ budget) */
  int64_t popped;        /* G-BFS: queue pops; random search: draws; N-A2C: episodes */
  int64_t skipped_illegit;
  int64_t skipped_visited;
  int64_t failed;        /* timed with cost +inf */
  double wall_s;
  int32_t stop_reason;   /* 0 budget, 1 queue empty, 2 time limit, 3 draws exhausted */
  int32_t reserved;
  double eval_s;         /* wall time spent timing candidates (launches, waits,
                            output checks; callback time in callback mode) */
  double device_s;       /* GPU time of the timed launches as the events
                            measured them (warm-ups included); 0 with a callback */
} gt_tune_result;

/* Fills the defaults listed in gt_tune_opts (budget 1000, seed 0, trace_fd -1).
 * opts: caller-owned. GT_EINVAL if opts is NULL. */
int gt_tune_opts_init(gt_tune_opts* opts);

/* G-BFS over the space. cost == NULL times gemm_run on the GPU with
 * opts->A/B/C/stream (and checks outputs when opts->check); otherwise
 * cost(cfg, rank, ctx) is called for every timed configuration. A candidate
 * that fails to launch or mismatches is logged with cost +inf and the search
 * goes on; a device error that outlives the failing call (a kernel fault)
 * ends the search with GT_EHIP, *out holding the search up to that point and
 * gt_last_error() naming the configuration that was being timed. Errors
 * before anything is timed: GT_EINVAL (null opts or out, budget or rho below
 * 1, a space make_space refuses, GPU mode without A, B or C, host memory
 * exhausted), GT_EDIMS (s0 not a member of the space), GT_EILLEGIT (J(s0) =
 * 0), GT_EHIP (the reference product could not be allocated or computed).
 * opts, its log buffer and out are caller-owned; the reference product made
 * when opts->c_ref is NULL is allocated and freed within the call. */
int tune_gbfs(const gt_space* sp, const gt_tune_opts* opts, gt_cost_fn cost,
              void* ctx, gt_tune_result* out);

/* Random search at an equal budget, the baseline the paper's tuners are
 * compared with (§5): ranks drawn uniformly, r = SplitMix64(opts->seed) mod
 * |ξ|; illegitimate and already-timed draws are skipped without cost; every
 * other draw is timed (GPU or callback exactly as in tune_gbfs) until
 * opts->budget configurations are timed, opts->t_max_s elapses, or
 * 64·budget + 1024 draws were made (stop_reason 3). opts->s0 and opts->rho
 * are not used (rho must still be ≥ 1). s* is the first minimum cost; with
 * nothing timed it is the configuration of rank 0 at cost +inf.
 * Same ownership and error behaviour as tune_gbfs. */
int tune_random(const gt_space* sp, const gt_tune_opts* opts, gt_cost_fn cost,
                void* ctx, gt_tune_result* out);

/* ---- N-A2C (§4.3, Alg.2) ------------------------------------------------ */

/* Settings of N-A2C. The paper fixes T = 3 (§5) and the reward (§4.1); the
 * rest are readings of what it leaves open. */
typedef struct gt_na2c_params {
  int32_t T;          /* steps per walk (𝒯), 1..64; default 3 */
  int32_t B;          /* len(B_test): states collected and timed per episode, ≤ 65536; 8 */
  int32_t H;          /* hidden tanh units of the actor and of the critic, 1..64; 32 */
  int32_t mem;        /* capacity of the FIFO memory 𝓜 (transitions), ≤ 65536; 256 */
  int32_t max_walks;  /* walks per episode before it is timed with fewer than B, ≤ 2^20; 64 */
  int32_t reward;     /* 0: r(s, a) = 1/cost(s') (§4.1, default); 1: variant
                         log(cost(s)/cost(s')) clipped to ±r_clip */
  int32_t eps_halving; /* 1: variant that also halves eps after an episode that
                          collects nothing; 0 (default): eps stays fixed */
  int32_t reserved;
  double eps;         /* probability of following π (else a uniform action); 0.8 */
  double gamma;       /* discount of the TD(0) advantage; 0.9 */
  double lr;          /* SGD step of actor and critic; 0.01 */
  double r_clip;      /* clip of the log-ratio reward variant; 5 */
} gt_na2c_params;

/* Fills the defaults listed in gt_na2c_params (§5 fixes T = 3; the rest are
 * the library's readings of §4.3). p: caller-owned. GT_EINVAL if p is NULL. */
int gt_na2c_params_init(gt_na2c_params* p);

/* N-A2C over the space, timed exactly as tune_gbfs (GPU or callback; same
 * opts: s0 (NULL: the paper's [D,1,…,1], MFMA 16), budget, t_max_s, seed,
 * log, progress). Actions: per dimension the ordered level pairs the
 * neighbour mode allows (×2 at one level, ÷2 at the other; available when the
 * halved factor is even), then the MFMA toggle. State features: each level's
 * share of its dimension's power-of-two exponent, plus the MFMA bit. Actor:
 * one hidden tanh layer, softmax over the available actions; critic: one
 * hidden tanh layer, linear output; weights U(±1/√fan_in) from
 * SplitMix64(seed ^ 0xA2C0A2C0A2C0A2C0), biases 0. Each episode walks T steps
 * from the centre (s0, then the best state so far) until B unvisited
 * legitimate states are collected (illegitimate states may be walked
 * through, never collected) or max_walks walks were made; with probability
 * eps a step samples π, else a uniform available action (SplitMix64(seed));
 * a walk ends at a state with no available action (one-configuration spaces).
 * An episode that collects nothing lengthens the walks by one step (the
 * paper lets the exploration step grow; params->eps_halving also halves eps),
 * up to T + 8 steps, after which the search stops (stop_reason 1); a new best
 * state resets the walk length and eps. The collected states are timed in
 * order; after each timing, every transition (s, a, r, s') into it from an
 * already-timed neighbour s joins 𝓜 (r = 1/cost(s'), §4.1, unless
 * params->reward selects the log-ratio variant) and one SGD pass over 𝓜
 * (oldest first) moves every parameter by lr·δ times its gradient — of V(s)
 * for the critic (TD(0), δ = r + γV(s') − V(s)), of log π(a|s) for the actor —
 * taken before the update. out->popped counts episodes. params NULL: the defaults. Same ownership and
 * error behaviour as tune_gbfs. */
int tune_na2c(const gt_space* sp, const gt_tune_opts* opts, const gt_na2c_params* params,
              gt_cost_fn cost, void* ctx, gt_tune_result* out);

/* Releases the device memory the library keeps between calls (the
 * per-GPU comparison buffers; each GPU's current device is restored).
 * Must not run concurrently with any other call of the library; later calls
 * allocate again as needed, so calling it twice, or a GEMM after it, is
 * fine. GT_EHIP if a hipFree fails (the remaining buffers are still
 * released). */
int gt_shutdown(void);

/* Thread-local message of the last failure. */
const char* gt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GEMMTUNE_H */
