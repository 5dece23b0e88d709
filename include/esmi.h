/*
 * esmi.h -- C-ABI of the MI355X (gfx950) evolution-strategy generation library.
 *
 * The library runs the ask / evaluate / tell loop of the evosax report
 * (arXiv 2212.04180, Sec. 2.1, Listing 1) for OpenAI-ES (Table 1, FDG class)
 * -- and PGPE, SNES and Sep-CMA-ES on the same path (es_strategy below) --
 * on R independent runs at once (the vmap over seeds of Sec. 2.2, Listing 3):
 *   ask      antithetic Gaussian perturbations x = m +- sigma*eps, eps drawn
 *            from a counter-based Philox-4x32-10 stream and regenerated on
 *            demand -- never stored;
 *   evaluate built-in benchmark problems (Sec. 3.2: sphere, shifted sphere,
 *            Rosenbrock, Rastrigin; a teacher-student MLP), fused with ask;
 *   tell     fitness shaping (Sec. 3.2: centered ranks as in App. B,
 *            z-scores, weight-decay regularisation), the finite-difference
 *            gradient estimate of Sec. 2.1, g = E^T y / (N sigma), and an
 *            Adam (or ClipUp) step on the mean (App. B); sigma and the learning rate
 *            then follow the exponential schedules of the App. B tables,
 *            per run (the vmap over hyper-parameters of Sec. 2.2).
 *
 * Conventions shared by every entry point:
 *   - Device pointers are HIP device addresses on the device that was
 *     current when es_init ran; host pointers are ordinary memory.  Arrays
 *     are dense, row-major, fp32 unless stated: a "[R][N]" array holds
 *     element (r, j) at r*N + j.
 *   - Every call only enqueues work on the stream given to es_init and
 *     returns without waiting, except where "synchronous" is stated.
 *     Outputs are valid once that stream has been synchronized (es_sync).
 *   - The caller owns every buffer it passes; the handle owns its state
 *     (mean, Adam moments, best-so-far, problem data, scratch).
 *   - No call throws.  A negative es_status reports an error; the message
 *     is available from es_last_error(h).  A failed call leaves the state
 *     unchanged unless it is ES_ERR_HIP (then the handle should be
 *     destroyed).
 *   - A handle is not thread-safe; distinct handles are independent.
 *   - The generation counter, sigma / lr buffer selection and sequence
 *     checks live on the host and the kernels take them as launch
 *     arguments, so a stream capture of es_ask / es_eval / es_tell records
 *     that one generation; a replay repeats it on the current state (for
 *     ES_PROB_MLP with OpenAI-ES on the inputs the replayed es_tell made for
 *     the generation after it), with the per-run sigma and lr of the
 *     captured generation: schedules and Sep-CMA-ES's step size do not
 *     advance from replay to replay.  For many generations per launch use
 *     es_run.
 *   - Minimisation is the default (Listing 1); maximize = 1 negates keys.
 */
#ifndef ESMI_H
#define ESMI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ES_OK = 0,
    ES_ERR_ARG = -1,         /* invalid argument or configuration            */
    ES_ERR_SEQUENCE = -2,    /* call out of ask -> (eval) -> tell order        */
    ES_ERR_HIP = -3,         /* a HIP runtime call failed                     */
    ES_ERR_OOM = -4,         /* device allocation failed                      */
    ES_ERR_UNSUPPORTED = -5  /* valid request the library does not implement  */
} es_status;

/* Fitness shaping (Sec. 3.2).  With key_j = f_j (minimise) or -f_j
 * (maximise), NaN the worst key (+inf), and -- when w_decay != 0 -- the
 * weight-decay penalty key_j = fl32(key_j + fl32(w_decay * pen_j)) for finite
 * keys, pen_j = (1/D) sum_d x_jd^2:
 *   CENTERED_RANK  y_j = (2 rank_j - (N-1)) / (2 (N-1)), one fp32 division of
 *                  exact integers; rank = position in a stable ascending sort
 *                  of the keys (ties by member index);
 *   RAW            y_j = key_j;
 *   Z_SCORE        y_j = fl32((key_j - mu) / (sd + 1e-10)), mu and sd the
 *                  fp64 mean and population standard deviation of the finite
 *                  keys; y_j = 0 for a non-finite key. */
typedef enum { ES_SHAPE_CENTERED_RANK = 0, ES_SHAPE_RAW = 1, ES_SHAPE_Z_SCORE = 2 } es_shaping;

typedef enum {
    ES_PROB_NONE = 0,           /* fitness only from the caller (es_tell)           */
    ES_PROB_SPHERE = 1,         /* sum x_i^2                                        */
    ES_PROB_SHIFTED_SPHERE = 2, /* sum (x_i - s_i)^2, s ~ N(0,1) from the base seed */
    ES_PROB_ROSENBROCK = 3,     /* sum_{i<D-1} 100 (x_{i+1} - x_i^2)^2 + (1 - x_i)^2 */
    ES_PROB_RASTRIGIN = 4,      /* A D + sum x_i^2 - A cos(2 pi x_i)                */
    ES_PROB_MLP = 5             /* -MSE of a 64-256-256-16 tanh MLP vs a teacher    */
} es_problem;

typedef enum { ES_INIT_UNIFORM = 0, ES_INIT_ZERO = 1, ES_INIT_FANIN_NORMAL = 2 } es_init_kind;

/* Strategies (Table 1).  All sample antithetic pairs x = m +- s (.) z_p with
 * z_p the Philox normals of pair p; s = sigma (OpenAI-ES) or a per-dimension
 * sigma vector (PGPE, SNES).  With a_p = y_p - y_{p+P}, b_p the second folded
 * weight, A_d = sum_p a_p z_pd and B_d = sum_p b_p (z_pd^2 - 1):
 *   OPENAI_ES  g = A / (N sigma); the optimiser steps the mean.
 *   PGPE       (Sehnke et al. 2010, symmetric sampling) b_p = (y_p +
 *              y_{p+P})/2 - mean(y); g = sigma_d A / N for the optimiser;
 *              sigma_d += clip(-sigma_lr sigma_d B / P, +-max_change sigma_d).
 *   SNES       (Schaul et al. 2011) y = softmax rank utilities of App. B,
 *              w = softmax(beta (rank'/N - 1/2)), rank' = N-1-rank (best
 *              largest), b_p = y_p + y_{p+P}; m += fl32(lr sigma_d) A,
 *              sigma_d *= exp(sigma_lr/2 B); the shaping field is ignored.
 * After each tell the sigma (vector) follows the schedule.  For PGPE and
 * SNES the run's sigma (cfg.sigma, es_get_hparams) is the value every
 * dimension starts from at es_init and stays fixed.
 *   SEP_CMA    Sep-CMA-ES (Ros & Hansen 2008): independent members
 *              x_j = m + s (.) z_j (Philox row j), s_d = fl32(sigma sqrtf(C_d));
 *              the mu = max(1, floor(elite_ratio N)) best members recombine
 *              with weights ln(mu + 1/2) - ln(i + 1) (normalised);
 *              evolution paths p_sigma, p_c, diagonal covariance C and
 *              path-length control of sigma with the standard CMA-ES
 *              settings and the separable rate factor (D + 2)/3.  m1 and v
 *              of es_get_state hold p_sigma and p_c; es_get_strategy_state's
 *              sigma_vec holds C; sigma is per run (es_get_hparams) and has
 *              no schedule.  The shaping field is ignored. */
typedef enum { ES_STRAT_OPENAI_ES = 0, ES_STRAT_PGPE = 1, ES_STRAT_SNES = 2, ES_STRAT_SEP_CMA = 3 } es_strategy;

/* Optimiser of the mean (OpenAI-ES, PGPE): Adam, or ClipUp (Toklu et al.
 * 2020, the ES optimiser named in Sec. 3.1): v = momentum v + lr g/|g|,
 * clipped to |v| <= clipup_max_speed, m -= v (norms in fp64 over the run). */
typedef enum { ES_OPT_ADAM = 0, ES_OPT_CLIPUP = 1 } es_optimizer;

/* Flags (es_config.flags). */
#define ES_FLAG_KEEP_GRAD 1u /* es_tell and es_run also store g [R][D] for es_get_grad */

/*
 * Strategy parameters (the default_params of Listing 1; App. B, OpenAI-ES
 * table).  Random streams: run r uses key seed + r; the shift vector, the
 * teacher network and the MLP inputs come from the base seed and are shared
 * by all runs.
 */
typedef struct es_config {
    int64_t num_dims;   /* D >= 1                                           */
    uint64_t seed;      /* base seed                                         */
    int32_t popsize;    /* N >= 2, even, <= 2^24: N/2 antithetic pairs       */
    int32_t num_runs;   /* R >= 1 independent runs                           */
    float sigma;        /* > 0, perturbation scale                           */
    float lr;           /* Adam learning rate                                */
    float beta1, beta2; /* Adam moment decays in [0, 1)                      */
    float eps;          /* Adam epsilon (outside the square root)            */
    int32_t maximize;   /* 0: minimise (default), 1: maximise               */
    int32_t shaping;    /* es_shaping                                        */
    int32_t init;       /* es_init_kind for the initial mean                 */
    float init_lo, init_hi; /* ES_INIT_UNIFORM range [lo, hi)                */
    int32_t problem;    /* es_problem used by es_eval / es_run               */
    float rastrigin_a;  /* A of Rastrigin (10)                               */
    int32_t mlp_batch;  /* ES_PROB_MLP: inputs per generation (256)          */
    int32_t mlp_bf16;   /* ES_PROB_MLP: 1 = bf16 matrix-core forward         */
    int32_t mlp_tanh_out; /* ES_PROB_MLP: 1 = tanh on the output layer       */
    uint32_t flags;     /* ES_FLAG_*                                         */
    /* Schedules (App. B, OpenAI-ES and PGPE tables: init / decay / final):
     * after every tell sigma <- max(fl32(sigma * sigma_decay), sigma_final)
     * and lr likewise, per run.  decay 1 and final 0 keep them constant. */
    float sigma_decay;  /* > 0                                               */
    float sigma_final;  /* >= 0                                              */
    float lr_decay;     /* > 0                                               */
    float lr_final;     /* >= 0                                              */
    float w_decay;      /* >= 0, weight-decay coefficient of the shaping     */
    int32_t strategy;   /* es_strategy                                       */
    int32_t optimizer;  /* es_optimizer (ignored by SNES)                    */
    float sigma_lr;     /* PGPE / SNES learning rate of sigma (> 0)          */
    float sigma_max_change; /* PGPE: |d sigma| <= max_change sigma, (0, 1)   */
    float clipup_max_speed; /* ClipUp velocity bound (> 0)                   */
    float clipup_momentum;  /* ClipUp velocity decay in [0, 1)               */
    float snes_temperature; /* SNES utility temperature beta (>= 0)          */
    float elite_ratio;  /* Sep-CMA-ES: share of the population recombined, (0, 1] */
    /* Launch plan (not part of the method; 0 = the library's choice, which
     * is what every result in the documentation refers to).  The first two
     * set how the fp32 partial sums are grouped, so they change the
     * summation order and therefore the low bits of the fitness and of the
     * gradient; plan_run_path only picks the code path of es_run.
     *   plan_eval_blocks  Philox blocks (4 dims) per evaluate chunk, >= 0;
     *                     each chunk's per-member partial is one fp32 sum
     *   plan_tell_split   gradient workgroups per group of 64 Philox blocks
     *                     (their fp64 partials are added in split order), >= 0;
     *                     the library may lower it to keep two pair groups
     *                     per slice, and ignores it where es_run's fused
     *                     loop would run (those keep the fused loop's order)
     *   plan_run_path     es_run: 1 = always the per-call kernels, 2 = the
     *                     fused loop wherever it supports the config (in
     *                     the fused loop's summation order, which equals the
     *                     per-call kernels' only where the library itself
     *                     would choose the fused loop), 3 = the grid loop
     *                     wherever it supports the config (always in the
     *                     per-call kernels' order, so the same bits); 0 =
     *                     the fused loop for small runs or many runs, the
     *                     grid loop where it applies (its workgroups keep
     *                     their share of the normals in LDS; at most 2^20
     *                     Philox pair-blocks in all, num_runs * popsize/2 *
     *                     ceil(D/4)), else the per-call kernels.  Both loops
     *                     run OpenAI-ES with Adam on the benchmark problems,
     *                     centered-rank or raw shaping, no weight decay; the
     *                     grid loop also needs popsize <= 8192
     *   plan_grid_workgroups  workgroups per run of the grid loop, 0..16
     *                     (0: about one per 2048 pair-blocks of a run),
     *                     lowered to what the evaluate chunks allow (each
     *                     workgroup owns whole chunk slices of the fitness
     *                     reduction: at most min(chunks, 16), beyond 16
     *                     chunks a divisor of 16); no effect on the results
     *   plan_rank_path    how the ranks are found (same ranks, same bits
     *                     either way): 1 = each workgroup counts against the
     *                     run's keys in LDS (popsize <= 16384), 2 = the
     *                     run's composite keys (key, member) are radix-sorted
     *                     and a member's position is its rank (also needs
     *                     num_runs * popsize < 2^31); 0 = the library's
     *                     choice: 2 above popsize 16384, and where
     *                     num_runs * popsize^2 > 1.2e8 (where it is the
     *                     faster), else 1
     *   plan_grid_spin_limit  polls of a word before a wait of the grid loop
     *                     gives up (0: 2^20, which a correct launch never
     *                     reaches; -1: every wait gives up at once, the
     *                     failure path, for tests); no effect on the results
     *                     of a launch whose waits all succeed.  A wait that
     *                     gives up ends the launch early with the state not
     *                     valid: es_sync reports it
     *   plan_grid_pack    placement of the grid loop's workgroups: 0 (the
     *                     library's choice) packs each run's workgroups onto
     *                     one XCD, whose L2 they then share for their
     *                     exchanges: the launch holds (XCDs) times the
     *                     workgroups, the hardware deals them to the XCDs in
     *                     turn, those of x index = r (mod XCDs) work for run
     *                     r and the others return at once; taken only where
     *                     the device holds the larger launch resident, else
     *                     as -1.  -1: one workgroup per participant.  No
     *                     effect on the results, only on the time          */
    int32_t plan_eval_blocks;
    int32_t plan_tell_split;
    int32_t plan_run_path;
    int32_t plan_rank_path;
    int32_t plan_grid_workgroups;
    int32_t plan_grid_spin_limit;
    int32_t plan_grid_pack;
} es_config;

typedef struct es_handle es_handle;

/* Create a strategy: validates cfg, allocates device state and enqueues the
 * initial mean (Listing 1 initialize), m1 = v = 0, t = 0, best = none.
 * hip_stream: a hipStream_t (NULL = the default stream) used by every later
 * call.  On success *out owns the handle (free with es_destroy). */
es_status es_init(const es_config* cfg, void* hip_stream, es_handle** out);

/* ask (Sec. 2.1 step 1): starts generation t.  x_out: NULL (the population
 * stays virtual and is regenerated where needed) or a device [R][N][D]
 * buffer that receives x_j = m + sigma*eps_j (j < N/2) and
 * m - sigma*eps_{j-N/2} (j >= N/2).  ES_ERR_SEQUENCE if the previous ask was
 * not followed by es_tell. */
es_status es_ask(es_handle* h, float* x_out);

/* evaluate (Sec. 2.1 step 2) with the configured built-in problem, fused
 * with the sampling: fitness_out device [R][N].  Requires a preceding es_ask
 * for this generation; ES_ERR_UNSUPPORTED for ES_PROB_NONE. */
es_status es_eval(es_handle* h, float* fitness_out);

/* Timing aid, not an operation of the paper: es_eval that also times its
 * main kernel.  start_event and stop_event
 * (hipEvent_t handles the caller created with timing enabled; either may be
 * NULL) are recorded by that kernel's dispatch itself (hipExtLaunchKernel),
 * at its start and at its end, so the stream carries no marker packet.  The
 * main kernel is the fused sample + evaluate (the benchmark problems; the
 * per-chunk sums are reduced by a second kernel after it) or the MLP forward
 * (a teacher kernel, when one runs, goes before it).  hipEventElapsedTime of
 * the two gives that kernel's time.  Same results as es_eval.  A timing
 * aid: not meant for a stream under capture. */
es_status es_eval_timed(es_handle* h, float* fitness_out, void* start_event, void* stop_event);

/* Allocation-free evaluate, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid
 * hipMalloc): es_eval's fused sample + evaluate without a handle.  It calls
 * no hipMalloc or hipFree and allocates nothing; its per-chunk partial sums
 * live in a static device array of 16 MiB per device (held until the
 * process ends), whose address is looked up on the first call on a device.
 *   cfg           a config es_init would accept; OpenAI-ES (scalar sigma)
 *                 and the benchmark problems only (ES_ERR_UNSUPPORTED else);
 *                 num_dims % 4 == 0 unless num_runs == 1 (ES_ERR_UNSUPPORTED)
 *   mean          device [R][D], the runs' means
 *   problem_data  device [D], the shift vector s for ES_PROB_SHIFTED_SPHERE
 *                 (es_get_problem_data of a handle with this config gives
 *                 it), NULL for the other problems
 *   sigma         device [R], each run's sigma of generation t
 *   t             generation whose noise is drawn, in [0, 2^32)
 *   fitness       device [R][N] output, the same bits es_eval gives a handle
 *                 with this config, mean, sigma and t
 *   hip_stream    hipStream_t the kernels are enqueued on (NULL: default)
 * ES_ERR_ARG when the evaluate's partial sums need more than 16 MiB (the
 * default plan needs about 12.6 MB for any run count and population; a
 * small cfg.plan_eval_blocks can need more).  Errors are reported through
 * es_last_error(NULL).  Calls that overlap on one device (several streams or
 * threads) share the array and race: serialise them. */
es_status es_eval_noalloc(const es_config* cfg, const float* mean, const float* problem_data, const float* sigma,
                          int64_t t, float* fitness, void* hip_stream);

/* tell (Sec. 2.1 step 3): fitness shaping (es_shaping; with weight decay the
 * penalty pass regenerates the population once more), g = E^T y / (N sigma)
 * with eps regenerated from the counter, Adam step on the mean, best-so-far
 * update on the raw fitness, schedule step of sigma and lr; t += 1.
 * fitness: device [R][N] from es_eval or from the caller's own evaluation
 * of the asked population.  ES_PROB_MLP with OpenAI-ES: the same launch also
 * makes the next generation's inputs and teacher outputs, which the next
 * es_eval then uses. */
es_status es_tell(es_handle* h, const float* fitness);

/* T fused generations (the scanned loop of Listing 2) with the built-in
 * problem.  log: NULL or device [T][R] receiving each generation's best
 * fitness (the member of rank 0).  Requires no open ask.  The code path
 * (per-call kernels, the fused loop of one workgroup per run, or the grid
 * loop of a cooperative launch per up to 256 generations) follows
 * cfg.plan_run_path. */
es_status es_run(es_handle* h, int32_t T, float* log);

/* Copy out / replace the search state (the state fields of Listing 1; the
 * paper defines no accessor: these are host-side plumbing).  m, m1, v:
 * device [R][D] (NULL to skip); t: number of completed generations.
 * es_set_state requires no open ask.  es_set_state and es_load_state also
 * clear the failure flag of the grid loop that es_sync reports. */
es_status es_get_state(es_handle* h, float* m, float* m1, float* v, int64_t* t);
es_status es_set_state(es_handle* h, const float* m, const float* m1, const float* v, int64_t t);

/* Best member and fitness seen so far (state fields of Listing 1).
 * member: device [R][D], fitness: device [R] (NaN while none). */
es_status es_get_best(es_handle* h, float* member, float* fitness);

/* Diagnostics of the last es_tell, not operations of the paper (they expose
 * intermediate values of the tell of Sec. 2.1 for inspection and tests):
 * shaped weights y [R][N], ranks [R][N] (int32), and -- when
 * ES_FLAG_KEEP_GRAD is set -- the gradient g [R][D].  Device pointers; NULL
 * to skip. */
es_status es_get_shaped(es_handle* h, float* y, int32_t* rank);
es_status es_get_grad(es_handle* h, float* g);

/* Per-run hyper-parameters (the vmap over hyper-parameters of Sec. 2.2):
 * sigma and lr of the next generation of every run.  Host arrays [R];
 * either may be NULL (left unchanged).  es_init sets every run to
 * cfg.sigma and cfg.lr; the schedules continue from the values set here.
 * Requires no open ask; sigma must be finite and > 0, lr finite and >= 0
 * (ES_ERR_ARG otherwise).  PGPE and SNES refuse a sigma (ES_ERR_UNSUPPORTED:
 * they sample with the per-dimension sigma of es_set_strategy_state).
 * es_get_hparams is synchronous. */
es_status es_set_hparams(es_handle* h, const float* sigma, const float* lr);
es_status es_get_hparams(es_handle* h, float* sigma, float* lr);

/* Per-dimension sigma (PGPE, SNES) -- for Sep-CMA-ES the diagonal
 * covariance C -- and ClipUp velocity of every run:
 * device [R][D] each; NULL to skip.  ES_ERR_UNSUPPORTED for a state the
 * configured strategy and optimiser do not keep.  es_set_strategy_state
 * requires no open ask. */
es_status es_get_strategy_state(es_handle* h, float* sigma_vec, float* velocity);
es_status es_set_strategy_state(es_handle* h, const float* sigma_vec, const float* velocity);

/* Diagnostic, not an operation of the paper: the weight-decay penalty of the
 * last es_tell (Sec. 3.2 shaping), pen [R][N] = (1/D) sum_d x_jd^2 of every
 * member (device pointer).  ES_ERR_UNSUPPORTED when w_decay = 0. */
es_status es_get_penalty(es_handle* h, float* pen);

/* Accessor, not an operation of the paper: the problem data shared by all
 * runs, the shift vector s [D] (shifted sphere) or the flattened teacher
 * network [D] (MLP).  Device pointer. */
es_status es_get_problem_data(es_handle* h, float* out);

/* Test aid, not an operation of the paper: the raw stream for one (run,
 * generation t, pair), the Philox words words[4*ceil(D/4)] (uint32) and the
 * normals eps[D] that ask (Sec. 2.1) perturbs with.  Device pointers; NULL
 * to skip.  Uses the same device code as ask, evaluate and tell. */
es_status es_debug_noise(es_handle* h, int32_t run, int64_t t, int32_t pair,
                         uint32_t* words, float* eps);

/* Checkpoint (synchronous; the paper defines none -- the state is that of
 * Listing 1): with host_buf NULL, *bytes receives the size;
 * otherwise the state (config, t, m, m1, v, best, per-run sigma and lr, the
 * sigma vector and velocity where kept) is written to host_buf.
 * es_load_state restores a checkpoint of a handle with the same config.
 * The random stream is a pure function of (seed, t), so resuming continues
 * the same trajectory bit for bit. */
es_status es_save_state(es_handle* h, void* host_buf, size_t* bytes);
es_status es_load_state(es_handle* h, const void* host_buf, size_t bytes);

/* Runtime plumbing below, not operations of the paper. */

/* Wait for all work enqueued by this handle (synchronous).  Not defined by
 * the paper.  Also reports ES_ERR_HIP if a grid-loop launch of es_run ended
 * early because a wait for another workgroup's values gave up (its
 * workgroups are resident together under a cooperative launch, so with the
 * default cfg.plan_grid_spin_limit only a library fault can cause that; the
 * state is then not valid, and stays reported until es_set_state or
 * es_load_state replaces it). */
es_status es_sync(es_handle* h);

/* Current generation counter t (host value; no device work). */
int64_t es_generation(const es_handle* h);

/* The code path es_run takes for this handle (host value; no device work;
 * not defined by the paper): 1 the per-call kernels, 2 the fused loop (one
 * workgroup per run), 3 the grid loop (a cooperative launch of several
 * workgroups per run); 0 for a NULL handle.  See cfg.plan_run_path.
 * keeps_normals (NULL to skip) receives 1 where that path's gradient reads
 * the normals its evaluate kept in LDS instead of regenerating them (the
 * grid loop always, the fused loop where they fit), else 0; the results are
 * the same bits either way. */
int32_t es_run_path(const es_handle* h, int32_t* keeps_normals);

/* Message of the last failed call on h ("" if none); with h == NULL, the
 * message of the last failed es_init on this thread.  Never NULL. */
const char* es_last_error(const es_handle* h);

/* Static description of a status code. */
const char* es_status_string(es_status s);

/* Release the handle and its device memory (waits for its stream). */
void es_destroy(es_handle* h);

#ifdef __cplusplus
}
#endif
#endif /* ESMI_H */
