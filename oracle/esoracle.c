/*
 * esoracle.c -- plain, slow CPU oracle for one OpenAI-ES generation.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of the
 * benchmark use it.  It shares no code, header, table or constant generator with
 * the HIP library: every step is written here again from its definition.
 *
 * What is computed (evosax report, arXiv 2212.04180):
 *   - the ask / evaluate / tell loop of Sec. 2.1 (Listing 1), run for several
 *     independent seeds as in Sec. 2.2 (Listing 3, vmap over keys);
 *   - OpenAI-ES (Table 1, FDG class): isotropic Gaussian perturbations with
 *     antithetic sampling, the finite-difference gradient estimator of Sec. 2.1
 *     (grad_m E f(m + s*eps) = (1/s) E[f(m + s*eps) eps]), centered-rank fitness
 *     shaping (Sec. 3.2; App. B, OpenAI-ES table) and an Adam update of the mean
 *     (Sec. 2.1; App. B).  Minimisation is the default (Listing 1).
 *   - The paper names no random-number generator, no rank formula and no Adam
 *     formula.  The readings used here (Philox-4x32-10 with a fixed counter
 *     layout, Box-Muller, the exact centered-rank fraction, Kingma & Ba Adam) are
 *     stated at each function.
 *
 * Arithmetic: fp64 accumulation everywhere a sum appears; fp32 where the
 * method's state is fp32.  Build with -ffp-contract=off so that no multiply-add
 * is fused unless written as fmaf().
 *
 * Parity status per function is recorded in the test-suite; the only part that
 * no outside fact pins is a free-running multi-generation trajectory (it is
 * pinned only stage by stage), which the test-suite marks "parity unpinned".
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Threads.  The loops over members (evaluation, population, penalty) and    */
/* over blocks of dimensions (gradient and noise sums) run in parallel with  */
/* OpenMP when the file is built with it.  Each parallel loop hands out      */
/* independent outputs (a member's fitness, a dimension's sum) and every     */
/* output's own sum keeps the serial order, so the results are bit-identical */
/* for any thread count.  n <= 0 restores OpenMP's default (OMP_NUM_THREADS, */
/* else all cores).                                                         */
/* ------------------------------------------------------------------------ */
void or_set_threads(int32_t n)
{
#ifdef _OPENMP
    static int32_t dflt = 0; /* OpenMP's own choice, seen before the first change */
    if (dflt == 0) dflt = (int32_t)omp_get_max_threads();
    omp_set_num_threads(n > 0 ? n : dflt);
#else
    (void)n;
#endif
}

int32_t or_get_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* Dimensions per work item of the dimension-parallel loops (a multiple of  */
/* the four dimensions of one generator block).                              */
#define OR_DIM_CHUNK 4096

/* ------------------------------------------------------------------------ */
/* Philox-4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11).  The paper uses JAX's splittable keys (Listing 1) */
/* and names no generator; the counter-based Philox stream replaces them.     */
/* ------------------------------------------------------------------------ */
#define OR_TWO_PI 6.283185307179586476925286766559
#define OR_PHILOX_M0 0xD2511F53u
#define OR_PHILOX_M1 0xCD9E8D57u
#define OR_PHILOX_W0 0x9E3779B9u
#define OR_PHILOX_W1 0xBB67AE85u

void or_philox4x32_10(uint32_t k0, uint32_t k1, const uint32_t ctr[4], uint32_t out[4])
{
    uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { /* key schedule: bump the key between rounds */
            k0 += OR_PHILOX_W0;
            k1 += OR_PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)OR_PHILOX_M0 * (uint64_t)c[0];
        uint64_t p1 = (uint64_t)OR_PHILOX_M1 * (uint64_t)c[2];
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c[1] ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c[3] ^ k1;
        uint32_t n3 = lo0;
        c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    }
    out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

/* Counter layout (reading): key = (lo32(seed_r), hi32(seed_r)),
 * counter = (block = d/4, row, t, domain).                                  */
enum { OR_DOM_NOISE = 0, OR_DOM_INIT = 1, OR_DOM_PROBLEM = 2, OR_DOM_EVAL = 3 };

void or_words(uint64_t seed, uint32_t domain, uint32_t row, uint32_t t,
              int64_t b0, int64_t nb, uint32_t* out)
{
    for (int64_t i = 0; i < nb; ++i) {
        uint32_t ctr[4] = {(uint32_t)(b0 + i), row, t, domain};
        or_philox4x32_10((uint32_t)seed, (uint32_t)(seed >> 32), ctr, out + 4 * i);
    }
}

/* Uniforms (reading): exact multiples of 2^-24. */
static double or_u_pos(uint32_t w) { return (double)((w >> 8) + 1u) * 0x1p-24; } /* (0,1] */
static double or_u_half(uint32_t w) { return (double)(w >> 8) * 0x1p-24; }       /* [0,1) */

/* Box-Muller (search distribution N(m, s^2 I) of Sec. 2.1): words (w0,w1)
 * give two normals r*cos(2 pi th), r*sin(2 pi th) with r = sqrt(-2 ln u),
 * computed in fp64 and rounded once to fp32.                               */
static void or_box_muller(const uint32_t w[4], float out[4])
{
    for (int h = 0; h < 2; ++h) {
        double r = sqrt(-2.0 * log(or_u_pos(w[2 * h])));
        double a = OR_TWO_PI * or_u_half(w[2 * h + 1]);
        out[2 * h] = (float)(r * cos(a));
        out[2 * h + 1] = (float)(r * sin(a));
    }
}

/* Normals for dims [d0, d0+nd) of the stream (seed, domain, row, t). */
void or_normals(uint64_t seed, uint32_t domain, uint32_t row, uint32_t t,
                int64_t d0, int64_t nd, float* out)
{
    int64_t d = d0;
    while (d < d0 + nd) {
        uint32_t w[4];
        float z[4];
        or_words(seed, domain, row, t, d / 4, 1, w);
        or_box_muller(w, z);
        for (int64_t k = d % 4; k < 4 && d < d0 + nd; ++k, ++d) out[d - d0] = z[k];
    }
}

/* ------------------------------------------------------------------------ */
/* Configuration (mirrors the fields of the library's config, declared here  */
/* again on purpose: the oracle includes nothing from the library).         */
/* ------------------------------------------------------------------------ */
enum { OR_PROB_NONE = 0, OR_PROB_SPHERE = 1, OR_PROB_SHIFTED_SPHERE = 2,
       OR_PROB_ROSENBROCK = 3, OR_PROB_RASTRIGIN = 4, OR_PROB_MLP = 5 };
enum { OR_INIT_UNIFORM = 0, OR_INIT_ZERO = 1, OR_INIT_FANIN_NORMAL = 2 };
enum { OR_SHAPE_CENTERED_RANK = 0, OR_SHAPE_RAW = 1, OR_SHAPE_Z_SCORE = 2 };
enum { OR_STRAT_OPENAI_ES = 0, OR_STRAT_PGPE = 1, OR_STRAT_SNES = 2, OR_STRAT_SEP_CMA = 3 };
enum { OR_OPT_ADAM = 0, OR_OPT_CLIPUP = 1 };

typedef struct {
    int64_t num_dims;   /* D */
    int32_t popsize;    /* N, even */
    int32_t num_runs;   /* R */
    float sigma, lr, beta1, beta2, eps;
    int32_t maximize;
    int32_t shaping;
    uint64_t seed;      /* run r uses seed + r */
    int32_t init;
    float init_lo, init_hi;
    int32_t problem;
    float rastrigin_a;
    int32_t mlp_batch;  /* inputs per generation */
    int32_t mlp_bf16;   /* 1: student forward rounds operands to bf16 */
    int32_t mlp_tanh_out;
    /* schedules (App. B tables: init / decay / final): after each tell       */
    /* sigma <- max(sigma * decay, final), lr likewise; 1 and 0 keep them      */
    /* constant.  sigma and lr above are the values of the current generation. */
    float sigma_decay, sigma_final, lr_decay, lr_final;
    float w_decay;      /* weight-decay coefficient of the fitness shaping   */
    /* Strategies of Table 1 beside OpenAI-ES (PGPE, SNES) and the ClipUp     */
    /* optimiser named in Sec. 3.1; parameters from the App. B tables.        */
    int32_t strategy;        /* OR_STRAT_*                                   */
    int32_t optimizer;       /* OR_OPT_* for the mean (OpenAI-ES, PGPE)       */
    float sigma_lr;          /* PGPE / SNES learning rate of sigma            */
    float sigma_max_change;  /* PGPE: bound of |d sigma| / sigma per step     */
    float clipup_max_speed;  /* ClipUp: bound of the velocity norm            */
    float clipup_momentum;   /* ClipUp: velocity decay                        */
    float snes_temperature;  /* SNES: beta of the softmax rank utilities      */
    const float* sigma_vec;  /* per-dimension sigma of this run (PGPE, SNES);   */
                             /* Sep-CMA-ES: the sampling scale sigma*sqrt(C)  */
    float elite_ratio;       /* Sep-CMA-ES: mu = max(1, floor(ratio * N))     */
} or_config;

/* MLP 64-256-256-16 layer table, flattened [out][in] row-major weights, then
 * bias, layer by layer (parameter reshaping, Sec. 3.2; flattening order is a
 * reading).                                                                */
#define OR_MLP_IN 64
#define OR_MLP_H 256
#define OR_MLP_OUT 16
static const int64_t or_mlp_fan_in[3] = {OR_MLP_IN, OR_MLP_H, OR_MLP_H};
static const int64_t or_mlp_fan_out[3] = {OR_MLP_H, OR_MLP_H, OR_MLP_OUT};

int64_t or_mlp_num_params(void)
{
    int64_t n = 0;
    for (int l = 0; l < 3; ++l) n += or_mlp_fan_in[l] * or_mlp_fan_out[l] + or_mlp_fan_out[l];
    return n;
}

/* For flat index i: layer, and whether it is a weight (1) or a bias (0). */
static int or_mlp_locate(int64_t i, int* layer)
{
    int64_t off = 0;
    for (int l = 0; l < 3; ++l) {
        int64_t nw = or_mlp_fan_in[l] * or_mlp_fan_out[l];
        if (i < off + nw) { *layer = l; return 1; }
        off += nw;
        if (i < off + or_mlp_fan_out[l]) { *layer = l; return 0; }
        off += or_mlp_fan_out[l];
    }
    *layer = -1;
    return 0;
}

/* Fan-in normal vector: weights z/sqrt(fan_in), biases 0 (reading of
 * "N(0, 1/fan_in) weights").                                                */
static void or_fanin_normal(uint64_t seed, uint32_t domain, int64_t D, float* out)
{
    float* z = (float*)malloc(sizeof(float) * (size_t)D);
    or_normals(seed, domain, 0, 0, 0, D, z);
    for (int64_t i = 0; i < D; ++i) {
        int l;
        if (or_mlp_locate(i, &l))
            out[i] = (float)((double)z[i] / sqrt((double)or_mlp_fan_in[l]));
        else
            out[i] = 0.0f;
    }
    free(z);
}

/* Initial mean of run r (reading: uniform from the INIT stream as
 * lo + (hi - lo) * u, one fp32 rounding; zero; or fan-in normal).          */
void or_init_mean(const or_config* c, int32_t run, float* m)
{
    uint64_t seed = c->seed + (uint64_t)run;
    int64_t D = c->num_dims;
    if (c->init == OR_INIT_ZERO) {
        for (int64_t i = 0; i < D; ++i) m[i] = 0.0f;
    } else if (c->init == OR_INIT_UNIFORM) {
        float range = c->init_hi - c->init_lo;
        for (int64_t i = 0; i < D; ++i) {
            uint32_t w[4];
            or_words(seed, OR_DOM_INIT, 0, 0, i / 4, 1, w);
            m[i] = fmaf(range, (float)or_u_half(w[i % 4]), c->init_lo);
        }
    } else {
        or_fanin_normal(seed, OR_DOM_INIT, D, m);
    }
}

/* Problem data shared by all runs: the shift vector s (D floats) of the
 * shifted sphere, or the teacher MLP (D floats) -- both from the base seed,
 * PROBLEM stream.                                                           */
void or_problem_data(const or_config* c, float* out)
{
    if (c->problem == OR_PROB_SHIFTED_SPHERE)
        or_normals(c->seed, OR_DOM_PROBLEM, 0, 0, 0, c->num_dims, out);
    else if (c->problem == OR_PROB_MLP)
        or_fanin_normal(c->seed, OR_DOM_PROBLEM, c->num_dims, out);
}

/* ------------------------------------------------------------------------ */
/* ask: antithetic population (Sec. 2.1 ask step; antithetic sampling named */
/* in the FDG item).  Reading: members 0..N/2-1 use +eps_p, members          */
/* N/2..N-1 use -eps_{j-N/2}; x = fmaf(+-sigma, eps, m), one rounding.       */
/* ------------------------------------------------------------------------ */
void or_member(const or_config* c, int32_t run, uint32_t t, const float* m, int32_t j, float* x)
{
    int32_t half = c->popsize / 2;
    int64_t D = c->num_dims;
    float* eps = (float*)malloc(sizeof(float) * (size_t)D);
    if (c->strategy == OR_STRAT_SEP_CMA) {
        /* independent samples, row = member: x = m + s (.) z_j */
        or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)j, t, 0, D, eps);
        for (int64_t d = 0; d < D; ++d) x[d] = fmaf(c->sigma_vec[d], eps[d], m[d]);
        free(eps);
        return;
    }
    int32_t p = j < half ? j : j - half;
    or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)p, t, 0, D, eps);
    for (int64_t d = 0; d < D; ++d) {
        /* PGPE / SNES: a diagonal Gaussian, per-dimension sigma */
        float sd = c->sigma_vec ? c->sigma_vec[d] : c->sigma;
        x[d] = fmaf(j < half ? sd : -sd, eps[d], m[d]);
    }
    free(eps);
}

void or_population(const or_config* c, int32_t run, uint32_t t, const float* m, float* x)
{
#pragma omp parallel for schedule(static)
    for (int32_t j = 0; j < c->popsize; ++j) or_member(c, run, t, m, j, x + (int64_t)j * c->num_dims);
}

/* ------------------------------------------------------------------------ */
/* evaluate: benchmark problems (BBOB family named in Sec. 3.2); formulas as  */
/* the workloads state them; fp64 accumulation over fp32 x, rounded once.    */
/* ------------------------------------------------------------------------ */
float or_fitness_bbob(int32_t problem, const float* x, int64_t D, const float* s, float a)
{
    double acc = 0.0;
    if (problem == OR_PROB_SPHERE) {
        for (int64_t i = 0; i < D; ++i) acc += (double)x[i] * (double)x[i];
    } else if (problem == OR_PROB_SHIFTED_SPHERE) {
        for (int64_t i = 0; i < D; ++i) {
            double d = (double)x[i] - (double)s[i];
            acc += d * d;
        }
    } else if (problem == OR_PROB_ROSENBROCK) {
        for (int64_t i = 0; i + 1 < D; ++i) {
            double xi = x[i], xn = x[i + 1];
            double q = xn - xi * xi;
            acc += 100.0 * q * q + (1.0 - xi) * (1.0 - xi);
        }
    } else if (problem == OR_PROB_RASTRIGIN) {
        acc = (double)a * (double)D;
        for (int64_t i = 0; i < D; ++i) {
            double xi = x[i];
            acc += xi * xi - (double)a * cos(OR_TWO_PI * xi);
        }
    } else {
        return NAN;
    }
    return (float)acc;
}

/* bf16 round-to-nearest-even of an fp32 value (NaN kept quiet). */
static float or_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) {
        u |= 0x400000u;
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    float r;
    memcpy(&r, &u, 4);
    return r;
}

/* Generation-t input batch X_t [B][64], N(0,1) from the EVAL stream of the
 * base seed (shared by every member and run).                               */
void or_mlp_inputs(const or_config* c, uint32_t t, float* X)
{
    or_normals(c->seed, OR_DOM_EVAL, 0, t, 0, (int64_t)c->mlp_batch * OR_MLP_IN, X);
}

/* Dense forward of the 64-256-256-16 MLP on B inputs.  bf16 = 1 rounds the
 * input, every weight and every hidden activation to bf16 (RNE); dot products
 * accumulate exactly in fp64 and the pre-activation is rounded to fp32.     */
static void or_mlp_forward(const float* p, const float* X, int32_t B, int bf16, int tanh_out, float* Y)
{
    int64_t maxw = OR_MLP_H;
    float* hin = (float*)malloc(sizeof(float) * (size_t)(B * maxw));
    float* hout = (float*)malloc(sizeof(float) * (size_t)(B * maxw));
    for (int64_t i = 0; i < (int64_t)B * OR_MLP_IN; ++i) hin[i] = bf16 ? or_bf16(X[i]) : X[i];
    const float* q = p;
    for (int l = 0; l < 3; ++l) {
        int64_t fi = or_mlp_fan_in[l], fo = or_mlp_fan_out[l];
        const float* W = q;
        const float* bias = q + fi * fo;
        for (int32_t n = 0; n < B; ++n) {
            for (int64_t o = 0; o < fo; ++o) {
                double acc = 0.0;
                for (int64_t k = 0; k < fi; ++k) {
                    float w = bf16 ? or_bf16(W[o * fi + k]) : W[o * fi + k];
                    acc += (double)hin[n * fi + k] * (double)w;
                }
                float pre = (float)(acc + (double)bias[o]);
                float h;
                if (l < 2 || tanh_out) h = (float)tanh((double)pre);
                else h = pre;
                if (l < 2 && bf16) h = or_bf16(h);
                hout[n * fo + o] = h;
            }
        }
        float* tmp = hin; hin = hout; hout = tmp;
        q += fi * fo + fo;
    }
    for (int64_t i = 0; i < (int64_t)B * OR_MLP_OUT; ++i) Y[i] = hin[i];
    free(hin);
    free(hout);
}

/* Teacher targets for generation t: fp32 teacher (no bf16) on X_t. */
void or_mlp_teacher_out(const or_config* c, const float* teacher, uint32_t t, float* YT)
{
    float* X = (float*)malloc(sizeof(float) * (size_t)c->mlp_batch * OR_MLP_IN);
    or_mlp_inputs(c, t, X);
    or_mlp_forward(teacher, X, c->mlp_batch, 0, c->mlp_tanh_out, YT);
    free(X);
}

/* MLP fitness of one parameter vector: -MSE against the teacher targets. */
float or_mlp_fitness(const or_config* c, const float* x, uint32_t t, const float* YT)
{
    int32_t B = c->mlp_batch;
    float* X = (float*)malloc(sizeof(float) * (size_t)B * OR_MLP_IN);
    float* Y = (float*)malloc(sizeof(float) * (size_t)B * OR_MLP_OUT);
    or_mlp_inputs(c, t, X);
    or_mlp_forward(x, X, B, c->mlp_bf16, c->mlp_tanh_out, Y);
    double acc = 0.0;
    for (int64_t i = 0; i < (int64_t)B * OR_MLP_OUT; ++i) {
        double d = (double)Y[i] - (double)YT[i];
        acc += d * d;
    }
    free(X);
    free(Y);
    return (float)(-(acc / (double)((int64_t)B * OR_MLP_OUT)));
}

/* Fitness of the listed members js[0..nj) of run r at generation t. */
void or_eval_members(const or_config* c, int32_t run, uint32_t t, const float* m,
                     const float* pdata, const int32_t* js, int32_t nj, float* f)
{
    int64_t D = c->num_dims;
    float* YT = NULL;
    if (c->problem == OR_PROB_MLP) {
        YT = (float*)malloc(sizeof(float) * (size_t)c->mlp_batch * OR_MLP_OUT);
        or_mlp_teacher_out(c, pdata, t, YT);
    }
#pragma omp parallel
    {
        float* x = (float*)malloc(sizeof(float) * (size_t)D);
#pragma omp for schedule(static)
        for (int32_t i = 0; i < nj; ++i) {
            or_member(c, run, t, m, js[i], x);
            if (c->problem == OR_PROB_MLP) f[i] = or_mlp_fitness(c, x, t, YT);
            else f[i] = or_fitness_bbob(c->problem, x, D, pdata, c->rastrigin_a);
        }
        free(x);
    }
    free(YT);
}

/* ------------------------------------------------------------------------ */
/* tell, step 1: fitness shaping (Sec. 3.2 "centered rank"; App. B).         */
/* Readings: key = f (minimise, Listing 1) or -f (maximise); NaN is the      */
/* worst value (+inf key); -0 == +0.  rank = position in a stable ascending   */
/* sort, i.e. ties broken by member index.                                   */
/* ------------------------------------------------------------------------ */
static double or_key(float f, int32_t maximize)
{
    double k = maximize ? -(double)f : (double)f;
    if (isnan(k)) k = INFINITY;
    return k;
}

void or_ranks(const float* f, int32_t N, int32_t maximize, int32_t* rank)
{
    for (int32_t j = 0; j < N; ++j) {
        double kj = or_key(f[j], maximize);
        int32_t r = 0;
        for (int32_t k = 0; k < N; ++k) {
            double kk = or_key(f[k], maximize);
            if (kk < kj || (kk == kj && k < j)) ++r;
        }
        rank[j] = r;
    }
}

/* Centered rank y = rank/(N-1) - 1/2, written as the single fp32 quotient
 * (2 rank - (N-1)) / (2 (N-1)) of two exact integers (reading that fixes the
 * bits).  RAW (test mode): y = key.                                         */
void or_shape(const float* f, int32_t N, int32_t maximize, int32_t shaping, float* y)
{
    if (shaping == OR_SHAPE_RAW) {
        for (int32_t j = 0; j < N; ++j) y[j] = maximize ? -f[j] : f[j];
        return;
    }
    int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    or_ranks(f, N, maximize, rank);
    float den = (float)(2 * (N - 1));
    for (int32_t j = 0; j < N; ++j) y[j] = (float)(2 * rank[j] - (N - 1)) / den;
    free(rank);
}

/* The other shaping transformations Sec. 3.2 names next to centered ranks:
 * z-scoring and weight-decay regularisation.
 * Readings.  Weight decay penalises the mean square parameter of a member in
 * the minimisation sense: with pen_j = (1/D) sum_d x_jd^2 (fp32),
 *   key_j = fl32(k_j + fl32(w_decay * pen_j)),  k_j = f_j or -f_j (maximise);
 * a NaN fitness stays the worst key (+inf).  Ranks and raw shaping then use
 * these keys.  z-score: over the n finite keys, mean mu and population
 * standard deviation sd in fp64, y_j = fl32((key_j - mu) / (sd + 1e-10));
 * members with a non-finite key get y = 0.                                  */
float or_shaped_key(float f, float pen, int32_t maximize, float w_decay)
{
    float k = maximize ? -f : f;
    if (isnan(k)) return INFINITY;
    if (w_decay != 0.0f && isfinite(k)) k = k + w_decay * pen;
    return k;
}

void or_shape_full(const float* f, const float* pen, int32_t N, int32_t maximize, int32_t shaping,
                   float w_decay, float* y)
{
    float* key = (float*)malloc(sizeof(float) * (size_t)N);
    for (int32_t j = 0; j < N; ++j) key[j] = or_shaped_key(f[j], pen ? pen[j] : 0.0f, maximize, w_decay);
    if (shaping == OR_SHAPE_RAW) {
        for (int32_t j = 0; j < N; ++j) y[j] = key[j];
    } else if (shaping == OR_SHAPE_Z_SCORE) {
        double sum = 0.0, n = 0.0;
        for (int32_t j = 0; j < N; ++j)
            if (isfinite(key[j])) { sum += (double)key[j]; n += 1.0; }
        double mu = n > 0.0 ? sum / n : 0.0, ss = 0.0;
        for (int32_t j = 0; j < N; ++j)
            if (isfinite(key[j])) ss += ((double)key[j] - mu) * ((double)key[j] - mu);
        double sd = n > 0.0 ? sqrt(ss / n) : 0.0;
        for (int32_t j = 0; j < N; ++j)
            y[j] = isfinite(key[j]) ? (float)(((double)key[j] - mu) / (sd + 1e-10)) : 0.0f;
    } else {
        /* centered ranks of the keys: key already minimisation-oriented */
        float den = (float)(2 * (N - 1));
        for (int32_t j = 0; j < N; ++j) {
            int32_t r = 0;
            for (int32_t k = 0; k < N; ++k)
                if (key[k] < key[j] || (key[k] == key[j] && k < j)) ++r;
            y[j] = (float)(2 * r - (N - 1)) / den;
        }
    }
    free(key);
}

/* Mean square parameter of every member of run r at generation t,
 * pen_j = fl32((sum_d x_jd^2 in fp64) / D).                                 */
void or_penalty(const or_config* c, int32_t run, uint32_t t, const float* m, float* pen)
{
    int64_t D = c->num_dims;
#pragma omp parallel
    {
        float* x = (float*)malloc(sizeof(float) * (size_t)D);
#pragma omp for schedule(static)
        for (int32_t j = 0; j < c->popsize; ++j) {
            or_member(c, run, t, m, j, x);
            double acc = 0.0;
            for (int64_t d = 0; d < D; ++d) acc += (double)x[d] * (double)x[d];
            pen[j] = (float)(acc / (double)D);
        }
        free(x);
    }
}

/* Exponential decay with a floor (App. B schedules), fp32: max(x*decay, final). */
float or_decay(float x, float decay, float final)
{
    float y = x * decay;
    return y > final ? y : final;
}

/* ------------------------------------------------------------------------ */
/* tell, step 2: FD gradient estimate (Sec. 2.1 estimator) over the whole    */
/* population, g = E^T y / (N sigma), E the N x D matrix of perturbations    */
/* (row j = +eps_j or -eps_{j-N/2}).  fp64 accumulation, one fp32 rounding.  */
/* Computes dims [d0, d0+nd) only.                                           */
/* ------------------------------------------------------------------------ */
void or_grad(const or_config* c, int32_t run, uint32_t t, const float* y,
             int64_t d0, int64_t nd, float* g)
{
    int32_t N = c->popsize, half = N / 2;
    double scale = (double)N * (double)c->sigma;
    int64_t nch = (nd + OR_DIM_CHUNK - 1) / OR_DIM_CHUNK;
    /* blocks of dims in parallel; each dim sums over j = 0..N-1 in order */
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < nch; ++k) {
        int64_t a = k * OR_DIM_CHUNK, n = nd - a < OR_DIM_CHUNK ? nd - a : OR_DIM_CHUNK;
        double* acc = (double*)calloc((size_t)n, sizeof(double));
        float* eps = (float*)malloc(sizeof(float) * (size_t)n);
        for (int32_t j = 0; j < N; ++j) {
            int32_t p = j < half ? j : j - half;
            double sgn = j < half ? 1.0 : -1.0;
            or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)p, t, d0 + a, n, eps);
            for (int64_t i = 0; i < n; ++i) acc[i] += (double)y[j] * sgn * (double)eps[i];
        }
        for (int64_t i = 0; i < n; ++i) g[a + i] = (float)(acc[i] / scale);
        free(acc);
        free(eps);
    }
}

/* ------------------------------------------------------------------------ */
/* tell, step 3: Adam (Kingma & Ba 2015, Algorithm 1) on the mean; the paper  */
/* names Adam as the optimiser (Sec. 2.1; App. B) without a formula.         */
/* Reading: fp32 state, t' = t + 1 counted from 1, bias corrections          */
/* bc = 1 - beta^t' evaluated in fp64 and rounded to fp32, eps outside sqrt,  */
/* this exact fp32 operation order:                                          */
/*   m1 = fmaf(b1, m1, (1-b1)*g);  v = fmaf(b2, v, (1-b2)*(g*g));           */
/*   q = (m1/bc1) / (sqrt(v/bc2) + eps);  m = fmaf(-lr, q, m).               */
/* ------------------------------------------------------------------------ */
void or_adam(const or_config* c, int64_t t, const float* g, int64_t n, float* m, float* m1, float* v)
{
    double tp = (double)(t + 1);
    float bc1 = (float)(1.0 - pow((double)c->beta1, tp));
    float bc2 = (float)(1.0 - pow((double)c->beta2, tp));
    float omb1 = (float)(1.0 - (double)c->beta1);
    float omb2 = (float)(1.0 - (double)c->beta2);
    for (int64_t i = 0; i < n; ++i) {
        float gi = g[i];
        float a = omb1 * gi;
        float nm1 = fmaf(c->beta1, m1[i], a);
        float gg = gi * gi;
        float b = omb2 * gg;
        float nv = fmaf(c->beta2, v[i], b);
        float mhat = nm1 / bc1;
        float vhat = nv / bc2;
        float den = sqrtf(vhat) + c->eps;
        float q = mhat / den;
        m[i] = fmaf(-c->lr, q, m[i]);
        m1[i] = nm1;
        v[i] = nv;
    }
}

/* ------------------------------------------------------------------------ */
/* Two weighted noise sums over the pairs, fp64:                             */
/*   A_d = sum_p a_p z_pd,   B_d = sum_p b_p (z_pd^2 - 1).                    */
/* ------------------------------------------------------------------------ */
void or_noise_sums(const or_config* c, int32_t run, uint32_t t, const float* a, const float* b,
                   double* A, double* B)
{
    int32_t P = c->popsize / 2;
    int64_t D = c->num_dims;
    int64_t nch = (D + OR_DIM_CHUNK - 1) / OR_DIM_CHUNK;
    /* blocks of dims in parallel; each dim sums over the pairs in order */
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < nch; ++k) {
        int64_t d0 = k * OR_DIM_CHUNK, n = D - d0 < OR_DIM_CHUNK ? D - d0 : OR_DIM_CHUNK;
        float* z = (float*)malloc(sizeof(float) * (size_t)n);
        for (int64_t d = d0; d < d0 + n; ++d) { A[d] = 0.0; B[d] = 0.0; }
        for (int32_t p = 0; p < P; ++p) {
            or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)p, t, d0, n, z);
            for (int64_t i = 0; i < n; ++i) {
                double zd = (double)z[i];
                A[d0 + i] += (double)a[p] * zd;
                B[d0 + i] += (double)b[p] * (zd * zd - 1.0);
            }
        }
        free(z);
    }
}

/* Error-bound helper for the tests (no step of the method): the fp64 sum   */
/* S_d = sum_p |a_p| |z_pd| over the pairs, the factor by which the normals' */
/* error bound moves a weighted noise sum such as the gradient's.            */
void or_abs_noise_sum(const or_config* c, int32_t run, uint32_t t, const float* a, double* S)
{
    int32_t P = c->popsize / 2;
    int64_t D = c->num_dims;
    int64_t nch = (D + OR_DIM_CHUNK - 1) / OR_DIM_CHUNK;
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < nch; ++k) {
        int64_t d0 = k * OR_DIM_CHUNK, n = D - d0 < OR_DIM_CHUNK ? D - d0 : OR_DIM_CHUNK;
        float* z = (float*)malloc(sizeof(float) * (size_t)n);
        for (int64_t d = d0; d < d0 + n; ++d) S[d] = 0.0;
        for (int32_t p = 0; p < P; ++p) {
            or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)p, t, d0, n, z);
            for (int64_t i = 0; i < n; ++i) S[d0 + i] += fabs((double)a[p]) * fabs((double)z[i]);
        }
        free(z);
    }
}

/* ClipUp (Toklu et al. 2020), the ES-adapted optimiser named in Sec. 3.1,
 * for minimisation.  Reading: with the fp64 norms |g| and |v'|,
 *   gh_d = fl32(g_d * fl32(1/|g|))          (0 when |g| = 0)
 *   v'_d = fmaf(lr, gh_d, fl32(momentum * v_d))
 *   v_d  = |v'| > max_speed ? fl32(v'_d * fl32(max_speed / |v'|)) : v'_d
 *   m_d  = m_d - v_d.                                                       */
void or_clipup(const or_config* c, float lr, const float* g, int64_t n, float* m, float* vel)
{
    double gg = 0.0;
    for (int64_t i = 0; i < n; ++i) gg += (double)g[i] * (double)g[i];
    float inv = gg > 0.0 ? (float)(1.0 / sqrt(gg)) : 0.0f;
    double vv = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        float gh = g[i] * inv;
        float mv = c->clipup_momentum * vel[i];
        vel[i] = fmaf(lr, gh, mv);
        vv += (double)vel[i] * (double)vel[i];
    }
    double nv = sqrt(vv);
    if (nv > (double)c->clipup_max_speed) {
        float sc = (float)((double)c->clipup_max_speed / nv);
        for (int64_t i = 0; i < n; ++i) vel[i] = vel[i] * sc;
    }
    for (int64_t i = 0; i < n; ++i) m[i] = m[i] - vel[i];
}

/* SNES utilities (App. B, SNES table): w_j = softmax(beta (rank'_j/N - 1/2))
 * with rank'_j = N - 1 - rank_j, so that the best member (rank 0 of the
 * minimisation keys) has the largest weight.  rank' is a permutation of
 * 0..N-1, so the weights form a table indexed by rank'; fp64, one fp32
 * rounding each.                                                           */
void or_snes_table(int32_t N, float beta, float* w)
{
    double S = 0.0;
    for (int32_t k = 0; k < N; ++k) S += exp((double)beta * ((double)k / (double)N - 0.5));
    for (int32_t k = 0; k < N; ++k) w[k] = (float)(exp((double)beta * ((double)k / (double)N - 0.5)) / S);
}

/* Ranks of the shaped minimisation keys (weight decay included). */
static void or_key_ranks(const float* f, const float* pen, int32_t N, int32_t maximize, float w_decay,
                         int32_t* rank)
{
    float* key = (float*)malloc(sizeof(float) * (size_t)N);
    for (int32_t j = 0; j < N; ++j) key[j] = or_shaped_key(f[j], pen ? pen[j] : 0.0f, maximize, w_decay);
    for (int32_t j = 0; j < N; ++j) {
        int32_t r = 0;
        for (int32_t k = 0; k < N; ++k)
            if (key[k] < key[j] || (key[k] == key[j] && k < j)) ++r;
        rank[j] = r;
    }
    free(key);
}

/* PGPE tell (Sehnke et al. 2010, symmetric sampling; FDG row of Table 1;
 * App. B PGPE table: sigma learning rate and maximum change).  Readings, for
 * shaped weights y (low = good) and pairs p with x = m +- sigma (.) z_p:
 *   mean gradient  g_d = fl32(sigma_d A_d / N),  a_p = y_p - y_{p+P};
 *   sigma gradient s_d = fl32(sigma_d B_d / P),  b_p = fl32((y_p + y_{p+P})/2 - ybar),
 *                  ybar the fp64 mean of y;
 *   mean step: the optimiser (Adam, or ClipUp) on g with learning rate lr;
 *   sigma step: dlt = -(sigma_lr * s_d), clipped to +- fl32(max_change * sigma_d),
 *                  sigma_d + dlt, then the schedule max(fl32(sigma*decay), final). */
void or_pgpe_update(const or_config* c, int32_t run, int64_t t, float lr, const float* y, float* m,
                    float* m1, float* v, float* vel, float* sig, float* g_out)
{
    int32_t N = c->popsize, P = N / 2;
    int64_t D = c->num_dims;
    double ybar = 0.0;
    for (int32_t j = 0; j < N; ++j) ybar += (double)y[j];
    ybar /= (double)N;
    float* a = (float*)malloc(sizeof(float) * (size_t)P);
    float* b = (float*)malloc(sizeof(float) * (size_t)P);
    for (int32_t p = 0; p < P; ++p) {
        a[p] = y[p] - y[p + P];
        b[p] = (float)(0.5 * ((double)y[p] + (double)y[p + P]) - ybar);
    }
    double* A = (double*)malloc(sizeof(double) * (size_t)D);
    double* B = (double*)malloc(sizeof(double) * (size_t)D);
    or_noise_sums(c, run, (uint32_t)t, a, b, A, B);
    float* g = (float*)malloc(sizeof(float) * (size_t)D);
    for (int64_t d = 0; d < D; ++d) g[d] = (float)((double)sig[d] * A[d] / (double)N);
    if (c->optimizer == OR_OPT_CLIPUP) {
        or_clipup(c, lr, g, D, m, vel);
    } else {
        or_config cc = *c;
        cc.lr = lr;
        or_adam(&cc, t, g, D, m, m1, v);
    }
    for (int64_t d = 0; d < D; ++d) {
        float sg = (float)((double)sig[d] * B[d] / (double)P);
        float dlt = -(c->sigma_lr * sg);
        float lim = c->sigma_max_change * sig[d];
        if (dlt > lim) dlt = lim;
        if (dlt < -lim) dlt = -lim;
        float ns = sig[d] + dlt;
        sig[d] = or_decay(ns, c->sigma_decay, c->sigma_final);
    }
    if (g_out) memcpy(g_out, g, sizeof(float) * (size_t)D);
    free(a); free(b); free(A); free(B); free(g);
}

/* SNES tell (Schaul et al. 2011; PFD row of Table 1) with the softmax rank
 * utilities of App. B.  Readings: w_j from or_snes_table over rank'_j (ranks
 * of the shaped keys, weight decay included); a_p = w_p - w_{p+P},
 * b_p = w_p + w_{p+P};
 *   m_d     = fmaf(fl32(lr * sigma_d), fl32(A_d), m_d)            (lr = eta_m)
 *   sigma_d = fl32(sigma_d * expf(fl32(fl32(sigma_lr / 2) * fl32(B_d)))),
 * then the sigma schedule.                                                 */
void or_snes_update(const or_config* c, int32_t run, int64_t t, float lr, const float* f, const float* pen,
                    float* m, float* sig, float* w_out)
{
    int32_t N = c->popsize, P = N / 2;
    int64_t D = c->num_dims;
    int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    or_key_ranks(f, pen, N, c->maximize, c->w_decay, rank);
    float* tab = (float*)malloc(sizeof(float) * (size_t)N);
    or_snes_table(N, c->snes_temperature, tab);
    float* w = (float*)malloc(sizeof(float) * (size_t)N);
    for (int32_t j = 0; j < N; ++j) w[j] = tab[N - 1 - rank[j]];
    float* a = (float*)malloc(sizeof(float) * (size_t)P);
    float* b = (float*)malloc(sizeof(float) * (size_t)P);
    for (int32_t p = 0; p < P; ++p) {
        a[p] = w[p] - w[p + P];
        b[p] = w[p] + w[p + P];
    }
    double* A = (double*)malloc(sizeof(double) * (size_t)D);
    double* B = (double*)malloc(sizeof(double) * (size_t)D);
    or_noise_sums(c, run, (uint32_t)t, a, b, A, B);
    float h = 0.5f * c->sigma_lr;
    for (int64_t d = 0; d < D; ++d) {
        m[d] = fmaf(lr * sig[d], (float)A[d], m[d]);
        float ns = sig[d] * expf(h * (float)B[d]);
        sig[d] = or_decay(ns, c->sigma_decay, c->sigma_final);
    }
    if (w_out) memcpy(w_out, w, sizeof(float) * (size_t)N);
    free(rank); free(tab); free(w); free(a); free(b); free(A); free(B);
}

/* ------------------------------------------------------------------------ */
/* Sep-CMA-ES (Ros & Hansen 2008; EOD row of Table 1, App. B table: sigma    */
/* init and elite ratio).  Readings (the paper gives no formula; these are   */
/* the standard CMA-ES settings of Hansen's tutorial with the separable      */
/* learning-rate scaling (D+2)/3 of Ros & Hansen):                           */
/*   mu = max(1, floor(ratio N)); w_i = (ln(mu + 1/2) - ln(i+1)) / sum,      */
/*   i = 0..mu-1 by rank; mu_eff = 1/sum w^2;                                */
/*   c_s = (mu_eff + 2)/(D + mu_eff + 5);                                    */
/*   d_s = 1 + 2 max(0, sqrt((mu_eff-1)/(D+1)) - 1) + c_s;                   */
/*   c_c = (4 + mu_eff/D)/(D + 4 + 2 mu_eff/D);                              */
/*   c1 = 2/((D+1.3)^2 + mu_eff);                                            */
/*   cmu = min(1 - c1, 2 (mu_eff - 2 + 1/mu_eff)/((D+2)^2 + mu_eff));        */
/*   separable: c1s = min(1, c1 (D+2)/3), cmus = min(1 - c1s, cmu (D+2)/3);  */
/*   chi = sqrt(D) (1 - 1/(4D) + 1/(21 D^2)).                                */
/* Sampling: s_d = fl32(sigma sqrtf(C_d)), x_j = fmaf(s, z_j, m) with z_j    */
/* the Philox normals of row j (independent members, no mirroring).          */
/* ------------------------------------------------------------------------ */
typedef struct {
    int32_t mu;
    double mu_eff, c_s, d_s, c_c, c1, cmu, chi;
} or_cma_consts;

int32_t or_cma_mu(const or_config* c)
{
    int32_t mu = (int32_t)floor((double)c->elite_ratio * (double)c->popsize);
    return mu < 1 ? 1 : mu;
}

void or_cma_weights(const or_config* c, double* w)
{
    int32_t mu = or_cma_mu(c);
    double s = 0.0;
    for (int32_t i = 0; i < mu; ++i) {
        w[i] = log((double)mu + 0.5) - log((double)(i + 1));
        s += w[i];
    }
    for (int32_t i = 0; i < mu; ++i) w[i] /= s;
}

static or_cma_consts or_cma_setup(const or_config* c, const double* w)
{
    or_cma_consts k;
    double D = (double)c->num_dims, s2 = 0.0;
    k.mu = or_cma_mu(c);
    for (int32_t i = 0; i < k.mu; ++i) s2 += w[i] * w[i];
    k.mu_eff = 1.0 / s2;
    k.c_s = (k.mu_eff + 2.0) / (D + k.mu_eff + 5.0);
    double q = sqrt((k.mu_eff - 1.0) / (D + 1.0)) - 1.0;
    k.d_s = 1.0 + 2.0 * (q > 0.0 ? q : 0.0) + k.c_s;
    k.c_c = (4.0 + k.mu_eff / D) / (D + 4.0 + 2.0 * k.mu_eff / D);
    double c1 = 2.0 / ((D + 1.3) * (D + 1.3) + k.mu_eff);
    double cmu = 2.0 * (k.mu_eff - 2.0 + 1.0 / k.mu_eff) / ((D + 2.0) * (D + 2.0) + k.mu_eff);
    if (cmu > 1.0 - c1) cmu = 1.0 - c1;
    k.c1 = c1 * (D + 2.0) / 3.0;
    if (k.c1 > 1.0) k.c1 = 1.0;
    k.cmu = cmu * (D + 2.0) / 3.0;
    if (k.cmu > 1.0 - k.c1) k.cmu = 1.0 - k.c1;
    k.chi = sqrt(D) * (1.0 - 1.0 / (4.0 * D) + 1.0 / (21.0 * D * D));
    return k;
}

void or_cma_scale(int64_t D, float sigma, const float* C, float* s)
{
    for (int64_t d = 0; d < D; ++d) s[d] = sigma * sqrtf(C[d]);
}

/* One Sep-CMA-ES tell.  Elites e_i = the member of rank i (shaped keys,
 * weight decay included); zw_d = sum_i w_i z_{e_i,d}, q_d = sum_i w_i
 * z_{e_i,d}^2 (fp64).  Then, in fp64 from the fp32 state, one rounding per
 * stored value, with s the generation's sampling scale:
 *   m_d   = m_d + s_d zw_d
 *   ps_d  = (1 - c_s) ps_d + sqrt(c_s (2 - c_s) mu_eff) zw_d
 *   h     = |ps| / sqrt(1 - (1 - c_s)^(2(t+1))) < (1.4 + 2/(D+1)) chi
 *   pc_d  = (1 - c_c) pc_d + h sqrt(c_c (2 - c_c) mu_eff) sqrt(C_d) zw_d
 *   C_d   = (1 - c1s - cmus) C_d + c1s (pc_d^2 + (1 - h) c_c (2 - c_c) C_d)
 *           + cmus C_d q_d
 *   sigma = sigma exp((c_s / d_s) (|ps| / chi - 1)).                       */
void or_sepcma_update(const or_config* c, int32_t run, int64_t t, const float* f, const float* pen, float* m,
                      float* sigma, float* C, float* ps, float* pc, const float* s, float* w_out)
{
    int32_t N = c->popsize;
    int64_t D = c->num_dims;
    double* w = (double*)malloc(sizeof(double) * (size_t)N);
    or_cma_weights(c, w);
    or_cma_consts k = or_cma_setup(c, w);
    int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    or_key_ranks(f, pen, N, c->maximize, c->w_decay, rank);
    int32_t* elite = (int32_t*)malloc(sizeof(int32_t) * (size_t)k.mu);
    for (int32_t j = 0; j < N; ++j)
        if (rank[j] < k.mu) elite[rank[j]] = j;
    double* zw = (double*)calloc((size_t)D, sizeof(double));
    double* q = (double*)calloc((size_t)D, sizeof(double));
    int64_t nch = (D + OR_DIM_CHUNK - 1) / OR_DIM_CHUNK;
    /* blocks of dims in parallel; each dim sums over the elites in order */
#pragma omp parallel for schedule(static)
    for (int64_t kc = 0; kc < nch; ++kc) {
        int64_t d0 = kc * OR_DIM_CHUNK, n = D - d0 < OR_DIM_CHUNK ? D - d0 : OR_DIM_CHUNK;
        float* z = (float*)malloc(sizeof(float) * (size_t)n);
        for (int32_t i = 0; i < k.mu; ++i) {
            or_normals(c->seed + (uint64_t)run, OR_DOM_NOISE, (uint32_t)elite[i], (uint32_t)t, d0, n, z);
            for (int64_t e = 0; e < n; ++e) {
                zw[d0 + e] += w[i] * (double)z[e];
                q[d0 + e] += w[i] * (double)z[e] * (double)z[e];
            }
        }
        free(z);
    }
    double a_s = sqrt(k.c_s * (2.0 - k.c_s) * k.mu_eff), n2 = 0.0;
    for (int64_t d = 0; d < D; ++d) {
        m[d] = (float)((double)m[d] + (double)s[d] * zw[d]);
        ps[d] = (float)((1.0 - k.c_s) * (double)ps[d] + a_s * zw[d]);
        n2 += (double)ps[d] * (double)ps[d];
    }
    double nps = sqrt(n2);
    double hth = nps / sqrt(1.0 - pow(1.0 - k.c_s, 2.0 * (double)(t + 1)));
    double h = hth < (1.4 + 2.0 / ((double)D + 1.0)) * k.chi ? 1.0 : 0.0;
    double a_c = sqrt(k.c_c * (2.0 - k.c_c) * k.mu_eff);
    for (int64_t d = 0; d < D; ++d) {
        double Cd = (double)C[d];
        pc[d] = (float)((1.0 - k.c_c) * (double)pc[d] + h * a_c * sqrt(Cd) * zw[d]);
        double pcd = (double)pc[d];
        C[d] = (float)((1.0 - k.c1 - k.cmu) * Cd + k.c1 * (pcd * pcd + (1.0 - h) * k.c_c * (2.0 - k.c_c) * Cd)
                       + k.cmu * Cd * q[d]);
    }
    *sigma = (float)((double)*sigma * exp((k.c_s / k.d_s) * (nps / k.chi - 1.0)));
    if (w_out)
        for (int32_t j = 0; j < N; ++j) w_out[j] = rank[j] < k.mu ? (float)w[rank[j]] : 0.0f;
    free(w); free(rank); free(elite); free(zw); free(q);
}

void or_generation_ex(const or_config* c0, int32_t run, int64_t t, const float* pdata,
                      float* m, float* m1, float* v, float* vel, float* sig, float* sigma_out,
                      const float* fit_in,
                      float* fit_out, float* y_out, float* g_out,
                      double* best_key, float* best_f, float* best_x);

/* ------------------------------------------------------------------------ */
/* One generation of one run (ask -> evaluate -> tell), the body of the      */
/* scanned loop of Sec. 2.2 (Listing 2).  fit_in != NULL replaces the        */
/* built-in evaluation (the user's own evaluate step).  Best-so-far member   */
/* and fitness (state fields of Listing 1) are updated from the generation's */
/* rank-0 member when it is strictly better.                                 */
/* Outputs (any may be NULL): fit_out[N], y_out[N], g_out[D].                 */
/* best_key / best_f / best_x carry the best-so-far state.                   */
/* ------------------------------------------------------------------------ */
void or_generation(const or_config* c, int32_t run, int64_t t, const float* pdata,
                   float* m, float* m1, float* v, const float* fit_in,
                   float* fit_out, float* y_out, float* g_out,
                   double* best_key, float* best_f, float* best_x)
{
    or_generation_ex(c, run, t, pdata, m, m1, v, NULL, NULL, NULL, fit_in, fit_out, y_out, g_out, best_key,
                     best_f, best_x);
}

/* As or_generation, for every strategy: vel = ClipUp velocity (or NULL),
 * sig = per-dimension sigma (PGPE, SNES; updated in place, and used as
 * c->sigma_vec for the sampling).  Sep-CMA-ES keeps C in sig, p_sigma in
 * m1 and p_c in v, and returns the run's new sigma in *sigma_out.          */
void or_generation_ex(const or_config* c0, int32_t run, int64_t t, const float* pdata,
                      float* m, float* m1, float* v, float* vel, float* sig, float* sigma_out,
                      const float* fit_in,
                      float* fit_out, float* y_out, float* g_out,
                      double* best_key, float* best_f, float* best_x)
{
    or_config cfg = *c0;
    const or_config* c = &cfg;
    float* scale = NULL;
    if (cfg.strategy == OR_STRAT_SEP_CMA) {
        /* state: sig = C, m1 = p_sigma, v = p_c; sampling scale sigma sqrt(C) */
        scale = (float*)malloc(sizeof(float) * (size_t)cfg.num_dims);
        or_cma_scale(cfg.num_dims, cfg.sigma, sig, scale);
        cfg.sigma_vec = scale;
    } else if (cfg.strategy != OR_STRAT_OPENAI_ES) {
        cfg.sigma_vec = sig;
    }
    int32_t N = c->popsize;
    int64_t D = c->num_dims;
    float* f = (float*)malloc(sizeof(float) * (size_t)N);
    float* y = (float*)malloc(sizeof(float) * (size_t)N);
    float* g = (float*)malloc(sizeof(float) * (size_t)D);
    int32_t* rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    if (fit_in) {
        memcpy(f, fit_in, sizeof(float) * (size_t)N);
    } else {
        int32_t* js = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
        for (int32_t j = 0; j < N; ++j) js[j] = j;
        or_eval_members(c, run, (uint32_t)t, m, pdata, js, N, f);
        free(js);
    }
    or_ranks(f, N, c->maximize, rank);
    int32_t jbest = 0;
    for (int32_t j = 0; j < N; ++j)
        if (rank[j] == 0) jbest = j;
    double kb = or_key(f[jbest], c->maximize);
    if (best_key && kb < *best_key) {
        *best_key = kb;
        if (best_f) *best_f = f[jbest];
        if (best_x) or_member(c, run, (uint32_t)t, m, jbest, best_x);
    }
    float* pen = NULL;
    if (c->w_decay != 0.0f) {
        pen = (float*)malloc(sizeof(float) * (size_t)N);
        or_penalty(c, run, (uint32_t)t, m, pen);
    }
    if (c->strategy == OR_STRAT_SEP_CMA) {
        float sg = c->sigma;
        or_sepcma_update(c, run, t, f, pen, m, &sg, sig, m1, v, scale, y);
        if (sigma_out) *sigma_out = sg;
        for (int64_t d = 0; d < D; ++d) g[d] = 0.0f;
    } else if (c->strategy == OR_STRAT_SNES) {
        /* m and sigma move together; sig is also c->sigma_vec */
        float* snew = (float*)malloc(sizeof(float) * (size_t)D);
        memcpy(snew, sig, sizeof(float) * (size_t)D);
        or_snes_update(c, run, t, c->lr, f, pen, m, snew, y);
        memcpy(sig, snew, sizeof(float) * (size_t)D);
        free(snew);
        for (int64_t d = 0; d < D; ++d) g[d] = 0.0f;
    } else {
        if (c->w_decay != 0.0f || c->shaping == OR_SHAPE_Z_SCORE)
            or_shape_full(f, pen, N, c->maximize, c->shaping, c->w_decay, y);
        else
            or_shape(f, N, c->maximize, c->shaping, y);
        if (c->strategy == OR_STRAT_PGPE) {
            float* snew = (float*)malloc(sizeof(float) * (size_t)D);
            memcpy(snew, sig, sizeof(float) * (size_t)D);
            or_pgpe_update(c, run, t, c->lr, y, m, m1, v, vel, snew, g);
            memcpy(sig, snew, sizeof(float) * (size_t)D);
            free(snew);
        } else {
            or_grad(c, run, (uint32_t)t, y, 0, D, g);
            if (c->optimizer == OR_OPT_CLIPUP) or_clipup(c, c->lr, g, D, m, vel);
            else or_adam(c, t, g, D, m, m1, v);
        }
    }
    free(pen);
    free(scale);
    if (fit_out) memcpy(fit_out, f, sizeof(float) * (size_t)N);
    if (y_out) memcpy(y_out, y, sizeof(float) * (size_t)N);
    if (g_out) memcpy(g_out, g, sizeof(float) * (size_t)D);
    free(f);
    free(y);
    free(g);
    free(rank);
}
