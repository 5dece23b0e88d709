// es_internal.hpp -- host-side declarations shared by the runtime (es_api.cpp)
// and the kernel launchers (es_kernels.hip).  Not part of the C-ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "es_teacher.hpp"
#include "esmi.h"

namespace esmi {

// Shapes of one strategy.  State rows are padded to Dp = 4 * nb floats so
// that every Philox block of four dims is one aligned float4.
struct Geometry {
    int64_t D;   // dims
    int64_t nb;  // Philox blocks per member, ceil(D / 4)
    int64_t Dp;  // padded row stride, 4 * nb
    int32_t N;   // population
    int32_t P;   // antithetic pairs, N / 2
    int32_t R;   // runs
};

// Adam constants of one step (host-rounded to fp32).
// Sep-CMA-ES settings (host-computed in fp64 from D, N and the elite ratio).
struct CmaConsts {
    int32_t mu;
    double mu_eff, c_s, d_s, c_c, c1, cmu, chi;
    double a_s, a_c;  // sqrt(c_s (2 - c_s) mu_eff), sqrt(c_c (2 - c_c) mu_eff)
    double wsum;      // sum of the fp32 recombination weights
};

// Adam constants of one generation (the learning rate is per run, beside sigma).
struct AdamConsts {
    float beta1, beta2, omb1, omb2, bc1, bc2, eps;
};

// Geometry of the fused sample+evaluate launch: pair groups of `wg` lanes,
// D split into chunks of `bc` Philox blocks; one fp32 partial sum per
// (chunk, run, member).
struct EvalPlan {
    int32_t wg;       // lanes (pairs) per workgroup
    int32_t n_pg;     // pair groups per run
    int64_t bc;       // blocks per chunk
    int64_t nchunks;  // chunks per member
};
EvalPlan eval_plan(const Geometry& g, int64_t bc_override);
int64_t eval_partial_elems(const Geometry& g, const EvalPlan& e);  // floats

hipError_t launch_init(const Geometry& g, const es_config& c, float* m, float* m1, float* v,
                       float* best_x, hipStream_t s);
hipError_t launch_problem_data(const Geometry& g, const es_config& c, float* pdata, hipStream_t s);
hipError_t launch_fill_rows(const Geometry& g, float* p, float value, hipStream_t s);  // [R][Dp], padding 0
hipError_t launch_cma_scale(const Geometry& g, float* svec, const float* C, const float* hp, hipStream_t s);
// hp: device [2][R], sigma then lr of every run for the current generation.
// svec: per-dimension sigma [R][Dp] (PGPE, SNES) or null.
hipError_t launch_ask(const Geometry& g, const es_config& c, uint32_t t, const float* m, float* x,
                      const float* hp, const float* svec, hipStream_t s);
// ev_start / ev_stop (either may be null): events that record the start and
// the end of the main evaluate kernel (es_eval_timed).
hipError_t launch_eval_bbob(const Geometry& g, const es_config& c, const EvalPlan& e, uint32_t t,
                            const float* m, const float* pdata, float* partial, float* fit,
                            const float* hp, const float* svec, double div, hipStream_t s,
                            hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// Sort-based ranks (populations beyond RANK_MAX_N, or on request): the
// composite keys run << (32 + bn) | order key << bn | member of all runs,
// sorted ascending over their low 32 + bn + br bits in one device-wide sort
// (bn, br: the bits of the largest member and run index; with R N < 2^31,
// 2^(bn + br) < 4 R N, so the key fits 64 bits).
struct RankSortBuffers {
    uint64_t* kin;     // [R][N] composite keys
    uint64_t* kout;    // [R][N] sorted (runs in order)
    uint32_t* keys;    // [R][N] shaped order keys
    double* stats;     // [R][4] per-run statistics of the shaped keys
    void* temp;        // sort scratch
    size_t temp_bytes;
    int32_t bn, br;    // member and run index bits
};
void rank_sort_bits(const Geometry& g, int32_t* bn, int32_t* br);
size_t rank_sort_temp_bytes(const Geometry& g);                                  // 0 on failure
hipError_t launch_rank_sort(const Geometry& g, const RankSortBuffers& rs, hipStream_t s);  // kin -> kout
// table: the shaping table indexed by rank (centered ranks, or SNES
// utilities by rank), ybar_table its mean; bfold: PGPE / SNES second weight;
// rs: sort-based ranks (null: counted in LDS, N <= RANK_MAX_N).
hipError_t launch_rank(const Geometry& g, const es_config& c, const float* fit, const float* pen,
                       const float* table, double ybar_table, float* y, int32_t* rank, float* wfold, float* bfold,
                       int32_t* elite, int32_t mu, uint32_t* best_okey, float* best_f, int32_t* best_j,
                       float* gen_best, const float* hp_cur, float* hp_next, const RankSortBuffers* rs,
                       hipStream_t s);
// Split of the gradient kernel's pairs: ps pair slices (one wave each) per
// workgroup, nsplit workgroups per group of 64 Philox blocks.  With nsplit > 1
// every workgroup stores its partial sums (part, fp64 [R][nsplit][nb][4]) and
// a second kernel adds them in split order and applies Adam.
struct TellPlan {
    int32_t ps = 1;
    int32_t nsplit = 1;
    int32_t sub = 1;  // lanes per Philox block (4: sub-slices of the pairs)
};
TellPlan tell_plan(const Geometry& g, bool fused_path, int64_t force_nsplit);
size_t tell_part_elems(const Geometry& g, const TellPlan& tp, int strategy);  // doubles
size_t tell_groups(const Geometry& g);  // groups of 64 Philox blocks per run

// Device buffers of one tell (null where the strategy has none).
struct TellBuffers {
    const float* wfold;    // [R][P]
    const float* bfold;    // [R][P] PGPE / SNES
    const int32_t* best_j; // [R]
    float* m;
    float* m1;
    float* v;
    float* grad;           // [R][Dp] with ES_FLAG_KEEP_GRAD
    float* best_x;
    float* sig;            // [R][Dp] PGPE / SNES per-dimension sigma
    float* vel;            // [R][Dp] ClipUp velocity
    float* gbuf;           // [R][Dp] ClipUp gradient
    double* gpart;         // [R][groups] ClipUp |g|^2 partials
    double* vpart;         // [R][groups] ClipUp |v|^2 partials
    double* part;          // split partial sums
    const float* hp;       // [2][R] sigma, lr
    float* hp_next;        // [2][R] next generation's (Sep-CMA-ES stores sigma')
    const int32_t* elite;  // [R][N] Sep-CMA-ES elites by rank
    const float* cw;       // [mu] recombination weights
    double* zw;            // [R][Dp]
    double* qd;            // [R][Dp]
    float* cmaC;           // [R][Dp] diagonal covariance
    CmaConsts cma;
    // MLP: the next generation's teacher work, run by MLP_BATCH extra
    // workgroups of the gradient launch (teacher.w null: none)
    TeacherJob teacher{};
};
hipError_t launch_tell(const Geometry& g, const es_config& c, const TellPlan& tp, uint32_t t, const AdamConsts& a,
                       const TellBuffers& tb, hipStream_t s);
// Whether the gradient launch of this plan can run teacher rows (tb.teacher).
bool tell_carries_teacher(const es_config& c, const TellPlan& tp);
hipError_t launch_debug_noise(const Geometry& g, const es_config& c, int32_t run, uint32_t t,
                              int32_t pair, uint32_t* words, float* eps, hipStream_t s);

// Pair slices of the gradient kernel (one wave each); the fused loop uses
// the same split so that both paths sum in the same order.
int32_t tell_slices(const Geometry& g);

// Fused multi-generation loop (one workgroup per run, state in LDS).
constexpr size_t FUSED_MAX_LDS = 60 * 1024;
size_t fused_lds_bytes(const Geometry& g, const EvalPlan& e);
// Whether the fused loop keeps the normals in LDS for the gradient (they fit)
bool fused_stash(const Geometry& g, const EvalPlan& e);
bool fused_supported(const Geometry& g, const EvalPlan& e, const es_config& c);
// Generations per fused launch: their Adam bias corrections (bcorr[i] =
// {bc1, bc2} of generation t0 + i) travel in the kernel arguments, so a
// launch needs no staging buffer; es_run splits longer runs into launches.
constexpr int32_t FUSED_MAX_T = 256;
hipError_t launch_run_fused(const Geometry& g, const es_config& c, const EvalPlan& e, uint32_t t0, int32_t T,
                            const AdamConsts& ac, const float (*bcorr)[2], float* m, float* m1, float* v, float* grad,
                            float* best_x, uint32_t* best_okey, float* best_f, const float* pdata, const float* table,
                            float* log, float* hp, hipStream_t s);

// Grid loop: T generations of each run on a cooperative launch of G
// workgroups per run, in the per-call plans' summation order.  words:
// grid_word_count tagged 64-bit words (slice sums, fitnesses, shaped weights,
// rank-0 members, Rosenbrock's chunk boundaries), zero at set-up and never
// cleared; seq: the launch's sequence number in [1, 2^24), different from
// the previous launch's, so that no word left by an earlier launch carries a
// tag this one waits for; err: set when a wait gave up (only a wrong kernel
// can make it).
constexpr int32_t GRID_MAX_G = 16;
constexpr int32_t GRID_MAX_N = 8192;            // every workgroup ranks the run's members
constexpr size_t GRID_MAX_LDS = 144 * 1024;     // of gfx950's 160 KB per workgroup
// es_run takes the grid loop by default up to this many pair-blocks (R P nb)
constexpr int64_t GRID_DEFAULT_WORK = 1 << 20;
int32_t grid_workgroups(const Geometry& g, const EvalPlan& e, int32_t want);  // want 0: the library's choice
inline size_t grid_word_count(const Geometry& g, const EvalPlan& e)
{
    return (size_t)g.R * ((size_t)16 * g.N * 2 + 2 * (size_t)g.N + 1 + (size_t)e.nchunks);
}
size_t grid_lds_bytes(const Geometry& g, const EvalPlan& e, const TellPlan& tp, int32_t G);
bool grid_supported(const Geometry& g, const EvalPlan& e, const TellPlan& tp, const es_config& c, int32_t G);
hipError_t grid_max_resident(int64_t* out);  // workgroups of the grid loop the device holds at once
hipError_t launch_run_grid(const Geometry& g, const es_config& c, const EvalPlan& e, const TellPlan& tp, int32_t G,
                           int32_t xs,
                           uint32_t t0, int32_t T, const AdamConsts& ac, const float (*bcorr)[2], float* m, float* m1,
                           float* v, float* grad, float* best_x, uint32_t* best_okey, float* best_f,
                           const float* pdata, const float* table, float* log, uint64_t* words, uint32_t seq,
                           uint32_t* err, float* hp, hipStream_t s);

// Neuroevolution problem (64-256-256-16 MLP vs a teacher).
constexpr int64_t MLP_NUM_PARAMS = 86544;
size_t mlp_scratch_bytes();  // X_t (fp32 and bf16), teacher outputs, transposed teacher
hipError_t launch_mlp_setup(const float* teacher, void* scratch, hipStream_t s);
size_t mlp_lds_bytes();
// run_teacher: also compute X_t and Y_T first (else the gradient launch of
// the previous generation left them in scratch).
hipError_t launch_eval_mlp(const Geometry& g, const es_config& c, uint32_t t, const float* m, const float* teacher,
                           void* scratch, float* fit, const float* hp, const float* svec, bool run_teacher,
                           hipStream_t s, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// The teacher work of generation t (X_t, Y_T into scratch).
TeacherJob mlp_teacher_job(const es_config& c, const float* teacher, void* scratch, uint32_t t);

// A kernel launch that, given events, has the dispatch itself record its start
// and end (hipExtLaunchKernel), so no marker packet sits between kernels.
template <typename... KArgs, typename... Args>
hipError_t launch_timed(void (*k)(KArgs...), dim3 grid, dim3 block, uint32_t lds, hipStream_t s, hipEvent_t ev_start,
                        hipEvent_t ev_stop, Args... args)
{
    if (!ev_start && !ev_stop) k<<<grid, block, lds, s>>>(args...);
    else hipExtLaunchKernelGGL(k, grid, block, lds, s, ev_start, ev_stop, 0u, args...);
    return hipGetLastError();
}

// Allocation-free evaluate: the static per-device scratch that holds its
// partial sums (16 MiB: the D = 1e6, N = 2048 evaluate needs 12.6 MB), and
// the current device's address of it (looked up once per device).
constexpr size_t NOALLOC_SCRATCH_FLOATS = (size_t)4 << 20;
hipError_t noalloc_scratch(float** out);

// Largest population the rank kernel stages in LDS; larger ones take the
// sort-based ranks, up to POP_MAX_N.
constexpr int32_t RANK_MAX_N = 16384;
constexpr int32_t POP_MAX_N = 1 << 24;
// The count costs R N^2 compares, the sort about R N log N plus a fixed
// part: the sort is the faster above about this R N^2 (measured, R N^2 in
// units of 1e8: one run 1.05 counted 58 us per generation against 59 sorted,
// 1.27 66 against 64; 16 runs 0.67 35 against 63, 2.7 85 against 73; 64 runs
// 0.67 33 against 72, 2.7 93 against 98).
constexpr double RANK_SORT_FROM_WORK = 1.2e8;

}  // namespace esmi
