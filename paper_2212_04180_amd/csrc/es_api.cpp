// es_api.cpp -- host runtime behind the C-ABI of esmi.h.
//
// Owns the handle (config, device state, scratch), validates arguments,
// enforces the ask -> (evaluate) -> tell order of Sec. 2.1 / Listing 1 and
// sequences the kernel launches on the caller's stream.  No call blocks
// unless esmi.h says it is synchronous.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <vector>
#include <new>

#include "es_internal.hpp"
#include "esmi.h"

using namespace esmi;

namespace {

enum Phase { READY = 0, ASKED = 1 };

constexpr uint32_t kCheckpointMagic = 0x45534d32u;  // "ESM2"
// no padding bytes: a checkpoint's config is compared byte for byte
static_assert(sizeof(es_config) == 168, "es_config has padding");

thread_local char g_init_err[256] = {0};

es_status init_fail(es_status s, const char* msg, const char* who = "es_init")
{
    std::snprintf(g_init_err, sizeof(g_init_err), "%s: %s", who, msg);
    return s;
}

}  // namespace

struct es_handle {
    es_config cfg;
    Geometry g;
    EvalPlan plan;
    hipStream_t stream = nullptr;
    int device = 0;
    int64_t t = 0;
    int phase = READY;
    // state [R][Dp]
    float* m = nullptr;
    float* m1 = nullptr;
    float* v = nullptr;
    float* best_x = nullptr;
    float* grad = nullptr;
    // per-run scalars
    uint32_t* best_okey = nullptr;
    float* best_f = nullptr;
    int32_t* best_j = nullptr;
    // per-generation scratch
    float* table = nullptr;  // centered weight per rank [N]
    float* y = nullptr;      // [R][N]
    int32_t* rank = nullptr; // [R][N]
    float* wfold = nullptr;  // [R][P]
    float* fit = nullptr;    // [R][N] fitness scratch for es_run
    float* partial = nullptr;
    // per-run sigma and lr ([2][R]) of the current generation and the next;
    // the rank kernel writes the schedule step into the other buffer
    float* hp[2] = {nullptr, nullptr};
    int hp_cur = 0;
    float* pen = nullptr;        // [R][N] weight-decay mean square of the last tell
    double ybar_table = 0.0;     // mean of the shaping table
    float* bfold = nullptr;      // [R][P] second folded weight (PGPE, SNES)
    float* sig = nullptr;        // [R][Dp] per-dimension sigma (PGPE, SNES)
    float* vel = nullptr;        // [R][Dp] ClipUp velocity
    float* gbuf = nullptr;       // [R][Dp] ClipUp gradient
    double* gpart = nullptr;     // [R][groups] ClipUp / Sep-CMA-ES partial norms
    double* vpart = nullptr;
    // Sep-CMA-ES
    CmaConsts cma{};
    int32_t* elite = nullptr;    // [R][N]
    float* cw = nullptr;         // [mu]
    float* cmaC = nullptr;       // [R][Dp]
    double* zw = nullptr;        // [R][Dp]
    double* qd = nullptr;        // [R][Dp]
    TellPlan tell;               // pair slices of the gradient kernel
    double* tell_part = nullptr; // per-workgroup gradient sums when tell.nsplit > 1
    float* pdata = nullptr;  // [Dp] shift vector or teacher
    void* mlp_scratch = nullptr;  // MLP inputs and teacher outputs of the current generation
    int64_t teacher_t = -1;       // generation whose inputs and teacher outputs are in mlp_scratch
    int run_path = 0;  // 0 auto, 1 per-call kernels, 2 fused loop, 3 grid loop
    int32_t grid_g = 0;             // workgroups per run of the grid loop (0: the grid loop does not apply)
    int32_t grid_xs = 1;            // x stride between a run's grid-loop workgroups (the XCD count when packed)
    uint64_t* grid_words = nullptr;  // the grid loop's tagged words
    uint32_t* grid_err = nullptr;    // the grid loop's error flag
    uint32_t grid_seq = 0;           // sequence number of the last grid-loop launch
    // sort-based ranks (populations beyond RANK_MAX_N, or plan_rank_path 2)
    bool rank_sort = false;
    RankSortBuffers rs{};
    char err[512] = {0};
};

namespace {

es_status fail(es_handle* h, es_status s, const char* fmt, ...)
{
    if (h) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(h->err, sizeof(h->err), fmt, ap);
        va_end(ap);
    }
    return s;
}

es_status hip_fail(es_handle* h, hipError_t e, const char* what)
{
    return fail(h, e == hipErrorOutOfMemory ? ES_ERR_OOM : ES_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define ES_HIP(h, call, what)                                   \
    do {                                                        \
        hipError_t e__ = (call);                                \
        if (e__ != hipSuccess) return hip_fail((h), e__, what); \
    } while (0)

template <typename T>
hipError_t dalloc(T** p, size_t n)
{
    *p = nullptr;
    if (n == 0) n = 1;
    return hipMalloc(reinterpret_cast<void**>(p), n * sizeof(T));
}

const char* validate(const es_config& c)
{
    if (c.num_dims < 1) return "num_dims must be >= 1";
    if (c.num_dims > ((int64_t)1 << 34)) return "num_dims exceeds 2^34";
    if (c.popsize < 2 || (c.popsize & 1)) return "popsize must be even and >= 2";
    if (c.popsize > POP_MAX_N) return "popsize exceeds 2^24";
    if (c.num_runs < 1 || c.num_runs > 65535) return "num_runs must be in [1, 65535]";
    if (!(c.sigma > 0.0f) || !std::isfinite(c.sigma)) return "sigma must be finite and > 0";
    if (!std::isfinite(c.lr) || c.lr < 0.0f) return "lr must be finite and >= 0";
    if (!(c.beta1 >= 0.0f && c.beta1 < 1.0f)) return "beta1 must be in [0, 1)";
    if (!(c.beta2 >= 0.0f && c.beta2 < 1.0f)) return "beta2 must be in [0, 1)";
    if (!(c.eps >= 0.0f) || !std::isfinite(c.eps)) return "eps must be finite and >= 0";
    if (c.maximize != 0 && c.maximize != 1) return "maximize must be 0 or 1";
    if (c.shaping != ES_SHAPE_CENTERED_RANK && c.shaping != ES_SHAPE_RAW && c.shaping != ES_SHAPE_Z_SCORE)
        return "unknown shaping";
    if (c.init < ES_INIT_UNIFORM || c.init > ES_INIT_FANIN_NORMAL) return "unknown init";
    if (c.init == ES_INIT_UNIFORM && !(c.init_hi > c.init_lo)) return "init range must have hi > lo";
    if (c.problem < ES_PROB_NONE || c.problem > ES_PROB_MLP) return "unknown problem";
    if (c.init == ES_INIT_FANIN_NORMAL && c.num_dims != MLP_NUM_PARAMS)
        return "fan-in normal init is defined for the 64-256-256-16 MLP (num_dims 86544)";
    if (c.problem == ES_PROB_MLP && c.num_dims != MLP_NUM_PARAMS) return "MLP problem needs num_dims 86544";
    if (c.problem == ES_PROB_MLP && c.mlp_batch != 256) return "MLP problem needs mlp_batch 256";
    if (c.problem == ES_PROB_MLP && c.mlp_bf16 != 1) return "the MLP forward runs on bf16 matrix cores (mlp_bf16 = 1)";
    if (c.problem == ES_PROB_RASTRIGIN && !std::isfinite(c.rastrigin_a)) return "rastrigin_a must be finite";
    if ((c.flags & ~ES_FLAG_KEEP_GRAD) != 0) return "unknown flags";
    if (!(c.sigma_decay > 0.0f) || !std::isfinite(c.sigma_decay)) return "sigma_decay must be finite and > 0";
    if (!(c.lr_decay > 0.0f) || !std::isfinite(c.lr_decay)) return "lr_decay must be finite and > 0";
    if (!(c.sigma_final >= 0.0f) || !std::isfinite(c.sigma_final)) return "sigma_final must be finite and >= 0";
    if (!(c.lr_final >= 0.0f) || !std::isfinite(c.lr_final)) return "lr_final must be finite and >= 0";
    if (!(c.w_decay >= 0.0f) || !std::isfinite(c.w_decay)) return "w_decay must be finite and >= 0";
    if (c.strategy < ES_STRAT_OPENAI_ES || c.strategy > ES_STRAT_SEP_CMA) return "unknown strategy";
    if (c.strategy == ES_STRAT_SEP_CMA && !(c.elite_ratio > 0.0f && c.elite_ratio <= 1.0f))
        return "elite_ratio must be in (0, 1]";
    if (c.plan_grid_workgroups < 0 || c.plan_grid_workgroups > GRID_MAX_G)
        return "plan_grid_workgroups must be in [0, 16]";
    if (c.plan_rank_path < 0 || c.plan_rank_path > 2) return "plan_rank_path must be 0, 1 or 2";
    if (c.plan_grid_spin_limit < -1) return "plan_grid_spin_limit must be >= -1";
    if (c.plan_grid_pack != 0 && c.plan_grid_pack != -1) return "plan_grid_pack must be 0 or -1";
    if (c.plan_rank_path == 1 && c.popsize > RANK_MAX_N)
        return "plan_rank_path 1 (ranks counted in LDS) takes popsize <= 16384";
    // (the library's own choice of the sort never needs more: it picks the
    // sort below RANK_MAX_N members only, where R N < 65536 * 16384)
    if ((c.popsize > RANK_MAX_N || c.plan_rank_path == 2) && (int64_t)c.popsize * c.num_runs > INT32_MAX)
        return "sort-based ranks need num_runs * popsize < 2^31";
    if (c.plan_eval_blocks < 0) return "plan_eval_blocks must be >= 0";
    if (c.plan_tell_split < 0 || c.plan_tell_split > 65535) return "plan_tell_split must be in [0, 65535]";
    if (c.plan_run_path < 0 || c.plan_run_path > 3) return "plan_run_path must be 0, 1, 2 or 3";
    if (c.strategy == ES_STRAT_SEP_CMA && c.problem == ES_PROB_MLP)
        return "Sep-CMA-ES takes the benchmark problems or the caller's fitness (the MLP evaluate kernel samples "
               "antithetic pairs)";
    if (c.optimizer != ES_OPT_ADAM && c.optimizer != ES_OPT_CLIPUP) return "unknown optimizer";
    if ((c.strategy == ES_STRAT_PGPE || c.strategy == ES_STRAT_SNES) && (!(c.sigma_lr > 0.0f) || !std::isfinite(c.sigma_lr)))
        return "sigma_lr must be finite and > 0";
    if (c.strategy == ES_STRAT_PGPE && !(c.sigma_max_change > 0.0f && c.sigma_max_change < 1.0f))
        return "sigma_max_change must be in (0, 1)";
    if ((c.strategy == ES_STRAT_OPENAI_ES || c.strategy == ES_STRAT_PGPE) && c.optimizer == ES_OPT_CLIPUP) {
        if (!(c.clipup_max_speed > 0.0f) || !std::isfinite(c.clipup_max_speed))
            return "clipup_max_speed must be finite and > 0";
        if (!(c.clipup_momentum >= 0.0f && c.clipup_momentum < 1.0f)) return "clipup_momentum must be in [0, 1)";
    }
    if (c.strategy == ES_STRAT_SNES && (!(c.snes_temperature >= 0.0f) || !std::isfinite(c.snes_temperature)))
        return "snes_temperature must be finite and >= 0";
    return nullptr;
}

// Sep-CMA-ES parent count: max(1, floor(elite_ratio N)).
int32_t cma_mu(const es_config& c)
{
    const int32_t mu = (int32_t)std::floor((double)c.elite_ratio * (double)c.popsize);
    return mu < 1 ? 1 : mu;
}

// Sep-CMA-ES settings (standard CMA-ES values, separable rate factor (D+2)/3)
// and recombination weights ln(mu + 1/2) - ln(i + 1), normalised in fp64.
CmaConsts cma_consts(const es_config& c, std::vector<double>& w)
{
    CmaConsts k{};
    const double D = (double)c.num_dims;
    k.mu = cma_mu(c);
    w.assign((size_t)k.mu, 0.0);
    double sum = 0.0, s2 = 0.0;
    for (int32_t i = 0; i < k.mu; ++i) sum += (w[i] = std::log((double)k.mu + 0.5) - std::log((double)(i + 1)));
    for (int32_t i = 0; i < k.mu; ++i) {
        w[i] /= sum;
        s2 += w[i] * w[i];
    }
    k.mu_eff = 1.0 / s2;
    k.c_s = (k.mu_eff + 2.0) / (D + k.mu_eff + 5.0);
    const double q = std::sqrt((k.mu_eff - 1.0) / (D + 1.0)) - 1.0;
    k.d_s = 1.0 + 2.0 * (q > 0.0 ? q : 0.0) + k.c_s;
    k.c_c = (4.0 + k.mu_eff / D) / (D + 4.0 + 2.0 * k.mu_eff / D);
    const double c1 = 2.0 / ((D + 1.3) * (D + 1.3) + k.mu_eff);
    double cmu = 2.0 * (k.mu_eff - 2.0 + 1.0 / k.mu_eff) / ((D + 2.0) * (D + 2.0) + k.mu_eff);
    if (cmu > 1.0 - c1) cmu = 1.0 - c1;
    k.c1 = std::min(1.0, c1 * (D + 2.0) / 3.0);
    k.cmu = std::min(1.0 - k.c1, cmu * (D + 2.0) / 3.0);
    k.chi = std::sqrt(D) * (1.0 - 1.0 / (4.0 * D) + 1.0 / (21.0 * D * D));
    k.a_s = std::sqrt(k.c_s * (2.0 - k.c_s) * k.mu_eff);
    k.a_c = std::sqrt(k.c_c * (2.0 - k.c_c) * k.mu_eff);
    k.wsum = 0.0;
    for (int32_t i = 0; i < k.mu; ++i) k.wsum += (double)(float)w[i];
    return k;
}

// Shaping weight of rank k.  Centered ranks: the fp32 quotient
// (2k - (N-1)) / (2(N-1)).  SNES: the softmax utility of rank' = N-1-k,
// exp(beta (rank'/N - 1/2)) / sum, in fp64 rounded once.  Sep-CMA-ES: the
// recombination weight of rank k < mu, else 0.  Returns the table's fp64 mean.
double weight_table(const es_config& c, int32_t N, float* out)
{
    if (c.strategy == ES_STRAT_SEP_CMA) {
        std::vector<double> w;
        const CmaConsts k = cma_consts(c, w);
        for (int32_t r = 0; r < N; ++r) out[r] = r < k.mu ? (float)w[r] : 0.0f;
    } else if (c.strategy == ES_STRAT_SNES) {
        double S = 0.0;
        for (int32_t k = 0; k < N; ++k) S += std::exp((double)c.snes_temperature * ((double)k / (double)N - 0.5));
        for (int32_t k = 0; k < N; ++k)
            out[k] = (float)(std::exp((double)c.snes_temperature * ((double)(N - 1 - k) / (double)N - 0.5)) / S);
    } else {
        const float den = (float)(2 * (N - 1));
        for (int32_t k = 0; k < N; ++k) out[k] = (float)(2 * k - (N - 1)) / den;
    }
    double sum = 0.0;
    for (int32_t k = 0; k < N; ++k) sum += (double)out[k];
    return sum / (double)N;
}

AdamConsts adam_consts(const es_config& c, int64_t t)
{
    AdamConsts a;
    const double tp = (double)(t + 1);
    a.beta1 = c.beta1;
    a.beta2 = c.beta2;
    a.omb1 = (float)(1.0 - (double)c.beta1);
    a.omb2 = (float)(1.0 - (double)c.beta2);
    a.bc1 = (float)(1.0 - std::pow((double)c.beta1, tp));
    a.bc2 = (float)(1.0 - std::pow((double)c.beta2, tp));
    a.eps = c.eps;
    return a;
}

// es_run's choice: the fused loop pays off when each run is small (per-call
// launches then dominate) or when the runs fill the chip one workgroup each.
bool fused_by_default(const Geometry& g, const EvalPlan& e, const es_config& c)
{
    return fused_supported(g, e, c) && ((int64_t)g.P * g.nb <= 8192 || g.R >= 128);
}

// Otherwise the grid loop, where the launches of the per-call kernels (about
// 2.5 us each, four per generation) would cost more than the work of a few
// runs on a few dozen CUs.
bool grid_by_default(const es_handle* h)
{
    const Geometry& g = h->g;
    return h->grid_g > 0 && !fused_by_default(g, h->plan, h->cfg) &&
           (int64_t)g.R * g.P * g.nb <= GRID_DEFAULT_WORK && (int64_t)g.R * h->grid_g <= 256;
}

// The path es_run takes: plan_run_path forces one (1 per-call kernels, 2
// fused loop, 3 grid loop, each where it supports the config; a forced fused
// loop on a geometry es_run would not fuse sums in its own order), 0 leaves
// it to the rules above.
int run_path_of(const es_handle* h)
{
    switch (h->run_path) {
    case 1: return 1;
    case 2: return fused_supported(h->g, h->plan, h->cfg) ? 2 : 1;
    case 3: return h->grid_g > 0 ? 3 : 1;
    default: return fused_by_default(h->g, h->plan, h->cfg) ? 2 : grid_by_default(h) ? 3 : 1;
    }
}

void free_all(es_handle* h)
{
    void* ptrs[] = {h->m, h->m1, h->v, h->best_x, h->grad, h->best_okey, h->best_f, h->best_j, h->table,
                    h->y, h->rank, h->wfold, h->fit, h->partial, h->pdata, h->mlp_scratch,
                    h->tell_part, h->hp[0], h->hp[1], h->pen, h->bfold, h->sig, h->vel, h->gbuf,
                    h->gpart, h->vpart, h->elite, h->cw, h->cmaC, h->zw, h->qd,
                    h->rs.kin, h->rs.kout, h->rs.keys, h->rs.stats, h->rs.temp, h->grid_words, h->grid_err};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
}

es_status enqueue_tell(es_handle* h, const float* fitness, float* gen_best)
{
    const Geometry& g = h->g;
    const float* hp = h->hp[h->hp_cur];
    if (h->cfg.w_decay != 0.0f) {
        // weight decay: the mean square of every member, one more pass of the
        // sampler through the sphere evaluation, divided by D in its reduction
        es_config sq = h->cfg;
        sq.problem = ES_PROB_SPHERE;
        ES_HIP(h, launch_eval_bbob(g, sq, h->plan, (uint32_t)h->t, h->m, nullptr, h->partial, h->pen, hp, h->sig,
                                   (double)g.D, h->stream),
               "weight-decay penalty pass");
    }
    ES_HIP(h, launch_rank(g, h->cfg, fitness, h->pen, h->table, h->ybar_table, h->y, h->rank, h->wfold, h->bfold,
                          h->elite, h->cma.mu, h->best_okey, h->best_f, h->best_j, gen_best, hp, h->hp[1 - h->hp_cur],
                          h->rank_sort ? &h->rs : nullptr, h->stream),
           "rank kernel");
    const AdamConsts a = adam_consts(h->cfg, h->t);
    TellBuffers tb;
    tb.wfold = h->wfold; tb.bfold = h->bfold; tb.best_j = h->best_j;
    tb.m = h->m; tb.m1 = h->m1; tb.v = h->v; tb.grad = h->grad; tb.best_x = h->best_x;
    tb.sig = h->sig; tb.vel = h->vel; tb.gbuf = h->gbuf; tb.gpart = h->gpart; tb.vpart = h->vpart;
    tb.part = h->tell_part; tb.hp = hp; tb.hp_next = h->hp[1 - h->hp_cur];
    tb.elite = h->elite; tb.cw = h->cw; tb.zw = h->zw; tb.qd = h->qd; tb.cmaC = h->cmaC; tb.cma = h->cma;
    // MLP: where the gradient kernel can carry them (OpenAI-ES), the next
    // generation's inputs and teacher outputs ride in the gradient launch (the
    // evaluate kernel of this generation has read them); otherwise the next
    // evaluate makes them
    const bool teach = h->mlp_scratch && tell_carries_teacher(h->cfg, h->tell) && h->t + 1 <= 0xFFFFFFFFll;
    if (teach) tb.teacher = mlp_teacher_job(h->cfg, h->pdata, h->mlp_scratch, (uint32_t)(h->t + 1));
    ES_HIP(h, launch_tell(g, h->cfg, h->tell, (uint32_t)h->t, a, tb, h->stream), "tell kernel");
    h->teacher_t = teach ? h->t + 1 : -1;
    h->hp_cur = 1 - h->hp_cur;  // the schedule step is next generation's sigma and lr
    return ES_OK;
}

es_status enqueue_eval(es_handle* h, float* fit, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr)
{
    if (h->cfg.problem == ES_PROB_NONE) return fail(h, ES_ERR_UNSUPPORTED, "no built-in problem configured");
    if (h->cfg.problem == ES_PROB_MLP) {
        ES_HIP(h, launch_eval_mlp(h->g, h->cfg, (uint32_t)h->t, h->m, h->pdata, h->mlp_scratch, fit,
                                  h->hp[h->hp_cur], h->sig, h->teacher_t != h->t, h->stream, ev_start, ev_stop),
               "MLP evaluate kernels");
        h->teacher_t = h->t;
        return ES_OK;
    }
    ES_HIP(h, launch_eval_bbob(h->g, h->cfg, h->plan, (uint32_t)h->t, h->m, h->pdata, h->partial, fit,
                               h->hp[h->hp_cur], h->sig, 1.0, h->stream, ev_start, ev_stop),
           "evaluate kernel");
    return ES_OK;
}

// Device rows [R][D] <-> state rows [R][Dp]: one copy when the rows are
// contiguous on both sides (Dp = D, or one run), one 2D copy for pitches the
// runtime takes (under 2 GiB), else a copy per row.
constexpr size_t kMaxCopyPitch = ((size_t)1 << 31) - 1;

hipError_t copy_rows(const Geometry& g, float* dst, size_t dpitch, const float* src, size_t spitch, hipStream_t s)
{
    const size_t width = (size_t)g.D * 4;
    if (g.R == 1 || g.Dp == g.D)
        return hipMemcpyAsync(dst, src, width * (size_t)g.R, hipMemcpyDeviceToDevice, s);
    if (dpitch <= kMaxCopyPitch && spitch <= kMaxCopyPitch)
        return hipMemcpy2DAsync(dst, dpitch, src, spitch, width, (size_t)g.R, hipMemcpyDeviceToDevice, s);
    for (int32_t r = 0; r < g.R; ++r) {
        const hipError_t e = hipMemcpyAsync(reinterpret_cast<char*>(dst) + (size_t)r * dpitch,
                                            reinterpret_cast<const char*>(src) + (size_t)r * spitch, width,
                                            hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

es_status copy_rows_out(es_handle* h, float* dst, const float* src)
{
    const Geometry& g = h->g;
    ES_HIP(h, copy_rows(g, dst, (size_t)g.D * 4, src, (size_t)g.Dp * 4, h->stream), "copy out");
    return ES_OK;
}

es_status copy_rows_in(es_handle* h, float* dst, const float* src)
{
    const Geometry& g = h->g;
    if (g.Dp != g.D)
        ES_HIP(h, hipMemsetAsync(dst, 0, (size_t)g.Dp * g.R * 4, h->stream), "clear padding");
    ES_HIP(h, copy_rows(g, dst, (size_t)g.Dp * 4, src, (size_t)g.D * 4, h->stream), "copy in");
    return ES_OK;
}

struct CkptHeader {
    uint32_t magic;
    uint32_t version;
    es_config cfg;
    int64_t t;
    int64_t D, R;
};

}  // namespace

extern "C" {

const char* es_status_string(es_status s)
{
    switch (s) {
    case ES_OK: return "ok";
    case ES_ERR_ARG: return "invalid argument";
    case ES_ERR_SEQUENCE: return "call out of ask/eval/tell order";
    case ES_ERR_HIP: return "HIP runtime error";
    case ES_ERR_OOM: return "device out of memory";
    case ES_ERR_UNSUPPORTED: return "unsupported request";
    }
    return "unknown status";
}

const char* es_last_error(const es_handle* h) { return h ? h->err : g_init_err; }

int64_t es_generation(const es_handle* h) { return h ? h->t : -1; }

int32_t es_run_path(const es_handle* h, int32_t* keeps_normals)
{
    const int32_t path = h ? run_path_of(h) : 0;
    if (keeps_normals)
        *keeps_normals = path == 3 || (path == 2 && fused_stash(h->g, h->plan)) ? 1 : 0;
    return path;
}

es_status es_init(const es_config* cfg, void* hip_stream, es_handle** out)
{
    if (!cfg || !out) return init_fail(ES_ERR_ARG, "null argument");
    *out = nullptr;
    if (const char* why = validate(*cfg)) return init_fail(ES_ERR_ARG, why);
    es_handle* h = new (std::nothrow) es_handle();
    if (!h) return init_fail(ES_ERR_OOM, "host allocation failed");
    h->cfg = *cfg;
    h->stream = reinterpret_cast<hipStream_t>(hip_stream);
    Geometry& g = h->g;
    g.D = cfg->num_dims;
    g.nb = (g.D + 3) / 4;
    g.Dp = 4 * g.nb;
    g.N = cfg->popsize;
    g.P = cfg->popsize / 2;
    g.R = cfg->num_runs;
    h->plan = eval_plan(g, cfg->plan_eval_blocks);
    // where es_run takes the fused loop (the rule of es_run), the per-call
    // gradient kernel sums in the fused loop's order, so both give the same bits
    h->tell = tell_plan(g, fused_by_default(g, h->plan, *cfg), cfg->plan_tell_split);
    h->run_path = cfg->plan_run_path;
    {
        const int32_t G = grid_workgroups(g, h->plan, cfg->plan_grid_workgroups);
        int64_t cap = 0;
        if (grid_supported(g, h->plan, h->tell, *cfg, G) && grid_max_resident(&cap) == hipSuccess &&
            (int64_t)G * g.R <= cap) {
            h->grid_g = G;
            // one XCD per run where the device holds the XCD count times the
            // workgroups at once (workgroups are dealt to the XCDs in turn)
            int dev = 0, xcc = 1;
            if (cfg->plan_grid_pack == 0 && hipGetDevice(&dev) == hipSuccess) {
                if (hipDeviceGetAttribute(&xcc, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess) {
                    // a runtime without the attribute: no packing, and no
                    // error left for the next launch's hipGetLastError
                    xcc = 1;
                    (void)hipGetLastError();
                }
                if (xcc > 1 && (int64_t)xcc * G * g.R <= cap) h->grid_xs = xcc;
            }
        }
    }
    hipError_t e = hipGetDevice(&h->device);
    const size_t rows = (size_t)g.Dp * g.R;
    if (e == hipSuccess) e = dalloc(&h->m, rows);
    if (e == hipSuccess) e = dalloc(&h->m1, rows);
    if (e == hipSuccess) e = dalloc(&h->v, rows);
    if (e == hipSuccess) e = dalloc(&h->best_x, rows);
    if (e == hipSuccess && (cfg->flags & ES_FLAG_KEEP_GRAD)) e = dalloc(&h->grad, rows);
    if (e == hipSuccess) e = dalloc(&h->best_okey, (size_t)g.R);
    if (e == hipSuccess) e = dalloc(&h->best_f, (size_t)g.R);
    if (e == hipSuccess) e = dalloc(&h->best_j, (size_t)g.R);
    if (e == hipSuccess) e = dalloc(&h->table, (size_t)g.N);
    if (e == hipSuccess) e = dalloc(&h->y, (size_t)g.N * g.R);
    if (e == hipSuccess) e = dalloc(&h->rank, (size_t)g.N * g.R);
    if (e == hipSuccess) e = dalloc(&h->wfold, (size_t)g.P * g.R);
    if (e == hipSuccess) e = dalloc(&h->fit, (size_t)g.N * g.R);
    if (e == hipSuccess && ((cfg->problem != ES_PROB_NONE && cfg->problem != ES_PROB_MLP) || cfg->w_decay != 0.0f))
        e = dalloc(&h->partial, (size_t)eval_partial_elems(g, h->plan));
    if (e == hipSuccess && cfg->w_decay != 0.0f) e = dalloc(&h->pen, (size_t)g.N * g.R);
    if (e == hipSuccess) e = dalloc(&h->hp[0], 2 * (size_t)g.R);
    if (e == hipSuccess) e = dalloc(&h->hp[1], 2 * (size_t)g.R);
    if (e == hipSuccess && (cfg->problem == ES_PROB_SHIFTED_SPHERE || cfg->problem == ES_PROB_MLP))
        e = dalloc(&h->pdata, (size_t)g.Dp);
    if (e == hipSuccess && cfg->problem == ES_PROB_MLP)
        e = dalloc(reinterpret_cast<char**>(&h->mlp_scratch), mlp_scratch_bytes());
    if (e == hipSuccess && h->tell.nsplit > 1)
        e = dalloc(&h->tell_part, tell_part_elems(g, h->tell, cfg->strategy));
    if (e == hipSuccess && h->grid_g > 0) {
        // zero tags: no launch waits for tag 0
        const size_t nw = grid_word_count(g, h->plan);
        e = dalloc(&h->grid_words, nw);
        if (e == hipSuccess) e = hipMemsetAsync(h->grid_words, 0, sizeof(uint64_t) * nw, h->stream);
        if (e == hipSuccess) e = dalloc(&h->grid_err, 1);
        if (e == hipSuccess) e = hipMemsetAsync(h->grid_err, 0, sizeof(uint32_t), h->stream);
    }
    const bool pgpe_snes = cfg->strategy == ES_STRAT_PGPE || cfg->strategy == ES_STRAT_SNES;
    const bool cma = cfg->strategy == ES_STRAT_SEP_CMA;
    if (e == hipSuccess && pgpe_snes) e = dalloc(&h->bfold, (size_t)g.P * g.R);
    if (e == hipSuccess && (pgpe_snes || cma)) e = dalloc(&h->sig, rows);
    std::vector<double> cma_w;
    if (cma) h->cma = cma_consts(*cfg, cma_w);
    if (e == hipSuccess && cma) e = dalloc(&h->elite, (size_t)g.N * g.R);
    if (e == hipSuccess && cma) e = dalloc(&h->cw, (size_t)h->cma.mu);
    if (e == hipSuccess && cma) e = dalloc(&h->cmaC, rows);
    if (e == hipSuccess && cma) e = dalloc(&h->zw, rows);
    if (e == hipSuccess && cma) e = dalloc(&h->qd, rows);
    if (e == hipSuccess && cma) e = dalloc(&h->gpart, tell_groups(g) * g.R);
    const bool clipup = (cfg->strategy == ES_STRAT_OPENAI_ES || cfg->strategy == ES_STRAT_PGPE) &&
                        cfg->optimizer == ES_OPT_CLIPUP;
    if (e == hipSuccess && clipup) e = dalloc(&h->vel, rows);
    if (e == hipSuccess && clipup) e = dalloc(&h->gbuf, rows);
    if (e == hipSuccess && clipup) e = dalloc(&h->gpart, tell_groups(g) * g.R);
    if (e == hipSuccess && clipup) e = dalloc(&h->vpart, tell_groups(g) * g.R);
    h->rank_sort = g.N > RANK_MAX_N || cfg->plan_rank_path == 2 ||
                   (cfg->plan_rank_path == 0 && (double)g.R * g.N * g.N > RANK_SORT_FROM_WORK);
    if (e == hipSuccess && h->rank_sort) {
        const size_t n = (size_t)g.N * g.R;
        e = dalloc(&h->rs.kin, n);
        if (e == hipSuccess) e = dalloc(&h->rs.kout, n);
        if (e == hipSuccess) e = dalloc(&h->rs.keys, n);
        if (e == hipSuccess) e = dalloc(&h->rs.stats, 4 * (size_t)g.R);
        rank_sort_bits(g, &h->rs.bn, &h->rs.br);
        h->rs.temp_bytes = rank_sort_temp_bytes(g);
        if (e == hipSuccess && h->rs.temp_bytes == 0) e = hipErrorInvalidValue;
        if (e == hipSuccess) e = dalloc(reinterpret_cast<char**>(&h->rs.temp), h->rs.temp_bytes);
    }
    if (e != hipSuccess) {
        free_all(h);
        delete h;
        return init_fail(e == hipErrorOutOfMemory ? ES_ERR_OOM : ES_ERR_HIP, hipGetErrorString(e));
    }
    // weight table (host-computed, exact fp32 quotients) and best-so-far init
    float* tab = static_cast<float*>(std::malloc(sizeof(float) * (size_t)g.N));
    uint32_t* ok = static_cast<uint32_t*>(std::malloc(sizeof(uint32_t) * (size_t)g.R));
    float* bf = static_cast<float*>(std::malloc(sizeof(float) * (size_t)g.R));
    float* hp = static_cast<float*>(std::malloc(sizeof(float) * 2 * (size_t)g.R));
    if (!tab || !ok || !bf || !hp) {
        std::free(tab); std::free(ok); std::free(bf); std::free(hp);
        free_all(h);
        delete h;
        return init_fail(ES_ERR_OOM, "host allocation failed");
    }
    h->ybar_table = weight_table(*cfg, g.N, tab);
    for (int32_t r = 0; r < g.R; ++r) {
        ok[r] = 0xFF800000u;  // order key of +inf: nothing is an improvement over it but a finite key
        bf[r] = NAN;
        hp[r] = cfg->sigma;
        hp[g.R + r] = cfg->lr;
    }
    e = hipMemcpyAsync(h->table, tab, sizeof(float) * (size_t)g.N, hipMemcpyHostToDevice, h->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(h->best_okey, ok, sizeof(uint32_t) * (size_t)g.R, hipMemcpyHostToDevice, h->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(h->best_f, bf, sizeof(float) * (size_t)g.R, hipMemcpyHostToDevice, h->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(h->hp[0], hp, sizeof(float) * 2 * (size_t)g.R, hipMemcpyHostToDevice, h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);  // host staging buffers are freed next
    std::free(tab); std::free(ok); std::free(bf); std::free(hp);
    if (e == hipSuccess) e = launch_init(g, *cfg, h->m, h->m1, h->v, h->best_x, h->stream);
    if (e == hipSuccess && h->sig) e = launch_fill_rows(g, h->sig, cfg->sigma, h->stream);
    if (e == hipSuccess && h->cmaC) e = launch_fill_rows(g, h->cmaC, 1.0f, h->stream);
    if (e == hipSuccess && h->cw) {
        std::vector<float> w32(cma_w.size());
        for (size_t i = 0; i < cma_w.size(); ++i) w32[i] = (float)cma_w[i];
        e = hipMemcpyAsync(h->cw, w32.data(), sizeof(float) * w32.size(), hipMemcpyHostToDevice, h->stream);
        if (e == hipSuccess) e = hipStreamSynchronize(h->stream);  // w32 is freed next
    }
    if (e == hipSuccess && h->vel) e = launch_fill_rows(g, h->vel, 0.0f, h->stream);
    if (e == hipSuccess && h->pdata) e = launch_problem_data(g, *cfg, h->pdata, h->stream);
    if (e == hipSuccess && h->mlp_scratch) e = launch_mlp_setup(h->pdata, h->mlp_scratch, h->stream);
    if (e != hipSuccess) {
        free_all(h);
        delete h;
        return init_fail(ES_ERR_HIP, hipGetErrorString(e));
    }
    g_init_err[0] = 0;
    *out = h;
    return ES_OK;
}

es_status es_ask(es_handle* h, float* x_out)
{
    if (!h) return ES_ERR_ARG;
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_ask: previous generation was not told");
    if (x_out)
        ES_HIP(h, launch_ask(h->g, h->cfg, (uint32_t)h->t, h->m, x_out, h->hp[h->hp_cur], h->sig, h->stream),
               "ask kernel");
    h->phase = ASKED;
    h->err[0] = 0;
    return ES_OK;
}

es_status es_eval(es_handle* h, float* fitness_out)
{
    if (!h || !fitness_out) return h ? fail(h, ES_ERR_ARG, "es_eval: null fitness buffer") : ES_ERR_ARG;
    if (h->phase != ASKED) return fail(h, ES_ERR_SEQUENCE, "es_eval: no open ask");
    return enqueue_eval(h, fitness_out);
}

es_status es_eval_timed(es_handle* h, float* fitness_out, void* start_event, void* stop_event)
{
    if (!h || !fitness_out) return h ? fail(h, ES_ERR_ARG, "es_eval_timed: null fitness buffer") : ES_ERR_ARG;
    if (h->phase != ASKED) return fail(h, ES_ERR_SEQUENCE, "es_eval_timed: no open ask");
    return enqueue_eval(h, fitness_out, reinterpret_cast<hipEvent_t>(start_event),
                        reinterpret_cast<hipEvent_t>(stop_event));
}

es_status es_eval_noalloc(const es_config* cfg, const float* mean, const float* problem_data, const float* sigma,
                          int64_t t, float* fitness, void* hip_stream)
{
    constexpr const char* kNoalloc = "es_eval_noalloc";
    if (!cfg || !mean || !sigma || !fitness) return init_fail(ES_ERR_ARG, "null argument", kNoalloc);
    if (const char* why = validate(*cfg)) return init_fail(ES_ERR_ARG, why, kNoalloc);
    if (cfg->strategy != ES_STRAT_OPENAI_ES)
        return init_fail(ES_ERR_UNSUPPORTED, "OpenAI-ES sampling (the run's scalar sigma) only", kNoalloc);
    if (cfg->problem != ES_PROB_SPHERE && cfg->problem != ES_PROB_SHIFTED_SPHERE && cfg->problem != ES_PROB_ROSENBROCK &&
        cfg->problem != ES_PROB_RASTRIGIN)
        return init_fail(ES_ERR_UNSUPPORTED, "the benchmark problems only (not the MLP, not none)", kNoalloc);
    if ((cfg->problem == ES_PROB_SHIFTED_SPHERE) != (problem_data != nullptr))
        return init_fail(ES_ERR_ARG, "problem_data is the shift vector of the shifted sphere "
                                     "(and NULL for the other problems)", kNoalloc);
    if (cfg->num_dims % 4 != 0 && cfg->num_runs != 1)
        return init_fail(ES_ERR_UNSUPPORTED, "several runs need num_dims % 4 == 0", kNoalloc);
    if (t < 0 || t > 0xFFFFFFFFll) return init_fail(ES_ERR_ARG, "t out of range", kNoalloc);
    Geometry g;
    g.D = cfg->num_dims;
    g.nb = (g.D + 3) / 4;
    g.Dp = 4 * g.nb;
    g.N = cfg->popsize;
    g.P = cfg->popsize / 2;
    g.R = cfg->num_runs;
    const EvalPlan plan = eval_plan(g, cfg->plan_eval_blocks);
    const int64_t need = eval_partial_elems(g, plan);
    if (need > (int64_t)NOALLOC_SCRATCH_FLOATS) {
        std::snprintf(g_init_err, sizeof(g_init_err),
                      "es_eval_noalloc: this evaluate needs %lld bytes of partial sums; the static scratch holds %zu",
                      (long long)need * 4, NOALLOC_SCRATCH_FLOATS * 4);
        return ES_ERR_ARG;
    }
    float* scratch = nullptr;
    hipError_t e = noalloc_scratch(&scratch);
    if (e != hipSuccess) return init_fail(ES_ERR_HIP, hipGetErrorString(e), kNoalloc);
    e = launch_eval_bbob(g, *cfg, plan, (uint32_t)t, mean, problem_data, scratch, fitness, sigma, nullptr, 1.0,
                         reinterpret_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return init_fail(ES_ERR_HIP, hipGetErrorString(e), kNoalloc);
    g_init_err[0] = 0;
    return ES_OK;
}

es_status es_tell(es_handle* h, const float* fitness)
{
    if (!h || !fitness) return h ? fail(h, ES_ERR_ARG, "es_tell: null fitness buffer") : ES_ERR_ARG;
    if (h->phase != ASKED) return fail(h, ES_ERR_SEQUENCE, "es_tell: no open ask");
    es_status s = enqueue_tell(h, fitness, nullptr);
    if (s != ES_OK) return s;
    h->t += 1;
    h->phase = READY;
    return ES_OK;
}

es_status es_run(es_handle* h, int32_t T, float* log)
{
    if (!h) return ES_ERR_ARG;
    if (T < 0) return fail(h, ES_ERR_ARG, "es_run: T must be >= 0");
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_run: an ask is open");
    if (h->cfg.problem == ES_PROB_NONE) return fail(h, ES_ERR_UNSUPPORTED, "es_run needs a built-in problem");
    if (T == 0) return ES_OK;
    if (h->t + T > 0xFFFFFFFFll) return fail(h, ES_ERR_ARG, "es_run: generation counter would exceed 2^32");
    const int path = run_path_of(h);
    if (path != 1) {
        // launches of up to FUSED_MAX_T generations, each with its generations'
        // Adam bias corrections in the kernel arguments
        float bcorr[FUSED_MAX_T][2];
        for (int32_t done = 0; done < T;) {
            const int32_t Tc = std::min(T - done, FUSED_MAX_T);
            for (int32_t i = 0; i < Tc; ++i) {
                const AdamConsts a = adam_consts(h->cfg, h->t + i);
                bcorr[i][0] = a.bc1;
                bcorr[i][1] = a.bc2;
            }
            float* lg = log ? log + (int64_t)done * h->g.R : nullptr;
            if (path == 2)
                ES_HIP(h, launch_run_fused(h->g, h->cfg, h->plan, (uint32_t)h->t, Tc, adam_consts(h->cfg, h->t), bcorr,
                                           h->m, h->m1, h->v, h->grad, h->best_x, h->best_okey, h->best_f, h->pdata,
                                           h->table,
                                           lg, h->hp[h->hp_cur], h->stream),
                       "fused generation loop");
            else {
                // a sequence number the previous launch did not use, so that
                // none of its words carries a tag this launch waits for
                h->grid_seq = h->grid_seq % 0xFFFFFFu + 1;
                ES_HIP(h, launch_run_grid(h->g, h->cfg, h->plan, h->tell, h->grid_g, h->grid_xs, (uint32_t)h->t, Tc,
                                          adam_consts(h->cfg, h->t), bcorr, h->m, h->m1, h->v, h->grad, h->best_x,
                                          h->best_okey, h->best_f, h->pdata, h->table, lg, h->grid_words, h->grid_seq,
                                          h->grid_err, h->hp[h->hp_cur], h->stream),
                       "grid generation loop");
            }
            h->t += Tc;
            done += Tc;
        }
        return ES_OK;
    }
    for (int32_t i = 0; i < T; ++i) {
        es_status s = enqueue_eval(h, h->fit);
        if (s != ES_OK) return s;
        s = enqueue_tell(h, h->fit, log ? log + (int64_t)i * h->g.R : nullptr);
        if (s != ES_OK) return s;
        h->t += 1;
    }
    return ES_OK;
}

es_status es_get_state(es_handle* h, float* m, float* m1, float* v, int64_t* t)
{
    if (!h) return ES_ERR_ARG;
    es_status s = ES_OK;
    if (m && (s = copy_rows_out(h, m, h->m)) != ES_OK) return s;
    if (m1 && (s = copy_rows_out(h, m1, h->m1)) != ES_OK) return s;
    if (v && (s = copy_rows_out(h, v, h->v)) != ES_OK) return s;
    if (t) *t = h->t;
    return ES_OK;
}

// A new state also makes the grid loop's failure flag stale: clear it (a
// copy rather than a memset, so that a captured stream records no memset).
static es_status clear_grid_flag(es_handle* h)
{
    static const uint32_t zero = 0;
    if (h->grid_err)
        ES_HIP(h, hipMemcpyAsync(h->grid_err, &zero, sizeof(zero), hipMemcpyHostToDevice, h->stream),
               "clear the grid loop flag");
    return ES_OK;
}

es_status es_set_state(es_handle* h, const float* m, const float* m1, const float* v, int64_t t)
{
    if (!h) return ES_ERR_ARG;
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_set_state: an ask is open");
    if (t < 0 || t > 0xFFFFFFFFll) return fail(h, ES_ERR_ARG, "es_set_state: t out of range");
    es_status s = ES_OK;
    if (m && (s = copy_rows_in(h, h->m, m)) != ES_OK) return s;
    if (m1 && (s = copy_rows_in(h, h->m1, m1)) != ES_OK) return s;
    if (v && (s = copy_rows_in(h, h->v, v)) != ES_OK) return s;
    if ((s = clear_grid_flag(h)) != ES_OK) return s;
    if (t != h->t) h->teacher_t = -1;
    h->t = t;
    return ES_OK;
}

es_status es_get_best(es_handle* h, float* member, float* fitness)
{
    if (!h) return ES_ERR_ARG;
    if (member) {
        es_status s = copy_rows_out(h, member, h->best_x);
        if (s != ES_OK) return s;
    }
    if (fitness)
        ES_HIP(h, hipMemcpyAsync(fitness, h->best_f, sizeof(float) * (size_t)h->g.R, hipMemcpyDeviceToDevice,
                                 h->stream),
               "copy best fitness");
    return ES_OK;
}

es_status es_get_shaped(es_handle* h, float* y, int32_t* rank)
{
    if (!h) return ES_ERR_ARG;
    const size_t n = (size_t)h->g.N * h->g.R;
    if (y) ES_HIP(h, hipMemcpyAsync(y, h->y, n * 4, hipMemcpyDeviceToDevice, h->stream), "copy y");
    if (rank) ES_HIP(h, hipMemcpyAsync(rank, h->rank, n * 4, hipMemcpyDeviceToDevice, h->stream), "copy ranks");
    return ES_OK;
}

es_status es_get_grad(es_handle* h, float* g)
{
    if (!h || !g) return h ? fail(h, ES_ERR_ARG, "es_get_grad: null buffer") : ES_ERR_ARG;
    if (!h->grad) return fail(h, ES_ERR_UNSUPPORTED, "es_get_grad needs ES_FLAG_KEEP_GRAD");
    return copy_rows_out(h, g, h->grad);
}

es_status es_set_hparams(es_handle* h, const float* sigma, const float* lr)
{
    if (!h) return ES_ERR_ARG;
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_set_hparams: an ask is open");
    if (sigma && (h->cfg.strategy == ES_STRAT_PGPE || h->cfg.strategy == ES_STRAT_SNES))
        return fail(h, ES_ERR_UNSUPPORTED, "es_set_hparams: PGPE and SNES sample with a per-dimension sigma "
                                           "(es_set_strategy_state)");
    const int32_t R = h->g.R;
    for (int32_t r = 0; r < R; ++r) {
        if (sigma && (!(sigma[r] > 0.0f) || !std::isfinite(sigma[r])))
            return fail(h, ES_ERR_ARG, "es_set_hparams: sigma[%d] must be finite and > 0", r);
        if (lr && (!(lr[r] >= 0.0f) || !std::isfinite(lr[r])))
            return fail(h, ES_ERR_ARG, "es_set_hparams: lr[%d] must be finite and >= 0", r);
    }
    float* d = h->hp[h->hp_cur];
    // synchronous copies: the caller's host arrays may be reused on return
    if (sigma) ES_HIP(h, hipMemcpyAsync(d, sigma, sizeof(float) * R, hipMemcpyHostToDevice, h->stream), "set sigma");
    if (lr) ES_HIP(h, hipMemcpyAsync(d + R, lr, sizeof(float) * R, hipMemcpyHostToDevice, h->stream), "set lr");
    if (sigma && h->cmaC) ES_HIP(h, launch_cma_scale(h->g, h->sig, h->cmaC, d, h->stream), "Sep-CMA-ES scale");
    ES_HIP(h, hipStreamSynchronize(h->stream), "set hparams");
    return ES_OK;
}

es_status es_get_hparams(es_handle* h, float* sigma, float* lr)
{
    if (!h) return ES_ERR_ARG;
    const int32_t R = h->g.R;
    const float* d = h->hp[h->hp_cur];
    if (sigma) ES_HIP(h, hipMemcpyAsync(sigma, d, sizeof(float) * R, hipMemcpyDeviceToHost, h->stream), "get sigma");
    if (lr) ES_HIP(h, hipMemcpyAsync(lr, d + R, sizeof(float) * R, hipMemcpyDeviceToHost, h->stream), "get lr");
    ES_HIP(h, hipStreamSynchronize(h->stream), "get hparams");
    return ES_OK;
}

es_status es_get_strategy_state(es_handle* h, float* sigma_vec, float* velocity)
{
    if (!h) return ES_ERR_ARG;
    if ((sigma_vec && !h->sig) || (velocity && !h->vel))
        return fail(h, ES_ERR_UNSUPPORTED, "es_get_strategy_state: the strategy keeps no such state");
    es_status s = ES_OK;
    // Sep-CMA-ES: the diagonal covariance (its sampling scale is derived)
    if (sigma_vec && (s = copy_rows_out(h, sigma_vec, h->cmaC ? h->cmaC : h->sig)) != ES_OK) return s;
    if (velocity && (s = copy_rows_out(h, velocity, h->vel)) != ES_OK) return s;
    return ES_OK;
}

es_status es_set_strategy_state(es_handle* h, const float* sigma_vec, const float* velocity)
{
    if (!h) return ES_ERR_ARG;
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_set_strategy_state: an ask is open");
    if ((sigma_vec && !h->sig) || (velocity && !h->vel))
        return fail(h, ES_ERR_UNSUPPORTED, "es_set_strategy_state: the strategy keeps no such state");
    es_status s = ES_OK;
    if (sigma_vec && (s = copy_rows_in(h, h->cmaC ? h->cmaC : h->sig, sigma_vec)) != ES_OK) return s;
    if (velocity && (s = copy_rows_in(h, h->vel, velocity)) != ES_OK) return s;
    if (sigma_vec && h->cmaC)
        ES_HIP(h, launch_cma_scale(h->g, h->sig, h->cmaC, h->hp[h->hp_cur], h->stream), "Sep-CMA-ES scale");
    return ES_OK;
}

es_status es_get_penalty(es_handle* h, float* pen)
{
    if (!h || !pen) return h ? fail(h, ES_ERR_ARG, "es_get_penalty: null buffer") : ES_ERR_ARG;
    if (!h->pen) return fail(h, ES_ERR_UNSUPPORTED, "es_get_penalty needs w_decay > 0");
    ES_HIP(h, hipMemcpyAsync(pen, h->pen, sizeof(float) * (size_t)h->g.N * h->g.R, hipMemcpyDeviceToDevice,
                             h->stream),
           "copy penalty");
    return ES_OK;
}

es_status es_get_problem_data(es_handle* h, float* out)
{
    if (!h || !out) return h ? fail(h, ES_ERR_ARG, "es_get_problem_data: null buffer") : ES_ERR_ARG;
    if (!h->pdata) return fail(h, ES_ERR_UNSUPPORTED, "this problem has no problem data");
    ES_HIP(h, hipMemcpyAsync(out, h->pdata, sizeof(float) * (size_t)h->g.D, hipMemcpyDeviceToDevice, h->stream),
           "copy problem data");
    return ES_OK;
}

es_status es_debug_noise(es_handle* h, int32_t run, int64_t t, int32_t pair, uint32_t* words, float* eps)
{
    if (!h) return ES_ERR_ARG;
    if (run < 0 || run >= h->g.R || pair < 0 || pair >= h->g.P || t < 0 || t > 0xFFFFFFFFll)
        return fail(h, ES_ERR_ARG, "es_debug_noise: run, pair or t out of range");
    ES_HIP(h, launch_debug_noise(h->g, h->cfg, run, (uint32_t)t, pair, words, eps, h->stream), "noise kernel");
    return ES_OK;
}

es_status es_save_state(es_handle* h, void* host_buf, size_t* bytes)
{
    if (!h || !bytes) return ES_ERR_ARG;
    const Geometry& g = h->g;
    const size_t rows = (size_t)g.Dp * g.R * sizeof(float);
    const size_t extra = (h->sig ? rows : 0) + (h->vel ? rows : 0) + (h->cmaC ? rows : 0);
    const size_t need = sizeof(CkptHeader) + 4 * rows + g.R * (sizeof(uint32_t) + 3 * sizeof(float)) + extra;
    if (!host_buf) {
        *bytes = need;
        return ES_OK;
    }
    if (*bytes < need) return fail(h, ES_ERR_ARG, "es_save_state: buffer too small (%zu < %zu)", *bytes, need);
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_save_state: an ask is open");
    char* p = static_cast<char*>(host_buf);
    CkptHeader hd;
    std::memset(&hd, 0, sizeof(hd));
    hd.magic = kCheckpointMagic;
    hd.version = 1;
    hd.cfg = h->cfg;
    hd.t = h->t;
    hd.D = g.D;
    hd.R = g.R;
    std::memcpy(p, &hd, sizeof(hd));
    p += sizeof(hd);
    const float* srcs[4] = {h->m, h->m1, h->v, h->best_x};
    for (const float* s : srcs) {
        ES_HIP(h, hipMemcpyAsync(p, s, rows, hipMemcpyDeviceToHost, h->stream), "save state");
        p += rows;
    }
    ES_HIP(h, hipMemcpyAsync(p, h->best_okey, g.R * sizeof(uint32_t), hipMemcpyDeviceToHost, h->stream), "save best");
    p += g.R * sizeof(uint32_t);
    ES_HIP(h, hipMemcpyAsync(p, h->best_f, g.R * sizeof(float), hipMemcpyDeviceToHost, h->stream), "save best");
    p += g.R * sizeof(float);
    ES_HIP(h, hipMemcpyAsync(p, h->hp[h->hp_cur], 2 * g.R * sizeof(float), hipMemcpyDeviceToHost, h->stream),
           "save sigma and lr");
    p += 2 * g.R * sizeof(float);
    for (const float* src : {static_cast<const float*>(h->sig), static_cast<const float*>(h->vel),
                             static_cast<const float*>(h->cmaC)}) {
        if (!src) continue;
        ES_HIP(h, hipMemcpyAsync(p, src, rows, hipMemcpyDeviceToHost, h->stream), "save strategy state");
        p += rows;
    }
    ES_HIP(h, hipStreamSynchronize(h->stream), "save sync");
    *bytes = need;
    return ES_OK;
}

es_status es_load_state(es_handle* h, const void* host_buf, size_t bytes)
{
    if (!h || !host_buf) return ES_ERR_ARG;
    if (h->phase != READY) return fail(h, ES_ERR_SEQUENCE, "es_load_state: an ask is open");
    const Geometry& g = h->g;
    const size_t rows = (size_t)g.Dp * g.R * sizeof(float);
    const size_t extra = (h->sig ? rows : 0) + (h->vel ? rows : 0) + (h->cmaC ? rows : 0);
    const size_t need = sizeof(CkptHeader) + 4 * rows + g.R * (sizeof(uint32_t) + 3 * sizeof(float)) + extra;
    if (bytes < need) return fail(h, ES_ERR_ARG, "es_load_state: checkpoint too small");
    CkptHeader hd;
    std::memcpy(&hd, host_buf, sizeof(hd));
    if (hd.magic != kCheckpointMagic || hd.version != 1)
        return fail(h, ES_ERR_ARG, "es_load_state: not a checkpoint of this library");
    if (std::memcmp(&hd.cfg, &h->cfg, sizeof(es_config)) != 0 || hd.D != g.D || hd.R != g.R)
        return fail(h, ES_ERR_ARG, "es_load_state: checkpoint was written with another config");
    const char* p = static_cast<const char*>(host_buf) + sizeof(hd);
    float* dsts[4] = {h->m, h->m1, h->v, h->best_x};
    for (float* d : dsts) {
        ES_HIP(h, hipMemcpyAsync(d, p, rows, hipMemcpyHostToDevice, h->stream), "load state");
        p += rows;
    }
    ES_HIP(h, hipMemcpyAsync(h->best_okey, p, g.R * sizeof(uint32_t), hipMemcpyHostToDevice, h->stream), "load best");
    p += g.R * sizeof(uint32_t);
    ES_HIP(h, hipMemcpyAsync(h->best_f, p, g.R * sizeof(float), hipMemcpyHostToDevice, h->stream), "load best");
    p += g.R * sizeof(float);
    ES_HIP(h, hipMemcpyAsync(h->hp[h->hp_cur], p, 2 * g.R * sizeof(float), hipMemcpyHostToDevice, h->stream),
           "load sigma and lr");
    p += 2 * g.R * sizeof(float);
    for (float* dst : {h->sig, h->vel, h->cmaC}) {
        if (!dst) continue;
        ES_HIP(h, hipMemcpyAsync(dst, p, rows, hipMemcpyHostToDevice, h->stream), "load strategy state");
        p += rows;
    }
    es_status st = clear_grid_flag(h);
    if (st != ES_OK) return st;
    ES_HIP(h, hipStreamSynchronize(h->stream), "load sync");
    if (hd.t != h->t) h->teacher_t = -1;
    h->t = hd.t;
    return ES_OK;
}

es_status es_sync(es_handle* h)
{
    if (!h) return ES_ERR_ARG;
    ES_HIP(h, hipStreamSynchronize(h->stream), "stream synchronize");
    if (h->grid_err) {
        uint32_t flag = 0;
        ES_HIP(h, hipMemcpy(&flag, h->grid_err, sizeof(flag), hipMemcpyDeviceToHost), "grid loop flag");
        if (flag) return fail(h, ES_ERR_HIP, "grid generation loop: a wait gave up; the state is not valid");
    }
    return ES_OK;
}

void es_destroy(es_handle* h)
{
    if (!h) return;
    (void)hipStreamSynchronize(h->stream);
    free_all(h);
    delete h;
}

}  // extern "C"
