// es_kernels.hip -- gfx950 kernels of one batched ES generation (OpenAI-ES,
// and the PGPE, SNES and Sep-CMA-ES strategies of Table 1 on the same path).
//
//   k_init            initial mean (Listing 1 initialize), zero Adam moments
//   k_problem_data    shift vector / teacher network from the base seed
//   k_fill_rows       per-dimension state rows (sigma vector, C) at init
//   k_ask             optional materialised population (Sec. 2.1 ask)
//   k_eval_bbob       fused sample + evaluate (Sec. 2.1 evaluate) for the
//                     benchmark problems; lane = antithetic pair (or member
//                     pair for independent sampling), D chunked
//   k_eval_reduce     fixed-order sum of the per-chunk partials -> fitness
//   k_rank            fitness shaping (Sec. 3.2): centered ranks with index
//                     tie-break, raw keys, z-scores, weight decay, the rank
//                     tables of SNES and Sep-CMA-ES; antithetic fold,
//                     best-so-far, the schedule step of sigma and lr
//   k_tell            noise sums over the pairs regenerated per Philox block
//                     (g = E^T y / (N sigma) for OpenAI-ES, Sec. 2.1), fused
//                     with the strategy's update; lane = a block of four dims;
//                     for the MLP problem its launch also runs the next
//                     generation's teacher rows (es_teacher.hpp)
//   k_tell_fold       the split gradient's partial sums in split order, then
//                     the update
//   k_clipup_velocity, k_clipup_apply   ClipUp's two norm passes
//   k_sepcma_finish, k_cma_scale        Sep-CMA-ES second pass, sampling scale
//   k_run_fused       T whole generations in one launch for small runs
//   k_debug_noise     raw words and normals of one stream (diagnostics)
//
// Every reduction runs in a fixed order (no floating-point atomics), so a
// launch is bit-reproducible.  Perturbation sums use short fp32 chains folded
// into fp64 accumulators.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stddef.h>

#include <mutex>
#include <type_traits>

#include "es_device.hpp"
#include "es_internal.hpp"

namespace esmi {

namespace {

constexpr int EVAL_MAX_WG = 1024; // lanes = antithetic pairs
constexpr int EVAL_FOLD = 4;      // Philox blocks summed in fp32 before the fp64 fold
constexpr int RED_SLICES = 16;    // chunk slices per member in the partial reduce
constexpr int RANK_PAIRS = 4;     // pairs per rank workgroup
constexpr int RANK_SLICES = 64;   // key slices per pair
constexpr int TELL_LANES = 64;    // Philox blocks per tell workgroup
constexpr int TELL_MAX_PS = 16;   // pair slices per tell workgroup (one wave each)
constexpr int TELL_GROUP = 16;    // fp32 pairs folded into the fp64 sum at once
constexpr int FUSED_WG = 256;     // threads of the fused multi-generation workgroup
constexpr int GRID_WG = 1024;      // threads of a grid-loop workgroup (four waves per SIMD)
constexpr uint32_t GRID_SPIN_LIMIT = 1u << 20;  // polls before a grid-loop wait gives up (the default)
constexpr int FUSED_PRIO = 3;     // wave priority of the fused loop's short phases (the highest)

// MLP 64-256-256-16, flattened [out][in] per layer then the bias.  Returns
// 1/sqrt(fan_in) for a weight and 0 for a bias.
__device__ __forceinline__ float mlp_init_scale(int64_t i)
{
    if (i < 16384) return 0.125f;   // W1 [256][64]
    if (i < 16640) return 0.0f;     // b1
    if (i < 82176) return 0.0625f;  // W2 [256][256]
    if (i < 82432) return 0.0f;     // b2
    if (i < 86528) return 0.0625f;  // W3 [16][256]
    return 0.0f;                    // b3
}

// ---------------------------------------------------------------------------
__global__ void k_init(float* __restrict__ m, float* __restrict__ m1, float* __restrict__ v,
                       float* __restrict__ best_x, uint64_t seed, int64_t D, int64_t nb, int32_t R,
                       int32_t init, float lo, float range)
{
    const int64_t total = (int64_t)R * nb;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / nb, b = i - r * nb;
        const uint64_t key = seed + (uint64_t)r;
        float o[4] = {0.f, 0.f, 0.f, 0.f};
        if (init == ES_INIT_UNIFORM) {
            const uint4 w = philox4x32_10((uint32_t)key, (uint32_t)(key >> 32), (uint32_t)b, 0, 0, DOM_INIT);
            const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) o[k] = fmaf(range, bm_turns(ww[k]), lo);
        } else if (init == ES_INIT_FANIN_NORMAL) {
            float e[4];
            normals4(key, (uint32_t)b, 0, 0, DOM_INIT, e);
#pragma unroll
            for (int k = 0; k < 4; ++k) o[k] = e[k] * mlp_init_scale(4 * b + k);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (4 * b + k >= D) o[k] = 0.f;
        const int64_t off = r * 4 * nb + 4 * b;
        *reinterpret_cast<float4*>(m + off) = make_float4(o[0], o[1], o[2], o[3]);
        *reinterpret_cast<float4*>(m1 + off) = make_float4(0.f, 0.f, 0.f, 0.f);
        *reinterpret_cast<float4*>(v + off) = make_float4(0.f, 0.f, 0.f, 0.f);
        *reinterpret_cast<float4*>(best_x + off) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

__global__ void k_problem_data(float* __restrict__ out, uint64_t seed, int64_t D, int64_t nb, int32_t problem)
{
    for (int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; b < nb;
         b += (int64_t)gridDim.x * blockDim.x) {
        float e[4];
        normals4(seed, (uint32_t)b, 0, 0, DOM_PROBLEM, e);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float o = problem == ES_PROB_MLP ? e[k] * mlp_init_scale(4 * b + k) : e[k];
            if (4 * b + k >= D) o = 0.f;
            out[4 * b + k] = o;
        }
    }
}

// ---------------------------------------------------------------------------
__global__ void k_ask(const float* __restrict__ m, float* __restrict__ x, uint64_t seed, uint32_t t,
                      int64_t D, int64_t nb, int32_t N, int32_t P, int32_t R, const float* __restrict__ hp,
                      const float* __restrict__ svec, int32_t indep)
{
    const int64_t total = (int64_t)R * P * nb;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = i % nb;
        const int64_t rp = i / nb;
        const int64_t p = rp % P, r = rp / P;
        float e[4], e2[4];
        normals4(seed + (uint64_t)r, (uint32_t)b, (uint32_t)p, t, DOM_NOISE, e);
        // independent members (Sep-CMA-ES): the second member has its own row
        if (indep) normals4(seed + (uint64_t)r, (uint32_t)b, (uint32_t)(p + P), t, DOM_NOISE, e2);
        const float* mr = m + r * 4 * nb;
        float* xp = x + (r * N + p) * D;
        float* xm = x + (r * N + p + P) * D;
        const float sigma = hp[r];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int64_t d = 4 * b + k;
            if (d < D) {
                const float g = svec ? svec[r * 4 * nb + d] : sigma;
                xp[d] = fmaf(g, e[k], mr[d]);
                xm[d] = indep ? fmaf(g, e2[k], mr[d]) : fmaf(-g, e[k], mr[d]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Fused sample + evaluate.  Workgroup = up to EVAL_MAX_WG antithetic pairs of
// one run over one chunk of Philox blocks.  The chunk's mean (and shift)
// words are the same for the whole workgroup, so they come through the
// scalar cache, EVAL_FOLD blocks (16 floats) per scalar load, fetched one
// group ahead; every lane regenerates its own pair's normals and scores both
// members.  Workgroup ids are dealt to the 8 XCDs round robin, so the pair
// groups of one chunk are given ids that share an XCD (and its L2).
template <int PROB>
struct BlockTerm;

// acc(s, x, shift, A): the running fp32 sum s plus one dim's term, each as
// one explicit operation (an fma where the term is a square), so that the
// rounding never depends on how the compiler contracts the code around it
template <>
struct BlockTerm<ES_PROB_SPHERE> {
    static __device__ __forceinline__ float acc(float s, float x, float, float) { return fmaf(x, x, s); }
};
template <>
struct BlockTerm<ES_PROB_SHIFTED_SPHERE> {
    static __device__ __forceinline__ float acc(float s, float x, float sh, float)
    {
        const float d = __fsub_rn(x, sh);
        return fmaf(d, d, s);
    }
};
template <>
struct BlockTerm<ES_PROB_RASTRIGIN> {
    static __device__ __forceinline__ float acc(float s, float x, float, float a)
    {
        return __fadd_rn(s, fmaf(x, x, __fmul_rn(-a, cos_2pi(x))));
    }
};

__device__ __forceinline__ float rosen_term(float xi, float xn)
{
    const float q = fmaf(-xi, xi, xn);
    const float o = 1.0f - xi;
    return fmaf(100.0f * q, q, o * o);
}

// Running state of one lane: both members' sums and, for Rosenbrock, the
// members' values at the previous dim.
struct EvalLane {
    double accp, accm;
    float xlp, xlm;
    bool have_prev;
};

// Sampling modes of the evaluate kernels: antithetic with the run's scalar
// sigma (OpenAI-ES), antithetic with a per-dimension sigma (PGPE, SNES), and
// independent members with a per-dimension scale (Sep-CMA-ES: the lane's
// second member uses Philox row p + P and the plus sign).
enum SampleMode { SM_SCALAR = 0, SM_VEC = 1, SM_INDEP = 2 };

// Terms of one full Philox block (four live dims) for both members: the
// first from normals e, the second from -e (antithetic) or e2 (independent).
template <int PROB, int SM>
__device__ __forceinline__ void block_terms(const float e[4], const float e2[4], const float mv[4], const float sv[4],
                                            const float* gv, float sg, float ra, EvalLane& L, float& sp, float& sm)
{
    if constexpr (PROB == ES_PROB_ROSENBROCK) {
        float xp[4], xm[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float g = SM != SM_SCALAR ? gv[k] : sg;
            xp[k] = fmaf(g, e[k], mv[k]);
            xm[k] = SM == SM_INDEP ? fmaf(g, e2[k], mv[k]) : fmaf(-g, e[k], mv[k]);
        }
        float tp = rosen_term(xp[0], xp[1]) + rosen_term(xp[1], xp[2]) + rosen_term(xp[2], xp[3]);
        float tm = rosen_term(xm[0], xm[1]) + rosen_term(xm[1], xm[2]) + rosen_term(xm[2], xm[3]);
        if (L.have_prev) {
            tp += rosen_term(L.xlp, xp[0]);
            tm += rosen_term(L.xlm, xm[0]);
        }
        L.have_prev = true;
        L.xlp = xp[3];
        L.xlm = xm[3];
        sp += tp;
        sm += tm;
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float g = SM != SM_SCALAR ? gv[k] : sg;
            sp = BlockTerm<PROB>::acc(sp, fmaf(g, e[k], mv[k]), sv[k], ra);
            sm = BlockTerm<PROB>::acc(sm, SM == SM_INDEP ? fmaf(g, e2[k], mv[k]) : fmaf(-g, e[k], mv[k]), sv[k], ra);
        }
    }
}

// Both members' sums of pair `row` over the Philox blocks [b0, b1) of one
// run: fp32 sums of EVAL_FOLD blocks folded into fp64, in block order.  The
// per-call kernel and the fused loop share this code, so both produce the
// same bits.  V names the counter word that varies across the wave.
template <int PROB, int V, int SM = SM_SCALAR>
__device__ __forceinline__ void eval_chunk(const float* __restrict__ mr, const float* __restrict__ pdata,
                                           uint32_t k0, uint32_t k1, uint32_t row, uint32_t t, int64_t b0,
                                           int64_t b1, int64_t D, float sg, float ra, double& accp, double& accm,
                                           const float* __restrict__ gr = nullptr, uint32_t row2 = 0, int64_t mshift = 0,
                                           float4* __restrict__ nout = nullptr, int32_t nstride = 0)
{
    // the mean of dim d is mr[d - mshift] (a window of the row in LDS); with
    // nout, the normals of block b0 + i are also stored at nout[i nstride]
    auto normals = [&](int64_t b, float e[4]) {
        box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)b, row, t, DOM_NOISE), e);
        if (nout) nout[(b - b0) * nstride] = make_float4(e[0], e[1], e[2], e[3]);
    };
    constexpr bool VEC = SM != SM_SCALAR;
    const int64_t nfull = D / 4;
    const int32_t nf = (int32_t)((b1 < nfull ? b1 : nfull) - b0);  // full blocks in [b0, b1) (may be <= 0)
    EvalLane L{0.0, 0.0, 0.f, 0.f, false};
    if (PROB == ES_PROB_ROSENBROCK && b0 > 0) {
        float e[4], e2[4] = {0.f, 0.f, 0.f, 0.f};
        box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)(b0 - 1), row, t, DOM_NOISE), e);
        if constexpr (SM == SM_INDEP) box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)(b0 - 1), row2, t, DOM_NOISE), e2);
        const float mv = mr[4 * b0 - 1 - mshift];
        const float g = VEC ? gr[4 * b0 - 1] : sg;
        L.xlp = fmaf(g, e[3], mv);
        L.xlm = SM == SM_INDEP ? fmaf(g, e2[3], mv) : fmaf(-g, e[3], mv);
        L.have_prev = true;
    }

    const float zero4[4] = {0.f, 0.f, 0.f, 0.f};
    int32_t i = 0;
    for (; i + EVAL_FOLD <= nf; i += EVAL_FOLD) {
        const int64_t bg = b0 + i;
        float mv[4 * EVAL_FOLD], sv[4 * EVAL_FOLD], gv[VEC ? 4 * EVAL_FOLD : 1];
#pragma unroll
        for (int q = 0; q < 4 * EVAL_FOLD; ++q) mv[q] = mr[4 * bg + q - mshift];
        if constexpr (VEC) {
#pragma unroll
            for (int q = 0; q < 4 * EVAL_FOLD; ++q) gv[q] = gr[4 * bg + q];
        }
        if constexpr (PROB == ES_PROB_SHIFTED_SPHERE) {
#pragma unroll
            for (int q = 0; q < 4 * EVAL_FOLD; ++q) sv[q] = pdata[4 * bg + q];
        }
        float sp = 0.f, sm = 0.f;
#pragma unroll
        for (int k = 0; k < EVAL_FOLD; ++k) {
            float e[4], e2[4] = {0.f, 0.f, 0.f, 0.f};
            normals(bg + k, e);
            if constexpr (SM == SM_INDEP)
                box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)(bg + k), row2, t, DOM_NOISE), e2);
            block_terms<PROB, SM>(e, e2, mv + 4 * k, PROB == ES_PROB_SHIFTED_SPHERE ? sv + 4 * k : zero4,
                                  VEC ? gv + 4 * k : nullptr, sg, ra, L, sp, sm);
        }
        L.accp += (double)sp;
        L.accm += (double)sm;
    }
    for (; i < nf; ++i) {
        const int64_t b = b0 + i;
        float mv[4], sv[4] = {0.f, 0.f, 0.f, 0.f}, gv[4] = {sg, sg, sg, sg};
#pragma unroll
        for (int q = 0; q < 4; ++q) mv[q] = mr[4 * b + q - mshift];
        if constexpr (VEC) {
#pragma unroll
            for (int q = 0; q < 4; ++q) gv[q] = gr[4 * b + q];
        }
        if constexpr (PROB == ES_PROB_SHIFTED_SPHERE) {
#pragma unroll
            for (int q = 0; q < 4; ++q) sv[q] = pdata[4 * b + q];
        }
        float e[4], e2[4] = {0.f, 0.f, 0.f, 0.f};
        normals(b, e);
        if constexpr (SM == SM_INDEP) box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)b, row2, t, DOM_NOISE), e2);
        float sp = 0.f, sm = 0.f;
        block_terms<PROB, SM>(e, e2, mv, sv, gv, sg, ra, L, sp, sm);
        L.accp += (double)sp;
        L.accm += (double)sm;
    }

    // Ragged tail: the last Philox block holds D % 4 live dims.
    if (b1 > nfull && nfull >= b0) {
        const int64_t b = nfull;
        const int nv = (int)(D - 4 * b);
        float e[4], e2[4] = {0.f, 0.f, 0.f, 0.f};
        normals(b, e);
        if constexpr (SM == SM_INDEP) box_muller4(philox4x32_10<V>(k0, k1, (uint32_t)b, row2, t, DOM_NOISE), e2);
        float sp = 0.f, sm = 0.f;
        for (int k = 0; k < nv; ++k) {
            const float mv = mr[4 * b + k - mshift];
            const float g = VEC ? gr[4 * b + k] : sg;
            const float xp = fmaf(g, e[k], mv), xm = SM == SM_INDEP ? fmaf(g, e2[k], mv) : fmaf(-g, e[k], mv);
            if constexpr (PROB == ES_PROB_ROSENBROCK) {
                if (L.have_prev) {
                    sp += rosen_term(L.xlp, xp);
                    sm += rosen_term(L.xlm, xm);
                }
                L.have_prev = true;
                L.xlp = xp;
                L.xlm = xm;
            } else {
                const float s = PROB == ES_PROB_SHIFTED_SPHERE ? pdata[4 * b + k] : 0.f;
                sp = BlockTerm<PROB>::acc(sp, xp, s, ra);
                sm = BlockTerm<PROB>::acc(sm, xm, s, ra);
            }
        }
        L.accp += (double)sp;
        L.accm += (double)sm;
    }
    accp = L.accp;
    accm = L.accm;
}

// Eight waves per SIMD (two 16-wave workgroups per CU): the compiler then
// keeps the kernel within the scalar register budget of that occupancy.
template <int PROB, int SM>
__global__ __launch_bounds__(EVAL_MAX_WG) __attribute__((amdgpu_waves_per_eu(8, 8))) void k_eval_bbob(
    const float* __restrict__ m, const float* __restrict__ pdata, float* __restrict__ partial,
    uint64_t seed, uint32_t t, int64_t D, int64_t nb, int32_t N, int32_t P, int64_t bc, int64_t nchunks,
    int32_t n_pg, const float* __restrict__ hp, float ra, const float* __restrict__ svec)
{
    const int32_t r = blockIdx.y;
    const float sigma = hp[r];
    const uint32_t w = blockIdx.x;
    const uint32_t slot = w >> 3, xcd = w & 7u;
    const int32_t pg = (int32_t)(slot % (uint32_t)n_pg);
    const int64_t chunk = (int64_t)(slot / (uint32_t)n_pg) * 8 + xcd;
    if (chunk >= nchunks) return;
    const int32_t p = pg * (int32_t)blockDim.x + (int32_t)threadIdx.x;
    const uint32_t row = (uint32_t)(p < P ? p : P - 1);
    const uint64_t key = seed + (uint64_t)r;
    const int64_t b0 = chunk * bc;
    const int64_t b1 = b0 + bc < nb ? b0 + bc : nb;
    // sigma lives in a VGPR so that fmaf(sigma, eps, m) can take m from an SGPR
    float sg;
    asm volatile("v_mov_b32 %0, %1" : "=v"(sg) : "s"(sigma));
    double accp, accm;
    eval_chunk<PROB, LANES_ROW, SM>(m + (int64_t)r * 4 * nb, pdata, (uint32_t)key, (uint32_t)(key >> 32), row, t, b0,
                                    b1, D, sg, ra, accp, accm, SM != SM_SCALAR ? svec + (int64_t)r * 4 * nb : nullptr,
                                    row + (uint32_t)P);
    if (p < P) {
        float* o = partial + (chunk * gridDim.y + r) * (int64_t)N;
        o[p] = (float)accp;
        o[p + P] = (float)accm;
    }
}

// fit[r][j] = (add + sum over chunks (fixed order) of the partials) / div
// (div = 1 for fitness, D for the weight-decay mean square).
// Workgroup = 64 members x RED_SLICES chunk slices.
__global__ __launch_bounds__(64 * RED_SLICES) void k_eval_reduce(const float* __restrict__ partial,
                                                                 float* __restrict__ fit, int32_t N, int32_t R,
                                                                 int64_t nchunks, double add, double div)
{
    __shared__ double red[RED_SLICES][64];
    const int32_t r = blockIdx.y;
    const int32_t tx = threadIdx.x & 63, s = threadIdx.x >> 6;
    const int32_t j = blockIdx.x * 64 + tx;
    double acc = 0.0;
    if (j < N) {
        const int64_t stride = (int64_t)RED_SLICES * R * N;
        const float* __restrict__ q = partial + ((int64_t)s * R + r) * N + j;
        int64_t c = s;
        // eight loads in flight, summed in chunk order
        for (; c + 7 * RED_SLICES < nchunks; c += 8 * RED_SLICES, q += 8 * stride) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = q[u * stride];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc += (double)v[u];
        }
        for (; c < nchunks; c += RED_SLICES, q += stride) acc += (double)*q;
    }
    red[s][tx] = acc;
    __syncthreads();
    if (s == 0 && j < N) {
        double tot = add;
#pragma unroll
        for (int q = 0; q < RED_SLICES; ++q) tot += red[q][tx];
        fit[(int64_t)r * N + j] = (float)(tot / div);
    }
}

// ---------------------------------------------------------------------------
// Fitness shaping (Sec. 3.2).  Workgroup = RANK_PAIRS pairs x RANK_SLICES key
// slices of one run; the run's order keys sit in LDS.  The shaped key is the
// fitness (negated when maximising, NaN the worst) plus, with weight decay,
// fl32(w * pen_j) for a finite key.  rank_j counts keys that sort before j in
// a stable ascending order: smaller key, or equal key and lower index.
// y_j: centered-rank table entry, the key itself (raw), or its z-score over
// the finite keys (fp64 mean and population deviation, reduced in a fixed
// order that every workgroup of the run repeats).  The first workgroup of a
// run also steps the run's sigma and learning-rate schedules.
struct ShapeArgs {
    const float* pen;       // [R][N] mean-square penalty or null
    const float* hp_cur;    // [2][R]: sigma, lr of this generation
    float* hp_next;         // [2][R]: after the schedule step
    float w_decay;
    float sigma_decay, sigma_final, lr_decay, lr_final;
    int32_t shaping;        // es_shaping
    int32_t maximize;
    // second folded weight per pair for the sigma-adapting strategies:
    // PGPE b_p = (y_p + y_{p+P})/2 - mean(y), SNES b_p = y_p + y_{p+P}
    float* bfold;           // [R][P] or null
    int32_t bmode;          // 0 none, 1 PGPE, 2 SNES, 3 Sep-CMA-ES (elite list)
    double ybar_table;      // mean of the shaping table (table shaping)
    int32_t* elite;         // [R][N] Sep-CMA-ES: member of rank i, i < mu
    int32_t mu;
    // Sort-based ranks (null: the workgroup counts in LDS): the shaped order
    // keys [R][N], the ranks [R][N] and the per-run statistics [R][4] of
    // k_rank_stats, all made by the kernels ahead of k_rank.
    const uint32_t* gkeys;
    const int32_t* pre_rank;
    const double* stats;
};

__device__ __forceinline__ float shaped_key(float f, float pen, int maximize, float w_decay)
{
    float k = maximize ? -f : f;
    if (k != k) return __builtin_inff();
    if (w_decay != 0.0f && __builtin_isfinite(k)) k = __fadd_rn(k, __fmul_rn(w_decay, pen));
    return k;
}

__device__ __forceinline__ float key_value(uint32_t K)
{
    return __uint_as_float((K & 0x80000000u) ? (K & 0x7FFFFFFFu) : ~K);
}

__device__ __forceinline__ float schedule_step(float x, float decay, float final)
{
    const float y = __fmul_rn(x, decay);
    return y > final ? y : final;
}

// Sum of v over the workgroup in a fixed tree order (blockDim.x = 256).
__device__ __forceinline__ double block_sum(double v, double* red)
{
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = RANK_PAIRS * RANK_SLICES / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const double out = red[0];
    __syncthreads();
    return out;
}

// Per-run statistics of the shaped keys kp[0, N) that the weights need:
// the z-score mean and 1 / (deviation + 1e-10) (fp64, finite keys), PGPE's
// mean of y when y is not a permutation of the table, and with weight decay
// the raw best (smallest raw order key, lowest index first) in raw_best[2].
// Sums over the run in one fixed order for a 256-lane workgroup, so every
// workgroup (and k_rank_stats) gets the same bits.
__device__ void rank_stats(const uint32_t* kp, const float* fr, const float* pr, int32_t N, const ShapeArgs& sa,
                           double* red, uint32_t* raw_best, double& mu_out, double& inv_sd_out, double& ybar_out)
{
    double mu = 0.0, inv_sd = 0.0;
    if (sa.shaping == ES_SHAPE_Z_SCORE) {
        double sum = 0.0, n = 0.0;
        for (int32_t k = threadIdx.x; k < N; k += blockDim.x) {
            const float v = key_value(kp[k]);
            if (__builtin_isfinite(v)) { sum += (double)v; n += 1.0; }
        }
        sum = block_sum(sum, red);
        n = block_sum(n, red);
        mu = n > 0.0 ? sum / n : 0.0;
        double ss = 0.0;
        for (int32_t k = threadIdx.x; k < N; k += blockDim.x) {
            const float v = key_value(kp[k]);
            if (__builtin_isfinite(v)) ss += ((double)v - mu) * ((double)v - mu);
        }
        ss = block_sum(ss, red);
        const double sd = n > 0.0 ? sqrt(ss / n) : 0.0;
        inv_sd = sd + 1e-10;
    }
    // PGPE baseline: the mean of y over the run (table shaping: the table's
    // own mean, as the ranks are a permutation)
    double ybar = sa.ybar_table;
    if (sa.bmode == 1 && sa.shaping != ES_SHAPE_CENTERED_RANK) {
        double acc = 0.0;
        for (int32_t k = threadIdx.x; k < N; k += blockDim.x) {
            float yk;
            if (sa.shaping == ES_SHAPE_RAW) {
                yk = sa.w_decay != 0.0f ? shaped_key(fr[k], pr[k], sa.maximize, sa.w_decay)
                                        : (sa.maximize ? -fr[k] : fr[k]);
            } else {
                const float v = key_value(kp[k]);
                yk = __builtin_isfinite(v) ? (float)(((double)v - mu) / inv_sd) : 0.0f;
            }
            acc += (double)yk;
        }
        ybar = block_sum(acc, red) / (double)N;
    }
    // With weight decay the best-so-far still follows the raw fitness: the
    // smallest raw key, lowest index first.
    const bool penalised = sa.w_decay != 0.0f;
    if (penalised) {
        if (threadIdx.x == 0) { raw_best[0] = 0xFFFFFFFFu; raw_best[1] = 0xFFFFFFFFu; }
        __syncthreads();
        uint32_t bk = 0xFFFFFFFFu, bj = 0xFFFFFFFFu;
        for (int32_t k = threadIdx.x; k < N; k += blockDim.x) {
            const uint32_t K = order_key(fr[k], sa.maximize);
            if (K < bk) { bk = K; bj = (uint32_t)k; }
        }
        atomicMin(&raw_best[0], bk);
        __syncthreads();
        if (bk == raw_best[0]) atomicMin(&raw_best[1], bj);
        __syncthreads();
    }

    mu_out = mu;
    inv_sd_out = inv_sd;
    ybar_out = ybar;
}

__global__ __launch_bounds__(RANK_PAIRS * RANK_SLICES) void k_rank(
    const float* __restrict__ fit, const float* __restrict__ table, float* __restrict__ y,
    int32_t* __restrict__ rank, float* __restrict__ wfold, uint32_t* __restrict__ best_okey,
    float* __restrict__ best_f, int32_t* __restrict__ best_j, float* __restrict__ gen_best, int32_t N,
    int32_t P, int32_t R, ShapeArgs sa)
{
    extern __shared__ uint32_t keys[];
    __shared__ int32_t cnt[RANK_SLICES][RANK_PAIRS][2];
    __shared__ double red[RANK_PAIRS * RANK_SLICES];
    __shared__ uint32_t raw_best[2];
    const int32_t r = blockIdx.y;
    const float* __restrict__ fr = fit + (int64_t)r * N;
    const float* __restrict__ pr = sa.pen ? sa.pen + (int64_t)r * N : nullptr;
    // this workgroup's own members, fetched first (used after the count)
    const int32_t tx = threadIdx.x % RANK_PAIRS, s = threadIdx.x / RANK_PAIRS;
    const int32_t p = blockIdx.x * RANK_PAIRS + tx;
    const bool valid = p < P;
    const int32_t j1 = valid ? p : 0, j2 = j1 + P;
    const float f1 = fr[j1], f2 = fr[j2];
    const bool pre = sa.gkeys != nullptr;
    // the run's keys: eight loads per lane in flight at once
    constexpr int KU = 8;
    for (int32_t k0 = threadIdx.x; !pre && k0 < N; k0 += KU * (int32_t)blockDim.x) {
        float fv[KU], pv[KU];
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int32_t k = k0 + u * (int32_t)blockDim.x;
            fv[u] = k < N ? fr[k] : 0.0f;
            pv[u] = pr && k < N ? pr[k] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int32_t k = k0 + u * (int32_t)blockDim.x;
            if (k < N) keys[k] = order_key(shaped_key(fv[u], pv[u], sa.maximize, sa.w_decay), 0);
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        sa.hp_next[r] = schedule_step(sa.hp_cur[r], sa.sigma_decay, sa.sigma_final);
        sa.hp_next[R + r] = schedule_step(sa.hp_cur[R + r], sa.lr_decay, sa.lr_final);
    }
    __syncthreads();

    double mu, inv_sd, ybar;
    const bool penalised = sa.w_decay != 0.0f;
    if (pre) {
        const double* st = sa.stats + 4 * (int64_t)r;
        mu = st[0];
        inv_sd = st[1];
        ybar = st[2];
        if (threadIdx.x == 0) {
            const uint64_t rb = __double_as_longlong(st[3]);
            raw_best[0] = (uint32_t)(rb >> 32);
            raw_best[1] = (uint32_t)rb;
        }
        __syncthreads();
    } else {
        rank_stats(keys, fr, pr, N, sa, red, raw_best, mu, inv_sd, ybar);
    }
    const uint32_t* kp = pre ? sa.gkeys + (int64_t)r * N : keys;
    const uint32_t K1 = kp[j1], K2 = kp[j2];
    // the count of slice s (the sort-based ranks arrive whole, in slice 0)
    const int32_t kb = pre ? 0 : (int32_t)(((int64_t)N * s) / RANK_SLICES);
    const int32_t ke = pre ? 0 : (int32_t)(((int64_t)N * (s + 1)) / RANK_SLICES);
    // rank_j = #{k : key_k < key_j} + #{k < j : key_k == key_j}, i.e. the
    // number of composites (key_k, k) below (key_j, j): one 64-bit compare
    int32_t c1 = 0, c2 = 0;
    const uint64_t cj1 = ((uint64_t)K1 << 32) | (uint32_t)j1, cj2 = ((uint64_t)K2 << 32) | (uint32_t)j2;
    int32_t k = kb;
    for (; k + 4 <= ke; k += 4) {
        uint32_t kk[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) kk[u] = keys[k + u];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint64_t ck = ((uint64_t)kk[u] << 32) | (uint32_t)(k + u);
            c1 += ck < cj1;
            c2 += ck < cj2;
        }
    }
    for (; k < ke; ++k) {
        const uint64_t ck = ((uint64_t)keys[k] << 32) | (uint32_t)k;
        c1 += ck < cj1;
        c2 += ck < cj2;
    }
    if (pre && s == 0) {
        c1 = sa.pre_rank[(int64_t)r * N + j1];
        c2 = sa.pre_rank[(int64_t)r * N + j2];
    }
    cnt[s][tx][0] = c1;
    cnt[s][tx][1] = c2;
    __syncthreads();
    if (s != 0 || !valid) return;

    int32_t r1 = 0, r2 = 0;
#pragma unroll
    for (int q = 0; q < RANK_SLICES; ++q) {
        r1 += cnt[q][tx][0];
        r2 += cnt[q][tx][1];
    }
    float y1, y2;
    if (sa.shaping == ES_SHAPE_RAW) {
        // the key itself; without weight decay the fitness keeps its NaN and sign of zero
        y1 = penalised ? shaped_key(f1, pr[j1], sa.maximize, sa.w_decay) : (sa.maximize ? -f1 : f1);
        y2 = penalised ? shaped_key(f2, pr[j2], sa.maximize, sa.w_decay) : (sa.maximize ? -f2 : f2);
    } else if (sa.shaping == ES_SHAPE_Z_SCORE) {
        const float v1 = key_value(K1), v2 = key_value(K2);
        y1 = __builtin_isfinite(v1) ? (float)(((double)v1 - mu) / inv_sd) : 0.0f;
        y2 = __builtin_isfinite(v2) ? (float)(((double)v2 - mu) / inv_sd) : 0.0f;
    } else {
        y1 = table[r1];
        y2 = table[r2];
    }
    float* yr = y + (int64_t)r * N;
    int32_t* rr = rank + (int64_t)r * N;
    yr[j1] = y1;
    yr[j2] = y2;
    rr[j1] = r1;
    rr[j2] = r2;
    wfold[(int64_t)r * P + p] = y1 - y2;
    if (sa.bmode == 1) sa.bfold[(int64_t)r * P + p] = (float)(0.5 * ((double)y1 + (double)y2) - ybar);
    if (sa.bmode == 2) sa.bfold[(int64_t)r * P + p] = y1 + y2;
    if (sa.bmode == 3) {
        if (r1 < sa.mu) sa.elite[(int64_t)r * N + r1] = j1;
        if (r2 < sa.mu) sa.elite[(int64_t)r * N + r2] = j2;
    }
    int32_t jb = -1;
    if (penalised) {
        if ((uint32_t)j1 == raw_best[1]) jb = j1;
        if ((uint32_t)j2 == raw_best[1]) jb = j2;
    } else if (r1 == 0 || r2 == 0) {
        jb = r1 == 0 ? j1 : j2;
    }
    if (jb >= 0) {
        const float fb = jb == j1 ? f1 : f2;
        const uint32_t kb0 = order_key(fb, sa.maximize);
        if (gen_best) gen_best[r] = fb;
        if (kb0 < best_okey[r]) {
            best_okey[r] = kb0;
            best_f[r] = fb;
            best_j[r] = jb;
        } else {
            best_j[r] = -1;
        }
    }
}

// Sort-based ranks, for populations whose keys do not fit a workgroup's LDS.
// Every member's composite key (run << (32 + bn) | order key << bn | member,
// bn = RankSortBuffers::bn) sorts ascending by run, then by key, then by
// index, so the runs come out in order, run r in [r N, (r + 1) N), and a
// member's position there is the count the rank kernel makes: the number of
// keys below its own plus the equal keys of lower index.
__global__ void k_rank_keys(const float* __restrict__ fit, const float* __restrict__ pen, int32_t N, int64_t total,
                            int32_t maximize, float w_decay, int32_t bn, uint32_t* __restrict__ keys,
                            uint64_t* __restrict__ comp)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t K = order_key(shaped_key(fit[i], pen ? pen[i] : 0.0f, maximize, w_decay), 0);
        keys[i] = K;
        const int64_t r = i / N;
        comp[i] = ((uint64_t)r << (32 + bn)) | ((uint64_t)K << bn) | (uint64_t)(i - r * N);
    }
}

// rank[r][member] = position of the member's composite key within run r's
// slice of the sorted keys
__global__ void k_rank_scatter(const uint64_t* __restrict__ sorted, int32_t N, int64_t total, int32_t bn,
                               int32_t* __restrict__ rank)
{
    const uint64_t mask = ((uint64_t)1 << bn) - 1;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / N;
        rank[r * N + (int64_t)(sorted[i] & mask)] = (int32_t)(i - r * N);
    }
}

// One workgroup per run: the statistics every rank workgroup of the run
// would compute (rank_stats, the same order), stored once:
// stats[r] = {mu, 1 / (deviation + 1e-10), ybar, raw best key << 32 | member}.
__global__ __launch_bounds__(RANK_PAIRS * RANK_SLICES) void k_rank_stats(const float* __restrict__ fit,
                                                                       const uint32_t* __restrict__ keys, int32_t N,
                                                                       ShapeArgs sa, double* __restrict__ stats)
{
    __shared__ double red[RANK_PAIRS * RANK_SLICES];
    __shared__ uint32_t raw_best[2];
    const int32_t r = blockIdx.x;
    const float* fr = fit + (int64_t)r * N;
    const float* pr = sa.pen ? sa.pen + (int64_t)r * N : nullptr;
    if (threadIdx.x == 0) { raw_best[0] = 0xFFFFFFFFu; raw_best[1] = 0xFFFFFFFFu; }
    __syncthreads();
    double mu, inv_sd, ybar;
    rank_stats(keys + (int64_t)r * N, fr, pr, N, sa, red, raw_best, mu, inv_sd, ybar);
    if (threadIdx.x == 0) {
        double* st = stats + 4 * (int64_t)r;
        st[0] = mu;
        st[1] = inv_sd;
        st[2] = ybar;
        st[3] = __longlong_as_double((long long)(((uint64_t)raw_best[0] << 32) | raw_best[1]));
    }
}

// ---------------------------------------------------------------------------
// Weighted noise sum of one Philox block over the pairs [pb, pe):
// a64[k] = sum_p w_p eps_{p, 4b+k}, fp32 over TELL_GROUP pairs folded into
// fp64, in pair order.  Shared by the per-call and the fused kernels.
template <int V>
__device__ __forceinline__ void tell_slice(const float* __restrict__ wr, uint32_t k0, uint32_t k1, uint32_t bb,
                                           uint32_t t, int32_t pb, int32_t pe, double a64[4])
{
    int32_t p0 = pb;
    float wv[TELL_GROUP];
    if (p0 + TELL_GROUP <= pe) {
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) wv[q] = wr[p0 + q];
    }
    for (; p0 + TELL_GROUP <= pe; p0 += TELL_GROUP) {
        // fetch the next group's weights while this group's noise is generated
        float wn[TELL_GROUP];
        const int32_t pn = p0 + 2 * TELL_GROUP <= pe ? p0 + TELL_GROUP : p0;  // stays in bounds
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) wn[q] = wr[pn + q];
        float a32[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) {
            float e[4];
            box_muller4(philox4x32_10<V>(k0, k1, bb, (uint32_t)(p0 + q), t, DOM_NOISE), e);
#pragma unroll
            for (int k = 0; k < 4; ++k) a32[k] = fmaf(wv[q], e[k], a32[k]);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) a64[k] += (double)a32[k];
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) wv[q] = wn[q];
    }
    float a32[4] = {0.f, 0.f, 0.f, 0.f};
    // the pairs past the last whole group: independent noise blocks, summed in order
#pragma unroll 4
    for (int32_t p = p0; p < pe; ++p) {
        float e[4];
        box_muller4(philox4x32_10<V>(k0, k1, bb, (uint32_t)p, t, DOM_NOISE), e);
        const float w = wr[p];
#pragma unroll
        for (int k = 0; k < 4; ++k) a32[k] = fmaf(w, e[k], a32[k]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) a64[k] += (double)a32[k];
}

// tell_slice with the pairs' normals of the block given (eps[p], as the
// evaluate stored them) instead of regenerated: the same groups of
// TELL_GROUP pairs folded into fp64, then the rest.
__device__ __forceinline__ void tell_slice_eps(const float* __restrict__ wr, const float4* __restrict__ eps, int32_t pb,
                                               int32_t pe, double a64[4])
{
    int32_t p0 = pb;
    for (; p0 + TELL_GROUP <= pe; p0 += TELL_GROUP) {
        float a32[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) {
            const float4 e = eps[p0 + q];
            const float w = wr[p0 + q];
            a32[0] = fmaf(w, e.x, a32[0]);
            a32[1] = fmaf(w, e.y, a32[1]);
            a32[2] = fmaf(w, e.z, a32[2]);
            a32[3] = fmaf(w, e.w, a32[3]);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) a64[k] += (double)a32[k];
    }
    float a32[4] = {0.f, 0.f, 0.f, 0.f};
    for (int32_t p = p0; p < pe; ++p) {
        const float4 e = eps[p];
        const float w = wr[p];
        a32[0] = fmaf(w, e.x, a32[0]);
        a32[1] = fmaf(w, e.y, a32[1]);
        a32[2] = fmaf(w, e.z, a32[2]);
        a32[3] = fmaf(w, e.w, a32[3]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) a64[k] += (double)a32[k];
}

// Both sums of one Philox block over the pairs [pb, pe) for the strategies
// that adapt a per-dimension sigma: a64[k] = sum_p a_p z_{p,4b+k} and
// b64[k] = sum_p b_p (z^2 - 1), fp32 over TELL_GROUP pairs folded into fp64.
// ROWS: the Philox row of each item comes from rows[] (Sep-CMA-ES: the
// elite members), else it is the item index (the pair).
template <int V, bool ROWS = false>
__device__ __forceinline__ void tell_slice2(const float* __restrict__ ar, const float* __restrict__ br, uint32_t k0,
                                            uint32_t k1, uint32_t bb, uint32_t t, int32_t pb, int32_t pe,
                                            double a64[4], double b64[4], const int32_t* __restrict__ rows = nullptr)
{
    int32_t p0 = pb;
    for (; p0 + TELL_GROUP <= pe; p0 += TELL_GROUP) {
        float av[TELL_GROUP], bv[TELL_GROUP];
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) {
            av[q] = ar[p0 + q];
            bv[q] = br[p0 + q];
        }
        float a32[4] = {0.f, 0.f, 0.f, 0.f}, b32[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < TELL_GROUP; ++q) {
            float e[4];
            const uint32_t row = ROWS ? (uint32_t)rows[p0 + q] : (uint32_t)(p0 + q);
            box_muller4(philox4x32_10<V>(k0, k1, bb, row, t, DOM_NOISE), e);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                a32[k] = fmaf(av[q], e[k], a32[k]);
                b32[k] = fmaf(bv[q], fmaf(e[k], e[k], -1.0f), b32[k]);
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a64[k] += (double)a32[k];
            b64[k] += (double)b32[k];
        }
    }
    float a32[4] = {0.f, 0.f, 0.f, 0.f}, b32[4] = {0.f, 0.f, 0.f, 0.f};
    for (int32_t p = p0; p < pe; ++p) {
        float e[4];
        box_muller4(philox4x32_10<V>(k0, k1, bb, ROWS ? (uint32_t)rows[p] : (uint32_t)p, t, DOM_NOISE), e);
        const float a = ar[p], b = br[p];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a32[k] = fmaf(a, e[k], a32[k]);
            b32[k] = fmaf(b, fmaf(e[k], e[k], -1.0f), b32[k]);
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        a64[k] += (double)a32[k];
        b64[k] += (double)b32[k];
    }
}

// g = sum / (N sigma), then Adam (Kingma & Ba) in fp32 in a fixed operation
// order on one dim; a dim at or beyond D stays zero.
__device__ __forceinline__ void adam_dim(double a64, double inv_ns, const AdamConsts& ac, float lr, int64_t d,
                                         int64_t D, float mo, float m1o, float vo, float& mn, float& m1n,
                                         float& vn, float& gg)
{
    const float g = (float)(a64 * inv_ns);
    gg = g;
    const float nm1 = __builtin_fmaf(ac.beta1, m1o, __fmul_rn(ac.omb1, g));
    const float nv = __builtin_fmaf(ac.beta2, vo, __fmul_rn(ac.omb2, __fmul_rn(g, g)));
    const float mhat = nm1 / ac.bc1;
    const float vhat = nv / ac.bc2;
    const float den = __fadd_rn(sqrtf(vhat), ac.eps);
    const float q = mhat / den;
    mn = __builtin_fmaf(-lr, q, mo);
    m1n = nm1;
    vn = nv;
    if (d >= D) { mn = 0.f; m1n = 0.f; vn = 0.f; gg = 0.f; }
}

// The same on the four dims of a Philox block.
__device__ __forceinline__ void adam_block(const double a64[4], double inv_ns, const AdamConsts& ac, float lr, int64_t d0,
                                           int64_t D, const float mo[4], const float m1o[4], const float vo[4],
                                           float mn[4], float m1n[4], float vn[4], float gg[4])
{
#pragma unroll
    for (int k = 0; k < 4; ++k) adam_dim(a64[k], inv_ns, ac, lr, d0 + k, D, mo[k], m1o[k], vo[k], mn[k], m1n[k], vn[k], gg[k]);
}

// Everything the gradient kernels need besides the geometry.
struct TellArgs {
    const float* wfold;    // [R][P] a_p = y_p - y_{p+P}
    const float* bfold;    // [R][P] second weight (PGPE, SNES) or null
    const int32_t* best_j; // [R]
    float* m;
    float* m1;
    float* v;
    float* grad;           // [R][Dp] or null
    float* best_x;
    float* sig;            // [R][Dp] per-dimension sigma (PGPE, SNES) or null
    float* gbuf;           // [R][Dp] ClipUp: the gradient, stepped by the ClipUp kernels
    double* gpart;         // [R][groups] ClipUp: |g|^2 of each group of 64 blocks
    double* part;          // split partial sums [R][nsplit][nb][4 or 8]
    const float* hp;       // [2][R] sigma, lr
    // Sep-CMA-ES: elite members by rank, recombination weights, the weighted
    // noise sums kept for the second pass
    const int32_t* elite;  // [R][N]
    const float* cw;       // [mu]
    double* zw;            // [R][Dp] sum_i w_i z_i
    double* qd;            // [R][Dp] sum_i w_i z_i^2
    CmaConsts cma;
    uint64_t seed;
    uint32_t t;
    int64_t D, nb;
    int32_t P, R, ps, nsplit;
    int32_t nitems;        // items the slices split: P pairs, or mu elites
    int32_t strategy, optimizer;
    float sigma_lr, max_change, sigma_decay, sigma_final;
    AdamConsts ac;
    // MLP: workgroups x < tshift of the launch (y = z = 0) run the next
    // generation's teacher rows; the gradient's workgroups follow them
    TeacherJob teacher;
    int32_t tshift;
};

__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Update of one Philox block from its noise sums a64 (and b64):
//   OpenAI-ES  g = a / (N sigma), Adam (or ClipUp, stepped later);
//   PGPE       g = sigma_d a / N, Adam or ClipUp on the mean;
//              s = sigma_d b / P, sigma += clip(-sigma_lr s, +-max_change sigma), schedule;
//   SNES       m += fl32(lr sigma_d) a, sigma *= exp(fl32(sigma_lr/2) b), schedule.
// Also the best member's parameters when the generation improved on the
// best so far (old mean and sigma), and the gradient when asked for.
// Returns this lane's share of |g|^2 (ClipUp), else 0.
__device__ __forceinline__ double tell_finish(const TellArgs& a, const double a64[4], const double b64[4], int64_t b,
                                              int32_t r, uint32_t k0, uint32_t k1)
{
    const int64_t off = (int64_t)r * 4 * a.nb + 4 * b;
    const float sigma = a.hp[r], lr = a.hp[a.R + r];
    const float4 m4 = *reinterpret_cast<const float4*>(a.m + off);
    const float mo[4] = {m4.x, m4.y, m4.z, m4.w};
    float so[4] = {sigma, sigma, sigma, sigma};
    if (a.sig) {
        const float4 s4 = *reinterpret_cast<const float4*>(a.sig + off);
        so[0] = s4.x; so[1] = s4.y; so[2] = s4.z; so[3] = s4.w;
    }
    const int32_t N = 2 * a.P;
    float mn[4] = {mo[0], mo[1], mo[2], mo[3]}, gg[4] = {0.f, 0.f, 0.f, 0.f}, sn[4] = {so[0], so[1], so[2], so[3]};
    double g2 = 0.0;
    if (a.strategy == ES_STRAT_SEP_CMA) {
        // first pass: mean, p_sigma (in m1), the sums for the second pass and
        // this lane's share of |p_sigma|^2; the best member (row = member, + sign)
        const float4 p4 = *reinterpret_cast<const float4*>(a.m1 + off);
        const float po[4] = {p4.x, p4.y, p4.z, p4.w};
        float pn[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const bool live = 4 * b + k < a.D;
            mn[k] = live ? (float)((double)mo[k] + (double)so[k] * a64[k]) : 0.f;
            pn[k] = live ? (float)((1.0 - a.cma.c_s) * (double)po[k] + a.cma.a_s * a64[k]) : 0.f;
            g2 += (double)pn[k] * (double)pn[k];
        }
        *reinterpret_cast<double4*>(a.zw + off) = make_double4(a64[0], a64[1], a64[2], a64[3]);
        *reinterpret_cast<double4*>(a.qd + off) =
            make_double4(b64[0] + a.cma.wsum, b64[1] + a.cma.wsum, b64[2] + a.cma.wsum, b64[3] + a.cma.wsum);
        *reinterpret_cast<float4*>(a.m1 + off) = make_float4(pn[0], pn[1], pn[2], pn[3]);
        const int32_t jb = a.best_j[r];
        if (jb >= 0) {
            float e[4];
            box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)b, (uint32_t)jb, a.t, DOM_NOISE), e);
            float bx[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) bx[k] = 4 * b + k < a.D ? fmaf(so[k], e[k], mo[k]) : 0.f;
            *reinterpret_cast<float4*>(a.best_x + off) = make_float4(bx[0], bx[1], bx[2], bx[3]);
        }
        *reinterpret_cast<float4*>(a.m + off) = make_float4(mn[0], mn[1], mn[2], mn[3]);
        if (a.grad)
            *reinterpret_cast<float4*>(a.grad + off) =
                make_float4((float)a64[0], (float)a64[1], (float)a64[2], (float)a64[3]);
        return g2;
    }
    if (a.strategy == ES_STRAT_SNES) {
        const float h = 0.5f * a.sigma_lr;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float A = (float)a64[k], B = (float)b64[k];
            if (4 * b + k < a.D) {
                mn[k] = fmaf(__fmul_rn(lr, so[k]), A, mo[k]);
                sn[k] = schedule_step(__fmul_rn(so[k], expf(__fmul_rn(h, B))), a.sigma_decay, a.sigma_final);
                gg[k] = __fmul_rn(so[k], A);
            } else {
                mn[k] = 0.f; sn[k] = 0.f;
            }
        }
    } else {
        const double inv_ns = 1.0 / ((double)N * (double)sigma);  // 1 / (N sigma)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            gg[k] = a.strategy == ES_STRAT_PGPE ? (float)((double)so[k] * a64[k] / (double)N) : (float)(a64[k] * inv_ns);
            if (4 * b + k >= a.D) gg[k] = 0.f;
        }
        if (a.optimizer == ES_OPT_CLIPUP) {
            *reinterpret_cast<float4*>(a.gbuf + off) = make_float4(gg[0], gg[1], gg[2], gg[3]);
#pragma unroll
            for (int k = 0; k < 4; ++k) g2 += (double)gg[k] * (double)gg[k];
        } else {
            const float4 m14 = *reinterpret_cast<const float4*>(a.m1 + off);
            const float4 v4 = *reinterpret_cast<const float4*>(a.v + off);
            const float m1o[4] = {m14.x, m14.y, m14.z, m14.w};
            const float vo[4] = {v4.x, v4.y, v4.z, v4.w};
            float m1n[4], vn[4], gd[4];
            const double a1[4] = {(double)gg[0], (double)gg[1], (double)gg[2], (double)gg[3]};
            adam_block(a1, 1.0, a.ac, lr, 4 * b, a.D, mo, m1o, vo, mn, m1n, vn, gd);
            *reinterpret_cast<float4*>(a.m1 + off) = make_float4(m1n[0], m1n[1], m1n[2], m1n[3]);
            *reinterpret_cast<float4*>(a.v + off) = make_float4(vn[0], vn[1], vn[2], vn[3]);
        }
        if (a.strategy == ES_STRAT_PGPE) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float sg = (float)((double)so[k] * b64[k] / (double)a.P);
                float dlt = -__fmul_rn(a.sigma_lr, sg);
                const float lim = __fmul_rn(a.max_change, so[k]);
                dlt = dlt > lim ? lim : dlt;
                dlt = dlt < -lim ? -lim : dlt;
                sn[k] = 4 * b + k < a.D ? schedule_step(__fadd_rn(so[k], dlt), a.sigma_decay, a.sigma_final) : 0.f;
            }
        }
    }
    const int32_t jb = a.best_j[r];
    if (jb >= 0) {
        const int32_t pbst = jb < a.P ? jb : jb - a.P;
        float e[4];
        box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)b, (uint32_t)pbst, a.t, DOM_NOISE), e);
        float bx[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) bx[k] = 4 * b + k < a.D ? fmaf(jb < a.P ? so[k] : -so[k], e[k], mo[k]) : 0.f;
        *reinterpret_cast<float4*>(a.best_x + off) = make_float4(bx[0], bx[1], bx[2], bx[3]);
    }
    if (a.strategy == ES_STRAT_SNES || a.optimizer != ES_OPT_CLIPUP)
        *reinterpret_cast<float4*>(a.m + off) = make_float4(mn[0], mn[1], mn[2], mn[3]);
    if (a.sig) *reinterpret_cast<float4*>(a.sig + off) = make_float4(sn[0], sn[1], sn[2], sn[3]);
    if (a.grad) *reinterpret_cast<float4*>(a.grad + off) = make_float4(gg[0], gg[1], gg[2], gg[3]);
    return g2;
}

// Gradient + update.  Workgroup = TELL_LANES Philox blocks x ps pair slices
// (ps <= TELL_MAX_PS, chosen per geometry) of one run.  Each lane walks its
// slice of pairs with the folded weights (uniform across the wave),
// regenerating the pair's normals, so the sums over pairs need no
// cross-lane reduction; the slices meet in LDS in a fixed order.  With
// nsplit > 1, grid.z = nsplit workgroups share a block group (workgroup z
// takes global slices z*ps .. z*ps+ps-1 of ps*nsplit equal slices of the
// pairs) and store their sums to part; k_tell_fold adds them in split order
// and applies the update.  TWO: the second sum b (PGPE, SNES, Sep-CMA-ES);
// ROWS: items are the elites (Sep-CMA-ES) rather than the pairs.
template <bool TWO, bool ROWS = false, int SUB = 1, bool TEACH = false>
__global__ __launch_bounds__(TELL_LANES * TELL_MAX_PS) void k_tell(TellArgs a)
{
    if constexpr (TEACH) {
        // the next generation's teacher rows, dispatched ahead of the gradient
        // workgroups so that they run in the shadow of the gradient's VALU work
        // (their own instantiation: the teacher's registers would otherwise
        // lower every gradient kernel's occupancy)
        if ((int32_t)blockIdx.x < a.tshift) {
            if (blockIdx.y == 0 && blockIdx.z == 0) teacher_row(a.teacher, blockIdx.x);
            return;
        }
    }
    const int32_t tsh = TEACH ? a.tshift : 0;
    const int32_t gx = (int32_t)blockIdx.x - tsh, gn = (int32_t)gridDim.x - tsh;
    // slices 1 .. ps-1 of every lane, sized by the launch: [ps-1][TELL_LANES][W]
    extern __shared__ double red[];
    constexpr int W = TWO ? 8 : 4;
    const int32_t r = blockIdx.y, z = blockIdx.z;
    const int32_t tx = threadIdx.x % TELL_LANES;
    // one wave per pair slice: make the slice index (and the pair loop) uniform
    const int32_t s = __builtin_amdgcn_readfirstlane(threadIdx.x / TELL_LANES);
    // SUB > 1: SUB neighbouring lanes share a block, each with a sub-slice of
    // the wave's pairs (a run with few block groups spread over more CUs);
    // SUB = 1 keeps the pair range uniform, so the weights come through the
    // scalar cache
    constexpr int32_t sub = SUB;
    const int32_t si = tx % sub;
    const int64_t b = (int64_t)gx * (TELL_LANES / sub) + tx / sub;
    const uint32_t bb = (uint32_t)(b < a.nb ? b : a.nb - 1);
    const uint64_t key = a.seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    const int64_t S = (int64_t)a.ps * a.nsplit * sub, gs = ((int64_t)z * a.ps + s) * sub + si;
    const int32_t pb = (int32_t)(((int64_t)a.nitems * gs) / S);
    const int32_t pe = (int32_t)(((int64_t)a.nitems * (gs + 1)) / S);

    double a64[4] = {0.0, 0.0, 0.0, 0.0}, b64[4] = {0.0, 0.0, 0.0, 0.0};
    if constexpr (ROWS)
        tell_slice2<LANES_BLOCK, true>(a.cw, a.cw, k0, k1, bb, a.t, pb, pe, a64, b64, a.elite + (int64_t)r * 2 * a.P);
    else if constexpr (TWO)
        tell_slice2<LANES_BLOCK>(a.wfold + (int64_t)r * a.P, a.bfold + (int64_t)r * a.P, k0, k1, bb, a.t, pb, pe,
                                 a64, b64);
    else
        tell_slice<LANES_BLOCK>(a.wfold + (int64_t)r * a.P, k0, k1, bb, a.t, pb, pe, a64);
    // sub-slices of one block: ((l0 + l1) + (l2 + l3)) in every lane of the group
#pragma unroll
    for (int off = 1; off < sub; off <<= 1) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a64[k] += __shfl_xor(a64[k], off);
            if constexpr (TWO) b64[k] += __shfl_xor(b64[k], off);
        }
    }
    if (s > 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            red[((s - 1) * TELL_LANES + tx) * W + k] = a64[k];
            if constexpr (TWO) red[((s - 1) * TELL_LANES + tx) * W + 4 + k] = b64[k];
        }
    }
    __syncthreads();
    if (s != 0) return;
    for (int q = 0; q < a.ps - 1; ++q)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            a64[k] += red[(q * TELL_LANES + tx) * W + k];
            if constexpr (TWO) b64[k] += red[(q * TELL_LANES + tx) * W + 4 + k];
        }
    if (a.nsplit > 1) {
        if (b < a.nb) {
            double* o = a.part + (((int64_t)r * a.nsplit + z) * a.nb + b) * (TWO ? 8 : 4);
            *reinterpret_cast<double4*>(o) = make_double4(a64[0], a64[1], a64[2], a64[3]);
            if constexpr (TWO) *reinterpret_cast<double4*>(o + 4) = make_double4(b64[0], b64[1], b64[2], b64[3]);
        }
        return;
    }
    if (SUB > 1 && si != 0) return;  // SUB > 1 only where no per-wave norm partials are kept
    const double g2 = b < a.nb ? tell_finish(a, a64, b64, b, r, k0, k1) : 0.0;
    if (a.gpart) {
        const double tot = wave_sum(g2);
        if (tx == 0) a.gpart[(int64_t)r * gn + gx] = tot;
    }
}

// Second half of a split gradient: the nsplit workgroup sums of each Philox
// block added in split order, then the update.  One lane per block; each
// wave covers one group of 64 blocks.
template <bool TWO>
__global__ __launch_bounds__(256) void k_tell_fold(TellArgs a)
{
    const int32_t r = blockIdx.y;
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t key = a.seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    double g2 = 0.0;
    if (b < a.nb) {
        constexpr int W = TWO ? 8 : 4;
        const double* p0 = a.part + ((int64_t)r * a.nsplit * a.nb + b) * W;
        double a64[4], b64[4] = {0.0, 0.0, 0.0, 0.0};
        const double4 q0 = *reinterpret_cast<const double4*>(p0);
        a64[0] = q0.x; a64[1] = q0.y; a64[2] = q0.z; a64[3] = q0.w;
        if constexpr (TWO) {
            const double4 r0 = *reinterpret_cast<const double4*>(p0 + 4);
            b64[0] = r0.x; b64[1] = r0.y; b64[2] = r0.z; b64[3] = r0.w;
        }
        for (int32_t q = 1; q < a.nsplit; ++q) {
            const double* pq = p0 + (int64_t)q * a.nb * W;
            const double4 qq = *reinterpret_cast<const double4*>(pq);
            a64[0] += qq.x; a64[1] += qq.y; a64[2] += qq.z; a64[3] += qq.w;
            if constexpr (TWO) {
                const double4 rr = *reinterpret_cast<const double4*>(pq + 4);
                b64[0] += rr.x; b64[1] += rr.y; b64[2] += rr.z; b64[3] += rr.w;
            }
        }
        g2 = tell_finish(a, a64, b64, b, r, k0, k1);
    }
    if (a.gpart) {
        const double tot = wave_sum(g2);
        const int64_t groups = (a.nb + TELL_LANES - 1) / TELL_LANES;
        if ((threadIdx.x & 63) == 0 && (b >> 6) < groups) a.gpart[(int64_t)r * groups + (b >> 6)] = tot;
    }
}

// ClipUp (Toklu et al. 2020) after the gradient kernel, two passes over the
// run's dims.  Each workgroup sums the per-group partials of |g|^2 (then
// |v'|^2) in the same fixed order, so every workgroup sees the same norm.
__device__ __forceinline__ double group_total(const double* __restrict__ part, int64_t n, double* red)
{
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) acc += part[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const double tot = red[0];
    __syncthreads();
    return tot;
}

// v' = fmaf(lr, g * fl32(1/|g|), momentum * v); stores v' and |v'|^2 per group.
__global__ __launch_bounds__(256) void k_clipup_velocity(const float* __restrict__ gbuf, float* __restrict__ vel,
                                                         const double* __restrict__ gpart, double* __restrict__ vpart,
                                                         const float* __restrict__ hp, int32_t R, int64_t nb,
                                                         int64_t groups, float momentum)
{
    __shared__ double red[256];
    const int32_t r = blockIdx.y;
    const double gg = group_total(gpart + (int64_t)r * groups, groups, red);
    const float inv = gg > 0.0 ? (float)(1.0 / sqrt(gg)) : 0.0f;
    const float lr = hp[R + r];
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    double v2 = 0.0;
    if (b < nb) {
        const int64_t off = (int64_t)r * 4 * nb + 4 * b;
        const float4 g4 = *reinterpret_cast<const float4*>(gbuf + off);
        const float4 v4 = *reinterpret_cast<const float4*>(vel + off);
        const float g[4] = {g4.x, g4.y, g4.z, g4.w}, vo[4] = {v4.x, v4.y, v4.z, v4.w};
        float vn[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            vn[k] = fmaf(lr, __fmul_rn(g[k], inv), __fmul_rn(momentum, vo[k]));
            v2 += (double)vn[k] * (double)vn[k];
        }
        *reinterpret_cast<float4*>(vel + off) = make_float4(vn[0], vn[1], vn[2], vn[3]);
    }
    const double tot = wave_sum(v2);
    if ((threadIdx.x & 63) == 0 && (b >> 6) < groups) vpart[(int64_t)r * groups + (b >> 6)] = tot;
}

// Sep-CMA-ES second pass: |p_sigma| from the groups' partials (fixed order),
// then per dim p_c (in v), C, and the next generation's sampling scale
// s = fl32(sigma' sqrtf(C)); the first workgroup stores the run's sigma'.
__global__ __launch_bounds__(256) void k_sepcma_finish(float* __restrict__ v, float* __restrict__ C,
                                                       float* __restrict__ svec, const double* __restrict__ zw,
                                                       const double* __restrict__ qd, const double* __restrict__ gpart,
                                                       const float* __restrict__ hp, float* __restrict__ hp_next,
                                                       int64_t D, int64_t nb, int64_t groups, uint32_t t, CmaConsts k)
{
    __shared__ double red[256];
    const int32_t r = blockIdx.y;
    const double nps = sqrt(group_total(gpart + (int64_t)r * groups, groups, red));
    const double hth = nps / sqrt(1.0 - pow(1.0 - k.c_s, 2.0 * ((double)t + 1.0)));
    const double h = hth < (1.4 + 2.0 / ((double)D + 1.0)) * k.chi ? 1.0 : 0.0;
    const float sig_new = (float)((double)hp[r] * exp((k.c_s / k.d_s) * (nps / k.chi - 1.0)));
    if (blockIdx.x == 0 && threadIdx.x == 0) hp_next[r] = sig_new;
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nb) return;
    const int64_t off = (int64_t)r * 4 * nb + 4 * b;
    const float4 pc4 = *reinterpret_cast<const float4*>(v + off);
    const float4 c4 = *reinterpret_cast<const float4*>(C + off);
    const double4 z4 = *reinterpret_cast<const double4*>(zw + off);
    const double4 q4 = *reinterpret_cast<const double4*>(qd + off);
    const float pco[4] = {pc4.x, pc4.y, pc4.z, pc4.w}, co[4] = {c4.x, c4.y, c4.z, c4.w};
    const double zv[4] = {z4.x, z4.y, z4.z, z4.w}, qv[4] = {q4.x, q4.y, q4.z, q4.w};
    float pcn[4], cn[4], sn[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (4 * b + j >= D) { pcn[j] = 0.f; cn[j] = 0.f; sn[j] = 0.f; continue; }
        const double Cd = (double)co[j];
        pcn[j] = (float)((1.0 - k.c_c) * (double)pco[j] + h * k.a_c * sqrt(Cd) * zv[j]);
        const double pcd = (double)pcn[j];
        cn[j] = (float)((1.0 - k.c1 - k.cmu) * Cd + k.c1 * (pcd * pcd + (1.0 - h) * k.c_c * (2.0 - k.c_c) * Cd) +
                        k.cmu * Cd * qv[j]);
        sn[j] = __fmul_rn(sig_new, sqrtf(cn[j]));
    }
    *reinterpret_cast<float4*>(v + off) = make_float4(pcn[0], pcn[1], pcn[2], pcn[3]);
    *reinterpret_cast<float4*>(C + off) = make_float4(cn[0], cn[1], cn[2], cn[3]);
    *reinterpret_cast<float4*>(svec + off) = make_float4(sn[0], sn[1], sn[2], sn[3]);
}

// s = fl32(sigma sqrtf(C)) for every run (after a change of sigma or C).
__global__ void k_cma_scale(float* __restrict__ svec, const float* __restrict__ C, const float* __restrict__ hp,
                            int64_t D, int64_t Dp, int64_t total)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / Dp;
        svec[i] = (i % Dp) < D ? __fmul_rn(hp[r], sqrtf(C[i])) : 0.0f;
    }
}

// v = v' * fl32(max_speed / |v'|) when |v'| > max_speed; m -= v.
__global__ __launch_bounds__(256) void k_clipup_apply(float* __restrict__ vel, float* __restrict__ m,
                                                      const double* __restrict__ vpart, int64_t nb, int64_t groups,
                                                      float max_speed)
{
    __shared__ double red[256];
    const int32_t r = blockIdx.y;
    const double nv = sqrt(group_total(vpart + (int64_t)r * groups, groups, red));
    const bool clip = nv > (double)max_speed;
    const float sc = clip ? (float)((double)max_speed / nv) : 1.0f;
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nb) return;
    const int64_t off = (int64_t)r * 4 * nb + 4 * b;
    float4 v4 = *reinterpret_cast<const float4*>(vel + off);
    float4 m4 = *reinterpret_cast<const float4*>(m + off);
    if (clip) {
        v4.x = __fmul_rn(v4.x, sc); v4.y = __fmul_rn(v4.y, sc); v4.z = __fmul_rn(v4.z, sc); v4.w = __fmul_rn(v4.w, sc);
        *reinterpret_cast<float4*>(vel + off) = v4;
    }
    m4.x = __fsub_rn(m4.x, v4.x); m4.y = __fsub_rn(m4.y, v4.y); m4.z = __fsub_rn(m4.z, v4.z); m4.w = __fsub_rn(m4.w, v4.w);
    *reinterpret_cast<float4*>(m + off) = m4;
}

// ---------------------------------------------------------------------------
// T whole generations in one launch (the scanned loop of Listing 2) for
// small strategies: one workgroup per run, the mean and Adam moments in LDS.
// Each phase repeats the per-call kernels' arithmetic in the same order
// (same chunking of the evaluation, same reduction order, same pair slices
// of the gradient), so es_run gives the same bits on either path.  STASH:
// the evaluate keeps every normal it makes in LDS and the gradient reads them
// back instead of regenerating them (where they fit).
struct FusedArgs {
    float* m;
    float* m1;
    float* v;
    float* grad;             // [R][Dp] or null
    float* best_x;
    uint32_t* best_okey;
    float* best_f;
    const float* pdata;
    const float* table;
    float* log;              // [T][R] or null
    uint64_t seed;
    uint32_t t0;
    int32_t T;
    int64_t D, nb;
    int32_t N, P, R;
    int64_t bc, nchunks;
    int32_t ps;
    float ra;
    double add;
    int32_t maximize, raw;
    float* hp;               // [2][R] sigma, lr: read at the start, the schedule's values written at the end
    float sigma_decay, sigma_final, lr_decay, lr_final;
    AdamConsts ac;           // the generation-independent Adam constants
    float bcorr[FUSED_MAX_T][2];  // bias corrections bc1, bc2 of generations t0 .. t0+T-1
};
static_assert(std::is_standard_layout<FusedArgs>::value, "offsetof(FusedArgs, bcorr) is used on the device");

// The value of the lane whose index differs in bit 0, 1 or 2 (bit 0 and 1:
// DPP quad permutations [1,0,3,2] and [2,3,0,1]; bit 2: ds_swizzle in
// bitmask mode, and_mask 31, xor_mask 4).  Every lane of the wave must be
// active.
__device__ __forceinline__ int32_t xor_lane1(int32_t x) { return __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false); }
__device__ __forceinline__ int32_t xor_lane2(int32_t x) { return __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false); }
__device__ __forceinline__ int32_t xor_lane4(int32_t x) { return __builtin_amdgcn_ds_swizzle(x, (4 << 10) | 0x1F); }

// Wave priority 0, 1 or 2 (s_setprio takes an immediate).
__device__ __forceinline__ void set_long_prio(uint32_t lp)
{
    if (lp == 0) __builtin_amdgcn_s_setprio(0);
    else if (lp == 1) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(2);
}

// Best-so-far of a run inside a multi-generation loop, kept on chip: the
// order key, fitness and member of the best so far, and the generation,
// member and sigma of the loop's last improvement (best_x gets its noise once,
// after the loop).
struct LoopBest {
    int32_t j;     // member improving on the best this generation, else -1
    uint32_t k;
    float fv;
    uint32_t t;
    int32_t jj;    // member of the last improvement (-1: none)
    float sg;
};

// One member's fitness from its chunk partials p[c * stride], c < nchunks,
// in the reduce kernel's order (chunk slices q < RED_SLICES, each summed in
// chunk order, added in slice order after `add`).
__device__ __forceinline__ double fitness_sum(const float* p, int32_t stride, int64_t nchunks, double add)
{
    const int nq = nchunks < RED_SLICES ? (int)nchunks : RED_SLICES;  // slices beyond add 0
    double tot = add;
    if (nchunks <= RED_SLICES) {
        // one chunk per slice: four loads in flight ahead of the sum
        for (int q0 = 0; q0 < nq; q0 += 4) {
            float pv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) pv[u] = p[(q0 + u < nq ? q0 + u : nq - 1) * stride];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (q0 + u < nq) {
                    double acc = 0.0;
                    acc += (double)pv[u];
                    tot += acc;
                }
        }
    } else {
        for (int q = 0; q < nq; ++q) {
            double acc = 0.0;
            for (int64_t c = q; c < nchunks; c += RED_SLICES) acc += (double)p[c * stride];
            tot += acc;
        }
    }
    return tot;
}

// Centered ranks of one generation from the run's order keys, the folded
// weights wf[p] = y_p - y_{p+P}, the best-so-far and (logp not null) the
// generation's best fitness.  Eight lanes per pair: lanes 4*mem + q count
// the keys of slice q below member p + mem*P (ties by index); the quad adds
// its counts and the two members' weights meet across the group.  WG lanes,
// all of them active.
template <int WG>
__device__ __forceinline__ void rank_pairs(const uint32_t* keys, const float* fit, const float* tab, float* wf,
                                           int32_t N, int32_t P, int32_t raw, int32_t maximize, LoopBest& bst,
                                           float* logp)
{
    const int32_t cs = ((N + 15) / 16) * 4;  // keys per slice, a multiple of 4
    const int32_t lg = threadIdx.x & 7, mem = lg >> 2, q = lg & 3;
    for (int32_t pb = 0; pb < P; pb += WG / 8) {
        const int32_t p = pb + (int32_t)(threadIdx.x >> 3);
        int32_t rk = 0, j = 0;
        uint32_t K = 0;
        if (p < P) {
            j = p + mem * P;
            K = keys[j];
            // member k sorts before j when (key_k, k) < (K, j): one 64-bit
            // compare per key
            const uint64_t cj = ((uint64_t)K << 32) | (uint32_t)j;
            const int32_t s0 = q * cs, s1 = s0 + cs < N ? s0 + cs : N;
            int32_t k = s0;
            for (; k + 8 <= s1; k += 8) {
                uint4 q4[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) q4[u] = *reinterpret_cast<const uint4*>(keys + k + 4 * u);
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const uint32_t kk = (uint32_t)(k + 4 * u);
                    rk += ((((uint64_t)q4[u].x) << 32) | kk) < cj;
                    rk += ((((uint64_t)q4[u].y) << 32) | (kk + 1)) < cj;
                    rk += ((((uint64_t)q4[u].z) << 32) | (kk + 2)) < cj;
                    rk += ((((uint64_t)q4[u].w) << 32) | (kk + 3)) < cj;
                }
            }
            for (; k < s1; ++k) rk += ((((uint64_t)keys[k]) << 32) | (uint32_t)k) < cj;
        }
        // every lane of the wave takes part in the exchanges (lane xor 1 and
        // xor 2 within the quad by DPP, xor 4 by swizzle)
        rk += xor_lane1(rk);
        rk += xor_lane2(rk);
        const float yj = p < P ? (raw ? (maximize ? -fit[j] : fit[j]) : tab[rk]) : 0.f;
        const float yo = __int_as_float(xor_lane4(__float_as_int(yj)));
        if (p < P && q == 0) {
            if (mem == 0) wf[p] = yj - yo;
            if (rk == 0) {
                if (logp) *logp = fit[j];
                if (K < bst.k) {
                    bst.k = K;
                    bst.fv = fit[j];
                    bst.j = j;
                } else {
                    bst.j = -1;
                }
            }
        }
    }
}

template <int PROB, bool STASH>
__global__ __launch_bounds__(FUSED_WG) void k_run_fused(FusedArgs a)
{
    extern __shared__ __align__(16) double smem[];
    const int32_t r = blockIdx.x;
    const int64_t Dp = 4 * a.nb;
    // LDS layout: tell slices (fp64) | normals (float4, STASH) | m | m1 | v | partial | fit | y | wf | keys (N
    // rounded up to 4) | table
    double* red = smem;                                  // [ps][nb][4]
    const int32_t es = a.P + 1;                          // normals of one block: one float4 per pair
    float4* eps = reinterpret_cast<float4*>(red + (int64_t)a.ps * a.nb * 4);  // [nb][P + 1]
    float* ms = reinterpret_cast<float*>(eps + (STASH ? a.nb * es : 0));
    float* m1s = ms + Dp;
    float* vs = m1s + Dp;
    float* part = vs + Dp;                               // [nchunks][N]
    float* fit = part + a.nchunks * a.N;                 // [N]
    float* y = fit + a.N;                                // [N]
    float* wf = y + a.N;                                 // [P]
    // keys start on a 16-byte boundary (they are read four at a time)
    uint32_t* keys = reinterpret_cast<uint32_t*>(ms + ((3 * Dp + a.nchunks * a.N + 2 * a.N + a.P + 3) & ~(int64_t)3));
    float* tab = reinterpret_cast<float*>(keys + ((a.N + 3) & ~3));  // [N] shaping table
    __shared__ LoopBest bst;

    const uint64_t key = a.seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    const int64_t goff = (int64_t)r * Dp;
    float sigma = a.hp[r], lr = a.hp[a.R + r];
    for (int64_t i = threadIdx.x; i < Dp; i += FUSED_WG) {
        ms[i] = a.m[goff + i];
        m1s[i] = a.m1[goff + i];
        vs[i] = a.v[goff + i];
    }
    for (int32_t j = threadIdx.x; j < a.N; j += FUSED_WG) tab[j] = a.table[j];
    // pair bounds of the gradient's slices: slice s takes pairs [P s / ps, P (s+1) / ps)
    __shared__ int32_t sl_bound[TELL_MAX_PS + 1];
    if (threadIdx.x <= (uint32_t)a.ps) sl_bound[threadIdx.x] = (int32_t)(((int64_t)a.P * threadIdx.x) / a.ps);
    if (threadIdx.x == 0) {
        bst.k = a.best_okey[r];
        bst.fv = a.best_f[r];
        bst.jj = -1;
    }
    __syncthreads();
    // Every generation a thread walks the same items: evaluate item i is
    // (pair i % P, chunk i / P), gradient item i is (slice i / nb, block
    // i % nb), for i = thread, thread + FUSED_WG, ...  The walks are set up
    // here once (all sizes of a fused run fit in 32 bits: its state is in LDS)
    // and stepped with additions inside the loop.
    const int32_t nb32 = (int32_t)a.nb, P32 = a.P;
    const int32_t ev_items = P32 * (int32_t)a.nchunks, tl_items = a.ps * nb32;
    const int32_t ev_p0 = (int32_t)threadIdx.x % P32, ev_c0 = (int32_t)threadIdx.x / P32;
    const int32_t ev_dp = FUSED_WG % P32, ev_dc = FUSED_WG / P32;
    const int32_t tl_b0 = (int32_t)threadIdx.x % nb32, tl_s0 = (int32_t)threadIdx.x / nb32;
    const int32_t tl_db = FUSED_WG % nb32, tl_ds = FUSED_WG / nb32;

    for (int32_t it = 0; it < a.T; ++it) {
        const uint32_t t = a.t0 + (uint32_t)it;
        // 1 / (N sigma) of this generation, used by the update at its end: the
        // empty asm keeps the fp64 division here, where its latency hides
        // under the evaluate phase, instead of on the update's critical path
        double inv_ns = 1.0 / (2.0 * (double)a.P * (double)sigma);
        asm volatile("" : "+v"(inv_ns));
        // this generation's Adam constants, from the kernel arguments: the
        // bias corrections are read through the kernarg segment pointer (the
        // launch's only explicit argument starts at its offset 0), because a
        // dynamic index into the by-value argument made the compiler hold the
        // array in VGPRs (92 -> 155 per lane, five waves per SIMD -> three)
        AdamConsts ac = a.ac;
        {
            const float* kb = reinterpret_cast<const float*>((const char*)__builtin_amdgcn_kernarg_segment_ptr() +
                                                             offsetof(FusedArgs, bcorr));
            ac.bc1 = kb[2 * it];
            ac.bc2 = kb[2 * it + 1];
        }
        // evaluate: items (pair, chunk).  The short phases (fitness, ranks,
        // update: latency chains on a few lanes) run at the highest wave
        // priority, so that the long phases of the other runs' workgroups on
        // the same CU fill the issue slots around them instead of delaying
        // them.  The long phases (evaluate, gradient) take turns: their
        // priority cycles through 0, 1, 2 over the generations, offset by the
        // workgroup index, so that no run of a CU is always the one served
        // last (the oldest wave otherwise wins every tie, and the youngest run
        // of a CU set the launch's length).
        const uint32_t lp = ((uint32_t)it + (blockIdx.x & 3u)) % 3u;
        set_long_prio(lp);
        {
            int32_t p = ev_p0, c = ev_c0;
            for (int32_t i = (int32_t)threadIdx.x; i < ev_items; i += FUSED_WG) {
                const int64_t b0 = (int64_t)c * a.bc, b1 = b0 + a.bc < a.nb ? b0 + a.bc : a.nb;
                double accp, accm;
                eval_chunk<PROB, LANES_BLOCK_AND_ROW>(ms, a.pdata, k0, k1, (uint32_t)p, t, b0, b1, a.D, sigma, a.ra,
                                                      accp, accm, nullptr, 0, 0,
                                                      STASH ? eps + b0 * es + p : nullptr, es);
                part[c * a.N + p] = (float)accp;
                part[c * a.N + p + P32] = (float)accm;
                p += ev_dp;
                c += ev_dc;
                if (p >= P32) {
                    p -= P32;
                    ++c;
                }
            }
        }
        __syncthreads();
        __builtin_amdgcn_s_setprio(FUSED_PRIO);
        // fitness in the reduce kernel's order, and order keys
        for (int32_t j = threadIdx.x; j < a.N; j += FUSED_WG) {
            const float f = (float)fitness_sum(part + j, a.N, a.nchunks, a.add);
            fit[j] = f;
            keys[j] = order_key(f, a.maximize);
        }
        __syncthreads();
        // centered ranks, the folded weights, best-so-far and the generation's
        // log entry
        rank_pairs<FUSED_WG>(keys, fit, tab, wf, a.N, a.P, a.raw, a.maximize, bst,
                             a.log ? a.log + (int64_t)it * a.R + r : nullptr);
        __syncthreads();
        set_long_prio(lp);
        // tell: items (block, pair slice), slices summed in order, then Adam
        {
            int32_t b = tl_b0, s = tl_s0;
            for (int32_t i = (int32_t)threadIdx.x; i < tl_items; i += FUSED_WG) {
                double a64[4] = {0.0, 0.0, 0.0, 0.0};
                if constexpr (STASH)
                    tell_slice_eps(wf, eps + (int64_t)b * es, sl_bound[s], sl_bound[s + 1], a64);
                else
                    tell_slice<LANES_BLOCK_AND_ROW>(wf, k0, k1, (uint32_t)b, t, sl_bound[s], sl_bound[s + 1], a64);
#pragma unroll
                for (int k = 0; k < 4; ++k) red[(s * nb32 + b) * 4 + k] = a64[k];
                b += tl_db;
                s += tl_ds;
                if (b >= nb32) {
                    b -= nb32;
                    ++s;
                }
            }
        }
        __syncthreads();
        __builtin_amdgcn_s_setprio(FUSED_PRIO);
        const int32_t jb = bst.j;
        for (int64_t i = threadIdx.x; i < 4 * a.nb; i += FUSED_WG) {
            // one dim per lane: the slices in order, then Adam
            // four slices' loads in flight ahead of the ordered sum
            double s64 = red[i];
            for (int q0 = 1; q0 < a.ps; q0 += 4) {
                double rv[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) rv[u] = red[(q0 + u < a.ps ? q0 + u : a.ps - 1) * 4 * nb32 + i];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (q0 + u < a.ps) s64 += rv[u];
            }
            const float mo = ms[i];
            float mn, m1n, vn, gg;
            adam_dim(s64, inv_ns, ac, lr, i, a.D, mo, m1s[i], vs[i], mn, m1n, vn, gg);
            // a new best: keep the mean it was sampled around; its noise is
            // added once, after the loop (same arithmetic as the per-call path)
            if (jb >= 0) a.best_x[goff + i] = mo;
            if (a.grad) a.grad[goff + i] = gg;
            ms[i] = mn;
            m1s[i] = m1n;
            vs[i] = vn;
        }
        if (jb >= 0 && threadIdx.x == 0) {
            bst.t = t;
            bst.jj = jb;
            bst.sg = sigma;
        }
        __syncthreads();
        sigma = schedule_step(sigma, a.sigma_decay, a.sigma_final);
        lr = schedule_step(lr, a.lr_decay, a.lr_final);
    }
    if (bst.jj >= 0) {
        const int32_t pbst = bst.jj < a.P ? bst.jj : bst.jj - a.P;
        const float sg = bst.jj < a.P ? bst.sg : -bst.sg;
        for (int64_t b = threadIdx.x; b < a.nb; b += FUSED_WG) {
            float e[4];
            box_muller4(philox4x32_10<LANES_BLOCK_AND_ROW>(k0, k1, (uint32_t)b, (uint32_t)pbst, bst.t, DOM_NOISE), e);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int64_t d = goff + 4 * b + k;
                a.best_x[d] = 4 * b + k < a.D ? fmaf(sg, e[k], a.best_x[d]) : 0.f;
            }
        }
    }
    if (threadIdx.x == 0) {
        a.hp[r] = sigma;
        a.hp[a.R + r] = lr;
        a.best_okey[r] = bst.k;
        a.best_f[r] = bst.fv;
    }
    for (int64_t i = threadIdx.x; i < Dp; i += FUSED_WG) {
        a.m[goff + i] = ms[i];
        a.m1[goff + i] = m1s[i];
        a.v[goff + i] = vs[i];
    }
}

// ---------------------------------------------------------------------------
// T whole generations of a run on a cooperative grid of G workgroups (grid.x;
// runs on grid.y): the scanned loop for runs too large for one workgroup yet
// too small to fill the chip per call, where the per-call launches would
// cost more than the work.  The work is split by dimension: workgroup w owns
// the evaluate chunks c = w + G i, which are whole chunk slices of the reduce
// kernel (slice q holds the chunks q, q + RED_SLICES, ...; G divides
// RED_SLICES, or every slice is one chunk), and for those chunks' Philox
// blocks it evaluates every pair, forms the gradient and the update, its
// mean, m1 and v staying in LDS.  The evaluate keeps the normals of the own
// blocks in LDS and the gradient reads them back instead of regenerating
// them (they never reach memory).
//
// Workgroups exchange values only as 64-bit words that carry a tag (the
// launch's sequence number and the generation) beside 32 bits of value: a
// reader waits until a word carries the tag it expects, and since each word
// is one location, no fence or barrier is needed.  Per generation: the
// members' fp64 slice sums (two words each, high and low half), from which
// workgroup w forms the fitness of members [N w / G, N (w+1) / G) in the
// reduce kernel's order; all fitnesses; the shaped weights and the rank-0
// member (each workgroup ranks its members against all N); and Rosenbrock's
// one dim before each chunk, owned by workgroup w - 1.  A word is written
// again only after every reader of its last value has used it, because each
// generation's words depend on every workgroup's reads of the one before.
// Chunking, reduction order and the gradient's sub-slices, slices and splits
// are those of the handle's per-call plans, so es_run gives the same bits on
// either path.
struct GridArgs {
    float* m;
    float* m1;
    float* v;
    float* grad;             // [R][Dp] or null
    float* best_x;
    uint32_t* best_okey;
    float* best_f;
    const float* pdata;
    const float* table;
    float* log;              // [T][R] or null
    uint64_t* sx;            // [R][RED_SLICES][N][2] tag | high, tag | low half of member j's slice sum q
    uint64_t* fx;            // [R][N] tag | fitness of member j
    uint64_t* yx;            // [R][N] tag | shaped weight of member j
    uint64_t* bestx;         // [R] tag | the rank-0 member
    uint64_t* halo;          // [R][nchunks] tag | the last dim of chunk c after the update
    uint32_t* err;           // set nonzero when a wait gives up
    uint32_t spin;           // SPIN_ARG: polls before a wait gives up; 0: at once, without polling
    uint32_t tag0;           // this launch's sequence number << 8; generation it's tag is tag0 | it
    int32_t xs;              // x stride between a run's workgroups: run r's are x = r mod xs, r mod xs + xs, ...
    uint64_t seed;
    uint32_t t0;
    int32_t T;
    int64_t D, nb;
    int32_t N, P, R;
    int64_t bc, nchunks;
    int32_t ps, nsplit, sub;  // the per-call gradient plan
    int32_t ncw;              // most chunks of one workgroup
    float ra;
    double add;
    int32_t maximize, raw;
    float* hp;               // [2][R] sigma, lr: read at the start, the schedule's values written at the end
    float sigma_decay, sigma_final, lr_decay, lr_final;
    AdamConsts ac;
    float bcorr[FUSED_MAX_T][2];
};
static_assert(std::is_standard_layout<GridArgs>::value, "offsetof(GridArgs, bcorr) is used on the device");

// Wait until the tagged word at src carries tag: false (with *err set) once
// the wait gives up, after GRID_SPIN_LIMIT polls (SPIN_ARG: `spin` polls,
// 0 giving up at once, so that a test can take the failure path) or when
// another workgroup gave up; the cooperative launch keeps all workgroups
// resident, so with the default limit only a wrong kernel can make it give
// up.  A workgroup whose wait gave up leaves the kernel at its next check,
// and so do the others once their waits see the flag.  (The limit is a
// template choice: as a kernel argument in the default instantiation it cost
// the loop about 8% per generation.)  The polls follow each other without a
// sleep: each is a load's round trip, and a sleep between them delayed the
// exchanges by about 1.5% of a generation.
template <bool SPIN_ARG>
__device__ __forceinline__ bool wait_word(const uint64_t* src, uint32_t tag, uint32_t* err, uint32_t spin,
                                          uint64_t& word)
{
    if constexpr (SPIN_ARG) {
        if (spin == 0) {
            __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
    }
    const uint32_t limit = SPIN_ARG ? spin - 1 : GRID_SPIN_LIMIT;
    for (uint32_t spins = 0;; ++spins) {
        word = __hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)(word >> 32) == tag) return true;
        if (spins >= limit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
            __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
    }
}

// Centered ranks, shared out: this workgroup ranks the members [N w / G,
// N (w+1) / G) against all N composites comp[k] = key_k << 32 | k (member k
// sorts before j exactly when comp[k] < comp[j]; one wave per member, a wave
// sum of the lanes' counts) and publishes their shaped weights as words
// tag << 32 | y_j, and the rank-0 member as tag << 32 | j in its own word.
// Every workgroup then reads all N weights (and the best) back: each word is
// one location, so no fence is needed.  Then the folded weights wf[p] = y_p
// - y_{p+P}, the best-so-far and (logp not null) the generation's best
// fitness.  false if a wait gave up.
template <bool SPIN_ARG>
__device__ __forceinline__ bool rank_exchange(const uint64_t* comp, const uint32_t* keys, const float* fit,
                                              const float* tab, float* y, float* wf, int32_t N, int32_t P, int32_t raw,
                                              int32_t maximize, uint32_t tag, uint64_t* yx, uint64_t* bestx, int32_t w,
                                              int32_t G, uint32_t* err, uint32_t spin, LoopBest& bst, float* logp, int32_t* ok)
{
    const int32_t wave = __builtin_amdgcn_readfirstlane((int32_t)(threadIdx.x / 64)), lane = threadIdx.x % 64;
    const int32_t j0 = (int32_t)(((int64_t)N * w) / G), j1 = (int32_t)(((int64_t)N * (w + 1)) / G);
    for (int32_t j = j0 + wave; j < j1; j += GRID_WG / 64) {
        const uint64_t cj = comp[j];
        int32_t rk = 0;
        for (int32_t k = lane; k < N; k += 64) rk += comp[k] < cj;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) rk += __shfl_xor(rk, off);
        if (lane == 0) {
            const float yj = raw ? (maximize ? -fit[j] : fit[j]) : tab[rk];
            __hip_atomic_store(yx + j, ((uint64_t)tag << 32) | __float_as_uint(yj), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            if (rk == 0)
                __hip_atomic_store(bestx, ((uint64_t)tag << 32) | (uint32_t)j, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (threadIdx.x == 0) *ok = 1;
    __syncthreads();
    for (int32_t j = threadIdx.x; j <= N; j += GRID_WG) {
        uint64_t word;
        if (!wait_word<SPIN_ARG>(j < N ? yx + j : bestx, tag, err, spin, word)) {
            *ok = 0;
            continue;
        }
        if (j < N) {
            y[j] = __uint_as_float((uint32_t)word);
        } else {
            const int32_t jb = (int32_t)(uint32_t)word;
            if (logp) *logp = fit[jb];
            const uint32_t K = keys[jb];
            if (K < bst.k) {
                bst.k = K;
                bst.fv = fit[jb];
                bst.j = jb;
            } else {
                bst.j = -1;
            }
        }
    }
    __syncthreads();
    if (!*ok) return false;
    for (int32_t p = threadIdx.x; p < P; p += GRID_WG) wf[p] = y[p] - y[p + P];
    return true;
}

template <int PROB, bool SPIN_ARG = false>
__global__ __launch_bounds__(GRID_WG) void k_run_grid(GridArgs a)
{
    extern __shared__ __align__(16) double smem[];
    // With xs > 1 the launch holds xs workgroups per working one: those with
    // x = r mod xs, r mod xs + xs, ... work for run r, the rest leave before
    // any access.
    // A row of the grid is a multiple of xs wide, so the workgroups of run r
    // all have linear index = r (mod xs): one XCD when xs is the XCD count.
    const int32_t r = blockIdx.y, xs = a.xs;
    if ((int32_t)blockIdx.x % xs != r % xs) return;
    const int32_t w = (int32_t)blockIdx.x / xs, G = (int32_t)gridDim.x / xs;
    const int32_t S = a.ps * a.nsplit * a.sub;  // the gradient's sub-slices of the pairs
    const int32_t nch = (int32_t)a.nchunks, bc = (int32_t)a.bc, nb = (int32_t)a.nb;
    const int32_t nq = nch < RED_SLICES ? nch : RED_SLICES;
    // own chunks c = w + G i, i < ncw; their blocks have local indices i bc + o
    const int32_t ncw = w < nch ? (nch - w + G - 1) / G : 0;
    const int32_t nlb = ncw * bc;        // local blocks (the last chunk's may pass nb)
    const int32_t CW = 1 + 4 * bc;       // mean of one chunk in LDS: the dim before it, then its dims
    // LDS: sub-slice sums (fp64) [S][ncw bc][4] | rank composites (u64) [N,
    // N padded to even] | own members' slice sums (fp64) [nmw][RED_SLICES] |
    // normals (float4) [ncw bc][P + 1] | mean [ncw][CW]
    // | m1, v [ncw bc][4] | partials [ncw][N] | fit [N] | y [N] | wf [P] |
    // keys [N, from a 16-byte boundary] | table [N] | pair bounds of the
    // sub-slices [S + 1]
    const int64_t st = 4 * (int64_t)a.ncw * bc;  // stride of one sub-slice in red
    const int32_t es = a.P + 1;                  // normals of one block: one float4 per pair (odd stride: no bank conflicts)
    double* red = smem;
    uint64_t* comp = reinterpret_cast<uint64_t*>(red + (int64_t)S * st);
    const int32_t j0 = (int32_t)(((int64_t)a.N * w) / G), nmw = (int32_t)(((int64_t)a.N * (w + 1)) / G) - j0;
    double* msl = reinterpret_cast<double*>(comp + ((a.N + 1) & ~1));
    float4* eps = reinterpret_cast<float4*>(msl + (int64_t)((a.N + G - 1) / G) * RED_SLICES);
    float* ms = reinterpret_cast<float*>(eps + (int64_t)a.ncw * bc * es);
    float* m1s = ms + a.ncw * CW;
    float* vs = m1s + st;
    float* part = vs + st;
    float* fit = part + a.ncw * a.N;
    float* y = fit + a.N;
    float* wf = y + a.N;
    uint32_t* keys = reinterpret_cast<uint32_t*>(ms + ((a.ncw * CW + 2 * st + a.ncw * a.N + 2 * a.N + a.P + 3) & ~(int64_t)3));
    float* tab = reinterpret_cast<float*>(keys + ((a.N + 3) & ~3));
    int32_t* sbd = reinterpret_cast<int32_t*>(tab + a.N);  // sub-slice gs takes the pairs [sbd[gs], sbd[gs + 1])
    __shared__ LoopBest bst;
    __shared__ int32_t ok;

    const uint64_t key = a.seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    const int64_t goff = (int64_t)r * 4 * a.nb;
    float sigma = a.hp[r], lr = a.hp[a.R + r];
    // own dims: local dim i = 4 (i_c bc + o) + k of chunk c = w + G i_c
    for (int32_t i = threadIdx.x; i < 4 * nlb; i += GRID_WG) {
        const int32_t lb = i >> 2, ic = lb / bc, o = lb - ic * bc;
        const int64_t b = (int64_t)(w + G * ic) * bc + o;
        float mv = 0.f, m1v = 0.f, vv = 0.f;  // padding blocks past nb stay zero
        if (b < nb) {
            const int64_t d = goff + 4 * b + (i & 3);
            mv = a.m[d];
            m1v = a.m1[d];
            vv = a.v[d];
        }
        ms[ic * CW + 1 + 4 * o + (i & 3)] = mv;
        m1s[i] = m1v;
        vs[i] = vv;
    }
    for (int32_t j = threadIdx.x; j < a.N; j += GRID_WG) tab[j] = a.table[j];
    for (int32_t g = threadIdx.x; g <= S; g += GRID_WG) sbd[g] = (int32_t)(((int64_t)a.P * g) / S);
    if (threadIdx.x == 0) {
        bst.k = a.best_okey[r];
        bst.fv = a.best_f[r];
        bst.jj = -1;
    }
    __syncthreads();
    uint64_t* halo = a.halo + (int64_t)r * nch;
    uint64_t* sxr = a.sx + (int64_t)r * RED_SLICES * a.N * 2;
    uint64_t* fxr = a.fx + (int64_t)r * a.N;
    const int32_t ev_items = a.P * ncw, tl_items = nlb * S;
    // Every generation a thread walks the same items, set up here and stepped
    // by additions: evaluate item i is (pair i % P, own chunk i / P), gradient
    // item i is (local block i % nlb, sub-slice i / nlb).
    const int32_t ev_p0 = (int32_t)threadIdx.x % a.P, ev_c0 = (int32_t)threadIdx.x / a.P;
    const int32_t ev_dp = GRID_WG % a.P, ev_dc = GRID_WG / a.P;
    const int32_t tl_l0 = nlb > 0 ? (int32_t)threadIdx.x % nlb : 0, tl_g0 = nlb > 0 ? (int32_t)threadIdx.x / nlb : 0;
    const int32_t tl_dl = nlb > 0 ? GRID_WG % nlb : 0, tl_dg = nlb > 0 ? GRID_WG / nlb : 0;

    for (int32_t it = 0; it < a.T; ++it) {
        const uint32_t t = a.t0 + (uint32_t)it, tag = a.tag0 | (uint32_t)it;
        double inv_ns = 1.0 / (2.0 * (double)a.P * (double)sigma);
        asm volatile("" : "+v"(inv_ns));
        AdamConsts ac = a.ac;
        {
            const float* kb = reinterpret_cast<const float*>((const char*)__builtin_amdgcn_kernarg_segment_ptr() +
                                                             offsetof(GridArgs, bcorr));
            ac.bc1 = kb[2 * it];
            ac.bc2 = kb[2 * it + 1];
        }
        if constexpr (PROB == ES_PROB_ROSENBROCK) {
            // the dim before each own chunk (the last of chunk c - 1, updated
            // by workgroup w - 1): from the state at the launch's first
            // generation, then from chunk c - 1's word once it carries the
            // previous generation's tag
            if (threadIdx.x == 0) ok = 1;
            __syncthreads();
            for (int32_t ic = threadIdx.x; ic < ncw; ic += GRID_WG) {
                const int32_t c = w + G * ic;
                float h = 0.f;
                if (c > 0 && it == 0) {
                    h = a.m[goff + 4 * (int64_t)c * bc - 1];
                } else if (c > 0) {
                    uint64_t word;
                    if (wait_word<SPIN_ARG>(halo + c - 1, tag - 1, a.err, a.spin, word)) h = __uint_as_float((uint32_t)word);
                    else ok = 0;
                }
                ms[ic * CW] = h;
            }
            __syncthreads();
            if (!ok) return;
        }
        // evaluate: items (pair, own chunk); the normals of the own blocks
        // also go to LDS for the gradient
        {
            int32_t p = ev_p0, ic = ev_c0;
            for (int32_t i = threadIdx.x; i < ev_items; i += GRID_WG) {
                const int64_t b0 = (int64_t)(w + G * ic) * bc, b1 = b0 + bc < nb ? b0 + bc : nb;
                double accp, accm;
                eval_chunk<PROB, LANES_BLOCK_AND_ROW>(ms + ic * CW + 1, a.pdata, k0, k1, (uint32_t)p, t, b0, b1, a.D,
                                                      sigma, a.ra, accp, accm, nullptr, 0, 4 * b0,
                                                      eps + (int64_t)ic * bc * es + p, es);
                part[ic * a.N + p] = (float)accp;
                part[ic * a.N + p + a.P] = (float)accm;
                p += ev_dp;
                ic += ev_dc;
                if (p >= a.P) {
                    p -= a.P;
                    ++ic;
                }
            }
        }
        __syncthreads();
        // slice sums of the own slices q = w + G u (chunks q, q + RED_SLICES,
        // ... in order), for every member, as two words each
        {
            const int32_t per = nch <= RED_SLICES ? 1 : RED_SLICES / G;  // own chunks between two of one slice
            const int32_t nsl = nch <= RED_SLICES ? ncw : (nq - w + G - 1) / G;
            for (int32_t i = threadIdx.x; i < nsl * a.N; i += GRID_WG) {
                const int32_t u = i / a.N, j = i - u * a.N;
                double acc = 0.0;
                for (int32_t ic = u; ic < ncw; ic += (nch <= RED_SLICES ? ncw : per)) acc += (double)part[ic * a.N + j];
                const uint64_t bits = (uint64_t)__double_as_longlong(acc);
                uint64_t* wq = sxr + ((int64_t)(w + G * u) * a.N + j) * 2;
                __hip_atomic_store(wq, ((uint64_t)tag << 32) | (bits >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(wq + 1, ((uint64_t)tag << 32) | (bits & 0xFFFFFFFFu), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        // the own members' slice sums, one (member, slice) per lane, then their
        // fitness: the slices in order after `add`, published as a word
        if (threadIdx.x == 0) ok = 1;
        __syncthreads();
        for (int32_t i = threadIdx.x; i < nmw * nq; i += GRID_WG) {
            const int32_t jl = i / nq, q = i - jl * nq;
            const uint64_t* wq = sxr + ((int64_t)q * a.N + j0 + jl) * 2;
            uint64_t hi, lo;
            if (wait_word<SPIN_ARG>(wq, tag, a.err, a.spin, hi) && wait_word<SPIN_ARG>(wq + 1, tag, a.err, a.spin, lo))
                msl[jl * RED_SLICES + q] = __longlong_as_double((long long)(((hi & 0xFFFFFFFFu) << 32) | (lo & 0xFFFFFFFFu)));
            else
                ok = 0;
        }
        __syncthreads();
        if (!ok) return;
        for (int32_t jl = threadIdx.x; jl < nmw; jl += GRID_WG) {
            double tot = a.add;
            for (int32_t q = 0; q < nq; ++q) tot += msl[jl * RED_SLICES + q];
            __hip_atomic_store(fxr + j0 + jl, ((uint64_t)tag << 32) | __float_as_uint((float)tot), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        // every member's fitness
        for (int32_t j = threadIdx.x; j < a.N; j += GRID_WG) {
            uint64_t word;
            if (!wait_word<SPIN_ARG>(fxr + j, tag, a.err, a.spin, word)) {
                ok = 0;
                continue;
            }
            const float f = __uint_as_float((uint32_t)word);
            fit[j] = f;
            const uint32_t K = order_key(f, a.maximize);
            keys[j] = K;
            comp[j] = ((uint64_t)K << 32) | (uint32_t)j;
        }
        __syncthreads();
        if (!ok) return;
        if (!rank_exchange<SPIN_ARG>(comp, keys, fit, tab, y, wf, a.N, a.P, a.raw, a.maximize, tag, a.yx + (int64_t)r * a.N,
                           a.bestx + r, w, G, a.err, a.spin, bst, (w == 0 && a.log) ? a.log + (int64_t)it * a.R + r : nullptr,
                           &ok))
            return;
        __syncthreads();
        // gradient of the own blocks: items (block, sub-slice gs), gs
        // numbering the pairs' sub-slices as the per-call kernel does:
        // ((split z) ps + slice s) sub + lane
        {
            int32_t lb = tl_l0, gs = tl_g0;
            for (int32_t i = threadIdx.x; i < tl_items; i += GRID_WG) {
                const int32_t ic = lb / bc;
                const int64_t b = (int64_t)(w + G * ic) * bc + (lb - ic * bc);
                if (b < nb) {
                    double a64[4] = {0.0, 0.0, 0.0, 0.0};
                    tell_slice_eps(wf, eps + (int64_t)lb * es, sbd[gs], sbd[gs + 1], a64);
#pragma unroll
                    for (int k = 0; k < 4; ++k) red[gs * st + 4 * lb + k] = a64[k];
                }
                lb += tl_dl;
                gs += tl_dg;
                if (lb >= nlb) {
                    lb -= nlb;
                    ++gs;
                }
            }
        }
        __syncthreads();
        // update of the own dims: the sub-slices combined in the per-call
        // order (the lanes of a block pairwise, into each slice's first
        // sub-slice, one (slice, dim) per lane; then per dim the slices in
        // order and the splits in order), then Adam
        if (a.sub > 1) {
            const int32_t dims = 4 * nlb;
            for (int32_t i = threadIdx.x; i < a.nsplit * a.ps * dims; i += GRID_WG) {
                const int32_t gi = i / dims, di = i - gi * dims;
                double* rv = red + (int64_t)gi * a.sub * st + di;
                double vsl = rv[0];
                if (a.sub == 2) vsl += rv[st];
                else vsl = (vsl + rv[st]) + (rv[2 * st] + rv[3 * st]);
                rv[0] = vsl;
            }
            __syncthreads();
        }
        const int32_t jb = bst.j;
        const int64_t gst = (int64_t)a.sub * st;  // from one slice's sum to the next
        for (int32_t i = threadIdx.x; i < 4 * nlb; i += GRID_WG) {
            const int32_t lb = i >> 2, ic = lb / bc, o = lb - ic * bc;
            const int64_t b = (int64_t)(w + G * ic) * bc + o;
            if (b >= nb) continue;
            double tot = 0.0;
            for (int32_t z = 0; z < a.nsplit; ++z) {
                // four slices' loads in flight ahead of the ordered sum
                const double* rz = red + (int64_t)z * a.ps * gst + i;
                double az = rz[0];
                for (int32_t s0 = 1; s0 < a.ps; s0 += 4) {
                    double v4[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) v4[u] = rz[(s0 + u < a.ps ? s0 + u : a.ps - 1) * gst];
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        if (s0 + u < a.ps) az += v4[u];
                }
                tot = z == 0 ? az : tot + az;
            }
            const int64_t d = 4 * b + (i & 3);
            float* mp = ms + ic * CW + 1 + 4 * o + (i & 3);
            const float mo = *mp;
            float mn, m1n, vn, gg;
            adam_dim(tot, inv_ns, ac, lr, d, a.D, mo, m1s[i], vs[i], mn, m1n, vn, gg);
            // a new best: keep the mean it was sampled around; its noise is
            // added once, after the loop
            if (jb >= 0) a.best_x[goff + d] = mo;
            *mp = mn;
            m1s[i] = m1n;
            vs[i] = vn;
            a.m[goff + d] = mn;
            if (a.grad) a.grad[goff + d] = gg;
            if constexpr (PROB == ES_PROB_ROSENBROCK) {
                // the last dim of a chunk that another chunk follows: published
                // for the next generation's evaluate of that chunk
                const int32_t c = w + G * ic;
                if (o == bc - 1 && (i & 3) == 3 && c + 1 < nch)
                    __hip_atomic_store(halo + c, ((uint64_t)tag << 32) | __float_as_uint(mn), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (jb >= 0 && threadIdx.x == 0) {
            bst.t = t;
            bst.jj = jb;
            bst.sg = sigma;
        }
        // the next generation's evaluate reads the updated mean (and its
        // ranks overwrite the best-so-far) only after every lane is done here
        __syncthreads();
        sigma = schedule_step(sigma, a.sigma_decay, a.sigma_final);
        lr = schedule_step(lr, a.lr_decay, a.lr_final);
    }
    __syncthreads();
    if (bst.jj >= 0) {
        const int32_t pbst = bst.jj < a.P ? bst.jj : bst.jj - a.P;
        const float sg = bst.jj < a.P ? bst.sg : -bst.sg;
        for (int32_t lb = threadIdx.x; lb < nlb; lb += GRID_WG) {
            const int32_t ic = lb / bc;
            const int64_t b = (int64_t)(w + G * ic) * bc + (lb - ic * bc);
            if (b >= nb) continue;
            float e[4];
            box_muller4(philox4x32_10<LANES_BLOCK_AND_ROW>(k0, k1, (uint32_t)b, (uint32_t)pbst, bst.t, DOM_NOISE), e);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int64_t d = goff + 4 * b + k;
                a.best_x[d] = 4 * b + k < a.D ? fmaf(sg, e[k], a.best_x[d]) : 0.f;
            }
        }
    }
    if (w == 0 && threadIdx.x == 0) {
        a.hp[r] = sigma;
        a.hp[a.R + r] = lr;
        a.best_okey[r] = bst.k;
        a.best_f[r] = bst.fv;
    }
    for (int32_t i = threadIdx.x; i < 4 * nlb; i += GRID_WG) {
        const int32_t lb = i >> 2, ic = lb / bc;
        const int64_t b = (int64_t)(w + G * ic) * bc + (lb - ic * bc);
        if (b >= nb) continue;
        const int64_t d = goff + 4 * b + (i & 3);
        a.m1[d] = m1s[i];
        a.v[d] = vs[i];
    }
}


// ---------------------------------------------------------------------------
__global__ void k_debug_noise(uint32_t* __restrict__ words, float* __restrict__ eps, uint64_t key,
                              uint32_t row, uint32_t t, int64_t D, int64_t nb)
{
    for (int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; b < nb;
         b += (int64_t)gridDim.x * blockDim.x) {
        const uint4 w = philox4x32_10((uint32_t)key, (uint32_t)(key >> 32), (uint32_t)b, row, t, DOM_NOISE);
        if (words) {
            words[4 * b + 0] = w.x;
            words[4 * b + 1] = w.y;
            words[4 * b + 2] = w.z;
            words[4 * b + 3] = w.w;
        }
        if (eps) {
            float e[4];
            box_muller4(w, e);
#pragma unroll
            for (int k = 0; k < 4; ++k)
                if (4 * b + k < D) eps[4 * b + k] = e[k];
        }
    }
}

// rows [R][Dp]: value on the live dims, 0 on the padding
__global__ void k_fill_rows(float* __restrict__ p, float value, int64_t D, int64_t Dp, int64_t total)
{
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = (i % Dp) < D ? value : 0.0f;
}

int grid_for(int64_t n, int threads)
{
    const int64_t g = (n + threads - 1) / threads;
    return (int)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

}  // namespace

// ---------------------------------------------------------------------------
EvalPlan eval_plan(const Geometry& g, int64_t bc_override)
{
    EvalPlan e;
    const int32_t P64 = (g.P + 63) / 64 * 64;
    e.wg = P64 < EVAL_MAX_WG ? P64 : EVAL_MAX_WG;
    e.n_pg = (g.P + e.wg - 1) / e.wg;
    int64_t bc;
    if (bc_override > 0) {
        bc = bc_override;
    } else {
        // About 24576 waves over the launch (three rounds of a full chip at
        // 8 waves per SIMD), with at least EVAL_FOLD blocks per chunk: the
        // shorter workgroups of three rounds leave a shorter tail while the
        // last round drains than those of two (D = 1e6, N = 2048: evaluate
        // 536 -> 524 us; four rounds gain no more and add partials to sum).
        const int64_t waves_per_chunk = (int64_t)e.n_pg * (e.wg / 64) * g.R;
        int64_t nch = (24576 + waves_per_chunk - 1) / waves_per_chunk;
        if (nch < 1) nch = 1;
        bc = (g.nb + nch - 1) / nch;
        if (bc < EVAL_FOLD) bc = EVAL_FOLD;
        // a small run: chunks short enough that the fused loop's workgroup
        // takes every (pair, chunk) item at once
        if ((int64_t)g.P * g.nb <= (int64_t)FUSED_WG * EVAL_FOLD) {
            const int64_t per = FUSED_WG / g.P > 1 ? FUSED_WG / g.P : 1;  // chunks per pair in one pass
            const int64_t bs = (g.nb + per - 1) / per;
            if (bs < bc) bc = bs;
        }
    }
    if (bc > g.nb) bc = g.nb;
    e.bc = bc;
    e.nchunks = (g.nb + bc - 1) / bc;
    return e;
}

int64_t eval_partial_elems(const Geometry& g, const EvalPlan& e) { return e.nchunks * g.R * (int64_t)g.N; }

hipError_t launch_init(const Geometry& g, const es_config& c, float* m, float* m1, float* v,
                       float* best_x, hipStream_t s)
{
    const float range = c.init_hi - c.init_lo;
    k_init<<<grid_for((int64_t)g.R * g.nb, 256), 256, 0, s>>>(m, m1, v, best_x, c.seed, g.D, g.nb, g.R,
                                                               c.init, c.init_lo, range);
    return hipGetLastError();
}

hipError_t launch_cma_scale(const Geometry& g, float* svec, const float* C, const float* hp, hipStream_t s)
{
    const int64_t total = g.Dp * (int64_t)g.R;
    k_cma_scale<<<grid_for(total, 256), 256, 0, s>>>(svec, C, hp, g.D, g.Dp, total);
    return hipGetLastError();
}

hipError_t launch_fill_rows(const Geometry& g, float* p, float value, hipStream_t s)
{
    const int64_t total = g.Dp * (int64_t)g.R;
    k_fill_rows<<<grid_for(total, 256), 256, 0, s>>>(p, value, g.D, g.Dp, total);
    return hipGetLastError();
}

hipError_t launch_problem_data(const Geometry& g, const es_config& c, float* pdata, hipStream_t s)
{
    k_problem_data<<<grid_for(g.nb, 256), 256, 0, s>>>(pdata, c.seed, g.D, g.nb, c.problem);
    return hipGetLastError();
}

hipError_t launch_ask(const Geometry& g, const es_config& c, uint32_t t, const float* m, float* x,
                      const float* hp, const float* svec, hipStream_t s)
{
    k_ask<<<grid_for((int64_t)g.R * g.P * g.nb, 256), 256, 0, s>>>(m, x, c.seed, t, g.D, g.nb, g.N, g.P,
                                                                   g.R, hp, svec, c.strategy == ES_STRAT_SEP_CMA);
    return hipGetLastError();
}

hipError_t launch_eval_bbob(const Geometry& g, const es_config& c, const EvalPlan& e, uint32_t t,
                            const float* m, const float* pdata, float* partial, float* fit,
                            const float* hp, const float* svec, double div, hipStream_t s, hipEvent_t ev_start,
                            hipEvent_t ev_stop)
{
    // chunk ids are dealt so that the pair groups of one chunk share an XCD
    const int64_t slots = (e.nchunks + 7) / 8 * e.n_pg;
    const dim3 grid((unsigned)(slots * 8), (unsigned)g.R);
    const dim3 block((unsigned)e.wg);
    const int sm = c.strategy == ES_STRAT_SEP_CMA ? SM_INDEP : svec ? SM_VEC : SM_SCALAR;
    const float* sv = sm == SM_SCALAR ? nullptr : svec;
#define ES_EVAL_LAUNCH(PROB, SM)                                                                                \
    launch_timed(k_eval_bbob<PROB, SM>, grid, block, 0, s, ev_start, ev_stop, m, pdata, partial, c.seed, t, g.D, \
                 g.nb, g.N, g.P, e.bc, e.nchunks, e.n_pg, hp, c.rastrigin_a, sv)
#define ES_EVAL_PROB(PROB)                                                                                      \
    (sm == SM_INDEP ? ES_EVAL_LAUNCH(PROB, SM_INDEP) : sm == SM_VEC ? ES_EVAL_LAUNCH(PROB, SM_VEC)               \
                                                                    : ES_EVAL_LAUNCH(PROB, SM_SCALAR))
    hipError_t err;
    switch (c.problem) {
    case ES_PROB_SPHERE: err = ES_EVAL_PROB(ES_PROB_SPHERE); break;
    case ES_PROB_SHIFTED_SPHERE: err = ES_EVAL_PROB(ES_PROB_SHIFTED_SPHERE); break;
    case ES_PROB_ROSENBROCK: err = ES_EVAL_PROB(ES_PROB_ROSENBROCK); break;
    case ES_PROB_RASTRIGIN: err = ES_EVAL_PROB(ES_PROB_RASTRIGIN); break;
    default: return hipErrorInvalidValue;
    }
#undef ES_EVAL_PROB
#undef ES_EVAL_LAUNCH
    if (err != hipSuccess) return err;
    const double add = c.problem == ES_PROB_RASTRIGIN ? (double)c.rastrigin_a * (double)g.D : 0.0;
    return launch_timed(k_eval_reduce, dim3((unsigned)((g.N + 63) / 64), (unsigned)g.R), dim3(64 * RED_SLICES), 0, s,
                        nullptr, nullptr, (const float*)partial, fit, g.N, g.R, e.nchunks, add, div);
}

hipError_t launch_rank(const Geometry& g, const es_config& c, const float* fit, const float* pen,
                       const float* table, double ybar_table, float* y, int32_t* rank, float* wfold, float* bfold,
                       int32_t* elite, int32_t mu, uint32_t* best_okey, float* best_f, int32_t* best_j,
                       float* gen_best, const float* hp_cur, float* hp_next, const RankSortBuffers* rs,
                       hipStream_t s)
{
    const dim3 grid((unsigned)((g.P + RANK_PAIRS - 1) / RANK_PAIRS), (unsigned)g.R);
    const size_t lds = rs ? 0 : sizeof(uint32_t) * (size_t)g.N;
    ShapeArgs sa;
    sa.pen = c.w_decay != 0.0f ? pen : nullptr;
    sa.hp_cur = hp_cur;
    sa.hp_next = hp_next;
    sa.w_decay = c.w_decay;
    // PGPE and SNES: the schedule acts on every dimension's sigma in the
    // tell; the run's sigma only seeded them and stays as it is
    const bool vec = c.strategy == ES_STRAT_PGPE || c.strategy == ES_STRAT_SNES;
    sa.sigma_decay = vec ? 1.0f : c.sigma_decay;
    sa.sigma_final = vec ? 0.0f : c.sigma_final;
    sa.lr_decay = c.lr_decay;
    sa.lr_final = c.lr_final;
    // SNES and Sep-CMA-ES shape by their weight tables (host-made, by rank)
    sa.shaping = c.strategy == ES_STRAT_SNES || c.strategy == ES_STRAT_SEP_CMA ? ES_SHAPE_CENTERED_RANK : c.shaping;
    sa.maximize = c.maximize;
    sa.bmode = c.strategy == ES_STRAT_PGPE ? 1 : c.strategy == ES_STRAT_SNES ? 2 : c.strategy == ES_STRAT_SEP_CMA ? 3 : 0;
    sa.bfold = bfold;
    sa.ybar_table = ybar_table;
    sa.elite = elite;
    sa.mu = mu;
    sa.gkeys = nullptr;
    sa.pre_rank = nullptr;
    sa.stats = nullptr;
    if (rs) {
        // keys, sort, ranks and the per-run statistics ahead of the rank kernel
        const int64_t total = (int64_t)g.R * g.N;
        k_rank_keys<<<grid_for(total, 256), 256, 0, s>>>(fit, sa.pen, g.N, total, c.maximize, c.w_decay, rs->bn,
                                                         rs->keys, rs->kin);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        e = launch_rank_sort(g, *rs, s);
        if (e != hipSuccess) return e;
        k_rank_scatter<<<grid_for(total, 256), 256, 0, s>>>(rs->kout, g.N, total, rs->bn, rank);
        k_rank_stats<<<g.R, RANK_PAIRS * RANK_SLICES, 0, s>>>(fit, rs->keys, g.N, sa, rs->stats);
        sa.gkeys = rs->keys;
        sa.pre_rank = rank;
        sa.stats = rs->stats;
    }
    k_rank<<<grid, RANK_PAIRS * RANK_SLICES, lds, s>>>(fit, table, y, rank, wfold, best_okey, best_f, best_j,
                                                       gen_best, g.N, g.P, g.R, sa);
    return hipGetLastError();
}

hipError_t launch_tell(const Geometry& g, const es_config& c, const TellPlan& tp, uint32_t t, const AdamConsts& ac,
                       const TellBuffers& tb, hipStream_t s)
{
    TellArgs a;
    a.wfold = tb.wfold; a.bfold = tb.bfold; a.best_j = tb.best_j;
    a.m = tb.m; a.m1 = tb.m1; a.v = tb.v; a.grad = tb.grad; a.best_x = tb.best_x;
    a.sig = tb.sig; a.gbuf = tb.gbuf; a.gpart = tb.gpart; a.part = tb.part; a.hp = tb.hp;
    a.elite = tb.elite; a.cw = tb.cw; a.zw = tb.zw; a.qd = tb.qd; a.cma = tb.cma;
    a.nitems = c.strategy == ES_STRAT_SEP_CMA ? tb.cma.mu : g.P;
    a.seed = c.seed; a.t = t; a.D = g.D; a.nb = g.nb; a.P = g.P; a.R = g.R; a.ps = tp.ps; a.nsplit = tp.nsplit;
    a.strategy = c.strategy; a.optimizer = c.optimizer;
    a.sigma_lr = c.sigma_lr; a.max_change = c.sigma_max_change;
    a.sigma_decay = c.sigma_decay; a.sigma_final = c.sigma_final;
    a.ac = ac;
    a.teacher = tb.teacher;
    a.tshift = tb.teacher.w ? MLP_BATCH : 0;
    const bool two = c.strategy != ES_STRAT_OPENAI_ES;
    const bool cma = c.strategy == ES_STRAT_SEP_CMA;
    const bool clipup = c.strategy != ES_STRAT_SNES && !cma && c.optimizer == ES_OPT_CLIPUP;
    if (!clipup && !cma) a.gpart = nullptr;
    // ClipUp and Sep-CMA-ES reduce per-wave norm partials: one lane per block
    const int sub = (!clipup && !cma && tp.nsplit == 1) ? tp.sub : 1;
    const int64_t groups = (g.nb + TELL_LANES / sub - 1) / (TELL_LANES / sub);
    if (a.tshift && !tell_carries_teacher(c, tp)) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(groups + a.tshift), (unsigned)g.R, (unsigned)tp.nsplit);
    const size_t lds = sizeof(double) * (size_t)(tp.ps - 1) * TELL_LANES * (two || cma ? 8 : 4);
    if (a.tshift) k_tell<false, false, 1, true><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    else if (cma) k_tell<true, true><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    else if (two && sub == 4) k_tell<true, false, 4><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    else if (two) k_tell<true><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    else if (sub == 4) k_tell<false, false, 4><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    else k_tell<false><<<grid, TELL_LANES * tp.ps, lds, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 fgrid((unsigned)((g.nb + 255) / 256), (unsigned)g.R);
    if (tp.nsplit > 1) {
        if (two) k_tell_fold<true><<<fgrid, 256, 0, s>>>(a);
        else k_tell_fold<false><<<fgrid, 256, 0, s>>>(a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (cma) {
        k_sepcma_finish<<<fgrid, 256, 0, s>>>(tb.v, tb.cmaC, tb.sig, tb.zw, tb.qd, tb.gpart, tb.hp, tb.hp_next, g.D,
                                               g.nb, groups, t, tb.cma);
        e = hipGetLastError();
    }
    if (clipup) {
        k_clipup_velocity<<<fgrid, 256, 0, s>>>(tb.gbuf, tb.vel, tb.gpart, tb.vpart, tb.hp, g.R, g.nb, groups,
                                                 c.clipup_momentum);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        k_clipup_apply<<<fgrid, 256, 0, s>>>(tb.vel, tb.m, tb.vpart, g.nb, groups, c.clipup_max_speed);
        e = hipGetLastError();
    }
    return e;
}

bool tell_carries_teacher(const es_config& c, const TellPlan& tp)
{
    // the one-sum kernel with one lane per block, in workgroups of at least
    // the teacher's thread count
    const bool clipup = c.optimizer == ES_OPT_CLIPUP;
    const int sub = (!clipup && tp.nsplit == 1) ? tp.sub : 1;
    return c.strategy == ES_STRAT_OPENAI_ES && sub == 1 && TELL_LANES * tp.ps >= TEACHER_THREADS;
}

TellPlan tell_plan(const Geometry& g, bool fused_path, int64_t force_nsplit)
{
    TellPlan tp;
    tp.ps = tell_slices(g);
    if (fused_path) return tp;  // the fused loop sums all slices in one workgroup
    // Few block groups (under four workgroups per CU) leave the CUs unevenly
    // loaded; then split each group's pairs over more, smaller workgroups
    // (four slices each; about 1024 workgroups, which all fit on the chip at
    // once), as long as every slice keeps two whole pair groups.
    const int64_t groups = (g.nb + TELL_LANES - 1) / TELL_LANES * g.R;
    int64_t nsplit = force_nsplit > 0 ? force_nsplit : groups >= 1024 ? 1 : (1024 + groups / 2) / groups;
    while (nsplit > 1 && g.P / (4 * nsplit) < 2 * TELL_GROUP) --nsplit;
    if (nsplit > 1 && nsplit <= 65535) {
        tp.ps = 4;
        tp.nsplit = (int32_t)nsplit;
        return tp;
    }
    // Too few pairs to split and few block groups: four lanes per block, so
    // the groups of 16 blocks spread the run over four times the CUs.
    if (groups < 64 && g.P >= 8 * tp.ps) tp.sub = 4;
    return tp;
}

size_t tell_part_elems(const Geometry& g, const TellPlan& tp, int strategy)
{
    const size_t w = strategy == ES_STRAT_OPENAI_ES ? 4 : 8;
    return tp.nsplit > 1 ? (size_t)g.R * tp.nsplit * g.nb * w : 0;
}

size_t tell_groups(const Geometry& g) { return (size_t)((g.nb + TELL_LANES - 1) / TELL_LANES); }

int32_t tell_slices(const Geometry& g)
{
    // about 4096 waves over the launch, at least 4 slices, at most one per pair
    const int64_t groups = (g.nb + TELL_LANES - 1) / TELL_LANES * g.R;
    int64_t ps = (4096 + groups - 1) / groups;
    if (ps < 4) ps = 4;
    // small runs: enough slices to keep a fused-loop workgroup's lanes busy
    if (ps * g.nb < FUSED_WG) ps = FUSED_WG / g.nb;
    if (ps > TELL_MAX_PS) ps = TELL_MAX_PS;
    if (ps > g.P) ps = g.P;
    // round up to a slice count that splits the pairs into whole groups
    for (int64_t q = ps; q <= TELL_MAX_PS && q <= g.P; ++q)
        if (g.P % q == 0 && (g.P / q) % TELL_GROUP == 0) return (int32_t)q;
    return (int32_t)ps;
}

size_t fused_lds_bytes(const Geometry& g, const EvalPlan& e)
{
    const size_t red = sizeof(double) * (size_t)tell_slices(g) * g.nb * 4;
    // m, m1, v | partials | fit, y | wf | keys (padded to 4) | table
    size_t f32 = (size_t)(3 * g.Dp + e.nchunks * g.N + 2 * g.N + g.P);
    f32 = (f32 + 3) & ~(size_t)3;  // the keys are read four at a time
    f32 += (size_t)((g.N + 3) & ~3) + (size_t)g.N;
    return red + sizeof(float) * f32;
}

size_t fused_stash_bytes(const Geometry& g) { return 16 * (size_t)g.nb * ((size_t)g.P + 1); }

// The normals stay in LDS when the workgroup still fits FUSED_MAX_LDS and the
// runs that share a CU (up to five of the loop's workgroups) still fit its
// 160 KB together.
bool fused_stash(const Geometry& g, const EvalPlan& e)
{
    const size_t per_run = fused_lds_bytes(g, e) + fused_stash_bytes(g);
    const int64_t per_cu = std::min<int64_t>((g.R + 255) / 256, 5);
    return per_run <= FUSED_MAX_LDS && per_run * (size_t)per_cu <= 160 * 1024;
}

bool fused_supported(const Geometry& g, const EvalPlan& e, const es_config& c)
{
    if (c.problem < ES_PROB_SPHERE || c.problem > ES_PROB_RASTRIGIN) return false;
    // the fused loop runs OpenAI-ES with Adam (not PGPE, SNES, Sep-CMA-ES)
    if (c.strategy != ES_STRAT_OPENAI_ES || c.optimizer != ES_OPT_ADAM) return false;
    // the fused loop shapes by centered ranks or raw keys, without weight decay
    if (c.shaping == ES_SHAPE_Z_SCORE || c.w_decay != 0.0f) return false;
    return fused_lds_bytes(g, e) <= FUSED_MAX_LDS;
}

hipError_t launch_run_fused(const Geometry& g, const es_config& c, const EvalPlan& e, uint32_t t0, int32_t T,
                            const AdamConsts& ac, const float (*bcorr)[2], float* m, float* m1, float* v, float* grad,
                            float* best_x, uint32_t* best_okey, float* best_f, const float* pdata, const float* table,
                            float* log, float* hp, hipStream_t s)
{
    if (T < 1 || T > FUSED_MAX_T) return hipErrorInvalidValue;
    FusedArgs a;
    a.m = m; a.m1 = m1; a.v = v; a.grad = grad; a.best_x = best_x; a.best_okey = best_okey; a.best_f = best_f;
    a.pdata = pdata; a.table = table; a.log = log;
    a.ac = ac;
    for (int32_t i = 0; i < T; ++i) {
        a.bcorr[i][0] = bcorr[i][0];
        a.bcorr[i][1] = bcorr[i][1];
    }
    a.seed = c.seed; a.t0 = t0; a.T = T; a.D = g.D; a.nb = g.nb; a.N = g.N; a.P = g.P; a.R = g.R;
    a.bc = e.bc; a.nchunks = e.nchunks; a.ps = tell_slices(g); a.ra = c.rastrigin_a;
    if (a.ps < 1 || a.ps > TELL_MAX_PS) return hipErrorInvalidValue;  // the kernel's slice table holds TELL_MAX_PS + 1
    a.add = c.problem == ES_PROB_RASTRIGIN ? (double)c.rastrigin_a * (double)g.D : 0.0;
    a.maximize = c.maximize; a.raw = c.shaping == ES_SHAPE_RAW;
    a.hp = hp;
    a.sigma_decay = c.sigma_decay; a.sigma_final = c.sigma_final; a.lr_decay = c.lr_decay; a.lr_final = c.lr_final;
    const bool stash = fused_stash(g, e);
    const size_t lds = fused_lds_bytes(g, e) + (stash ? fused_stash_bytes(g) : 0);
#define ES_FUSED_LAUNCH(PROB)                                                     \
    (stash ? (k_run_fused<PROB, true><<<g.R, FUSED_WG, lds, s>>>(a), 0)           \
           : (k_run_fused<PROB, false><<<g.R, FUSED_WG, lds, s>>>(a), 0))
    switch (c.problem) {
    case ES_PROB_SPHERE: ES_FUSED_LAUNCH(ES_PROB_SPHERE); break;
    case ES_PROB_SHIFTED_SPHERE: ES_FUSED_LAUNCH(ES_PROB_SHIFTED_SPHERE); break;
    case ES_PROB_ROSENBROCK: ES_FUSED_LAUNCH(ES_PROB_ROSENBROCK); break;
    case ES_PROB_RASTRIGIN: ES_FUSED_LAUNCH(ES_PROB_RASTRIGIN); break;
    default: return hipErrorInvalidValue;
    }
#undef ES_FUSED_LAUNCH
    return hipGetLastError();
}

int32_t grid_workgroups(const Geometry& g, const EvalPlan& e, int32_t want)
{
    // about 2048 pair-blocks of each of evaluate and gradient per workgroup,
    // at most one per chunk slice of the reduce kernel and, beyond
    // RED_SLICES chunks, a divisor of RED_SLICES (workgroups own whole slices)
    const int64_t nq = e.nchunks < RED_SLICES ? e.nchunks : RED_SLICES;
    int64_t G = want > 0 ? want : ((int64_t)g.P * g.nb + 2047) / 2048;
    if (G > nq) G = nq;
    if (G < 1) G = 1;
    if (e.nchunks > RED_SLICES)
        while (RED_SLICES % G != 0) --G;
    return (int32_t)G;
}

size_t grid_lds_bytes(const Geometry& g, const EvalPlan& e, const TellPlan& tp, int32_t G)
{
    const int64_t S = (int64_t)tp.ps * tp.nsplit * tp.sub;
    const int64_t ncw = (e.nchunks + G - 1) / G, st = 4 * ncw * e.bc;
    // sub-slice sums | rank composites | own members' slice sums | normals | mean windows | m1, v | partials | fit |
    // y | wf | keys (from a 16-byte boundary) | table | pair bounds
    size_t f32 = (size_t)(ncw * (1 + 4 * e.bc) + 2 * st + ncw * g.N + 2 * g.N + g.P);
    f32 = (f32 + 3) & ~(size_t)3;
    f32 += (size_t)((g.N + 3) & ~3) + (size_t)g.N + (size_t)(S + 1);
    const size_t eps = 16 * (size_t)(ncw * e.bc) * ((size_t)g.P + 1);  // float4 normals
    const size_t msl = (size_t)((g.N + G - 1) / G) * RED_SLICES;
    return sizeof(double) * (size_t)(S * st + ((g.N + 1) & ~1) + msl) + eps + sizeof(float) * f32;
}

bool grid_supported(const Geometry& g, const EvalPlan& e, const TellPlan& tp, const es_config& c, int32_t G)
{
    // what the fused loop runs (OpenAI-ES with Adam, centered ranks or raw
    // keys, no weight decay), with every workgroup ranking the run's members
    if (c.problem < ES_PROB_SPHERE || c.problem > ES_PROB_RASTRIGIN) return false;
    if (c.strategy != ES_STRAT_OPENAI_ES || c.optimizer != ES_OPT_ADAM) return false;
    if (c.shaping == ES_SHAPE_Z_SCORE || c.w_decay != 0.0f) return false;
    if (g.N > GRID_MAX_N || (int64_t)G * g.R > 65535) return false;
    if (tp.sub != 1 && tp.sub != 2 && tp.sub != 4) return false;
    if ((int64_t)tp.ps * tp.nsplit * tp.sub > g.P) return false;  // every sub-slice is a pair range
    // workgroups own whole chunk slices
    const int64_t nq = e.nchunks < RED_SLICES ? e.nchunks : RED_SLICES;
    if (G < 1 || G > nq || (e.nchunks > RED_SLICES && RED_SLICES % G != 0)) return false;
    return grid_lds_bytes(g, e, tp, G) <= GRID_MAX_LDS;
}

static_assert(RED_SLICES == 16, "grid_word_count sizes the slice sums for 16 slices");

hipError_t grid_max_resident(int64_t* out)
{
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    // every grid-loop launch stays within GRID_MAX_LDS of dynamic LDS
    if (e == hipSuccess)
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_run_grid<ES_PROB_ROSENBROCK>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)GRID_MAX_LDS);
    if (e == hipSuccess)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(&k_run_grid<ES_PROB_ROSENBROCK>),
                                                         GRID_WG, GRID_MAX_LDS);
    *out = e == hipSuccess ? (int64_t)cus * per_cu : 0;
    return e;
}

hipError_t launch_run_grid(const Geometry& g, const es_config& c, const EvalPlan& e, const TellPlan& tp, int32_t G,
                           int32_t xs,
                           uint32_t t0, int32_t T, const AdamConsts& ac, const float (*bcorr)[2], float* m, float* m1,
                           float* v, float* grad, float* best_x, uint32_t* best_okey, float* best_f,
                           const float* pdata, const float* table, float* log, uint64_t* words, uint32_t seq,
                           uint32_t* err, float* hp, hipStream_t s)
{
    if (T < 1 || T > FUSED_MAX_T || G < 1 || G > GRID_MAX_G || xs < 1 || xs > 64) return hipErrorInvalidValue;
    if (!grid_supported(g, e, tp, c, G)) return hipErrorInvalidValue;
    GridArgs a;
    a.m = m; a.m1 = m1; a.v = v; a.grad = grad; a.best_x = best_x; a.best_okey = best_okey; a.best_f = best_f;
    a.pdata = pdata; a.table = table; a.log = log;
    a.sx = words;
    a.fx = a.sx + (size_t)g.R * RED_SLICES * g.N * 2;
    a.yx = a.fx + (size_t)g.R * g.N;
    a.bestx = a.yx + (size_t)g.R * g.N;
    a.halo = a.bestx + g.R;
    a.err = err;
    // polls before a wait gives up: the library's limit, a caller's, or
    // none at all (-1: every wait gives up at once)
    a.spin = c.plan_grid_spin_limit == 0 ? GRID_SPIN_LIMIT
             : c.plan_grid_spin_limit < 0 ? 0u
                                          : (uint32_t)c.plan_grid_spin_limit;
    if (seq < 1 || seq >= (1u << 24)) return hipErrorInvalidValue;
    a.tag0 = seq << 8;
    a.xs = xs;
    a.ac = ac;
    for (int32_t i = 0; i < T; ++i) {
        a.bcorr[i][0] = bcorr[i][0];
        a.bcorr[i][1] = bcorr[i][1];
    }
    a.seed = c.seed; a.t0 = t0; a.T = T; a.D = g.D; a.nb = g.nb; a.N = g.N; a.P = g.P; a.R = g.R;
    a.bc = e.bc; a.nchunks = e.nchunks; a.ps = tp.ps; a.nsplit = tp.nsplit; a.sub = tp.sub;
    a.ncw = (int32_t)((e.nchunks + G - 1) / G);
    a.ra = c.rastrigin_a;
    a.add = c.problem == ES_PROB_RASTRIGIN ? (double)c.rastrigin_a * (double)g.D : 0.0;
    a.maximize = c.maximize; a.raw = c.shaping == ES_SHAPE_RAW;
    a.hp = hp;
    a.sigma_decay = c.sigma_decay; a.sigma_final = c.sigma_final; a.lr_decay = c.lr_decay; a.lr_final = c.lr_final;
    hipError_t herr;
    const uint32_t lds = (uint32_t)grid_lds_bytes(g, e, tp, G);
    void* args[] = {&a};
    const void* k;
    const bool spin_arg = c.plan_grid_spin_limit != 0;
#define ES_GRID_KERNEL(PROB)                                                                       \
    (spin_arg ? reinterpret_cast<const void*>(&k_run_grid<PROB, true>)                             \
              : reinterpret_cast<const void*>(&k_run_grid<PROB, false>))
    switch (c.problem) {
    case ES_PROB_SPHERE: k = ES_GRID_KERNEL(ES_PROB_SPHERE); break;
    case ES_PROB_SHIFTED_SPHERE: k = ES_GRID_KERNEL(ES_PROB_SHIFTED_SPHERE); break;
    case ES_PROB_ROSENBROCK: k = ES_GRID_KERNEL(ES_PROB_ROSENBROCK); break;
    case ES_PROB_RASTRIGIN: k = ES_GRID_KERNEL(ES_PROB_RASTRIGIN); break;
    default: return hipErrorInvalidValue;
    }
#undef ES_GRID_KERNEL
    // more than 64 KB of LDS per workgroup: allowed per kernel (cheap to repeat)
    herr = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)GRID_MAX_LDS);
    if (herr != hipSuccess) return herr;
    return hipLaunchCooperativeKernel(k, dim3((unsigned)(G * xs), (unsigned)g.R), dim3(GRID_WG), args, lds, s);
}

hipError_t launch_debug_noise(const Geometry& g, const es_config& c, int32_t run, uint32_t t,
                              int32_t pair, uint32_t* words, float* eps, hipStream_t s)
{
    k_debug_noise<<<grid_for(g.nb, 256), 256, 0, s>>>(words, eps, c.seed + (uint64_t)run, (uint32_t)pair, t,
                                                      g.D, g.nb);
    return hipGetLastError();
}

// Scratch of the allocation-free evaluate (es_eval_noalloc): the per-chunk
// partial sums live in this array, one copy per device, held until the
// process ends.  Host code never passes the array's name to a kernel (on the
// host it is a stand-in, not a device address): noalloc_scratch looks up each
// device's address once, with that device current, and hands that out.
static __device__ __align__(256) float scratch[NOALLOC_SCRATCH_FLOATS];

hipError_t noalloc_scratch(float** out)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float* addr[kMaxDevices] = {};
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<float*>(p);
    }
    *out = addr[dev];
    return hipSuccess;
}

}  // namespace esmi
