// es_mlp.hip -- neuroevolution fitness on gfx950: a 64-256-256-16 tanh MLP
// whose flat parameter vector is the search point (network definitions and
// parameter reshaping, Sec. 3.2 of the evosax report), scored by -MSE
// against a fixed random teacher network of the same shape.
//
//   k_mlp_teacher  X_t [256][64] ~ N(0,1) from the EVAL stream of the base
//                  seed (fp32 for the teacher, bf16 for the students) and
//                  the fp32 teacher forward on it -> Y_T [256][16]; after
//                  the first generation the gradient launch of generation
//                  t computes them for t+1 (es_teacher.hpp)
//   k_eval_mlp     one workgroup per antithetic pair: the pair's noise is
//                  regenerated once and turned into both members' weights
//                  (bf16(m +- sigma*eps), biases fp32) in LDS; the forward
//                  runs on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
//
// Layout of the flat vector: per layer the [out][in] row-major weights, then
// the bias: W1 [256][64], b1 [256], W2 [256][256], b2 [256], W3 [16][256],
// b3 [16]; D = 86,544.  Every boundary is a multiple of 4, so no Philox block
// straddles two tensors.
//
// MFMA mapping.  The layers are computed transposed, Z^T = W . H^T, so the
// weights are the A operand (16 out-rows x 32 in) and the activations the B
// operand (32 in x 16 batch).  Each wave owns 32 batch columns (two B tiles)
// for the whole network, so activations never leave registers: the 16x16
// accumulator tiles of rows [r0, r0+16) and [r0+16, r0+32) hold, per lane,
// rows 4q+i and 16+4q+i (q = lane/16, i < 4) of batch column lane%16, which
// is exactly a B operand of the next layer whose 32 K-slots are taken in the
// order pi(8q+i) = 4q+i, pi(8q+4+i) = 16+4q+i.  The next layer's weights are
// read from LDS in the same K order, so the contraction is unchanged.
#include <hip/hip_runtime.h>
#include <math.h>

#include "es_device.hpp"
#include "es_internal.hpp"
#include "es_teacher.hpp"

namespace esmi {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int MLP_WAVES = 16;          // per member: 8 waves x 32 batch columns = 256 inputs
constexpr int MLP_THREADS = 64 * MLP_WAVES;
constexpr int W2_ROWS = 32;            // W2 rows per LDS chunk (one K-step of layer 3)
constexpr int W2_CHUNKS = MLP_H / W2_ROWS;
constexpr int W2_BLOCKS_PER_THREAD = W2_ROWS * MLP_H / 4 / MLP_THREADS;  // Philox blocks per lane per chunk
static_assert(W2_BLOCKS_PER_THREAD * MLP_THREADS * 4 == W2_ROWS * MLP_H, "W2 chunk must split evenly");
static_assert(8 % W2_BLOCKS_PER_THREAD == 0, "generation steps must divide the K loop");
// LDS row strides (bf16 elements), padded so that the A-operand reads of a
// 16-lane group hit distinct banks
constexpr int W1S = MLP_IN + 8;        // W1 tile [256][64]
constexpr int W2S = MLP_H + 4;         // W2 chunk [32][256]
constexpr int W3S = MLP_H + 4;         // W3 [16][256]
constexpr int W1_TILE = MLP_H * W1S;
constexpr int W2_TILE = W2_ROWS * W2S;

// The W1 tiles are dead once layer 1 is done, so the second W2 chunk buffer
// reuses their space.
struct MlpSmem {
    union {
        __bf16 w1[2][W1_TILE];     // member +, member -
        __bf16 w2b[2][W2_TILE];    // W2 chunk buffer 1
    } a;
    __bf16 w2a[2][W2_TILE];        // W2 chunk buffer 0
    __bf16 w3[2][MLP_OUT * W3S];
    float b1[2][MLP_H], b2[2][MLP_H], b3[2][MLP_OUT];  // b1, b2 times 2 log2(e)
    double red[MLP_WAVES];
};

// tanh x = 1 - 2 / (2^u + 1) with u = 2 log2(e) x: v_exp_f32 and v_rcp_f32,
// saturating to +-1.  The hidden layers keep their biases pre-multiplied by
// 2 log2(e) so that u = fma(z, 2 log2(e), that product) is one instruction.
constexpr float TWO_LOG2E = 2.88539008177792681472f;

__device__ __forceinline__ float tanh_scaled(float u)
{
    return fmaf(-2.0f, __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f(u) + 1.0f), 1.0f);
}

__device__ __forceinline__ float tanh_fast(float x) { return tanh_scaled(x * TWO_LOG2E); }

__device__ __forceinline__ bf16x8 cat(bf16x4 lo, bf16x4 hi)
{
    bf16x8 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[i] = lo[i];
        r[4 + i] = hi[i];
    }
    return r;
}

// Bias, activation and bf16 rounding of two stacked accumulator tiles
// (rows r0+4q+i and r0+16+4q+i) into one B operand of the next layer;
// biasK holds the layer's biases times 2 log2(e).
__device__ __forceinline__ bf16x8 activate(const floatx4& lo, const floatx4& hi, const float* biasK, int r0, int q)
{
    bf16x8 h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h[i] = (__bf16)tanh_scaled(fmaf(lo[i], TWO_LOG2E, biasK[r0 + 4 * q + i]));
        h[4 + i] = (__bf16)tanh_scaled(fmaf(hi[i], TWO_LOG2E, biasK[r0 + 16 + 4 * q + i]));
    }
    return h;
}

// Two fp32 values rounded to bf16 (round to nearest even) in one
// v_cvt_pk_bf16_f32: lo in bits 0-15, hi in bits 16-31.  Written out because
// the compiler otherwise paired the two members' values and repacked them.
__device__ __forceinline__ uint32_t pk_bf16(float lo, float hi)
{
    uint32_t r;
    asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
    return r;
}

// One Philox block (4 weights) of W2 chunk `chunk` into the chunk buffers.
// VEC: per-dimension sigma from sr (PGPE, SNES).
template <bool VEC>
__device__ __forceinline__ void gen_w2_block(const float* __restrict__ mr, const float* __restrict__ sr, uint32_t k0,
                                             uint32_t k1, uint32_t pair, uint32_t t, int chunk, int i, float sigma,
                                             __bf16* wp, __bf16* wm)
{
    const int64_t b = (OFF_W2 + (int64_t)chunk * W2_ROWS * MLP_H) / 4 + i;
    float e[4];
    box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)b, pair, t, DOM_NOISE), e);
    const float4 m4 = *reinterpret_cast<const float4*>(mr + 4 * b);
    const float mv[4] = {m4.x, m4.y, m4.z, m4.w};
    float sv[4] = {sigma, sigma, sigma, sigma};
    if constexpr (VEC) {
        const float4 s4 = *reinterpret_cast<const float4*>(sr + 4 * b);
        sv[0] = s4.x; sv[1] = s4.y; sv[2] = s4.z; sv[3] = s4.w;
    }
    float xp[4], xm[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        xp[k] = fmaf(sv[k], e[k], mv[k]);
        xm[k] = fmaf(-sv[k], e[k], mv[k]);
    }
    const int row = (4 * i) / MLP_H, col = (4 * i) % MLP_H;
    *reinterpret_cast<uint2*>(wp + row * W2S + col) = make_uint2(pk_bf16(xp[0], xp[1]), pk_bf16(xp[2], xp[3]));
    *reinterpret_cast<uint2*>(wm + row * W2S + col) = make_uint2(pk_bf16(xm[0], xm[1]), pk_bf16(xm[2], xm[3]));
}

// Layer 2 on one W2 chunk (rows [W2_ROWS*c, +W2_ROWS)) for this wave's
// member: acc = W2[chunk] . H1^T.
__device__ __forceinline__ void layer2_mfma(const __bf16* wc, const bf16x8 (&h1)[8][2], floatx4 (&acc)[2][2], int q,
                                            int l16)
{
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < 8; ++g)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
            const __bf16* row = wc + (16 * mt + l16) * W2S + 32 * g;
            const bf16x8 A = cat(*reinterpret_cast<const bf16x4*>(row + 4 * q),
                                 *reinterpret_cast<const bf16x4*>(row + 16 + 4 * q));
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, h1[g][nt], acc[mt][nt], 0, 0, 0);
        }
}

// Bias + tanh + bf16 of the chunk's layer-2 rows, then that chunk's share of
// layer 3 (the chunk's rows are layer 3's K range).
__device__ __forceinline__ void layer2_act(const MlpSmem& S, const floatx4 (&acc)[2][2], int c, int mem,
                                           floatx4 (&y)[2], int q, int l16)
{
    const int r0 = W2_ROWS * c;
    const __bf16* w3row = S.w3[mem] + l16 * W3S + r0;
    const bf16x8 A3 = cat(*reinterpret_cast<const bf16x4*>(w3row + 4 * q),
                          *reinterpret_cast<const bf16x4*>(w3row + 16 + 4 * q));
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const bf16x8 hb = activate(acc[0][nt], acc[1][nt], S.b2[mem], r0, q);
        y[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A3, hb, y[nt], 0, 0, 0);
    }
}

// One workgroup per antithetic pair: waves 0-7 evaluate member p (+eps),
// waves 8-15 member p + N/2 (-eps); each wave owns 32 batch columns.
template <bool VEC>
__global__ __launch_bounds__(MLP_THREADS) void k_eval_mlp(const float* __restrict__ m, const __bf16* __restrict__ xb,
                                                          const float* __restrict__ yt, float* __restrict__ fit,
                                                          uint64_t seed, uint32_t t, int64_t Dp, int32_t N,
                                                          int32_t P, const float* __restrict__ hp, int32_t tanh_out,
                                                          const float* __restrict__ svec)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    MlpSmem& S = *reinterpret_cast<MlpSmem*>(smem_raw);
    const int32_t p = blockIdx.x, r = blockIdx.y;
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, q = lane / 16, l16 = lane % 16;
    const int mem = wave / 8;                 // 0: +eps, 1: -eps
    const int nbase = 32 * (wave % 8);        // this wave's batch columns
    const uint64_t key = seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    const float* __restrict__ mr = m + (int64_t)r * Dp;
    const float* __restrict__ sr = VEC ? svec + (int64_t)r * Dp : nullptr;
    const float sigma = hp[r];

    // ---- layer 1 and layer 3 weights, W2 chunk 0, all biases.  Each thread
    // owns seven weight blocks (W1: tid + 1024k, W3: tid, W2 chunk 0: tid and
    // tid + 1024); the 132 bias blocks go to the last threads.  All mean
    // words are fetched before the first Philox block is generated.
    {
        const int tid = (int)threadIdx.x;
        constexpr int NB1 = MLP_H * MLP_IN / 4, NB3 = MLP_OUT * MLP_H / 4;
        static_assert(NB1 == 4 * MLP_THREADS && NB3 == MLP_THREADS && W2_ROWS * MLP_H / 4 == 2 * MLP_THREADS,
                      "prologue block split");
        constexpr int NBIAS = (2 * MLP_H + MLP_OUT) / 4;
        const int64_t blk[7] = {OFF_W1 / 4 + tid, OFF_W1 / 4 + tid + MLP_THREADS, OFF_W1 / 4 + tid + 2 * MLP_THREADS,
                                OFF_W1 / 4 + tid + 3 * MLP_THREADS, OFF_W3 / 4 + tid, OFF_W2 / 4 + tid,
                                OFF_W2 / 4 + tid + MLP_THREADS};
        float4 mw[7], sw[VEC ? 7 : 1];
#pragma unroll
        for (int k = 0; k < 7; ++k) mw[k] = *reinterpret_cast<const float4*>(mr + 4 * blk[k]);
        if constexpr (VEC) {
#pragma unroll
            for (int k = 0; k < 7; ++k) sw[k] = *reinterpret_cast<const float4*>(sr + 4 * blk[k]);
        }
        const int jb = tid - (MLP_THREADS - NBIAS);  // bias block of this thread, if >= 0
        const int64_t bblk = jb < MLP_H / 4 ? OFF_B1 / 4 + jb : jb < MLP_H / 2 ? OFF_B2 / 4 + (jb - MLP_H / 4)
                                                                                : OFF_B3 / 4 + (jb - MLP_H / 2);
        float4 mb = make_float4(0.f, 0.f, 0.f, 0.f);
        if (jb >= 0) mb = *reinterpret_cast<const float4*>(mr + 4 * bblk);
#pragma unroll
        for (int k = 0; k < 7; ++k) {
            float e[4];
            box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)blk[k], (uint32_t)p, t, DOM_NOISE), e);
            const float mv[4] = {mw[k].x, mw[k].y, mw[k].z, mw[k].w};
            float sv[4] = {sigma, sigma, sigma, sigma};
            if constexpr (VEC) {
                sv[0] = sw[k].x; sv[1] = sw[k].y; sv[2] = sw[k].z; sv[3] = sw[k].w;
            }
            float xp[4], xm[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                xp[i] = fmaf(sv[i], e[i], mv[i]);
                xm[i] = fmaf(-sv[i], e[i], mv[i]);
            }
            const uint2 vp = make_uint2(pk_bf16(xp[0], xp[1]), pk_bf16(xp[2], xp[3]));
            const uint2 vm = make_uint2(pk_bf16(xm[0], xm[1]), pk_bf16(xm[2], xm[3]));
            __bf16 *dp, *dm;
            if (k < 4) {  // W1 [256][64]
                const int i4 = 4 * (tid + k * MLP_THREADS);
                dp = S.a.w1[0] + (i4 / MLP_IN) * W1S + i4 % MLP_IN;
                dm = S.a.w1[1] + (i4 / MLP_IN) * W1S + i4 % MLP_IN;
            } else if (k == 4) {  // W3 [16][256]
                const int i4 = 4 * tid;
                dp = S.w3[0] + (i4 / MLP_H) * W3S + i4 % MLP_H;
                dm = S.w3[1] + (i4 / MLP_H) * W3S + i4 % MLP_H;
            } else {  // W2 chunk 0 [32][256]
                const int i4 = 4 * (tid + (k - 5) * MLP_THREADS);
                dp = S.w2a[0] + (i4 / MLP_H) * W2S + i4 % MLP_H;
                dm = S.w2a[1] + (i4 / MLP_H) * W2S + i4 % MLP_H;
            }
            *reinterpret_cast<uint2*>(dp) = vp;
            *reinterpret_cast<uint2*>(dm) = vm;
        }
        if (jb >= 0) {
            float e[4];
            box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)bblk, (uint32_t)p, t, DOM_NOISE), e);
            const float mv[4] = {mb.x, mb.y, mb.z, mb.w};
            float sv[4] = {sigma, sigma, sigma, sigma};
            if constexpr (VEC) {
                const float4 s4 = *reinterpret_cast<const float4*>(sr + 4 * bblk);
                sv[0] = s4.x; sv[1] = s4.y; sv[2] = s4.z; sv[3] = s4.w;
            }
            float *bp, *bm;
            if (jb < MLP_H / 4) {
                bp = S.b1[0] + 4 * jb; bm = S.b1[1] + 4 * jb;
            } else if (jb < MLP_H / 2) {
                bp = S.b2[0] + 4 * (jb - MLP_H / 4); bm = S.b2[1] + 4 * (jb - MLP_H / 4);
            } else {
                bp = S.b3[0] + 4 * (jb - MLP_H / 2); bm = S.b3[1] + 4 * (jb - MLP_H / 2);
            }
            const float sc = jb < MLP_H / 2 ? TWO_LOG2E : 1.0f;  // hidden-layer biases pre-scaled
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                bp[i] = fmaf(sv[i], e[i], mv[i]) * sc;
                bm[i] = fmaf(-sv[i], e[i], mv[i]) * sc;
            }
        }
    }

    // input B operands: X[n][32ks + 8q + i] for batch column n of tile nt
    bf16x8 xop[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
            xop[ks][nt] = *reinterpret_cast<const bf16x8*>(xb + (nbase + 16 * nt + l16) * MLP_IN + 32 * ks + 8 * q);
    __syncthreads();

    // ---- layer 1: H1^T (256 x 32), kept as layer-2 B operands
    bf16x8 h1[8][2];
    const __bf16* W1 = S.a.w1[mem];
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        floatx4 cc[2][2];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) cc[a][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 A = *reinterpret_cast<const bf16x8*>(W1 + (32 * g + 16 * a + l16) * W1S + 32 * ks + 8 * q);
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
                    cc[a][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, xop[ks][nt], cc[a][nt], 0, 0, 0);
            }
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) h1[g][nt] = activate(cc[0][nt], cc[1][nt], S.b1[mem], 32 * g, q);
    }
    __syncthreads();  // W1 is dead from here on; its space holds chunk buffer 1

    // teacher outputs of this lane's (batch column, output) entries, fetched
    // early: Y_T[n][4q .. 4q+3] for n = nbase + 16 nt + l16
    float4 yref[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
        yref[nt] = *reinterpret_cast<const float4*>(yt + (nbase + 16 * nt + l16) * MLP_OUT + 4 * q);

    // ---- layer 2 chunk by chunk, generating the next chunk meanwhile
    floatx4 y[2] = {floatx4{0.f, 0.f, 0.f, 0.f}, floatx4{0.f, 0.f, 0.f, 0.f}};
    for (int c = 0; c < W2_CHUNKS; ++c) {
        // Even chunks live in buffer 0, odd ones in buffer 1.  Each lane also
        // generates its share of chunk c+1 into the other buffer: the waves of
        // member + do that before their matrix work, those of member - after
        // it, so that every SIMD has VALU and MFMA work in flight together.
        __bf16* nb_p = (c & 1) ? S.w2a[0] : S.a.w2b[0];
        __bf16* nb_m = (c & 1) ? S.w2a[1] : S.a.w2b[1];
        const __bf16* wc = (c & 1) ? S.a.w2b[mem] : S.w2a[mem];
        const bool gen = c + 1 < W2_CHUNKS;
        if (mem == 0 && gen)
#pragma unroll
            for (int j = 0; j < W2_BLOCKS_PER_THREAD; ++j)
                gen_w2_block<VEC>(mr, sr, k0, k1, (uint32_t)p, t, c + 1, (int)threadIdx.x + j * MLP_THREADS, sigma, nb_p,
                                  nb_m);
        {
            floatx4 acc[2][2];
            layer2_mfma(wc, h1, acc, q, l16);
            layer2_act(S, acc, c, mem, y, q, l16);
        }
        if (mem == 1 && gen)
#pragma unroll
            for (int j = 0; j < W2_BLOCKS_PER_THREAD; ++j)
                gen_w2_block<VEC>(mr, sr, k0, k1, (uint32_t)p, t, c + 1, (int)threadIdx.x + j * MLP_THREADS, sigma, nb_p,
                                  nb_m);
        __syncthreads();
    }

    // ---- output layer bias, squared error against the teacher
    double se = 0.0;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const float yr[4] = {yref[nt].x, yref[nt].y, yref[nt].z, yref[nt].w};
        float sq = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int o = 4 * q + i;
            float v = y[nt][i] + S.b3[mem][o];
            if (tanh_out) v = tanh_fast(v);
            const float d = v - yr[i];
            sq = fmaf(d, d, sq);
        }
        se += (double)sq;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off);
    if (lane == 0) S.red[wave] = se;
    __syncthreads();
    if (threadIdx.x < 2) {
        double tot = 0.0;
        for (int w = 0; w < 8; ++w) tot += S.red[8 * threadIdx.x + w];
        const double mse = tot / (double)(MLP_BATCH * MLP_OUT);
        fit[(int64_t)r * N + p + (threadIdx.x ? P : 0)] = (float)(-mse);
    }
}

// The teacher's weights transposed once at set-up: W1^T [64][256],
// W2^T [256][256], W3^T [256][16] (the biases are not copied), so that the
// per-generation forward reads them coalesced.
__global__ void k_mlp_transpose(const float* __restrict__ w, float* __restrict__ wt)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;  // destination index
    if (i < MLP_IN * MLP_H) {
        const int k = i / MLP_H, o = i % MLP_H;
        wt[OFF_W1 + i] = w[OFF_W1 + o * MLP_IN + k];
    } else if (i < MLP_IN * MLP_H + MLP_H * MLP_H) {
        const int j = i - MLP_IN * MLP_H, k = j / MLP_H, o = j % MLP_H;
        wt[OFF_W2 + j] = w[OFF_W2 + o * MLP_H + k];
    } else if (i < MLP_IN * MLP_H + MLP_H * MLP_H + MLP_H * MLP_OUT) {
        const int j = i - MLP_IN * MLP_H - MLP_H * MLP_H, k = j / MLP_OUT, o = j % MLP_OUT;
        wt[OFF_W3 + j] = w[OFF_W3 + o * MLP_H + k];
    }
}

// Per generation: X_t and Y_T, one workgroup per input row.
__global__ __launch_bounds__(TEACHER_THREADS) void k_mlp_teacher(TeacherJob j) { teacher_row(j, blockIdx.x); }

}  // namespace

size_t mlp_scratch_bytes()
{
    // X_t fp32, X_t bf16, Y_T, transposed teacher
    return sizeof(float) * MLP_BATCH * MLP_IN + sizeof(__bf16) * MLP_BATCH * MLP_IN + sizeof(float) * MLP_BATCH * MLP_OUT +
           sizeof(float) * MLP_NUM_PARAMS;
}

hipError_t launch_mlp_setup(const float* teacher, void* scratch, hipStream_t s)
{
    float* wt = reinterpret_cast<float*>(static_cast<char*>(scratch) + mlp_scratch_bytes() - sizeof(float) * MLP_NUM_PARAMS);
    const int n = MLP_IN * MLP_H + MLP_H * MLP_H + MLP_H * MLP_OUT;
    k_mlp_transpose<<<(n + 255) / 256, 256, 0, s>>>(teacher, wt);
    return hipGetLastError();
}

size_t mlp_lds_bytes() { return sizeof(MlpSmem); }

TeacherJob mlp_teacher_job(const es_config& c, const float* teacher, void* scratch, uint32_t t)
{
    TeacherJob j;
    j.xf = static_cast<float*>(scratch);
    j.xb = reinterpret_cast<__bf16*>(j.xf + MLP_BATCH * MLP_IN);
    j.yt = reinterpret_cast<float*>(j.xb + MLP_BATCH * MLP_IN);
    j.wt = reinterpret_cast<const float*>(static_cast<const char*>(scratch) + mlp_scratch_bytes() -
                                          sizeof(float) * MLP_NUM_PARAMS);
    j.w = teacher;
    j.seed = c.seed;
    j.t = t;
    j.tanh_out = c.mlp_tanh_out;
    return j;
}

hipError_t launch_eval_mlp(const Geometry& g, const es_config& c, uint32_t t, const float* m, const float* teacher,
                           void* scratch, float* fit, const float* hp, const float* svec, bool run_teacher,
                           hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop)
{
    const TeacherJob j = mlp_teacher_job(c, teacher, scratch, t);
    const __bf16* xb = j.xb;
    const float* yt = j.yt;
    if (run_teacher) {
        hipError_t e = launch_timed(k_mlp_teacher, dim3(MLP_BATCH), dim3(TEACHER_THREADS), 0, s, nullptr, nullptr, j);
        if (e != hipSuccess) return e;
    }
    // more than 64 KB of LDS per workgroup: allowed per kernel (cheap to repeat)
    const void* kern = svec ? reinterpret_cast<const void*>(&k_eval_mlp<true>)
                            : reinterpret_cast<const void*>(&k_eval_mlp<false>);
    const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(MlpSmem));
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)g.P, (unsigned)g.R);
    if (svec)
        return launch_timed(k_eval_mlp<true>, grid, dim3(MLP_THREADS), (uint32_t)sizeof(MlpSmem), s, ev_start, ev_stop,
                            m, xb, yt, fit, c.seed, t, g.Dp, g.N, g.P, hp, c.mlp_tanh_out, svec);
    return launch_timed(k_eval_mlp<false>, grid, dim3(MLP_THREADS), (uint32_t)sizeof(MlpSmem), s, ev_start, ev_stop,
                        m, xb, yt, fit, c.seed, t, g.Dp, g.N, g.P, hp, c.mlp_tanh_out, (const float*)nullptr);
}

}  // namespace esmi
