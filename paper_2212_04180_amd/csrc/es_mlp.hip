// es_mlp.hip -- neuroevolution fitness on gfx950: a 64-256-256-16 tanh MLP
// whose flat parameter vector is the search point (network definitions and
// parameter reshaping, Sec. 3.2 of the evosax report), scored by -MSE
// against a fixed random teacher network of the same shape.
//
//   k_mlp_inputs   X_t [256][64] ~ N(0,1) from the EVAL stream of the base
//                  seed: fp32 for the teacher, bf16 for the students
//   k_mlp_teacher  fp32 teacher forward on X_t -> Y_T [256][16]
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

namespace esmi {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int MLP_IN = 64, MLP_H = 256, MLP_OUT = 16, MLP_BATCH = 256;
constexpr int64_t OFF_W1 = 0, OFF_B1 = 16384, OFF_W2 = 16640, OFF_B2 = 82176, OFF_W3 = 82432, OFF_B3 = 86528;
constexpr int MLP_WAVES = 8;           // 8 x 32 batch columns = 256 inputs
constexpr int MLP_THREADS = 64 * MLP_WAVES;
constexpr int W2_ROWS = 64;            // W2 rows generated per LDS round
// LDS row strides (bf16 elements), padded against bank conflicts
constexpr int W1S = MLP_IN + 8;        // W1 tile [256][64]
constexpr int W2S = MLP_H + 8;         // W2 chunk [64][256]
constexpr int W3S = MLP_H + 8;         // W3 [16][256]
constexpr int WTILE = (MLP_H * W1S > W2_ROWS * W2S) ? MLP_H * W1S : W2_ROWS * W2S;

struct MlpSmem {
    __bf16 w[2][WTILE];            // member +, member -: W1 or the current W2 chunk
    __bf16 w3[2][MLP_OUT * W3S];
    float b1[2][MLP_H], b2[2][MLP_H], b3[2][MLP_OUT];
    double red[MLP_WAVES][2];
};

// tanh x = 1 - 2 / (e^{2x} + 1): v_exp_f32 and v_rcp_f32, saturating to +-1.
__device__ __forceinline__ float tanh_fast(float x)
{
    const float e = __builtin_amdgcn_exp2f(x * 2.88539008177792681472f);
    return fmaf(-2.0f, __builtin_amdgcn_rcpf(e + 1.0f), 1.0f);
}

// Perturbed weights of flat range [off, off + rows*cols) (a [rows][cols]
// block of one tensor), written as bf16 to two LDS tiles with row stride ld.
// Lanes vary in the Philox block; the pair is uniform.
__device__ __forceinline__ void gen_weights(const float* __restrict__ mr, uint32_t k0, uint32_t k1, uint32_t pair,
                                            uint32_t t, int64_t off, int rows, int cols, float sigma, __bf16* wp,
                                            __bf16* wm, int ld)
{
    const int nblk = rows * cols / 4;
    for (int i = threadIdx.x; i < nblk; i += blockDim.x) {
        const int64_t b = off / 4 + i;
        float e[4];
        box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)b, pair, t, DOM_NOISE), e);
        const float4 m4 = *reinterpret_cast<const float4*>(mr + 4 * b);
        const float mv[4] = {m4.x, m4.y, m4.z, m4.w};
        bf16x4 vp, vm;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            vp[k] = (__bf16)fmaf(sigma, e[k], mv[k]);
            vm[k] = (__bf16)fmaf(-sigma, e[k], mv[k]);
        }
        const int row = (4 * i) / cols, col = (4 * i) % cols;
        *reinterpret_cast<bf16x4*>(wp + row * ld + col) = vp;
        *reinterpret_cast<bf16x4*>(wm + row * ld + col) = vm;
    }
}

// Perturbed biases of flat range [off, off + n), fp32.
__device__ __forceinline__ void gen_bias(const float* __restrict__ mr, uint32_t k0, uint32_t k1, uint32_t pair,
                                         uint32_t t, int64_t off, int n, float sigma, float* bp, float* bm)
{
    for (int i = threadIdx.x; i < n / 4; i += blockDim.x) {
        const int64_t b = off / 4 + i;
        float e[4];
        box_muller4(philox4x32_10<LANES_BLOCK>(k0, k1, (uint32_t)b, pair, t, DOM_NOISE), e);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bp[4 * i + k] = fmaf(sigma, e[k], mr[4 * b + k]);
            bm[4 * i + k] = fmaf(-sigma, e[k], mr[4 * b + k]);
        }
    }
}

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
// (rows r0+4q+i and r0+16+4q+i) into one B operand of the next layer.
__device__ __forceinline__ bf16x8 activate(const floatx4& lo, const floatx4& hi, const float* bias, int r0, int q)
{
    bf16x8 h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h[i] = (__bf16)tanh_fast(lo[i] + bias[r0 + 4 * q + i]);
        h[4 + i] = (__bf16)tanh_fast(hi[i] + bias[r0 + 16 + 4 * q + i]);
    }
    return h;
}

__global__ __launch_bounds__(MLP_THREADS) void k_eval_mlp(const float* __restrict__ m, const __bf16* __restrict__ xb,
                                                          const float* __restrict__ yt, float* __restrict__ fit,
                                                          uint64_t seed, uint32_t t, int64_t Dp, int32_t N,
                                                          int32_t P, float sigma, int32_t tanh_out)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    MlpSmem& S = *reinterpret_cast<MlpSmem*>(smem_raw);
    const int32_t p = blockIdx.x, r = blockIdx.y;
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64, q = lane / 16, l16 = lane % 16;
    const uint64_t key = seed + (uint64_t)r;
    const uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    const float* __restrict__ mr = m + (int64_t)r * Dp;
    const int nbase = 32 * wave;  // this wave's batch columns

    // ---- layer 1 weights, all biases, layer 3 weights
    gen_weights(mr, k0, k1, (uint32_t)p, t, OFF_W1, MLP_H, MLP_IN, sigma, S.w[0], S.w[1], W1S);
    gen_weights(mr, k0, k1, (uint32_t)p, t, OFF_W3, MLP_OUT, MLP_H, sigma, S.w3[0], S.w3[1], W3S);
    gen_bias(mr, k0, k1, (uint32_t)p, t, OFF_B1, MLP_H, sigma, S.b1[0], S.b1[1]);
    gen_bias(mr, k0, k1, (uint32_t)p, t, OFF_B2, MLP_H, sigma, S.b2[0], S.b2[1]);
    gen_bias(mr, k0, k1, (uint32_t)p, t, OFF_B3, MLP_OUT, sigma, S.b3[0], S.b3[1]);

    // input B operands: X[n][32ks + 8q + i] for batch column n of tile nt
    bf16x8 xop[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
            xop[ks][nt] = *reinterpret_cast<const bf16x8*>(xb + (nbase + 16 * nt + l16) * MLP_IN + 32 * ks + 8 * q);
    __syncthreads();

    // ---- layer 1: H1^T (256 x 32) per member, kept as layer-2 B operands
    bf16x8 h1[2][8][2];
#pragma unroll
    for (int mem = 0; mem < 2; ++mem) {
        const __bf16* W = S.w[mem];
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            floatx4 c[2][2];
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) c[a][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8 A = *reinterpret_cast<const bf16x8*>(W + (32 * g + 16 * a + l16) * W1S + 32 * ks + 8 * q);
#pragma unroll
                    for (int nt = 0; nt < 2; ++nt)
                        c[a][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, xop[ks][nt], c[a][nt], 0, 0, 0);
                }
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) h1[mem][g][nt] = activate(c[0][nt], c[1][nt], S.b1[mem], 32 * g, q);
        }
    }
    __syncthreads();  // W1 tiles are reused for W2

    // ---- layer 2 in chunks of W2_ROWS output rows, each followed by its
    // share of layer 3 (the chunk's rows are layer 3's K range)
    floatx4 y[2][2];
#pragma unroll
    for (int mem = 0; mem < 2; ++mem)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) y[mem][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < MLP_H / W2_ROWS; ++c) {
        gen_weights(mr, k0, k1, (uint32_t)p, t, OFF_W2 + (int64_t)c * W2_ROWS * MLP_H, W2_ROWS, MLP_H, sigma, S.w[0],
                    S.w[1], W2S);
        __syncthreads();
#pragma unroll
        for (int mem = 0; mem < 2; ++mem) {
            const __bf16* W = S.w[mem];
            floatx4 acc[4][2];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int g = 0; g < 8; ++g)
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const __bf16* row = W + (16 * mt + l16) * W2S + 32 * g;
                    const bf16x8 A = cat(*reinterpret_cast<const bf16x4*>(row + 4 * q),
                                         *reinterpret_cast<const bf16x4*>(row + 16 + 4 * q));
#pragma unroll
                    for (int nt = 0; nt < 2; ++nt)
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, h1[mem][g][nt], acc[mt][nt], 0, 0, 0);
                }
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int r0 = W2_ROWS * c + 32 * h;  // layer-2 output rows = layer-3 K range
                const __bf16* w3row = S.w3[mem] + l16 * W3S + r0;
                const bf16x8 A3 = cat(*reinterpret_cast<const bf16x4*>(w3row + 4 * q),
                                      *reinterpret_cast<const bf16x4*>(w3row + 16 + 4 * q));
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    const bf16x8 hb = activate(acc[2 * h][nt], acc[2 * h + 1][nt], S.b2[mem], r0, q);
                    y[mem][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A3, hb, y[mem][nt], 0, 0, 0);
                }
            }
        }
        __syncthreads();  // before the next chunk overwrites the tiles
    }

    // ---- output layer bias, squared error against the teacher
    double se[2] = {0.0, 0.0};
#pragma unroll
    for (int mem = 0; mem < 2; ++mem)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            const int n = nbase + 16 * nt + l16;
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int o = 4 * q + i;
                float v = y[mem][nt][i] + S.b3[mem][o];
                if (tanh_out) v = tanh_fast(v);
                const float d = v - yt[n * MLP_OUT + o];
                s = fmaf(d, d, s);
            }
            se[mem] += (double)s;
        }
#pragma unroll
    for (int mem = 0; mem < 2; ++mem)
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) se[mem] += __shfl_xor(se[mem], off);
    if (lane == 0) {
        S.red[wave][0] = se[0];
        S.red[wave][1] = se[1];
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        double tot = 0.0;
        for (int w = 0; w < MLP_WAVES; ++w) tot += S.red[w][threadIdx.x];
        const double mse = tot / (double)(MLP_BATCH * MLP_OUT);
        fit[(int64_t)r * N + p + (threadIdx.x ? P : 0)] = (float)(-mse);
    }
}

// X_t: 256 x 64 normals from the EVAL stream (row 0, counter block = flat/4).
__global__ void k_mlp_inputs(float* __restrict__ xf, __bf16* __restrict__ xb, uint64_t seed, uint32_t t)
{
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= MLP_BATCH * MLP_IN / 4) return;
    float e[4];
    normals4(seed, (uint32_t)b, 0, t, DOM_EVAL, e);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        xf[4 * b + k] = e[k];
        xb[4 * b + k] = (__bf16)e[k];
    }
}

// Teacher forward in fp32: one workgroup per input row, one thread per
// hidden unit; Y_T[n][o].
__global__ __launch_bounds__(MLP_H) void k_mlp_teacher(const float* __restrict__ w, const float* __restrict__ xf,
                                                       float* __restrict__ yt, int32_t tanh_out)
{
    __shared__ float x[MLP_IN], h1[MLP_H], h2[MLP_H];
    const int n = blockIdx.x, o = threadIdx.x;
    if (o < MLP_IN) x[o] = xf[n * MLP_IN + o];
    __syncthreads();
    float a = 0.f;
    for (int k = 0; k < MLP_IN; ++k) a = fmaf(x[k], w[OFF_W1 + o * MLP_IN + k], a);
    h1[o] = tanhf(a + w[OFF_B1 + o]);
    __syncthreads();
    a = 0.f;
    for (int k = 0; k < MLP_H; ++k) a = fmaf(h1[k], w[OFF_W2 + o * MLP_H + k], a);
    h2[o] = tanhf(a + w[OFF_B2 + o]);
    __syncthreads();
    if (o < MLP_OUT) {
        a = 0.f;
        for (int k = 0; k < MLP_H; ++k) a = fmaf(h2[k], w[OFF_W3 + o * MLP_H + k], a);
        a += w[OFF_B3 + o];
        yt[n * MLP_OUT + o] = tanh_out ? tanhf(a) : a;
    }
}

}  // namespace

size_t mlp_scratch_bytes()
{
    return sizeof(float) * MLP_BATCH * MLP_IN + sizeof(__bf16) * MLP_BATCH * MLP_IN + sizeof(float) * MLP_BATCH * MLP_OUT;
}

size_t mlp_lds_bytes() { return sizeof(MlpSmem); }

hipError_t launch_eval_mlp(const Geometry& g, const es_config& c, uint32_t t, const float* m, const float* teacher,
                           void* scratch, float* fit, hipStream_t s)
{
    float* xf = static_cast<float*>(scratch);
    __bf16* xb = reinterpret_cast<__bf16*>(xf + MLP_BATCH * MLP_IN);
    float* yt = reinterpret_cast<float*>(xb + MLP_BATCH * MLP_IN);
    k_mlp_inputs<<<(MLP_BATCH * MLP_IN / 4 + 255) / 256, 256, 0, s>>>(xf, xb, c.seed, t);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_mlp_teacher<<<MLP_BATCH, MLP_H, 0, s>>>(teacher, xf, yt, c.mlp_tanh_out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    static bool lds_attr_set = false;  // more than 64 KB of LDS per workgroup
    if (!lds_attr_set) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_eval_mlp),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(MlpSmem));
        if (e != hipSuccess) return e;
        lds_attr_set = true;
    }
    k_eval_mlp<<<dim3((unsigned)g.P, (unsigned)g.R), MLP_THREADS, sizeof(MlpSmem), s>>>(
        m, xb, yt, fit, c.seed, t, g.Dp, g.N, g.P, c.sigma, c.mlp_tanh_out);
    return hipGetLastError();
}

}  // namespace esmi
