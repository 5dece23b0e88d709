// es_teacher.hpp -- layout of the 64-256-256-16 MLP's flat parameter vector
// and the fp32 teacher forward of one input row.  Used by the teacher kernel
// and by the gradient kernel, whose launch carries the next generation's
// teacher rows in workgroups of their own (Sec. 3.2 network definitions; the
// teacher-student fitness is this library's neuroevolution workload).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "es_device.hpp"

namespace esmi {

// Per layer the [out][in] row-major weights, then the bias: W1 [256][64],
// b1 [256], W2 [256][256], b2 [256], W3 [16][256], b3 [16].
constexpr int MLP_IN = 64, MLP_H = 256, MLP_OUT = 16, MLP_BATCH = 256;
constexpr int64_t OFF_W1 = 0, OFF_B1 = 16384, OFF_W2 = 16640, OFF_B2 = 82176, OFF_W3 = 82432, OFF_B3 = 86528;

// The teacher's summation order: the inner sums of layers 1 and 2 are split
// into TEACHER_SLICES contiguous K ranges (layer 3 into L3_SLICES ranges of
// 4) whose fp32 partials are added in slice order.
constexpr int TEACHER_SLICES = 4;
constexpr int TEACHER_THREADS = MLP_H;                     // threads that compute (one per hidden unit)
constexpr int L3_SLICES = TEACHER_SLICES * MLP_H / MLP_OUT;  // layer 3: 64 K ranges of 4

// One generation's teacher work: X_t and Y_T of generation t.
struct TeacherJob {
    const float* w;   // teacher, flat [86544]; null: no job
    const float* wt;  // its weight matrices transposed ([in][out])
    float* xf;        // X_t fp32 [256][64]
    __bf16* xb;       // X_t bf16 [256][64]
    float* yt;        // Y_T [256][16]
    uint64_t seed;    // base seed (EVAL stream)
    uint32_t t;
    int32_t tanh_out;
};

// Slice partials of hidden unit o for one layer: TEACHER_SLICES fma chains
// over their K ranges in increasing k, run side by side (independent loads
// in flight), then added in slice order.
template <int K>
__device__ __forceinline__ float teacher_unit(const float* __restrict__ in, const float* __restrict__ wt, int o)
{
    constexpr int KS = K / TEACHER_SLICES;
    float a[TEACHER_SLICES];
#pragma unroll
    for (int s = 0; s < TEACHER_SLICES; ++s) a[s] = 0.f;
#pragma unroll 8
    for (int k = 0; k < KS; ++k)
#pragma unroll
        for (int s = 0; s < TEACHER_SLICES; ++s) a[s] = fmaf(in[s * KS + k], wt[(s * KS + k) * MLP_H + o], a[s]);
    float z = a[0];
#pragma unroll
    for (int s = 1; s < TEACHER_SLICES; ++s) z += a[s];
    return z;
}

// Input row n of X_t (64 normals from the EVAL stream, counter block = flat
// index / 4) in fp32 and bf16, and the teacher forward on it -> Y_T[n][:].
// Needs blockDim.x >= TEACHER_THREADS; the results do not depend on it.
__device__ __forceinline__ void teacher_row(const TeacherJob& j, int n)
{
    __shared__ float x[MLP_IN], h1[MLP_H], h2[MLP_H], part[L3_SLICES * MLP_OUT];
    const int tid = threadIdx.x;
    if (tid < MLP_IN / 4) {
        float e[4];
        normals4(j.seed, (uint32_t)(n * (MLP_IN / 4) + tid), 0, j.t, DOM_EVAL, e);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            x[4 * tid + k] = e[k];
            j.xf[n * MLP_IN + 4 * tid + k] = e[k];
            j.xb[n * MLP_IN + 4 * tid + k] = (__bf16)e[k];
        }
    }
    __syncthreads();
    if (tid < TEACHER_THREADS) h1[tid] = tanhf(teacher_unit<MLP_IN>(x, j.wt + OFF_W1, tid) + j.w[OFF_B1 + tid]);
    __syncthreads();
    if (tid < TEACHER_THREADS) h2[tid] = tanhf(teacher_unit<MLP_H>(h1, j.wt + OFF_W2, tid) + j.w[OFF_B2 + tid]);
    __syncthreads();
    // layer 3: item i = (K range i / 16, output i % 16), four per thread
    constexpr int K3 = MLP_H / L3_SLICES, IPT = L3_SLICES * MLP_OUT / TEACHER_THREADS;
    if (tid < TEACHER_THREADS) {
        float a[IPT];
#pragma unroll
        for (int q = 0; q < IPT; ++q) a[q] = 0.f;
#pragma unroll
        for (int k = 0; k < K3; ++k)
#pragma unroll
            for (int q = 0; q < IPT; ++q) {
                const int i = tid + q * TEACHER_THREADS, kk = (i / MLP_OUT) * K3 + k;
                a[q] = fmaf(h2[kk], j.wt[OFF_W3 + kk * MLP_OUT + i % MLP_OUT], a[q]);
            }
#pragma unroll
        for (int q = 0; q < IPT; ++q) part[tid + q * TEACHER_THREADS] = a[q];
    }
    __syncthreads();
    if (tid < MLP_OUT) {
        float z = part[tid];
        for (int s = 1; s < L3_SLICES; ++s) z += part[s * MLP_OUT + tid];
        z += j.w[OFF_B3 + tid];
        j.yt[n * MLP_OUT + tid] = j.tanh_out ? tanhf(z) : z;
    }
}

}  // namespace esmi
