// es_probe.hip -- issue-rate probe of the gfx950 instructions the library's
// kernels are built from (a measurement aid behind the roofline figures of
// the benchmark, not a step of the method; built into libesmi_probe.so).
//
// Each kernel runs CHAINS independent dependency chains of one instruction
// per lane, unrolled, on 2048 workgroups of 256 threads (eight waves per SIMD
// on 256 CUs), so the issue rate, not the latency, bounds it.  Wave
// instructions per launch = 2048 * 4 * iters * CHAINS; their rate relative to
// v_fma_f32's is the instruction's issue cost in full-rate slots.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "esmi_probe.h"

namespace {

constexpr int CHAINS = 8;
constexpr int PROBE_WG = 256;
constexpr int PROBE_GRID = 2048;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int OP>
__global__ __launch_bounds__(PROBE_WG) void k_issue(int64_t iters, uint32_t* __restrict__ sink)
{
    const uint32_t gid = blockIdx.x * PROBE_WG + threadIdx.x;
    uint32_t sum = 0;
    if constexpr (OP == ES_PROBE_MFMA_BF16) {
        floatx4 acc[CHAINS];
        bf16x8 a, b;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            a[k] = (__bf16)(1.0f + (float)(gid & 7) * 0.125f);
            b[k] = (__bf16)(0.5f + (float)k * 0.0625f);
        }
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) acc[c] = floatx4{(float)c, 0.f, 0.f, 0.f};
        for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
            for (int c = 0; c < CHAINS; ++c)
                asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc[c]) : "v"(a), "v"(b));
        }
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) sum += __float_as_uint(acc[c][0] + acc[c][3]);
    } else if constexpr (OP == ES_PROBE_FMA_F64 || OP == ES_PROBE_ADD_F64) {
        double x[CHAINS];
        const double p = 1.0000001, q = 1e-9;
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) x[c] = (double)(gid + c);
        for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
            for (int c = 0; c < CHAINS; ++c) {
                if constexpr (OP == ES_PROBE_FMA_F64) asm volatile("v_fma_f64 %0, %0, %1, 0.5" : "+v"(x[c]) : "s"(p));
                else asm volatile("v_add_f64 %0, %0, %1" : "+v"(x[c]) : "s"(q));
            }
        }
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) sum += (uint32_t)__double_as_longlong(x[c]);
    } else if constexpr (OP == ES_PROBE_MAD_U64_U32) {
        uint32_t u[CHAINS];
        const uint32_t mul = 0xD2511F53u;
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) u[c] = gid * 8u + (uint32_t)c;
        for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
            for (int c = 0; c < CHAINS; ++c) {
                uint64_t r;
                asm volatile("v_mad_u64_u32 %0, vcc, %1, %2, 0" : "=v"(r) : "v"(u[c]), "s"(mul) : "vcc");
                u[c] = (uint32_t)r;
            }
        }
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) sum += u[c];
    } else {
        float x[CHAINS];
        const float p = 1.0000001f, q = 1e-7f;
        const uint32_t kk = 0x9E3779B9u;
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) x[c] = 0.5f + (float)((gid + c) & 255) * 0.001f;
        for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
            for (int c = 0; c < CHAINS; ++c) {
                // one VGPR source per instruction (the others a scalar register or
                // an inline constant), as in most instructions of the hot kernels;
                // ES_PROBE_FMA_F32_VVV reads three VGPRs
                if constexpr (OP == ES_PROBE_FMA_F32) asm volatile("v_fma_f32 %0, %0, %1, 0.5" : "+v"(x[c]) : "s"(p));
                else if constexpr (OP == ES_PROBE_FMA_F32_VVV) asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x[c]) : "v"(p), "v"(q));
                else if constexpr (OP == ES_PROBE_MUL_F32) asm volatile("v_mul_f32_e32 %0, %1, %0" : "+v"(x[c]) : "s"(p));
                else if constexpr (OP == ES_PROBE_XOR_B32) asm volatile("v_xor_b32_e32 %0, %1, %0" : "+v"(x[c]) : "s"(kk));
                else if constexpr (OP == ES_PROBE_BITOP3) asm volatile("v_bitop3_b32 %0, %0, %1, %0 bitop3:0x96" : "+v"(x[c]) : "s"(kk));
                else if constexpr (OP == ES_PROBE_CVT_F32_U32) asm volatile("v_cvt_f32_u32_e32 %0, %0" : "+v"(x[c]));
                else if constexpr (OP == ES_PROBE_CVT_PK_BF16) asm volatile("v_cvt_pk_bf16_f32 %0, %0, %1" : "+v"(x[c]) : "s"(p));
                else if constexpr (OP == ES_PROBE_LOG) asm volatile("v_log_f32_e32 %0, %0" : "+v"(x[c]));
                else if constexpr (OP == ES_PROBE_EXP) asm volatile("v_exp_f32_e32 %0, %0" : "+v"(x[c]));
                else if constexpr (OP == ES_PROBE_RCP) asm volatile("v_rcp_f32_e32 %0, %0" : "+v"(x[c]));
                else if constexpr (OP == ES_PROBE_SQRT) asm volatile("v_sqrt_f32_e32 %0, %0" : "+v"(x[c]));
                else if constexpr (OP == ES_PROBE_SIN) asm volatile("v_sin_f32_e32 %0, %0" : "+v"(x[c]));
                else asm volatile("v_cos_f32_e32 %0, %0" : "+v"(x[c]));
            }
        }
#pragma unroll
        for (int c = 0; c < CHAINS; ++c) sum += __float_as_uint(x[c]);
    }
    sink[gid] = sum;
}

template <int OP>
hipError_t launch_issue(int64_t iters, uint32_t* sink, hipStream_t s)
{
    k_issue<OP><<<PROBE_GRID, PROBE_WG, 0, s>>>(iters, sink);
    return hipGetLastError();
}

}  // namespace

extern "C" {

int64_t es_probe_threads(void) { return (int64_t)PROBE_GRID * PROBE_WG; }

int32_t es_probe_chains(void) { return CHAINS; }

int32_t es_probe_issue(int32_t op, int64_t iters, uint32_t* sink, void* hip_stream)
{
    if (!sink || iters < 1) return (int32_t)hipErrorInvalidValue;
    hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    switch (op) {
    case ES_PROBE_FMA_F32: return (int32_t)launch_issue<ES_PROBE_FMA_F32>(iters, sink, s);
    case ES_PROBE_BITOP3: return (int32_t)launch_issue<ES_PROBE_BITOP3>(iters, sink, s);
    case ES_PROBE_MAD_U64_U32: return (int32_t)launch_issue<ES_PROBE_MAD_U64_U32>(iters, sink, s);
    case ES_PROBE_CVT_F32_U32: return (int32_t)launch_issue<ES_PROBE_CVT_F32_U32>(iters, sink, s);
    case ES_PROBE_CVT_PK_BF16: return (int32_t)launch_issue<ES_PROBE_CVT_PK_BF16>(iters, sink, s);
    case ES_PROBE_LOG: return (int32_t)launch_issue<ES_PROBE_LOG>(iters, sink, s);
    case ES_PROBE_EXP: return (int32_t)launch_issue<ES_PROBE_EXP>(iters, sink, s);
    case ES_PROBE_RCP: return (int32_t)launch_issue<ES_PROBE_RCP>(iters, sink, s);
    case ES_PROBE_SQRT: return (int32_t)launch_issue<ES_PROBE_SQRT>(iters, sink, s);
    case ES_PROBE_SIN: return (int32_t)launch_issue<ES_PROBE_SIN>(iters, sink, s);
    case ES_PROBE_COS: return (int32_t)launch_issue<ES_PROBE_COS>(iters, sink, s);
    case ES_PROBE_FMA_F64: return (int32_t)launch_issue<ES_PROBE_FMA_F64>(iters, sink, s);
    case ES_PROBE_ADD_F64: return (int32_t)launch_issue<ES_PROBE_ADD_F64>(iters, sink, s);
    case ES_PROBE_MFMA_BF16: return (int32_t)launch_issue<ES_PROBE_MFMA_BF16>(iters, sink, s);
    case ES_PROBE_MUL_F32: return (int32_t)launch_issue<ES_PROBE_MUL_F32>(iters, sink, s);
    case ES_PROBE_XOR_B32: return (int32_t)launch_issue<ES_PROBE_XOR_B32>(iters, sink, s);
    case ES_PROBE_FMA_F32_VVV: return (int32_t)launch_issue<ES_PROBE_FMA_F32_VVV>(iters, sink, s);
    }
    return (int32_t)hipErrorInvalidValue;
}

}  // extern "C"
