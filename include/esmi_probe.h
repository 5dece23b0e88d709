/*
 * esmi_probe.h -- issue-rate probe of gfx950 instructions (libesmi_probe.so).
 *
 * A measurement aid, not an operation of the paper and not part of the
 * generation's path: the benchmark's roofline figures count the hot kernels'
 * work in full-rate VALU slots (v_fma_f32 = 1), and this probe measures the
 * slot cost of each instruction those kernels issue.  Each launch runs
 * es_probe_chains() independent chains of one instruction per lane, `iters`
 * times, on es_probe_threads() threads (eight waves per SIMD on 256 CUs):
 * es_probe_threads() / 64 * iters * es_probe_chains() wave instructions.
 * The caller times the launch (events on hip_stream) and owns `sink`, a
 * device uint32 array of es_probe_threads() entries that receives one value
 * per thread.  Returns a hipError_t value (0 = success); an unknown op or
 * iters < 1 gives hipErrorInvalidValue and launches nothing.
 */
#ifndef ESMI_PROBE_H
#define ESMI_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ES_PROBE_FMA_F32 = 0,     /* v_fma_f32                          */
    ES_PROBE_BITOP3 = 1,      /* v_bitop3_b32 (three-input xor)     */
    ES_PROBE_MAD_U64_U32 = 2, /* v_mad_u64_u32 (32x32 -> 64 product) */
    ES_PROBE_CVT_F32_U32 = 3, /* v_cvt_f32_u32                      */
    ES_PROBE_CVT_PK_BF16 = 4, /* v_cvt_pk_bf16_f32                  */
    ES_PROBE_LOG = 5,         /* v_log_f32                          */
    ES_PROBE_EXP = 6,         /* v_exp_f32                          */
    ES_PROBE_RCP = 7,         /* v_rcp_f32                          */
    ES_PROBE_SQRT = 8,        /* v_sqrt_f32                         */
    ES_PROBE_SIN = 9,         /* v_sin_f32                          */
    ES_PROBE_COS = 10,        /* v_cos_f32                          */
    ES_PROBE_FMA_F64 = 11,    /* v_fma_f64                          */
    ES_PROBE_ADD_F64 = 12,    /* v_add_f64                          */
    ES_PROBE_MFMA_BF16 = 13,  /* v_mfma_f32_16x16x32_bf16           */
    ES_PROBE_MUL_F32 = 14,    /* v_mul_f32                          */
    ES_PROBE_XOR_B32 = 15,    /* v_xor_b32                          */
    ES_PROBE_FMA_F32_VVV = 16, /* v_fma_f32 with three VGPR sources */
    ES_PROBE_NUM_OPS = 17
};

int32_t es_probe_issue(int32_t op, int64_t iters, uint32_t* sink, void* hip_stream);
int64_t es_probe_threads(void);
int32_t es_probe_chains(void);

#ifdef __cplusplus
}
#endif
#endif /* ESMI_PROBE_H */
