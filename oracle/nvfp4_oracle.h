/*
 * NVFP4 ScaleSweep oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Declarations of the plain CPU reference used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg.  Nothing in the product library includes this header or
 * links this code; the two implementations share no source, header or table.
 *
 * Conventions (host pointers, row-major):
 *   x            [rows, cols] of dtype 0 = binary32, 1 = bfloat16 (raw 16-bit patterns)
 *   block        micro-block length n in {16, 32, 64, 128}, blocks run along cols
 *   q            [rows, cols/2] bytes, element 2j in bits 3:0 of byte j, 2j+1 in bits 7:4,
 *                nibble = sign << 3 | E2M1 magnitude code
 *   scales       [rows, cols/block] E4M3 codes (0..126)
 *   tensor_scale the binary32 global scale S
 * Return codes match the numeric status codes of the product library's C interface.
 */
#ifndef NVFP4_ORACLE_H
#define NVFP4_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    REF_OK = 0,
    REF_ERR_NULL = -1,
    REF_ERR_SHAPE = -2,
    REF_ERR_BLOCK = -3,
    REF_ERR_DTYPE = -4,
    REF_ERR_ARG = -5,
    REF_ERR_NONFINITE = -9
};

enum { REF_ABSMAX = 0, REF_FOUR_OVER_SIX = 1, REF_SCALESWEEP_MSE = 2, REF_SCALESWEEP_WMSE = 3 };
enum { REF_WINDOW_OFFSETS = 0, REF_WINDOW_TIGHT = 1 };
enum { REF_SCALES_ROW_MAJOR = 0, REF_SCALES_SWIZZLED = 1 };

/* Number formats (Appendix A). */
double nvfp4_ref_eemm_value(int e, int m, int code);
double nvfp4_ref_e2m1(int k);
double nvfp4_ref_e4m3(int c);

/* Rounding (Notation section). */
int nvfp4_ref_round_fp4(double a, double s);
int nvfp4_ref_floor_fp8(double v_num, double v_den);
int nvfp4_ref_nearest_fp8(double v_num, double v_den);

/* Block objective and block-scale selection (Method section). */
double nvfp4_ref_block_loss(const float* y, const float* w, int n, double s);
int nvfp4_ref_window_lower(int method, int n);
int nvfp4_ref_window_upper(void);
int nvfp4_ref_block_sweep(const float* y, const float* w, int n, int L, int U,
                          int* c0, int* lo, int* hi, int* c_win, int* c_full, double* J127);
int nvfp4_ref_block_choose(int method, const float* y, const float* w, int n);

/* Window variants (Tables 1 and 2; the sweep-range study). */
int nvfp4_ref_window_tight(int method, int n, int b, int* lower, int* upper);
int nvfp4_ref_window_codes(int method, int n, int mode, int lo_off, int hi_off, int c0,
                           int* lo, int* hi);

/* Tensor-level calls. */
int nvfp4_ref_tensor_scale(const void* x, int dtype, int64_t count, float fp8_range, float* S);
int nvfp4_ref_quantize(int method, const void* x, int dtype, int64_t rows, int64_t cols,
                       int block, float fp8_range, float static_scale, const float* col_weight,
                       float* tensor_scale, uint8_t* q, uint8_t* scales);
int nvfp4_ref_quant_absmax(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                           float fp8_range, float static_scale, float* tensor_scale,
                           uint8_t* q, uint8_t* scales);
int nvfp4_ref_quant_four_over_six(const void* x, int dtype, int64_t rows, int64_t cols,
                                  int block, float fp8_range, float static_scale,
                                  const float* col_weight, float* tensor_scale, uint8_t* q,
                                  uint8_t* scales);
int nvfp4_ref_quant_scalesweep_mse(const void* x, int dtype, int64_t rows, int64_t cols,
                                   int block, float fp8_range, float static_scale,
                                   float* tensor_scale, uint8_t* q, uint8_t* scales);
int nvfp4_ref_quant_scalesweep_wmse(const void* x, int dtype, int64_t rows, int64_t cols,
                                    int block, float fp8_range, float static_scale,
                                    const float* col_weight, float* tensor_scale, uint8_t* q,
                                    uint8_t* scales);
int nvfp4_ref_quant_scalesweep_window(const void* x, int dtype, int64_t rows, int64_t cols,
                                      int block, const float* col_weight, int win_mode,
                                      int lo_off, int hi_off, float fp8_range,
                                      float static_scale, float* tensor_scale, uint8_t* q,
                                      uint8_t* scales);
/* Online quantization (implementation details; importance vectors of the WMSE section). */
int64_t nvfp4_ref_swizzled_offset(int64_t m, int64_t k, int64_t k16);
int64_t nvfp4_ref_scales_bytes(int64_t rows, int64_t cols, int block, int layout);
int nvfp4_ref_quant_online(int method, const void* x, int dtype, int64_t rows, int64_t cols,
                           int block, const float* importance, int64_t imp_groups,
                           int64_t imp_group_rows, float static_scale, int layout,
                           float* tensor_scale, uint8_t* q, uint8_t* scales);
/* SwiGLU producer of the fused online quantizer: e^x as specified in nvfp4_oracle.c, and
 * h = bf16(RN(silu(g) * u)) over bfloat16 bit patterns; non-finite inputs: REF_ERR_NONFINITE. */
float nvfp4_ref_swiglu_exp(float x);
int nvfp4_ref_swiglu(const uint16_t* gate, const uint16_t* up, int64_t count, uint16_t* h);
int nvfp4_ref_channel_sq_norms(const void* x, int dtype, int64_t rows, int64_t cols,
                               int64_t group_rows, int64_t groups, int64_t group_div,
                               int64_t rep_out, float* out);
/* GPTQ / LDLQ with fixed block scales (implementation details, GPTQ paragraph). */
int nvfp4_ref_ldlq_order(const double* H, int64_t n, int64_t* perm);
int nvfp4_ref_ldlq_factor(const double* H, int64_t n, double damp, const int64_t* perm,
                          double* U, double* D);
int nvfp4_ref_ldlq(const void* w, int dtype, int64_t rows, int64_t n, int block, const double* H,
                   const uint8_t* scales, float S, double damp, uint8_t* q);
int nvfp4_ref_dequant(const uint8_t* q, const uint8_t* scales, float tensor_scale,
                      int64_t rows, int64_t cols, int block, float* out);

/* Scale-quality references (appendix on the optimal FP32 block scale). */
double nvfp4_ref_continuous_opt(const float* y, const float* w, int n, double* s_opt);
int nvfp4_ref_fp8_quantized_opt(const float* y, const float* w, int n, double* loss);

/* Tensor error metrics (Notation section): out[0..3] = MSE, NMSE, WMSE, NWMSE. */
int nvfp4_ref_metrics(const void* x, int dtype, const float* xhat, int64_t rows, int64_t cols,
                      const float* col_weight, double* out4);

#ifdef __cplusplus
}
#endif

#endif
