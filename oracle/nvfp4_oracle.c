/*
 * NVFP4 ScaleSweep oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, single-threaded, deliberately slow CPU implementation of the ScaleSweep hot path
 * (Lin & Wan, "ScaleSweep: Accurate NVFP4 Post-Training Quantization of LLMs via Block Scale
 * Initialization", arXiv 2606.07618), written from the paper.  Only the tests, the smoke check
 * and the benchmark's CPU-baseline leg load it; the product library neither links nor calls
 * it, and the two share no code, header, table or generator.
 *
 * Precision.  The global scale S and the normalized values y = x / S are IEEE binary32 (C
 * float division, round to nearest even).  Every objective value is computed in binary64.
 * Build with -O2 -ffp-contract=off and without fast-math, so that no multiply-add is fused.
 *
 * Readings of points the paper leaves open are marked "reading:" where they are used; the
 * design document lists all of them.  Every function here is pinned by the CPU test-suite
 * (paper values, closed forms, invariants, brute force); none is "parity unpinned".
 */
#include "nvfp4_oracle.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define E2M1_CODES 8        /* non-negative E2M1 magnitudes, codes 0..7 */
#define E4M3_MAX_CODE 126   /* codes 1..126 are the 126 positive finite E4M3 values */
#define MAX_BLOCK 128

/* ------------------------------------------------------------------------------------- */
/* Number formats: Appendix A (floating-point representation).                            */
/* ------------------------------------------------------------------------------------- */

/* Value of the non-negative EeMm bit pattern code = a * 2^m + b (sign c = 0), with bias
 * B = 2^(e-1) - 1:  a != 0 -> 2^(a-B) (1 + b / 2^m),  a == 0 -> 2^(1-B) b / 2^m.
 * For a positive value the bit-pattern integer I(v) of Appendix A is the code itself. */
double nvfp4_ref_eemm_value(int e, int m, int code)
{
    int bias = (1 << (e - 1)) - 1;
    int a = code >> m;
    int b = code & ((1 << m) - 1);
    double mant = (double)(1 << m);
    if (a != 0) return ldexp(1.0 + (double)b / mant, a - bias);
    return ldexp((double)b / mant, 1 - bias);
}

static double g_e2m1[E2M1_CODES];
static double g_e4m3[E4M3_MAX_CODE + 1];
static int g_tables_ready = 0;

static void tables_init(void)
{
    if (g_tables_ready) return;
    for (int k = 0; k < E2M1_CODES; ++k) g_e2m1[k] = nvfp4_ref_eemm_value(2, 1, k);
    for (int c = 0; c <= E4M3_MAX_CODE; ++c) g_e4m3[c] = nvfp4_ref_eemm_value(4, 3, c);
    g_tables_ready = 1;
}

/* FP4 E2M1 magnitude of code k in 0..7: {0, 0.5, 1, 1.5, 2, 3, 4, 6} (NVFP4 section). */
double nvfp4_ref_e2m1(int k)
{
    tables_init();
    return (k >= 0 && k < E2M1_CODES) ? g_e2m1[k] : NAN;
}

/* FP8 E4M3 value of code c in 0..126; code 127 (exponent 15, mantissa 7) is NaN and is not a
 * candidate: the paper counts 126 positive finite scales, the largest being 448. */
double nvfp4_ref_e4m3(int c)
{
    tables_init();
    return (c >= 0 && c <= E4M3_MAX_CODE) ? g_e4m3[c] : NAN;
}

/* ------------------------------------------------------------------------------------- */
/* Rounding: Notation section (round to nearest / down onto a grid).                      */
/* ------------------------------------------------------------------------------------- */

/* Nearest point of the scaled grid FP4(s) = { s * v : v in G_FP4 } to a >= 0, returned as the
 * E2M1 magnitude code.  a lies above the midpoint between codes k and k+1 exactly when the
 * nearest point is past k.  reading: an exact midpoint goes to the even code (ties-to-even,
 * as IEEE and OCP conversions do).  Each midpoint (v_k + v_{k+1}) / 2 * s has at most 7
 * significant bits, so every comparison is exact.  FP4(0) = {0}. */
int nvfp4_ref_round_fp4(double a, double s)
{
    if (s == 0.0) return 0;
    int k = 0;
    while (k < E2M1_CODES - 1) {
        double mid = 0.5 * (nvfp4_ref_e2m1(k) + nvfp4_ref_e2m1(k + 1)) * s;
        if (a > mid || (a == mid && ((k + 1) % 2) == 0))
            k++;
        else
            break;
    }
    return k;
}

/* Round down onto the FP8 grid, of the ratio v_num / v_den (v_den in {4, 6}):
 * the largest code c in 0..126 with v_den * E4M3(c) <= v_num.  The products are exact. */
int nvfp4_ref_floor_fp8(double v_num, double v_den)
{
    int c = E4M3_MAX_CODE;
    while (c > 0 && v_den * nvfp4_ref_e4m3(c) > v_num) c--;
    return c;
}

/* Round to nearest onto the FP8 grid, of v_num / v_den.  reading: ties go to the even code
 * and values beyond 448 saturate to 448 (code 126); the result may be code 0. */
int nvfp4_ref_nearest_fp8(double v_num, double v_den)
{
    int c = nvfp4_ref_floor_fp8(v_num, v_den);
    if (c < E4M3_MAX_CODE) {
        double mid = 0.5 * v_den * (nvfp4_ref_e4m3(c) + nvfp4_ref_e4m3(c + 1));
        if (v_num > mid || (v_num == mid && ((c + 1) % 2) == 0)) c++;
    }
    return c;
}

/* ------------------------------------------------------------------------------------- */
/* Objective: Eq. (weighted_quantization_loss) and Eq. (mse_quantization_loss).          */
/* ------------------------------------------------------------------------------------- */

/* L(s; y, w) = sum_i w_i (y_i - round_FP4(s)(y_i))^2 over one micro-block of n normalized
 * values (w == NULL: all w_i = 1).  The grid is symmetric, so the error of y_i equals that of
 * |y_i|.  Terms are added in order i = 0 .. n-1 in binary64; the difference |y_i| - g s is
 * exact in binary64 for every finite binary32 y_i the dynamic global scale can produce. */
double nvfp4_ref_block_loss(const float* y, const float* w, int n, double s)
{
    double J = 0.0;
    for (int i = 0; i < n; ++i) {
        double a = fabs((double)y[i]);
        double g = nvfp4_ref_e2m1(nvfp4_ref_round_fp4(a, s));
        double e = a - g * s;
        double t = e * e;
        if (w) t = (double)w[i] * t;
        J = J + t;
    }
    return J;
}

/* ------------------------------------------------------------------------------------- */
/* Block scale selection: Method section (ScaleSweep, block scale bounds).               */
/* ------------------------------------------------------------------------------------- */

/* Offset of the lowest swept code below I(s_base^FP8).
 *   MSE,  n = 16: 3 (Lemma 3: the argmin is >= 4/5 s_base^FP8, i.e. 3 codes down).
 *   WMSE, n = 16: 8 (the empirical s_base / 2 bound).
 *   reading for n > 16: MSE 5 / 7 / 11 for n = 32 / 64 / 128, from the r <= 3/4 step of the
 *   proof of Lemma 3 with n - 1 non-maximal coordinates; WMSE max(8, MSE offset).
 * AbsMax and 4/6 do not sweep (returns 0). */
int nvfp4_ref_window_lower(int method, int n)
{
    int mse = (n == 16) ? 3 : (n == 32) ? 5 : (n == 64) ? 7 : (n == 128) ? 11 : -1;
    if (mse < 0) return -1;
    if (method == REF_SCALESWEEP_MSE) return mse;
    if (method == REF_SCALESWEEP_WMSE) return mse > 8 ? mse : 8;
    return 0;
}

/* Offset of the highest swept code above I(s_base^FP8): 7, from Lemma 1 (no scale above
 * 12/7 s_base can beat its half) and Lemma 2 with alpha = 12/7 (Table 1). */
int nvfp4_ref_window_upper(void) { return 7; }

static double block_ymax(const float* y, int n)
{
    double m = 0.0;
    for (int i = 0; i < n; ++i) {
        double a = fabs((double)y[i]);
        if (a > m) m = a;
    }
    return m;
}

/* ScaleSweep on one block: s_base = max|y| / 6, s_base^FP8 = round-down of s_base onto the
 * FP8 grid, c0 = I(s_base^FP8); sweep codes [max(1, c0-L), min(126, c0+U)] and keep the
 * argmin of L (reading: the smallest code wins a tie).  Also sweeps all 126 positive codes
 * (the exhaustive search the window is meant to reproduce).  J127, if given, receives L at
 * every code 0..126 (code 0 is the zero scale, whose loss is sum w y^2). */
int nvfp4_ref_block_sweep(const float* y, const float* w, int n, int L, int U,
                          int* c0_out, int* lo_out, int* hi_out, int* c_win, int* c_full,
                          double* J127)
{
    double ymax = block_ymax(y, n);
    int c0 = nvfp4_ref_floor_fp8(ymax, 6.0);
    int lo = c0 - L < 1 ? 1 : c0 - L;
    int hi = c0 + U > E4M3_MAX_CODE ? E4M3_MAX_CODE : c0 + U;
    int best_w = -1, best_f = -1;
    double jw = 0.0, jf = 0.0;
    for (int c = 0; c <= E4M3_MAX_CODE; ++c) {
        double J = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(c));
        if (J127) J127[c] = J;
        if (c == 0) continue;
        if (best_f < 0 || J < jf) { best_f = c; jf = J; }
        if (c >= lo && c <= hi && (best_w < 0 || J < jw)) { best_w = c; jw = J; }
    }
    if (c0_out) *c0_out = c0;
    if (lo_out) *lo_out = lo;
    if (hi_out) *hi_out = hi;
    if (c_win) *c_win = best_w;
    if (c_full) *c_full = best_f;
    return REF_OK;
}

/* Argmin of L over the codes lo..hi, the smallest code on a tie (reading). */
static int argmin_codes(const float* y, const float* w, int n, int lo, int hi)
{
    int best = lo;
    double jb = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(lo));
    for (int c = lo + 1; c <= hi; ++c) {
        double J = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(c));
        if (J < jb) { best = c; jb = J; }
    }
    return best;
}

/* The scale code a method picks for one block of normalized values.
 *   AbsMax (NVFP4 section): s = round-to-nearest-FP8(max|y| / 6).
 *   4/6 (Introduction; Related Work): also try round-to-nearest-FP8(max|y| / 4), which maps the
 *     block maximum to 4 instead of 6, and keep it only if its loss is strictly lower
 *     (reading: loss as in the call -- weighted when weights are given -- ties keep /6).
 *   ScaleSweep (Method section): argmin of L over the window only. */
int nvfp4_ref_block_choose(int method, const float* y, const float* w, int n)
{
    double ymax = block_ymax(y, n);
    if (method == REF_ABSMAX) return nvfp4_ref_nearest_fp8(ymax, 6.0);
    if (method == REF_FOUR_OVER_SIX) {
        int c6 = nvfp4_ref_nearest_fp8(ymax, 6.0);
        int c4 = nvfp4_ref_nearest_fp8(ymax, 4.0);
        double j6 = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(c6));
        double j4 = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(c4));
        return (j4 < j6) ? c4 : c6;
    }
    int L = nvfp4_ref_window_lower(method, n);
    int U = nvfp4_ref_window_upper();
    int c0 = nvfp4_ref_floor_fp8(ymax, 6.0);
    int lo = c0 - L < 1 ? 1 : c0 - L;
    int hi = c0 + U > E4M3_MAX_CODE ? E4M3_MAX_CODE : c0 + U;
    const float* wm = (method == REF_SCALESWEEP_WMSE) ? w : NULL;
    return argmin_codes(y, wm, n, lo, hi);
}

/* ------------------------------------------------------------------------------------- */
/* Window variants (Block Scale Upper Bound / Lower Bound paragraphs; the sweep-range      */
/* study of the Experiment section).                                                      */
/* ------------------------------------------------------------------------------------- */

/* Per-mantissa offsets for a base code whose mantissa field is b (Tables 1 and 2), derived
 * on a normal base code (exponent field 7, s_base^FP8 = 1 + b/8) from the bounds' meaning:
 *   upper: I of the largest round-down of (12/7) s_base, over s_base from s_base^FP8 up to the
 *          next FP8 value (closed at the top, as the printed sup column is), minus I(s_base^FP8)
 *          -- Lemma 1 with Lemma 2 at alpha = 12/7; it holds for either objective and any n;
 *   lower: MSE objective with n = 16: I(s_base^FP8) minus I of the round-up of
 *          (4/5) s_base^FP8 (Lemma 3); otherwise the method's standard lower offset. */
int nvfp4_ref_window_tight(int method, int n, int b, int* lower, int* upper)
{
    if (!lower || !upper) return REF_ERR_NULL;
    if (b < 0 || b > 7) return REF_ERR_ARG;
    if (method != REF_SCALESWEEP_MSE && method != REF_SCALESWEEP_WMSE) return REF_ERR_ARG;
    int std_lower = nvfp4_ref_window_lower(method, n);
    if (std_lower < 0) return REF_ERR_BLOCK;
    int c0 = 8 * 7 + b;
    double s0 = nvfp4_ref_e4m3(c0);
    double s1 = nvfp4_ref_e4m3(c0 + 1);
    *upper = nvfp4_ref_floor_fp8(12.0 * s1, 7.0) - c0;
    if (method == REF_SCALESWEEP_MSE && n == 16) {
        int c_inf = c0;
        while (c_inf > 1 && 5.0 * nvfp4_ref_e4m3(c_inf - 1) >= 4.0 * s0) --c_inf;
        *lower = c0 - c_inf;
    } else {
        *lower = std_lower;
    }
    return REF_OK;
}

/* The codes one block sweeps under a window variant, from its base code c0 = I(s_base^FP8):
 *   mode REF_WINDOW_OFFSETS: offsets [lo_off, hi_off] around c0 (the [l, r] of the sweep-range
 *     study; the standard windows are [-3, 7] and [-8, 7] at n = 16);
 *   mode REF_WINDOW_TIGHT: the per-mantissa offsets of nvfp4_ref_window_tight for b = c0 & 7.
 * reading: each end is clamped into the positive codes 1..126, so a window that lies wholly
 * outside them sweeps the nearest end code alone; [-126, 126] is the exhaustive sweep. */
int nvfp4_ref_window_codes(int method, int n, int mode, int lo_off, int hi_off, int c0,
                           int* lo, int* hi)
{
    if (!lo || !hi) return REF_ERR_NULL;
    if (mode == REF_WINDOW_TIGHT) {
        int rc = nvfp4_ref_window_tight(method, n, c0 & 7, &lo_off, &hi_off);
        if (rc != REF_OK) return rc;
        lo_off = -lo_off;
    } else if (mode != REF_WINDOW_OFFSETS || lo_off < -E4M3_MAX_CODE || hi_off > E4M3_MAX_CODE ||
               lo_off > hi_off) {
        return REF_ERR_ARG;
    }
    int l = c0 + lo_off, h = c0 + hi_off;
    *lo = l < 1 ? 1 : l > E4M3_MAX_CODE ? E4M3_MAX_CODE : l;
    *hi = h < 1 ? 1 : h > E4M3_MAX_CODE ? E4M3_MAX_CODE : h;
    return REF_OK;
}

/* ------------------------------------------------------------------------------------- */
/* Tensor level: global scale (NVFP4 section; Global Scale Selection) and packing.        */
/* ------------------------------------------------------------------------------------- */

static float load_elem(const void* x, int dtype, int64_t i)
{
    if (dtype == 0) return ((const float*)x)[i];
    uint32_t bits = (uint32_t)((const uint16_t*)x)[i] << 16;   /* bfloat16 -> binary32, exact */
    float f;
    memcpy(&f, &bits, sizeof f);
    return f;
}

static int valid_block(int block)
{
    return block == 16 || block == 32 || block == 64 || block == 128;
}

static int valid_range(float d) { return isfinite(d) && d > 0.0f && d <= 448.0f; }

/* S = amax / (6 D) in binary32 (D = 448 for AbsMax in the NVFP4 section, D = 256 for the
 * global scale selection of ScaleSweep and 4/6).  reading: the denominator 6 D is formed in
 * binary32 first; an all-zero tensor gets S = 1; a quotient that underflows to zero is raised
 * to the smallest positive binary32 value.  A non-finite element is an error. */
int nvfp4_ref_tensor_scale(const void* x, int dtype, int64_t count, float fp8_range, float* S)
{
    if (!S || (count > 0 && !x)) return REF_ERR_NULL;
    if (dtype != 0 && dtype != 1) return REF_ERR_DTYPE;
    if (count < 0) return REF_ERR_SHAPE;
    if (!valid_range(fp8_range)) return REF_ERR_ARG;
    float amax = 0.0f;
    for (int64_t i = 0; i < count; ++i) {
        float v = load_elem(x, dtype, i);
        if (!isfinite(v)) return REF_ERR_NONFINITE;
        float a = fabsf(v);
        if (a > amax) amax = a;
    }
    if (amax == 0.0f) {
        *S = 1.0f;
        return REF_OK;
    }
    float denom = 6.0f * fp8_range;
    float s = amax / denom;
    if (s == 0.0f) s = FLT_TRUE_MIN;
    *S = s;
    return REF_OK;
}

/* win_mode < 0: the method's own block-scale rule; otherwise ScaleSweep over the window
 * variant (win_mode, lo_off, hi_off) of nvfp4_ref_window_codes. */
static int quantize_impl(int method, int win_mode, int lo_off, int hi_off, const void* x,
                         int dtype, int64_t rows, int64_t cols, int block, float fp8_range,
                         float static_scale, const float* col_weight, float* tensor_scale,
                         uint8_t* q, uint8_t* scales)
{
    if (method < REF_ABSMAX || method > REF_SCALESWEEP_WMSE) return REF_ERR_ARG;
    if (!tensor_scale) return REF_ERR_NULL;
    if (dtype != 0 && dtype != 1) return REF_ERR_DTYPE;
    if (!valid_block(block)) return REF_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return REF_ERR_SHAPE;
    if (!valid_range(fp8_range)) return REF_ERR_ARG;
    if (!isfinite(static_scale) || static_scale < 0.0f) return REF_ERR_ARG;
    if (method == REF_SCALESWEEP_WMSE && !col_weight) return REF_ERR_NULL;
    if (win_mode >= 0) {
        int lo, hi;
        int rc = nvfp4_ref_window_codes(method, block, win_mode, lo_off, hi_off, 0, &lo, &hi);
        if (rc != REF_OK) return rc;
    }
    int64_t count = rows * cols;
    if (count > 0 && (!x || !q || !scales)) return REF_ERR_NULL;
    const float* w = (method == REF_SCALESWEEP_WMSE || method == REF_FOUR_OVER_SIX)
                         ? col_weight : NULL;
    if (w) {
        for (int64_t j = 0; j < cols; ++j)
            if (!isfinite(w[j]) || w[j] < 0.0f) return REF_ERR_ARG;
    }

    float S = static_scale;
    if (S == 0.0f) {
        int rc = nvfp4_ref_tensor_scale(x, dtype, count, fp8_range, &S);
        if (rc != REF_OK) return rc;
    }

    int64_t nb_row = cols / block;
    float y[MAX_BLOCK];
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t kb = 0; kb < nb_row; ++kb) {
            int64_t base = r * cols + kb * block;
            for (int i = 0; i < block; ++i) {
                float v = load_elem(x, dtype, base + i);
                y[i] = v / S;                        /* y = RN32(x / S) */
                if (!isfinite(v) || !isfinite(y[i])) return REF_ERR_NONFINITE;
            }
            const float* wb = w ? w + kb * block : NULL;
            int c;
            if (win_mode < 0) {
                c = nvfp4_ref_block_choose(method, y, wb, block);
            } else {
                int lo, hi;
                int c0 = nvfp4_ref_floor_fp8(block_ymax(y, block), 6.0);
                nvfp4_ref_window_codes(method, block, win_mode, lo_off, hi_off, c0, &lo, &hi);
                c = argmin_codes(y, wb, block, lo, hi);
            }
            scales[r * nb_row + kb] = (uint8_t)c;
            double s = nvfp4_ref_e4m3(c);
            for (int i = 0; i < block; ++i) {
                int k = nvfp4_ref_round_fp4(fabs((double)y[i]), s);
                int nib = (signbit(y[i]) ? 8 : 0) | k;
                int64_t e = base + i;
                uint8_t* byte = &q[e >> 1];
                if ((e & 1) == 0)
                    *byte = (uint8_t)((*byte & 0xF0) | nib);
                else
                    *byte = (uint8_t)((*byte & 0x0F) | (nib << 4));
            }
        }
    }
    *tensor_scale = S;
    return REF_OK;
}

int nvfp4_ref_quantize(int method, const void* x, int dtype, int64_t rows, int64_t cols,
                       int block, float fp8_range, float static_scale, const float* col_weight,
                       float* tensor_scale, uint8_t* q, uint8_t* scales)
{
    return quantize_impl(method, -1, 0, 0, x, dtype, rows, cols, block, fp8_range,
                         static_scale, col_weight, tensor_scale, q, scales);
}

/* ScaleSweep with a window variant; col_weight NULL selects the MSE objective, otherwise
 * the WMSE objective with those per-column weights. */
int nvfp4_ref_quant_scalesweep_window(const void* x, int dtype, int64_t rows, int64_t cols,
                                      int block, const float* col_weight, int win_mode,
                                      int lo_off, int hi_off, float fp8_range,
                                      float static_scale, float* tensor_scale, uint8_t* q,
                                      uint8_t* scales)
{
    if (win_mode != REF_WINDOW_OFFSETS && win_mode != REF_WINDOW_TIGHT) return REF_ERR_ARG;
    int method = col_weight ? REF_SCALESWEEP_WMSE : REF_SCALESWEEP_MSE;
    return quantize_impl(method, win_mode, lo_off, hi_off, x, dtype, rows, cols, block,
                         fp8_range, static_scale, col_weight, tensor_scale, q, scales);
}

/* ------------------------------------------------------------------------------------- */
/* Online quantization of activations, KV cache and queries (implementation details:     */
/* static global scale; importance vectors of the WMSE section; the swizzled scale layout  */
/* of the operator benchmark).                                                            */
/* ------------------------------------------------------------------------------------- */

/* Byte offset of the scale of row m, scale column k in the swizzled layout of a scale matrix
 * with k16 columns: the matrix is padded to a multiple of 128 rows and 4 columns and stored
 * as tiles of 128 rows x 4 columns, tile-row-major; inside a tile, row m of the tile sits at
 * (m mod 32) * 16 + (m div 32) * 4 and column k at k mod 4.  reading: this is the layout of
 * vLLM's NVFP4 operators, which the paper's operator benchmark uses. */
int64_t nvfp4_ref_swizzled_offset(int64_t m, int64_t k, int64_t k16)
{
    int64_t kt = (k16 + 3) / 4;
    int64_t tile = (m / 128) * kt + k / 4;
    int64_t mm = m % 128;
    return tile * 512 + (mm % 32) * 16 + (mm / 32) * 4 + k % 4;
}

int64_t nvfp4_ref_scales_bytes(int64_t rows, int64_t cols, int block, int layout)
{
    if (!valid_block(block) || rows < 0 || cols < 0 || cols % block != 0) return -1;
    int64_t k16 = cols / block;
    if (layout == REF_SCALES_ROW_MAJOR) return rows * k16;
    if (layout == REF_SCALES_SWIZZLED && block == 16)
        return ((rows + 127) / 128 * 128) * ((k16 + 3) / 4 * 4);
    return -1;
}

/* Quantize with a given (static, calibrated) global scale, the importance vector of row r
 * being importance[((r / imp_group_rows) mod imp_groups) * cols ...] (imp_groups = 1: one
 * vector for every row, as for activations; K, V and Q as [batch * heads * tokens, head_dim]
 * rows take imp_group_rows = tokens and imp_groups = heads).  Each row is quantized on its
 * own with its vector, exactly as a one-row tensor with that column weight and the same S.
 * Scales go row-major or swizzled (block 16 only; padding bytes are 0).  importance may be
 * NULL for the unweighted methods; tensor_scale may be NULL. */
int nvfp4_ref_quant_online(int method, const void* x, int dtype, int64_t rows, int64_t cols,
                           int block, const float* importance, int64_t imp_groups,
                           int64_t imp_group_rows, float static_scale, int layout,
                           float* tensor_scale, uint8_t* q, uint8_t* scales)
{
    if (method < REF_ABSMAX || method > REF_SCALESWEEP_WMSE) return REF_ERR_ARG;
    if (dtype != 0 && dtype != 1) return REF_ERR_DTYPE;
    if (!valid_block(block)) return REF_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return REF_ERR_SHAPE;
    if (!(static_scale > 0.0f) || !isfinite(static_scale)) return REF_ERR_ARG;
    if (method == REF_SCALESWEEP_WMSE && !importance) return REF_ERR_NULL;
    if (importance && (imp_groups < 1 || imp_group_rows < 1)) return REF_ERR_ARG;
    int64_t nbytes = nvfp4_ref_scales_bytes(rows, cols, block, layout);
    if (nbytes < 0) return REF_ERR_ARG;
    if (rows * cols > 0 && (!x || !q || !scales)) return REF_ERR_NULL;
    int64_t k16 = cols / block;
    uint8_t* row_scales = k16 > 0 ? (uint8_t*)malloc((size_t)k16) : NULL;
    if (k16 > 0 && !row_scales) return REF_ERR_ARG;
    if (layout == REF_SCALES_SWIZZLED) memset(scales, 0, (size_t)nbytes);
    size_t esz = dtype == 0 ? 4 : 2;
    int rc = REF_OK;
    for (int64_t r = 0; r < rows && rc == REF_OK; ++r) {
        const float* w = importance
                             ? importance + ((r / imp_group_rows) % imp_groups) * cols
                             : NULL;
        float S;
        rc = nvfp4_ref_quantize(method, (const char*)x + (size_t)(r * cols) * esz, dtype, 1,
                                cols, block, 448.0f, static_scale, w, &S, q + r * (cols / 2),
                                row_scales);
        for (int64_t k = 0; k < k16; ++k) {
            int64_t off = layout == REF_SCALES_SWIZZLED ? nvfp4_ref_swizzled_offset(r, k, k16)
                                                        : r * k16 + k;
            scales[off] = row_scales[k];
        }
    }
    free(row_scales);
    if (rc == REF_OK && tensor_scale) *tensor_scale = static_scale;
    return rc;
}

/* ------------------------------------------------------------------------------------- */
/* A producer for the fused online quantizer: the SwiGLU product of a Llama MLP.           */
/* ------------------------------------------------------------------------------------- */

/* reading: the paper leaves the producer of a fused quantizer open (Overhead Analysis: the
 * operators are memory-bound, fusion is the next step).  The product silu(g) * u of a
 * SwiGLU MLP, the input of its down projection, is taken, with its binary32 arithmetic fixed
 * so that a plain implementation reproduces it bit for bit:
 *   e^x: zero below x = -80 (then 1 + e^x rounds to 1 anyway) and +inf from x = 89; else
 *        n = rint(RN(x * RN(log2 e))), the reduced argument r = x - n ln2 with ln2 split as
 *        0.693145751953125 + RN(ln2 - 0.693145751953125) (two fused multiply-adds), the
 *        Taylor polynomial of degree 6 with coefficients RN(1/k!) in Horner form (fused
 *        multiply-adds), times 2^n (exact: the result stays normal);
 *   silu(g) = RN(g / RN(1 + e^-g)) (a correctly rounded division); h = RN(silu(g) * u),
 *   rounded to nearest even onto bfloat16. */
float nvfp4_ref_swiglu_exp(float x)
{
    if (x < -80.0f) return 0.0f;
    if (x >= 89.0f) return INFINITY;
    const float log2e = 1.44269502162933349609375f;          /* RN32(1 / ln 2) */
    const float ln2_hi = 0.693145751953125f;
    const float ln2_lo = (float)(0.6931471805599453094 - 0.693145751953125);
    float t = x * log2e;
    float n = rintf(t);
    float r = fmaf(-n, ln2_hi, x);
    r = fmaf(-n, ln2_lo, r);
    float c[7];
    double f = 1.0;
    for (int k = 0; k < 7; ++k) {
        if (k > 0) f *= (double)k;
        c[k] = (float)(1.0 / f);                               /* RN32(1 / k!) */
    }
    float p = c[6];
    for (int k = 5; k >= 0; --k) p = fmaf(p, r, c[k]);
    return ldexpf(p, (int)n);
}

static uint16_t bf16_round(float v)
{
    uint32_t b;
    memcpy(&b, &v, 4);
    /* round to nearest even at bit 16 (finite values and infinities) */
    uint32_t r = b + 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(r >> 16);
}

static float bf16_value(uint16_t h)
{
    uint32_t b = (uint32_t)h << 16;
    float v;
    memcpy(&v, &b, 4);
    return v;
}

/* h = bf16(RN(silu(g) * u)) elementwise over bfloat16 gate and up (count elements). */
int nvfp4_ref_swiglu(const uint16_t* gate, const uint16_t* up, int64_t count, uint16_t* h)
{
    if (count < 0) return REF_ERR_SHAPE;
    if (count > 0 && (!gate || !up || !h)) return REF_ERR_NULL;
    for (int64_t i = 0; i < count; ++i) {
        float g = bf16_value(gate[i]), u = bf16_value(up[i]);
        if (!isfinite(g) || !isfinite(u)) return REF_ERR_NONFINITE;
        float e = nvfp4_ref_swiglu_exp(-g);
        float d = 1.0f + e;
        float sg = g / d;
        h[i] = bf16_round(sg * u);
    }
    return REF_OK;
}

/* Squared norms of the input channels (the importance scores of the WMSE section): for a
 * matrix x [rows, cols], out[g][c] = sum over the rows r of group g of x[r][c]^2, where row
 * r belongs to group ((r / group_rows) mod groups) / group_div, summed in row order in
 * binary64 and rounded once to binary32; each group's vector is written rep_out times
 * (out has groups / group_div * rep_out vectors).  Activations: the weight matrix
 * [d_out, d_in] with one group; queries from keys and keys from queries of grouped-query
 * attention: rows [batch * heads * tokens, head_dim] with group_rows = tokens; values from
 * W^O [d_model, heads * head_dim] viewed as [d_model * heads, head_dim] with group_rows = 1
 * and groups = heads. */
int nvfp4_ref_channel_sq_norms(const void* x, int dtype, int64_t rows, int64_t cols,
                               int64_t group_rows, int64_t groups, int64_t group_div,
                               int64_t rep_out, float* out)
{
    if (dtype != 0 && dtype != 1) return REF_ERR_DTYPE;
    if (rows < 0 || cols < 0) return REF_ERR_SHAPE;
    if (group_rows < 1 || groups < 1 || group_div < 1 || rep_out < 1 || groups % group_div)
        return REF_ERR_ARG;
    if (!out || (rows * cols > 0 && !x)) return REF_ERR_NULL;
    int64_t gout = groups / group_div;
    double* acc = (double*)calloc((size_t)(gout * cols > 0 ? gout * cols : 1), sizeof(double));
    if (!acc) return REF_ERR_ARG;
    for (int64_t r = 0; r < rows; ++r) {
        int64_t g = ((r / group_rows) % groups) / group_div;
        for (int64_t c = 0; c < cols; ++c) {
            double v = (double)load_elem(x, dtype, r * cols + c);
            acc[g * cols + c] += v * v;
        }
    }
    for (int64_t g = 0; g < gout; ++g)
        for (int64_t j = 0; j < rep_out; ++j)
            for (int64_t c = 0; c < cols; ++c)
                out[(g * rep_out + j) * cols + c] = (float)acc[g * cols + c];
    free(acc);
    return REF_OK;
}

/* ------------------------------------------------------------------------------------- */
/* GPTQ with fixed block scales (implementation details, GPTQ paragraph): LDLQ, damping    */
/* 0.01 x the mean Hessian diagonal, static reordering by descending Hessian diagonal,     */
/* block scales chosen before the pass.                                                   */
/* ------------------------------------------------------------------------------------- */

/* Column order of the pass: indices sorted by H_cc descending, ties by ascending index. */
int nvfp4_ref_ldlq_order(const double* H, int64_t n, int64_t* perm)
{
    if (!H || !perm) return REF_ERR_NULL;
    for (int64_t i = 0; i < n; ++i) perm[i] = i;
    for (int64_t i = 1; i < n; ++i) {               /* insertion sort: stable */
        int64_t v = perm[i];
        double d = H[v * n + v];
        int64_t j = i;
        while (j > 0 && H[perm[j - 1] * n + perm[j - 1]] < d) {
            perm[j] = perm[j - 1];
            --j;
        }
        perm[j] = v;
    }
    return REF_OK;
}

/* Hp = P^T H P + lambda I with lambda = damp * (sum_c H_cc) / n (the diagonal summed in index
 * order), P the column order; then Hp = (U + I) D (U + I)^T with U strictly upper triangular
 * and D diagonal, computed from the last column backwards:
 *   D_j  = Hp_jj - sum_{k > j} (U_jk U_jk) D_k
 *   U_ij = (Hp_ij - sum_{k > j} (U_ik U_jk) D_k) / D_j      (i < j)
 * each sum subtracted term by term from the largest k down.  U is returned row-major [n, n]
 * (diagonal and lower part 0).  A non-positive or non-finite D_j is an error. */
int nvfp4_ref_ldlq_factor(const double* H, int64_t n, double damp, const int64_t* perm,
                          double* U, double* D)
{
    if (!H || !perm || !U || !D) return REF_ERR_NULL;
    if (!(damp >= 0.0) || !isfinite(damp)) return REF_ERR_ARG;
    double tr = 0.0;
    for (int64_t c = 0; c < n; ++c) tr += H[c * n + c];
    double lambda = n > 0 ? damp * (tr / (double)n) : 0.0;
    for (int64_t i = 0; i < n * n; ++i) U[i] = 0.0;
    for (int64_t j = n - 1; j >= 0; --j) {
        double dj = H[perm[j] * n + perm[j]] + lambda;
        for (int64_t k = n - 1; k > j; --k) dj = dj - (U[j * n + k] * U[j * n + k]) * D[k];
        if (!(dj > 0.0) || !isfinite(dj)) return REF_ERR_ARG;
        D[j] = dj;
        for (int64_t i = 0; i < j; ++i) {
            double acc = H[perm[i] * n + perm[j]];
            for (int64_t k = n - 1; k > j; --k) acc = acc - (U[i * n + k] * U[j * n + k]) * D[k];
            U[i * n + j] = acc / dj;
        }
    }
    return REF_OK;
}

/* LDLQ (equivalent to GPTQ): in the column order, each column's values are
 *   x_a = w_a + sum_{b < a} (w_b - w^_b) U_ba        (terms added from b = 0 up)
 * and w^_a is x_a quantized with the block's fixed scale: y = RN32(RN32(x_a) / S), nibble =
 * sign(y) << 3 | RNE_FP4(|y| / s), w^_a = +-E2M1 * s * S (exact in binary64).  w [rows, n]
 * in binary32 or bfloat16, H [n, n] binary64, scales [rows, n / block] E4M3 codes fixed
 * beforehand, S the global scale; q [rows, n / 2] nibbles as the quantizers pack them. */
int nvfp4_ref_ldlq(const void* w, int dtype, int64_t rows, int64_t n, int block, const double* H,
                   const uint8_t* scales, float S, double damp, uint8_t* q)
{
    if (dtype != 0 && dtype != 1) return REF_ERR_DTYPE;
    if (!valid_block(block)) return REF_ERR_BLOCK;
    if (rows < 0 || n < 0 || n % block != 0) return REF_ERR_SHAPE;
    if (!(S > 0.0f) || !isfinite(S)) return REF_ERR_ARG;
    if (rows * n > 0 && (!w || !H || !scales || !q)) return REF_ERR_NULL;
    if (n == 0 || rows == 0) return REF_OK;
    int64_t* perm = (int64_t*)malloc((size_t)n * sizeof(int64_t));
    double* U = (double*)malloc((size_t)(n * n) * sizeof(double));
    double* D = (double*)malloc((size_t)n * sizeof(double));
    double* e = (double*)malloc((size_t)n * sizeof(double));
    int rc = (perm && U && D && e) ? REF_OK : REF_ERR_ARG;
    if (rc == REF_OK) rc = nvfp4_ref_ldlq_order(H, n, perm);
    if (rc == REF_OK) rc = nvfp4_ref_ldlq_factor(H, n, damp, perm, U, D);
    int64_t nb = n / block;
    for (int64_t r = 0; r < rows && rc == REF_OK; ++r) {
        for (int64_t a = 0; a < n; ++a) {
            int64_t c = perm[a];
            double wv = (double)load_elem(w, dtype, r * n + c);
            double x = wv;
            for (int64_t b = 0; b < a; ++b) x = x + e[b] * U[b * n + a];
            float y = (float)x / S;
            double s = nvfp4_ref_e4m3(scales[r * nb + c / block]);
            int k = nvfp4_ref_round_fp4(fabs((double)y), s);
            double wq = nvfp4_ref_e2m1(k) * s * (double)S;
            if (signbit(y)) wq = -wq;
            e[a] = wv - wq;
            int nib = (signbit(y) ? 8 : 0) | k;
            int64_t el = r * n + c;
            uint8_t* byte = &q[el >> 1];
            if ((el & 1) == 0)
                *byte = (uint8_t)((*byte & 0xF0) | nib);
            else
                *byte = (uint8_t)((*byte & 0x0F) | (nib << 4));
        }
    }
    free(perm);
    free(U);
    free(D);
    free(e);
    return rc;
}

int nvfp4_ref_quant_absmax(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                           float fp8_range, float static_scale, float* tensor_scale,
                           uint8_t* q, uint8_t* scales)
{
    return nvfp4_ref_quantize(REF_ABSMAX, x, dtype, rows, cols, block, fp8_range,
                              static_scale, NULL, tensor_scale, q, scales);
}

int nvfp4_ref_quant_four_over_six(const void* x, int dtype, int64_t rows, int64_t cols,
                                  int block, float fp8_range, float static_scale,
                                  const float* col_weight, float* tensor_scale, uint8_t* q,
                                  uint8_t* scales)
{
    return nvfp4_ref_quantize(REF_FOUR_OVER_SIX, x, dtype, rows, cols, block, fp8_range,
                              static_scale, col_weight, tensor_scale, q, scales);
}

int nvfp4_ref_quant_scalesweep_mse(const void* x, int dtype, int64_t rows, int64_t cols,
                                   int block, float fp8_range, float static_scale,
                                   float* tensor_scale, uint8_t* q, uint8_t* scales)
{
    return nvfp4_ref_quantize(REF_SCALESWEEP_MSE, x, dtype, rows, cols, block, fp8_range,
                              static_scale, NULL, tensor_scale, q, scales);
}

int nvfp4_ref_quant_scalesweep_wmse(const void* x, int dtype, int64_t rows, int64_t cols,
                                    int block, float fp8_range, float static_scale,
                                    const float* col_weight, float* tensor_scale, uint8_t* q,
                                    uint8_t* scales)
{
    return nvfp4_ref_quantize(REF_SCALESWEEP_WMSE, x, dtype, rows, cols, block, fp8_range,
                              static_scale, col_weight, tensor_scale, q, scales);
}

/* Reconstruction x_hat_i = q_i * s_{block(i)} * S (NVFP4 section).  q * s is exact (at most 6
 * significant bits); the product with S is formed exactly in binary64 and rounded once. */
int nvfp4_ref_dequant(const uint8_t* q, const uint8_t* scales, float tensor_scale,
                      int64_t rows, int64_t cols, int block, float* out)
{
    if (!valid_block(block)) return REF_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return REF_ERR_SHAPE;
    if (rows * cols > 0 && (!q || !scales || !out)) return REF_ERR_NULL;
    int64_t nb_row = cols / block;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t j = 0; j < cols; ++j) {
            int64_t e = r * cols + j;
            int nib = (e & 1) ? (q[e >> 1] >> 4) : (q[e >> 1] & 15);
            double v = nvfp4_ref_e2m1(nib & 7);
            if (nib & 8) v = -v;
            double qs = v * nvfp4_ref_e4m3(scales[r * nb_row + j / block]);
            out[e] = (float)(qs * (double)tensor_scale);
        }
    }
    return REF_OK;
}

/* ------------------------------------------------------------------------------------- */
/* Appendix: optimal FP32 block scale, and its FP8-quantized version.                     */
/* ------------------------------------------------------------------------------------- */

static int cmp_double(const void* a, const void* b)
{
    double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/* Loss of the block at a real scale s with the rounding index of each element held fixed at
 * the one it takes at s_ref: the quadratic A - 2 B s + C s^2 of one segment. */
static void segment_quadratic(const float* y, const float* w, int n, double s_ref, double* A,
                              double* B, double* C)
{
    *A = *B = *C = 0.0;
    for (int i = 0; i < n; ++i) {
        double a = fabs((double)y[i]);
        double wi = w ? (double)w[i] : 1.0;
        double g = nvfp4_ref_e2m1(nvfp4_ref_round_fp4(a, s_ref));
        *A += wi * a * a;
        *B += wi * a * g;
        *C += wi * g * g;
    }
}

/* min over real s > 0 of L(s; y, w).  Each element's error is a piecewise quadratic in s
 * whose breakpoints are the s at which |y_i| / s meets an FP4 midpoint; between consecutive
 * breakpoints of the whole block the rounding indices are constant, so L is one quadratic
 * there.  Enumerate the segments, minimize each quadratic on its closed segment, keep the
 * least.  Returns the minimum; *s_opt receives the minimizer. */
double nvfp4_ref_continuous_opt(const float* y, const float* w, int n, double* s_opt)
{
    double bp[7 * MAX_BLOCK + 2];
    int nb = 0;
    for (int i = 0; i < n; ++i) {
        double a = fabs((double)y[i]);
        if (a == 0.0) continue;
        for (int k = 0; k < E2M1_CODES - 1; ++k) {
            double mid = 0.5 * (nvfp4_ref_e2m1(k) + nvfp4_ref_e2m1(k + 1));
            bp[nb++] = a / mid;
        }
    }
    double A0 = 0.0;
    for (int i = 0; i < n; ++i) {
        double a = (double)y[i];
        A0 += (w ? (double)w[i] : 1.0) * a * a;
    }
    double best = A0;           /* s -> infinity: everything rounds to zero */
    double best_s = INFINITY;
    if (nb == 0) {
        if (s_opt) *s_opt = 1.0;
        return 0.0;
    }
    qsort(bp, (size_t)nb, sizeof(double), cmp_double);
    for (int seg = 0; seg <= nb; ++seg) {
        double lo = (seg == 0) ? 0.0 : bp[seg - 1];
        double hi = (seg == nb) ? INFINITY : bp[seg];
        if (!(hi > lo)) continue;
        double s_ref = (seg == 0) ? 0.5 * hi : (seg == nb) ? 2.0 * lo : 0.5 * (lo + hi);
        double A, B, C;
        segment_quadratic(y, w, n, s_ref, &A, &B, &C);
        if (C <= 0.0) {
            if (A < best) { best = A; best_s = s_ref; }
            continue;
        }
        double s = B / C;
        if (s < lo) s = lo;
        if (s > hi) s = hi;
        if (s <= 0.0) continue;
        double val = A - 2.0 * B * s + C * s * s;
        if (val < 0.0) val = 0.0;
        if (val < best) { best = val; best_s = s; }
    }
    if (s_opt) *s_opt = best_s;
    return best;
}

/* FP8-quantized optimal scale: the better (by L) of the FP8 values just below and just above
 * the optimal real block scale, in the normalized domain y = x / S.  Returns the code. */
int nvfp4_ref_fp8_quantized_opt(const float* y, const float* w, int n, double* loss)
{
    double s_opt;
    nvfp4_ref_continuous_opt(y, w, n, &s_opt);
    int cf = nvfp4_ref_floor_fp8(s_opt, 1.0);
    int cc = cf;
    if (nvfp4_ref_e4m3(cf) < s_opt && cf < E4M3_MAX_CODE) cc = cf + 1;
    if (cf < 1) cf = 1;
    if (cc < 1) cc = 1;
    double jf = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(cf));
    double jc = nvfp4_ref_block_loss(y, w, n, nvfp4_ref_e4m3(cc));
    int c = (jc < jf) ? cc : cf;
    if (loss) *loss = (jc < jf) ? jc : jf;
    return c;
}

/* ------------------------------------------------------------------------------------- */
/* Metrics: Notation section.                                                             */
/* ------------------------------------------------------------------------------------- */

/* MSE = |x - xh|^2 / N, NMSE = |x - xh|^2 / |x|^2, WMSE = sum w (x - xh)^2 / sum w,
 * NWMSE = sum w (x - xh)^2 / sum w x^2, with the per-column weight broadcast over rows. */
int nvfp4_ref_metrics(const void* x, int dtype, const float* xhat, int64_t rows, int64_t cols,
                      const float* col_weight, double* out4)
{
    if (!out4 || (rows * cols > 0 && (!x || !xhat))) return REF_ERR_NULL;
    double se = 0.0, sx = 0.0, wse = 0.0, wsx = 0.0, sw = 0.0;
    for (int64_t r = 0; r < rows; ++r) {
        for (int64_t j = 0; j < cols; ++j) {
            double v = (double)load_elem(x, dtype, r * cols + j);
            double d = v - (double)xhat[r * cols + j];
            double wj = col_weight ? (double)col_weight[j] : 1.0;
            se += d * d;
            sx += v * v;
            wse += wj * d * d;
            wsx += wj * v * v;
            sw += wj;
        }
    }
    double N = (double)(rows * cols);
    out4[0] = N > 0 ? se / N : 0.0;
    out4[1] = sx > 0 ? se / sx : 0.0;
    out4[2] = sw > 0 ? wse / sw : 0.0;
    out4[3] = wsx > 0 ? wse / wsx : 0.0;
    return REF_OK;
}
