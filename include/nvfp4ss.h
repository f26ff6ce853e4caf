/*
 * nvfp4ss.h -- C interface of the NVFP4 ScaleSweep quantizer for AMD Instinct MI355X (gfx950).
 *
 * NVFP4 (ScaleSweep paper, arXiv 2606.07618, "NVFP4 Quantization" section) represents a tensor
 * x as (q, s, S): FP4 E2M1 values q, one FP8 E4M3 scale s per micro-block of 16 consecutive
 * elements, and one binary32 global scale S, reconstructing x_hat_i = q_i * s_{block(i)} * S.
 * The calls below compute (q, s, S) with four block-scale rules:
 *   nvfp4_quant_absmax          AbsMax (NVFP4 Quantization section)
 *   nvfp4_quant_four_over_six   4/6 (Introduction and Related Work)
 *   nvfp4_quant_scalesweep_mse  ScaleSweep with the MSE objective (Method section)
 *   nvfp4_quant_scalesweep_wmse ScaleSweep with the WMSE objective (Method section)
 * plus nvfp4_quant_scalesweep_window (ScaleSweep over other sweep windows: Tables 1 and 2,
 * and the sweep-range study of the Experiment section)
 * and nvfp4_dequant computes x_hat.
 *
 * Common conventions
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library never
 *     allocates, frees or keeps them.  Inputs and outputs must not overlap.
 *   - Every call validates its arguments synchronously on the host, before any launch; on an
 *     error it returns a negative nvfp4_status and has launched nothing and written nothing.
 *   - On success the work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *     the call returns NVFP4_OK without waiting.  A failed launch returns NVFP4_ERR_HIP.
 *   - Conditions that depend on the data cannot be reported synchronously: if x holds a NaN
 *     or an infinity, the dynamic global scale is NaN and the other outputs are unspecified
 *     (the kernels still terminate normally).  Check *tensor_scale after synchronizing.
 *   - Calls are thread-safe; the library holds no global state.  Two calls that are in
 *     flight at the same time must not share a workspace.
 *
 * Layouts (row-major)
 *   x       [rows, cols], dtype NVFP4_IN_F32 (binary32) or NVFP4_IN_BF16 (bfloat16);
 *           16-byte aligned.  Micro-blocks are `block` consecutive elements of a row
 *           (block in {16, 32, 64, 128}; cols % block == 0), i.e. they run along the input
 *           dimension d_in of a weight stored [d_out, d_in], as in Eq. (nvfp4_MSE).
 *   q       [rows, cols/2] bytes, 8-byte aligned; element 2j sits in bits 3:0 of byte j and
 *           element 2j+1 in bits 7:4; a nibble is (sign << 3) | E2M1 code, the code k of the
 *           magnitude {0, 0.5, 1, 1.5, 2, 3, 4, 6}[k].  The sign of x is kept, also on zero.
 *   scales  [rows, cols/block] bytes, the E4M3 bit pattern (0..126) of each block scale.
 *   tensor_scale  one binary32 in device memory, receives S.
 */
#ifndef NVFP4SS_H
#define NVFP4SS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { NVFP4_IN_F32 = 0, NVFP4_IN_BF16 = 1 } nvfp4_dtype;

typedef enum {
    NVFP4_OK = 0,
    NVFP4_ERR_NULL = -1,      /* a required pointer is NULL */
    NVFP4_ERR_SHAPE = -2,     /* rows < 0, cols < 0, or cols % block != 0 */
    NVFP4_ERR_BLOCK = -3,     /* block not in {16, 32, 64, 128} */
    NVFP4_ERR_DTYPE = -4,     /* dtype / out_dtype not supported */
    NVFP4_ERR_ARG = -5,       /* fp8_range, static_scale or a window out of range */
    NVFP4_ERR_WORKSPACE = -6, /* dynamic scale requested without a large enough workspace */
    NVFP4_ERR_ALIGN = -7,     /* x, col_weight or workspace not 16-byte aligned, q not 8 */
    NVFP4_ERR_HIP = -8,       /* a kernel launch failed */
    NVFP4_ERR_LIMIT = -10     /* more than the no-allocation entry point's fixed scratch holds */
} nvfp4_status;

/* Bytes of device workspace the dynamic-scale path needs (a small constant, 10 KiB).
 * It carries the per-workgroup |x| maxima of the reduction kernel and the resulting S and 1/S
 * to the quantization kernel of the same call; it needs no initialization and holds nothing
 * between calls.  Static-scale calls do not touch it (it may be NULL). */
size_t nvfp4_workspace_bytes(void);

/* Text for a status code (a static string; never NULL). */
const char* nvfp4_status_string(int status);

/*
 * Global scale and arguments shared by the quantizers.
 *   fp8_range     D in S = max_i |x_i| / (6 D): 448 for AbsMax (NVFP4 Quantization section),
 *                 256 for ScaleSweep and 4/6 (Global Scale Selection).  Finite, 0 < D <= 448,
 *                 else NVFP4_ERR_ARG.  6 D is formed in binary32, then S = RN32(amax / (6 D));
 *                 an all-zero tensor gets S = 1, a quotient that underflows gets the smallest
 *                 positive binary32.
 *   static_scale  0: dynamic -- a first kernel reduces max |x| over the tensor and writes S.
 *                 Finite > 0: a given (calibrated) global scale, as used for activations, KV
 *                 cache and queries (implementation details appendix); no reduction pass;
 *                 S = static_scale is still written to *tensor_scale.  Every |x| / S must be
 *                 finite.  Negative, NaN or infinite: NVFP4_ERR_ARG.
 *   workspace     >= nvfp4_workspace_bytes() bytes, 16-byte aligned, for dynamic S (see above);
 *                 otherwise NVFP4_ERR_WORKSPACE (NULL with static_scale > 0 is fine).
 * Every quantizer normalizes y_i = RN32(x_i / S) (a correctly rounded division) and works on
 * blocks of y, as the Block Scale Optimization section does; FP4 rounding is to nearest with
 * ties to the even code; the objective L(s; y, w) is Eq. (weighted_quantization_loss).
 */

/* AbsMax (NVFP4 Quantization section): s = round-to-nearest-even FP8(max|y| / 6), saturating
 * at 448 (the code may be 0: then every value of the block is 0); q_i = RNE FP4(y_i / s). */
int nvfp4_quant_absmax(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                       float fp8_range, float static_scale, float* tensor_scale, uint8_t* q,
                       uint8_t* scales, void* workspace, size_t workspace_bytes, void* stream);

/* 4/6: the FP8 scales round-to-nearest(max|y|/6) and round-to-nearest(max|y|/4) (mapping the
 * block maximum to 6 or to 4); keeps the /4 scale only if its loss is strictly lower.
 * col_weight: [cols] binary32 column importance (16-byte aligned) for a weighted loss, or
 * NULL for the unweighted one.  Weights must be finite and >= 0 (not checked). */
int nvfp4_quant_four_over_six(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                              const float* col_weight, float fp8_range, float static_scale,
                              float* tensor_scale, uint8_t* q, uint8_t* scales,
                              void* workspace, size_t workspace_bytes, void* stream);

/* ScaleSweep, MSE objective (Block Scale Optimization; Lemmas 1-3): with s0 the FP8 value
 * just below max|y| / 6 and c0 = I(s0) its bit pattern, sweep every E4M3 code c in
 * [max(1, c0 - L), min(126, c0 + 7)] and keep the argmin of L(E4M3(c); y), the smallest code
 * on a tie.  L = 3 for block 16 (Lemma 3); 5 / 7 / 11 for block 32 / 64 / 128 (the lemma's
 * argument extended to larger blocks).  The result equals the exact argmin over the window
 * for every block: near-ties are re-decided in binary64. */
int nvfp4_quant_scalesweep_mse(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                               float fp8_range, float static_scale, float* tensor_scale,
                               uint8_t* q, uint8_t* scales, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ScaleSweep, WMSE objective (Eq. nvfp4_WMSE): as above with the weighted loss
 * sum_i Imp_i (y_i - q_i s)^2, Imp the per-input-column importance ||X_{:,i}||^2 (or any
 * positive multiple of it, e.g. the mean over calibration tokens), and L = 8 (the empirical
 * s_base / 2 bound; 11 for block 128).  col_weight: [cols] binary32, required (NULL ->
 * NVFP4_ERR_NULL), 16-byte aligned, finite and >= 0 (not checked). */
int nvfp4_quant_scalesweep_wmse(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                                const float* col_weight, float fp8_range, float static_scale,
                                float* tensor_scale, uint8_t* q, uint8_t* scales,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Window of nvfp4_quant_scalesweep_window. */
typedef enum { NVFP4_WINDOW_OFFSETS = 0, NVFP4_WINDOW_TIGHT = 1 } nvfp4_window;

/* ScaleSweep over a chosen window of E4M3 bit patterns around c0 = I(s0) (s0 the FP8 value
 * just below max|y| / 6, as above).  A block sweeps the codes [lo, hi] and keeps the exact
 * argmin of L, the smallest code on a tie, where
 *   window_mode NVFP4_WINDOW_OFFSETS: lo = c0 + window_lo, hi = c0 + window_hi -- the [l, r]
 *     bit-pattern bounds of the sweep-range study (Experiment section, Scale Sweep Range);
 *     -126 <= window_lo <= window_hi <= 126 (else NVFP4_ERR_ARG).  [-3, 7] is
 *     nvfp4_quant_scalesweep_mse at block 16, [-8, 7] nvfp4_quant_scalesweep_wmse, and
 *     [-126, 126] the exhaustive sweep over all 126 positive scales;
 *   window_mode NVFP4_WINDOW_TIGHT: per-mantissa offsets for the mantissa field b = c0 & 7
 *     (window_lo / window_hi ignored): hi = c0 + 7, or c0 + 6 for b = 6, 7 (Table 1, from
 *     Lemmas 1 and 2; any objective and block); lo = c0 - 3 for b = 0, 7 and c0 - 2 otherwise
 *     (Table 2, from Lemma 3) with the MSE objective at block 16, else the standard lower
 *     offset of the objective.  Where the lemmas hold (normal s0 with 11/7 s0 <= 448) it
 *     picks the same codes as the standard windows with 9 to 11 candidates instead of 11.
 * Each end is clamped into 1..126, so a window wholly outside them sweeps that end code alone.
 * col_weight NULL selects the MSE objective, otherwise the WMSE objective with those
 * per-column weights (as nvfp4_quant_scalesweep_wmse).  Other arguments, layouts and errors
 * as nvfp4_quant_scalesweep_wmse. */
int nvfp4_quant_scalesweep_window(const void* x, int dtype, int64_t rows, int64_t cols,
                                  int block, const float* col_weight, int window_mode,
                                  int window_lo, int window_hi, float fp8_range,
                                  float static_scale, float* tensor_scale, uint8_t* q,
                                  uint8_t* scales, void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * Online quantization of activations, KV cache and query states (implementation details:
 * a static global scale found at calibration; importance vectors as in the WMSE section).
 */
typedef enum { NVFP4_SCALES_ROW_MAJOR = 0, NVFP4_SCALES_SWIZZLED = 1 } nvfp4_scale_layout;

/* Bytes of the scale output of a [rows, cols] tensor: rows * cols / block row-major; for the
 * swizzled layout (block 16 only) the scale matrix padded to multiples of 128 rows and 4
 * columns.  A negative nvfp4_status for invalid arguments. */
int64_t nvfp4_scales_bytes(int64_t rows, int64_t cols, int block, int layout);

/* Quantizes x [rows, cols] with a given static global scale S = static_scale (finite, > 0,
 * else NVFP4_ERR_ARG; every |x| / S must be finite) and method 0 AbsMax, 1 4/6,
 * 2 ScaleSweep-MSE, 3 ScaleSweep-WMSE (same block-scale rules as the single-tensor calls).
 * importance: [imp_groups, cols] binary32 (16-byte aligned, finite, >= 0), the weights of
 * row r being vector ((r / imp_group_rows) mod imp_groups): one vector for activations
 * [tokens, d_in] (imp_groups = 1), per head for K, V or Q laid out as
 * [batch * heads * tokens, head_dim] (imp_groups = heads, imp_group_rows = tokens).  Required
 * for method 3, optional for 4/6, ignored otherwise.  scale_layout NVFP4_SCALES_ROW_MAJOR
 * writes scales [rows, cols/block]; NVFP4_SCALES_SWIZZLED (block 16) writes the 128 x 4 tiled
 * layout of vLLM's NVFP4 GEMM operands -- byte
 *   ((m / 128) * kt + k / 4) * 512 + (m mod 32) * 16 + ((m / 32) mod 4) * 4 + k mod 4
 * for row m, scale column k, kt = ceil(cols / 64) -- and zeroes its padding; the buffer holds
 * nvfp4_scales_bytes() bytes.  tensor_scale: NULL, or a device float that receives S.  No
 * workspace, no reduction pass: one quantization kernel (plus a padding kernel for the
 * swizzled layout), asynchronous on `stream`.  Other errors as the single-tensor calls. */
int nvfp4_quant_online(int method, const void* x, int dtype, int64_t rows, int64_t cols, int block,
                       const float* importance, int64_t imp_groups, int64_t imp_group_rows,
                       float static_scale, int scale_layout, float* tensor_scale, uint8_t* q,
                       uint8_t* scales, void* stream);

/* The producer of a quantized activation fused with its quantizer (the Overhead Analysis:
 * the operators are memory-bound and open to fusion).  The producer is the SwiGLU product of
 * a Llama MLP, the input of its down projection: over bfloat16 gate and up [rows, cols],
 *   h = bf16(RN(silu(g) * u)),  silu(g) = RN(g / RN(1 + e^-g)) (a correctly rounded division),
 * with e^x computed as: 0 for x < -80, +inf for x >= 89, otherwise n = rint(RN(x * RN32(1/ln 2))),
 * r = fma(-n, 0.693145751953125, x), r = fma(-n, RN32(ln 2 - 0.693145751953125), r), the
 * degree-6 Taylor polynomial in r with coefficients RN32(1/k!) in Horner form (fused
 * multiply-adds), times 2^n; bfloat16 rounding to nearest even.
 * nvfp4_swiglu writes h [rows, cols] (bfloat16; the unfused producer).
 * nvfp4_quant_online_swiglu quantizes h without writing it: it equals nvfp4_swiglu followed by
 * nvfp4_quant_online on h with dtype NVFP4_IN_BF16 and block 16 (same arguments otherwise),
 * bit for bit, and reads 4 bytes per element instead of 8 (4 + 2 + 2).  gate, up: 16-byte
 * aligned device pointers; cols % 16 == 0; non-finite inputs give unspecified outputs.  Errors
 * as nvfp4_quant_online (up NULL: NVFP4_ERR_NULL). */
int nvfp4_swiglu(const void* gate, const void* up, int64_t rows, int64_t cols, void* h, void* stream);
int nvfp4_quant_online_swiglu(int method, const void* gate, const void* up, int64_t rows, int64_t cols,
                              const float* importance, int64_t imp_groups, int64_t imp_group_rows,
                              float static_scale, int scale_layout, float* tensor_scale, uint8_t* q,
                              uint8_t* scales, void* stream);

/* Importance vectors (WMSE section): squared norms of input channels.  For x [rows, cols]
 * (binary32 or bfloat16), out[g][c] = sum of x[r][c]^2 over the rows r of group
 * g = ((r / group_rows) mod groups) / group_div, accumulated in binary64 and rounded once to
 * binary32, each group's vector written rep_out times: out is
 * [groups / group_div * rep_out, cols] binary32.  groups % group_div == 0 and
 * groups / group_div <= 64, else NVFP4_ERR_ARG.  Uses:
 *   activations of a linear layer: x = its weight [d_out, d_in], one group;
 *   query states from keys (grouped-query attention, heads_q = rep * heads_kv): x = K as
 *     [batch * heads_kv * tokens, head_dim], group_rows = tokens, groups = heads_kv,
 *     rep_out = rep -- one vector per query head;
 *   keys from queries: x = Q as [batch * heads_q * tokens, head_dim], group_rows = tokens,
 *     groups = heads_q, group_div = rep;
 *   values from W^O [d_model, heads_q * head_dim]: x = W^O viewed as
 *     [d_model * heads_q, head_dim], group_rows = 1, groups = heads_q, group_div = rep.
 * Deterministic (fixed summation order: column-wise over 256-row chunks, then over chunks).
 * workspace: >= nvfp4_channel_sq_norms_workspace_bytes() bytes, 8-byte aligned. */
int64_t nvfp4_channel_sq_norms_workspace_bytes(int64_t rows, int64_t cols, int64_t groups,
                                               int64_t group_div);
int nvfp4_channel_sq_norms(const void* x, int dtype, int64_t rows, int64_t cols, int64_t group_rows,
                           int64_t groups, int64_t group_div, int64_t rep_out, float* out,
                           void* workspace, size_t workspace_bytes, void* stream);

/* GPTQ with fixed block scales (implementation details, GPTQ paragraph), in the LDLQ form the
 * paper uses: the block scales (scales [rows, cols/block] E4M3 codes, row-major) and the
 * global scale (*tensor_scale, device) are chosen beforehand by a quantizer call; the input
 * channels are visited in descending order of the Hessian diagonal (ties by index); the
 * Hessian hessian [cols, cols] (binary64, row-major, symmetric positive semi-definite, e.g.
 * X^T X over calibration activations) is damped by damp x its mean diagonal (damp = 0.01 in
 * the paper) and factored as (U + I) D (U + I)^T with U strictly upper triangular; then each
 * value, in that order, is its weight plus the earlier errors (w - w^) times U, quantized with
 * its block's fixed scale as the quantizers round: y = RN32(RN32(x) / S), nibble
 * sign(y) << 3 | RNE_FP4(|y| / s).  Outputs q [rows, cols/2] nibbles as the quantizers pack
 * them.  w: [rows, cols] binary32 or bfloat16.  cols must be a multiple of 64.  *status
 * (device int) is set to 0, or 1 if the damped Hessian is not positive definite (then q is
 * unspecified): check it after synchronizing.  workspace: >= nvfp4_ldlq_workspace_bytes()
 * bytes (about 8 (cols^2 + 2 rows cols) bytes), 256-byte aligned, no initialization.  All
 * arithmetic is binary64 in a fixed order (no atomics), so results are deterministic. */
size_t nvfp4_ldlq_workspace_bytes(int64_t rows, int64_t cols);
int nvfp4_ldlq(const void* w, int dtype, int64_t rows, int64_t cols, int block, const double* hessian,
               const uint8_t* scales, const float* tensor_scale, double damp, uint8_t* q, int* status,
               void* workspace, size_t workspace_bytes, void* stream);

/* One tensor of a batched call: device pointers and shape, as in the single-tensor calls
 * (col_weight: NULL unless the method uses weights). */
typedef struct {
    const void* x;
    int64_t rows, cols;
    const float* col_weight;
    float* tensor_scale;
    uint8_t* q;
    uint8_t* scales;
} nvfp4_tensor;

/* Workspace bytes for a batched call over `count` tensors (count single-call workspaces). */
size_t nvfp4_batched_workspace_bytes(int count);

/* Quantizes `count` tensors with one method (0 AbsMax, 1 4/6, 2 ScaleSweep-MSE,
 * 3 ScaleSweep-WMSE), each with its own dynamic global scale: the per-tensor round-to-nearest
 * pipeline of the experiment setup applied to, e.g., the weights of one decoder layer.  Every
 * tensor's outputs are bit-identical to its single-tensor call.  `tensors` is a host array;
 * the descriptors may be reused once the call returns.  Everything runs on `stream`: the
 * smallest non-empty tensor's |x| reduction first, then one quantization kernel per tensor in
 * ascending size, each of which also reduces max |x| of the next tensor (atomic maxima into
 * that tensor's workspace), so that only the smallest reduction is not overlapped with a
 * sweep.  workspace: >= nvfp4_batched_workspace_bytes(count), 16-byte aligned, no
 * initialization; two calls in flight at the same time must not share it.  The call allocates
 * no host or device memory for any count (the ascending order is found by rescanning the
 * descriptors).  Errors as for the single-tensor calls (validated for every tensor before any
 * launch); count < 0 or an unknown method: NVFP4_ERR_ARG. */
int nvfp4_quant_batched(int method, const nvfp4_tensor* tensors, int count, int dtype, int block,
                        float fp8_range, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): nvfp4_quant_batched without a workspace argument.
 * The scratch it needs (amax partials, S and 1/S, |x| maximum slots: nvfp4_workspace_bytes()
 * per tensor) lives in a fixed device array of NVFP4_NOALLOC_MAX_TENSORS such workspaces
 * (320 KiB) that the library defines and each GPU holds until the process ends; the call
 * allocates nothing, host or device.  On its first call for a device it looks up that device's
 * copy of the array (hipGetSymbolAddress; the device is the stream's, or the current one for
 * the null stream).  Outputs are bit-identical to nvfp4_quant_batched's.  count above
 * NVFP4_NOALLOC_MAX_TENSORS: NVFP4_ERR_LIMIT, nothing launched; other errors as for
 * nvfp4_quant_batched.  Every call on one GPU shares that GPU's array and leaves its last
 * contents there (the chain clears what must start at zero with a kernel of its own): calls
 * that overlap in time on one GPU (other streams, other host threads) race and must not be
 * issued; calls ordered on one stream are safe. */
#define NVFP4_NOALLOC_MAX_TENSORS 32
int nvfp4_quant_batched_noalloc(int method, const nvfp4_tensor* tensors, int count, int dtype,
                                int block, float fp8_range, void* stream);

/* Reconstruction x_hat_i = q_i * s_{block(i)} * S (NVFP4 Quantization section) into out
 * [rows, cols] binary32 (out_dtype must be NVFP4_IN_F32): q * s is exact, so each output is the
 * single rounding RN32((q * s) * S).  tensor_scale is read from device memory. */
int nvfp4_dequant(const uint8_t* q, const uint8_t* scales, const float* tensor_scale,
                  int64_t rows, int64_t cols, int block, int out_dtype, void* out, void* stream);

/*
 * Reference scales and exact losses for gap reports (appendix "Optimal FP32 Scale for FP4
 * Quantization"; the relative gaps of Figures 1 and 4).  These are analysis calls, not
 * quantizers.  Each works on y = RN32(x / S) with S read from the device float
 * *tensor_scale (e.g. the one a quantizer call wrote), blocks and weights as in the
 * quantizers (col_weight NULL: MSE objective).  Outputs are per micro-block, in block order
 * (row-major over [rows, cols/block]); every value is computed in binary64 with a fixed
 * order of correctly rounded operations.  x needs only its element alignment here.
 */

/* Optimal real block scale (appendix, first paragraph): opt_loss[b] = min over real s > 0 of
 * L(s; y, w), found by enumerating the pieces between the breakpoints |y_i| / m_k
 * (m_k the midpoints between neighbouring E2M1 values), on each of which L is a quadratic in
 * s, and minimizing every piece on its closed interval; the lowest piece wins a tie, and the
 * all-zero reconstruction (s -> infinity) wins a tie with any piece.  opt_scale[b] receives
 * the minimizer (+infinity for the all-zero reconstruction, 1 for an all-zero block).
 * FP8-quantized optimal scale (appendix, second paragraph): of the two E4M3 values just below
 * and just above opt_scale[b] (codes >= 1), the one with the lower L, the lower one on a tie:
 * fp8_code[b] its code and fp8_loss[b] its loss.  opt_loss [nblocks] is required (8-byte
 * aligned); opt_scale, fp8_code and fp8_loss may be NULL.  One wavefront per block; binary64
 * ALU-bound. */
int nvfp4_block_optimum(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                        const float* col_weight, const float* tensor_scale, double* opt_loss,
                        double* opt_scale, uint8_t* fp8_code, double* fp8_loss, void* stream);

/* Exact loss L(E4M3(scales[b]); y, w) of every block at its given scale code (0..126; larger
 * codes are read as 126), summed in element order in binary64: loss [nblocks], 8-byte
 * aligned.  With the codes a quantizer chose, sum(loss) / sum(opt_loss) - 1 is its gap. */
int nvfp4_block_loss(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                     const float* col_weight, const float* tensor_scale, const uint8_t* scales,
                     double* loss, void* stream);

/* Deterministic sum of v[0..n) in binary64 into the device double *out (a fixed reduction
 * order that depends on n only).  workspace: >= nvfp4_sum_workspace_bytes() bytes, 8-byte
 * aligned, no initialization. */
size_t nvfp4_sum_workspace_bytes(void);
int nvfp4_sum_f64(const double* v, int64_t n, double* out, void* workspace,
                  size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* NVFP4SS_H */
