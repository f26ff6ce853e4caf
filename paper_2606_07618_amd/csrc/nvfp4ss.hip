// NVFP4 ScaleSweep quantizer for AMD Instinct MI355X (gfx950): kernels and the C interface
// declared in include/nvfp4ss.h.
//
// Method (ScaleSweep, arXiv 2606.07618): with a global scale S fixed, every micro-block of
// normalized values y = x / S picks its FP8 E4M3 scale independently (Global Scale
// Selection).  ScaleSweep evaluates the block loss of Eq. (weighted_quantization_loss) at
// every E4M3 bit pattern in a short window around I(s_base^FP8) (Lemmas 1-3; the window
// summary at the end of the Block Scale Lower Bound paragraph) and keeps the argmin.
//
// Design for gfx950:
//  * One lane owns 16 consecutive elements; a micro-block of n elements is n/16 adjacent
//    lanes.  Everything per block (max, window, argmin) lives in registers; partial losses
//    of multi-lane blocks are combined with ds_swizzle exchanges.
//  * The FP4 rounding of two elements is one v_cvt_scalef32_pk_fp4_f32 (round to nearest
//    even onto E2M1 of src / 2^exponent(scale), saturating at 6) and the decode back one
//    v_cvt_scalef32_pk_f32_fp4.  A scale s = M 2^E (M in [1, 2)) is applied as u = |y| / M,
//    computed once and shared by the codes c, c+8, c+16 (same M, exponent +1, +2), and the
//    conversion's power-of-two scale 2^E.
//  * The sweep scores candidates in binary32 with the quotient |y| * (1/M) rounded once, so
//    an element within about an ulp of an FP4 midpoint may round the other way.  That moves a
//    loss by at most ~4e-6 of itself; candidates within a relative band of 2^-14 of the best
//    are re-scored exactly in binary64 in the order the definition sums them, which makes the
//    chosen code the exact argmin (smallest code on a tie).
//  * Exact roundings use exactly rounded quotients: y = RN32(x / S) and u = RN32(y / M) come
//    from a multiply by the correctly rounded reciprocal and one fused-multiply-add
//    correction (Markstein), exact when no intermediate underflows; tiny inputs fall back to
//    IEEE division.  RN32(y / M) then rounds to the same E2M1 value as y / M itself, because
//    an E2M1 midpoint times M has few enough bits that a 24-bit y cannot lie within half an
//    ulp of the quotient's midpoint without hitting it.
//  * The dynamic global scale needs max |x| first: a streaming kernel writes one maximum per
//    workgroup (at most 256) into the workspace, a one-wave kernel folds them into S and 1/S,
//    and the quantization kernel reads those two words.  Kernel boundaries order the passes.
//    Measured alternatives were slower: folding the partials in every quantization workgroup
//    (its prologue latency), and a last-arriving-workgroup fold in the reduction kernel (an
//    L2 write-back per workgroup for the release; with a full fence, also an L2 invalidate).
#include <hip/hip_runtime.h>

#include <float.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "nvfp4ss.h"

namespace {

constexpr int kThreads = 256;
constexpr int kLaneElems = 16;

enum Method { kAbsMax = 0, kFourSix = 1, kSweepMse = 2, kSweepWmse = 3, kWindowMse = 4, kWindowWmse = 5 };

// Workspace words: one |x|-maximum bit pattern per workgroup of the reduction pass, then S
// and 1/S; from word kSlotWord0 on, 64 |x|-maximum slots, each on its own 128-byte line,
// which the workgroups of the quantization kernel of the preceding tensor of a batched call
// raise atomically (slot = workgroup index mod 64).  Atomics on one line serialize (about
// 11 ns apiece measured on MI355X, i.e. 160 us for one per workgroup of a 14336-workgroup
// grid); spread over 64 lines they cost nothing measurable.
constexpr int kMaxPartials = 256;
constexpr int kWsScale = kMaxPartials, kWsRecip = kMaxPartials + 1;
constexpr int kSlotWord0 = 512, kSlotStride = 32, kSlots = 64;
constexpr size_t kWorkspaceBytes = (kSlotWord0 + kSlots * kSlotStride) * sizeof(uint32_t);


// Candidate band for the exact re-scoring (relative, plus an absolute floor for losses that
// underflow binary32).
constexpr float kBand = 0x1p-14f;
constexpr float kBandAbs = 0x1p-120f;

typedef float float2v __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------------------
// Formats.
// ---------------------------------------------------------------------------------------

// E4M3 code c (0..126) -> value.  Normal codes (c >= 8) have binary32 exponent field
// (c >> 3) + 120 and the top three mantissa bits c & 7, which is (c << 20) + (120 << 23);
// subnormal codes are c * 2^-9.
__device__ __forceinline__ float e4m3_value(int c) {
    return c >= 8 ? __uint_as_float(((uint32_t)c << 20) + 0x3C000000u) : (float)c * 0x1p-9f;
}

// Per-code constants, kept in LDS: s = M 2^E with M in [1, 2); rM = RN32(1 / M); cvs is the
// conversion scale (any value with exponent E; 1 for the zero code).
struct Scale {
    float M, rM, s, cvs;
};

// The table covers codes -16..143 so that a window's candidates index it without clamping.
// Codes that are not candidates get NaN in M, rM and cvs, so their loss comes out NaN and
// loses every comparison: codes outside 0..126, and code 0 unless the zero scale is allowed
// (AbsMax and 4/6 may pick it; a ScaleSweep window starts at code 1).
constexpr int kTabLo = 16, kTabSize = 160;

struct ScaleTable {
    Scale e[kTabSize];
};

constexpr float pow2(int k) {
    float r = 1.0f;
    for (; k > 0; --k) r *= 2.0f;
    for (; k < 0; ++k) r *= 0.5f;
    return r;
}

// Built at compile time (all steps exact except 1/M, which constant folding rounds to
// nearest even): E4M3 code c = a*8 + b has value 2^(a-7) (1 + b/8) for a > 0 and
// 2^-6 (b/8) for a = 0 (Appendix A with e = 4, m = 3).
template <bool ZERO_SCALE>
constexpr ScaleTable make_scale_table() {
    ScaleTable t{};
    const float nan = __builtin_nanf("");
    for (int i = 0; i < kTabSize; ++i) {
        const int c = i - kTabLo;
        Scale e{nan, nan, nan, nan};
        if (c >= 0 && c <= 126) {
            const int a = c >> 3, b = c & 7;
            const float s = a ? pow2(a - 7) * (1.0f + (float)b / 8.0f) : pow2(-6) * ((float)b / 8.0f);
            e.s = s;
            if (c == 0) {
                if (ZERO_SCALE) {
                    e.M = 0.0f;
                    e.rM = 0.0f;
                    e.cvs = 1.0f;
                }
            } else {
                float M = s;                       // significand of s in [1, 2)
                while (M >= 2.0f) M *= 0.5f;
                while (M < 1.0f) M *= 2.0f;
                e.M = M;
                e.rM = 1.0f / M;
                e.cvs = s;
            }
        }
        t.e[i] = e;
    }
    return t;
}

__device__ constexpr ScaleTable kSweepTable = make_scale_table<false>();
__device__ constexpr ScaleTable kNearestTable = make_scale_table<true>();

// Copies the table into LDS (threads 0..159); the caller synchronizes before reading it.
template <bool ZERO_SCALE>
__device__ __forceinline__ void fill_scale_table(Scale* tab_all) {
    if (threadIdx.x < kTabSize)
        tab_all[threadIdx.x] = (ZERO_SCALE ? kNearestTable : kSweepTable).e[threadIdx.x];
}

__device__ __forceinline__ int clamp_code(int c) { return c < 0 ? 0 : (c > 126 ? 126 : c); }

// Largest code c with div * E4M3(c) <= v (round-down onto the FP8 grid of v / div), exact: an
// estimate from the bits of v * (1/div) is off by at most one code and is fixed with exact
// comparisons (div * E4M3(c) has at most six significant bits).
__device__ __forceinline__ int floor_code(float v, float div, float rdiv, const Scale* tab) {
    const float t = v * rdiv;
    int c = t >= 0x1p-6f ? (int)(__float_as_uint(t) >> 20) - 960 : (int)(t * 512.0f);
    c = clamp_code(c);
    if (c > 0 && div * tab[c].s > v) c--;
    if (c < 126 && div * tab[c + 1].s <= v) c++;
    return c;
}

// Round-to-nearest-even code of v / div from its round-down code cf; saturates at 126.
__device__ __forceinline__ int nearest_code(float v, float div, int cf, const Scale* tab) {
    if (cf >= 126) return 126;
    const float mid = 0.5f * div * (tab[cf].s + tab[cf + 1].s);   // exact
    return (v > mid || (v == mid && ((cf + 1) & 1) == 0)) ? cf + 1 : cf;
}

// ---------------------------------------------------------------------------------------
// Lane exchanges inside groups of 2 / 4 / 8 lanes (ds_swizzle, bit-mask mode: xor).
// ---------------------------------------------------------------------------------------

template <int XOR>
__device__ __forceinline__ float swz_xor(float v) {
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), (XOR << 10) | 0x1F));
}

template <int LPB>
__device__ __forceinline__ float group_sum(float v) {
    if (LPB >= 2) v += swz_xor<1>(v);
    if (LPB >= 4) v += swz_xor<2>(v);
    if (LPB >= 8) v += swz_xor<4>(v);
    return v;
}

template <int LPB>
__device__ __forceinline__ float group_max(float v) {
    if (LPB >= 2) v = fmaxf(v, swz_xor<1>(v));
    if (LPB >= 4) v = fmaxf(v, swz_xor<2>(v));
    if (LPB >= 8) v = fmaxf(v, swz_xor<4>(v));
    return v;
}

// ---------------------------------------------------------------------------------------
// Loads.
// ---------------------------------------------------------------------------------------

template <typename In>
struct Loader;

template <>
struct Loader<float> {
    static __device__ __forceinline__ void load(const float* p, float (&v)[kLaneElems]) {
        const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float4 t = q[k];
            v[4 * k] = t.x;
            v[4 * k + 1] = t.y;
            v[4 * k + 2] = t.z;
            v[4 * k + 3] = t.w;
        }
    }
};

template <>
struct Loader<uint16_t> {   // bfloat16 bit patterns; widening to binary32 is exact
    static __device__ __forceinline__ void load(const uint16_t* p, float (&v)[kLaneElems]) {
        const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const uint4 t = q[k];
            const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                v[8 * k + 2 * j] = __uint_as_float(w[j] << 16);
                v[8 * k + 2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
            }
        }
    }
};

__device__ __forceinline__ void load_weights(const float* p, float (&w)[kLaneElems]) {
    const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float4 t = q[k];
        w[4 * k] = t.x;
        w[4 * k + 1] = t.y;
        w[4 * k + 2] = t.z;
        w[4 * k + 3] = t.w;
    }
}

// ---------------------------------------------------------------------------------------
// SwiGLU producer of the fused online quantizer: h = bf16(RN(silu(g) * u)).
// ---------------------------------------------------------------------------------------

// e^x in binary32 with every step fixed, so that a plain implementation reproduces it bit for
// bit: 0 below -80 (1 + e^x then rounds to 1 anyway), +inf from 89; otherwise Cody-Waite
// reduction x = n ln2 + r (ln2 as 0.693145751953125 plus the rounded rest, two fused
// multiply-adds), the degree-6 Taylor polynomial with coefficients RN32(1/k!) in Horner form,
// and the exact scaling by 2^n (the result is normal for x >= -80).  At most ~4 ulps from e^x.
__device__ __forceinline__ float swiglu_exp(float x) {
    if (x < -80.0f) return 0.0f;
    if (x >= 89.0f) return __builtin_inff();
    const float n = __builtin_rintf(x * 0x1.715476p+0f);   // RN32(1 / ln 2)
    float r = fmaf(-n, 0x1.62e4p-1f, x);
    r = fmaf(-n, 0x1.7f7d1cp-20f, r);                      // RN32(ln 2 - 0.693145751953125)
    float q = 0x1.6c16c2p-10f;                             // 1/720
    q = fmaf(q, r, 0x1.111112p-7f);                        // 1/120
    q = fmaf(q, r, 0x1.555556p-5f);                        // 1/24
    q = fmaf(q, r, 0x1.555556p-3f);                        // 1/6
    q = fmaf(q, r, 0.5f);
    q = fmaf(q, r, 1.0f);
    q = fmaf(q, r, 1.0f);
    return ldexpf(q, (int)n);
}

// The bfloat16 bit pattern (round to nearest even) of silu(g) * u = RN(RN(g / RN(1 + e^-g)) u),
// with a correctly rounded division.  Finite inputs.
__device__ __forceinline__ uint32_t swiglu_bf16(float g, float u) {
    const float d = 1.0f + swiglu_exp(-g);
    const float h = __fdiv_rn(g, d) * u;
    const uint32_t b = __float_as_uint(h);
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// The 16 producer outputs of one lane (bfloat16 values widened to binary32, exactly).
__device__ __forceinline__ void swiglu_lane(const uint16_t* gate, const uint16_t* up, float (&h)[kLaneElems]) {
    float g[kLaneElems], u[kLaneElems];
    Loader<uint16_t>::load(gate, g);
    Loader<uint16_t>::load(up, u);
#pragma unroll
    for (int i = 0; i < kLaneElems; ++i) h[i] = __uint_as_float(swiglu_bf16(g[i], u[i]) << 16);
}

// ---------------------------------------------------------------------------------------
// Block loss of one candidate scale, binary32 (fast screen).
// ---------------------------------------------------------------------------------------

// A register whose value does not matter: the FP4 conversion writes one byte of its
// destination and keeps the other three from this operand, and only that byte is read back.
__device__ __forceinline__ uint32_t any_bits() {
    uint32_t v;
    asm volatile("" : "=v"(v));
    return v;
}

// u[i] ~ |y_i| / M (rounded once); the conversion divides by 2^E exactly and rounds to E2M1;
// its decode gives g 2^E and e = |y| - (g 2^E) M is formed with one fused multiply-add.
template <bool WEIGHTED>
__device__ __forceinline__ float cand_loss(const float (&u)[kLaneElems], const float (&y)[kLaneElems],
                                           const float (&w)[kLaneElems], float cvs, float M) {
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
    for (int i = 0; i < kLaneElems; i += 2) {
        const uint32_t p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(any_bits(), u[i], u[i + 1], cvs, 0);
        const float2v g = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(p, cvs, 0);
        const float e0 = fmaf(-g.x, M, fabsf(y[i]));
        const float e1 = fmaf(-g.y, M, fabsf(y[i + 1]));
        if (WEIGHTED) {
            acc0 = fmaf(w[i] * e0, e0, acc0);
            acc1 = fmaf(w[i + 1] * e1, e1, acc1);
        } else {
            acc0 = fmaf(e0, e0, acc0);
            acc1 = fmaf(e1, e1, acc1);
        }
    }
    return acc0 + acc1;
}

// Losses of the window candidates d, d + 8, d + 16 (those below NC), normal codes only: the
// three share the significand M, so each element's quotient u = |y| * (1/M) is formed once
// and fed to the three conversions (scales 2^E, 2^(E+1), 2^(E+2)).  Element-major order keeps
// two quotients live instead of sixteen.  Each loss is the same binary32 operation sequence
// as cand_loss (even and odd elements in two chains, added at the end), so the values are
// bit-identical; a code past 126 has NaN in M and cvs and scores NaN as there.
template <bool WEIGHTED, int LPB, int NC>
__device__ __forceinline__ void significand_group_losses(const float (&y)[kLaneElems],
                                                         const float (&w)[kLaneElems],
                                                         const Scale* tab, int cb, int d,
                                                         float (&J)[NC], int dmin = 0, int dlim = NC) {
    // members d + 8k below dmin or at dlim and above are left out (and keep their J)
    constexpr int KMAX = (NC + 7) / 8;
    const float rM = tab[cb + d].rM;
    float M[KMAX], cvs[KMAX], acc0[KMAX], acc1[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
        if (d + 8 * k < dlim && d + 8 * k >= dmin) {
            M[k] = tab[cb + d + 8 * k].M;
            cvs[k] = tab[cb + d + 8 * k].cvs;
        }
        acc0[k] = 0.f;
        acc1[k] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < kLaneElems; i += 2) {
        float u0 = fabsf(y[i]) * rM, u1 = fabsf(y[i + 1]) * rM;
        // not rematerializable: the compiler would otherwise recompute them per candidate
        asm volatile("" : "+v"(u0), "+v"(u1));
#pragma unroll
        for (int k = 0; k < KMAX; ++k) {
            if (d + 8 * k >= dlim || d + 8 * k < dmin) continue;
            const uint32_t p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(any_bits(), u0, u1, cvs[k], 0);
            const float2v g = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(p, cvs[k], 0);
            const float e0 = fmaf(-g.x, M[k], fabsf(y[i]));
            const float e1 = fmaf(-g.y, M[k], fabsf(y[i + 1]));
            if (WEIGHTED) {
                acc0[k] = fmaf(w[i] * e0, e0, acc0[k]);
                acc1[k] = fmaf(w[i + 1] * e1, e1, acc1[k]);
            } else {
                acc0[k] = fmaf(e0, e0, acc0[k]);
                acc1[k] = fmaf(e1, e1, acc1[k]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
        if (d + 8 * k < dlim && d + 8 * k >= dmin) J[d + 8 * k] = group_sum<LPB>(acc0[k] + acc1[k]);
}

// The unweighted losses with the instruction order fixed by hand.  gfx950 issues two
// consecutive VALU instructions of a wave together when they are independent and read no
// common register; the compiler emits each element-candidate as a dependent chain
// (conversion, decode, error, accumulate), which leaves that pairing mostly unused.  Here the
// two candidates of a significand group (codes d and d + 8) are interleaved so that
// neighbours are independent and share no operand; a lone candidate keeps M in a second
// register for its odd elements.  Per element pair: one block with both conversions and
// decodes, one with the errors e = |y| - g M (a fused multiply-add) and the accumulations
// acc += e e.  The operations and their order per accumulator are those of
// significand_group_losses, so the values are bit-identical.  Plain VALU instructions need no
// wait states between them, and a conversion or decode may read a VALU result of the
// previous instruction on gfx950.  (The weighted loss gains nothing from this order and
// keeps the compiler's.)
template <int LPB, int NC>
__device__ __forceinline__ void significand_group_losses_sched(const float (&y)[kLaneElems],
                                                               const Scale* tab, int cb, int d,
                                                               float (&J)[NC]) {
    const float rM = tab[cb + d].rM;
    const float m0 = tab[cb + d].M;
    if (d + 8 < NC) {
        const float m1 = tab[cb + d + 8].M;   // equal to m0, or NaN past code 126
        const float s0 = tab[cb + d].cvs, s1 = tab[cb + d + 8].cvs;
        float a00 = 0.f, a01 = 0.f, a10 = 0.f, a11 = 0.f;   // [candidate][element parity]
#pragma unroll
        for (int i = 0; i < kLaneElems; i += 2) {
            const float u0 = fabsf(y[i]) * rM, u1 = fabsf(y[i + 1]) * rM;
            uint32_t p0, p1;
            float2v g0, g1;
            asm volatile(
                "v_cvt_scalef32_pk_fp4_f32 %[p0], %[u0], %[u1], %[s0]\n\t"
                "v_cvt_scalef32_pk_fp4_f32 %[p1], %[u0], %[u1], %[s1]\n\t"
                "v_cvt_scalef32_pk_f32_fp4 %[g0], %[p0], %[s0]\n\t"
                "v_cvt_scalef32_pk_f32_fp4 %[g1], %[p1], %[s1]"
                : [p0] "=&v"(p0), [p1] "=&v"(p1), [g0] "=&v"(g0), [g1] "=&v"(g1)
                : [u0] "v"(u0), [u1] "v"(u1), [s0] "v"(s0), [s1] "v"(s1));
            float T0, T1;   // errors e_cp (candidate c, element parity p)
            asm volatile(
                "v_fma_f32 %[T0], -%[g0x], %[m0], |%[y0]|\n\t"    // e00
                "v_fma_f32 %[T1], -%[g1y], %[m1], |%[y1]|\n\t"    // e11
                "v_fmac_f32 %[a00], %[T0], %[T0]\n\t"
                "v_fmac_f32 %[a11], %[T1], %[T1]\n\t"
                "v_fma_f32 %[T0], -%[g0y], %[m0], |%[y1]|\n\t"    // e01
                "v_fma_f32 %[T1], -%[g1x], %[m1], |%[y0]|\n\t"    // e10
                "v_fmac_f32 %[a01], %[T0], %[T0]\n\t"
                "v_fmac_f32 %[a10], %[T1], %[T1]"
                : [T0] "=&v"(T0), [T1] "=&v"(T1),
                  [a00] "+v"(a00), [a01] "+v"(a01), [a10] "+v"(a10), [a11] "+v"(a11)
                : [g0x] "v"(g0.x), [g0y] "v"(g0.y), [g1x] "v"(g1.x), [g1y] "v"(g1.y),
                  [m0] "v"(m0), [m1] "v"(m1), [y0] "v"(y[i]), [y1] "v"(y[i + 1]));
        }
        J[d] = group_sum<LPB>(a00 + a01);
        J[d + 8] = group_sum<LPB>(a10 + a11);
    } else {
        float m1;
        asm volatile("v_mov_b32 %0, %1" : "=v"(m1) : "v"(m0));   // M in a second register
        const float s0 = tab[cb + d].cvs;
        float a00 = 0.f, a01 = 0.f;
#pragma unroll
        for (int i = 0; i < kLaneElems; i += 2) {
            const float u0 = fabsf(y[i]) * rM, u1 = fabsf(y[i + 1]) * rM;
            uint32_t p0;
            float2v g0;
            asm volatile(
                "v_cvt_scalef32_pk_fp4_f32 %[p0], %[u0], %[u1], %[s0]\n\t"
                "v_cvt_scalef32_pk_f32_fp4 %[g0], %[p0], %[s0]"
                : [p0] "=&v"(p0), [g0] "=&v"(g0)
                : [u0] "v"(u0), [u1] "v"(u1), [s0] "v"(s0));
            float e00, e01;
            asm volatile(
                "v_fma_f32 %[e00], -%[g0x], %[m0], |%[y0]|\n\t"
                "v_fma_f32 %[e01], -%[g0y], %[m1], |%[y1]|\n\t"
                "v_fmac_f32 %[a00], %[e00], %[e00]\n\t"
                "v_fmac_f32 %[a01], %[e01], %[e01]"
                : [e00] "=&v"(e00), [e01] "=&v"(e01), [a00] "+v"(a00), [a01] "+v"(a01)
                : [g0x] "v"(g0.x), [g0y] "v"(g0.y), [m0] "v"(m0), [m1] "v"(m1),
                  [y0] "v"(y[i]), [y1] "v"(y[i + 1]));
        }
        J[d] = group_sum<LPB>(a00 + a01);
    }
}

// ---------------------------------------------------------------------------------------
// Weighted ScaleSweep with provably losing candidates skipped.
// ---------------------------------------------------------------------------------------

// The (block, candidate) items of a wave that the in-place sweep leaves to a shared pass,
// compacted block by block: the owner block's first lane in bits 5:0, candidate code in bits
// 12:6; each slot then receives its item's loss.  A block has at most 8 items at n = 16 (64
// blocks per wave) and 11 at n = 128 (window -11..7; 8 blocks per wave); the 64 slots past the
// most a wave can hold take the writes that land past the list's end.  Beside the list, every lane's |y|
// (4 x 16 bytes, stored transposed: chunk k of lane L at ay[k][L], so that the stores are
// contiguous across the wave), read back by the lanes that score its items.
constexpr int kItemSlots = 64 * 8 + 64;
struct PrunedLds {
    uint32_t item[kThreads / 64][kItemSlots];
    float4 ay[kThreads / 64][4][64];
};

__device__ __forceinline__ float bperm(int src_lane, float v) {
    return __int_as_float(__builtin_amdgcn_ds_bpermute(src_lane << 2, __float_as_int(v)));
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// E4M3 value of a normal code c (8..126) from its bits, as e4m3_value without the subnormal case.
__device__ __forceinline__ float e4m3_normal(int c) {
    return __uint_as_float(((uint32_t)c << 20) + 0x3C000000u);
}

// Losses J[d] of the WMSE window (codes cb + d, d = 0..NC-1, offsets -L..7 with L = NC - 8; all
// codes normal), for blocks of n = 16 LPB elements on LPB adjacent lanes.
//
// Offsets -1..6 (d = L-1..L+6) are scored in place for every block.  The other candidates are
// scored only where they can still be the window's argmin:
//  * Lower candidates d < L-1 (offsets -L..-2): their scale s is below s0 <= max|y| / 6, so the
//    block's largest element saturates to 6 s and its term alone, w1 (y1 - 6 s)^2, bounds the
//    candidate's loss from below.  That term is computed in the operation order the sweep uses
//    for it (e = RN(y1 - 6 s), which the sweep's fused multiply-add also yields; then
//    RN(RN(w1 e) e)), and a binary32 sum of non-negative terms accumulated with fused
//    multiply-adds is never below any one of its products, so the sweep's loss of d is >= the
//    bound (w1 is the weight of any one element with |y| = max|y|).  The bound grows as
//    s falls, so the candidates a block keeps are the top ones, d = dk .. L-2, and dk comes from
//    a binary search.
//  * Offset +7 (d = NC-1, code c0 + 7 >= 23): its half is offset -1, an E4M3 value of the window.
//    When 3.5 s > max|y|, every element rounds at s to a point of the half scale's grid (the
//    Block Scale Upper Bound lemma), so its exact loss is >= that of offset -1, which wins a
//    tie as the smaller code: +7 cannot be the argmin.  Otherwise the largest element's term,
//    formed exactly as the sweep forms it, bounds its loss as above.
// A candidate whose bound exceeds the best in-place loss by more than the re-scoring band (or
// that the lemma rules out) can be neither the binary32 minimum nor inside the band, nor the
// exact argmin, so skipping it (loss +inf) leaves the argmin and the band decisions exactly as
// with the full sweep.
//
// The kept (block, candidate) items of the wave (on Llama-like weights about 0.8 per block at
// n = 16 and 4.9 at n = 128: one or two rounds, or about five) go into one list, entered by each
// block's first lane, and are scored by all lanes together, LPB lanes per item.  Lane j of an
// item's group reads part j of the owner block: its |y| from LDS (four 16-byte loads) and its
// weights, at n = 16 from memory (four 16-byte loads, cache hits: the owner has just loaded
// them), at n > 16 from the owner lane's registers (lane permutes, which keep memory latency
// out of the several rounds).  The group's partial losses are summed as in the sweep and the
// first lane leaves the loss in the item's slot: the losses are the operation sequence of
// cand_loss, bit-identical to in-place scoring.  Called in uniform control flow with all 64
// lanes of the wave running; wblk is the offset of the block's weights in colw in units of n
// elements, part the lane's part of its block.
template <int NC, int LPB>
__device__ __forceinline__ void pruned_wmse_losses(const float (&y)[kLaneElems], const float (&w)[kLaneElems],
                                                   float ymax, bool active, const Scale* tab, int cb,
                                                   float (&J)[NC], PrunedLds& lds, const float* colw,
                                                   uint32_t wblk, int part) {
    constexpr int L = NC - 8;                        // lowest offset -L
    constexpr int kLow = L - 1;                      // lower candidates d = 0..kLow-1
    constexpr int kTop = NC - 1;                     // d of offset +7
    constexpr int kBits = kLow < 8 ? 3 : 4;          // binary digits of a lower count 0..kLow
    constexpr int kG = 64 / LPB;                     // blocks (items of a round) per wave
    static_assert(L >= 8 && kLow + 1 <= 16, "WMSE windows -8..7 / -11..7");
    static_assert(kG * (kLow + 1) + kLow <= kItemSlots, "the writes past a list stay in it");
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        significand_group_losses<true, LPB, NC>(y, w, tab, cb, r, J, kLow, kTop);
        // finished here, before the next group's quotients are formed: one group live at a time
#pragma unroll
        for (int d = r; d < NC; d += 8)
            if (d >= kLow && d < kTop) asm volatile("" : "+v"(J[d]));
    }
    asm volatile("" : "+v"(ymax));                  // the bounds below are formed after the sweep
    float jb = J[kLow];
#pragma unroll
    for (int d = kLow + 1; d < kTop; ++d) jb = fminf(jb, J[d]);   // NaN codes past 126 drop out
    // inactive lanes (past the last block) keep nothing
    const float thr = active ? fmaf(jb, kBand, jb) + kBandAbs : -__builtin_inff();
    float w1 = 0.f;                                  // weight of an element with |y| = max|y|
#pragma unroll
    for (int i = 0; i < kLaneElems; ++i) w1 = fabsf(y[i]) == ymax ? w[i] : w1;
    w1 = group_max<LPB>(w1);                         // lanes without such an element offer 0

    // lower candidates: d is kept iff its bound is not above thr; the kept ones are d >= dk
    auto low_keep = [&](int d) {
        const float e = ymax - 6.0f * e4m3_normal(cb + d);   // 6 s is exact
        const float t = w1 * e;
        return !(t * e > thr);
    };
    int dk = 0, dhi = kLow;                          // first kept d in [dk, dhi] (kLow: none)
#pragma unroll
    for (int it = 0; it < kBits; ++it) {
        const int mid = (dk + dhi) >> 1;
        if (dk < dhi) {
            if (low_keep(mid)) dhi = mid;
            else dk = mid + 1;
        }
    }
    const uint32_t nlow = (uint32_t)(kLow - dk);
    // offset +7
    bool keep_top = false;
    {
        const int ct = cb + kTop;
        const Scale st = tab[ct];                    // NaN entries past code 126
        if (ct <= 126 && !(3.5f * st.s > ymax)) {
            const float u1 = ymax * st.rM;           // the sweep's quotient of this element
            const float2v g = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(
                __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(any_bits(), u1, u1, st.cvs, 0), st.cvs, 0);
            const float e = fmaf(-g.x, st.M, ymax);
            const float t = w1 * e;
            keep_top = !(t * e > thr);
        }
        keep_top = keep_top && active;
    }
    // each block's items are entered by its first lane; list positions from a prefix count over
    // the blocks (binary digits, by ballot; only first lanes vote, so the count of set lanes
    // below this lane is the count over the blocks before its block)
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const bool leader = part == 0;
    uint32_t* items = lds.item[wv];
    uint32_t pos = 0u, total = 0u;
#pragma unroll
    for (int b = 0; b < kBits; ++b) {
        const uint64_t m = __ballot(leader && ((nlow >> b) & 1u));
        pos += lanes_below(m) << b;
        total += (uint32_t)__popcll(m) << b;
    }
    {
        const uint64_t m = __ballot(leader && keep_top);
        pos += lanes_below(m);
        total += (uint32_t)__popcll(m);
    }
    // A block's items: offset +7 first when kept (t = 1), then the lower candidates from d =
    // kLow - 1 down.  Every block with items writes all kLow + 1 slots from its position, last
    // slot first; the slots past its own items are overwritten by the blocks that follow (their
    // writes of those slots come later, at smaller offsets), or lie past the end of the list.
    const uint32_t t = keep_top ? 1u : 0u;
    if (leader && nlow + t != 0u) {
        const uint32_t v0 = (uint32_t)lane | ((uint32_t)(cb + kLow - 1) << 6);
        uint32_t* mine = items + pos;
        // one store per slot, in this order (a wave's LDS stores complete in issue order; the
        // empty asm keeps the compiler from reordering or pairing them)
#pragma unroll
        for (int j = kLow; j >= 1; --j) {
            mine[j] = v0 + (t << 6) - ((uint32_t)j << 6);
            asm volatile("" ::: "memory");
        }
        mine[0] = keep_top ? (uint32_t)lane | ((uint32_t)(cb + kTop) << 6) : v0;
    }
    if (total != 0u) {                               // uniform
        const uint32_t g = (uint32_t)lane / LPB;     // this lane's item of a round, and its part
        const int jp = lane % LPB;
        // loss of the item in slot pidx, left there by the group's first lane (slots past total:
        // idle, never read); wload(q) gives weights 4q..4q+3 of this lane's part
        auto score = [&](uint32_t pidx, uint32_t it, auto wload) {
            const int src = (int)(it & 63u) + jp;    // the owner block's lane for this part
            const Scale sc = tab[(int)(it >> 6)];
            float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
            for (int h = 0; h < 2; ++h) {            // two halves of 8 elements
                float a[8], wo[8];
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const float4 v = lds.ay[wv][2 * h + k][src];
                    a[4 * k] = v.x;
                    a[4 * k + 1] = v.y;
                    a[4 * k + 2] = v.z;
                    a[4 * k + 3] = v.w;
                    const float4 q4 = wload(2 * h + k);
                    wo[4 * k] = q4.x;
                    wo[4 * k + 1] = q4.y;
                    wo[4 * k + 2] = q4.z;
                    wo[4 * k + 3] = q4.w;
                }
#pragma unroll
                for (int i = 0; i < 8; i += 2) {
                    const float u0 = a[i] * sc.rM, u1 = a[i + 1] * sc.rM;
                    const uint32_t pk = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(any_bits(), u0, u1, sc.cvs, 0);
                    const float2v gv = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pk, sc.cvs, 0);
                    const float e0 = fmaf(-gv.x, sc.M, a[i]);
                    const float e1 = fmaf(-gv.y, sc.M, a[i + 1]);
                    acc0 = fmaf(wo[i] * e0, e0, acc0);
                    acc1 = fmaf(wo[i + 1] * e1, e1, acc1);
                }
            }
            const float loss = group_sum<LPB>(acc0 + acc1);
            if (jp == 0) items[pidx] = __float_as_uint(loss);
        };
        auto stage_ay = [&]() {
#pragma unroll
            for (int k = 0; k < 4; ++k)
                lds.ay[wv][k][lane] = make_float4(fabsf(y[4 * k]), fabsf(y[4 * k + 1]), fabsf(y[4 * k + 2]),
                                                  fabsf(y[4 * k + 3]));
        };
        auto wave_sync = []() {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        };
        if constexpr (LPB == 1) {
            // n = 16 (about one round per wave): the weights come from memory, where the owner
            // has just loaded them
            stage_ay();
            wave_sync();
#pragma unroll 1
            for (uint32_t r = 0; r < total; r += kG) {   // uniform; every lane takes an item or idles
                const uint32_t pidx = r + g;
                const uint32_t it = pidx < total ? items[pidx] : 0u;
                const uint32_t ob = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(it & 63u) << 2, (int)wblk);
                const float4* p4 = reinterpret_cast<const float4*>(colw + (uint64_t)ob * 16);
                score(pidx, it, [&](int q) { return p4[q]; });
            }
        } else {
            // n > 16: the weights come from the owner lane's registers
            stage_ay();
            wave_sync();
#pragma unroll 1
            for (uint32_t r = 0; r < total; r += kG) {   // uniform; every group takes an item or idles
                const uint32_t pidx = r + g;
                const uint32_t it = pidx < total ? items[pidx] : 0u;
                const int src = (int)(it & 63u) + jp;
                score(pidx, it, [&](int q) {
                    return make_float4(bperm(src, w[4 * q]), bperm(src, w[4 * q + 1]),
                                       bperm(src, w[4 * q + 2]), bperm(src, w[4 * q + 3]));
                });
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // every lane of a block reads the block's losses (pos, dk, nlow, keep_top are block-wide)
    const uint32_t bpos = LPB == 1 ? pos : (uint32_t)__shfl((int)pos, lane - part, 64);
    const uint32_t* mine = items + bpos;
#pragma unroll
    for (int d = 0; d < kLow; ++d)
        J[d] = d >= dk ? __uint_as_float(mine[t + (uint32_t)(kLow - 1 - d)]) : __builtin_inff();
    J[kTop] = keep_top ? __uint_as_float(mine[0]) : __builtin_inff();
}

// max(|a|, |b|, c) in one instruction (abs source modifiers); c >= 0.  The inputs come from
// arithmetic, so none is a signaling NaN and no canonicalization is needed.
__device__ __forceinline__ float max3_abs(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, |%1|, |%2|, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// Exactly rounded u = RN32(v / M) for M in [1, 2) with rM = RN32(1 / M) (Markstein): the
// remainder u M - v is exact in one fused multiply-add and corrects u once.  Written as
// u - (u M - v) rM so that a zero quotient keeps the sign of v (-0 + -0 = -0), which the
// nibble's sign bit needs; with M = rM = 0 (the zero scale) it returns +-0 as well.
__device__ __forceinline__ float div_by_significand(float v, float M, float rM) {
    const float u = v * rM;
    const float r = fmaf(u, M, -v);
    return fmaf(-r, rM, u);
}

// Exact block loss in binary64, summed in element order 0..n-1 across the block's lanes:
// e = |y| - g s exactly, term = e * e (times the weight), J = J + term.
template <bool WEIGHTED, int LPB>
__device__ double exact_loss(const float (&y)[kLaneElems], const float (&w)[kLaneElems], const Scale& sc,
                             int part, int group_base_lane) {
    double acc = 0.0;
#pragma unroll 1
    for (int l = 0; l < LPB; ++l) {
        if (part == l) {
#pragma unroll
            for (int i = 0; i < kLaneElems; ++i) {
                float a = fabsf(y[i]);
                float wi = w[i];
                // keeps the binary64 conversions of |y| and w inside this rarely taken path
                // (hoisted out of the candidate loop they would hold 64 registers everywhere)
                asm volatile("" : "+v"(a), "+v"(wi));
                const float u = div_by_significand(a, sc.M, sc.rM);
                const uint32_t p = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, u, 0.f, sc.cvs, 0);
                const float2v g = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(p, sc.cvs, 0);
                const float gs = g.x * sc.M;                       // exact
                const double e = (double)a - (double)gs;
                double t = e * e;
                if (WEIGHTED) t = (double)wi * t;
                acc = acc + t;
            }
        }
        if (LPB > 1) acc = __shfl(acc, group_base_lane + l, 64);
    }
    return acc;
}

// Whether the scales s0 = M 2^E and s1 = M 2^(E+1) (codes c and c + 8) reconstruct every
// element of the block identically: the exact E2M1 rounding of u = RN32(|y| / M) (the quotient
// the emit uses) at both scales gives the same g 2^E for all n elements.  Then every term of the
// loss, weighted or not, is the same for both codes, and so are the two sums.
template <int LPB>
__device__ bool same_reconstruction(const float (&y)[kLaneElems], const Scale& s0, const Scale& s1) {
    uint32_t differ = 0u;
#pragma unroll
    for (int i = 0; i < kLaneElems; i += 2) {
        const float u0 = div_by_significand(fabsf(y[i]), s0.M, s0.rM);
        const float u1 = div_by_significand(fabsf(y[i + 1]), s0.M, s0.rM);
        const float2v g0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(
            __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, u0, u1, s0.cvs, 0), s0.cvs, 0);
        const float2v g1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(
            __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, u0, u1, s1.cvs, 0), s1.cvs, 0);
        differ |= (__float_as_uint(g0.x) ^ __float_as_uint(g1.x)) | (__float_as_uint(g0.y) ^ __float_as_uint(g1.y));
    }
    return group_sum<LPB>(differ != 0u ? 1.0f : 0.0f) == 0.0f;
}

// ---------------------------------------------------------------------------------------
// Global scale: max |x| over the tensor.
// ---------------------------------------------------------------------------------------

__device__ __forceinline__ uint32_t absmax_bits(uint4 d, float) {
    uint32_t m = d.x & 0x7FFFFFFFu;
    m = max(m, d.y & 0x7FFFFFFFu);
    m = max(m, d.z & 0x7FFFFFFFu);
    return max(m, d.w & 0x7FFFFFFFu);
}

__device__ __forceinline__ uint32_t absmax_bits(uint4 d, uint16_t) {
    // bfloat16 pairs: |x| bits of both halves, placed as binary32 bit patterns
    uint32_t m = max((d.x << 16) & 0x7FFF0000u, d.x & 0x7FFF0000u);
    m = max(m, max((d.y << 16) & 0x7FFF0000u, d.y & 0x7FFF0000u));
    m = max(m, max((d.z << 16) & 0x7FFF0000u, d.z & 0x7FFF0000u));
    return max(m, max((d.w << 16) & 0x7FFF0000u, d.w & 0x7FFF0000u));
}

// S = RN32(amax / denom) with denom = RN32(6 D); an all-zero tensor gets 1, an underflowing
// quotient the smallest positive binary32, a non-finite input NaN.
__device__ __forceinline__ float global_scale(uint32_t amax_bits, float denom) {
    if (amax_bits >= 0x7F800000u) return __uint_as_float(0x7FC00000u);
    if (amax_bits == 0u) return 1.0f;
    const float s = __fdiv_rn(__uint_as_float(amax_bits), denom);
    return s == 0.0f ? FLT_TRUE_MIN : s;
}

template <typename In>
__global__ __launch_bounds__(kThreads) void amax_kernel(const In* __restrict__ x, int64_t nvec,
                                                        uint32_t* __restrict__ partials) {
    const uint4* v = reinterpret_cast<const uint4*>(x);
    uint32_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + 7 * stride < nvec; i += 8 * stride) {
        uint4 d[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) d[k] = v[i + k * stride];
#pragma unroll
        for (int k = 0; k < 8; ++k) m = max(m, absmax_bits(d[k], In()));
    }
    for (; i < nvec; i += stride) m = max(m, absmax_bits(v[i], In()));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
    __shared__ uint32_t part[kThreads / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) partials[blockIdx.x] = max(max(part[0], part[1]), max(part[2], part[3]));
}

// Folds the per-workgroup maxima into S and 1/S (one wave): S goes to the caller's output
// and, with 1/S, to the workspace words after the partials, for the quantization kernel.
// With zero_count > 0 it also clears the |x|-maximum slots of zero_count workspaces laid out
// zero_stride words apart from zero_base (the other tensors of a batched call).
__global__ __launch_bounds__(64) void scale_kernel(uint32_t* __restrict__ ws, int npart,
                                                   float denom, float* __restrict__ tensor_scale,
                                                   uint32_t* __restrict__ zero_base, int zero_count,
                                                   int64_t zero_stride) {
    for (int t = threadIdx.x; t < zero_count * kSlots; t += 64)
        zero_base[(t / kSlots) * zero_stride + kSlotWord0 + (t % kSlots) * kSlotStride] = 0u;
    uint32_t m = 0;
    for (int i = threadIdx.x; i < npart; i += 64) m = max(m, ws[i]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
    if (threadIdx.x == 0) {
        const float S = global_scale(m, denom);
        tensor_scale[0] = S;
        ws[kWsScale] = __float_as_uint(S);
        ws[kWsRecip] = __float_as_uint(__fdiv_rn(1.0f, S));
    }
}

__global__ void write_scale_kernel(float* tensor_scale, float S) { tensor_scale[0] = S; }

// ---------------------------------------------------------------------------------------
// Quantization kernel.
// ---------------------------------------------------------------------------------------

// Source of the global scale in the quantization kernel.
enum ScaleSource {
    kScaleStatic = 0,         // Params::S, Params::rS (given by the caller)
    kScaleWorkspace = 1,      // S and 1/S formed by scale_kernel earlier on the stream
    kScaleSlots = 2,          // the maximum of the workspace's |x| slots (raised atomically by
                              // the preceding kernel of a batched call), folded here
};

struct Params {
    int64_t nblocks;          // micro-blocks in the tensor
    uint32_t bpr;             // micro-blocks per row
    uint32_t bpr_magic;       // blk / bpr = (umulhi(blk, magic) + ((blk - hi) >> 1)) >> (shift - 1)
    uint32_t bpr_shift;
    int scale_src;            // where S comes from (ScaleSource)
    float S, rS;              // static global scale and its reciprocal
    float denom;              // 6 D, for kScaleSlots
    const uint32_t* ws;       // workspace of the dynamic path
    float* tensor_scale;      // static and slot paths: written once, by the first lane of the grid
    const uint4* nx;          // batched calls: the next tensor, whose |x| maximum every
    int64_t nx_vec;           //   workgroup reduces a share of (nx_per of its nx_vec 16-byte
    int64_t nx_per;           //   vectors) into nx_slots; nx_per = 0: no next tensor
    uint32_t* nx_slots;
    int win_tight;            // window variants: per-mantissa offsets (else win_lo..win_hi)
    int win_lo, win_hi;
    int swizzled;             // scales in 128 x 4 tiles (else row-major)
    const uint16_t* up;       // fused SwiGLU input: x is the gate, this the up projection
    uint32_t sw_kt;           // 4-column scale tiles per tile row
    uint32_t wgroups;         // importance vectors: row r uses ((r / wg_rows) mod wgroups)
    uint32_t wgr_magic, wgr_shift, wgn_magic, wgn_shift;   // dividers by wg_rows, wgroups
};

// n / d for the invariant divisor d behind (magic, shift) (shift 0: d = 1).
__device__ __forceinline__ uint32_t div_magic(uint32_t n, uint32_t magic, uint32_t shift) {
    if (shift == 0) return n;
    const uint32_t hi = __umulhi(n, magic);
    return (hi + ((n - hi) >> 1)) >> (shift - 1);
}

__device__ __forceinline__ uint32_t div_bpr(uint32_t n, const Params& p) {
    return div_magic(n, p.bpr_magic, p.bpr_shift);
}

// Index of the importance vector of a row: (row / wg_rows) mod wgroups.
__device__ __forceinline__ uint32_t weight_group(uint32_t row, const Params& p) {
    const uint32_t t = div_magic(row, p.wgr_magic, p.wgr_shift);
    return t - div_magic(t, p.wgn_magic, p.wgn_shift) * p.wgroups;
}

// Byte offset of the scale of row m, scale column k in the swizzled layout: the scale matrix,
// padded to multiples of 128 rows and 4 columns, is stored as 512-byte tiles of 128 x 4,
// tile-row-major; inside a tile row m sits at (m mod 32) * 16 + ((m / 32) mod 4) * 4 and column
// k at k mod 4 (the layout of vLLM's NVFP4 operators, used by the paper's operator benchmark).
__device__ __forceinline__ uint32_t swizzled_offset(uint32_t m, uint32_t k, uint32_t kt) {
    return ((m >> 7) * kt + (k >> 2)) * 512u + (m & 31u) * 16u + ((m >> 5) & 3u) * 4u + (k & 3u);
}

// Workgroups are dispatched to the 8 XCDs of the GPU round-robin (workgroup i to XCD i mod 8),
// and each XCD has its own L2.  This regrouping gives the workgroups of XCD x a contiguous
// eighth of the tiles (rows), so every workgroup that writes into one 512-byte scale tile of the
// swizzled layout (128 rows) runs on the same XCD: that L2 merges their 4-byte pieces into whole
// lines before they go to memory, instead of eight L2s writing partial lines.  Any grid size;
// a bijection on 0..grid-1.
constexpr uint32_t kXcds = 8;
__device__ __forceinline__ uint32_t xcd_tile(uint32_t i, uint32_t grid) {
    const uint32_t x = i % kXcds, j = i / kXcds;
    const uint32_t q = grid / kXcds, r = grid % kXcds;
    return x * q + min(x, r) + j;
}

template <int METHOD, int N>
struct Window {
    static constexpr int L = METHOD == kSweepMse
                                 ? (N == 16 ? 3 : N == 32 ? 5 : N == 64 ? 7 : 11)
                                 : (N == 128 ? 11 : 8);
    static constexpr int U = 7;
    static constexpr int NC = L + U + 1;
};

// Window variants of ScaleSweep (Tables 1 and 2; the sweep-range study of the Experiment
// section): the block sweeps the codes [lo, hi] = [c0 + lo_off, c0 + hi_off], each end clamped
// into 1..126, with per-mantissa offsets in the tight mode:
//   upper (Table 1, Lemmas 1-2 with alpha = 12/7, any objective and n): 7, or 6 for b >= 6;
//   lower (Table 2, Lemma 3, MSE with n = 16): 3 for b = 0 and b = 7, else 2; otherwise the
//   standard lower offset.
// The window has 1..126 codes and may differ between the lanes of a wave, so the candidate
// losses are not kept: a running minimum and second minimum of the keys decide the argmin and
// whether the band re-scoring is needed, and that rare path scores the candidates again.
template <bool WGT, int LPB>
__device__ int choose_window(const float (&y)[kLaneElems], const float (&w)[kLaneElems], float ymax,
                             const Scale* tab, const Params& p, int part, int group_base,
                             int std_lower, bool table2) {
    const int c0 = floor_code(ymax, 6.0f, 1.0f / 6.0f, tab);
    int lo_off = p.win_lo, hi_off = p.win_hi;
    if (p.win_tight) {
        const int b = c0 & 7;
        hi_off = b >= 6 ? 6 : 7;
        lo_off = table2 ? ((b == 0 || b == 7) ? -3 : -2) : -std_lower;
    }
    const int lo = min(max(c0 + lo_off, 1), 126);
    const int hi = min(max(c0 + hi_off, 1), 126);
    const int ncand = hi - lo + 1;
    uint32_t best1 = 0xFFFFFFFFu, best2 = 0xFFFFFFFFu;
    auto take = [&](float J, int j) {
        const uint32_t key = (__float_as_uint(J) & 0xFFFFFF80u) | (uint32_t)j;
        best2 = min(best2, max(best1, key));
        best1 = min(best1, key);
    };
    float u[kLaneElems];
    if (__all(lo >= 8)) {
        // normal codes only: lo + t, lo + t + 8, ... share the significand of lo + t
        for (int t = 0; t < 8 && __any(t < ncand); ++t) {
            const Scale st = tab[t < ncand ? lo + t : -kTabLo];        // -16: a NaN entry
#pragma unroll
            for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * st.rM;
            for (int j = t; __any(j < ncand); j += 8) {
                const Scale sj = tab[j < ncand ? lo + j : -kTabLo];
                take(group_sum<LPB>(cand_loss<WGT>(u, y, w, sj.cvs, sj.M)), j);
            }
        }
    } else {
        for (int j = 0; __any(j < ncand); ++j) {
            const Scale sj = tab[j < ncand ? lo + j : -kTabLo];
#pragma unroll
            for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * sj.rM;
            take(group_sum<LPB>(cand_loss<WGT>(u, y, w, sj.cvs, sj.M)), j);
        }
    }
    int dstar = (int)(best1 & 0x7Fu);
    const float j1 = __uint_as_float(best1 & 0xFFFFFF80u);
    const float bound = fmaf(j1, kBand, j1) + kBandAbs;
    const bool near = __uint_as_float(best2 & 0xFFFFFF80u) <= bound;
    if (__any(near)) {
        if (near) {      // every lane of a block takes the same path (its losses are shared)
            double jb = 0.0;
            int db = -1;
            for (int j = 0; j < ncand; ++j) {
                const Scale sj = tab[lo + j];
#pragma unroll
                for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * sj.rM;
                const float J = group_sum<LPB>(cand_loss<WGT>(u, y, w, sj.cvs, sj.M));
                if (__uint_as_float(__float_as_uint(J) & 0xFFFFFF80u) <= bound) {
                    const double jd = exact_loss<WGT, LPB>(y, w, sj, part, group_base);
                    if (db < 0 || jd < jb) {
                        jb = jd;
                        db = j;
                    }
                }
            }
            if (db >= 0) dstar = db;
        }
    }
    return dstar < ncand ? lo + dstar : lo;   // dstar >= ncand only if every loss is NaN
}

// Batched calls: every workgroup of a quantization grid also reads an equal share of the
// next tensor (at most 4 loads of 16 bytes per lane in flight, issued behind the tile's own
// loads) and each wave raises slot (4 * workgroup + wave) mod 64 of that tensor's workspace
// with one relaxed device-scope atomic maximum; the next kernel on the stream folds the slots
// after this grid has completed.  Spread this way the next tensor streams at a modest rate
// for the whole sweep; dedicated reducer workgroups at the head of the grid instead burst
// it at full bandwidth, queueing the first sweep tiles' loads and holding wave slots.
template <typename In>
__device__ __forceinline__ uint32_t next_share_max(const Params& p, uint32_t tile) {
    const int64_t v0 = (int64_t)tile * p.nx_per;
    const int64_t v1 = min(v0 + p.nx_per, p.nx_vec);
    uint32_t m = 0;
    for (int64_t v = v0 + threadIdx.x; v < v1; v += 4 * kThreads) {
        uint4 d[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            d[k] = v + k * kThreads < v1 ? p.nx[v + k * kThreads] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
        for (int k = 0; k < 4; ++k) m = max(m, absmax_bits(d[k], In()));
    }
    return m;
}

__device__ __forceinline__ void raise_next_slot(const Params& p, uint32_t tile, uint32_t m) {
    // wave maximum: xor exchanges inside 32-lane halves, then the two halves' lane 0
    m = max(m, (uint32_t)__builtin_amdgcn_ds_swizzle((int)m, (1 << 10) | 0x1F));
    m = max(m, (uint32_t)__builtin_amdgcn_ds_swizzle((int)m, (2 << 10) | 0x1F));
    m = max(m, (uint32_t)__builtin_amdgcn_ds_swizzle((int)m, (4 << 10) | 0x1F));
    m = max(m, (uint32_t)__builtin_amdgcn_ds_swizzle((int)m, (8 << 10) | 0x1F));
    m = max(m, (uint32_t)__builtin_amdgcn_ds_swizzle((int)m, (16 << 10) | 0x1F));
    m = max((uint32_t)__builtin_amdgcn_readlane((int)m, 0), (uint32_t)__builtin_amdgcn_readlane((int)m, 32));
    if ((threadIdx.x & 63) == 0 && m != 0u)
        __hip_atomic_fetch_max(p.nx_slots + ((tile * 4u + (threadIdx.x >> 6)) & (kSlots - 1)) * kSlotStride,
                               m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int METHOD, typename In, int N, bool SWIGLU = false>
__global__ __launch_bounds__(kThreads) void quant_kernel(const In* __restrict__ x,
                                                         const float* __restrict__ colw,
                                                         uint8_t* __restrict__ q,
                                                         uint8_t* __restrict__ scales, Params p) {
    constexpr int LPB = N / kLaneElems;
    constexpr bool WEIGHTED_OBJ = METHOD == kSweepWmse || METHOD == kFourSix || METHOD == kWindowWmse;
    __shared__ Scale tab_all[kTabSize];
    Scale* tab = tab_all + kTabLo;                 // tab[c] for codes c in -16..143
    // the workgroup's tile of this tensor; with swizzled scales, tiles are regrouped by XCD
    const uint32_t tile = p.swizzled ? xcd_tile(blockIdx.x, gridDim.x) : blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int64_t gtid = (int64_t)tile * kThreads + threadIdx.x;
    const int64_t blk = gtid / LPB;
    const int part = (int)(gtid % LPB);
    const int group_base = lane - part;
    const bool active = blk < p.nblocks;
    const int64_t blk_c = active ? blk : 0;   // inactive lanes run on block 0, store nothing

    // The tile's loads go out first; the table fill and the global-scale fold overlap them.
    float y[kLaneElems];
    if constexpr (SWIGLU) {           // the tensor is the producer's output, formed here
        static_assert(N == 16, "fused producer at block 16");
        swiglu_lane(reinterpret_cast<const uint16_t*>(x) + blk_c * N, p.up + blk_c * N, y);
    } else {
        Loader<In>::load(x + blk_c * N + part * kLaneElems, y);
    }
    float w[kLaneElems];
    const bool use_w = WEIGHTED_OBJ && colw != nullptr;
    uint32_t row = 0, kb = 0;         // the block's row and block column
    if (use_w || p.swizzled) {
        row = div_bpr((uint32_t)blk_c, p);
        kb = (uint32_t)blk_c - row * p.bpr;
    }
    // the block's weights in colw, in units of N elements: below rows * cols / N < 2^31
    uint32_t wblk = 0;
    if (use_w) {
        wblk = (p.wgroups > 1 ? weight_group(row, p) * p.bpr : 0u) + kb;
        load_weights(colw + (int64_t)wblk * N + part * kLaneElems, w);
    } else {
#pragma unroll
        for (int i = 0; i < kLaneElems; ++i) w[i] = 1.0f;
    }
    fill_scale_table<METHOD == kAbsMax || METHOD == kFourSix>(tab_all);
    if (p.nx_per > 0) raise_next_slot(p, tile, next_share_max<In>(p, tile));   // uniform
    __shared__ float s_scale[2];
    if (p.scale_src == kScaleSlots && threadIdx.x < 64) {
        // the slots were raised by the previous kernel on the stream: wave 0 folds them
        uint32_t m = p.ws[kSlotWord0 + threadIdx.x * kSlotStride];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
        if (threadIdx.x == 0) {
            const float Sg = global_scale(m, p.denom);
            s_scale[0] = Sg;
            s_scale[1] = __fdiv_rn(1.0f, Sg);
        }
    }
    __syncthreads();
    float S, rS;
    if (p.scale_src == kScaleWorkspace) {      // formed by scale_kernel, earlier on the stream
        S = __uint_as_float(p.ws[kWsScale]);
        rS = __uint_as_float(p.ws[kWsRecip]);
    } else {
        if (p.scale_src == kScaleSlots) {
            S = s_scale[0];
            rS = s_scale[1];
        } else {
            S = p.S;
            rS = p.rS;
        }
        if (tile == 0 && threadIdx.x == 0 && p.tensor_scale) p.tensor_scale[0] = S;
    }
    const bool fast_div = S >= 0x1p-26f && S <= 0x1p26f;

    {
    // ---- normalize y = RN32(x / S) -----------------------------------------------------
#pragma unroll
    for (int i = 0; i < kLaneElems; ++i) {
        const float xv = y[i];
        if (fast_div && fabsf(xv) >= 0x1p-74f) {
            y[i] = div_by_significand(xv, S, rS);    // exact for these ranges (Markstein)
        } else {
            y[i] = __fdiv_rn(xv, S);
        }
    }
    float ymax = 0.f;
#pragma unroll
    for (int i = 0; i < kLaneElems; i += 2) ymax = max3_abs(y[i], y[i + 1], ymax);
    ymax = group_max<LPB>(ymax);

    // ---- choose the block scale code ---------------------------------------------------
    int code;
    if (METHOD == kAbsMax) {
        const int cf = floor_code(ymax, 6.0f, 1.0f / 6.0f, tab);
        code = nearest_code(ymax, 6.0f, cf, tab);
    } else if (METHOD == kFourSix) {
        const int c6 = nearest_code(ymax, 6.0f, floor_code(ymax, 6.0f, 1.0f / 6.0f, tab), tab);
        const int c4 = nearest_code(ymax, 4.0f, floor_code(ymax, 4.0f, 0.25f, tab), tab);
        float u[kLaneElems];
        const Scale s6 = tab[c6], s4 = tab[c4];
#pragma unroll
        for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * s6.rM;
        float j6 = group_sum<LPB>(use_w ? cand_loss<true>(u, y, w, s6.cvs, s6.M)
                                        : cand_loss<false>(u, y, w, s6.cvs, s6.M));
#pragma unroll
        for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * s4.rM;
        float j4 = group_sum<LPB>(use_w ? cand_loss<true>(u, y, w, s4.cvs, s4.M)
                                        : cand_loss<false>(u, y, w, s4.cvs, s4.M));
        code = j4 < j6 ? c4 : c6;
        const float lo = fminf(j4, j6), hi = fmaxf(j4, j6);
        const bool near = c4 != c6 && !(hi > fmaf(lo, 2.0f * kBand, lo) + kBandAbs);
        if (__any(near)) {
            if (near) {
                const double e6 = use_w ? exact_loss<true, LPB>(y, w, s6, part, group_base)
                                        : exact_loss<false, LPB>(y, w, s6, part, group_base);
                const double e4 = use_w ? exact_loss<true, LPB>(y, w, s4, part, group_base)
                                        : exact_loss<false, LPB>(y, w, s4, part, group_base);
                code = e4 < e6 ? c4 : c6;
            }
        }
    } else if (METHOD == kWindowMse || METHOD == kWindowWmse) {
        constexpr bool WGT = METHOD == kWindowWmse;
        constexpr int STD_LOWER = Window<WGT ? kSweepWmse : kSweepMse, N>::L;
        code = choose_window<WGT, LPB>(y, w, ymax, tab, p, part, group_base, STD_LOWER,
                                        !WGT && N == 16);
    } else {
        using Win = Window<METHOD, N>;
        constexpr int NC = Win::NC;
        constexpr bool WGT = METHOD == kSweepWmse;
        const int c0 = floor_code(ymax, 6.0f, 1.0f / 6.0f, tab);
        const int cb = c0 - Win::L;                 // candidate d is code cb + d
        float J[NC];
        if constexpr (WGT) {
            __shared__ PrunedLds pl;
            if (__all(cb >= 8)) {
                pruned_wmse_losses<NC, LPB>(y, w, ymax, active, tab, cb, J, pl, colw, wblk, part);
            } else {
#pragma unroll
                for (int d = 0; d < NC; ++d) {
                    const Scale sd = tab[cb + d];
                    float u[kLaneElems];
#pragma unroll
                    for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * sd.rM;
                    J[d] = group_sum<LPB>(cand_loss<WGT>(u, y, w, sd.cvs, sd.M));
                }
            }
        } else if (!WGT && N == 16 && __all(cb >= 8)) {
            // MSE, offsets -3..7: the lowest candidate (d = 0, scored with offset 5 in one
            // significand group) comes last and is skipped by the wave when no block needs it.
            // Its scale is below max|y| / 6, so the largest element saturates there and
            // RN(RN(y1 - 6 s)^2) bounds its loss from below (the bound of pruned_wmse_losses
            // with w = 1): above the best other loss plus the band, the candidate can neither
            // be the minimum nor enter the band, and it scores +inf.
#pragma unroll
            for (int d = 1; d < 8; ++d) significand_group_losses_sched<LPB, NC>(y, tab, cb, d, J);
            float jb = J[1];
#pragma unroll
            for (int d = 2; d < NC; ++d)
                if (d != 8) jb = fminf(jb, J[d]);
            const float thr = active ? fmaf(jb, kBand, jb) + kBandAbs : -__builtin_inff();
            const float e = ymax - 6.0f * e4m3_value(cb);   // 6 s is exact
            if (__any(!(e * e > thr))) {
                significand_group_losses_sched<LPB, NC>(y, tab, cb, 0, J);
            } else {
                J[0] = __builtin_inff();
                significand_group_losses_sched<LPB, NC>(y, tab, cb, 8, J);   // offset 5 alone
            }
        } else if (!WGT && N > 16 && __all(cb >= 8)) {
            // MSE at n = 32, 64, 128 (offsets -L..7): offsets -1..7 first (grouped by
            // significand), then the lower candidates from the highest down, each scored only
            // when a block of the wave may need it: the saturation bound of the n = 16 case,
            // against the best loss scored so far.  Bound and losses are block-wide, so the
            // lanes of a block decide alike; a skipped candidate scores +inf.
            constexpr int DU = Win::L - 1;          // d of offset -1
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                if constexpr (NC <= 16) {
                    if (r >= DU) significand_group_losses_sched<LPB, NC>(y, tab, cb, r, J);
                    else if (r + 8 < NC) significand_group_losses_sched<LPB, NC>(y, tab, cb, r + 8, J);
                } else {
                    significand_group_losses<false, LPB, NC>(y, w, tab, cb, r, J, DU);
                }
            }
            float jb = J[DU];
#pragma unroll
            for (int d = DU + 1; d < NC; ++d) jb = fminf(jb, J[d]);   // NaN codes past 126 drop out
#pragma unroll
            for (int d = DU - 1; d >= 0; --d) {
                const float thr = fmaf(jb, kBand, jb) + kBandAbs;
                const float e = ymax - 6.0f * e4m3_value(cb + d);   // 6 s is exact
                if (__any(active && !(e * e > thr))) {
                    const Scale sd = tab[cb + d];
                    float u[kLaneElems];
#pragma unroll
                    for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * sd.rM;
                    J[d] = group_sum<LPB>(cand_loss<false>(u, y, w, sd.cvs, sd.M));
                    jb = fminf(jb, J[d]);
                } else {
                    J[d] = __builtin_inff();
                }
            }
        } else if (__all(cb >= 8)) {
            // normal codes only: c, c+8, c+16 share the significand M and differ in 2^E
#pragma unroll
            for (int d = 0; d < 8 && d < NC; ++d)
                if constexpr (!WGT && NC <= 16)
                    significand_group_losses_sched<LPB, NC>(y, tab, cb, d, J);
                else
                    significand_group_losses<WGT, LPB, NC>(y, w, tab, cb, d, J);
        } else {
#pragma unroll
            for (int d = 0; d < NC; ++d) {
                const Scale sd = tab[cb + d];
                float u[kLaneElems];
#pragma unroll
                for (int i = 0; i < kLaneElems; ++i) u[i] = fabsf(y[i]) * sd.rM;
                J[d] = group_sum<LPB>(cand_loss<WGT>(u, y, w, sd.cvs, sd.M));
            }
        }
        // (codes outside 1..126 scored NaN through their table entries)
        // argmin on the loss with its 7 low bits replaced by the candidate index: exact
        // ordering except between losses within 2^-16 of each other, which the band re-scores
        uint32_t best = 0xFFFFFFFFu;
#pragma unroll
        for (int d = 0; d < NC; d += 2) {
            const uint32_t k0 = (__float_as_uint(J[d]) & 0xFFFFFF80u) | (uint32_t)d;
            const uint32_t k1 = d + 1 < NC ? (__float_as_uint(J[d + 1]) & 0xFFFFFF80u) | (uint32_t)(d + 1)
                                           : 0xFFFFFFFFu;
            best = min(best, min(k0, k1));
        }
        int dstar = (int)(best & 0x7Fu);
        const float j1 = __uint_as_float(best & 0xFFFFFF80u);
        const float bound = fmaf(j1, kBand, j1) + kBandAbs;
        // candidates inside the band, counted per lane (a compare and an add with carry each)
        uint32_t inb = 0u;
#pragma unroll
        for (int d = 0; d < NC; ++d) inb += J[d] <= bound ? 1u : 0u;
        const bool near = inb >= 2u;
        if (__any(near)) {
            if (near) {
                // candidates in the band; two of them eight codes apart (one significand,
                // scales s and 2s) that reconstruct every element identically have equal
                // exact losses, so the smaller code wins without summing in binary64
                uint32_t inband = 0u;
#pragma unroll
                for (int d = 0; d < NC; ++d)
                    if (J[d] <= bound && cb + d >= 1 && cb + d <= 126) inband |= 1u << d;
                const int d0 = __builtin_ctz(inband | 0x80000000u), d1 = 31 - __builtin_clz(inband | 1u);
                const bool pair8 = __builtin_popcount(inband) == 2 && d1 == d0 + 8;
                if (pair8 && same_reconstruction<LPB>(y, tab[cb + d0], tab[cb + d1])) {
                    dstar = d0;
                } else {
                    double jb = 0.0;
                    int db = -1;
                    // the weights again, from memory: this rare path keeps no registers
                    // occupied across the sweep
                    float wx[kLaneElems];
                    if (WGT) {
                        load_weights(colw + (int64_t)wblk * N + part * kLaneElems, wx);
                    } else {
#pragma unroll
                        for (int i = 0; i < kLaneElems; ++i) wx[i] = 1.0f;
                    }
#pragma unroll 1
                    for (int d = 0; d < NC; ++d) {
                        if ((inband >> d) & 1u) {
                            const Scale sd = tab[cb + d];
                            const double jd = exact_loss<WGT, LPB>(y, wx, sd, part, group_base);
                            if (db < 0 || jd < jb) {
                                jb = jd;
                                db = d;
                            }
                        }
                    }
                    if (db >= 0) dstar = db;
                }
            }
        }
        code = clamp_code(cb + dstar);   // always a window code unless every loss is NaN
    }

    // ---- emit: exact FP4 codes at the chosen scale, packed two per byte ------------------
    const Scale sc = tab[code];
    uint32_t packed[2] = {0u, 0u};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        float u[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            u[i] = div_by_significand(y[8 * h + i], sc.M, sc.rM);
        }
        uint32_t r = 0u;
        r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, u[0], u[1], sc.cvs, 0);
        r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, u[2], u[3], sc.cvs, 1);
        r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, u[4], u[5], sc.cvs, 2);
        r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, u[6], u[7], sc.cvs, 3);
        packed[h] = r;
    }
    if (active) {
        uint2* dst = reinterpret_cast<uint2*>(q + ((blk * N + part * kLaneElems) >> 1));
        // streamed past the caches (nothing here reads them again): 2-5 % for the
        // bandwidth-bound AbsMax and 4/6 launches
        u32x2 pv;
        pv.x = packed[0];
        pv.y = packed[1];
        __builtin_nontemporal_store(pv, reinterpret_cast<u32x2*>(dst));
        if (part == 0) {
            if (p.swizzled)      // through L2, which merges the 4-byte pieces of a tile's lines
                scales[swizzled_offset(row, kb, p.sw_kt)] = (uint8_t)code;
            else
                __builtin_nontemporal_store((uint8_t)code, scales + blk);
        }
    }
    }
}

// Zero bytes of the swizzled scale layout that no block owns: rows rows..mp-1 (all kp columns),
// then columns k16..kp-1 of rows 0..rows-1.  Disjoint from the bytes the quantization kernel
// writes, so the two may run in either order.
__global__ __launch_bounds__(256) void swizzle_pad_kernel(uint8_t* __restrict__ scales, uint32_t rows,
                                                          uint32_t k16, uint32_t mp, uint32_t kp) {
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    const uint32_t n_rows = (mp - rows) * kp;
    const uint32_t wcols = kp - k16;
    uint32_t m, k;
    if (t < n_rows) {
        m = rows + t / kp;
        k = t % kp;
    } else if (t < n_rows + rows * wcols) {
        const uint32_t u = t - n_rows;
        m = u / wcols;
        k = k16 + u % wcols;
    } else {
        return;
    }
    scales[swizzled_offset(m, k, kp / 4)] = 0;
}

// ---------------------------------------------------------------------------------------
// Dequantization: x_hat = RN32((q s) S).
// ---------------------------------------------------------------------------------------

typedef float float4v __attribute__((ext_vector_type(4)));

// A wave writes 1024 consecutive outputs (4 KiB) as four stores of 16 bytes per lane, each
// store contiguous across the wave: store k of lane L holds elements base + 256 k + 4 L ...
// + 3, decoded from the byte pair of their nibbles and the scale of their block.  (Sixteen
// consecutive outputs per lane, 64 bytes apart between lanes, reached 3.6 TB/s on MI355X; the
// wave-contiguous stores 5.8 TB/s, and streaming them past the caches 6.8 TB/s.)
template <int N>
__global__ __launch_bounds__(kThreads) void dequant_kernel(const uint8_t* __restrict__ q,
                                                           const uint8_t* __restrict__ scales,
                                                           const float* __restrict__ tensor_scale,
                                                           int64_t n, float* __restrict__ out) {
    const int64_t base = ((int64_t)blockIdx.x * kThreads + (threadIdx.x & ~63)) * kLaneElems;
    const int lane = threadIdx.x & 63;
    const float S = tensor_scale[0];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int64_t e = base + 256 * k + 4 * lane;      // n is a multiple of 16: all or none
        if (e < n) {
            const uint32_t pair = *reinterpret_cast<const uint16_t*>(q + (e >> 1));
            const int code = scales[e / N];
            const float s = e4m3_value(code);
            const float cvs = code == 0 ? 1.0f : s;
            const float M = code == 0 ? 0.f : __uint_as_float((__float_as_uint(s) & 0x007FFFFFu) | 0x3F800000u);
            const float2v g0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pair, cvs, 0);
            const float2v g1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(pair, cvs, 1);
            float4v v;                          // g 2^E M = q s exactly, then one rounding
            v.x = (g0.x * M) * S;
            v.y = (g0.y * M) * S;
            v.z = (g1.x * M) * S;
            v.w = (g1.y * M) * S;
            __builtin_nontemporal_store(v, reinterpret_cast<float4v*>(out + e));
        }
    }
}

// The SwiGLU producer alone (the unfused path): h = bf16(silu(gate) * up), 16 elements per
// lane, two 16-byte stores per lane.
__global__ __launch_bounds__(kThreads) void swiglu_kernel(const uint16_t* __restrict__ gate,
                                                          const uint16_t* __restrict__ up, int64_t n,
                                                          uint16_t* __restrict__ h) {
    const int64_t e = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kLaneElems;
    if (e >= n) return;                               // n is a multiple of 16
    float v[kLaneElems];
    swiglu_lane(gate + e, up + e, v);
    uint32_t w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = (__float_as_uint(v[2 * j]) >> 16) | (__float_as_uint(v[2 * j + 1]) & 0xFFFF0000u);
    uint4* dst = reinterpret_cast<uint4*>(h + e);
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
}

// ---------------------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------------------

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool valid_block(int block) { return block == 16 || block == 32 || block == 64 || block == 128; }

// Unsigned division by an invariant d >= 1: magic m and shift l with
// n / d = (hi + ((n - hi) >> 1)) >> (l - 1), hi = umulhi(n, m), l = ceil(log2 d) (l = 0: d = 1).
void make_divider(uint32_t d, uint32_t* magic, uint32_t* shift) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    *shift = l;
    *magic = l == 0 ? 0u : (uint32_t)((((1ull << l) - d) << 32) / d + 1);
}

struct Call {
    int method;
    const void* x;
    int dtype;
    int64_t rows, cols;
    int block;
    const float* colw;
    float fp8_range, static_scale;
    float* tensor_scale;
    uint8_t* q;
    uint8_t* scales;
    void* ws;
    size_t ws_bytes;
    hipStream_t stream;
    int win_mode = 0, win_lo = 0, win_hi = 0;     // window variants only
    int layout = NVFP4_SCALES_ROW_MAJOR;          // online calls only
    int64_t wgroups = 1, wgroup_rows = 1;
    const void* up = nullptr;                     // fused SwiGLU calls: x is the gate
};

// Workgroups of the quantization kernel: one lane per 16 elements, one workgroup per tile.
int64_t quant_grid(const Call& c) {
    const int64_t lanes = c.rows * c.cols / kLaneElems;
    return (lanes + kThreads - 1) / kThreads;
}

template <int METHOD, typename In, int N, bool SWIGLU = false>
hipError_t launch_quant(const Call& c, const Params& p) {
    const int64_t grid = quant_grid(c);
    hipLaunchKernelGGL((quant_kernel<METHOD, In, N, SWIGLU>), dim3((unsigned)grid), dim3(kThreads), 0,
                       c.stream, static_cast<const In*>(c.x), c.colw, c.q, c.scales, p);
    return hipGetLastError();
}

template <int METHOD, typename In>
hipError_t launch_quant_n(const Call& c, const Params& p) {
    switch (c.block) {
        case 16: return launch_quant<METHOD, In, 16>(c, p);
        case 32: return launch_quant<METHOD, In, 32>(c, p);
        case 64: return launch_quant<METHOD, In, 64>(c, p);
        default: return launch_quant<METHOD, In, 128>(c, p);
    }
}

template <int METHOD>
hipError_t launch_quant_m(const Call& c, const Params& p) {
    return c.dtype == NVFP4_IN_F32 ? launch_quant_n<METHOD, float>(c, p)
                                   : launch_quant_n<METHOD, uint16_t>(c, p);
}

// Synchronous argument checks shared by every entry point; nothing is launched.
int validate(const Call& c) {
    if (!c.tensor_scale) return NVFP4_ERR_NULL;
    if (c.dtype != NVFP4_IN_F32 && c.dtype != NVFP4_IN_BF16) return NVFP4_ERR_DTYPE;
    if (!valid_block(c.block)) return NVFP4_ERR_BLOCK;
    if (c.rows < 0 || c.cols < 0 || c.cols % c.block != 0) return NVFP4_ERR_SHAPE;
    if (!(c.fp8_range > 0.0f && c.fp8_range <= 448.0f)) return NVFP4_ERR_ARG;
    if (!(c.static_scale >= 0.0f && c.static_scale <= FLT_MAX)) return NVFP4_ERR_ARG;
    if ((c.method == kSweepWmse || c.method == kWindowWmse) && !c.colw) return NVFP4_ERR_NULL;
    if (c.method == kWindowMse || c.method == kWindowWmse) {
        if (c.win_mode == NVFP4_WINDOW_OFFSETS) {
            if (c.win_lo < -126 || c.win_hi > 126 || c.win_lo > c.win_hi) return NVFP4_ERR_ARG;
        } else if (c.win_mode != NVFP4_WINDOW_TIGHT) {
            return NVFP4_ERR_ARG;
        }
    }
    const int64_t n = c.rows * c.cols;
    if (n > 0 && (!c.x || !c.q || !c.scales)) return NVFP4_ERR_NULL;
    if (c.static_scale == 0.0f) {
        if (!c.ws) return NVFP4_ERR_WORKSPACE;
        if (c.ws_bytes < kWorkspaceBytes) return NVFP4_ERR_WORKSPACE;
        if (!aligned(c.ws, 16)) return NVFP4_ERR_ALIGN;
    }
    if (n > 0 && (!aligned(c.x, 16) || !aligned(c.q, 8))) return NVFP4_ERR_ALIGN;
    if (c.colw && !aligned(c.colw, 16)) return NVFP4_ERR_ALIGN;
    if (n / c.block > 0x7FFFFFFFLL) return NVFP4_ERR_SHAPE;     // 32-bit block indexing
    return NVFP4_OK;
}

// Dynamic global scale of a non-empty tensor: the |x| reduction and the fold into S, 1/S
// (which also clears the |x| slots of zero_count workspaces from zero_base, for a batched call).
hipError_t launch_scale(const Call& c, hipStream_t stream, int* npart, void* zero_base = nullptr,
                        int zero_count = 0) {
    const int64_t n = c.rows * c.cols;
    const int64_t nvec = n * (c.dtype == NVFP4_IN_F32 ? 4 : 2) / 16;
    int64_t g = (nvec + kThreads * 8 - 1) / (kThreads * 8);
    if (g < 1) g = 1;
    if (g > kMaxPartials) g = kMaxPartials;
    *npart = (int)g;
    if (c.dtype == NVFP4_IN_F32)
        hipLaunchKernelGGL(amax_kernel<float>, dim3((unsigned)g), dim3(kThreads), 0, stream,
                           static_cast<const float*>(c.x), nvec, static_cast<uint32_t*>(c.ws));
    else
        hipLaunchKernelGGL(amax_kernel<uint16_t>, dim3((unsigned)g), dim3(kThreads), 0, stream,
                           static_cast<const uint16_t*>(c.x), nvec, static_cast<uint32_t*>(c.ws));
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(scale_kernel, dim3(1), dim3(64), 0, stream, static_cast<uint32_t*>(c.ws),
                       (int)g, 6.0f * c.fp8_range, c.tensor_scale, static_cast<uint32_t*>(zero_base),
                       zero_count, (int64_t)(kWorkspaceBytes / sizeof(uint32_t)));
    return hipGetLastError();
}

// What a quantization kernel of a batched call does beyond its own tensor: where its S comes
// from, and the next tensor whose |x| maximum it reduces (nullptr: none).
struct Chain {
    int scale_src = kScaleWorkspace;
    const void* nx = nullptr;
    int64_t nx_bytes = 0;
    uint32_t* nx_ws = nullptr;
};


// The quantization kernel of a non-empty tensor (after launch_scale for a dynamic scale, or
// after the kernel that raised its |x| slots in a batched call).
hipError_t launch_main(const Call& c, hipStream_t stream, const Chain& chain = Chain()) {
    const bool dynamic = c.static_scale == 0.0f;
    Params p;
    p.nblocks = c.rows * c.cols / c.block;
    p.bpr = (uint32_t)(c.cols / c.block);
    make_divider(p.bpr, &p.bpr_magic, &p.bpr_shift);
    p.scale_src = dynamic ? chain.scale_src : kScaleStatic;
    p.S = dynamic ? 0.0f : c.static_scale;
    p.rS = dynamic ? 0.0f : 1.0f / c.static_scale;
    p.denom = 6.0f * c.fp8_range;
    p.ws = static_cast<const uint32_t*>(c.ws);
    p.tensor_scale = c.tensor_scale;
    p.nx = static_cast<const uint4*>(chain.nx);
    p.nx_vec = chain.nx ? chain.nx_bytes / 16 : 0;
    const int64_t tiles = quant_grid(c);
    p.nx_per = p.nx_vec > 0 ? (p.nx_vec + tiles - 1) / tiles : 0;
    p.nx_slots = chain.nx_ws ? chain.nx_ws + kSlotWord0 : nullptr;
    p.swizzled = c.layout == NVFP4_SCALES_SWIZZLED ? 1 : 0;
    p.sw_kt = (uint32_t)((c.cols / c.block + 3) / 4);
    p.wgroups = (uint32_t)c.wgroups;
    make_divider((uint32_t)c.wgroup_rows, &p.wgr_magic, &p.wgr_shift);
    make_divider((uint32_t)c.wgroups, &p.wgn_magic, &p.wgn_shift);
    p.win_tight = c.win_mode == NVFP4_WINDOW_TIGHT ? 1 : 0;
    p.win_lo = c.win_lo;
    p.win_hi = c.win_hi;
    p.up = static_cast<const uint16_t*>(c.up);
    Call cs = c;
    cs.stream = stream;
    if (c.up) {                       // fused SwiGLU producer: bfloat16, block 16
        switch (c.method) {
            case kAbsMax: return launch_quant<kAbsMax, uint16_t, 16, true>(cs, p);
            case kFourSix: return launch_quant<kFourSix, uint16_t, 16, true>(cs, p);
            case kSweepMse: return launch_quant<kSweepMse, uint16_t, 16, true>(cs, p);
            default: return launch_quant<kSweepWmse, uint16_t, 16, true>(cs, p);
        }
    }
    switch (c.method) {
        case kAbsMax: return launch_quant_m<kAbsMax>(cs, p);
        case kFourSix: return launch_quant_m<kFourSix>(cs, p);
        case kSweepMse: return launch_quant_m<kSweepMse>(cs, p);
        case kWindowMse: return launch_quant_m<kWindowMse>(cs, p);
        case kWindowWmse: return launch_quant_m<kWindowWmse>(cs, p);
        default: return launch_quant_m<kSweepWmse>(cs, p);
    }
}

// S of an empty tensor is 1 (or the given S).
hipError_t launch_empty(const Call& c, hipStream_t stream) {
    hipLaunchKernelGGL(write_scale_kernel, dim3(1), dim3(1), 0, stream, c.tensor_scale,
                       c.static_scale == 0.0f ? 1.0f : c.static_scale);
    return hipGetLastError();
}

int run_quant(const Call& c) {
    const int rc = validate(c);
    if (rc != NVFP4_OK) return rc;
    if (c.rows * c.cols == 0) return launch_empty(c, c.stream) == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
    int npart = 0;
    if (c.static_scale == 0.0f && launch_scale(c, c.stream, &npart) != hipSuccess) return NVFP4_ERR_HIP;
    return launch_main(c, c.stream) == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

// Several tensors, dynamic scales, one stream.  The non-empty tensors form a chain in
// ascending size: the first is reduced by amax_kernel and folded by scale_kernel (which also
// clears every tensor's |x| slots); each quantization kernel then also reduces the next
// tensor of the chain into that tensor's slots, and the next kernel folds them into its S.
// So every reduction but the smallest tensor's rides along with an arithmetic-bound sweep,
// and no kernel sits between two sweeps.  Ascending order keeps the next tensor's share per
// workgroup small (at most 4x its own tile for a decoder layer).  The chain is walked in
// place: each step scans the list for the smallest (size, index) after the current one, so
// the call allocates nothing for any count (count^2 comparisons on the host).
int run_batched(int method, const nvfp4_tensor* t, int count, int dtype, int block,
                float fp8_range, void* ws, size_t ws_bytes, hipStream_t main) {
    if (count < 0) return NVFP4_ERR_ARG;
    if (count > 0 && !t) return NVFP4_ERR_NULL;
    if (method < kAbsMax || method > kSweepWmse) return NVFP4_ERR_ARG;
    if (count > 0 && (!ws || ws_bytes < (size_t)count * kWorkspaceBytes)) return NVFP4_ERR_WORKSPACE;
    if (count > 0 && !aligned(ws, 16)) return NVFP4_ERR_ALIGN;
    auto ws_of = [&](int k) { return static_cast<char*>(ws) + (size_t)k * kWorkspaceBytes; };
    auto call_of = [&](int k) {
        return Call{method, t[k].x, dtype, t[k].rows, t[k].cols, block, t[k].col_weight,
                    fp8_range, 0.0f, t[k].tensor_scale, t[k].q, t[k].scales,
                    ws_of(k), kWorkspaceBytes, main};
    };
    auto size_of = [&](int k) { return t[k].rows * t[k].cols; };
    for (int k = 0; k < count; ++k) {
        const int rc = validate(call_of(k));
        if (rc != NVFP4_OK) return rc;
    }
    // the non-empty tensor that follows k in ascending (size, index) order (k < 0: the first),
    // or -1 after the last
    auto next_of = [&](int k) {
        int best = -1;
        for (int j = 0; j < count; ++j) {
            const int64_t sj = size_of(j);
            if (sj == 0) continue;
            if (k >= 0 && (sj < size_of(k) || (sj == size_of(k) && j <= k))) continue;
            if (best < 0 || sj < size_of(best)) best = j;   // ties keep the lower index
        }
        return best;
    };
    const int64_t elem_bytes = dtype == NVFP4_IN_F32 ? 4 : 2;
    bool ok = true;
    for (int k = 0; ok && k < count; ++k)
        if (size_of(k) == 0) ok = launch_empty(call_of(k), main) == hipSuccess;
    int cur = next_of(-1);
    int npart = 0;
    if (ok && cur >= 0) ok = launch_scale(call_of(cur), main, &npart, ws, count) == hipSuccess;
    for (bool first = true; ok && cur >= 0; first = false) {
        const int kn = next_of(cur);
        Chain ch;
        ch.scale_src = first ? kScaleWorkspace : kScaleSlots;
        if (kn >= 0) {
            ch.nx = t[kn].x;
            ch.nx_bytes = size_of(kn) * elem_bytes;
            ch.nx_ws = reinterpret_cast<uint32_t*>(ws_of(kn));
        }
        ok = launch_main(call_of(cur), main, ch) == hipSuccess;
        cur = kn;
    }
    return ok ? NVFP4_OK : NVFP4_ERR_HIP;
}

// Bytes of the scale output for a layout, or a negative status.
int64_t scales_bytes(int64_t rows, int64_t cols, int block, int layout) {
    if (!valid_block(block)) return NVFP4_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return NVFP4_ERR_SHAPE;
    const int64_t k16 = cols / block;
    if (layout == NVFP4_SCALES_ROW_MAJOR) return rows * k16;
    if (layout != NVFP4_SCALES_SWIZZLED || block != 16) return NVFP4_ERR_ARG;
    return (rows + 127) / 128 * 128 * ((k16 + 3) / 4 * 4);
}

int run_online(const Call& c) {
    if (c.method < kAbsMax || c.method > kSweepWmse) return NVFP4_ERR_ARG;
    if (c.dtype != NVFP4_IN_F32 && c.dtype != NVFP4_IN_BF16) return NVFP4_ERR_DTYPE;
    const int64_t nbytes = scales_bytes(c.rows, c.cols, c.block, c.layout);
    if (nbytes < 0) return (int)nbytes;
    if (!(c.static_scale > 0.0f && c.static_scale <= FLT_MAX)) return NVFP4_ERR_ARG;
    if (c.method == kSweepWmse && !c.colw) return NVFP4_ERR_NULL;
    if (c.colw && (c.wgroups < 1 || c.wgroup_rows < 1 || c.wgroups > 0xFFFFFFFFLL ||
                   c.wgroup_rows > 0xFFFFFFFFLL))
        return NVFP4_ERR_ARG;
    const int64_t n = c.rows * c.cols;
    if (n > 0 && (!c.x || !c.q || !c.scales)) return NVFP4_ERR_NULL;
    if (n > 0 && (!aligned(c.x, 16) || !aligned(c.q, 8))) return NVFP4_ERR_ALIGN;
    if (c.colw && !aligned(c.colw, 16)) return NVFP4_ERR_ALIGN;
    if (n / c.block > 0x7FFFFFFFLL || nbytes > 0x7FFFFFFFLL) return NVFP4_ERR_SHAPE;
    if (n == 0) {
        if (!c.tensor_scale) return NVFP4_OK;
        return launch_empty(c, c.stream) == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
    }
    Call cc = c;
    if (!c.colw) cc.wgroups = cc.wgroup_rows = 1;
    if (launch_main(cc, c.stream) != hipSuccess) return NVFP4_ERR_HIP;
    if (c.layout == NVFP4_SCALES_SWIZZLED) {
        const uint32_t rows = (uint32_t)c.rows, k16 = (uint32_t)(c.cols / 16);
        const uint32_t mp = (rows + 127) / 128 * 128, kp = (k16 + 3) / 4 * 4;
        const uint64_t pad = (uint64_t)(mp - rows) * kp + (uint64_t)rows * (kp - k16);
        if (pad > 0) {
            hipLaunchKernelGGL(swizzle_pad_kernel, dim3((unsigned)((pad + 255) / 256)), dim3(256), 0,
                               c.stream, c.scales, rows, k16, mp, kp);
            if (hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
        }
    }
    return NVFP4_OK;
}

}  // namespace

// ---------------------------------------------------------------------------------------
// Fixed scratch of the no-allocation batched entry point.
// ---------------------------------------------------------------------------------------

namespace nvfp4ss_noalloc {

constexpr int kMaxTensors = NVFP4_NOALLOC_MAX_TENSORS;
constexpr int kMaxDevices = 64;

// One workspace per tensor of a call.  On the host this name is only a stand-in for the
// symbol: each device holds its own copy, whose address hipGetSymbolAddress returns.
__device__ __align__(256) uint8_t scratch[kMaxTensors * kWorkspaceBytes];

std::mutex lookup_mu;
void* device_ptr[kMaxDevices];     // per device: that device's copy of `scratch`

// The address of `scratch` on the device that runs `stream`, looked up once per device with
// that device current.
int scratch_for(hipStream_t stream, void** out) {
    int dev = -1;
    if (stream == nullptr) {
        if (hipGetDevice(&dev) != hipSuccess) return NVFP4_ERR_HIP;
    } else if (hipStreamGetDevice(stream, &dev) != hipSuccess) {
        return NVFP4_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) return NVFP4_ERR_ARG;
    std::lock_guard<std::mutex> lock(lookup_mu);
    if (!device_ptr[dev]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return NVFP4_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return NVFP4_ERR_HIP;
        void* ptr = nullptr;
        const hipError_t err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev) (void)hipSetDevice(cur);
        if (err != hipSuccess || !ptr) return NVFP4_ERR_HIP;
        device_ptr[dev] = ptr;
    }
    *out = device_ptr[dev];
    return NVFP4_OK;
}

}  // namespace nvfp4ss_noalloc

extern "C" {

int nvfp4_quant_batched_noalloc(int method, const nvfp4_tensor* tensors, int count, int dtype,
                                int block, float fp8_range, void* stream) {
    if (count < 0) return NVFP4_ERR_ARG;
    if (count > nvfp4ss_noalloc::kMaxTensors) return NVFP4_ERR_LIMIT;
    if (count == 0) return run_batched(method, tensors, 0, dtype, block, fp8_range, nullptr, 0,
                                       (hipStream_t)stream);
    if (!tensors) return NVFP4_ERR_NULL;
    void* ws = nullptr;
    const int rc = nvfp4ss_noalloc::scratch_for((hipStream_t)stream, &ws);
    if (rc != NVFP4_OK) return rc;
    return run_batched(method, tensors, count, dtype, block, fp8_range, ws,
                       (size_t)count * kWorkspaceBytes, (hipStream_t)stream);
}

int64_t nvfp4_scales_bytes(int64_t rows, int64_t cols, int block, int layout) {
    return scales_bytes(rows, cols, block, layout);
}

int nvfp4_quant_online(int method, const void* x, int dtype, int64_t rows, int64_t cols, int block,
                       const float* importance, int64_t imp_groups, int64_t imp_group_rows,
                       float static_scale, int scale_layout, float* tensor_scale, uint8_t* q,
                       uint8_t* scales, void* stream) {
    Call c{method, x, dtype, rows, cols, block,
           (method == kSweepWmse || method == kFourSix) ? importance : nullptr, 448.0f,
           static_scale, tensor_scale, q, scales, nullptr, 0, (hipStream_t)stream};
    c.layout = scale_layout;
    c.wgroups = imp_groups;
    c.wgroup_rows = imp_group_rows;
    return run_online(c);
}

int nvfp4_quant_online_swiglu(int method, const void* gate, const void* up, int64_t rows, int64_t cols,
                              const float* importance, int64_t imp_groups, int64_t imp_group_rows,
                              float static_scale, int scale_layout, float* tensor_scale, uint8_t* q,
                              uint8_t* scales, void* stream) {
    if (!up && rows * cols > 0) return NVFP4_ERR_NULL;
    if (rows * cols > 0 && !aligned(up, 16)) return NVFP4_ERR_ALIGN;
    Call c{method, gate, NVFP4_IN_BF16, rows, cols, 16,
           (method == kSweepWmse || method == kFourSix) ? importance : nullptr, 448.0f,
           static_scale, tensor_scale, q, scales, nullptr, 0, (hipStream_t)stream};
    c.layout = scale_layout;
    c.wgroups = imp_groups;
    c.wgroup_rows = imp_group_rows;
    c.up = up;
    return run_online(c);
}

int nvfp4_swiglu(const void* gate, const void* up, int64_t rows, int64_t cols, void* h, void* stream) {
    if (rows < 0 || cols < 0 || cols % 16 != 0) return NVFP4_ERR_SHAPE;
    const int64_t n = rows * cols;
    if (n == 0) return NVFP4_OK;
    if (!gate || !up || !h) return NVFP4_ERR_NULL;
    if (!aligned(gate, 16) || !aligned(up, 16) || !aligned(h, 16)) return NVFP4_ERR_ALIGN;
    const int64_t grid = (n / kLaneElems + kThreads - 1) / kThreads;
    if (grid > 0x7FFFFFFFLL) return NVFP4_ERR_SHAPE;
    hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)grid), dim3(kThreads), 0, (hipStream_t)stream,
                       static_cast<const uint16_t*>(gate), static_cast<const uint16_t*>(up), n,
                       static_cast<uint16_t*>(h));
    return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

size_t nvfp4_workspace_bytes(void) { return kWorkspaceBytes; }

size_t nvfp4_batched_workspace_bytes(int count) {
    return count > 0 ? (size_t)count * kWorkspaceBytes : 0;
}

int nvfp4_quant_batched(int method, const nvfp4_tensor* tensors, int count, int dtype, int block,
                        float fp8_range, void* workspace, size_t workspace_bytes, void* stream) {
    return run_batched(method, tensors, count, dtype, block, fp8_range, workspace,
                       workspace_bytes, (hipStream_t)stream);
}

const char* nvfp4_status_string(int status) {
    switch (status) {
        case NVFP4_OK: return "ok";
        case NVFP4_ERR_NULL: return "a required pointer is NULL";
        case NVFP4_ERR_SHAPE: return "bad shape (rows/cols negative, cols not a multiple of block, or too many blocks)";
        case NVFP4_ERR_BLOCK: return "block must be 16, 32, 64 or 128";
        case NVFP4_ERR_DTYPE: return "unsupported dtype";
        case NVFP4_ERR_ARG: return "fp8_range, static_scale or window out of range";
        case NVFP4_ERR_WORKSPACE: return "dynamic global scale needs a workspace of nvfp4_workspace_bytes() bytes";
        case NVFP4_ERR_ALIGN: return "misaligned pointer (x, col_weight, workspace: 16 bytes; q: 8 bytes)";
        case NVFP4_ERR_HIP: return "HIP kernel launch failed";
        case NVFP4_ERR_LIMIT: return "more tensors than the no-allocation call's fixed scratch holds (NVFP4_NOALLOC_MAX_TENSORS)";
        default: return "unknown status";
    }
}

int nvfp4_quant_absmax(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                       float fp8_range, float static_scale, float* tensor_scale, uint8_t* q,
                       uint8_t* scales, void* workspace, size_t workspace_bytes, void* stream) {
    return run_quant({kAbsMax, x, dtype, rows, cols, block, nullptr, fp8_range, static_scale,
                      tensor_scale, q, scales, workspace, workspace_bytes, (hipStream_t)stream});
}

int nvfp4_quant_four_over_six(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                              const float* col_weight, float fp8_range, float static_scale,
                              float* tensor_scale, uint8_t* q, uint8_t* scales,
                              void* workspace, size_t workspace_bytes, void* stream) {
    return run_quant({kFourSix, x, dtype, rows, cols, block, col_weight, fp8_range, static_scale,
                      tensor_scale, q, scales, workspace, workspace_bytes, (hipStream_t)stream});
}

int nvfp4_quant_scalesweep_mse(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                               float fp8_range, float static_scale, float* tensor_scale,
                               uint8_t* q, uint8_t* scales, void* workspace,
                               size_t workspace_bytes, void* stream) {
    return run_quant({kSweepMse, x, dtype, rows, cols, block, nullptr, fp8_range, static_scale,
                      tensor_scale, q, scales, workspace, workspace_bytes, (hipStream_t)stream});
}

int nvfp4_quant_scalesweep_wmse(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                                const float* col_weight, float fp8_range, float static_scale,
                                float* tensor_scale, uint8_t* q, uint8_t* scales,
                                void* workspace, size_t workspace_bytes, void* stream) {
    return run_quant({kSweepWmse, x, dtype, rows, cols, block, col_weight, fp8_range,
                      static_scale, tensor_scale, q, scales, workspace, workspace_bytes,
                      (hipStream_t)stream});
}

int nvfp4_quant_scalesweep_window(const void* x, int dtype, int64_t rows, int64_t cols,
                                  int block, const float* col_weight, int window_mode,
                                  int window_lo, int window_hi, float fp8_range,
                                  float static_scale, float* tensor_scale, uint8_t* q,
                                  uint8_t* scales, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    Call c{col_weight ? kWindowWmse : kWindowMse, x, dtype, rows, cols, block, col_weight,
           fp8_range, static_scale, tensor_scale, q, scales, workspace, workspace_bytes,
           (hipStream_t)stream};
    c.win_mode = window_mode;
    c.win_lo = window_lo;
    c.win_hi = window_hi;
    return run_quant(c);
}

int nvfp4_dequant(const uint8_t* q, const uint8_t* scales, const float* tensor_scale,
                  int64_t rows, int64_t cols, int block, int out_dtype, void* out, void* stream) {
    if (!tensor_scale) return NVFP4_ERR_NULL;
    if (out_dtype != NVFP4_IN_F32) return NVFP4_ERR_DTYPE;
    if (!valid_block(block)) return NVFP4_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return NVFP4_ERR_SHAPE;
    const int64_t n = rows * cols;
    if (n == 0) return NVFP4_OK;
    if (!q || !scales || !out) return NVFP4_ERR_NULL;
    if (!aligned(q, 8) || !aligned(out, 16)) return NVFP4_ERR_ALIGN;
    const int64_t grid = (n / kLaneElems + kThreads - 1) / kThreads;   // 4096 outputs each
    hipStream_t s = (hipStream_t)stream;
    switch (block) {
        case 16: hipLaunchKernelGGL(dequant_kernel<16>, dim3((unsigned)grid), dim3(kThreads), 0, s, q, scales, tensor_scale, n, (float*)out); break;
        case 32: hipLaunchKernelGGL(dequant_kernel<32>, dim3((unsigned)grid), dim3(kThreads), 0, s, q, scales, tensor_scale, n, (float*)out); break;
        case 64: hipLaunchKernelGGL(dequant_kernel<64>, dim3((unsigned)grid), dim3(kThreads), 0, s, q, scales, tensor_scale, n, (float*)out); break;
        default: hipLaunchKernelGGL(dequant_kernel<128>, dim3((unsigned)grid), dim3(kThreads), 0, s, q, scales, tensor_scale, n, (float*)out); break;
    }
    return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

}  // extern "C"
