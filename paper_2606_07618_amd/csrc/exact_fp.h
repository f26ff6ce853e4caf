// Exact FP4 / FP8 helpers in binary64 shared by the analysis and GPTQ kernels: E2M1 values and
// the midpoints between them, E4M3 code values, and the nearest-E2M1 index of a / s by exact
// comparisons (NVFP4 section; Appendix A for the formats).
#pragma once

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

namespace nvfp4_exact {

// Midpoints between consecutive E2M1 magnitudes {0, 0.5, 1, 1.5, 2, 3, 4, 6}: 4 m_k is
// 1, 3, 5, 7, 10, 14, 20 for k = 0..6, one byte each of a 64-bit constant (exact; a shift
// and a conversion even when k is not a compile-time constant).
__device__ __forceinline__ double e2m1_mid(int k) {
    const uint64_t quads = 0x00140E0A07050301ull;
    return (double)(int)((quads >> (8 * k)) & 0xFFu) * 0.25;
}

// E2M1 magnitude of index k (0..7): twice the values, 0 1 2 3 4 6 8 12, are the nibbles of one
// 32-bit constant (no branch).
__device__ __forceinline__ double e2m1_value(int k) {
    return (double)((0xC8643210u >> (4 * k)) & 15u) * 0.5;
}

// E4M3 code c = a * 8 + b (0..126): 2^(a - 7) (1 + b/8) for a > 0, 2^-6 (b/8) for a = 0, i.e.
// (8 + b) 2^(a - 10) and b 2^-9 (no branch).
__device__ __forceinline__ double e4m3_f64(int c) {
    const int a = c >> 3, b = c & 7;
    return ldexp((double)(a ? 8 + b : b), (a ? a : 1) - 10);
}

// Index of the E2M1 value nearest to a / s (a >= 0, s > 0): the number of midpoints m_j with
// a > m_j s, where a midpoint that a meets exactly counts only if it leads to an even code.
// The products m_j s are rounded once in binary64 (exact when s is an E4M3 value).  They
// increase with j, so the count is found by a binary search over the seven midpoints (three
// products instead of seven).
__device__ __forceinline__ bool fp4_passes(double a, double s, int j) {
    const double m = e2m1_mid(j) * s;
    return a > m || (a == m && ((j + 1) & 1) == 0);
}

__device__ __forceinline__ int round_fp4_index(double a, double s) {
    if (s == 0.0) return 0;
    int k = fp4_passes(a, s, 3) ? 4 : 0;            // midpoints 0..3 all passed, or not 3
    k += fp4_passes(a, s, k + 1) ? 2 : 0;           // then j = k+1 decides two more
    k += fp4_passes(a, s, k) ? 1 : 0;               // and j = k one more
    return k;
}

// Largest code c in 0..126 with E4M3(c) <= v (v >= 0; +inf gives 126).
__device__ __forceinline__ int floor_e4m3(double v) {
    int lo = 0, hi = 126;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (e4m3_f64(mid) <= v) lo = mid; else hi = mid - 1;
    }
    return lo;
}

}  // namespace nvfp4_exact
