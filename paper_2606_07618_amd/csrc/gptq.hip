// GPTQ with fixed NVFP4 block scales on AMD Instinct MI355X (gfx950), in its LDLQ form
// (implementation details, GPTQ paragraph): the block scales are chosen before the pass (by
// any of the quantizers), the input channels are visited in descending order of the Hessian
// diagonal, the Hessian is damped by 0.01 x its mean diagonal, and
//   x_a = w_a + sum_{b < a} (w_b - w^_b) U_ba,     w^_a = Q(x_a)
// with Hp = (U + I) D (U + I)^T the factorization of the damped, reordered Hessian (U strictly
// upper triangular).  LDLQ and GPTQ give the same result.  Everything is binary64 with a
// fixed order of correctly rounded operations per value:
//   * factor: Hp is factored in place (column-major) in 64-column blocks from the last: the
//     block's own columns right-looking from its last column (rows in registers, each
//     column's updates to the block's remaining triangle in parallel); then the rows above
//     it, each a 64-column triangular solve, also right-looking; then the block's
//     contribution (U_ik U_jk) D_k, k walked downwards, is subtracted from the rest of the
//     upper triangle in tiles, first the column of tiles the next block needs, then the rest
//     beside the next block's own factor (look-ahead).  So each element receives its terms
//     k = n-1, ..., j+1 in that order.
//   * quantize: columns are taken in tiles of 64.  A tile kernel gives each row a quad of
//     lanes holding the tile's running values in registers: column b's value is quantized and
//     its error times U added to the tile's later columns, b = a0, a0 + 1, ... in order.  A
//     trailing-update kernel then adds the tile's 64 errors times U to every later column,
//     term by term in tile order: first to the next tile's columns, then to the rest beside
//     the next tile's kernel (look-ahead).  Every x_a therefore receives its terms
//     b = 0, 1, ... in ascending order, as the sequential definition adds them.
//   The sequential kernels (diagonal block, panel, tile) hold no branch per step: the columns
//   are interleaved over a quad's lanes (column 4m + q in lane q), so a step's updates need at
//   most one select, and its operands that do not depend on the running values are formed
//   ahead of the dependent chain.
// Q(x) is the quantizers' rounding: y = RN32(RN32(x) / S), nibble sign(y) << 3 | RNE_FP4(|y| /
// s), w^ = +-E2M1 * s * S (exact in binary64).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <utility>

#include "exact_fp.h"
#include "nvfp4ss.h"

namespace {

using namespace nvfp4_exact;

constexpr int kTile = 64;

template <typename In>
__device__ __forceinline__ float load_w(const In* w, int64_t i);

template <>
__device__ __forceinline__ float load_w<float>(const float* w, int64_t i) { return w[i]; }

template <>
__device__ __forceinline__ float load_w<uint16_t>(const uint16_t* w, int64_t i) {
    return __uint_as_float((uint32_t)w[i] << 16);
}

// f(integral_constant<int, B>) for B = 0, 1, ... in order (the calls unrolled at compile time).
template <typename F, int... B>
__device__ __forceinline__ void for_each_index(F&& f, std::integer_sequence<int, B...>) {
    (f(std::integral_constant<int, B>()), ...);
}

// Lane l of a quad broadcasts v to the quad's four lanes (a DPP quad permutation).
template <int L>
__device__ __forceinline__ uint32_t quad_bcast_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, L * 0x55, 0xF, 0xF, false);
}

// Lane l of each 16-lane row broadcasts v to the row's lanes (DPP row_newbcast).
template <int L>
__device__ __forceinline__ double row_bcast(double v) {
    constexpr int ctrl = 0x150 + L;
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, ctrl, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), ctrl, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

template <int L>
__device__ __forceinline__ double quad_bcast(double v) {
    constexpr int ctrl = L * 0x55;                    // quad_perm(L, L, L, L)
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, ctrl, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), ctrl, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// ---- column order and damping ------------------------------------------------------------

__global__ __launch_bounds__(256) void diag_kernel(const double* __restrict__ H, int64_t n,
                                                   double* __restrict__ diag) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) diag[i] = H[i * n + i];
}

// perm[rank(i)] = i, rank = number of columns with a larger diagonal, or an equal one and a
// smaller index (a stable descending order).  64 columns i per workgroup; each of its 16 waves
// counts over a sixteenth of every 1024-value chunk of the diagonal staged in LDS (one value per
// step, read by the wave's lanes alike), and the sixteen counts are added.
constexpr int kOrderParts = 16;
__global__ __launch_bounds__(64 * kOrderParts) void order_kernel(const double* __restrict__ diag, int64_t n,
                                                                 int* __restrict__ perm) {
    constexpr int kChunk = 1024, kPer = kChunk / kOrderParts;
    __shared__ double chunk[kChunk];
    __shared__ int part_rank[kOrderParts][64];
    const int il = threadIdx.x & 63, part = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * 64 + il;
    const double d = i < n ? diag[i] : 0.0;
    int rank = 0;
    for (int64_t c0 = 0; c0 < n; c0 += kChunk) {
        __syncthreads();                                          // the previous chunk is used
        chunk[threadIdx.x] = c0 + threadIdx.x < n ? diag[c0 + threadIdx.x] : 0.0;
        __syncthreads();
        const int64_t jb = c0 + part * kPer;
        const int m = (int)(n - jb < kPer ? (n - jb > 0 ? n - jb : 0) : kPer);
#pragma unroll 8
        for (int jj = 0; jj < m; ++jj) {
            const double e = chunk[part * kPer + jj];
            rank += (e > d || (e == d && jb + jj < i)) ? 1 : 0;
        }
    }
    part_rank[part][il] = rank;
    __syncthreads();
    if (part == 0 && i < n) {
        int r = 0;
        for (int k = 0; k < kOrderParts; ++k) r += part_rank[k][il];
        perm[r] = (int)i;
    }
}

// lambda = damp * (sum of the diagonal in index order) / n: one wave stages the diagonal in
// chunks, one lane adds.
__global__ __launch_bounds__(64) void damping_kernel(const double* __restrict__ diag, int64_t n, double damp,
                                                     double* __restrict__ lambda) {
    __shared__ double buf[1024];
    double tr = 0.0;
    for (int64_t c0 = 0; c0 < n; c0 += 1024) {
        __syncthreads();
        for (int t = threadIdx.x; t < 1024; t += 64) buf[t] = c0 + t < n ? diag[c0 + t] : 0.0;
        __syncthreads();
        if (threadIdx.x == 0) {
            const int m = (int)(n - c0 < 1024 ? n - c0 : 1024);
#pragma unroll 16
            for (int k = 0; k < m; ++k) tr += buf[k];
        }
    }
    if (threadIdx.x == 0) lambda[0] = damp * (tr / (double)n);
}

// ---- factor: blocked, from the last 64-column block backwards ---------------------------
// Uc holds A = Hp column-major (Uc[j n + i] = A_ij for i <= j; the lower triangle is never
// written, and the values the kernels read from it feed only results they discard) and is
// overwritten in place by U.  Element (i, j) must receive its terms k = n-1, n-2, ..., j+1 in that order; the blocks
// are finished last-first and every kernel walks k downwards, so it does.

__global__ __launch_bounds__(256) void init_a_kernel(const double* __restrict__ H,
                                                     const int* __restrict__ perm,
                                                     const double* __restrict__ lambda, int64_t n,
                                                     double* __restrict__ Uc) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= n * n) return;
    const int64_t j = t / n, i = t % n;
    if (i > j) return;                       // only the upper triangle is ever read as A
    double v = H[(int64_t)perm[i] * n + perm[j]];
    if (i == j) v = v + lambda[0];
    Uc[t] = v;
}

// The diagonal block [k0, k0 + 64): its D and its U, column by column from the last.  The
// block's own 64 columns, right-looking: at step kk (from the last) D_kk is the updated
// diagonal, U_i,kk = A_i,kk / D_kk for i < kk, and every A_ij (i <= j < kk) then loses
// (U_ik U_jk) D_k, so each element receives its terms k = 63, 62, ... in the order the
// column-by-column definition sums them.  A quad of threads per row, thread q holding the
// row's values of columns 4m + q in registers; column kk of U goes through LDS.  One barrier
// per step: after its updates every thread forms D_(kk-1) itself from the value its owner
// published before the step (the owner's own update, the same operations), so the threads
// holding column kk - 1 can divide at once and publish that column for the next step.
struct alignas(16) DiagLds {
    double col[2][kTile];          // col[kk & 1][16 (i & 3) + (i >> 2)] = U_{k0+i, k0+kk}
    double pre[2];                 // pre[kk & 1]: A_(kk-1),(kk-1) before step kk
    double Db[kTile];
};

__device__ __forceinline__ int quad_slot(int j) { return 16 * (j & 3) + (j >> 2); }

__device__ __forceinline__ void factor_diag_body(double* __restrict__ Uc, double* __restrict__ D,
                                                 int64_t n, int64_t k0, int* __restrict__ status,
                                                 DiagLds& L) {
    const int tid = threadIdx.x;
    const int i = tid >> 2, q = tid & 3;
    double v[16];                            // A (then U) of (k0 + i, k0 + 4m + q)
#pragma unroll
    for (int m = 0; m < 16; ++m) v[m] = Uc[(k0 + 4 * m + q) * n + k0 + i];
    // the column buffers start at zero: a step reads slots of rows it does not update (their
    // results are discarded by the selects)
    if (tid < 2 * kTile) L.col[tid / kTile][tid % kTile] = 0.0;
    // column 63: its diagonal, then its U, and A_62,62 for step 63
    if (i == kTile - 1 && q == 3) L.Db[kTile - 1] = v[15];
    __syncthreads();
    {
        const double d = L.Db[kTile - 1];
        const double u = v[15] / d;
        if (q == 3 && i < kTile - 1) {
            v[15] = u;
            L.col[1][quad_slot(i)] = u;
        }
        if (i == kTile - 2 && q == 2) L.pre[1] = v[15];
    }
    __syncthreads();
    auto step = [&](auto kc) {
        constexpr int kk = kTile - 1 - decltype(kc)::value, par = kk & 1;
        const double d = L.Db[kk];
        const double* c = &L.col[par][0];
        const double ui = c[quad_slot(i)];
        const double* cq = c + 16 * q;
        // the updates of this step: A_ij, i <= j = 4m + q < kk, in two halves of eight columns
        // (U values read together first).  Values left of the diagonal (j < i) are updated too:
        // they feed nothing (no diagonal, division, published value or store reads them), so
        // only the column bound j < kk needs a select, in one register per step.
#pragma unroll
        for (int h = 0; h < 16; h += 8) {
            double uj[8];
#pragma unroll
            for (int m = 0; m < 8; ++m) uj[m] = 4 * (h + m) < kk ? cq[h + m] : 0.0;
#pragma unroll
            for (int m = 0; m < 8; ++m) {
                const int mm = h + m;
                if (4 * mm < kk) {
                    double nv = v[mm] - (ui * uj[m]) * d;
                    asm volatile("" : "+v"(nv));     // formed in every lane, then selected (no
                                                     // branch around the update and its reads)
                    v[mm] = (4 * mm + 3 < kk || q < kk - 4 * mm) ? nv : v[mm];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (kk >= 1) {
            constexpr int k1 = kk - 1, q1 = k1 & 3, m1 = k1 >> 2;
            // D_(kk-1): its owner's update of this step, formed by every thread alike
            const double u1 = c[quad_slot(k1)];
            const double d1 = L.pre[par] - (u1 * u1) * d;
            const double u = v[m1] / d1;
            if (q == q1 && i < k1) {
                v[m1] = u;
                L.col[par ^ 1][quad_slot(i)] = u;
            }
            if (tid == 0) L.Db[k1] = d1;
            if constexpr (kk >= 2) {
                constexpr int k2 = kk - 2, q2 = k2 & 3, m2 = k2 >> 2;
                if (i == k2 && q == q2) L.pre[par ^ 1] = v[m2];
            }
            __syncthreads();
        }
    };
    for_each_index(step, std::make_integer_sequence<int, kTile>());
#pragma unroll
    for (int m = 0; m < 16; ++m) {
        const int j = 4 * m + q;
        if (i < j) Uc[(k0 + j) * n + k0 + i] = v[m];
    }
    if (tid < kTile) {
        const double d = L.Db[tid];
        D[k0 + tid] = d;
        if (!(d > 0.0) || !isfinite(d)) status[0] = 1;           // not positive definite
    }
}

__global__ __launch_bounds__(4 * kTile) void factor_diag_kernel(double* __restrict__ Uc, double* __restrict__ D,
                                                                int64_t n, int64_t k0, int* __restrict__ status) {
    __shared__ DiagLds L;
    factor_diag_body(Uc, D, n, k0, status, L);
}

// Rows above the block (i < k0), 16 per workgroup, a 16-lane row of lanes per matrix row: lane
// q holds the row's values of block columns 16m + q (m = 0..3) in registers.  Each row is a
// triangular solve from the block's last column, right-looking: at step kk the row's value of
// column kk is final, U_i,kk = A_i,kk / D_kk (broadcast in the lane row), and each of the
// row's columns j < kk loses (U_i,kk U_j,kk) D_kk.  So each value receives its terms kk = 63,
// 62, ... in the order the column-by-column definition sums them.  A step holds no branch and
// at most four updates per lane; the block's U and D are staged in LDS (each lane's columns of
// a U row contiguous).
constexpr int kPanelRows = 16;
__device__ __forceinline__ int row16_slot(int j) { return 4 * (j & 15) + (j >> 4); }

__global__ __launch_bounds__(256) void factor_panel_kernel(double* __restrict__ Uc,
                                                           const double* __restrict__ D, int64_t n,
                                                           int64_t k0) {
    __shared__ double Ub[kTile][kTile];       // Ub[kk][4 q + m] = U_{k0+16m+q, k0+kk}
    __shared__ double Db[kTile];
    const int tid = threadIdx.x;
    const int64_t i0 = (int64_t)blockIdx.x * kPanelRows;
    for (int t = tid; t < kTile * kTile; t += 256) {
        const int kk = t / kTile, jj = t % kTile;                 // coalesced over jj
        Ub[kk][row16_slot(jj)] = Uc[(k0 + kk) * n + k0 + jj];
    }
    if (tid < kTile) Db[tid] = D[k0 + tid];
    const int rr = tid >> 4, q = tid & 15;
    const int64_t i = i0 + rr;
    double v[4];
    if (i < k0) {
#pragma unroll
        for (int m = 0; m < 4; ++m) v[m] = Uc[(k0 + 16 * m + q) * n + i];
    }
    __syncthreads();
    if (i >= k0) return;                     // whole lane rows; rows share nothing
    const double* Up = &Ub[0][4 * q];
    auto step = [&](auto kc) {
        constexpr int kk = kTile - 1 - decltype(kc)::value, qk = kk & 15, mk = kk >> 4;
        const double dk = Db[kk];
        const double u = row_bcast<qk>(v[mk]) / dk;
        Uc[(k0 + kk) * n + i] = u;           // the row's lanes store the same value
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            if (16 * m < kk) {               // some lane of the row holds a column before kk
                const double nv = v[m] - (u * Up[kk * kTile + m]) * dk;
                v[m] = (16 * m + 15 < kk || q < kk - 16 * m) ? nv : v[m];
            }
        }
    };
    for_each_index(step, std::make_integer_sequence<int, kTile>());
}

// A_ij -= sum over the block's k, downwards, of (U_ik U_jk) D_k for i <= j < k0: one
// 16R x 16R tile of the upper triangle (rows i0.., columns j0..) per workgroup (tiles wholly
// below it exit), R x R values per lane; the block's 64 k in two halves of 32 (the upper
// first), so that four workgroups of the 64 x 64 tiles fit a CU's LDS: four waves per SIMD to
// issue the binary64 chains.  The 32 x 32 tiles (R = 2) serve the column of tiles the next
// block needs, which is on the critical path: four times the workgroups, a quarter of the
// chain per lane.
constexpr int kHalf = kTile / 2;
template <int R>
struct alignas(16) FTrailLdsT {
    double Ui[kHalf][16 * R + 2];  // Ui[kk][ii] = U_{i0+ii, k0+h+kk} (rows padded: 16-byte rows)
    double Uj[kHalf][16 * R + 2];
    double Dk[kTile];
};
using FTrailLds = FTrailLdsT<4>;

// Lane (tr, tc) owns rows i0 + R tr .. + R - 1 and columns j0 + R tc .. + R - 1, so that its
// values of a column and its operands of a step sit in 16-byte pairs.
template <int R>
__device__ __forceinline__ void factor_trailing_body(double* __restrict__ Uc, const double* __restrict__ D,
                                                     int64_t n, int64_t k0, int64_t i0, int64_t j0,
                                                     FTrailLdsT<R>& L) {
    static_assert(R % 2 == 0, "pairs of values");
    constexpr int B = 16 * R;
    if (i0 > j0 + B - 1) return;
    if (threadIdx.x < kTile) L.Dk[threadIdx.x] = D[k0 + threadIdx.x];
    const int tr = threadIdx.x / 16, tc = threadIdx.x % 16;
    const int64_t ir = i0 + R * tr, jc = j0 + R * tc;
    double acc[R][R];                        // acc[a][b]: (ir + a, jc + b)
#pragma unroll
    for (int b = 0; b < R; ++b) {
        const double2* src = reinterpret_cast<const double2*>(Uc + (jc + b) * n + ir);
#pragma unroll
        for (int a = 0; a < R; a += 2) {
            const double2 v = src[a / 2];
            acc[a][b] = v.x;
            acc[a + 1][b] = v.y;
        }
    }
    // each half's operands are loaded into registers while the previous half is computed
    constexpr int kPer = B * kHalf / 256;
    double pi[kPer], pj[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int t = threadIdx.x + 256 * e, kk = t / B, r = t % B;      // coalesced over r
        pi[e] = Uc[(k0 + kHalf + kk) * n + i0 + r];
        pj[e] = Uc[(k0 + kHalf + kk) * n + j0 + r];
    }
    for (int h = kHalf; h >= 0; h -= kHalf) {
        __syncthreads();                                          // the previous half is used
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int t = threadIdx.x + 256 * e, kk = t / B, r = t % B;
            L.Ui[kk][r] = pi[e];
            L.Uj[kk][r] = pj[e];
        }
        __syncthreads();
        if (h > 0) {
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                const int t = threadIdx.x + 256 * e, kk = t / B, r = t % B;
                pi[e] = Uc[(k0 + kk) * n + i0 + r];
                pj[e] = Uc[(k0 + kk) * n + j0 + r];
            }
        }
#pragma unroll(R == 2 ? 4 : 2)
        for (int kk = kHalf - 1; kk >= 0; --kk) {
            double ua[R], ub[R];
            const double2* ap = reinterpret_cast<const double2*>(&L.Ui[kk][R * tr]);
            const double2* bp = reinterpret_cast<const double2*>(&L.Uj[kk][R * tc]);
#pragma unroll
            for (int a = 0; a < R; a += 2) {
                const double2 av = ap[a / 2], bv = bp[a / 2];
                ua[a] = av.x;
                ua[a + 1] = av.y;
                ub[a] = bv.x;
                ub[a + 1] = bv.y;
            }
            const double dk = L.Dk[h + kk];
#pragma unroll
            for (int a = 0; a < R; ++a)
#pragma unroll
                for (int b = 0; b < R; ++b) acc[a][b] = acc[a][b] - (ua[a] * ub[b]) * dk;
        }
    }
#pragma unroll
    for (int b = 0; b < R; ++b)
#pragma unroll
        for (int a = 0; a < R; ++a) {
            const int64_t i = ir + a, j = jc + b;
            if (i <= j) Uc[j * n + i] = acc[a][b];
        }
}

// Tiles (blockIdx.y, blockIdx.x) of 16R x 16R in the columns from j0.
template <int R>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void factor_trailing_kernel(
        double* __restrict__ Uc, const double* __restrict__ D, int64_t n, int64_t k0, int64_t j0) {
    __shared__ FTrailLdsT<R> L;
    factor_trailing_body<R>(Uc, D, n, k0, (int64_t)blockIdx.y * 16 * R, j0 + (int64_t)blockIdx.x * 16 * R, L);
}

// Look-ahead: the next diagonal block [kd, kd + 64) (workgroup 0, once the column of tiles it
// needs has been updated) beside the rest of the current block's trailing update, tiles with
// bj < nb (the other workgroups, nb x nb of them).  The two touch disjoint elements.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void factor_lookahead_kernel(
        double* __restrict__ Uc, double* __restrict__ D, int64_t n, int64_t k0, int64_t nb, int64_t kd,
        int* __restrict__ status) {
    __shared__ union {
        DiagLds d;
        FTrailLds t;
    } L;
    if (blockIdx.x == 0) {
        factor_diag_body(Uc, D, n, kd, status, L.d);
    } else {
        const int64_t idx = blockIdx.x - 1;
        factor_trailing_body<4>(Uc, D, n, k0, idx / nb * kTile, idx % nb * kTile, L.t);
    }
}

// ---- quantize -----------------------------------------------------------------------------

template <typename In>
__global__ __launch_bounds__(256) void init_x_kernel(const In* __restrict__ w, const int* __restrict__ perm,
                                                     int64_t rows, int64_t n, double* __restrict__ X) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= rows * n) return;
    const int64_t r = t / n, a = t % n;
    X[t] = (double)load_w<In>(w, r * n + perm[a]);
}

// One tile of 64 columns, right-looking, four lanes (a quad) per row and 64 rows per
// workgroup: lane p of a quad holds the running values of tile columns 4j + p, j = 0..15, in
// registers, with their weights and scale codes.  Column b's value is broadcast to the quad,
// which quantizes it (every lane the same operations, so the same error), and each lane then
// adds error_b * U_b,a to each of its columns a > b.  Every value thus receives its terms
// b = a0, a0 + 1, ... in ascending order, as the sequential definition adds them.  U's tile
// block is staged in LDS, each lane's columns of a U row contiguous.  A column's work holds
// no branch: its scale, weight, midpoint products and U values do not depend on the running
// value, so they are formed ahead of the chain value -> quotient -> E2M1 index -> error -> the
// next column's value that bounds the walk.
struct alignas(16) TileLds {
    double T[kTile][kTile + 2];    // T[b][16 p + j] = U_{a0+b, a0+4j+p} (rows padded: the staging
                                   // writes of a wave, one per row, spread over the banks)
    int pc[kTile];
};

template <typename In>
__device__ __forceinline__ void tile_body(const In* __restrict__ w, const int* __restrict__ perm,
                                          const double* __restrict__ Uc, const uint8_t* __restrict__ scales,
                                          const float* __restrict__ tensor_scale, int64_t rows, int64_t n,
                                          int block, int64_t a0, const double* __restrict__ X,
                                          double* __restrict__ Et, uint8_t* __restrict__ codes,
                                          int64_t rblock, TileLds& L) {
    const int tid = threadIdx.x;
    for (int t = tid; t < kTile * kTile; t += 4 * kTile) {
        const int a = t / kTile, b = t % kTile;                   // coalesced over b
        L.T[b][16 * (a & 3) + (a >> 2)] = Uc[(a0 + a) * n + a0 + b];
    }
    if (tid < kTile) L.pc[tid] = perm[a0 + tid];
    __syncthreads();
    const int rr = tid >> 2, p = tid & 3;
    const int64_t r = rblock * kTile + rr;
    if (r >= rows) return;                   // whole quads: the broadcasts stay inside live rows
    const int64_t nb = n / block;
    double x[16];
    float wr[16];                            // weights of this lane's columns
    uint32_t sc4[4] = {0u, 0u, 0u, 0u};      // their scale codes, four to a register
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int c = L.pc[4 * j + p];
        x[j] = X[r * n + a0 + 4 * j + p];
        wr[j] = load_w<In>(w, r * n + c);
        sc4[j >> 2] |= (uint32_t)scales[r * nb + c / block] << (8 * (j & 3));
    }
    const float S = tensor_scale[0];
    const double halfS = 0.5 * (double)S;
    const double* Tp = &L.T[0][16 * p];
    constexpr int kTRow = kTile + 2;
    uint8_t* crow = codes + r * n;
    double* erow = Et + r * kTile;
    auto column = [&](auto bc) {
        constexpr int b = decltype(bc)::value, pb = b & 3, jb = b >> 2;
        // independent of the running values
        const int code = (int)((quad_bcast_u32<pb>(sc4[jb >> 2]) >> (8 * (jb & 3))) & 0xFFu);
        const double s = e4m3_f64(code);
        const double wv = (double)__uint_as_float(quad_bcast_u32<pb>(__float_as_uint(wr[jb])));
        const double gscale = s * halfS;     // E2M1(k) s S = (2 E2M1(k)) (s S / 2), all exact
        double m[7];                          // the midpoints times s (exact: <= 7 significant bits)
#pragma unroll
        for (int jm = 0; jm < 7; ++jm) m[jm] = e2m1_mid(jm) * s;
        // the chain
        const double xb = quad_bcast<pb>(x[jb]);
        const float y = __fdiv_rn(__double2float_rn(xb), S);
        const double ay = fabs((double)y);
        // index of the nearest E2M1 value: the midpoints passed, a tie counting only toward an
        // even index (midpoints 1, 3, 5); none for a zero scale
        int k = 0;
#pragma unroll
        for (int jm = 0; jm < 7; ++jm) k += ((jm & 1) ? ay >= m[jm] : ay > m[jm]) ? 1 : 0;
        k = code == 0 ? 0 : k;
        const bool neg = signbit(y);
        const double wq = (double)((0xC8643210u >> (4 * k)) & 15u) * gscale;
        const double e = wv - (neg ? -wq : wq);
        // the quad's four lanes store the same code and error
        crow[L.pc[b]] = (uint8_t)((neg ? 8 : 0) | k);
        erow[b] = e;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (4 * j + 3 > b) {             // some lane of the quad holds a column past b
                const double v = x[j] + e * Tp[b * kTRow + j];
                x[j] = (4 * j > b || p > pb) ? v : x[j];
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    for_each_index(column, std::make_integer_sequence<int, kTile>());
}

template <typename In>
__global__ __launch_bounds__(4 * kTile) void tile_kernel(const In* __restrict__ w, const int* __restrict__ perm,
                                                         const double* __restrict__ Uc,
                                                         const uint8_t* __restrict__ scales,
                                                         const float* __restrict__ tensor_scale,
                                                         int64_t rows, int64_t n, int block, int64_t a0,
                                                         const double* __restrict__ X,
                                                         double* __restrict__ Et,
                                                         uint8_t* __restrict__ codes) {
    __shared__ TileLds L;
    tile_body<In>(w, perm, Uc, scales, tensor_scale, rows, n, block, a0, X, Et, codes, blockIdx.x, L);
}

// X[r][k] += sum over the tile's b (in order) of Et[r][b] * U_{a0+b, k}, for k in [kstart,
// kend): one 16R x 16R output block (column block bx, row block by) per workgroup, R x R values
// per lane, the terms staged 32 at a time (so that four workgroups of the 64 x 64 blocks fit a
// CU's LDS: four waves per SIMD to issue the binary64 chains).  The 32 x 32 blocks (R = 2)
// serve the next tile's columns, which are on the critical path.
template <int R>
struct alignas(16) QTrailLdsT {
    double Es[kHalf][16 * R + 2];  // Es[b][row] (rows padded: 16-byte rows, staging writes spread)
    double Us[kHalf][16 * R + 2];  // Us[b][col]
};
using QTrailLds = QTrailLdsT<4>;

// Lane (tr, tc) owns rows r0 + R tr .. + R - 1 and columns k0 + R tc .. + R - 1, so that its X
// values and its operands of a step sit in 16-byte pairs.  kstart, kend and the blocks' columns
// are multiples of 32, so a lane's columns are all inside [kstart, kend) or all outside.
template <int R>
__device__ __forceinline__ void trailing_body(const double* __restrict__ Et, const double* __restrict__ Uc,
                                              int64_t rows, int64_t n, int64_t a0, int64_t kstart,
                                              int64_t kend, double* __restrict__ X, int64_t bx,
                                              int64_t by, QTrailLdsT<R>& L) {
    static_assert(R % 2 == 0, "pairs of values");
    constexpr int B = 16 * R;
    const int64_t r0 = by * B;
    const int64_t k0 = kstart + bx * B;
    const int tr = threadIdx.x / 16, tc = threadIdx.x % 16;      // 16 x 16 lanes, R x R each
    const int64_t kc = k0 + R * tc;
    const bool cols_in = kc < kend;
    double acc[R][R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t r = r0 + R * tr + i;
        const double2* src = reinterpret_cast<const double2*>(X + r * n + kc);
#pragma unroll
        for (int j = 0; j < R; j += 2) {
            const double2 v = (r < rows && cols_in) ? src[j / 2] : make_double2(0.0, 0.0);
            acc[i][j] = v.x;
            acc[i][j + 1] = v.y;
        }
    }
    // each half's operands are loaded into registers while the previous half is computed
    constexpr int kPer = B * kHalf / 256;
    double pe[kPer], pu[kPer];
    auto fetch = [&](int h) {
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int t = threadIdx.x + 256 * e, rr = t / kHalf, b = t % kHalf;   // coalesced over b
            pe[e] = r0 + rr < rows ? Et[(r0 + rr) * kTile + h + b] : 0.0;
            pu[e] = k0 + rr < kend ? Uc[(k0 + rr) * n + a0 + h + b] : 0.0;
        }
    };
    fetch(0);
    for (int h = 0; h < kTile; h += kHalf) {
        __syncthreads();                                          // the previous half is used
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int t = threadIdx.x + 256 * e, rr = t / kHalf, b = t % kHalf;
            L.Es[b][rr] = pe[e];
            L.Us[b][rr] = pu[e];
        }
        __syncthreads();
        if (h + kHalf < kTile) fetch(h + kHalf);
#pragma unroll(R == 2 ? 4 : 2)
        for (int b = 0; b < kHalf; ++b) {
            double e[R], u[R];
            const double2* ep = reinterpret_cast<const double2*>(&L.Es[b][R * tr]);
            const double2* up = reinterpret_cast<const double2*>(&L.Us[b][R * tc]);
#pragma unroll
            for (int i = 0; i < R; i += 2) {
                const double2 ev = ep[i / 2], uv = up[i / 2];
                e[i] = ev.x;
                e[i + 1] = ev.y;
                u[i] = uv.x;
                u[i + 1] = uv.y;
            }
#pragma unroll
            for (int i = 0; i < R; ++i)
#pragma unroll
                for (int j = 0; j < R; ++j) acc[i][j] = acc[i][j] + e[i] * u[j];
        }
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t r = r0 + R * tr + i;
        if (r < rows && cols_in) {
            double2* dst = reinterpret_cast<double2*>(X + r * n + kc);
#pragma unroll
            for (int j = 0; j < R; j += 2) dst[j / 2] = make_double2(acc[i][j], acc[i][j + 1]);
        }
    }
}

template <int R>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void trailing_kernel(
        const double* __restrict__ Et, const double* __restrict__ Uc, int64_t rows, int64_t n, int64_t a0,
        int64_t kstart, int64_t kend, double* __restrict__ X) {
    __shared__ QTrailLdsT<R> L;
    trailing_body<R>(Et, Uc, rows, n, a0, kstart, kend, X, blockIdx.x, blockIdx.y, L);
}

// Look-ahead: the next tile (workgroups 0 .. ntile-1, its errors into Etn) beside the rest of
// the current tile's trailing update, columns [kstart, n) with the current tile's errors Etc
// (the other workgroups, ncb column blocks per row block).  The next tile's columns already
// hold every earlier term; the two touch disjoint values.
template <typename In>
__global__ __launch_bounds__(4 * kTile) __attribute__((amdgpu_waves_per_eu(4))) void tile_lookahead_kernel(
        const In* __restrict__ w, const int* __restrict__ perm, const double* __restrict__ Uc,
        const uint8_t* __restrict__ scales, const float* __restrict__ tensor_scale, int64_t rows,
        int64_t n, int block, int64_t a0n, double* __restrict__ X, double* __restrict__ Etn,
        uint8_t* __restrict__ codes, int64_t ntile, const double* __restrict__ Etc, int64_t a0c,
        int64_t kstart, int64_t ncb) {
    __shared__ union {
        TileLds t;
        QTrailLds q;
    } L;
    if ((int64_t)blockIdx.x < ntile) {
        tile_body<In>(w, perm, Uc, scales, tensor_scale, rows, n, block, a0n, X, Etn, codes, blockIdx.x,
                      L.t);
    } else {
        const int64_t idx = blockIdx.x - ntile;
        trailing_body<4>(Etc, Uc, rows, n, a0c, kstart, n, X, idx % ncb, idx / ncb, L.q);
    }
}

__global__ __launch_bounds__(256) void pack_kernel(const uint8_t* __restrict__ codes, int64_t npairs,
                                                   uint8_t* __restrict__ q) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t < npairs) q[t] = (uint8_t)(codes[2 * t] | (codes[2 * t + 1] << 4));
}

__global__ void clear_status_kernel(int* status) { status[0] = 0; }

// ---- workspace ---------------------------------------------------------------------------

struct Layout {
    size_t perm, diag, lambda, D, Uc, X, Et, codes, total;
};

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

Layout layout_of(int64_t rows, int64_t n) {
    Layout l;
    size_t o = 0;
    l.perm = o;   o = align256(o + (size_t)n * sizeof(int));
    l.diag = o;   o = align256(o + (size_t)n * sizeof(double));
    l.lambda = o; o = align256(o + sizeof(double));
    l.D = o;      o = align256(o + (size_t)n * sizeof(double));
    l.Uc = o;     o = align256(o + (size_t)n * n * sizeof(double));
    l.X = o;      o = align256(o + (size_t)rows * n * sizeof(double));
    l.Et = o;     o = align256(o + (size_t)2 * rows * kTile * sizeof(double));   // two tiles in turn
    l.codes = o;  o = align256(o + (size_t)rows * n);
    l.total = o;
    return l;
}

unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

template <typename In>
int run_ldlq(const void* wv, int64_t rows, int64_t n, int block, const double* H,
             const uint8_t* scales, const float* S, double damp, uint8_t* q, int* status,
             char* ws, hipStream_t st) {
    const In* w = static_cast<const In*>(wv);
    const Layout l = layout_of(rows, n);
    int* perm = reinterpret_cast<int*>(ws + l.perm);
    double* diag = reinterpret_cast<double*>(ws + l.diag);
    double* lambda = reinterpret_cast<double*>(ws + l.lambda);
    double* D = reinterpret_cast<double*>(ws + l.D);
    double* Uc = reinterpret_cast<double*>(ws + l.Uc);
    double* X = reinterpret_cast<double*>(ws + l.X);
    double* Et = reinterpret_cast<double*>(ws + l.Et);
    uint8_t* codes = reinterpret_cast<uint8_t*>(ws + l.codes);

    hipLaunchKernelGGL(clear_status_kernel, dim3(1), dim3(1), 0, st, status);
    hipLaunchKernelGGL(diag_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, H, n, diag);
    hipLaunchKernelGGL(order_kernel, dim3(blocks_for(n, 64)), dim3(64 * kOrderParts), 0, st, diag, n, perm);
    hipLaunchKernelGGL(damping_kernel, dim3(1), dim3(64), 0, st, diag, n, damp, lambda);
    if (hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
    hipLaunchKernelGGL(init_a_kernel, dim3(blocks_for(n * n, 256)), dim3(256), 0, st, H, perm, lambda,
                       n, Uc);
    // factor, from the last block: its diagonal block, then per block the panel above it, the
    // column of tiles the next diagonal block and panel need, and then the next diagonal block
    // beside the rest of the trailing update (look-ahead)
    hipLaunchKernelGGL(factor_diag_kernel, dim3(1), dim3(4 * kTile), 0, st, Uc, D, n, n - kTile, status);
    for (int64_t k0 = n - kTile; k0 > 0; k0 -= kTile) {
        hipLaunchKernelGGL(factor_panel_kernel, dim3(blocks_for(k0, kPanelRows)), dim3(256), 0, st, Uc, D,
                           n, k0);
        const int64_t nb = k0 / kTile - 1;                         // the next block's tile column
        hipLaunchKernelGGL(factor_trailing_kernel<2>, dim3(2, (unsigned)(2 * (nb + 1))), dim3(256), 0, st, Uc,
                           D, n, k0, nb * kTile);
        hipLaunchKernelGGL(factor_lookahead_kernel, dim3((unsigned)(1 + nb * nb)), dim3(256), 0, st, Uc, D,
                           n, k0, nb > 0 ? nb : 1, k0 - kTile, status);
        if (hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
    }
    hipLaunchKernelGGL(init_x_kernel<In>, dim3(blocks_for(rows * n, 256)), dim3(256), 0, st, w, perm,
                       rows, n, X);
    // quantize: tile 0, then per tile the next tile's columns, and then the next tile beside
    // the rest of the trailing update (look-ahead); the tiles' errors alternate between two
    // buffers
    const unsigned rblocks = blocks_for(rows, kTile);
    hipLaunchKernelGGL(tile_kernel<In>, dim3(rblocks), dim3(4 * kTile), 0, st, w, perm, Uc, scales, S,
                       rows, n, block, (int64_t)0, X, Et, codes);
    for (int64_t a0 = 0; a0 + kTile < n; a0 += kTile) {
        double* Etc = Et + ((a0 / kTile) & 1) * rows * kTile;
        double* Etn = Et + (((a0 / kTile) + 1) & 1) * rows * kTile;
        hipLaunchKernelGGL(trailing_kernel<2>, dim3(2, blocks_for(rows, 32)), dim3(256), 0, st, Etc, Uc, rows,
                           n, a0, a0 + kTile, a0 + 2 * kTile, X);
        const int64_t rest = n - (a0 + 2 * kTile);                  // columns past the next tile
        const int64_t ncb = (rest + kTile - 1) / kTile;
        hipLaunchKernelGGL(tile_lookahead_kernel<In>, dim3((unsigned)(rblocks + ncb * rblocks)),
                           dim3(4 * kTile), 0, st, w, perm, Uc, scales, S, rows, n, block, a0 + kTile, X, Etn,
                           codes, (int64_t)rblocks, Etc, a0, a0 + 2 * kTile, ncb > 0 ? ncb : 1);
        if (hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
    }
    hipLaunchKernelGGL(pack_kernel, dim3(blocks_for(rows * n / 2, 256)), dim3(256), 0, st, codes,
                       rows * n / 2, q);
    return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

}  // namespace

extern "C" {

size_t nvfp4_ldlq_workspace_bytes(int64_t rows, int64_t cols) {
    if (rows < 0 || cols < 0) return 0;
    return layout_of(rows, cols).total;
}

int nvfp4_ldlq(const void* w, int dtype, int64_t rows, int64_t cols, int block, const double* hessian,
               const uint8_t* scales, const float* tensor_scale, double damp, uint8_t* q, int* status,
               void* workspace, size_t workspace_bytes, void* stream) {
    if (dtype != NVFP4_IN_F32 && dtype != NVFP4_IN_BF16) return NVFP4_ERR_DTYPE;
    if (block != 16 && block != 32 && block != 64 && block != 128) return NVFP4_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % kTile != 0) return NVFP4_ERR_SHAPE;
    if (cols > 0x7FFFFFFF || rows * cols > ((int64_t)1 << 40)) return NVFP4_ERR_SHAPE;
    if (!(damp >= 0.0) || !isfinite(damp)) return NVFP4_ERR_ARG;
    if (!status || !tensor_scale) return NVFP4_ERR_NULL;
    if (rows * cols > 0 && (!w || !hessian || !scales || !q)) return NVFP4_ERR_NULL;
    if (((uintptr_t)hessian & 7) || ((uintptr_t)status & 3)) return NVFP4_ERR_ALIGN;
    hipStream_t st = (hipStream_t)stream;
    if (rows * cols == 0) {
        hipLaunchKernelGGL(clear_status_kernel, dim3(1), dim3(1), 0, st, status);
        return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
    }
    if (!workspace || workspace_bytes < layout_of(rows, cols).total) return NVFP4_ERR_WORKSPACE;
    if ((uintptr_t)workspace & 255) return NVFP4_ERR_ALIGN;
    char* ws = static_cast<char*>(workspace);
    return dtype == NVFP4_IN_F32
        ? run_ldlq<float>(w, rows, cols, block, hessian, scales, tensor_scale, damp, q, status, ws, st)
        : run_ldlq<uint16_t>(w, rows, cols, block, hessian, scales, tensor_scale, damp, q, status, ws, st);
}

}  // extern "C"
