// Reference block scales for NVFP4 gap reports, on AMD Instinct MI355X (gfx950):
//   * the optimal real (FP32) block scale and its loss (appendix "Optimal FP32 Scale for FP4
//     Quantization", first paragraph);
//   * the FP8-quantized optimal scale (same appendix, second paragraph);
//   * the exact loss of given E4M3 block scales, and a deterministic binary64 sum,
// for the relative gaps of AbsMax, 4/6 and ScaleSweep to the optimum (Figures 1 and 4).
//
// The loss of one block, L(s) = sum_i w_i (|y_i| - RNE_FP4(|y_i| / s) s)^2, is piecewise
// quadratic in s; it changes pieces where |y_i| / s crosses a midpoint between neighbouring
// E2M1 values, i.e. at the 7 breakpoints |y_i| / m_k of every non-zero element.  Between two
// consecutive breakpoints the rounding of every element is fixed, so L = A - 2 B s + C s^2
// there and its minimum on the closed piece is at B / C clamped to the piece.
//
// Work layout: one wavefront per micro-block.  The wave writes the block's 7 n breakpoints
// to LDS (padded with +inf to a power of two), sorts them with a bitonic network, and then
// every lane scores every 64th piece: the piece's rounding indices are taken at its
// midpoint, its coefficients summed in element order, and its minimum formed as above.  A
// wave-wide lexicographic minimum (loss, piece index) picks the optimum, the lowest piece on
// a tie, and the all-zero reconstruction (s -> infinity) ahead of any piece of equal loss.
// Everything is binary64 with correctly rounded division and no contraction, so each
// value is a fixed sequence of IEEE operations.  This is analysis work, bound by binary64
// ALU throughput, not part of the quantizers' hot path.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "exact_fp.h"
#include "nvfp4ss.h"

namespace {

constexpr int kWave = 64;

using namespace nvfp4_exact;

template <typename In>
__device__ __forceinline__ float load_elem(const In* x, int64_t i);

template <>
__device__ __forceinline__ float load_elem<float>(const float* x, int64_t i) { return x[i]; }

template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* x, int64_t i) {
    return __uint_as_float((uint32_t)x[i] << 16);        // bfloat16 -> binary32, exact
}

// Exact loss of one block at the scale s, summed in element order (binary64).
template <int N>
__device__ double block_loss_f64(const float* ys, const float* ws, bool weighted, double s) {
    double J = 0.0;
#pragma unroll 2
    for (int i = 0; i < N; ++i) {
        const double a = fabs((double)ys[i]);
        const double g = e2m1_value(round_fp4_index(a, s));
        const double e = a - g * s;
        double t = e * e;
        if (weighted) t = (double)ws[i] * t;
        J = J + t;
    }
    return J;
}

struct Best {
    double val, s;
    int seg;                 // -1: the all-zero reconstruction
};

__device__ __forceinline__ bool better(const Best& a, const Best& b) {
    return a.val < b.val || (a.val == b.val && a.seg < b.seg);
}

template <int N>
struct Pow2Breaks {
    static constexpr int M = 7 * N;
    static constexpr int P = M <= 128 ? 128 : M <= 256 ? 256 : M <= 512 ? 512 : 1024;
};

template <typename In, int N>
__global__ __launch_bounds__(kWave) void optimum_kernel(const In* __restrict__ x,
                                                        const float* __restrict__ colw,
                                                        const float* __restrict__ tensor_scale,
                                                        int64_t nblocks, int64_t bpr,
                                                        double* __restrict__ opt_loss,
                                                        double* __restrict__ opt_scale,
                                                        uint8_t* __restrict__ fp8_code,
                                                        double* __restrict__ fp8_loss) {
    constexpr int P = Pow2Breaks<N>::P;
    __shared__ double bp[P];
    __shared__ float ys[N], wsh[N];
    __shared__ double ad[N], wd[N], wad[N];   // |y|, w, w |y| in binary64 (per block)
    __shared__ double g_tab[8];
    if (threadIdx.x < 8) g_tab[threadIdx.x] = e2m1_value(threadIdx.x);
    const int lane = threadIdx.x;
    const float S = tensor_scale[0];
    const bool weighted = colw != nullptr;

    for (int64_t blk = blockIdx.x; blk < nblocks; blk += gridDim.x) {
        const int64_t kb = blk % bpr;
        int nonzero = 0;
        for (int i = lane; i < N; i += kWave) {
            const float y = __fdiv_rn(load_elem<In>(x, blk * N + i), S);   // y = RN32(x / S)
            ys[i] = y;
            wsh[i] = weighted ? colw[kb * N + i] : 1.0f;
            const double a = fabs((double)y);
            const double wi = weighted ? (double)wsh[i] : 1.0;
            ad[i] = a;
            wd[i] = wi;
            wad[i] = wi * a;
        }
        __syncthreads();
        for (int i = 0; i < N; i += kWave) {
            const bool nz = i + lane < N && ys[i + lane] != 0.0f;
            nonzero += __popcll(__ballot(nz));
        }
        const int nb = 7 * nonzero;
        for (int t = lane; t < P; t += kWave) {
            double v = INFINITY;
            if (t < 7 * N) {
                const double a = fabs((double)ys[t / 7]);
                if (a != 0.0) v = a / e2m1_mid(t % 7);
            }
            bp[t] = v;
        }
        __syncthreads();
        // ascending bitonic sort of the P breakpoints (+inf padding sorts last)
        for (int size = 2; size <= P; size <<= 1) {
            for (int ls = __builtin_ctz(size) - 1; ls >= 0; --ls) {   // stride = 2^ls
                const int stride = 1 << ls;
                for (int t = lane; t < P / 2; t += kWave) {
                    const int i = ((t >> ls) << (ls + 1)) + (t & (stride - 1));
                    const int j = i + stride;
                    const bool asc = (i & size) == 0;
                    const double u = bp[i], v = bp[j];
                    if ((u > v) == asc) {
                        bp[i] = v;
                        bp[j] = u;
                    }
                }
                __syncthreads();
            }
        }

        double A0 = 0.0;                       // the all-zero reconstruction: sum w y^2
        for (int i = 0; i < N; ++i) {
            const double a = (double)ys[i];
            A0 += (weighted ? (double)wsh[i] : 1.0) * a * a;
        }
        Best best{A0, INFINITY, -1};
        for (int seg = lane; seg <= nb; seg += kWave) {
            const double lo = seg == 0 ? 0.0 : bp[seg - 1];
            const double hi = seg == nb ? INFINITY : bp[seg];
            if (!(hi > lo)) continue;
            const double s_ref = seg == 0 ? 0.5 * hi : seg == nb ? 2.0 * lo : 0.5 * (lo + hi);
            // A = sum w y^2 is the same on every piece (and equals A0 bit for bit: w |y| |y|
            // and w y y round alike), so only B and C are summed here
            const double A = A0;
            double B = 0.0, C = 0.0;
#pragma unroll 4
            for (int i = 0; i < N; ++i) {
                const double g = g_tab[round_fp4_index(ad[i], s_ref)];
                B += wad[i] * g;                 // (w |y|) g, as w * a * g associates
                C += wd[i] * g * g;
            }
            Best cand{0.0, 0.0, seg};
            if (C <= 0.0) {
                cand.val = A;
                cand.s = s_ref;
            } else {
                double s = B / C;
                if (s < lo) s = lo;
                if (s > hi) s = hi;
                if (s <= 0.0) continue;
                double val = A - 2.0 * B * s + C * s * s;
                if (val < 0.0) val = 0.0;
                cand.val = val;
                cand.s = s;
            }
            if (better(cand, best)) best = cand;
        }
        for (int off = kWave / 2; off > 0; off >>= 1) {
            Best o;
            o.val = __shfl_xor(best.val, off, kWave);
            o.s = __shfl_xor(best.s, off, kWave);
            o.seg = __shfl_xor(best.seg, off, kWave);
            if (better(o, best)) best = o;
        }
        double J = best.val, s_opt = best.s;
        if (nb == 0) {                          // all-zero block: zero loss at any scale
            J = 0.0;
            s_opt = 1.0;
        }
        if (lane == 0) {
            opt_loss[blk] = J;
            if (opt_scale) opt_scale[blk] = s_opt;
            if (fp8_code || fp8_loss) {
                // the FP8 values just below and just above s_opt; the lower-loss one (the
                // lower value on a tie); positive codes only
                int cf = floor_e4m3(s_opt);
                int cc = (e4m3_f64(cf) < s_opt && cf < 126) ? cf + 1 : cf;
                cf = cf < 1 ? 1 : cf;
                cc = cc < 1 ? 1 : cc;
                const double jf = block_loss_f64<N>(ys, wsh, weighted, e4m3_f64(cf));
                const double jc = block_loss_f64<N>(ys, wsh, weighted, e4m3_f64(cc));
                if (fp8_code) fp8_code[blk] = (uint8_t)(jc < jf ? cc : cf);
                if (fp8_loss) fp8_loss[blk] = jc < jf ? jc : jf;
            }
        }
        __syncthreads();                        // LDS is reused by the next block
    }
}

// Exact loss of each block at its given E4M3 scale code: one lane per block.
template <typename In, int N>
__global__ __launch_bounds__(256) void block_loss_kernel(const In* __restrict__ x,
                                                         const float* __restrict__ colw,
                                                         const float* __restrict__ tensor_scale,
                                                         const uint8_t* __restrict__ scales,
                                                         int64_t nblocks, int64_t bpr,
                                                         double* __restrict__ loss) {
    const int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (blk >= nblocks) return;
    const float S = tensor_scale[0];
    const int64_t kb = blk % bpr;
    const int code = scales[blk] > 126 ? 126 : scales[blk];
    const double s = e4m3_f64(code);
    double J = 0.0;
    for (int i = 0; i < N; ++i) {
        const float y = __fdiv_rn(load_elem<In>(x, blk * N + i), S);
        const double a = fabs((double)y);
        const double g = e2m1_value(round_fp4_index(a, s));
        const double e = a - g * s;
        double t = e * e;
        if (colw) t = (double)colw[kb * N + i] * t;
        J = J + t;
    }
    loss[blk] = J;
}

// Deterministic binary64 sum: each of G <= 256 workgroups sums a fixed slice (a strided
// per-thread sum, then a fixed tree), and one wave adds the G partials in a fixed tree.
constexpr int kSumThreads = 256, kSumParts = 256;

__global__ __launch_bounds__(kSumThreads) void sum_partial_kernel(const double* __restrict__ v,
                                                                  int64_t n, double* __restrict__ part) {
    __shared__ double sh[kSumThreads];
    double acc = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * kSumThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kSumThreads)
        acc += v[i];
    sh[threadIdx.x] = acc;
    __syncthreads();
    for (int h = kSumThreads / 2; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) sh[threadIdx.x] += sh[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) part[blockIdx.x] = sh[0];
}

__global__ __launch_bounds__(kWave) void sum_final_kernel(const double* __restrict__ part, int g,
                                                          double* __restrict__ out) {
    double acc = 0.0;
    for (int i = threadIdx.x; i < g; i += kWave) acc += part[i];
    for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
    if (threadIdx.x == 0) out[0] = acc;
}

bool aligned_to(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int check_tensor(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                 const float* col_weight, const float* tensor_scale) {
    if (!tensor_scale) return NVFP4_ERR_NULL;
    if (dtype != NVFP4_IN_F32 && dtype != NVFP4_IN_BF16) return NVFP4_ERR_DTYPE;
    if (block != 16 && block != 32 && block != 64 && block != 128) return NVFP4_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block != 0) return NVFP4_ERR_SHAPE;
    if (rows * cols > 0 && !x) return NVFP4_ERR_NULL;
    if (x && !aligned_to(x, dtype == NVFP4_IN_F32 ? 4 : 2)) return NVFP4_ERR_ALIGN;
    if (col_weight && !aligned_to(col_weight, 4)) return NVFP4_ERR_ALIGN;
    return NVFP4_OK;
}

template <typename In, int N>
hipError_t launch_optimum(const void* x, const float* colw, const float* S, int64_t nblocks,
                          int64_t bpr, double* opt_loss, double* opt_scale, uint8_t* code,
                          double* fp8_loss, hipStream_t st) {
    const int64_t grid = nblocks < 65536 ? nblocks : 65536;    // grid-stride over blocks
    hipLaunchKernelGGL((optimum_kernel<In, N>), dim3((unsigned)grid), dim3(kWave), 0, st,
                       static_cast<const In*>(x), colw, S, nblocks, bpr, opt_loss, opt_scale,
                       code, fp8_loss);
    return hipGetLastError();
}

template <typename In, int N>
hipError_t launch_loss(const void* x, const float* colw, const float* S, const uint8_t* scales,
                       int64_t nblocks, int64_t bpr, double* loss, hipStream_t st) {
    const int64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL((block_loss_kernel<In, N>), dim3((unsigned)grid), dim3(256), 0, st,
                       static_cast<const In*>(x), colw, S, scales, nblocks, bpr, loss);
    return hipGetLastError();
}

template <typename In>
hipError_t dispatch_optimum(int block, const void* x, const float* colw, const float* S,
                            int64_t nblocks, int64_t bpr, double* l, double* s, uint8_t* c,
                            double* f, hipStream_t st) {
    switch (block) {
        case 16: return launch_optimum<In, 16>(x, colw, S, nblocks, bpr, l, s, c, f, st);
        case 32: return launch_optimum<In, 32>(x, colw, S, nblocks, bpr, l, s, c, f, st);
        case 64: return launch_optimum<In, 64>(x, colw, S, nblocks, bpr, l, s, c, f, st);
        default: return launch_optimum<In, 128>(x, colw, S, nblocks, bpr, l, s, c, f, st);
    }
}

template <typename In>
hipError_t dispatch_loss(int block, const void* x, const float* colw, const float* S,
                         const uint8_t* scales, int64_t nblocks, int64_t bpr, double* loss,
                         hipStream_t st) {
    switch (block) {
        case 16: return launch_loss<In, 16>(x, colw, S, scales, nblocks, bpr, loss, st);
        case 32: return launch_loss<In, 32>(x, colw, S, scales, nblocks, bpr, loss, st);
        case 64: return launch_loss<In, 64>(x, colw, S, scales, nblocks, bpr, loss, st);
        default: return launch_loss<In, 128>(x, colw, S, scales, nblocks, bpr, loss, st);
    }
}

}  // namespace

extern "C" {

int nvfp4_block_optimum(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                        const float* col_weight, const float* tensor_scale, double* opt_loss,
                        double* opt_scale, uint8_t* fp8_code, double* fp8_loss, void* stream) {
    const int rc = check_tensor(x, dtype, rows, cols, block, col_weight, tensor_scale);
    if (rc != NVFP4_OK) return rc;
    const int64_t nblocks = rows * cols / block;
    if (nblocks == 0) return NVFP4_OK;
    if (!opt_loss) return NVFP4_ERR_NULL;
    if (!aligned_to(opt_loss, 8) || (opt_scale && !aligned_to(opt_scale, 8)) ||
        (fp8_loss && !aligned_to(fp8_loss, 8)))
        return NVFP4_ERR_ALIGN;
    hipStream_t st = (hipStream_t)stream;
    const hipError_t e = dtype == NVFP4_IN_F32
        ? dispatch_optimum<float>(block, x, col_weight, tensor_scale, nblocks, cols / block,
                                  opt_loss, opt_scale, fp8_code, fp8_loss, st)
        : dispatch_optimum<uint16_t>(block, x, col_weight, tensor_scale, nblocks, cols / block,
                                     opt_loss, opt_scale, fp8_code, fp8_loss, st);
    return e == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

int nvfp4_block_loss(const void* x, int dtype, int64_t rows, int64_t cols, int block,
                     const float* col_weight, const float* tensor_scale, const uint8_t* scales,
                     double* loss, void* stream) {
    const int rc = check_tensor(x, dtype, rows, cols, block, col_weight, tensor_scale);
    if (rc != NVFP4_OK) return rc;
    const int64_t nblocks = rows * cols / block;
    if (nblocks == 0) return NVFP4_OK;
    if (!scales || !loss) return NVFP4_ERR_NULL;
    if (!aligned_to(loss, 8)) return NVFP4_ERR_ALIGN;
    hipStream_t st = (hipStream_t)stream;
    const hipError_t e = dtype == NVFP4_IN_F32
        ? dispatch_loss<float>(block, x, col_weight, tensor_scale, scales, nblocks, cols / block, loss, st)
        : dispatch_loss<uint16_t>(block, x, col_weight, tensor_scale, scales, nblocks, cols / block, loss, st);
    return e == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

size_t nvfp4_sum_workspace_bytes(void) { return kSumParts * sizeof(double); }

int nvfp4_sum_f64(const double* v, int64_t n, double* out, void* workspace,
                  size_t workspace_bytes, void* stream) {
    if (!out) return NVFP4_ERR_NULL;
    if (n < 0) return NVFP4_ERR_SHAPE;
    if (n > 0 && !v) return NVFP4_ERR_NULL;
    if (!workspace || workspace_bytes < kSumParts * sizeof(double)) return NVFP4_ERR_WORKSPACE;
    if (!aligned_to(workspace, 8) || !aligned_to(out, 8) || (v && !aligned_to(v, 8)))
        return NVFP4_ERR_ALIGN;
    hipStream_t st = (hipStream_t)stream;
    int64_t g = (n + kSumThreads * 8 - 1) / (kSumThreads * 8);
    if (g < 1) g = 1;
    if (g > kSumParts) g = kSumParts;
    double* part = static_cast<double*>(workspace);
    hipLaunchKernelGGL(sum_partial_kernel, dim3((unsigned)g), dim3(kSumThreads), 0, st, v, n, part);
    if (hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
    hipLaunchKernelGGL(sum_final_kernel, dim3(1), dim3(kWave), 0, st, part, (int)g, out);
    return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

}  // extern "C"
