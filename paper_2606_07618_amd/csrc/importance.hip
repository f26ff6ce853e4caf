// Importance vectors for the WMSE objective on AMD Instinct MI355X (gfx950): squared norms
// of input channels (WMSE section; "Quantization" paragraph of the implementation details).
//   * weights W [d_out, d_in]: Imp_j = ||W[:, j]||^2 over the calibration activations X of
//     the layer -- here any matrix whose column norms are wanted;
//   * activations: the squared norms of the consuming weight's input channels;
//   * query states, key cache, value cache: the input-channel squared norms of K, Q and W^O.
// A matrix x [rows, cols] is reduced column-wise into groups of rows: row r belongs to group
// ((r / group_rows) mod groups) / group_div, so attention tensors laid out as
// [batch * heads * tokens, head_dim] reduce per head (group_rows = tokens, groups = heads),
// and group_div merges the query heads that share a KV head.
//
// Pass 1: a wavefront owns 64 adjacent columns of a chunk of rows (256 or more, at most 2048
// chunks); each lane walks its column down the chunk in runs of rows of one group (eight
// coalesced row segments in flight), accumulating in binary64 into an LDS accumulator per
// group, then writes the chunk's per-group partial sums.  Pass 2 adds the partials of each
// (group, column) in a fixed order (sixteen contiguous runs of chunks, then the sixteen run
// sums) and rounds once to binary32.  The order is fixed, so results are deterministic.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "nvfp4ss.h"

namespace {

constexpr int kLanes = 64;
constexpr int64_t kMinChunkRows = 256;
constexpr int64_t kMaxChunks = 2048;

// Rows per chunk: at least 256, and few enough chunks that the final pass stays short.
int64_t chunk_rows_for(int64_t rows) {
    const int64_t c = (rows + kMaxChunks - 1) / kMaxChunks;
    return c <= kMinChunkRows ? kMinChunkRows : (c + 7) / 8 * 8;
}
constexpr int kMaxGroups = 64;

template <typename In>
__device__ __forceinline__ float load_value(const In* x, int64_t i);

template <>
__device__ __forceinline__ float load_value<float>(const float* x, int64_t i) { return x[i]; }

template <>
__device__ __forceinline__ float load_value<uint16_t>(const uint16_t* x, int64_t i) {
    return __uint_as_float((uint32_t)x[i] << 16);
}

template <typename In>
__global__ __launch_bounds__(kLanes) void norms_partial_kernel(const In* __restrict__ x, int64_t rows,
                                                               int64_t cols, int64_t group_rows,
                                                               int64_t groups, int64_t group_div,
                                                               int gout, int64_t chunk_rows,
                                                               double* __restrict__ part) {
    extern __shared__ double acc_lds[];          // [gout][64]: sized at launch
    double (*acc_g)[kLanes] = reinterpret_cast<double (*)[kLanes]>(acc_lds);
    const int lane = threadIdx.x;
    const int64_t c = (int64_t)blockIdx.x * kLanes + lane;
    const int64_t r0 = (int64_t)blockIdx.y * chunk_rows;
    const int64_t r1 = r0 + chunk_rows < rows ? r0 + chunk_rows : rows;
    for (int g = 0; g < gout; ++g) acc_g[g][lane] = 0.0;
    // rows are walked in runs of one group: r = q * group_rows + rem, and q mod groups =
    // gd * group_div + gm, so a run ends after (group_div - gm) * group_rows - rem rows
    int64_t rem = r0 % group_rows;
    const int64_t gi = (r0 / group_rows) % groups;
    int64_t gm = gi % group_div;
    int gd = (int)(gi / group_div);
    const bool col_ok = c < cols;
    const In* xc = x + (col_ok ? c : 0);
    for (int64_t r = r0; r < r1;) {
        const int64_t run = (group_div - gm) * group_rows - rem;
        const int64_t end = r + run < r1 ? r + run : r1;
        double acc = 0.0;
        int64_t rr = r;
        for (; rr + 8 <= end; rr += 8) {          // eight independent loads in flight
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = load_value<In>(xc, (rr + j) * cols);
#pragma unroll
            for (int j = 0; j < 8; ++j) acc += (double)v[j] * (double)v[j];
        }
        for (; rr < end; ++rr) {
            const double v = (double)load_value<In>(xc, rr * cols);
            acc += v * v;
        }
        if (col_ok) acc_g[gd][lane] += acc;
        r = end;
        rem = 0;
        gm = 0;
        gd = gd + 1 == gout ? 0 : gd + 1;
    }
    if (c < cols)
        for (int g = 0; g < gout; ++g)
            part[((int64_t)blockIdx.y * gout + g) * cols + c] = acc_g[g][lane];
}

// One workgroup per (group, 64 columns): 16 waves each add a contiguous sixteenth of the chunk
// partials in order (eight loads in flight), then the sixteen sums are added in order.
constexpr int kFinalSubs = 16;

__global__ __launch_bounds__(kLanes * kFinalSubs) void norms_final_kernel(
        const double* __restrict__ part, int64_t nchunks, int64_t cols, int gout, int64_t rep_out,
        float* __restrict__ out) {
    __shared__ double sub_sum[kFinalSubs][kLanes];
    const int lane = threadIdx.x % kLanes, sub = threadIdx.x / kLanes;
    const int64_t tiles = (cols + kLanes - 1) / kLanes;
    const int64_t g = blockIdx.x / tiles;
    const int64_t c = (blockIdx.x % tiles) * kLanes + lane;
    const int64_t per = (nchunks + kFinalSubs - 1) / kFinalSubs;
    const int64_t k0 = sub * per, k1 = k0 + per < nchunks ? k0 + per : nchunks;
    double s = 0.0;
    if (c < cols) {
        const double* p = part + g * cols + c;
        const int64_t stride = (int64_t)gout * cols;
        int64_t k = k0;
        for (; k + 8 <= k1; k += 8) {
            double v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = p[(k + j) * stride];
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[j];
        }
        for (; k < k1; ++k) s += p[k * stride];
    }
    sub_sum[sub][lane] = s;
    __syncthreads();
    if (sub == 0 && c < cols) {
        double t = 0.0;
        for (int j = 0; j < kFinalSubs; ++j) t += sub_sum[j][lane];
        const float v = (float)t;
        for (int64_t j = 0; j < rep_out; ++j) out[(g * rep_out + j) * cols + c] = v;
    }
}

int64_t workspace_bytes(int64_t rows, int64_t cols, int64_t groups, int64_t group_div) {
    if (rows < 0 || cols < 0) return NVFP4_ERR_SHAPE;
    if (groups < 1 || group_div < 1 || groups % group_div) return NVFP4_ERR_ARG;
    const int64_t gout = groups / group_div;
    if (gout > kMaxGroups) return NVFP4_ERR_ARG;
    const int64_t cr = chunk_rows_for(rows);
    const int64_t nchunks = (rows + cr - 1) / cr;
    return nchunks * gout * cols * (int64_t)sizeof(double);
}

}  // namespace

extern "C" {

int64_t nvfp4_channel_sq_norms_workspace_bytes(int64_t rows, int64_t cols, int64_t groups,
                                               int64_t group_div) {
    return workspace_bytes(rows, cols, groups, group_div);
}

int nvfp4_channel_sq_norms(const void* x, int dtype, int64_t rows, int64_t cols, int64_t group_rows,
                           int64_t groups, int64_t group_div, int64_t rep_out, float* out,
                           void* workspace, size_t ws_bytes, void* stream) {
    if (dtype != NVFP4_IN_F32 && dtype != NVFP4_IN_BF16) return NVFP4_ERR_DTYPE;
    const int64_t need = workspace_bytes(rows, cols, groups, group_div);
    if (need < 0) return (int)need;
    if (group_rows < 1 || rep_out < 1) return NVFP4_ERR_ARG;
    if (!out) return NVFP4_ERR_NULL;
    const int64_t gout = groups / group_div;
    const int64_t cr = chunk_rows_for(rows);
    const int64_t nchunks = (rows + cr - 1) / cr;
    if ((cols + kLanes - 1) / kLanes > 0x7FFFFFFF) return NVFP4_ERR_SHAPE;
    if (cols == 0) return NVFP4_OK;
    hipStream_t st = (hipStream_t)stream;
    if (rows > 0 && !x) return NVFP4_ERR_NULL;
    if (rows > 0 && (!workspace || (int64_t)ws_bytes < need)) return NVFP4_ERR_WORKSPACE;
    if (((uintptr_t)workspace & 7) || ((uintptr_t)out & 3)) return NVFP4_ERR_ALIGN;
    double* part = static_cast<double*>(workspace);
    const dim3 grid((unsigned)((cols + kLanes - 1) / kLanes), (unsigned)nchunks);
    const size_t lds = (size_t)gout * kLanes * sizeof(double);
    if (rows == 0) {
        // no rows: the final pass writes zeros (it reads no partials)
    } else if (dtype == NVFP4_IN_F32)
        hipLaunchKernelGGL(norms_partial_kernel<float>, grid, dim3(kLanes), lds, st,
                           static_cast<const float*>(x), rows, cols, group_rows, groups, group_div,
                           (int)gout, cr, part);
    else
        hipLaunchKernelGGL(norms_partial_kernel<uint16_t>, grid, dim3(kLanes), lds, st,
                           static_cast<const uint16_t*>(x), rows, cols, group_rows, groups,
                           group_div, (int)gout, cr, part);
    if (rows > 0 && hipGetLastError() != hipSuccess) return NVFP4_ERR_HIP;
    const int64_t nwg = gout * ((cols + kLanes - 1) / kLanes);
    hipLaunchKernelGGL(norms_final_kernel, dim3((unsigned)nwg), dim3(kLanes * kFinalSubs), 0, st, part,
                       rows > 0 ? nchunks : 0, cols, (int)gout, rep_out, out);
    return hipGetLastError() == hipSuccess ? NVFP4_OK : NVFP4_ERR_HIP;
}

}  // extern "C"
