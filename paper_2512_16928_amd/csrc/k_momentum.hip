// K1: momentum accumulate fused with the line-norm reduction.
//
// M <- fl32(M + G) in place (Algorithm 1, accumulate step) and, for every line of
// the selection axis, the l1 norm (Select_alpha, Default rule) and the
// squared l2 norm (for ||M[K]||_F, the Newton-Schulz normalisation).
// The l1 norm is accumulated in double-double from the fp32 values and
// rounded once at the end, which gives the exactly rounded sum unless the
// exact sum lies within ~n*2^-106 (relative) of an fp64 rounding boundary.
//
// Row mode: one wave per row (four rows per 256-thread block); every lane
// streams 4-element vectors (16 B of M, 8 B of bf16 G), eight vectors in
// flight, and the wave reduces in a fixed shuffle order. M and G are
// streamed with non-temporal loads and stores (each is touched once).
// Column mode: M is only read here (the gather pass rewrites whole rows of
// M once the selection is known, so the sum is stored once); each thread
// owns 4 adjacent columns of a block of rows and writes double-double
// partials, and a second pass folds the row blocks in order. No
// floating-point atomics anywhere: results are run-to-run bitwise
// reproducible.
#include <type_traits>

#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void accumulate(double x, double& hi, double& lo, double& s2) {
    double s, e;
    two_sum(hi, x, s, e);
    hi = s;
    lo += e;
    s2 += x * x;
}

// Fixed-order wave reduction of (hi, lo, s2); result valid in every lane.
__device__ __forceinline__ void wave_reduce(double& hi, double& lo, double& s2) {
    for (int off = 32; off > 0; off >>= 1) {
        double ohi = __shfl_xor(hi, off);
        double olo = __shfl_xor(lo, off);
        double os2 = __shfl_xor(s2, off);
        dd_add(hi, lo, ohi, olo);
        s2 += os2;
    }
}

constexpr int kRowsPerBlock = kThreads / 64;
constexpr int kRowVecs = 8;   // 4-element vectors per lane in flight

template <int VEC, typename GT>
__global__ __launch_bounds__(kThreads) void momentum_rows(MatSet ms, int64_t rows, int64_t cols,
                                                          double* __restrict__ l1,
                                                          double* __restrict__ sq) {
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;   // whole wave
    float* __restrict__ M = ms.m(b) + row * cols;
    const GT* __restrict__ G = ms.g<GT>(b) + row * cols;
    // four independent accumulators (element v of each vector goes to set v)
    // keep the fp64 dependency chains short; they are folded in a fixed order
    double h4[4] = {0.0, 0.0, 0.0, 0.0}, l4[4] = {0.0, 0.0, 0.0, 0.0}, q4[4] = {0.0, 0.0, 0.0, 0.0};
    if constexpr (VEC == 4) {
        constexpr int kStep = 64 * 4 * kRowVecs;
        int64_t c = 0;
        for (; c + kStep <= cols; c += kStep) {
            float m[kRowVecs][4], g[kRowVecs][4];
#pragma unroll
            for (int u = 0; u < kRowVecs; ++u) {
                unpack4(ldg_nt<float4>(M + c + (u * 64 + lane) * 4), m[u]);
                unpack4(ldg_nt<typename std::conditional<sizeof(GT) == 2, uint2, float4>::type>(
                            G + c + (u * 64 + lane) * 4), g[u]);
            }
#pragma unroll
            for (int u = 0; u < kRowVecs; ++u) {
#pragma unroll
                for (int v = 0; v < 4; ++v) m[u][v] = m[u][v] + g[u][v];
                stg_nt(M + c + (u * 64 + lane) * 4, make_float4(m[u][0], m[u][1], m[u][2], m[u][3]));
#pragma unroll
                for (int v = 0; v < 4; ++v) accumulate(fabs((double)m[u][v]), h4[v], l4[v], q4[v]);
            }
        }
        for (int64_t cc = c + lane * 4; cc < cols; cc += 64 * 4) {
            float m[4], g[4];
            load4(M + cc, m);
            load4(G + cc, g);
#pragma unroll
            for (int v = 0; v < 4; ++v) m[v] = m[v] + g[v];
            stg(M + cc, make_float4(m[0], m[1], m[2], m[3]));
#pragma unroll
            for (int v = 0; v < 4; ++v) accumulate(fabs((double)m[v]), h4[v], l4[v], q4[v]);
        }
    } else {
        for (int64_t c = lane; c < cols; c += 64) {
            const float m = ldg<float>(M + c) + Elem<GT>::load(G + c);
            stg(M + c, m);
            accumulate(fabs((double)m), h4[0], l4[0], q4[0]);
        }
    }
    double hi = h4[0], lo = l4[0], s2 = q4[0];
#pragma unroll
    for (int v = 1; v < 4; ++v) {
        dd_add(hi, lo, h4[v], l4[v]);
        s2 += q4[v];
    }
    wave_reduce(hi, lo, s2);
    if (lane == 0) {
        l1[(int64_t)b * rows + row] = hi + lo;
        sq[(int64_t)b * rows + row] = s2;
    }
}

template <int VEC, typename GT>
__global__ __launch_bounds__(kThreads) void momentum_cols_partial(MatSet ms, int64_t rows,
                                                                  int64_t cols, int rb_rows,
                                                                  int nrb,
                                                                  double* __restrict__ part) {
    const int b = blockIdx.z;
    const int rb = blockIdx.y;
    const int64_t c0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC;
    if (c0 >= cols) return;
    const int64_t r0 = (int64_t)rb * rb_rows;
    const int64_t r1 = r0 + rb_rows < rows ? r0 + rb_rows : rows;
    const float* __restrict__ M = ms.m(b);
    const GT* __restrict__ G = ms.g<GT>(b);
    double hi[VEC], lo[VEC], s2[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) hi[v] = lo[v] = s2[v] = 0.0;
#pragma unroll 4
    for (int64_t r = r0; r < r1; ++r) {
        const float* p = M + r * cols + c0;
        const GT* q = G + r * cols + c0;
        if constexpr (VEC == 4) {
            float m[4], g[4];
            unpack4(ldg_nt<float4>(p), m);
            unpack4(ldg_nt<typename std::conditional<sizeof(GT) == 2, uint2, float4>::type>(q), g);
#pragma unroll
            for (int v = 0; v < 4; ++v) m[v] = m[v] + g[v];
#pragma unroll
            for (int v = 0; v < VEC; ++v) accumulate(fabs((double)m[v]), hi[v], lo[v], s2[v]);
        } else {
            const float m = ldg<float>(p) + Elem<GT>::load(q);
            accumulate(fabs((double)m), hi[0], lo[0], s2[0]);
        }
    }
    double* out = part + ((int64_t)b * nrb + rb) * 3 * cols;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        out[c0 + v] = hi[v];
        out[cols + c0 + v] = lo[v];
        out[2 * cols + c0 + v] = s2[v];
    }
}

__global__ __launch_bounds__(kThreads) void momentum_cols_final(const double* __restrict__ part,
                                                                int nrb, int64_t cols,
                                                                double* __restrict__ l1,
                                                                double* __restrict__ sq) {
    const int b = blockIdx.y;
    const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (c >= cols) return;
    double hi = 0.0, lo = 0.0, s2 = 0.0;
    for (int rb = 0; rb < nrb; ++rb) {
        const double* p = part + ((int64_t)b * nrb + rb) * 3 * cols;
        dd_add(hi, lo, p[c], p[cols + c]);
        s2 += p[2 * cols + c];
    }
    l1[(int64_t)b * cols + c] = hi + lo;
    sq[(int64_t)b * cols + c] = s2;
}

template <int VEC, typename GT>
hipError_t launch_typed(const MomentumArgs& a, int axis, hipStream_t s) {
    if (axis == 0) {
        dim3 grid((unsigned)((a.rows + kRowsPerBlock - 1) / kRowsPerBlock), (unsigned)a.batch);
        hipLaunchKernelGGL((momentum_rows<VEC, GT>), grid, dim3(kThreads), 0, s, a.ms, a.rows,
                           a.cols, a.l1, a.sq);
    } else {
        // Blocks of four waves where they tile the row exactly, else of one
        // wave, so a row that is not a multiple of 256 * VEC columns wide
        // leaves at most part of one wave idle (1408 columns: 8% of the
        // lanes instead of 31%). Each column's rows are summed in the same
        // order either way.
        const int threads = a.cols % ((int64_t)kThreads * VEC) == 0 ? kThreads : 64;
        const int64_t per_block = (int64_t)threads * VEC;
        dim3 grid((unsigned)((a.cols + per_block - 1) / per_block), (unsigned)a.nrb,
                  (unsigned)a.batch);
        hipLaunchKernelGGL((momentum_cols_partial<VEC, GT>), grid, dim3(threads), 0, s, a.ms,
                           a.rows, a.cols, a.rb_rows, a.nrb, a.part);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        dim3 grid2((unsigned)((a.cols + kThreads - 1) / kThreads), (unsigned)a.batch);
        hipLaunchKernelGGL(momentum_cols_final, grid2, dim3(kThreads), 0, s, a.part, a.nrb,
                           a.cols, a.l1, a.sq);
    }
    return hipGetLastError();
}

}  // namespace

// Row blocking of the column-mode reduction: blocks of 256 rows keep the
// partials small next to the matrix while giving enough blocks to fill the
// chip.
int64_t momentum_col_blocks(int64_t rows, int* rb_rows) {
    const int rb = 256;
    *rb_rows = rb;
    return (rows + rb - 1) / rb;
}

hipError_t launch_momentum(const MomentumArgs& a, int axis, int g_bf16, hipStream_t s) {
    const bool vec = (a.cols % 4) == 0;
    if (g_bf16) {
        return vec ? launch_typed<4, uint16_t>(a, axis, s) : launch_typed<1, uint16_t>(a, axis, s);
    }
    return vec ? launch_typed<4, float>(a, axis, s) : launch_typed<1, float>(a, axis, s);
}

}  // namespace dion2
