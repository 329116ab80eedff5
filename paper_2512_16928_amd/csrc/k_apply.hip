// K5: the sparse weight update step of Algorithm 1 with the scale of
// eq. (1):
//   W_line(K[p])[j] <- round_W( W_line(K[p])[j] - lr*sqrt(rows/cols) * O[p][j] )
// O is the fp32 Newton-Schulz output in the compact L layout [kpad][opad].
// The product and the difference are taken in fp64 (one rounding each, no
// contraction) and the result is rounded once, to nearest even, to W's
// storage type; lines outside K are never touched. Optionally O itself is
// copied out unpadded for inspection.
//
// Row mode reads O rows and W rows along j (both contiguous). Column mode
// streams W by rows and reads O transposed.
#include <type_traits>

#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kThreads = 256;

template <typename WT>
__device__ __forceinline__ void update(WT* w, float o, double lr_eff) {
    const double x = (double)Elem<WT>::load(w);
    const double r = __dsub_rn(x, __dmul_rn(lr_eff, (double)o));
    Elem<WT>::store_f64(w, r);
}

// four consecutive elements of W: load as fp32, store rounded from fp64
__device__ __forceinline__ void load4w(const float* p, float (&v)[4]) { load4(p, v); }
__device__ __forceinline__ void load4w(const uint16_t* p, float (&v)[4]) { load4(p, v); }
__device__ __forceinline__ void store4w(float* p, const double (&r)[4]) {
    stg(p, make_float4((float)r[0], (float)r[1], (float)r[2], (float)r[3]));
}
__device__ __forceinline__ void store4w(uint16_t* p, const double (&r)[4]) {
    uint2 u;
    u.x = (uint32_t)f64_to_bf16(r[0]) | ((uint32_t)f64_to_bf16(r[1]) << 16);
    u.y = (uint32_t)f64_to_bf16(r[2]) | ((uint32_t)f64_to_bf16(r[3]) << 16);
    stg(p, u);
}

// Row mode: one wave per selected line p, four elements per lane.
template <int VEC, typename WT>
__global__ __launch_bounds__(kThreads) void apply_rows(ApplyArgs a) {
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int p = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (p >= a.k) return;   // whole wave
    WT* __restrict__ w = a.ms.w<WT>(b) + (int64_t)a.sel[(int64_t)b * a.k + p] * a.cols;
    const float* __restrict__ o = a.O + (int64_t)b * a.kpad * a.opad + (int64_t)p * a.opad;
    float* dbg = a.dbg ? a.dbg + ((int64_t)b * a.k + p) * a.d_oth : nullptr;
    if constexpr (VEC == 4) {
        for (int j = 4 * lane; j < a.d_oth; j += 256) {
            float x[4], u[4];
            load4w(w + j, x);
            load4(o + j, u);
            double r[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) r[v] = __dsub_rn((double)x[v], __dmul_rn(a.lr_eff, (double)u[v]));
            store4w(w + j, r);
            if (dbg) *reinterpret_cast<float4*>(dbg + j) = make_float4(u[0], u[1], u[2], u[3]);
        }
    } else {
        for (int j = lane; j < a.d_oth; j += 64) {
            update(w + j, o[j], a.lr_eff);
            if (dbg) dbg[j] = o[j];
        }
    }
}

// Column mode: the selected columns are spread through every row of W, so
// W is streamed row by row. O comes in the L^T layout [opad][kpad], so the
// values a row needs, O^T[r][rank[c]] for its selected columns c, sit
// together in one row of O^T. A block covers kCW columns x kRB rows; each
// lane owns four columns of kRB / 4 rows and issues all its loads before
// any store. Every four-column group is written back, unselected entries
// with their own bits, so each cache line of W is rewritten whole.
constexpr int kCW = 256;
constexpr int kRB = 64;

template <int VEC, typename WT>
__global__ __launch_bounds__(kThreads) void apply_cols(ApplyArgs a) {
    const int b = blockIdx.z;
    const int64_t c0 = (int64_t)blockIdx.x * kCW;
    const int r0 = blockIdx.y * kRB;
    const int32_t* __restrict__ rank = a.rank + (int64_t)b * (a.cols + 1);
    WT* __restrict__ W = a.ms.w<WT>(b);
    const float* __restrict__ OT = a.O + (int64_t)b * a.opad * a.kpad;
    const int cq = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int64_t c = c0 + 4 * cq;
    int p[4];   // line of each column, -1 if unselected
    {
        int rk[5];   // rank[c .. c + 4], clamped to the array (branch-free loads)
#pragma unroll
        for (int v = 0; v < 5; ++v) rk[v] = ldg<int32_t>(rank + (c + v < a.cols ? c + v : a.cols));
#pragma unroll
        for (int v = 0; v < 4; ++v) p[v] = (c + v < a.cols && rk[v + 1] > rk[v]) ? rk[v] : -1;
    }
    constexpr int kR = kRB / 4;   // rows per thread
    if (VEC == 4 && c + 3 < a.cols) {
        typedef typename std::conditional<sizeof(WT) == 2, uint2, float4>::type Raw;
        Raw raw[kR];
        float o[kR][4];
        // branch-free loads so all of them are in flight together: an
        // unselected column reads the block's first line (a word of the same
        // row segment, so no extra cache line; unused), rows past the matrix
        // read its last row
        const int pfirst = ldg<int32_t>(rank + c0);
        int pc[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) pc[v] = p[v] >= 0 ? p[v] : pfirst;
#pragma unroll
        for (int i = 0; i < kR; ++i) {
            int64_t r = r0 + rg + 4 * i;
            r = r < a.rows ? r : a.rows - 1;
            raw[i] = ldg_nt<Raw>(W + r * a.cols + c);
#pragma unroll
            for (int v = 0; v < 4; ++v) o[i][v] = OT[r * a.kpad + pc[v]];
        }
#pragma unroll
        for (int i = 0; i < kR; ++i) {
            const int64_t r = r0 + rg + 4 * i;
            if (r >= a.rows) continue;
            // unselected entries are written back with their own bits
            if constexpr (sizeof(WT) == 2) {
                const uint2 x = reinterpret_cast<const uint2&>(raw[i]);
                uint32_t h[4] = {x.x & 0xffffu, x.x >> 16, x.y & 0xffffu, x.y >> 16};
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (p[v] >= 0)
                        h[v] = f64_to_bf16(__dsub_rn((double)bf16_bits_to_f32(h[v]),
                                                     __dmul_rn(a.lr_eff, (double)o[i][v])));
                stg_nt(W + r * a.cols + c, make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16)));
            } else {
                float4 x = reinterpret_cast<const float4&>(raw[i]);
                float f[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (p[v] >= 0) f[v] = (float)__dsub_rn((double)f[v], __dmul_rn(a.lr_eff, (double)o[i][v]));
                stg_nt(W + r * a.cols + c, make_float4(f[0], f[1], f[2], f[3]));
            }
        }
    } else {
        for (int rl = rg; rl < kRB; rl += 4) {
            const int64_t r = r0 + rl;
            if (r >= a.rows) break;
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (p[v] >= 0) update(W + r * a.cols + c + v, OT[r * a.kpad + p[v]], a.lr_eff);
        }
    }
    if (a.dbg) {   // O in the [k][d_oth] layout (inspection only)
        for (int rl = rg; rl < kRB; rl += 4) {
            const int64_t r = r0 + rl;
            if (r >= a.rows) break;
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (p[v] >= 0) a.dbg[((int64_t)b * a.k + p[v]) * a.d_oth + r] = OT[r * a.kpad + p[v]];
        }
    }
}

}  // namespace

hipError_t launch_apply(const ApplyArgs& a, int axis, int w_bf16, hipStream_t s) {
    const bool vec = a.cols % 4 == 0;
    if (axis == 0) {
        dim3 grid((unsigned)((a.k + 3) / 4), (unsigned)a.batch);
        if (w_bf16) {
            if (vec) hipLaunchKernelGGL((apply_rows<4, uint16_t>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((apply_rows<1, uint16_t>), grid, dim3(kThreads), 0, s, a);
        } else {
            if (vec) hipLaunchKernelGGL((apply_rows<4, float>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((apply_rows<1, float>), grid, dim3(kThreads), 0, s, a);
        }
    } else {
        dim3 grid((unsigned)((a.cols + kCW - 1) / kCW), (unsigned)((a.rows + kRB - 1) / kRB),
                  (unsigned)a.batch);
        if (w_bf16) {
            if (vec) hipLaunchKernelGGL((apply_cols<4, uint16_t>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((apply_cols<1, uint16_t>), grid, dim3(kThreads), 0, s, a);
        } else {
            if (vec) hipLaunchKernelGGL((apply_cols<4, float>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((apply_cols<1, float>), grid, dim3(kThreads), 0, s, a);
        }
    }
    return hipGetLastError();
}

}  // namespace dion2
