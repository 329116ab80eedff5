// K3: gather the selected lines into the compact bf16 submatrix, scaled for
// Newton-Schulz, fused with the selective decay of eq. (2).
//
//   L[p][j]  = bf16(M_line(K[p])[j] / (||M[K]||_F + eps))   [kpad][opad]
//   LT[j][p] = L[p][j]                                       [opad][kpad]
//   M_line(K[p]) <- fl32(mu * M_line(K[p]))                   (Algorithm 1, decay step)
//
// Only the orientation Newton-Schulz iterates on is written (the wide one;
// the other pointer is null). One 256-thread block handles a 64 x 64 tile of
// (line p, other index j): the side that is contiguous in M is read and
// written directly, the other side goes through an LDS tile. Tiles cover the
// padded extents, and padding (p >= k or j >= d_oth) is written as zero.
#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kT = 64;   // tile edge
constexpr int kThreads = 256;

// Row mode: line p is row K[p] of M; j runs along the row (contiguous).
template <int VEC>
__global__ __launch_bounds__(kThreads) void gather_rows(GatherArgs a) {
    __shared__ float tile[kT][kT + 1];
    const int b = blockIdx.z;
    const int p0 = blockIdx.y * kT, j0 = blockIdx.x * kT;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float* __restrict__ M = a.ms.m(b);
    const int32_t* __restrict__ K = a.sel + (int64_t)b * a.k;
    const float sc = (float)a.scale[b];
    uint16_t* __restrict__ L = a.L ? a.L + (int64_t)b * a.kpad * a.opad : nullptr;
    uint16_t* __restrict__ LT = a.LT ? a.LT + (int64_t)b * a.opad * a.kpad : nullptr;
    float* __restrict__ O = a.O ? a.O + (int64_t)b * a.kpad * a.opad : nullptr;
    const int j = j0 + 4 * tx;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pl = ty + 16 * i;
        const int p = p0 + pl;
        float x[4] = {0.f, 0.f, 0.f, 0.f};
        if (p < a.k) {
            float* row = M + (int64_t)K[p] * a.cols;
            if (VEC == 4 && j + 3 < a.d_oth) {
                float m[4];
                load4(row + j, m);
#pragma unroll
                for (int v = 0; v < 4; ++v) x[v] = m[v] * sc;
                if (a.decay) {
                    *reinterpret_cast<float4*>(row + j) =
                        make_float4(a.mu * m[0], a.mu * m[1], a.mu * m[2], a.mu * m[3]);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    if (j + v < a.d_oth) {
                        const float m = row[j + v];
                        x[v] = m * sc;
                        if (a.decay) row[j + v] = a.mu * m;
                    }
                }
            }
        }
        if (L) {
            uint2 packed;
            packed.x = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
            packed.y = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
            *reinterpret_cast<uint2*>(L + (int64_t)p * a.opad + j) = packed;
        }
        if (O) *reinterpret_cast<float4*>(O + (int64_t)p * a.opad + j) = make_float4(x[0], x[1], x[2], x[3]);
#pragma unroll
        for (int v = 0; v < 4; ++v) tile[pl][4 * tx + v] = x[v];
    }
    if (!LT) return;   // uniform over the block
    __syncthreads();
    // transposed: LT[j][p], p contiguous
    const int p = p0 + 4 * tx;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int jl = ty + 16 * i;
        uint2 packed;
        packed.x = (uint32_t)f32_to_bf16(tile[4 * tx + 0][jl]) |
                   ((uint32_t)f32_to_bf16(tile[4 * tx + 1][jl]) << 16);
        packed.y = (uint32_t)f32_to_bf16(tile[4 * tx + 2][jl]) |
                   ((uint32_t)f32_to_bf16(tile[4 * tx + 3][jl]) << 16);
        *reinterpret_cast<uint2*>(LT + (int64_t)(j0 + jl) * a.kpad + p) = packed;
    }
}

// Column mode: line p is column K[p] of M; the other index r is the row.
// Reading along a row picks K[p], K[p+1], ... (ascending, nearby columns).
__global__ __launch_bounds__(kThreads) void gather_cols(GatherArgs a) {
    __shared__ float tile[kT][kT + 1];   // [p local][r local]
    const int b = blockIdx.z;
    const int p0 = blockIdx.y * kT, r0 = blockIdx.x * kT;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float* __restrict__ M = a.ms.m(b);
    const int32_t* __restrict__ K = a.sel + (int64_t)b * a.k;
    const float sc = (float)a.scale[b];
    uint16_t* __restrict__ L = a.L ? a.L + (int64_t)b * a.kpad * a.opad : nullptr;
    uint16_t* __restrict__ LT = a.LT ? a.LT + (int64_t)b * a.opad * a.kpad : nullptr;
    float* __restrict__ O = a.O ? a.O + (int64_t)b * a.kpad * a.opad : nullptr;
    const int p = p0 + 4 * tx;
    int col[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) col[v] = (p + v < a.k) ? K[p + v] : -1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rl = ty + 16 * i;
        const int r = r0 + rl;
        float x[4] = {0.f, 0.f, 0.f, 0.f};
        if (r < a.d_oth) {
            float* row = M + (int64_t)r * a.cols;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                if (col[v] >= 0) {
                    const float m = row[col[v]];
                    x[v] = m * sc;
                    if (a.decay) row[col[v]] = a.mu * m;
                }
            }
        }
        if (LT) {
            uint2 packed;
            packed.x = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
            packed.y = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
            *reinterpret_cast<uint2*>(LT + (int64_t)r * a.kpad + p) = packed;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) tile[4 * tx + v][rl] = x[v];
    }
    if (!L && !O) return;   // uniform over the block
    __syncthreads();
    // L[p][r], r contiguous
    const int r = r0 + 4 * tx;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pl = ty + 16 * i;
        float x[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) x[v] = tile[pl][4 * tx + v];
        if (L) {
            uint2 packed;
            packed.x = (uint32_t)f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
            packed.y = (uint32_t)f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
            *reinterpret_cast<uint2*>(L + (int64_t)(p0 + pl) * a.opad + r) = packed;
        }
        if (O) *reinterpret_cast<float4*>(O + (int64_t)(p0 + pl) * a.opad + r) = make_float4(x[0], x[1], x[2], x[3]);
    }
}

__global__ __launch_bounds__(kThreads) void decay_all(DecayAllArgs a) {
    const int b = blockIdx.y;
    float* __restrict__ M = a.ms.m(b);
    const int64_t n = a.rows * a.cols;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads) {
        M[i] = a.mu * M[i];
    }
}

}  // namespace

hipError_t launch_gather(const GatherArgs& a, int axis, hipStream_t s) {
    dim3 grid((unsigned)(a.opad / kT), (unsigned)(a.kpad / kT), (unsigned)a.batch);
    if (axis == 0) {
        if (a.cols % 4 == 0) {
            hipLaunchKernelGGL((gather_rows<4>), grid, dim3(kThreads), 0, s, a);
        } else {
            hipLaunchKernelGGL((gather_rows<1>), grid, dim3(kThreads), 0, s, a);
        }
    } else {
        hipLaunchKernelGGL(gather_cols, grid, dim3(kThreads), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_decay_all(const DecayAllArgs& a, hipStream_t s) {
    const int64_t n = a.rows * a.cols;
    int64_t blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(decay_all, dim3((unsigned)blocks, (unsigned)a.batch), dim3(kThreads), 0, s,
                       a);
    return hipGetLastError();
}

}  // namespace dion2
