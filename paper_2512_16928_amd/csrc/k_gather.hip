// K3: gather the selected lines into the compact bf16 submatrix, scaled for
// Newton-Schulz, fused with the selective decay of eq. (2) (and, in column
// mode, with the store of the accumulated momentum).
//
//   L[p][j]  = bf16(M_line(K[p])[j] / (||M[K]||_F + eps))   [kpad][opad]
//   LT[j][p] = L[p][j]                                       [opad][kpad]
//   M_line(K[p]) <- fl32(mu * M_line(K[p]))                   (Algorithm 1, decay step)
//
// Only the orientation Newton-Schulz iterates on is written (the wide one;
// the other pointer is null). For the fp32-master Newton-Schulz the lo
// halves bf16(x - bf16(x)) go out beside it (Llo / LTlo). One 256-thread block handles a 64 x 64 tile of
// (line p, other index j): the side that is contiguous in M is read and
// written directly, the other side goes through an LDS tile. Tiles cover the
// padded extents, and padding (p >= k or j >= d_oth) is written as zero.
#include <type_traits>

#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kT = 64;   // tile edge
constexpr int kThreads = 256;

// Four values as packed bf16 his, and their lo halves bf16(x - hi).
__device__ __forceinline__ void pack_hilo4(const float (&x)[4], uint2* hi, uint2* lo) {
    uint16_t h[4], l[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        h[v] = f32_to_bf16(x[v]);
        l[v] = f32_to_bf16(x[v] - bf16_bits_to_f32(h[v]));
    }
    hi->x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
    hi->y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
    lo->x = (uint32_t)l[0] | ((uint32_t)l[1] << 16);
    lo->y = (uint32_t)l[2] | ((uint32_t)l[3] << 16);
}

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
    // the four rows' indices and values are all requested before the first
    // store: memory counters retire in issue order, so a load issued after a
    // store would also wait for the store's acknowledgement
    int64_t roff[4];
    float4 mv[4];
    const bool vec = VEC == 4 && j + 3 < a.d_oth;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int p = p0 + ty + 16 * i;
        roff[i] = (int64_t)ldg<int32_t>(K + (p < a.k ? p : a.k - 1)) * a.cols;
    }
    if (vec) {
#pragma unroll
        for (int i = 0; i < 4; ++i) mv[i] = ldg_nt<float4>(M + roff[i] + j);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int pl = ty + 16 * i;
        const int p = p0 + pl;
        float x[4] = {0.f, 0.f, 0.f, 0.f};
        if (p < a.k) {
            float* row = M + roff[i];
            if (vec) {
                float m[4];
                unpack4(mv[i], m);
#pragma unroll
                for (int v = 0; v < 4; ++v) x[v] = m[v] * sc;
                if (a.decay) stg_nt(row + j, make_float4(a.mu * m[0], a.mu * m[1], a.mu * m[2], a.mu * m[3]));
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    if (j + v < a.d_oth) {
                        const float m = ldg<float>(row + j + v);
                        x[v] = m * sc;
                        if (a.decay) stg(row + j + v, a.mu * m);
                    }
                }
            }
        }
        if (L) {
            uint2 hi, lo;
            pack_hilo4(x, &hi, &lo);
            *reinterpret_cast<uint2*>(L + (int64_t)p * a.opad + j) = hi;
            if (a.Llo) *reinterpret_cast<uint2*>(a.Llo + (int64_t)b * a.kpad * a.opad + (int64_t)p * a.opad + j) = lo;
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
        const float x[4] = {tile[4 * tx + 0][jl], tile[4 * tx + 1][jl], tile[4 * tx + 2][jl],
                            tile[4 * tx + 3][jl]};
        uint2 hi, lo;
        pack_hilo4(x, &hi, &lo);
        *reinterpret_cast<uint2*>(LT + (int64_t)(j0 + jl) * a.kpad + p) = hi;
        if (a.LTlo)
            *reinterpret_cast<uint2*>(a.LTlo + (int64_t)b * a.opad * a.kpad + (int64_t)(j0 + jl) * a.kpad + p) = lo;
    }
}

// Column mode: line p is column K[p] of M; the other index r is the row.
// Selected columns are scattered through every row, so decaying them in
// place would dirty every cache line of M anyway; instead this pass streams
// whole rows once: M <- fl32(M + G) (the momentum pass only read M to get
// the column norms), times mu on the selected columns (every column with
// decay == 2), and the selected columns, scaled, go through an LDS tile
// into the compact matrix. A block covers kCW columns x kRB rows; rank[c]
// (selected columns below c) gives each selected column its line p, and
// the block's lines are p0 = rank[c0] .. p1 = rank[c0 + kCW].
constexpr int kCW = 256;
constexpr int kRB = 64;

template <int VEC, typename GT>
__global__ __launch_bounds__(kThreads) void update_cols(GatherArgs a) {
    __shared__ float tile[kCW][kRB + 1];   // [p - p0][r - r0]
    const int b = blockIdx.z;
    const int64_t c0 = (int64_t)blockIdx.x * kCW;
    const int r0 = blockIdx.y * kRB;
    const int64_t cend = c0 + kCW < a.cols ? c0 + kCW : a.cols;
    const int32_t* __restrict__ rank = a.rank + (int64_t)b * (a.cols + 1);
    const int p0 = rank[c0], p1 = rank[cend];
    float* __restrict__ M = a.ms.m(b);
    const GT* __restrict__ G = a.ms.g<GT>(b);
    // the single pass (sq_part) copies the columns unscaled: their norm is
    // known only once every row has been read
    const float sc = a.sq_part ? 1.0f : (float)a.scale[b];
    const int cq = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int64_t c = c0 + 4 * cq;
    int pl[4];        // tile row of each of the four columns, -1 if unselected
    bool in[4];
    {
        int rk[5];   // rank[c .. c + 4], clamped to the array (branch-free loads)
#pragma unroll
        for (int v = 0; v < 5; ++v) rk[v] = ldg<int32_t>(rank + (c + v < a.cols ? c + v : a.cols));
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            in[v] = c + v < a.cols;
            pl[v] = (in[v] && rk[v + 1] > rk[v]) ? rk[v] - p0 : -1;
        }
    }
    constexpr int kR = kRB / 4;   // rows per thread
    if (VEC == 4 && in[3]) {
        // every row's M and G are loaded before the first store
        typedef typename std::conditional<sizeof(GT) == 2, uint2, float4>::type GRaw;
        float4 mr[kR];
        GRaw gr[kR];
#pragma unroll
        for (int i = 0; i < kR; ++i) {
            const int64_t r = r0 + rg + 4 * i;
            if (r < a.rows) {
                mr[i] = ldg_nt<float4>(M + r * a.cols + c);
                gr[i] = ldg_nt<GRaw>(G + r * a.cols + c);
            }
        }
#pragma unroll
        for (int i = 0; i < kR; ++i) {
            const int rl = rg + 4 * i;
            const int64_t r = r0 + rl;
            float m[4] = {0.f, 0.f, 0.f, 0.f};
            if (r < a.rows) {
                float g[4];
                unpack4(gr[i], g);
                m[0] = mr[i].x + g[0];
                m[1] = mr[i].y + g[1];
                m[2] = mr[i].z + g[2];
                m[3] = mr[i].w + g[3];
                float o[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    o[v] = (a.decay == 2 || (a.decay == 1 && pl[v] >= 0)) ? a.mu * m[v] : m[v];
                stg_nt(M + r * a.cols + c, make_float4(o[0], o[1], o[2], o[3]));
            }
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (pl[v] >= 0) tile[pl[v]][rl] = m[v] * sc;   // rows past d_oth give zeros
        }
    } else {
        for (int i = 0; i < kR; ++i) {
            const int rl = rg + 4 * i;
            const int64_t r = r0 + rl;
            float m[4] = {0.f, 0.f, 0.f, 0.f};
            if (r < a.rows) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    if (in[v]) {
                        m[v] = ldg<float>(M + r * a.cols + c + v) + Elem<GT>::load(G + r * a.cols + c + v);
                        stg(M + r * a.cols + c + v,
                            (a.decay == 2 || (a.decay == 1 && pl[v] >= 0)) ? a.mu * m[v] : m[v]);
                    }
                }
            }
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (pl[v] >= 0) tile[pl[v]][rl] = m[v] * sc;
        }
    }
    __syncthreads();
    const int np = p1 - p0;
    const bool last = cend == a.cols;   // this chunk also zeroes the padded lines k..kpad
    if (a.sq_part) {
        // sum of squares of this block's 64 rows of each selected column, in row order
        double* sp = a.sq_part + ((int64_t)b * (a.opad / kRB) + blockIdx.y) * a.kpad + p0;
        for (int pi = threadIdx.x; pi < np; pi += kThreads) {
            double q = 0.0;
            for (int rl = 0; rl < kRB; ++rl) {
                const double x = (double)tile[pi][rl];
                q += x * x;
            }
            sp[pi] = q;
        }
    }
    if (a.L) {
        // L[p][r0 .. r0 + 64), four rows per thread
        const int q = threadIdx.x & 15;
        for (int pi = threadIdx.x >> 4; pi < np; pi += kThreads / 16) {
            float x[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) x[v] = tile[pi][4 * q + v];
            const int64_t off = (int64_t)b * a.kpad * a.opad + (int64_t)(p0 + pi) * a.opad + r0 + 4 * q;
            uint2 hi, lo;
            pack_hilo4(x, &hi, &lo);
            *reinterpret_cast<uint2*>(a.L + off) = hi;
            if (a.Llo) *reinterpret_cast<uint2*>(a.Llo + off) = lo;
        }
        if (last) {
            for (int pi = a.k + (threadIdx.x >> 4); pi < a.kpad; pi += kThreads / 16) {
                const int64_t off = (int64_t)b * a.kpad * a.opad + (int64_t)pi * a.opad + r0 + 4 * q;
                *reinterpret_cast<uint2*>(a.L + off) = make_uint2(0u, 0u);
                if (a.Llo) *reinterpret_cast<uint2*>(a.Llo + off) = make_uint2(0u, 0u);
            }
        }
    }
    if (a.O) {
        // fp32 O^T[r][p0 .. p1), p contiguous (the layout the apply pass reads)
        float* O = a.O + (int64_t)b * a.opad * a.kpad;
        for (int idx = threadIdx.x; idx < kRB * np; idx += kThreads) {
            const int rl = idx / np, pi = idx % np;
            O[(int64_t)(r0 + rl) * a.kpad + p0 + pi] = tile[pi][rl];
        }
    }
    if (a.LT) {
        // L^T[r][p0 .. p1), p contiguous
        uint16_t* LT = a.LT + (int64_t)b * a.opad * a.kpad;
        uint16_t* LTlo = a.LTlo ? a.LTlo + (int64_t)b * a.opad * a.kpad : nullptr;
        for (int idx = threadIdx.x; idx < kRB * np; idx += kThreads) {
            const int rl = idx / np, pi = idx % np;
            const float x = tile[pi][rl];
            const uint16_t h = f32_to_bf16(x);
            LT[(int64_t)(r0 + rl) * a.kpad + p0 + pi] = h;
            if (LTlo) LTlo[(int64_t)(r0 + rl) * a.kpad + p0 + pi] = f32_to_bf16(x - bf16_bits_to_f32(h));
        }
        if (last) {
            const int npad = a.kpad - a.k;
            for (int idx = threadIdx.x; idx < kRB * npad; idx += kThreads) {
                const int rl = idx / npad, pi = idx % npad;
                LT[(int64_t)(r0 + rl) * a.kpad + a.k + pi] = 0;
                if (LTlo) LTlo[(int64_t)(r0 + rl) * a.kpad + a.k + pi] = 0;
            }
        }
    }
}

__global__ __launch_bounds__(kThreads) void decay_all(DecayAllArgs a) {
    const int b = blockIdx.y;
    float* __restrict__ M = a.ms.m(b);
    const int64_t n = a.rows * a.cols;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads) {
        stg(M + i, a.mu * ldg<float>(M + i));
    }
}

__global__ __launch_bounds__(kThreads) void copy_compact(CompactCopyArgs a) {
    const int b = blockIdx.y;
    const int64_t n = (int64_t)a.k * a.d_oth;
    const uint16_t* __restrict__ Z = a.Z + (int64_t)b * a.kpad * a.opad;
    uint16_t* __restrict__ out = a.out + (int64_t)b * n;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads) {
        const int64_t p = i / a.d_oth, j = i % a.d_oth;
        out[i] = a.transposed ? Z[j * a.kpad + p] : Z[p * a.opad + j];
    }
}

}  // namespace

hipError_t launch_copy_compact(const CompactCopyArgs& a, hipStream_t s) {
    const int64_t n = (int64_t)a.k * a.d_oth;
    int64_t blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(copy_compact, dim3((unsigned)blocks, (unsigned)a.batch), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

// ---- the end of the single column pass (see ColpassArgs)

namespace {

// Sums of squares of the selected columns from update_cols' partials
// sq_part[b][rb][p] (rb = 64-row block), in a fixed order. Level 1: a block
// takes 64 lines and up to 256 row blocks (four quarters, one per group of 64
// threads, each summed in row order with its loads issued ahead), folds the
// quarters in order and writes the result in place of the chunk's first row
// block.
constexpr int kChunk = 256;   // row blocks folded by one level-1 block

__global__ __launch_bounds__(kThreads) void colpass_fold(ColpassArgs a) {
    __shared__ double part[4][64];
    const int b = blockIdx.z;
    const int nrb = a.opad / kRB;
    const int p = blockIdx.x * 64 + (threadIdx.x & 63);
    const int quarter = threadIdx.x >> 6;
    const int rb0 = blockIdx.y * kChunk;
    const int rb1 = rb0 + kChunk < nrb ? rb0 + kChunk : nrb;
    const int per = (rb1 - rb0 + 3) / 4;
    const int q0 = rb0 + quarter * per;
    const int q1 = q0 + per < rb1 ? q0 + per : rb1;
    double* sp = a.sq_part + (int64_t)b * nrb * a.kpad;
    double q = 0.0;
    if (p < a.k) {
        int rb = q0;
        for (; rb + 8 <= q1; rb += 8) {
            double v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = sp[(int64_t)(rb + u) * a.kpad + p];
#pragma unroll
            for (int u = 0; u < 8; ++u) q += v[u];
        }
        for (; rb < q1; ++rb) q += sp[(int64_t)rb * a.kpad + p];
    }
    part[quarter][threadIdx.x & 63] = q;
    __syncthreads();
    if (quarter == 0 && p < a.k) {
        const int l = threadIdx.x;
        sp[(int64_t)rb0 * a.kpad + p] = ((part[0][l] + part[1][l]) + part[2][l]) + part[3][l];
    }
}

// Level 2, one block per matrix: each line's chunks in order, the lines in a
// fixed order, then scale = 1 / (sqrt(sum) + eps).
__global__ __launch_bounds__(kThreads) void colpass_scale(ColpassArgs a) {
    const int b = blockIdx.x;
    const int nrb = a.opad / kRB;
    const double* sp = a.sq_part + (int64_t)b * nrb * a.kpad;
    double f = 0.0;
    for (int p = threadIdx.x; p < a.k; p += kThreads) {
        double q = 0.0;
        for (int rb0 = 0; rb0 < nrb; rb0 += kChunk) q += sp[(int64_t)rb0 * a.kpad + p];
        f += q;
    }
    __shared__ double red[kThreads / 64];
    for (int off = 32; off > 0; off >>= 1) f += __shfl_xor(f, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = f;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) t += red[w];
        const double d = sqrt(t) + a.eps;   // zero X with eps = 0: scale 0, X stays 0
        a.scale[b] = d > 0.0 ? 1.0 / d : 0.0;
    }
}

// 64 rows x 64 lines per block through an LDS tile; every store writes eight
// consecutive bf16 (16 bytes).
__global__ __launch_bounds__(kThreads) void colpass_compact(ColpassArgs a) {
    __shared__ float t[64][65];
    const int b = blockIdx.z;
    const int r0 = blockIdx.y * 64, p0 = blockIdx.x * 64;
    const float sc = (float)a.scale[b];
    const float* Ot = a.Ot + (int64_t)b * a.opad * a.kpad;
    for (int idx = threadIdx.x; idx < 64 * 16; idx += kThreads) {
        const int r = idx >> 4, pq = (idx & 15) * 4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (p0 + pq < a.k) v = ldg<float4>(Ot + (int64_t)(r0 + r) * a.kpad + p0 + pq);
        const float x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) t[r][pq + u] = p0 + pq + u < a.k ? x[u] * sc : 0.f;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 64 * 8; idx += kThreads) {
        const int row = idx >> 3, c8 = (idx & 7) * 8;   // output row, first of eight entries
        uint32_t w[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float x0 = a.LT ? t[row][c8 + 2 * u] : t[c8 + 2 * u][row];
            const float x1 = a.LT ? t[row][c8 + 2 * u + 1] : t[c8 + 2 * u + 1][row];
            w[u] = (uint32_t)f32_to_bf16(x0) | ((uint32_t)f32_to_bf16(x1) << 16);
        }
        uint16_t* dst = a.LT ? a.LT + (int64_t)b * a.opad * a.kpad + (int64_t)(r0 + row) * a.kpad + p0 + c8
                             : a.L + (int64_t)b * a.kpad * a.opad + (int64_t)(p0 + row) * a.opad + r0 + c8;
        stg(dst, make_uint4(w[0], w[1], w[2], w[3]));
    }
}

}  // namespace

hipError_t launch_colpass_finish(const ColpassArgs& a, hipStream_t s) {
    if (a.kpad % 64 || a.opad % 64 || a.batch < 1 || a.batch > 65535 || (!a.L) == (!a.LT))
        return hipErrorInvalidValue;
    const int nrb = a.opad / kRB;
    const dim3 fold((unsigned)((a.k + 63) / 64), (unsigned)((nrb + kChunk - 1) / kChunk), (unsigned)a.batch);
    hipLaunchKernelGGL(colpass_fold, fold, dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(colpass_scale, dim3((unsigned)a.batch), dim3(kThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(a.kpad / 64), (unsigned)(a.opad / 64), (unsigned)a.batch);
    hipLaunchKernelGGL(colpass_compact, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs& a, int axis, int g_bf16, hipStream_t s) {
    if (axis == 0) {
        dim3 grid((unsigned)(a.opad / kT), (unsigned)(a.kpad / kT), (unsigned)a.batch);
        if (a.cols % 4 == 0) {
            hipLaunchKernelGGL((gather_rows<4>), grid, dim3(kThreads), 0, s, a);
        } else {
            hipLaunchKernelGGL((gather_rows<1>), grid, dim3(kThreads), 0, s, a);
        }
    } else {
        dim3 grid((unsigned)((a.cols + kCW - 1) / kCW), (unsigned)(a.opad / kRB), (unsigned)a.batch);
        const bool vec = a.cols % 4 == 0;
        if (g_bf16) {
            if (vec) hipLaunchKernelGGL((update_cols<4, uint16_t>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((update_cols<1, uint16_t>), grid, dim3(kThreads), 0, s, a);
        } else {
            if (vec) hipLaunchKernelGGL((update_cols<4, float>), grid, dim3(kThreads), 0, s, a);
            else hipLaunchKernelGGL((update_cols<1, float>), grid, dim3(kThreads), 0, s, a);
        }
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
