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
// stages a 64 x 64 tile of O in LDS so that W is walked along its rows,
// touching the selected columns K[p] of each row in ascending order.
#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kT = 64;
constexpr int kThreads = 256;

template <typename WT>
__device__ __forceinline__ void update(WT* w, float o, double lr_eff) {
    const double x = (double)Elem<WT>::load(w);
    const double r = __dsub_rn(x, __dmul_rn(lr_eff, (double)o));
    Elem<WT>::store_f64(w, r);
}

template <typename WT>
__global__ __launch_bounds__(kThreads) void apply_rows(ApplyArgs a) {
    const int b = blockIdx.z;
    const int p0 = blockIdx.y * kT, j0 = blockIdx.x * kT;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    WT* __restrict__ W = a.ms.w<WT>(b);
    const int32_t* __restrict__ K = a.sel + (int64_t)b * a.k;
    const float* __restrict__ O = a.O + (int64_t)b * a.kpad * a.opad;
    const int j = j0 + tx;
    if (j >= a.d_oth) return;
    for (int pl = ty; pl < kT; pl += 4) {
        const int p = p0 + pl;
        if (p >= a.k) break;
        const float o = O[(int64_t)p * a.opad + j];
        update(W + (int64_t)K[p] * a.cols + j, o, a.lr_eff);
        if (a.dbg) a.dbg[((int64_t)b * a.k + p) * a.d_oth + j] = o;
    }
}

template <typename WT>
__global__ __launch_bounds__(kThreads) void apply_cols(ApplyArgs a) {
    __shared__ float tile[kT][kT + 1];   // [p local][r local]
    const int b = blockIdx.z;
    const int p0 = blockIdx.y * kT, r0 = blockIdx.x * kT;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    WT* __restrict__ W = a.ms.w<WT>(b);
    const int32_t* __restrict__ K = a.sel + (int64_t)b * a.k;
    const float* __restrict__ O = a.O + (int64_t)b * a.kpad * a.opad;
    // load O[p][r] along r (contiguous); padding of O is in bounds
    for (int pl = ty; pl < kT; pl += 4) {
        const int p = p0 + pl;
        const float o = O[(int64_t)p * a.opad + r0 + tx];
        tile[pl][tx] = o;
        if (a.dbg && p < a.k && r0 + tx < a.d_oth)
            a.dbg[((int64_t)b * a.k + p) * a.d_oth + r0 + tx] = o;
    }
    __syncthreads();
    const int p = p0 + tx;
    if (p >= a.k) return;
    const int col = K[p];
    for (int rl = ty; rl < kT; rl += 4) {
        const int r = r0 + rl;
        if (r >= a.d_oth) break;
        update(W + (int64_t)r * a.cols + col, tile[tx][rl], a.lr_eff);
    }
}

}  // namespace

hipError_t launch_apply(const ApplyArgs& a, int axis, int w_bf16, hipStream_t s) {
    const unsigned gj = (unsigned)((a.d_oth + kT - 1) / kT);
    const unsigned gp = (unsigned)((a.k + kT - 1) / kT);
    dim3 grid(gj, gp, (unsigned)a.batch);
    if (axis == 0) {
        if (w_bf16) hipLaunchKernelGGL((apply_rows<uint16_t>), grid, dim3(kThreads), 0, s, a);
        else hipLaunchKernelGGL((apply_rows<float>), grid, dim3(kThreads), 0, s, a);
    } else {
        if (w_bf16) hipLaunchKernelGGL((apply_cols<uint16_t>), grid, dim3(kThreads), 0, s, a);
        else hipLaunchKernelGGL((apply_cols<float>), grid, dim3(kThreads), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace dion2
