// K4: the Newton-Schulz GEMMs on MFMA (bf16 operands, fp32 accumulation).
//
// One Newton-Schulz step on the wide compact matrix Z (s x l, s <= l) is
//   A  = Z Z^T                              gemm_nt<1, EPI_SPLIT>
//   B  = b A + c A^2                        gemm_nt<3, EPI_POLY>
//   Z' = a Z + B Z                          gemm_nt<1, EPI_AXPY | EPI_FINAL>
// All three are "NT" products C[i][j] = sum_k A[i][k] B[j][k] whose operands
// are K-contiguous rows: Z Z^T reads Z twice; A^2 = A A^T because A is
// symmetric; B Z reads B and the transposed copy Z^T that the previous step
// wrote. A is kept as a bf16 hi/lo pair and A^2 is formed from three passes
// (hi*hi + hi*lo + lo*hi), which keeps the rounding of A out of A^2.
//
// Tiling for gfx950: 256 threads (4 wave64) per 128 x 128 output tile, each
// wave a 64 x 64 quadrant of 2 x 2 v_mfma_f32_32x32x16_bf16 blocks. Operand
// tiles are staged through LDS, double-buffered, with the next K-slice
// fetched into registers while the current one feeds the MFMAs. The
// epilogue stages the fp32 tile in LDS so both the row-major and the
// transposed output are written with 16-byte coalesced stores.
//
// All dimensions are multiples of 128 (compact buffers are zero padded).
#include "dion2_device.h"

namespace dion2 {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kThreads = 256;
constexpr int BM = 128, BN = 128;
constexpr int kCLd = BN + 4;   // fp32 staging row stride

template <int NPASS> struct Cfg {
    static constexpr int BK = NPASS == 1 ? 64 : 32;
    static constexpr int LDK = BK + 8;              // bf16 row stride in LDS
    static constexpr int NTILE = NPASS == 1 ? 2 : 4;  // operand tiles per stage
    static constexpr int TILE = BM * LDK;           // elements per operand tile
    static constexpr int STAGE = NTILE * TILE;
    static constexpr int CPR = BK / 8;              // 16-byte chunks per tile row
    static constexpr int PER_T = BM * CPR / kThreads;  // chunks per thread per tile
    static constexpr int SMEM_OPS = 2 * STAGE * 2;  // bytes
    static constexpr int SMEM_EPI = BM * kCLd * 4;
    static constexpr int SMEM = SMEM_OPS > SMEM_EPI ? SMEM_OPS : SMEM_EPI;
};

__device__ __forceinline__ uint32_t pack2(float x, float y) {
    return (uint32_t)f32_to_bf16(x) | ((uint32_t)f32_to_bf16(y) << 16);
}

template <int NPASS, int EPI>
__global__ __launch_bounds__(kThreads, 2) void gemm_nt(GemmArgs a) {
    using C = Cfg<NPASS>;
    __shared__ __attribute__((aligned(16))) unsigned char smem_raw[C::SMEM];
    uint16_t* smem = reinterpret_cast<uint16_t*>(smem_raw);

    const int b = blockIdx.z;
    const int row0 = blockIdx.y * BM;   // output rows (M)
    const int col0 = blockIdx.x * BN;   // output cols (N)
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // Operand tiles of this block: NPASS==1 {A0, B0}; NPASS==3 {A0, A1, B0, B1}.
    // Every thread stages eight 16-byte chunks per K-slice (NTILE * PER_T == 8),
    // held in eight named registers so none of them can live in scratch.
    static_assert(C::NTILE * C::PER_T == 8, "eight staged chunks per thread");
    const uint16_t* tsrc[4];
    int tld[4];
    tsrc[0] = a.A0 + (int64_t)b * a.sA + (int64_t)row0 * a.lda;
    tld[0] = a.lda;
    if constexpr (NPASS == 1) {
        tsrc[1] = a.B0 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb;
        tld[1] = a.ldb;
        tsrc[2] = tsrc[3] = nullptr;
        tld[2] = tld[3] = 0;
    } else {
        tsrc[1] = a.A1 + (int64_t)b * a.sA + (int64_t)row0 * a.lda;
        tsrc[2] = a.B0 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb;
        tsrc[3] = a.B1 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb;
        tld[1] = a.lda;
        tld[2] = tld[3] = a.ldb;
    }
#define DION2_CHUNK_PTR(I)                                                              \
    const uint16_t* gp##I;                                                              \
    int so##I;                                                                          \
    {                                                                                   \
        constexpr int t = (I) / C::PER_T, i = (I) % C::PER_T;                           \
        const int c = tid + i * kThreads;                                               \
        gp##I = tsrc[t] + (int64_t)(c / C::CPR) * tld[t] + (c % C::CPR) * 8;            \
        so##I = t * C::TILE + (c / C::CPR) * C::LDK + (c % C::CPR) * 8;                 \
    }
    DION2_CHUNK_PTR(0) DION2_CHUNK_PTR(1) DION2_CHUNK_PTR(2) DION2_CHUNK_PTR(3)
    DION2_CHUNK_PTR(4) DION2_CHUNK_PTR(5) DION2_CHUNK_PTR(6) DION2_CHUNK_PTR(7)
#undef DION2_CHUNK_PTR
    uint4 r0, r1, r2, r3, r4, r5, r6, r7;
#define DION2_GLOAD(K0)                                                                 \
    r0 = *reinterpret_cast<const uint4*>(gp0 + (K0));                                   \
    r1 = *reinterpret_cast<const uint4*>(gp1 + (K0));                                   \
    r2 = *reinterpret_cast<const uint4*>(gp2 + (K0));                                   \
    r3 = *reinterpret_cast<const uint4*>(gp3 + (K0));                                   \
    r4 = *reinterpret_cast<const uint4*>(gp4 + (K0));                                   \
    r5 = *reinterpret_cast<const uint4*>(gp5 + (K0));                                   \
    r6 = *reinterpret_cast<const uint4*>(gp6 + (K0));                                   \
    r7 = *reinterpret_cast<const uint4*>(gp7 + (K0));
#define DION2_SSTORE(BASE)                                                              \
    *reinterpret_cast<uint4*>((BASE) + so0) = r0;                                       \
    *reinterpret_cast<uint4*>((BASE) + so1) = r1;                                       \
    *reinterpret_cast<uint4*>((BASE) + so2) = r2;                                       \
    *reinterpret_cast<uint4*>((BASE) + so3) = r3;                                       \
    *reinterpret_cast<uint4*>((BASE) + so4) = r4;                                       \
    *reinterpret_cast<uint4*>((BASE) + so5) = r5;                                       \
    *reinterpret_cast<uint4*>((BASE) + so6) = r6;                                       \
    *reinterpret_cast<uint4*>((BASE) + so7) = r7;

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = a.K / C::BK;
    DION2_GLOAD(0)
    DION2_SSTORE(smem)
    __syncthreads();
    const int arow = wm * 64 + (lane & 31);
    const int brow = wn * 64 + (lane & 31);
    const int kl = 8 * (lane >> 5);
    for (int kt = 0; kt < nk; ++kt) {
        // next K-slice (the last iteration re-reads the current one, which is
        // in bounds, and stages it into the idle buffer)
        const int k0 = (kt + 1 < nk ? kt + 1 : kt) * C::BK;
        DION2_GLOAD(k0)
        // keep the prefetch ahead of the MFMAs so its latency overlaps them
        __builtin_amdgcn_sched_barrier(0);
        const uint16_t* st = smem + (kt & 1) * C::STAGE;
#pragma unroll
        for (int kk = 0; kk < C::BK / 16; ++kk) {
            const int ko = kk * 16 + kl;
            if constexpr (NPASS == 1) {
                bf16x8 fa[2], fb[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    fa[i] = *reinterpret_cast<const bf16x8*>(st + (arow + i * 32) * C::LDK + ko);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    fb[j] = *reinterpret_cast<const bf16x8*>(st + C::TILE + (brow + j * 32) * C::LDK + ko);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            } else {
                bf16x8 fa0[2], fa1[2], fb0[2], fb1[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    fa0[i] = *reinterpret_cast<const bf16x8*>(st + (arow + i * 32) * C::LDK + ko);
                    fa1[i] = *reinterpret_cast<const bf16x8*>(st + C::TILE + (arow + i * 32) * C::LDK + ko);
                }
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    fb0[j] = *reinterpret_cast<const bf16x8*>(st + 2 * C::TILE + (brow + j * 32) * C::LDK + ko);
                    fb1[j] = *reinterpret_cast<const bf16x8*>(st + 3 * C::TILE + (brow + j * 32) * C::LDK + ko);
                }
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa0[i], fb1[j], acc[i][j], 0, 0, 0);
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa1[i], fb0[j], acc[i][j], 0, 0, 0);
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa0[i], fb0[j], acc[i][j], 0, 0, 0);
                    }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        {
            uint16_t* dst = smem + ((kt + 1) & 1) * C::STAGE;
            DION2_SSTORE(dst)
        }
        __syncthreads();
    }
#undef DION2_GLOAD
#undef DION2_SSTORE

    // ---- epilogue: stage the fp32 tile in LDS
    float* Cs = reinterpret_cast<float*>(smem_raw);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                const int n = wn * 64 + j * 32 + (lane & 31);
                Cs[m * kCLd + n] = acc[i][j][r];
            }
    __syncthreads();

    const int ec = (tid & 15) * 8;   // 8 consecutive columns
    if constexpr (EPI == EPI_SPLIT) {
        uint16_t* hiP = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0;
        uint16_t* loP = static_cast<uint16_t*>(a.out1) + (int64_t)b * a.sOut1;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int er = (tid >> 4) + 16 * i;
            uint32_t h[4], l[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float v0 = Cs[er * kCLd + ec + 2 * q];
                const float v1 = Cs[er * kCLd + ec + 2 * q + 1];
                const uint16_t h0 = f32_to_bf16(v0), h1 = f32_to_bf16(v1);
                h[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                l[q] = pack2(v0 - bf16_bits_to_f32(h0), v1 - bf16_bits_to_f32(h1));
            }
            const int64_t off = (int64_t)(row0 + er) * a.ldo0 + col0 + ec;
            *reinterpret_cast<uint4*>(hiP + off) = make_uint4(h[0], h[1], h[2], h[3]);
            *reinterpret_cast<uint4*>(loP + (int64_t)(row0 + er) * a.ldo1 + col0 + ec) =
                make_uint4(l[0], l[1], l[2], l[3]);
        }
    } else if constexpr (EPI == EPI_POLY) {
        const uint16_t* hiP = a.E0 + (int64_t)b * a.sE;
        const uint16_t* loP = a.E1 + (int64_t)b * a.sE;
        uint16_t* outP = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int er = (tid >> 4) + 16 * i;
            const int64_t eoff = (int64_t)(row0 + er) * a.lde + col0 + ec;
            const uint4 hv = *reinterpret_cast<const uint4*>(hiP + eoff);
            const uint4 lv = *reinterpret_cast<const uint4*>(loP + eoff);
            const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
            const uint32_t lw[4] = {lv.x, lv.y, lv.z, lv.w};
            uint32_t o[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float a0 = bf16_bits_to_f32(hw[q] & 0xffffu) + bf16_bits_to_f32(lw[q] & 0xffffu);
                const float a1 = bf16_bits_to_f32(hw[q] >> 16) + bf16_bits_to_f32(lw[q] >> 16);
                const float v0 = a.cb * a0 + a.cc * Cs[er * kCLd + ec + 2 * q];
                const float v1 = a.cb * a1 + a.cc * Cs[er * kCLd + ec + 2 * q + 1];
                o[q] = pack2(v0, v1);
            }
            *reinterpret_cast<uint4*>(outP + (int64_t)(row0 + er) * a.ldo0 + col0 + ec) =
                make_uint4(o[0], o[1], o[2], o[3]);
        }
    } else {
        // EPI_AXPY / EPI_FINAL: Z' = a Z + C
        const uint16_t* zP = a.E0 + (int64_t)b * a.sE;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int er = (tid >> 4) + 16 * i;
            const uint4 zv = *reinterpret_cast<const uint4*>(zP + (int64_t)(row0 + er) * a.lde + col0 + ec);
            const uint32_t zw[4] = {zv.x, zv.y, zv.z, zv.w};
            float v[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                v[2 * q] = a.ca * bf16_bits_to_f32(zw[q] & 0xffffu) + Cs[er * kCLd + ec + 2 * q];
                v[2 * q + 1] = a.ca * bf16_bits_to_f32(zw[q] >> 16) + Cs[er * kCLd + ec + 2 * q + 1];
            }
            if constexpr (EPI == EPI_AXPY) {
                uint16_t* outP = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0;
                *reinterpret_cast<uint4*>(outP + (int64_t)(row0 + er) * a.ldo0 + col0 + ec) =
                    make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
            } else {
                if (!a.out_transposed) {
                    float* outP = static_cast<float*>(a.out0) + (int64_t)b * a.sOut0;
                    float* d = outP + (int64_t)(row0 + er) * a.ldo0 + col0 + ec;
                    *reinterpret_cast<float4*>(d) = make_float4(v[0], v[1], v[2], v[3]);
                    *reinterpret_cast<float4*>(d + 4) = make_float4(v[4], v[5], v[6], v[7]);
                }
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) Cs[er * kCLd + ec + q] = v[q];
        }
        const bool transposed_out = (EPI == EPI_AXPY) || a.out_transposed;
        if (transposed_out) {
            __syncthreads();
            // transposed tile: output row = tile column tc, 8 consecutive tile rows
            const int tr = (tid & 15) * 8;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int tc = (tid >> 4) + 16 * i;
                float v[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = Cs[(tr + q) * kCLd + tc];
                if constexpr (EPI == EPI_AXPY) {
                    uint16_t* outP = static_cast<uint16_t*>(a.out1) + (int64_t)b * a.sOut1;
                    *reinterpret_cast<uint4*>(outP + (int64_t)(col0 + tc) * a.ldo1 + row0 + tr) =
                        make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
                } else {
                    float* outP = static_cast<float*>(a.out0) + (int64_t)b * a.sOut0;
                    float* d = outP + (int64_t)(col0 + tc) * a.ldo0 + row0 + tr;
                    *reinterpret_cast<float4*>(d) = make_float4(v[0], v[1], v[2], v[3]);
                    *reinterpret_cast<float4*>(d + 4) = make_float4(v[4], v[5], v[6], v[7]);
                }
            }
        }
    }
}

template <int NPASS, int EPI>
hipError_t launch_one(const GemmArgs& a, hipStream_t s) {
    dim3 grid((unsigned)(a.N / BN), (unsigned)(a.M / BM), (unsigned)a.batch);
    hipLaunchKernelGGL((gemm_nt<NPASS, EPI>), grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, hipStream_t s) {
    if (a.M % BM || a.N % BN || a.K % 64) return hipErrorInvalidValue;
    switch (epi) {
        case EPI_SPLIT: return launch_one<1, EPI_SPLIT>(a, s);
        case EPI_POLY: return launch_one<3, EPI_POLY>(a, s);
        case EPI_AXPY: return launch_one<1, EPI_AXPY>(a, s);
        case EPI_FINAL: return launch_one<1, EPI_FINAL>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace dion2
