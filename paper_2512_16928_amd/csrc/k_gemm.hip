// K4: the Newton-Schulz GEMMs on MFMA (bf16 operands, fp32 accumulation).
//
// One Newton-Schulz step on the wide compact matrix Z (s x l, s <= l) is
//   A  = Z Z^T                     gemm<1, BT=0, EPI_SPLIT>   A kept as bf16 hi + lo
//   B  = b A + c A^2               gemm<3, BT=0, EPI_POLY>    A^2 = A A^T from three
//                                                             passes hi*hi+hi*lo+lo*hi
//   Z' = a Z + B Z                 gemm<1, BT=1, EPI_UPDATE | EPI_FINAL>
// The a Z term is added in fp32 in the epilogue rather than folded into the
// diagonal of B: with it separate, lines of Z that are exactly equal stay
// exactly equal through every step (their rows of A, B and Z' come from
// identical inputs), so no rounding noise enters the null space, where the
// polynomial would amplify it by a per step.
//
// C[i][j] = sum_k A[i][k] B[k][j]. The A operand is always given as rows
// with K contiguous. The B operand is given either as rows with K
// contiguous (BT = 0: Z Z^T reads Z twice, A^2 reads A, which is symmetric)
// or as a row-major [K][N] matrix (BT = 1: the update reads Z itself). For
// BT = 1 the K-slice of Z is staged in LDS as is and the MFMA fragments are
// read with gfx950's transposing LDS read (ds_read_b64_tr_b16): a lane of
// a 16-lane group receives element (i mod 4) of the 8 bytes addressed by
// source lane 4e + i/4 for e = 0..3, so pointing source lane s at row s/4,
// column 4 (s mod 4) hands lane i four consecutive K values of column i.
//
// Tiling for gfx950: a BM x BN output tile per block of WM x WN wave64s,
// each wave a (BM/WM) x (BN/WN) tile of v_mfma_f32_32x32x16_bf16 blocks.
// Operand K-slices (BK deep) are staged through LDS, double-buffered; the
// next slice is fetched into named registers before the current slice's
// MFMAs so its latency overlaps them. Tiles are numbered XCD-aware. The
// epilogue goes through a per-wave 32 x 32 LDS tile so row-major and
// transposed outputs are both written as 16-byte chunks.
//
// All dimensions are multiples of the tile (compact buffers are zero padded
// to 128, and the padding stays zero through every step).
#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kXcds = 8;   // accelerator complex dies on MI355X

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

__device__ __forceinline__ uint32_t pack2(float x, float y) {
    return (uint32_t)f32_to_bf16(x) | ((uint32_t)f32_to_bf16(y) << 16);
}

template <int NPASS, int BT_, int BM_, int BN_, int BK_, int WM_, int WN_>
struct Tile {
    static constexpr int BT = BT_;
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int THREADS = 64 * WM * WN;
    static constexpr int TM = BM / WM, TN = BN / WN;     // wave tile
    static constexpr int FM = TM / 32, FN = TN / 32;     // MFMA blocks per wave
    static constexpr int NA = NPASS == 1 ? 1 : 2;        // A operand tiles (hi[, lo])
    static constexpr int NB = NPASS == 1 ? 1 : 2;        // B operand tiles
    static constexpr int LDK = BK + 8;                   // padded K-major LDS row (bf16)
    static constexpr int LDN = BN + 16;                  // padded N-major LDS row (BT = 1)
    static constexpr int CPR = BK / 8;                   // 16-byte chunks per K-major row
    static constexpr int A_CH = BM * CPR, B_CH = BN * CPR;
    static constexpr int NCH = (NA * A_CH + NB * B_CH) / THREADS;  // chunks per thread
    static constexpr int A_TILE = BM * LDK;
    static constexpr int B_TILE = BT ? BK * LDN : BN * LDK;
    static constexpr int STAGE = NA * A_TILE + NB * B_TILE;        // elements
    static constexpr int EPI_LD = 33;                    // fp32 staging row (32 + 1)
    static constexpr int EPI_BYTES = WM * WN * 32 * EPI_LD * 4;
    static constexpr int SMEM = (2 * STAGE * 2 > EPI_BYTES) ? 2 * STAGE * 2 : EPI_BYTES;
    static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile is whole 32x32 blocks");
    static_assert(A_CH % THREADS == 0 && B_CH % THREADS == 0, "chunks split evenly");
    static_assert(NCH >= 1 && NCH <= 16, "at most 16 staged chunks per thread");
    static_assert(BK % 16 == 0, "BK is a multiple of the MFMA K");
    static_assert(!BT || NPASS == 1, "the transposed B operand is single-pass");
};

// Tile and in-tile position of a thread's I-th staged chunk. Chunks run over
// the A tiles, then the B tiles; every chunk index I maps all threads of the
// block into one tile (the tiles are whole multiples of the block size).
template <typename T, int I>
struct Chunk {
    static constexpr int flat0 = I * T::THREADS;
    static constexpr bool is_a = flat0 < T::NA * T::A_CH;
    static constexpr int tile = is_a ? flat0 / T::A_CH : (flat0 - T::NA * T::A_CH) / T::B_CH;
    static constexpr int within0 = is_a ? flat0 % T::A_CH : (flat0 - T::NA * T::A_CH) % T::B_CH;
    static constexpr int lds_base = is_a ? tile * T::A_TILE : T::NA * T::A_TILE + tile * T::B_TILE;
};

// B fragment (8 consecutive K of one column) through two transposing reads.
// `col` is the fragment's first column in the staged [BK][LDN] tile.
template <typename T>
__device__ __forceinline__ bf16x8 b_frag_tr(const uint16_t* sb, int krow, int col, int lane) {
    const int g = lane >> 4, s = lane & 15;
    const int row = krow + 8 * (g >> 1) + (s >> 2);
    const int c = col + 16 * (g & 1) + 4 * (s & 3);
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sb + row * T::LDN + c));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sb + (row + 4) * T::LDN + c));
    typedef __attribute__((ext_vector_type(8))) short i16x8;
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// MFMAs of one BK-deep K-slice staged at `st`, fragments software-pipelined
// (k-step kk+1 is read from LDS while the MFMAs of kk run).
template <int NPASS, typename T>
__device__ __forceinline__ void mma_slice(f32x16 (&acc)[T::FM][T::FN], const uint16_t* st,
                                          int wm, int wn, int lane) {
    const uint16_t* sa0 = st;
    const uint16_t* sa1 = st + T::A_TILE;
    const uint16_t* sb0 = st + T::NA * T::A_TILE;
    const uint16_t* sb1 = sb0 + T::B_TILE;
    const int arow = wm * T::TM + (lane & 31);
    const int brow = wn * T::TN + (lane & 31);
    const int kl = 8 * (lane >> 5);
    constexpr int KK = T::BK / 16;
    bf16x8 fa0[2][T::FM], fb0[2][T::FN], fa1[2][T::FM], fb1[2][T::FN];
#pragma unroll
    for (int kk = 0; kk <= KK; ++kk) {
        if (kk < KK) {
            const int ko = kk * 16 + kl;
            const int slot = kk & 1;
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
                fa0[slot][i] = *reinterpret_cast<const bf16x8*>(sa0 + (arow + i * 32) * T::LDK + ko);
#pragma unroll
            for (int j = 0; j < T::FN; ++j) {
                if constexpr (T::BT) {
                    fb0[slot][j] = b_frag_tr<T>(sb0, kk * 16, wn * T::TN + j * 32, lane);
                } else {
                    fb0[slot][j] = *reinterpret_cast<const bf16x8*>(sb0 + (brow + j * 32) * T::LDK + ko);
                }
            }
            if constexpr (NPASS == 3) {
#pragma unroll
                for (int i = 0; i < T::FM; ++i)
                    fa1[slot][i] = *reinterpret_cast<const bf16x8*>(sa1 + (arow + i * 32) * T::LDK + ko);
#pragma unroll
                for (int j = 0; j < T::FN; ++j)
                    fb1[slot][j] = *reinterpret_cast<const bf16x8*>(sb1 + (brow + j * 32) * T::LDK + ko);
            }
        }
        if (kk > 0) {
            const int slot = (kk - 1) & 1;
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j) {
                    if constexpr (NPASS == 3) {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa0[slot][i], fb1[slot][j], acc[i][j], 0, 0, 0);
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa1[slot][i], fb0[slot][j], acc[i][j], 0, 0, 0);
                    }
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa0[slot][i], fb0[slot][j], acc[i][j], 0, 0, 0);
                }
        }
    }
}

template <int NPASS, int EPI, typename T>
__global__ __launch_bounds__(T::THREADS) void gemm(GemmArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char smem_raw[T::SMEM];
    uint16_t* smem = reinterpret_cast<uint16_t*>(smem_raw);

    // XCD-aware tile order. Workgroups are dispatched round-robin over the
    // eight XCDs, each with its own L2; renumbering puts consecutive tiles --
    // the tiles of one matrix, which share its operands -- on one XCD, so a
    // matrix's compact operands are fetched into one L2 instead of eight.
    const int nx = gridDim.x, ny = gridDim.y;
    const int total = nx * ny * gridDim.z;
    const int hw = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    const int logical = (total % kXcds == 0) ? (hw % kXcds) * (total / kXcds) + hw / kXcds : hw;
    const int b = logical / (nx * ny);
    const int row0 = ((logical / nx) % ny) * T::BM;   // output rows (M)
    const int col0 = (logical % nx) * T::BN;          // output cols (N)
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WN, wn = wave % T::WN;

    const uint16_t* abase[2];
    const uint16_t* bbase[2];
    abase[0] = a.A0 + (int64_t)b * a.sA + (int64_t)row0 * a.lda;
    abase[1] = NPASS == 3 ? a.A1 + (int64_t)b * a.sA + (int64_t)row0 * a.lda : abase[0];
    if constexpr (T::BT) {
        bbase[0] = bbase[1] = a.B0 + (int64_t)b * a.sB + col0;
    } else {
        bbase[0] = a.B0 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb;
        bbase[1] = NPASS == 3 ? a.B1 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb : bbase[0];
    }
    // elements between consecutive K-slices of one staged chunk
    const int64_t astep = T::BK;
    const int64_t bstep = T::BT ? (int64_t)T::BK * a.ldb : T::BK;

    // staged chunk I: global pointer of slice 0, per-slice stride, LDS offset
#define DION2_CH_DECL(I) const uint16_t* gp##I = nullptr; int64_t gs##I = 0; int so##I = 0; uint4 r##I;
#define DION2_CH_INIT(I)                                                                \
    if constexpr ((I) < T::NCH) {                                                       \
        using CI = Chunk<T, I>;                                                         \
        const int w = CI::within0 + tid;                                                \
        if constexpr (CI::is_a) {                                                       \
            const int rr = w / T::CPR, kc = w % T::CPR;                                 \
            gp##I = abase[CI::tile] + (int64_t)rr * a.lda + kc * 8;                     \
            gs##I = astep;                                                              \
            so##I = CI::lds_base + rr * T::LDK + kc * 8;                                \
        } else if constexpr (T::BT) {                                                   \
            const int kr = w / (T::BN / 8), c8 = w % (T::BN / 8);                       \
            gp##I = bbase[CI::tile] + (int64_t)kr * a.ldb + c8 * 8;                     \
            gs##I = bstep;                                                              \
            so##I = CI::lds_base + kr * T::LDN + c8 * 8;                                \
        } else {                                                                        \
            const int rr = w / T::CPR, kc = w % T::CPR;                                 \
            gp##I = bbase[CI::tile] + (int64_t)rr * a.ldb + kc * 8;                     \
            gs##I = bstep;                                                              \
            so##I = CI::lds_base + rr * T::LDK + kc * 8;                                \
        }                                                                               \
    }
#define DION2_CH_LOAD(I, KT)                                                            \
    if constexpr ((I) < T::NCH) r##I = *reinterpret_cast<const uint4*>(gp##I + (KT) * gs##I);
#define DION2_CH_STORE(I, BASE)                                                         \
    if constexpr ((I) < T::NCH) *reinterpret_cast<uint4*>((BASE) + so##I) = r##I;
#define DION2_CH_ALL(M, ...)                                                            \
    M(0, __VA_ARGS__) M(1, __VA_ARGS__) M(2, __VA_ARGS__) M(3, __VA_ARGS__)             \
    M(4, __VA_ARGS__) M(5, __VA_ARGS__) M(6, __VA_ARGS__) M(7, __VA_ARGS__)             \
    M(8, __VA_ARGS__) M(9, __VA_ARGS__) M(10, __VA_ARGS__) M(11, __VA_ARGS__)           \
    M(12, __VA_ARGS__) M(13, __VA_ARGS__) M(14, __VA_ARGS__) M(15, __VA_ARGS__)
#define DION2_CH_DECL_(I, ...) DION2_CH_DECL(I)
#define DION2_CH_INIT_(I, ...) DION2_CH_INIT(I)
    DION2_CH_ALL(DION2_CH_DECL_, 0)
    DION2_CH_ALL(DION2_CH_INIT_, 0)

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = a.K / T::BK;
    DION2_CH_ALL(DION2_CH_LOAD, 0)
    DION2_CH_ALL(DION2_CH_STORE, smem)
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        // next K-slice (the last iteration re-reads the current one, which is
        // in bounds, and stages it into the idle buffer)
        const int kn = kt + 1 < nk ? kt + 1 : kt;
        DION2_CH_ALL(DION2_CH_LOAD, kn)
        __builtin_amdgcn_sched_barrier(0);
        mma_slice<NPASS, T>(acc, smem + (kt & 1) * T::STAGE, wm, wn, lane);
        __builtin_amdgcn_sched_barrier(0);
        DION2_CH_ALL(DION2_CH_STORE, smem + ((kt + 1) & 1) * T::STAGE)
        __syncthreads();
    }
#undef DION2_CH_DECL
#undef DION2_CH_INIT
#undef DION2_CH_LOAD
#undef DION2_CH_STORE
#undef DION2_CH_ALL
#undef DION2_CH_DECL_
#undef DION2_CH_INIT_

    // ---- epilogue, one 32 x 32 block at a time through a per-wave LDS tile.
    // The tile belongs to its wave alone and LDS accesses of one wave complete
    // in issue order, so wave barriers order the staging.
    float* stage = reinterpret_cast<float*>(smem_raw) + wave * 32 * T::EPI_LD;
    const int er = lane >> 1;          // row (or transposed row) handled by this lane
    const int ec = (lane & 1) * 16;    // 16 consecutive columns
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
            const int R = row0 + wm * T::TM + i * 32;   // block origin in the output
            const int Cc = col0 + wn * T::TN + j * 32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                stage[m * T::EPI_LD + (lane & 31)] = acc[i][j][r];
            }
            __builtin_amdgcn_wave_barrier();
            float v[16];
            const bool transposed = EPI == EPI_FINAL && a.out_transposed;
            if (!transposed) {
#pragma unroll
                for (int q = 0; q < 16; ++q) v[q] = stage[er * T::EPI_LD + ec + q];
            } else {
                // output row = block column er, 16 consecutive block rows
#pragma unroll
                for (int q = 0; q < 16; ++q) v[q] = stage[(ec + q) * T::EPI_LD + er];
            }
            const int64_t orow = transposed ? Cc + er : R + er;
            const int64_t ocol = transposed ? R + ec : Cc + ec;
            if constexpr (EPI == EPI_UPDATE || EPI == EPI_FINAL) {
                // a Z at this lane's 16 block entries (row zr, columns zc..zc+15)
                const int64_t zr = transposed ? R + ec : R + er;
                const int64_t zc = transposed ? Cc + er : Cc + ec;
                if (!transposed) {
                    const uint16_t* zp = a.E0 + (int64_t)b * a.sE + zr * a.lde + zc;
                    const uint4 z0 = reinterpret_cast<const uint4*>(zp)[0];
                    const uint4 z1 = reinterpret_cast<const uint4*>(zp)[1];
                    const uint32_t zw[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        v[2 * q] += a.ca * bf16_bits_to_f32(zw[q] & 0xffffu);
                        v[2 * q + 1] += a.ca * bf16_bits_to_f32(zw[q] >> 16);
                    }
                } else {
                    // transposed output: entry q is Z[R + ec + q][Cc + er]
                    const uint16_t* zp = a.E0 + (int64_t)b * a.sE + zr * a.lde + zc;
#pragma unroll
                    for (int q = 0; q < 16; ++q) v[q] += a.ca * bf16_bits_to_f32(zp[(int64_t)q * a.lde]);
                }
            }
            if constexpr (EPI == EPI_SPLIT) {
                uint32_t h[8], l[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const uint16_t h0 = f32_to_bf16(v[2 * q]), h1 = f32_to_bf16(v[2 * q + 1]);
                    h[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                    l[q] = pack2(v[2 * q] - bf16_bits_to_f32(h0), v[2 * q + 1] - bf16_bits_to_f32(h1));
                }
                uint16_t* hp = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + orow * a.ldo0 + ocol;
                uint16_t* lp = static_cast<uint16_t*>(a.out1) + (int64_t)b * a.sOut1 + orow * a.ldo1 + ocol;
                reinterpret_cast<uint4*>(hp)[0] = make_uint4(h[0], h[1], h[2], h[3]);
                reinterpret_cast<uint4*>(hp)[1] = make_uint4(h[4], h[5], h[6], h[7]);
                reinterpret_cast<uint4*>(lp)[0] = make_uint4(l[0], l[1], l[2], l[3]);
                reinterpret_cast<uint4*>(lp)[1] = make_uint4(l[4], l[5], l[6], l[7]);
            } else if constexpr (EPI == EPI_POLY) {
                // B = b (A_hi + A_lo) + c A^2
                const int64_t eo = (int64_t)b * a.sE + orow * a.lde + ocol;
                const uint4 h0 = reinterpret_cast<const uint4*>(a.E0 + eo)[0];
                const uint4 h1 = reinterpret_cast<const uint4*>(a.E0 + eo)[1];
                const uint4 l0 = reinterpret_cast<const uint4*>(a.E1 + eo)[0];
                const uint4 l1 = reinterpret_cast<const uint4*>(a.E1 + eo)[1];
                const uint32_t hw[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
                const uint32_t lw[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
                uint32_t o[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float a0 = bf16_bits_to_f32(hw[q] & 0xffffu) + bf16_bits_to_f32(lw[q] & 0xffffu);
                    const float a1 = bf16_bits_to_f32(hw[q] >> 16) + bf16_bits_to_f32(lw[q] >> 16);
                    o[q] = pack2(a.cb * a0 + a.cc * v[2 * q], a.cb * a1 + a.cc * v[2 * q + 1]);
                }
                uint16_t* op = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + orow * a.ldo0 + ocol;
                reinterpret_cast<uint4*>(op)[0] = make_uint4(o[0], o[1], o[2], o[3]);
                reinterpret_cast<uint4*>(op)[1] = make_uint4(o[4], o[5], o[6], o[7]);
            } else if constexpr (EPI == EPI_UPDATE) {
                uint16_t* op = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + orow * a.ldo0 + ocol;
                reinterpret_cast<uint4*>(op)[0] = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]),
                                                             pack2(v[4], v[5]), pack2(v[6], v[7]));
                reinterpret_cast<uint4*>(op)[1] = make_uint4(pack2(v[8], v[9]), pack2(v[10], v[11]),
                                                             pack2(v[12], v[13]), pack2(v[14], v[15]));
            } else {
                float* op = static_cast<float*>(a.out0) + (int64_t)b * a.sOut0 + orow * a.ldo0 + ocol;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    reinterpret_cast<float4*>(op)[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
            }
            __builtin_amdgcn_wave_barrier();   // the stage tile is rewritten next
        }
    }
}

template <int NPASS, int EPI, typename T>
hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
    if (a.M % T::BM || a.N % T::BN || a.K % T::BK) return hipErrorInvalidValue;
    dim3 grid((unsigned)(a.N / T::BN), (unsigned)(a.M / T::BM), (unsigned)a.batch);
    hipLaunchKernelGGL((gemm<NPASS, EPI, T>), grid, dim3(T::THREADS), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, hipStream_t s) {
    using TG = Tile<1, 0, 128, 128, 64, 2, 2>;   // Gram
    using TP = Tile<3, 0, 128, 128, 32, 2, 2>;   // polynomial (three passes)
    using TU = Tile<1, 1, 128, 128, 64, 2, 2>;   // update (B operand [K][N])
    switch (epi) {
        case EPI_SPLIT: return launch_tile<1, EPI_SPLIT, TG>(a, s);
        case EPI_POLY: return launch_tile<3, EPI_POLY, TP>(a, s);
        case EPI_UPDATE: return launch_tile<1, EPI_UPDATE, TU>(a, s);
        case EPI_FINAL: return launch_tile<1, EPI_FINAL, TU>(a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace dion2
