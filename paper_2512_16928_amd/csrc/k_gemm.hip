// K4: the Newton-Schulz GEMMs on MFMA (bf16 operands, fp32 accumulation).
//
// One Newton-Schulz step on the wide compact matrix Z (s x l, s <= l) is
//   A  = Z Z^T                     gemm<1, EPI_H16>, B as rows    A kept as fp16 (scaled)
//   B  = b A + c A^2               gemm<1, EPI_POLY_H16>, B as rows  A^2 = A A^T, one fp16 pass
//   Z' = a Z + B Z                 gemm<1, EPI_UPDATE | EPI_FINAL>, B operand = Z as [K][N]
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
// BT = 1 the MFMA fragments are read with gfx950's transposing LDS read
// (ds_read_b64_tr_b16): a lane of a 16-lane group receives element (i mod 4)
// of the 8 bytes addressed by source lane 4e + i/4 for e = 0..3, so pointing
// source lane s at row s/4, column 4 (s mod 4) hands lane i four
// consecutive K values of column i.
//
// The GRAM form's chain of s x s products runs the same way on bf16 hi / lo
// pairs (three passes), or, as an option, on scaled fp16 matrices with
// v_mfma_f32_32x32x16_f16 (one pass; EPI_H16 and EPI_QPOLY_H16 store fp16).
// For s <= 64 the whole chain is one launch instead (chain_small): one block
// per matrix keeps its s x s matrices in LDS and computes every product as
// the launches would, bitwise.
// With the fp32 master Z itself is a hi / lo pair: the Gram matrix takes
// three passes, and so does the final product, whose [K][N] operand then
// has a lo tile read through the same transposing LDS reads.
//
// Tiling for gfx950: a BM x BN output tile per block of WM x WN wave64s,
// each wave a (BM/WM) x (BN/WN) tile of v_mfma_f32_32x32x16_bf16 blocks.
// K-slices (BK deep) go from global memory straight into an S-stage LDS
// ring with global_load_lds_dwordx4 (each lane's 16 bytes land at the
// wave's LDS base + 16 * lane), S - 1 slices ahead of the MFMAs, so no
// registers stage the operands and a slice's load latency is covered by
// S - 2 slices of compute. Tiles are stored unpadded with an XOR swizzle of
// their 16-byte chunks, chosen so both the fragment reads (ds_read_b128)
// and the transposing reads hit distinct LDS banks; each lane fetches the
// global chunk that belongs in its LDS slot. Tiles are numbered XCD-aware;
// the symmetric products (A and B) compute only the tiles on and above the
// diagonal and write each one twice, so that the stored matrix is exactly
// symmetric. The epilogue goes through a per-wave 32 x 32 LDS tile: each
// lane finishes 16 entries of a row there, and the
// block then leaves in whole row segments (64 bytes of bf16 or 128 bytes of
// fp32 per row), row-major or transposed for the mirrored copy.
//
// All dimensions are multiples of the tile (compact buffers are zero padded
// to 128, and the padding stays zero through every step).
#include <type_traits>

#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kXcds = 8;   // accelerator complex dies on MI355X

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((address_space(3))) void lds_void;

// two fp32 -> packed bf16 pair (RNE), one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack2(float x, float y) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
    const bf16x2 v = {(__bf16)x, (__bf16)y};
    return __builtin_bit_cast(uint32_t, v);
}

// two fp32 -> packed fp16 pair (RNE)
__device__ __forceinline__ uint32_t pack2h(float x, float y) {
    typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;
    const f16x2 v = {(_Float16)x, (_Float16)y};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// One 32 x 32 x 16 MFMA block on bf16 or fp16 fragments.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma32(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

template <int NPASS, int BT_, int BM_, int BN_, int BK_, int WM_, int WN_, int S_, bool F16_ = false>
struct Tile {
    static constexpr int BT = BT_, S = S_;
    static constexpr bool F16 = F16_;                    // fp16 operands (else bf16)
    using Frag = typename std::conditional<F16_, f16x8, bf16x8>::type;
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int WAVES = WM * WN;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int TM = BM / WM, TN = BN / WN;     // wave tile
    static constexpr int FM = TM / 32, FN = TN / 32;     // MFMA blocks per wave
    static constexpr int NA = NPASS == 1 ? 1 : 2;        // A operand tiles (hi[, lo])
    static constexpr int NB = NPASS == 3 ? 2 : 1;        // B operand tiles
    // K-major tiles: rows of BK bf16 (pitch PK bytes), CPR chunks of 16 B
    static constexpr int PK = BK * 2;
    static constexpr int CPR = BK / 8;
    static constexpr int GK = 256 / PK;                  // rows sharing one bank sweep
    // N-major tile (BT = 1): rows of BN bf16 (pitch PN bytes)
    static constexpr int PN = BN * 2;
    static constexpr int A_BYTES = BM * PK;
    static constexpr int B_BYTES = BN * PK;              // same size either layout
    static constexpr int STAGE_BYTES = NA * A_BYTES + NB * B_BYTES;
    static constexpr int STAGE_INSTS = STAGE_BYTES / 1024;   // 1 KB per wave instruction
    static constexpr int IPW = STAGE_INSTS / WAVES;      // load instructions per wave per slice
    static constexpr int EPI_LD = 33;                    // fp32 staging row (32 + 1)
    static constexpr int EPI_BYTES = WAVES * 32 * EPI_LD * 4;
    static constexpr int SMEM = (S * STAGE_BYTES > EPI_BYTES) ? S * STAGE_BYTES : EPI_BYTES;
    static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile is whole 32x32 blocks");
    static_assert(BK % 16 == 0 && (BK == 32 || BK == 64), "BK of 32 or 64");
    static_assert(A_BYTES % 1024 == 0 && B_BYTES % 1024 == 0, "tiles are whole 1 KB blocks");
    static_assert(STAGE_INSTS % WAVES == 0, "load instructions split evenly over waves");
    static_assert(NPASS >= 1 && NPASS <= 3, "one to three passes");
    static_assert(!BT || BN == 128, "the [K][N] B operand: BN 128");
    static_assert(S >= 2 && S <= 4, "two to four stages");
    static_assert(!F16 || (NPASS == 1 && !BT), "fp16 operands: one pass, B as rows");
};

// Byte offset, inside a K-major tile, of logical 16-byte chunk c of row r.
template <typename T>
__device__ __forceinline__ int kmajor_off(int r, int c) {
    return r * T::PK + 16 * (c ^ ((r / T::GK) % T::CPR));
}
// Byte offset, inside the [BK][BN] tile, of logical 16-byte chunk c of row r.
__device__ __forceinline__ int nmajor_off(int r, int c) {
    return r * 256 + 16 * (c ^ ((r & 3) << 2));
}

// Issue the direct-to-LDS load `q` (0 <= q < IPW) of this wave's part of
// K-slice `kt` into the stage at `dst`. Wave w owns the stage's 1 KB blocks
// w, w + WAVES, ...; lane i of a block fills the block's 16-byte slot i with
// the global chunk that belongs there.
template <int NPASS, typename T>
__device__ __forceinline__ void load_one(const GemmArgs& a, unsigned char* dst, int kt,
                                         const uint16_t* const (&abase)[2],
                                         const uint16_t* const (&bbase)[2], int wave, int lane, int q) {
    const int blk = wave + q * T::WAVES;   // 1 KB block of the stage (wave-uniform)
    const uint16_t* src;
    if (blk * 1024 < T::NA * T::A_BYTES) {
        // K-major A tile: the block holds 1024 / PK whole rows
        const int t = (blk * 1024) / T::A_BYTES;
        const int lb = (blk * 1024) % T::A_BYTES + lane * 16;
        const int r = lb / T::PK, slot = (lb % T::PK) / 16;
        const int c = slot ^ ((r / T::GK) % T::CPR);
        src = (t ? abase[1] : abase[0]) + (int64_t)r * a.lda + (int64_t)kt * T::BK + c * 8;
    } else {
        const int bb = blk * 1024 - T::NA * T::A_BYTES;
        const int t = bb / T::B_BYTES;
        const int lb = bb % T::B_BYTES + lane * 16;
        if constexpr (T::BT) {
            const int r = lb / 256, slot = (lb % 256) / 16;
            const int c = slot ^ ((r & 3) << 2);
            src = (t ? bbase[1] : bbase[0]) + ((int64_t)kt * T::BK + r) * a.ldb + c * 8;
        } else {
            const int r = lb / T::PK, slot = (lb % T::PK) / 16;
            const int c = slot ^ ((r / T::GK) % T::CPR);
            src = (t ? bbase[1] : bbase[0]) + (int64_t)r * a.ldb + (int64_t)kt * T::BK + c * 8;
        }
    }
    __builtin_amdgcn_global_load_lds(src, (lds_void*)(dst + blk * 1024), 16, 0, 0);
}

// All of this wave's loads of K-slice `kt` (the ring's prologue).
template <int NPASS, typename T>
__device__ __forceinline__ void load_slice(const GemmArgs& a, unsigned char* dst, int kt,
                                           const uint16_t* const (&abase)[2],
                                           const uint16_t* const (&bbase)[2], int wave, int lane) {
#pragma unroll
    for (int q = 0; q < T::IPW; ++q) load_one<NPASS, T>(a, dst, kt, abase, bbase, wave, lane, q);
}

// Wait until at most N vector-memory loads of this wave are outstanding
// (vmcnt only; lgkmcnt and expcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// B fragment (8 consecutive K of one column) from the [BK][BN] tile through
// two transposing reads; `col` is the fragment's first column.
template <typename T>
__device__ __forceinline__ bf16x8 b_frag_tr(const unsigned char* sb, int krow, int col, int lane) {
    const int g = lane >> 4, s = lane & 15;
    const int row = krow + 8 * (g >> 1) + (s >> 2);
    const int c = col + 16 * (g & 1) + 4 * (s & 3);
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(sb + nmajor_off(row, c >> 3) + 2 * (c & 7)));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(sb + nmajor_off(row + 4, c >> 3) + 2 * (c & 7)));
    typedef __attribute__((ext_vector_type(8))) short i16x8;
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// MFMAs of one BK-deep K-slice staged at `st`, fragments software-pipelined
// (k-step kk+1 is read from LDS while the MFMAs of kk run). The loads of
// slice `kn` into the stage at `ldst` are spread between the MFMAs, each
// fenced in place: issued in one burst ahead of the MFMAs they hold the
// wave in the vector-memory issue queue while its matrix pipe idles.
template <int NPASS, typename T>
__device__ __forceinline__ void mma_slice(f32x16 (&acc)[T::FM][T::FN], const unsigned char* st,
                                          int wm, int wn, int lane, const GemmArgs& a, unsigned char* ldst,
                                          int kn, const uint16_t* const (&abase)[2],
                                          const uint16_t* const (&bbase)[2], int wave) {
    const unsigned char* sa0 = st;
    const unsigned char* sa1 = st + T::A_BYTES;
    const unsigned char* sb0 = st + T::NA * T::A_BYTES;
    const unsigned char* sb1 = sb0 + T::B_BYTES;
    const int arow = wm * T::TM + (lane & 31);
    const int brow = wn * T::TN + (lane & 31);
    const int half = lane >> 5;
    constexpr int KK = T::BK / 16;
    constexpr int NM = T::FM * T::FN * NPASS;            // MFMAs per k-step
    constexpr int NL = (T::IPW + KK - 1) / KK;           // loads per k-step
    constexpr int EVERY = NM / NL > 0 ? NM / NL : 1;     // MFMAs between two loads
    using Frag = typename T::Frag;
    Frag fa0[2][T::FM], fb0[2][T::FN], fa1[2][T::FM], fb1[2][T::FN];
    int q = 0;   // next load of slice kn (compile-time after unrolling)
#pragma unroll
    for (int kk = 0; kk <= KK; ++kk) {
        if (kk < KK) {
            const int c = 2 * kk + half;   // logical 16-byte chunk of the K-major rows
            const int slot = kk & 1;
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
                fa0[slot][i] = *reinterpret_cast<const Frag*>(sa0 + kmajor_off<T>(arow + i * 32, c));
#pragma unroll
            for (int j = 0; j < T::FN; ++j) {
                if constexpr (T::BT) {
                    fb0[slot][j] = b_frag_tr<T>(sb0, kk * 16, wn * T::TN + j * 32, lane);
                } else {
                    fb0[slot][j] = *reinterpret_cast<const Frag*>(sb0 + kmajor_off<T>(brow + j * 32, c));
                }
            }
            if constexpr (NPASS >= 2) {
#pragma unroll
                for (int i = 0; i < T::FM; ++i)
                    fa1[slot][i] = *reinterpret_cast<const Frag*>(sa1 + kmajor_off<T>(arow + i * 32, c));
            }
            if constexpr (NPASS == 3) {
#pragma unroll
                for (int j = 0; j < T::FN; ++j) {
                    if constexpr (T::BT) {
                        fb1[slot][j] = b_frag_tr<T>(sb1, kk * 16, wn * T::TN + j * 32, lane);
                    } else {
                        fb1[slot][j] = *reinterpret_cast<const Frag*>(sb1 + kmajor_off<T>(brow + j * 32, c));
                    }
                }
            }
        }
        if (kk > 0) {
            const int slot = (kk - 1) & 1;
            int m = 0;
#pragma unroll
            for (int i = 0; i < T::FM; ++i)
#pragma unroll
                for (int j = 0; j < T::FN; ++j)
#pragma unroll
                    for (int p = 0; p < NPASS; ++p) {
                        // per block: hi*lo, lo*hi, then hi*hi (the order of the sums)
                        if (NPASS == 3 && p == 0) acc[i][j] = mfma32(fa0[slot][i], fb1[slot][j], acc[i][j]);
                        else if (NPASS >= 2 && p == NPASS - 2) acc[i][j] = mfma32(fa1[slot][i], fb0[slot][j], acc[i][j]);
                        else acc[i][j] = mfma32(fa0[slot][i], fb0[slot][j], acc[i][j]);
                        if (++m % EVERY == 0 && q < T::IPW && q < kk * NL) {
                            __builtin_amdgcn_sched_barrier(0);
                            load_one<NPASS, T>(a, ldst, kn, abase, bbase, wave, lane, q);
                            __builtin_amdgcn_sched_barrier(0);
                            ++q;
                        }
                    }
        }
    }
#pragma unroll
    for (; q < T::IPW; ++q) load_one<NPASS, T>(a, ldst, kn, abase, bbase, wave, lane, q);
}

// Store a wave's finished 32 x 32 block from its LDS tile (fp32, row pitch
// EPI_LD) to output rows orow0 .. orow0 + 31, columns ocol0 .. ocol0 + 31, in
// the epilogue's output form. Lanes take whole row segments: for bf16
// outputs four lanes cover a row's 64 bytes (16 rows per instruction), for
// fp32 eight lanes its 128 bytes, so every store instruction writes
// contiguous segments of few cache lines. With TR the tile is read
// transposed (output row q = tile column q), for the mirrored block; with
// DIAG (a block on the diagonal of a symmetric product) the entries below
// the diagonal are taken from their mirror images above it. O1 sends a bf16
// block to out1 instead of out0 (EPI_UPDATE's transposed copy).
template <int EPI, typename T, bool TR, bool DIAG = false, bool O1 = false>
__device__ __forceinline__ void store_block(const GemmArgs& a, int b, const float* stage, int64_t orow0,
                                            int64_t ocol0, int lane) {
    auto at = [&](int r, int c) {
        if (DIAG && c < r) return stage[c * T::EPI_LD + r];
        return TR ? stage[c * T::EPI_LD + r] : stage[r * T::EPI_LD + c];
    };
    if constexpr (EPI == EPI_FINAL) {
        const int c4 = 4 * (lane & 7);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = 8 * q + (lane >> 3);
            float* op = static_cast<float*>(a.out0) + (int64_t)b * a.sOut0 + (orow0 + r) * a.ldo0 + ocol0 + c4;
            *reinterpret_cast<float4*>(op) = make_float4(at(r, c4), at(r, c4 + 1), at(r, c4 + 2), at(r, c4 + 3));
        }
    } else {
        const int c8 = 8 * (lane & 3);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int r = 16 * q + (lane >> 2);
            float v[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) v[t] = at(r, c8 + t);
            if constexpr (EPI == EPI_SPLIT || EPI == EPI_QPOLY) {
                uint32_t h[4], l[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint16_t h0 = f32_to_bf16(v[2 * t]), h1 = f32_to_bf16(v[2 * t + 1]);
                    h[t] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                    l[t] = pack2(v[2 * t] - bf16_bits_to_f32(h0), v[2 * t + 1] - bf16_bits_to_f32(h1));
                }
                uint16_t* hp = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + (orow0 + r) * a.ldo0 + ocol0 + c8;
                uint16_t* lp = static_cast<uint16_t*>(a.out1) + (int64_t)b * a.sOut1 + (orow0 + r) * a.ldo1 + ocol0 + c8;
                *reinterpret_cast<uint4*>(hp) = make_uint4(h[0], h[1], h[2], h[3]);
                *reinterpret_cast<uint4*>(lp) = make_uint4(l[0], l[1], l[2], l[3]);
            } else if constexpr (EPI == EPI_H16 || EPI == EPI_QPOLY_H16) {
                uint16_t* op = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + (orow0 + r) * a.ldo0 + ocol0 + c8;
                *reinterpret_cast<uint4*>(op) = make_uint4(pack2h(v[0], v[1]), pack2h(v[2], v[3]),
                                                           pack2h(v[4], v[5]), pack2h(v[6], v[7]));
            } else if constexpr (O1) {   // EPI_UPDATE's transposed copy: bf16
                uint16_t* op = static_cast<uint16_t*>(a.out1) + (int64_t)b * a.sOut1 + (orow0 + r) * a.ldo1 + ocol0 + c8;
                *reinterpret_cast<uint4*>(op) = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]),
                                                           pack2(v[4], v[5]), pack2(v[6], v[7]));
            } else {   // EPI_POLY, EPI_UPDATE: bf16
                uint16_t* op = static_cast<uint16_t*>(a.out0) + (int64_t)b * a.sOut0 + (orow0 + r) * a.ldo0 + ocol0 + c8;
                *reinterpret_cast<uint4*>(op) = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]),
                                                           pack2(v[4], v[5]), pack2(v[6], v[7]));
            }
        }
    }
}

template <int NPASS, int EPI, typename T, bool SYM>
__global__ __launch_bounds__(T::THREADS) void gemm(GemmArgs a) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem_raw[T::SMEM];

    // XCD-aware tile order. Workgroups are dispatched round-robin over the
    // eight XCDs, each with its own L2; renumbering puts consecutive tiles --
    // the tiles of one matrix, which share its operands -- on one XCD, so a
    // matrix's compact operands are fetched into one L2 instead of eight.
    const int nx = gridDim.x, ny = gridDim.y;
    const int total = nx * ny * gridDim.z;
    const int hw = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    const int logical = (total % kXcds == 0) ? (hw % kXcds) * (total / kXcds) + hw / kXcds : hw;
    int b = logical / (nx * ny);
    if (a.dual) {
        // matrix b's two products are neighbours in the tile order, so the
        // shared A operand is fetched into one L2 for both
        if (b & 1) {
            a.B0 = a.B0x;
            a.B1 = a.B1x;
            a.out0 = a.out0x;
            a.out1 = a.out1x;
            a.oexp = a.oexpx;
        }
        b >>= 1;
    }
    // Within a matrix the tiles run down each column strip first: the ny
    // tiles that read one strip of the B operand are dispatched together, so
    // the strip is fetched into L2 once, while the A operand (the s x s
    // factor, the smaller one) stays resident across strips.
    int row0 = (logical % ny) * T::BM;          // output rows (M)
    int col0 = ((logical / ny) % nx) * T::BN;   // output cols (N)
    if constexpr (SYM) {
        // symmetric output: x enumerates the upper-triangle tiles I <= J
        // row by row; each is written at (I, J) and mirrored to (J, I)
        const int tiles = a.M / T::BM;
        int rem = logical % nx, I = 0;
        while (rem >= tiles - I) {
            rem -= tiles - I;
            ++I;
        }
        row0 = I * T::BM;
        col0 = (I + rem) * T::BN;
    }
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int wm = wave / T::WN, wn = wave % T::WN;

    const uint16_t* abase[2];
    const uint16_t* bbase[2];
    abase[0] = a.A0 + (int64_t)b * a.sA + (int64_t)row0 * a.lda;
    abase[1] = NPASS >= 2 ? a.A1 + (int64_t)b * a.sA + (int64_t)row0 * a.lda : abase[0];
    if constexpr (T::BT) {
        bbase[0] = a.B0 + (int64_t)b * a.sB + col0;
        bbase[1] = NPASS == 3 ? a.B1 + (int64_t)b * a.sB + col0 : bbase[0];
    } else {
        bbase[0] = a.B0 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb;
        bbase[1] = NPASS == 3 ? a.B1 + (int64_t)b * a.sB + (int64_t)col0 * a.ldb : bbase[0];
    }

    // Epilogue operands (Z for a Z, or A's hi / lo for the polynomial) are
    // fetched first so their latency hides behind the main loop.
    const int er = lane >> 1;          // epilogue: row (or transposed row) of this lane
    const int ec = (lane & 1) * 16;    // epilogue: 16 consecutive columns
    constexpr bool kPreE0 = EPI == EPI_POLY || EPI == EPI_QPOLY || EPI == EPI_UPDATE || EPI == EPI_FINAL ||
                            EPI == EPI_APPLY || EPI == EPI_QPOLY_H16 || EPI == EPI_POLY_H16;
    constexpr bool kPreE1 = EPI == EPI_POLY || EPI == EPI_QPOLY;
    const bool pre = kPreE0 && a.E0 != nullptr && !(EPI == EPI_FINAL && a.out_transposed);
    uint4 e0[T::FM][T::FN][2], e1[T::FM][T::FN][2];
    if (pre) {
#pragma unroll
        for (int i = 0; i < T::FM; ++i)
#pragma unroll
            for (int j = 0; j < T::FN; ++j) {
                const int64_t eo = (int64_t)b * a.sE + (int64_t)(row0 + wm * T::TM + i * 32 + er) * a.lde +
                                   col0 + wn * T::TN + j * 32 + ec;
                e0[i][j][0] = reinterpret_cast<const uint4*>(a.E0 + eo)[0];
                e0[i][j][1] = reinterpret_cast<const uint4*>(a.E0 + eo)[1];
                if constexpr (kPreE1) {
                    e1[i][j][0] = reinterpret_cast<const uint4*>(a.E1 + eo)[0];
                    e1[i][j][1] = reinterpret_cast<const uint4*>(a.E1 + eo)[1];
                }
            }
    }

    // EPI_APPLY: the W entries this lane updates (16 consecutive bf16 per
    // block, row K[p] of W) are fetched before the main loop as well.
    // Addresses are clamped into W so the loads are unconditional; the
    // epilogue uses them only where they are the right entries.
    int32_t wrow[T::FM];
    uint4 wv[T::FM][T::FN][2];
    if constexpr (EPI == EPI_APPLY) {
        const uint16_t* W = a.ms.w<uint16_t>(b);
#pragma unroll
        for (int i = 0; i < T::FM; ++i) {
            const int p = row0 + wm * T::TM + i * 32 + er;
            wrow[i] = ldg<int32_t>(a.sel + (int64_t)b * a.k + (p < a.k ? p : a.k - 1));
#pragma unroll
            for (int j = 0; j < T::FN; ++j) {
                int64_t jc = col0 + wn * T::TN + j * 32 + ec;
                jc = jc + 16 <= a.cols ? jc : a.cols - 16;
                const uint16_t* src = W + (int64_t)wrow[i] * a.cols + jc;
                wv[i][j][0] = ldg<uint4>(src);
                wv[i][j][1] = ldg<uint4>(src + 8);
            }
        }
    }

    f32x16 acc[T::FM][T::FN];
#pragma unroll
    for (int i = 0; i < T::FM; ++i)
#pragma unroll
        for (int j = 0; j < T::FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // S-stage ring: slices 0..S-2 in flight before the first MFMA; at
    // iteration kt slice kt+S-1 is requested into the stage freed by kt-1.
    // Requests past the last slice re-read it (in bounds) so every iteration
    // issues the same number of loads and the vmcnt wait stays exact.
    const int nk = a.K / T::BK;
#pragma unroll
    for (int p = 0; p < T::S - 1; ++p)
        load_slice<NPASS, T>(a, smem_raw + p * T::STAGE_BYTES, p < nk ? p : nk - 1, abase, bbase, wave, lane);
    for (int kt = 0; kt < nk; ++kt) {
        // This wave's part of slice kt has landed; the bare barrier then makes
        // every wave's part visible and frees stage kt-1 (its fragments were
        // consumed by MFMAs issued before the barrier). A full __syncthreads
        // would also drain the loads of the slices in flight behind kt.
        wait_vmcnt<(T::S - 2) * T::IPW>();
        __builtin_amdgcn_s_barrier();
        const int kn = kt + T::S - 1;
        mma_slice<NPASS, T>(acc, smem_raw + (kt % T::S) * T::STAGE_BYTES, wm, wn, lane, a,
                            smem_raw + (kn % T::S) * T::STAGE_BYTES, kn < nk ? kn : nk - 1, abase, bbase, wave);
    }
    wait_vmcnt<0>();   // no load may land in the ring once the epilogue reuses it
    __syncthreads();

    // ---- epilogue, one 32 x 32 block at a time through a per-wave LDS tile.
    // The tile belongs to its wave alone and LDS accesses of one wave complete
    // in issue order, so wave barriers order the staging.
    float* stage = reinterpret_cast<float*>(smem_raw) + wave * 32 * T::EPI_LD;
    // the fp16 chain's products carry power-of-two scales (exact)
    constexpr bool kScaled = T::F16 || EPI == EPI_H16;
    const float osc = kScaled ? __builtin_amdgcn_ldexpf(1.0f, a.oexp) : 1.0f;
#pragma unroll
    for (int i = 0; i < T::FM; ++i) {
#pragma unroll
        for (int j = 0; j < T::FN; ++j) {
            const int R = row0 + wm * T::TM + i * 32;   // block origin in the output
            const int Cc = col0 + wn * T::TN + j * 32;
            // A symmetric product is stored exactly symmetric: blocks above
            // the diagonal are written twice, blocks on it from their upper
            // triangle, and blocks below it (in diagonal tiles) not at all.
            // Rounding leaves the computed product slightly asymmetric;
            // carried along, that asymmetry feeds the Gram chain's unstable
            // directions.
            if (SYM && R > Cc) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                stage[m * T::EPI_LD + (lane & 31)] = kScaled ? acc[i][j][r] * osc : acc[i][j][r];
            }
            __builtin_amdgcn_wave_barrier();
            if constexpr (EPI == EPI_SPLIT || EPI == EPI_H16) {
                // no arithmetic after the accumulators: they leave the tile as staged
                if (SYM && R == Cc) {
                    store_block<EPI, T, false, true>(a, b, stage, (int64_t)R, (int64_t)Cc, lane);
                } else {
                    store_block<EPI, T, false>(a, b, stage, (int64_t)R, (int64_t)Cc, lane);
                    if (SYM) store_block<EPI, T, true>(a, b, stage, (int64_t)Cc, (int64_t)R, lane);
                }
                __builtin_amdgcn_wave_barrier();   // the stage tile is rewritten next
                continue;
            }
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
            if constexpr (EPI == EPI_UPDATE || EPI == EPI_FINAL || EPI == EPI_APPLY) {
                // + a Z at this lane's 16 entries (none when E0 is null)
                if (pre) {
                    const uint4 z0 = e0[i][j][0];
                    const uint4 z1 = e0[i][j][1];
                    const uint32_t zw[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        v[2 * q] += a.ca * bf16_bits_to_f32(zw[q] & 0xffffu);
                        v[2 * q + 1] += a.ca * bf16_bits_to_f32(zw[q] >> 16);
                    }
                } else if (transposed && a.E0) {
                    // transposed output: entry q is Z[R + ec + q][Cc + er]
                    const uint16_t* zp = a.E0 + (int64_t)b * a.sE + (int64_t)(R + ec) * a.lde + Cc + er;
#pragma unroll
                    for (int q = 0; q < 16; ++q) v[q] += a.ca * bf16_bits_to_f32(zp[(int64_t)q * a.lde]);
                }
            } else if constexpr (EPI == EPI_POLY || EPI == EPI_QPOLY) {
                // b (A_hi + A_lo) + c A^2 [+ a I]
                const uint4 h0 = e0[i][j][0];
                const uint4 h1 = e0[i][j][1];
                const uint4 l0 = e1[i][j][0];
                const uint4 l1 = e1[i][j][1];
                const uint32_t hw[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
                const uint32_t lw[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float a0 = bf16_bits_to_f32(hw[q] & 0xffffu) + bf16_bits_to_f32(lw[q] & 0xffffu);
                    const float a1 = bf16_bits_to_f32(hw[q] >> 16) + bf16_bits_to_f32(lw[q] >> 16);
                    v[2 * q] = a.cb * a0 + a.cc * v[2 * q];
                    v[2 * q + 1] = a.cb * a1 + a.cc * v[2 * q + 1];
                }
                if constexpr (EPI == EPI_QPOLY) {
                    // entry (R + er, Cc + ec + q) is on the diagonal iff er == ec + q
                    if (R == Cc) {
#pragma unroll
                        for (int q = 0; q < 16; ++q)
                            if (er == ec + q) v[q] += a.ca;
                    }
                }
            } else if constexpr (EPI == EPI_QPOLY_H16 || EPI == EPI_POLY_H16) {
                // b A + c A^2 from the fp16 A (scale 2^eexp back to A); the
                // chain's Q adds a I and is stored as fp16(2^sexp Q)
                const float esc = __builtin_amdgcn_ldexpf(1.0f, a.eexp);
                const uint4 h0 = e0[i][j][0];
                const uint4 h1 = e0[i][j][1];
                const uint32_t hw[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    v[2 * q] = a.cb * (esc * f16_bits_to_f32(hw[q] & 0xffffu)) + a.cc * v[2 * q];
                    v[2 * q + 1] = a.cb * (esc * f16_bits_to_f32(hw[q] >> 16)) + a.cc * v[2 * q + 1];
                }
                if constexpr (EPI == EPI_QPOLY_H16) {
                    const float ssc = __builtin_amdgcn_ldexpf(1.0f, a.sexp);
                    if (R == Cc) {
#pragma unroll
                        for (int q = 0; q < 16; ++q)
                            if (er == ec + q) v[q] += a.ca;
                    }
#pragma unroll
                    for (int q = 0; q < 16; ++q) v[q] *= ssc;
                }
            }
            if constexpr (EPI == EPI_APPLY) {
                // W[K[p]][j] <- bf16(W[K[p]][j] - lr_eff O[p][j]) (update step, eq. (1))
                if (orow < a.k) {
                    uint16_t* w = a.ms.w<uint16_t>(b) + (int64_t)wrow[i] * a.cols + ocol;
                    if (ocol + 16 <= a.d_oth) {
                        const uint32_t ww[8] = {wv[i][j][0].x, wv[i][j][0].y, wv[i][j][0].z, wv[i][j][0].w,
                                                wv[i][j][1].x, wv[i][j][1].y, wv[i][j][1].z, wv[i][j][1].w};
                        uint32_t o[8];
#pragma unroll
                        for (int q = 0; q < 8; ++q) {
                            const double w0 = (double)bf16_bits_to_f32(ww[q] & 0xffffu);
                            const double w1 = (double)bf16_bits_to_f32(ww[q] >> 16);
                            o[q] = (uint32_t)f64_to_bf16(__dsub_rn(w0, __dmul_rn(a.lr_eff, (double)v[2 * q]))) |
                                   ((uint32_t)f64_to_bf16(__dsub_rn(w1, __dmul_rn(a.lr_eff, (double)v[2 * q + 1]))) << 16);
                        }
                        stg(w, make_uint4(o[0], o[1], o[2], o[3]));
                        stg(w + 8, make_uint4(o[4], o[5], o[6], o[7]));
                    } else {
#pragma unroll
                        for (int q = 0; q < 16; ++q) {
                            if (ocol + q < a.d_oth) {
                                const double x = (double)bf16_bits_to_f32(ldg<uint16_t>(w + q));
                                stg(w + q, f64_to_bf16(__dsub_rn(x, __dmul_rn(a.lr_eff, (double)v[q]))));
                            }
                        }
                    }
                    if (a.dbg) {
#pragma unroll
                        for (int q = 0; q < 16; ++q)
                            if (ocol + q < a.d_oth) a.dbg[((int64_t)b * a.k + orow) * a.d_oth + ocol + q] = v[q];
                    }
                }
            } else {
                // the finished values go back to the tile (this lane's own
                // entries) and leave it in whole row segments
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int q = 0; q < 16; ++q) stage[er * T::EPI_LD + ec + q] = v[q];
                __builtin_amdgcn_wave_barrier();
                if (SYM && R == Cc) {
                    store_block<EPI, T, false, true>(a, b, stage, orow - er, ocol - ec, lane);
                } else {
                    store_block<EPI, T, false>(a, b, stage, orow - er, ocol - ec, lane);
                    if (SYM) store_block<EPI, T, true>(a, b, stage, (int64_t)Cc, (int64_t)R, lane);
                }
                if constexpr (EPI == EPI_UPDATE) {
                    // X' also as X'^T, the next step's B operand given as rows
                    if (a.out1) store_block<EPI, T, true, false, true>(a, b, stage, (int64_t)Cc, (int64_t)R, lane);
                }
            }
            __builtin_amdgcn_wave_barrier();   // the stage tile is rewritten next
        }
    }
}

// ---- the GRAM chain of a compact matrix with s <= 64, in one block
//
// The s x s matrices stay in LDS as bf16 hi / lo planes of 64 rows (pitch
// kSmallPitch entries: 144-byte rows put the 32 rows of a fragment read on
// distinct banks). Every product is the one the launch-per-product chain
// makes: per 16-deep k-step hi*lo, lo*hi, then hi*hi into fp32
// accumulators, the same epilogue arithmetic and hi / lo split, and exactly
// symmetric storage (entries on and above the diagonal computed, mirrored
// below it). Waves 0..2 take the upper 32 x 32 blocks (0,0), (0,1), (1,1);
// with s_k = 32 (KS) only the first. Entries past s_k are never read.
constexpr int kSmallPitch = 72;
constexpr int kSmallPlane = kSmallChainS * kSmallPitch;
enum { SP_A = 0, SP_Q = 2, SP_T = 4, SP_P = 6, SP_PLANES = 10 };   // hi, lo; P twice (6 and 8)

// dst[p] = x y[p] (x, y[p] symmetric, given by rows) on this wave's block
// (bi, bj), for NP products sharing x; their MFMA chains interleave, each in
// its own order. With QPOLY (NP = 1, x = y = A_t) dst = c x y + b x + a I:
// Q_t.
template <int KS, int NP, bool QPOLY>
__device__ __forceinline__ void small_products(uint16_t* pl, int x, const int (&y)[NP], const int (&dst)[NP],
                                               int bi, int bj, int lane, float ca, float cb, float cc) {
    static_assert(!QPOLY || NP == 1, "the polynomial epilogue takes one product");
    constexpr int NK = KS / 16;
    const uint16_t* xh = pl + x * kSmallPlane;
    const uint16_t* xl = xh + kSmallPlane;
    const int arow = bi * 32 + (lane & 31), brow = bj * 32 + (lane & 31);
    const int half = lane >> 5;
    auto entry = [&](int r, int& m, int& n) {
        m = bi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        n = bj * 32 + (lane & 31);
    };
    // the epilogue's A entries (QPOLY) and every fragment first, then the MFMAs
    float a0[16];
    if constexpr (QPOLY) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            int m, n;
            entry(r, m, n);
            a0[r] = bf16_bits_to_f32(xh[m * kSmallPitch + n]) + bf16_bits_to_f32(xl[m * kSmallPitch + n]);
        }
    }
    bf16x8 ah[NK], al[NK], bh[NP][NK], bl[NP][NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int kc = 16 * k + 8 * half;
        ah[k] = *reinterpret_cast<const bf16x8*>(xh + arow * kSmallPitch + kc);
        al[k] = *reinterpret_cast<const bf16x8*>(xl + arow * kSmallPitch + kc);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const uint16_t* yh = pl + y[p] * kSmallPlane;
            bh[p][k] = *reinterpret_cast<const bf16x8*>(yh + brow * kSmallPitch + kc);
            bl[p][k] = *reinterpret_cast<const bf16x8*>(yh + kSmallPlane + brow * kSmallPitch + kc);
        }
    }
    f32x16 acc[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[p][r] = 0.f;
#pragma unroll
    for (int k = 0; k < NK; ++k) {
#pragma unroll
        for (int p = 0; p < NP; ++p) acc[p] = mfma32(ah[k], bl[p][k], acc[p]);
#pragma unroll
        for (int p = 0; p < NP; ++p) acc[p] = mfma32(al[k], bh[p][k], acc[p]);
#pragma unroll
        for (int p = 0; p < NP; ++p) acc[p] = mfma32(ah[k], bh[p][k], acc[p]);
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        uint16_t* oh = pl + dst[p] * kSmallPlane;
        uint16_t* ol = oh + kSmallPlane;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            int m, n;
            entry(r, m, n);
            if (bi == bj && m > n) continue;   // below the diagonal: the mirror of (n, m)
            float v = acc[p][r];
            if constexpr (QPOLY) {
                v = cb * a0[r] + cc * v;
                if (m == n) v += ca;
            }
            const uint16_t h = f32_to_bf16(v);
            const uint16_t l = (uint16_t)(pack2(v - bf16_bits_to_f32(h), 0.f) & 0xffffu);
            oh[m * kSmallPitch + n] = h;
            ol[m * kSmallPitch + n] = l;
            if (m != n) {
                oh[n * kSmallPitch + m] = h;
                ol[n * kSmallPitch + m] = l;
            }
        }
    }
}

template <int KS>
__global__ __launch_bounds__(256) void chain_small(SmallChainArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t pl[SP_PLANES * kSmallPlane];
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t s2 = a.s_pad * a.s_pad;
    // A_0's [0, 64)^2 corner (zero past s_k) into the A planes, 16 bytes a lane
    constexpr int kChunks = kSmallChainS * (kSmallChainS / 8);   // per plane
    for (int i = tid; i < 2 * kChunks; i += 256) {
        const int plane = i / kChunks, r = (i % kChunks) / 8, c = i % 8;
        const uint16_t* src = (plane ? a.Al : a.Ah) + (int64_t)b * s2 + (int64_t)r * a.s_pad + 8 * c;
        *reinterpret_cast<uint4*>(pl + (SP_A + plane) * kSmallPlane + r * kSmallPitch + 8 * c) = ldg<uint4>(src);
    }
    __syncthreads();
    const int bi = wave == 2 ? 1 : 0, bj = wave == 0 ? 0 : 1;
    const bool active = wave == 0 || (KS > 32 && wave < 3);
    int cur = 0;
    for (int t = 0; t < a.ns_steps; ++t) {
        const float ca = a.cf[t][0], cb = a.cf[t][1], cc = a.cf[t][2];
        const int q = t == 0 ? SP_P : SP_Q;   // the first Q_t is P itself
        if (active) small_products<KS, 1, true>(pl, SP_A, {SP_A}, {q}, bi, bj, lane, ca, cb, cc);
        __syncthreads();
        // P <- Q_t P (t > 0) and T = Q_t A (t < T - 1), then A <- Q_t T
        const bool do_p = t > 0, do_t = t + 1 < a.ns_steps;
        const int pin = SP_P + 2 * cur, pout = SP_P + 2 * (1 - cur);
        if (active) {
            if (do_p && do_t) small_products<KS, 2, false>(pl, q, {pin, SP_A}, {pout, SP_T}, bi, bj, lane, 0.f, 0.f, 0.f);
            else if (do_p) small_products<KS, 1, false>(pl, q, {pin}, {pout}, bi, bj, lane, 0.f, 0.f, 0.f);
            else if (do_t) small_products<KS, 1, false>(pl, q, {SP_A}, {SP_T}, bi, bj, lane, 0.f, 0.f, 0.f);
        }
        __syncthreads();
        if (do_p) cur = 1 - cur;
        if (do_t) {
            if (active) small_products<KS, 1, false>(pl, q, {SP_T}, {SP_A}, bi, bj, lane, 0.f, 0.f, 0.f);
            __syncthreads();
        }
    }
    // P_T out: [0, s_k)^2 from LDS, zero elsewhere
    const uint16_t* ph = pl + (SP_P + 2 * cur) * kSmallPlane;
    const int64_t cpr = a.s_pad / 8;   // 16-byte chunks per row
    for (int64_t i = tid; i < 2 * a.s_pad * cpr; i += 256) {
        const int plane = (int)(i / (a.s_pad * cpr));
        const int64_t rem = i % (a.s_pad * cpr);
        const int64_t r = rem / cpr, c = rem % cpr;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (r < KS && 8 * c < KS) v = *reinterpret_cast<const uint4*>(ph + plane * kSmallPlane + r * kSmallPitch + 8 * c);
        stg((plane ? a.Pl : a.Ph) + (int64_t)b * s2 + r * a.s_pad + 8 * c, v);
    }
}

constexpr unsigned kMaxGridZ = 65535;   // the grid's z extent holds the batch

template <int NPASS, int EPI, typename T, bool SYM = false>
hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
    if (a.M % T::BM || a.N % T::BN || a.K % T::BK) return hipErrorInvalidValue;
    const unsigned per = a.dual ? 2u : 1u;
    if (SYM && (unsigned)a.batch * per > kMaxGridZ) {
        // A dual launch of more than 32767 matrices: consecutive launches
        // over slices of the batch (the symmetric products' operands and
        // outputs are all bf16 / fp16 stacks with a batch stride).
        const int chunk = (int)(kMaxGridZ / per);
        auto at = [](const void* p, int64_t elems) {
            return p ? static_cast<const uint16_t*>(p) + elems : nullptr;
        };
        for (int b0 = 0; b0 < a.batch; b0 += chunk) {
            GemmArgs c = a;
            c.batch = a.batch - b0 < chunk ? a.batch - b0 : chunk;
            c.A0 = at(a.A0, b0 * a.sA);
            c.A1 = at(a.A1, b0 * a.sA);
            c.B0 = at(a.B0, b0 * a.sB);
            c.B1 = at(a.B1, b0 * a.sB);
            c.B0x = at(a.B0x, b0 * a.sB);
            c.B1x = at(a.B1x, b0 * a.sB);
            c.E0 = at(a.E0, b0 * a.sE);
            c.E1 = at(a.E1, b0 * a.sE);
            c.out0 = const_cast<uint16_t*>(at(a.out0, b0 * a.sOut0));
            c.out1 = const_cast<uint16_t*>(at(a.out1, b0 * a.sOut1));
            c.out0x = const_cast<uint16_t*>(at(a.out0x, b0 * a.sOut0));
            c.out1x = const_cast<uint16_t*>(at(a.out1x, b0 * a.sOut1));
            const hipError_t e = launch_tile<NPASS, EPI, T, SYM>(c, s);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    const unsigned zb = (unsigned)a.batch * per;
    if (zb > kMaxGridZ) return hipErrorInvalidValue;
    dim3 grid((unsigned)(a.N / T::BN), (unsigned)(a.M / T::BM), zb);
    if (SYM) {
        if (a.M != a.N || T::BM != T::BN) return hipErrorInvalidValue;
        const unsigned tiles = (unsigned)(a.M / T::BM);
        grid = dim3(tiles * (tiles + 1) / 2, 1, zb);
    }
    hipLaunchKernelGGL((gemm<NPASS, EPI, T, SYM>), grid, dim3(T::THREADS), 0, s, a);
    return hipGetLastError();
}

}  // namespace

// A three-pass symmetric s x s product without a polynomial epilogue goes
// on 256 x 256 tiles (one block of eight waves per compute unit) when s is
// a multiple of 256 and the launch has enough of those tiles to fill the
// chip twice; otherwise on 128 x 128.
bool big_sym(const GemmArgs& a) {
    if (a.M < 1024 || a.M % 256) return false;
    const int64_t t = a.M / 256;
    return (int64_t)a.batch * (a.dual ? 2 : 1) * (t * (t + 1) / 2) >= 512;
}

// bf16 transpose through a 64 x 64 LDS tile (row pitch 66 elements, so the
// column reads spread over the banks): 16-byte row segments in and out.
__global__ __launch_bounds__(256) void transpose_bf16(const uint16_t* __restrict__ in, uint16_t* __restrict__ out,
                                                      int64_t rows, int64_t cols, int64_t stride) {
    __shared__ uint16_t t[64][66];
    const int64_t b = blockIdx.z;
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const uint16_t* src = in + b * stride + r0 * cols + c0;
    uint16_t* dst = out + b * stride + c0 * rows + r0;
    for (int i = threadIdx.x; i < 64 * 8; i += 256) {
        const int r = i >> 3, c = (i & 7) * 8;
        const uint4 v = ldg<uint4>(src + (int64_t)r * cols + c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            t[r][c + 2 * q] = (uint16_t)(w[q] & 0xffffu);
            t[r][c + 2 * q + 1] = (uint16_t)(w[q] >> 16);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 64 * 8; i += 256) {
        const int r = i >> 3, c = (i & 7) * 8;   // output row r (input column), input rows c .. c + 7
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = (uint32_t)t[c + 2 * q][r] | ((uint32_t)t[c + 2 * q + 1][r] << 16);
        stg(dst + (int64_t)r * rows + c, make_uint4(w[0], w[1], w[2], w[3]));
    }
}

hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, int npass, hipStream_t s) {
    // Tile choices measured on MI355X at the Newton-Schulz shapes. The Gram
    // matrix keeps four stages of 32-deep slices on 128 x 128 tiles, two
    // blocks of four waves per CU (64-deep slices fetch whole 128-byte lines
    // per row, but either cost blocks per CU, which slows the step whose
    // groups run side by side, or a stage in flight); from s = 1024 it runs
    // on 256 x 256 tiles.
    // The fp16 s x s products (one pass) run on 128 x 128 tiles of four
    // waves, and from s = 2048 on 256 x 256 tiles of eight (12% faster at
    // s = 2048, 24% at 4096; 13% slower at 1024).
    // The three-pass s x s products keep 128 x 128 tiles, two blocks per CU,
    // except large launches of the plain (hi / lo) products, which run on
    // 256 x 256. The X-side products use a two-stage ring, which leaves
    // room for three blocks per CU; with the update applied in the
    // epilogue eight waves per block hide more of the W traffic. Given X^T
    // as rows (b_rows) they run on 256 x 256 plain-read tiles, or 256 x 128
    // where l is not a multiple of 256 and for the fused update step.
    using TG = Tile<1, 0, 128, 128, kSliceK, 2, 2, 4>;    // Gram
    using TGL = Tile<1, 0, 256, 256, kSliceK, 4, 2, 3>;   // Gram, large s
    using TP = Tile<3, 0, 128, 128, kSliceK, 4, 2, 2>;    // three-pass symmetric products
    using TPL = Tile<3, 0, 256, 256, kSliceK, 2, 4, 2>;   // three-pass symmetric products, large s
    using TU = Tile<1, 1, 128, 128, kSliceK, 2, 2, 2>;    // update (B operand [K][N])
    using TU2 = Tile<2, 1, 128, 128, kSliceK, 2, 2, 2>;   // two-pass final product
    using TU2A = Tile<2, 1, 128, 128, kSliceK, 4, 2, 2>;  // two-pass final product applying the update
    using TU3 = Tile<3, 1, 128, 128, kSliceK, 2, 2, 2>;   // three-pass final product (fp32 master)
    using TR = Tile<1, 0, 256, 256, kSliceK, 2, 4, 3>;    // X-side products, B operand as rows (X^T)
    using TRN = Tile<1, 0, 256, 128, kSliceK, 4, 2, 4>;   // the same, l not a multiple of 256; fused update
    using TH = Tile<1, 0, 128, 128, kSliceK, 2, 2, 4, true>;   // fp16 s x s products
    using THL = Tile<1, 0, 256, 256, kSliceK, 4, 2, 3, true>;  // fp16 s x s products from s = 2048
    if (a.f16) {
        if (npass != 1) return hipErrorInvalidValue;
        const bool big = a.M >= 2048 && a.M % 256 == 0;
        if (a.dual && epi != EPI_H16) return hipErrorInvalidValue;   // the chain's P and T
        switch (epi) {
            case EPI_SPLIT:
                return big ? launch_tile<1, EPI_SPLIT, THL, true>(a, s) : launch_tile<1, EPI_SPLIT, TH, true>(a, s);
            case EPI_H16:
                return big ? launch_tile<1, EPI_H16, THL, true>(a, s) : launch_tile<1, EPI_H16, TH, true>(a, s);
            case EPI_QPOLY_H16:
                return big ? launch_tile<1, EPI_QPOLY_H16, THL, true>(a, s)
                           : launch_tile<1, EPI_QPOLY_H16, TH, true>(a, s);
            case EPI_POLY_H16:   // the Direct form's B = b A + c A^2
                return big ? launch_tile<1, EPI_POLY_H16, THL, true>(a, s)
                           : launch_tile<1, EPI_POLY_H16, TH, true>(a, s);
            default: break;
        }
        return hipErrorInvalidValue;
    }
    if (a.dual && !(epi == EPI_SPLIT && npass == 3)) return hipErrorInvalidValue;
    if (a.b_rows) {
        // the Direct form's X-side products from s = 2048: X^T as rows lets
        // them run on the wide plain-read tiles (28% faster at s = 2048, 35%
        // at 4096 than the transposing reads of the [K][N] operand)
        if (npass != 1 || a.M % 256) return hipErrorInvalidValue;
        const bool wide = a.N % 256 == 0;
        switch (epi) {
            case EPI_UPDATE:
                return wide ? launch_tile<1, EPI_UPDATE, TR>(a, s) : launch_tile<1, EPI_UPDATE, TRN>(a, s);
            case EPI_FINAL:
                return wide ? launch_tile<1, EPI_FINAL, TR>(a, s) : launch_tile<1, EPI_FINAL, TRN>(a, s);
            case EPI_APPLY:   // (its W rows spill on 256 x 256)
                if (a.cols % 8 || a.cols < 16 || a.out_transposed) break;
                return launch_tile<1, EPI_APPLY, TRN>(a, s);
            default: break;
        }
        return hipErrorInvalidValue;
    }
    switch (epi) {
        case EPI_SPLIT:
            if (npass == 3) {
                if (big_sym(a)) return launch_tile<3, EPI_SPLIT, TPL, true>(a, s);
                return launch_tile<3, EPI_SPLIT, TP, true>(a, s);
            }
            if (npass != 1) break;
            if (a.M >= 1024 && a.M % 256 == 0) return launch_tile<1, EPI_SPLIT, TGL, true>(a, s);
            return launch_tile<1, EPI_SPLIT, TG, true>(a, s);
        case EPI_H16:   // the Gram matrix of bf16 Z into the fp16 chain
            if (npass != 1) break;
            if (a.M >= 1024 && a.M % 256 == 0) return launch_tile<1, EPI_H16, TGL, true>(a, s);
            return launch_tile<1, EPI_H16, TG, true>(a, s);
        case EPI_POLY:   // (the polynomial epilogues keep 128 x 128: on 256 x 256 they spill)
            if (npass == 3) return launch_tile<3, EPI_POLY, TP, true>(a, s);
            break;
        case EPI_QPOLY:
            if (npass == 3) return launch_tile<3, EPI_QPOLY, TP, true>(a, s);
            break;
        case EPI_UPDATE:
            if (npass == 1) return launch_tile<1, EPI_UPDATE, TU>(a, s);
            break;
        case EPI_FINAL:
            if (npass == 1) return launch_tile<1, EPI_FINAL, TU>(a, s);
            if (npass == 2) return launch_tile<2, EPI_FINAL, TU2>(a, s);
            if (npass == 3) return launch_tile<3, EPI_FINAL, TU3>(a, s);
            break;
        case EPI_APPLY:
            if (a.cols % 8 || a.cols < 16 || a.out_transposed) break;
            if (npass == 1) return launch_tile<1, EPI_APPLY, TU>(a, s);
            if (npass == 2) return launch_tile<2, EPI_APPLY, TU2A>(a, s);
            if (npass == 3) return launch_tile<3, EPI_APPLY, TU3>(a, s);
            break;
        default:   // the fp16 epilogues run only with fp16 operands (above)
            break;
    }
    return hipErrorInvalidValue;
}

hipError_t launch_chain_small(const SmallChainArgs& a, hipStream_t s) {
    if (a.s_k < 32 || a.s_k > kSmallChainS || a.s_k % 32 || a.s_pad < kSmallChainS || a.s_pad % 8 ||
        a.ns_steps < 1 || a.ns_steps > kChainMaxSteps || a.batch < 1)
        return hipErrorInvalidValue;
    if (a.s_k == 32) hipLaunchKernelGGL(chain_small<32>, dim3((unsigned)a.batch), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(chain_small<64>, dim3((unsigned)a.batch), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_transpose_bf16(const uint16_t* in, uint16_t* out, int64_t rows, int64_t cols, int batch,
                                 int64_t stride, hipStream_t s) {
    if (rows < 64 || cols < 64 || rows % 64 || cols % 64 || rows / 64 > 65535 || batch < 1 || batch > 65535)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)(cols / 64), (unsigned)(rows / 64), (unsigned)batch);
    hipLaunchKernelGGL(transpose_bf16, grid, dim3(256), 0, s, in, out, rows, cols, stride);
    return hipGetLastError();
}

}  // namespace dion2
