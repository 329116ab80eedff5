// Device-side helpers and launch interfaces shared by the Dion2 kernels.
//
// Layout conventions (all row-major):
//   W, G : [rows][cols] in their storage type (bf16 or fp32), M : fp32.
//   A "line" is a row (axis = rows) or a column (axis = columns) of M / W;
//   d_sel lines exist, each of length d_oth.
//   Compact submatrix L  : [kpad][opad] bf16, row p = selected line K[p]
//                           scaled by 1 / (||M[K]||_F + eps), zero padding.
//   Its transpose     LT : [opad][kpad] bf16. Newton-Schulz iterates on the
//                           wide one of the two (L when k <= d_oth).
//   kpad, opad are k and d_oth rounded up to the GEMM tile (128); every
//   padded entry is zero, which the Newton-Schulz polynomial keeps at zero.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dion2 {

constexpr int kTile = 128;  // padding granule of the compact buffers
constexpr int kSliceK = 32;  // K depth of one slice in every GEMM tile

// A batch of same-shape matrices: either one strided stack (tables == null)
// or device-resident tables of per-matrix pointers.
struct MatSet {
    void* W;                // stack base, or unused with tables
    float* M;
    const void* G;
    int64_t stride;         // elements between consecutive matrices
    void* const* Wt;        // device tables (nullable)
    float* const* Mt;
    const void* const* Gt;

    template <typename T>
    __device__ __forceinline__ T* w(int b) const {
        return Wt ? static_cast<T*>(Wt[b]) : static_cast<T*>(W) + (int64_t)b * stride;
    }
    __device__ __forceinline__ float* m(int b) const {
        return Mt ? Mt[b] : M + (int64_t)b * stride;
    }
    template <typename T>
    __device__ __forceinline__ const T* g(int b) const {
        return Gt ? static_cast<const T*>(Gt[b]) : static_cast<const T*>(G) + (int64_t)b * stride;
    }
};

// ------------------------------------------------------- global accesses
// Pointers reached through MatSet (possibly from a device pointer table) are
// generic; these helpers access them as global memory, so the compiler emits
// global (not flat) loads and stores and waits on vmcnt alone.
#define DION2_GLOBAL __attribute__((address_space(1)))
template <int N> struct RawBits;
template <> struct RawBits<2> { typedef unsigned short T; };
template <> struct RawBits<4> { typedef unsigned int T; };
template <> struct RawBits<8> { typedef unsigned int T __attribute__((ext_vector_type(2))); };
template <> struct RawBits<16> { typedef unsigned int T __attribute__((ext_vector_type(4))); };
template <typename V>
__device__ __forceinline__ V ldg(const void* p) {
    typedef typename RawBits<sizeof(V)>::T R;
    const R r = *(const DION2_GLOBAL R*)p;
    V v;
    __builtin_memcpy(&v, &r, sizeof(V));
    return v;
}
template <typename V>
__device__ __forceinline__ void stg(void* p, const V& v) {
    typedef typename RawBits<sizeof(V)>::T R;
    R r;
    __builtin_memcpy(&r, &v, sizeof(V));
    *(DION2_GLOBAL R*)p = r;
}

// Non-temporal variants for data touched once per step (streamed past the
// caches rather than kept).
template <typename V>
__device__ __forceinline__ V ldg_nt(const void* p) {
    typedef typename RawBits<sizeof(V)>::T R;
    const R r = __builtin_nontemporal_load((const DION2_GLOBAL R*)p);
    V v;
    __builtin_memcpy(&v, &r, sizeof(V));
    return v;
}
template <typename V>
__device__ __forceinline__ void stg_nt(void* p, const V& v) {
    typedef typename RawBits<sizeof(V)>::T R;
    R r;
    __builtin_memcpy(&r, &v, sizeof(V));
    __builtin_nontemporal_store(r, (DION2_GLOBAL R*)p);
}

// ------------------------------------------------------------ conversions

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
    return __uint_as_float(h << 16);
}

// fp32 -> bf16, round to nearest even (gfx950's v_cvt_pk_bf16_f32); NaN
// stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// fp64 -> bf16 with a single round-to-nearest-even: first to fp32 with
// round-to-odd (toward zero, then the last bit forced when inexact), which
// keeps the second rounding exact because fp32 carries more than 8 + 2 bits.
// Round-to-odd is built from the hardware's nearest-even conversion: where
// that rounded away from zero the magnitude steps back one unit (the bit
// pattern minus one, also from inf to the largest finite value). A NaN
// stays a NaN. About eight vector instructions, where a directed-rounding
// conversion is emulated with some twenty.
__device__ __forceinline__ uint16_t f64_to_bf16(double d) {
    const float f = (float)d;
    const double back = (double)f;
    uint32_t u = __float_as_uint(f);
    u -= __builtin_fabs(back) > __builtin_fabs(d) ? 1u : 0u;
    u |= back != d ? 1u : 0u;
    return f32_to_bf16(__uint_as_float(u));
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float load(const float* p) { return ldg<float>(p); }
    static __device__ __forceinline__ void store_f64(float* p, double v) { stg<float>(p, (float)v); }
    // the same on an LDS copy
    static __device__ __forceinline__ float lds_load(const float* p) { return *p; }
    static __device__ __forceinline__ void lds_store_f64(float* p, double v) { *p = (float)v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p) { return bf16_bits_to_f32(ldg<uint16_t>(p)); }
    static __device__ __forceinline__ void store_f64(uint16_t* p, double v) { stg<uint16_t>(p, f64_to_bf16(v)); }
    static __device__ __forceinline__ float lds_load(const uint16_t* p) { return bf16_bits_to_f32(*p); }
    static __device__ __forceinline__ void lds_store_f64(uint16_t* p, double v) { *p = f64_to_bf16(v); }
};

// four consecutive elements as fp32 (p is 8-byte aligned for bf16, 16 for fp32)
__device__ __forceinline__ void load4(const float* p, float (&v)[4]) {
    const float4 x = ldg<float4>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
__device__ __forceinline__ void load4(const uint16_t* p, float (&v)[4]) {
    const uint2 x = ldg<uint2>(p);
    v[0] = bf16_bits_to_f32(x.x & 0xffffu); v[1] = bf16_bits_to_f32(x.x >> 16);
    v[2] = bf16_bits_to_f32(x.y & 0xffffu); v[3] = bf16_bits_to_f32(x.y >> 16);
}

// the same four values from a vector already in registers
__device__ __forceinline__ void unpack4(const float4& x, float (&v)[4]) {
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
__device__ __forceinline__ void unpack4(const uint2& x, float (&v)[4]) {
    v[0] = bf16_bits_to_f32(x.x & 0xffffu); v[1] = bf16_bits_to_f32(x.x >> 16);
    v[2] = bf16_bits_to_f32(x.y & 0xffffu); v[3] = bf16_bits_to_f32(x.y >> 16);
}

// ------------------------------------------------------- double-double sum

// Error-free transformation a + b = s + e (Knuth's TwoSum; no branch).
__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
    s = a + b;
    double bb = s - a;
    e = (a - (s - bb)) + (b - bb);
}

// (hi, lo) += (bhi, blo)
__device__ __forceinline__ void dd_add(double& hi, double& lo, double bhi, double blo) {
    double s, e;
    two_sum(hi, bhi, s, e);
    hi = s;
    lo = lo + (blo + e);
}

// ------------------------------------------------------------------ launch
// Every launcher enqueues on `stream` and returns the launch status.

struct MomentumArgs {
    MatSet ms;
    int64_t rows, cols;
    int batch;
    double* l1;        // [batch][d_sel]
    double* sq;        // [batch][d_sel]
    double* part;      // column mode partials [batch][nrb][3][cols]
    int rb_rows, nrb;  // column mode row blocking
    float mu;          // used when decay_all (M <- mu (M + G) after use)
};
hipError_t launch_momentum(const MomentumArgs& a, int axis, int g_bf16, hipStream_t s);
int64_t momentum_col_blocks(int64_t rows, int* rb_rows);

struct SelectArgs {
    const double* l1;
    const double* sq;
    int d_sel, k, batch;
    double eps;
    int32_t* sel;      // [batch][k] ascending
    double* scale;     // [batch] 1 / (sqrt(sum sq over K) + eps); not written when sq is null
    int32_t* rank;     // nullable [batch][d_sel + 1]: selected lines below i
    int rule;          // 0: largest l1 norms, 1: smallest Philox keys (Random rule)
    uint64_t seed, step;
    int64_t matrix0;   // Random rule: counter word of the batch's first matrix
};
hipError_t launch_select(const SelectArgs& a, hipStream_t s);

struct GatherArgs {
    MatSet ms;
    int64_t rows, cols;
    int batch, k, d_oth, kpad, opad;
    const int32_t* sel;
    const int32_t* rank;   // column mode: [batch][cols + 1], see SelectArgs
    const double* scale;
    float mu;
    int decay;         // 0: none, 1: M[K] <- mu M[K] here, 2: M <- mu M (column mode)
    uint16_t* L;       // nullable [batch][kpad][opad]
    uint16_t* LT;      // nullable [batch][opad][kpad] (one of L, LT is written)
    uint16_t* Llo;     // nullable: with L (LT), the lo halves bf16(x - L) of the
    uint16_t* LTlo;    // same entries, for the fp32-master Newton-Schulz
    float* O;          // nullable: fp32 copy (no Newton-Schulz step), L layout for
                       // rows, L^T layout [opad][kpad] for columns
    double* sq_part;   // columns, single pass (the Random rule: K known before M is
                       // read): scale is not read; O gets the unscaled selected
                       // columns and sq_part[batch][opad / 64][kpad] the sums of
                       // squares of each 64-row block of each selected column
};
hipError_t launch_gather(const GatherArgs& a, int axis, int g_bf16, hipStream_t s);

// The end of the single column pass: scale[b] = 1 / (sqrt(sum of sq_part over
// K's lines and the row blocks, in a fixed order) + eps), then the compact
// matrix bf16(fl32(x * fl32(scale))) from the unscaled copy Ot [opad][kpad],
// into L [kpad][opad] or LT [opad][kpad] (padded lines zero).
struct ColpassArgs {
    const float* Ot;
    double* sq_part;   // folded in place
    double* scale;
    uint16_t* L;
    uint16_t* LT;
    int batch, k, kpad, opad;
    double eps;
};
hipError_t launch_colpass_finish(const ColpassArgs& a, hipStream_t s);

struct DecayAllArgs {
    MatSet ms;
    int64_t rows, cols;
    int batch;
    float mu;
};
hipError_t launch_decay_all(const DecayAllArgs& a, hipStream_t s);

// Copy of the compact matrix (hi or lo half) as the gather left it, unpadded,
// line p in row p: out[b][p][j] for p < k, j < d_oth.
struct CompactCopyArgs {
    const uint16_t* Z;   // [batch][kpad][opad], or [batch][opad][kpad] when transposed
    uint16_t* out;       // [batch][k][d_oth]
    int batch, k, d_oth, kpad, opad;
    int transposed;
};
hipError_t launch_copy_compact(const CompactCopyArgs& a, hipStream_t s);

// Newton-Schulz GEMMs, C = A B with A given as rows [M][K]. With npass = 3
// both operands come as bf16 hi + lo pairs (A0/A1, B0/B1) and
// C = A0 B0 + A0 B1 + A1 B0; with npass = 2 only A does (C = A0 B0 + A1 B0).
//   EPI_SPLIT  (B as rows [N][K], symmetric C; npass 1 or 3):
//              out0 = bf16(C), out1 = bf16(C - out0)
//   EPI_POLY   (B as rows [N][K], npass 3): out0 = bf16(cb (E0 + E1) + cc C)
//   EPI_QPOLY  (B as rows [N][K], npass 3): Q = ca I + cb (E0 + E1) + cc C,
//              out0 = bf16(Q), out1 = bf16(Q - out0)
//   EPI_UPDATE (B as [K][N], or as rows with b_rows; npass 1):
//              out0 = bf16(ca E0 + C), and out1 = its transpose when set
//   EPI_FINAL  (B as [K][N], npass 1 to 3; as rows with b_rows, npass 1):
//              out0 = ca E0 + C in fp32 (no E0 term when E0 is null), or its
//              transpose when out_transposed
//   EPI_APPLY  (B as [K][N], npass 1 to 3; as rows with b_rows, npass 1):
//              O = ca E0 + C (row selection, O in the L layout) is not
//              stored; the update step is applied directly:
//              W[K[p]][j] <- bf16(W[K[p]][j] - lr_eff O[p][j]) for p < k,
//              j < d_oth (bf16 W, cols % 8 == 0); dbg gets O if set
//   EPI_H16    (B as rows [N][K], symmetric C; npass 1): out0 = fp16(2^oexp C)
//   EPI_QPOLY_H16 (B as rows [N][K], npass 1, fp16 operands and E0):
//              Q = ca I + cb 2^eexp E0 + cc 2^oexp C, out0 = fp16(2^sexp Q)
//   EPI_POLY_H16 (B as rows [N][K], npass 1, fp16 operands and E0):
//              out0 = bf16(cb 2^eexp E0 + cc 2^oexp C)
// With f16 set the operands are fp16 (one pass); EPI_SPLIT then stores
// 2^oexp C as the hi / lo pair. The power-of-two exponents keep the fp16
// values of the Gram-form chain clear of fp16's overflow and subnormal range.
// The symmetric products (EPI_SPLIT, EPI_POLY, EPI_QPOLY, EPI_H16,
// EPI_QPOLY_H16, EPI_POLY_H16) compute the tiles on and above the diagonal
// and mirror them.
enum GemmEpi { EPI_SPLIT = 0, EPI_POLY = 1, EPI_UPDATE = 2, EPI_FINAL = 3, EPI_QPOLY = 4,
               EPI_APPLY = 5, EPI_H16 = 6, EPI_QPOLY_H16 = 7, EPI_POLY_H16 = 8 };
struct GemmArgs {
    const uint16_t* A0; const uint16_t* A1;   // A operand(s), [M][K] ld lda
    const uint16_t* B0; const uint16_t* B1;   // B operand(s), [N][K] or [K][N], ld ldb
    int64_t sA, sB;                           // batch strides (elements)
    int M, N, K, lda, ldb;
    int batch;
    float ca, cb, cc;                         // polynomial coefficients
    // epilogue inputs / outputs (batch stride in elements, ld in elements)
    const uint16_t* E0; const uint16_t* E1; int64_t sE; int lde;  // A hi / lo, or Z
    void* out0; int64_t sOut0; int ldo0;
    void* out1; int64_t sOut1; int ldo1;
    int out_transposed;                        // EPI_FINAL: write out0[j][i]
    // X-side products (EPI_UPDATE, EPI_FINAL, EPI_APPLY): the B operand given
    // as rows [N][K] (X^T) instead of [K][N]; EPI_UPDATE then also writes the
    // transpose of its output to out1 (ld ldo1) when out1 is set
    int b_rows;
    // dual launch (EPI_SPLIT npass 3, or EPI_H16): a second product with the
    // same A operand, B = B0x/B1x into out0x/out1x (scale 2^oexpx), computed
    // in the same grid
    int dual;
    const uint16_t* B0x; const uint16_t* B1x;
    void* out0x; void* out1x;
    // fp16 Gram-form chain: fp16 operands, and the scale exponents above
    int f16;
    int oexp, oexpx, eexp, sexp;
    // EPI_APPLY only
    MatSet ms;                                 // W
    const int32_t* sel;                        // [batch][k]
    int k, d_oth;
    int64_t cols;
    double lr_eff;
    float* dbg;                                // nullable [batch][k][d_oth]
};
hipError_t launch_gemm(const GemmArgs& a, GemmEpi epi, int npass, hipStream_t s);

// The GRAM form's chain of s x s products for s <= 64 (s_k, the K extent,
// 32 or 64) in one launch, one block per matrix: A_0 in, P_T out, both as
// bf16 hi / lo pairs [batch][s_pad][s_pad]; P_T is zero outside
// [0, s_k)^2. Every product is computed as the launch-per-product chain
// computes it, so P_T is bitwise that chain's on [0, s_k)^2.
constexpr int kSmallChainS = 64;
constexpr int kChainMaxSteps = 16;   // DION2_MAX_NS_STEPS
struct SmallChainArgs {
    const uint16_t* Ah;
    const uint16_t* Al;
    uint16_t* Ph;
    uint16_t* Pl;
    int64_t s_pad;
    int s_k, ns_steps, batch;
    float cf[kChainMaxSteps][3];   // (a, b, c) per step
};
hipError_t launch_chain_small(const SmallChainArgs& a, hipStream_t s);

// out[b][j][i] = in[b][i][j] for bf16 [batch][rows][cols] stacks (both sides
// multiples of 64; `stride` elements between matrices on both sides).
hipError_t launch_transpose_bf16(const uint16_t* in, uint16_t* out, int64_t rows, int64_t cols, int batch,
                                 int64_t stride, hipStream_t s);

struct ApplyArgs {
    MatSet ms;
    int64_t rows, cols;
    int batch, k, d_oth, kpad, opad;
    const int32_t* sel;
    const int32_t* rank;   // column mode: [batch][cols + 1], see SelectArgs
    const float* O;    // [batch][kpad][opad] (rows) or [batch][opad][kpad] (columns)
    double lr_eff;     // lr * sqrt(rows / cols)
    float* dbg;        // nullable [batch][k][d_oth]
};
hipError_t launch_apply(const ApplyArgs& a, int axis, int w_bf16, hipStream_t s);

}  // namespace dion2
