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
// streams W by rows and reads O transposed, in one of three kernels:
//   apply_cols_sel    column count a multiple of 8 and a row of W within
//                     8 KB (the common case): one row per wave, copied into
//                     LDS, one fp64 update per selected entry per lane;
//   apply_cols_strip  wider rows: 512-column strips, the strip's slice of
//                     O^T staged in LDS, only chunks with a selected column
//                     rewritten;
//   apply_cols        other column counts: four (or one) columns per lane.
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

// Column mode, cols % 8 == 0. A block covers a strip of kStrip columns x
// kStripRows rows; lane l owns columns c .. c + 7 (c = strip + 8 l) of the
// four rows of its wave. The selected columns of a strip have consecutive
// ranks [rank[s0], rank[s1]), so the values the strip needs sit in one
// contiguous slice of each O^T row; every wave copies the slices of its own
// rows into LDS with aligned 16-byte loads (the slice start rounded down to
// a multiple of 4) and then reads O^T[r][rank[c]] from there. A chunk with
// no selected column is neither read nor written; in the others the
// unselected entries keep their bits.
constexpr int kLaneCols = 8;
constexpr int kStrip = 64 * kLaneCols;
constexpr int kStripRows = 16;
constexpr int kRowsPerWave = kStripRows / 4;
constexpr int kOtPitch = kStrip + 4;   // floats: a slice spans at most kStrip + 3

template <typename WT>
struct Chunk8;   // eight consecutive W entries
template <>
struct Chunk8<uint16_t> {
    uint4 u;
    __device__ __forceinline__ void load(const uint16_t* p) { u = ldg_nt<uint4>(p); }
    __device__ __forceinline__ void store(uint16_t* p) const { stg_nt(p, u); }
    __device__ __forceinline__ void put(uint16_t* lds) const { *reinterpret_cast<uint4*>(lds) = u; }
    __device__ __forceinline__ void get_lds(const uint16_t* lds) { u = *reinterpret_cast<const uint4*>(lds); }
    __device__ __forceinline__ float get(int v) const {
        const uint32_t w = v < 2 ? u.x : v < 4 ? u.y : v < 6 ? u.z : u.w;
        return bf16_bits_to_f32((v & 1) ? (w >> 16) : (w & 0xffffu));
    }
    __device__ __forceinline__ void set(int v, double r) {
        const uint32_t h = f64_to_bf16(r);
        uint32_t& w = v < 2 ? u.x : v < 4 ? u.y : v < 6 ? u.z : u.w;
        w = (v & 1) ? ((w & 0xffffu) | (h << 16)) : ((w & 0xffff0000u) | h);
    }
};
template <>
struct Chunk8<float> {
    float f[8];
    __device__ __forceinline__ void load(const float* p) {
        unpack4(ldg_nt<float4>(p), *reinterpret_cast<float(*)[4]>(&f[0]));
        unpack4(ldg_nt<float4>(p + 4), *reinterpret_cast<float(*)[4]>(&f[4]));
    }
    __device__ __forceinline__ void store(float* p) const {
        stg_nt(p, make_float4(f[0], f[1], f[2], f[3]));
        stg_nt(p + 4, make_float4(f[4], f[5], f[6], f[7]));
    }
    __device__ __forceinline__ void put(float* lds) const {
        reinterpret_cast<float4*>(lds)[0] = make_float4(f[0], f[1], f[2], f[3]);
        reinterpret_cast<float4*>(lds)[1] = make_float4(f[4], f[5], f[6], f[7]);
    }
    __device__ __forceinline__ void get_lds(const float* lds) {
        unpack4(reinterpret_cast<const float4*>(lds)[0], *reinterpret_cast<float(*)[4]>(&f[0]));
        unpack4(reinterpret_cast<const float4*>(lds)[1], *reinterpret_cast<float(*)[4]>(&f[4]));
    }
    __device__ __forceinline__ float get(int v) const { return f[v]; }
    __device__ __forceinline__ void set(int v, double r) { f[v] = (float)r; }
};

template <typename WT>
__global__ __launch_bounds__(kThreads) void apply_cols_strip(ApplyArgs a) {
    __shared__ __attribute__((aligned(16))) float ot[kStripRows][kOtPitch];
    const int b = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // one grid dimension: blocks run along the strips of one row block, then
    // the next row block
    const int64_t nstrips = (a.cols + kStrip - 1) / kStrip;
    const int64_t s0 = ((int64_t)blockIdx.x % nstrips) * kStrip;
    const int64_t s1 = s0 + kStrip < a.cols ? s0 + kStrip : a.cols;
    const int64_t r0 = ((int64_t)blockIdx.x / nstrips) * kStripRows;
    const int32_t* __restrict__ rank = a.rank + (int64_t)b * (a.cols + 1);
    WT* __restrict__ W = a.ms.w<WT>(b);
    const float* __restrict__ OT = a.O + (int64_t)b * a.opad * a.kpad;

    // ranks of this lane's columns (clamped past the strip: no column)
    const int64_t c = s0 + kLaneCols * lane;
    int rk[kLaneCols + 1];
#pragma unroll
    for (int v = 0; v <= kLaneCols; ++v) rk[v] = ldg<int32_t>(rank + (c < s1 ? c + v : s1));
    unsigned m = 0;
#pragma unroll
    for (int v = 0; v < kLaneCols; ++v) m |= (rk[v + 1] > rk[v] ? 1u : 0u) << v;

    // this wave's rows (past the matrix: its last row, never stored)
    int64_t rr[kRowsPerWave];
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
        const int64_t r = r0 + wave + 4 * i;
        rr[i] = r < a.rows ? r : a.rows - 1;
    }
    Chunk8<WT> w[kRowsPerWave];
    if (m) {
#pragma unroll
        for (int i = 0; i < kRowsPerWave; ++i) w[i].load(W + rr[i] * a.cols + c);
    }

    // the strip's O^T slices of this wave's rows into LDS
    const int R0 = ldg<int32_t>(rank + s0) & ~3;
    const int R1 = ldg<int32_t>(rank + s1);
    const int nq = (R1 - R0 + 3) >> 2;   // 16-byte pieces per row; R0 + 4 nq <= kpad
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
        const float* src = OT + rr[i] * a.kpad + R0;
        float* dst = &ot[wave + 4 * i][0];
        for (int q = lane; q < nq; q += 64) {
            const float4 x = ldg<float4>(src + 4 * q);
            *reinterpret_cast<float4*>(dst + 4 * q) = x;
        }
    }
    // LDS accesses of one wave complete in issue order: no block barrier
    __builtin_amdgcn_wave_barrier();
    if (!m) return;

#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
        const int64_t r = r0 + wave + 4 * i;
        if (r >= a.rows) break;
        const float* o = &ot[wave + 4 * i][0];
#pragma unroll
        for (int v = 0; v < kLaneCols; ++v) {
            if (m & (1u << v)) {
                const float ov = o[rk[v] - R0];
                w[i].set(v, __dsub_rn((double)w[i].get(v), __dmul_rn(a.lr_eff, (double)ov)));
                if (a.dbg) a.dbg[((int64_t)b * a.k + rk[v]) * a.d_oth + r] = ov;
            }
        }
        w[i].store(W + r * a.cols + c);
    }
}

// Column mode, cols % 8 == 0 and a row of W within 8 KB: whole
// rows per wave, the arithmetic spread over the selected entries rather
// than over the columns. A wave copies its row of W into LDS (16-byte
// chunks), lane l updates there the entries of ranks p = l + 64 t (column
// K[p], value O^T[r][p], read coalesced), and the row goes back to W whole.
// Every lane does the same number of updates, so nothing diverges; K is
// staged in LDS once per block. The first 64 KT ranks of a row are fetched
// with the row (one row ahead); larger k take further passes of 64 KT.
constexpr int kSelRows = 32;                 // rows per block (8 per wave)
constexpr int kSelRowBytes = 8192;           // LDS row buffer per wave
constexpr int kSelMaxK = 4096;               // k <= cols <= 4096 (bf16) or 2048 (fp32)

template <typename WT, int NCH, int KT>
__global__ __launch_bounds__(kThreads) void apply_cols_sel(ApplyArgs a) {
    __shared__ __attribute__((aligned(16))) WT row_s[4][kSelRowBytes / sizeof(WT)];
    extern __shared__ int32_t sel_s[];   // k entries (dynamic: k * 4 bytes)
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    {
        const int32_t* sel = a.sel + (int64_t)b * a.k;
        for (int i0 = 0; i0 < a.k; i0 += 4 * kThreads) {
            int32_t t[4];   // four loads in flight before the LDS writes
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = i0 + threadIdx.x + q * kThreads;
                t[q] = ldg<int32_t>(sel + (i < a.k ? i : a.k - 1));
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = i0 + threadIdx.x + q * kThreads;
                if (i < a.k) sel_s[i] = t[q];
            }
        }
    }
    __syncthreads();

    WT* __restrict__ W = a.ms.w<WT>(b);
    const float* __restrict__ OT = a.O + (int64_t)b * a.opad * a.kpad;
    WT* rs = row_s[wave];
    int coff[NCH];   // this lane's chunks; past the row end: clamped, unused
    bool cval[NCH];
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int c = kLaneCols * (lane + 64 * j);
        cval[j] = c < a.cols;
        coff[j] = cval[j] ? c : (int)a.cols - kLaneCols;
    }
    // Software pipelined over the wave's rows: the loads of the next row are
    // issued before the stores of this one. Vector memory counters retire in
    // issue order, so a wait for loads issued after a row's stores would also
    // wait for those stores to be acknowledged; issued before them, it does
    // not. The last row's "next" loads re-read that row, unused.
    auto load_row = [&](int64_t r, Chunk8<WT> (&w)[NCH], float (&o)[KT]) {
#pragma unroll
        for (int j = 0; j < NCH; ++j) w[j].load(W + r * a.cols + coff[j]);
        const float* src = OT + r * a.kpad;
#pragma unroll
        for (int t = 0; t < KT; ++t) {
            const int p = lane + 64 * t;
            o[t] = ldg<float>(src + (p < a.k ? p : a.k - 1));
        }
    };
    const int64_t r_end = (int64_t)(blockIdx.x + 1) * kSelRows < a.rows ? (int64_t)(blockIdx.x + 1) * kSelRows
                                                                         : a.rows;
    int64_t r = (int64_t)blockIdx.x * kSelRows + wave;
    if (r >= r_end) return;   // whole wave; no block barrier follows
    Chunk8<WT> w[NCH], wn[NCH];
    float o[KT], on[KT];
    load_row(r, w, o);
    for (; r < r_end; r += 4) {
        load_row(r + 4 < r_end ? r + 4 : r, wn, on);
#pragma unroll
        for (int j = 0; j < NCH; ++j)
            if (cval[j]) w[j].put(rs + coff[j]);
        // LDS accesses of one wave complete in issue order
        __builtin_amdgcn_wave_barrier();
        auto update = [&](int p, float ov) {
            if (p < a.k) {
                WT* e = rs + sel_s[p];
                Elem<WT>::lds_store_f64(e, __dsub_rn((double)Elem<WT>::lds_load(e), __dmul_rn(a.lr_eff, (double)ov)));
                if (a.dbg) a.dbg[((int64_t)b * a.k + p) * a.d_oth + r] = ov;
            }
        };
#pragma unroll
        for (int t = 0; t < KT; ++t) update(lane + 64 * t, o[t]);
        for (int p0 = 64 * KT; p0 < a.k; p0 += 64 * 8) {   // k > 64 KT only
            const float* src = OT + r * a.kpad;
            float ox[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int p = p0 + lane + 64 * t;
                ox[t] = ldg<float>(src + (p < a.k ? p : a.k - 1));
            }
#pragma unroll
            for (int t = 0; t < 8; ++t) update(p0 + lane + 64 * t, ox[t]);
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            if (cval[j]) {
                w[j].get_lds(rs + coff[j]);
                w[j].store(W + r * a.cols + coff[j]);
            }
        }
        __builtin_amdgcn_wave_barrier();   // the row buffer is rewritten next
#pragma unroll
        for (int j = 0; j < NCH; ++j) w[j] = wn[j];
#pragma unroll
        for (int t = 0; t < KT; ++t) o[t] = on[t];
    }
}

template <typename WT, int NCH>
void launch_cols_sel_k(const ApplyArgs& a, hipStream_t s) {
    dim3 grid((unsigned)((a.rows + kSelRows - 1) / kSelRows), (unsigned)a.batch);
    const size_t lds = (size_t)a.k * sizeof(int32_t);   // K's copy; the row buffers are static
    if (a.k <= 256) hipLaunchKernelGGL((apply_cols_sel<WT, NCH, 4>), grid, dim3(kThreads), lds, s, a);
    else if (a.k <= 512) hipLaunchKernelGGL((apply_cols_sel<WT, NCH, 8>), grid, dim3(kThreads), lds, s, a);
    else hipLaunchKernelGGL((apply_cols_sel<WT, NCH, 16>), grid, dim3(kThreads), lds, s, a);
}

template <typename WT>
bool launch_cols_sel(const ApplyArgs& a, hipStream_t s) {
    constexpr int64_t kMaxCols = kSelRowBytes / sizeof(WT);
    if (a.cols % kLaneCols || a.cols > kMaxCols || a.k > kSelMaxK) return false;
    const int64_t nch = (a.cols + kStrip - 1) / kStrip;
    if (nch <= 1) launch_cols_sel_k<WT, 1>(a, s);
    else if (nch <= 2) launch_cols_sel_k<WT, 2>(a, s);
    else if (nch <= 4) launch_cols_sel_k<WT, 4>(a, s);
    else if constexpr (kMaxCols > 2048) launch_cols_sel_k<WT, 8>(a, s);
    else return false;
    return true;
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
    } else if (w_bf16 ? launch_cols_sel<uint16_t>(a, s) : launch_cols_sel<float>(a, s)) {
        // whole rows per wave, one update per selected entry
    } else if (a.cols % kLaneCols == 0) {
        const int64_t blocks = (a.cols + kStrip - 1) / kStrip * ((a.rows + kStripRows - 1) / kStripRows);
        dim3 grid((unsigned)blocks, 1, (unsigned)a.batch);
        if (w_bf16) hipLaunchKernelGGL((apply_cols_strip<uint16_t>), grid, dim3(kThreads), 0, s, a);
        else hipLaunchKernelGGL((apply_cols_strip<float>), grid, dim3(kThreads), 0, s, a);
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
