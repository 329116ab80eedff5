// K2: Select_alpha -- the k lines of largest l1 norm (Default rule), or k
// lines uniformly at random (Random rule) from counter-based Philox keys.
//
// One 1024-thread block per matrix. Norms are non-negative fp64, so their
// bit patterns order like unsigned integers; NaN is mapped to +inf's pattern
// (a corrupted line ranks first and shows in W). An MSD radix select over
// the 64-bit keys, 8 bits per pass with an LDS histogram, finds the k-th
// largest key T and how many of the lines equal to T are still needed; the
// digit of each pass comes from a suffix scan of the histogram by one wave.
// Keys are cached in LDS when the matrix has at most kCache lines. A
// second sweep in index order keeps every key > T and the lowest-indexed
// keys == T (ties to the lower index) and compacts them with wave ballots
// into K, which therefore comes out ascending.
//
// The block also sums the selected lines' squared l2 norms in a fixed order
// and stores 1 / (||M[K]||_F + eps), the Newton-Schulz normalisation, and
// optionally rank[i] = the number of selected lines below i (i <= d_sel),
// which the column-mode gather uses to place line i at rank[i].
#include "dion2_device.h"

namespace dion2 {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr uint64_t kInfBits = 0x7ff0000000000000ull;
constexpr int kCache = 8192;   // lines whose keys are kept in LDS (64 KB)

// Random rule: Philox-4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011), ten
// rounds of two 32 x 32 -> 64-bit products with the halves swapped and the
// round key mixed in, the key bumped by the Weyl constants between rounds.
// The line's key is the first two output words, high first.
__device__ __forceinline__ uint64_t philox_line_key(uint32_t line, uint32_t matrix, uint64_t step,
                                                    uint64_t seed) {
    uint32_t c0 = line, c1 = matrix, c2 = (uint32_t)step, c3 = (uint32_t)(step >> 32);
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
        const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    return ((uint64_t)c0 << 32) | c1;
}

__device__ __forceinline__ uint64_t key_of(double v) {
    uint64_t u = (uint64_t)__double_as_longlong(v);
    u &= 0x7fffffffffffffffull;           // -0.0 orders as +0.0
    return u > kInfBits ? kInfBits : u;   // NaN ranks as +inf
}

// Exclusive prefix count of `flag` over the block in thread order, and the
// block total. Uses wave ballots and one LDS round.
__device__ __forceinline__ int block_excl_prefix(bool flag, int* wave_tot, int& total) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const uint64_t mask = __ballot(flag);
    const int within = __popcll(mask & ((1ull << lane) - 1ull));
    __syncthreads();   // wave_tot may still be read by the previous call
    if (lane == 0) wave_tot[wave] = __popcll(mask);
    __syncthreads();
    int before = 0;
    total = 0;
    for (int w = 0; w < kWaves; ++w) {
        const int t = wave_tot[w];
        before += (w < wave) ? t : 0;
        total += t;
    }
    return before + within;
}

__global__ __launch_bounds__(kThreads) void select_topk(SelectArgs a) {
    const int b = blockIdx.x;
    const double* __restrict__ nrm = a.l1 + (int64_t)b * a.d_sel;
    const double* __restrict__ sq = a.sq ? a.sq + (int64_t)b * a.d_sel : nullptr;
    int32_t* __restrict__ out = a.sel + (int64_t)b * a.k;
    int32_t* __restrict__ rank = a.rank ? a.rank + (int64_t)b * (a.d_sel + 1) : nullptr;

    __shared__ uint64_t cache[kCache];
    __shared__ unsigned hist[256];
    __shared__ uint64_t s_prefix;
    __shared__ int s_need;
    __shared__ int wave_tot[kWaves];
    __shared__ double red[kWaves];

    // Keys ordered so that the k largest are taken: l1 norms as they are,
    // Philox keys complemented (the k smallest keys win; equal keys stay
    // equal, so ties still go to the lower index).
    const uint32_t mtx = (uint32_t)(a.matrix0 + b);
    auto make_key = [&](int i) {
        return a.rule ? ~philox_line_key((uint32_t)i, mtx, a.step, a.seed) : key_of(nrm[i]);
    };
    const bool cached = a.d_sel <= kCache;   // uniform
    if (cached)
        for (int i = threadIdx.x; i < a.d_sel; i += kThreads) cache[i] = make_key(i);
    auto key_at = [&](int i) { return cached ? cache[i] : make_key(i); };
    const int lane = threadIdx.x & 63;

    uint64_t prefix = 0, mask = 0;
    int need = a.k;   // how many still to take at or below the current prefix
    for (int shift = 56; shift >= 0; shift -= 8) {
        if (threadIdx.x < 256) hist[threadIdx.x] = 0;
        __syncthreads();
        for (int base = 0; base < a.d_sel; base += kThreads) {
            const int i = base + threadIdx.x;
            const uint64_t key = i < a.d_sel ? key_at(i) : 0;
            const bool in = i < a.d_sel && (key & mask) == prefix;
            const unsigned digit = (unsigned)(key >> shift) & 0xffu;
            // one atomic per wave when every candidate lane has the same digit
            const uint64_t cand = __ballot(in);
            if (cand == 0) continue;
            const int first = __builtin_ctzll(cand);
            const unsigned d0 = __shfl(digit, first);
            if (__ballot(in && digit != d0) == 0) {
                if (lane == first) atomicAdd(&hist[d0], (unsigned)__popcll(cand));
            } else if (in) {
                atomicAdd(&hist[digit], 1u);
            }
        }
        __syncthreads();
        if (threadIdx.x < 64) {
            // lane l owns bins 4l .. 4l+3; above[l] = count in bins > 4l+3
            unsigned c[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) c[q] = hist[4 * lane + q];
            const unsigned own = c[0] + c[1] + c[2] + c[3];
            unsigned incl = own;   // inclusive suffix sum over lanes >= l
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const unsigned v = __shfl_down(incl, off);
                if (lane + off < 64) incl += v;
            }
            unsigned above = incl - own;
            // the digit is the largest d whose suffix count reaches `need`
#pragma unroll
            for (int q = 3; q >= 0; --q) {
                if (above < (unsigned)need && above + c[q] >= (unsigned)need) {
                    s_prefix = prefix | ((uint64_t)(4 * lane + q) << shift);
                    s_need = need - (int)above;
                }
                above += c[q];
            }
        }
        __syncthreads();
        prefix = s_prefix;
        need = s_need;
        mask |= 0xffull << shift;
    }
    // prefix == T (the k-th largest key); `need` of the keys equal to T go in.
    const uint64_t T = prefix;
    int taken = 0, ties_seen = 0;
    double fro = 0.0;
    for (int base = 0; base < a.d_sel; base += kThreads) {
        const int i = base + threadIdx.x;
        const bool valid = i < a.d_sel;
        const uint64_t key = valid ? key_at(i) : 0;
        const bool eq = valid && key == T;
        int eq_total;
        const int eq_rank = ties_seen + block_excl_prefix(eq, wave_tot, eq_total);
        const bool pick = valid && (key > T || (eq && eq_rank < need));
        int pick_total;
        const int pos = taken + block_excl_prefix(pick, wave_tot, pick_total);
        if (pick) {
            out[pos] = i;
            if (sq) fro += sq[i];
        }
        if (rank && valid) rank[i] = pos;   // selected lines before i
        taken += pick_total;
        ties_seen += eq_total;
    }
    // fixed-order reduction of the selected squared norms
    for (int off = 32; off > 0; off >>= 1) fro += __shfl_xor(fro, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = fro;
    __syncthreads();
    if (threadIdx.x == 0) {
        double f = 0.0;
        for (int w = 0; w < kWaves; ++w) f += red[w];
        if (sq) {   // a zero X with eps = 0: scale 0 (X / (||X||_F + eps) -> 0 as eps -> 0+)
            const double d = sqrt(f) + a.eps;
            a.scale[b] = d > 0.0 ? 1.0 / d : 0.0;
        }
        if (rank) rank[a.d_sel] = a.k;
    }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(select_topk, dim3((unsigned)a.batch), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace dion2
