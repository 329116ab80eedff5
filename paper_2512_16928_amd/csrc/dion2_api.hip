// Host side of the Dion2 C ABI: argument validation, planning, workspace
// management and the launch sequence of one step (Algorithm 1):
//
//   K1 momentum + line norms -> K2 top-k select -> K3 gather + decay
//   -> K4 Newton-Schulz, DIRECT: ns_steps x (Gram split -> A^2 combine -> a Z + B Z)
//                        GRAM:   Gram split -> ns_steps x (s x s products) -> P Z
//   -> K5 scatter-apply
//
// Nothing here computes part of the step on the host; the host only decides
// shapes, carves the workspace and enqueues kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "dion2.h"
#include "dion2_device.h"

using namespace dion2;

namespace {

thread_local std::string g_last_error = "no error";

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(DION2_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr float kMuonQuintic[3] = {3.4445f, -4.7750f, 2.0315f};
constexpr int64_t kMaxDim = int64_t(1) << 20;

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Plan {
    int axis;                 // resolved: 0 rows, 1 columns
    int64_t rows, cols;
    int64_t d_sel, d_oth, k;
    int64_t kpad, opad;
    bool z_is_L;              // Newton-Schulz iterates on L (k <= d_oth) or L^T
    int64_t s_pad, l_pad;
    int64_t s_k, l_k;         // K extents of the s- and l-deep products (see make_plan)
    int batch;
    int nrb, rb_rows;         // column-mode reduction blocking
    bool gram;                // Newton-Schulz on s x s matrices (DION2_NS_GRAM)
    bool master;              // X kept as a hi / lo pair (DION2_MASTER_FP32; implies gram)
    bool xrows;               // DIRECT from s = 2048: X also kept as X^T for the update's B operand
    bool colpass;             // columns under the Random rule: one pass over M and G (see front)
    // workspace offsets
    size_t o_l1, o_sq, o_part, o_sel, o_rank, o_scale, o_Z, o_Z1, o_ZT, o_sqp, o_S, S_bytes, o_O, o_tables,
        total;
};

// s x s buffers of the two Newton-Schulz forms (bf16 [batch][s_pad][s_pad])
enum { SQ_AHI, SQ_ALO, SQ_B, SQ_DIRECT_COUNT = 3 };
enum { SQ_QHI = 2, SQ_QLO, SQ_THI, SQ_TLO, SQ_P0HI, SQ_P0LO, SQ_P1HI, SQ_P1LO, SQ_GRAM_COUNT };

// The DIRECT form rounds X to bf16 after every step, so its distance from
// the exact iteration grows with the step count. An emulation of its bf16
// arithmetic on the compact shapes it is chosen for (near-square, from
// 80 x 640 to 1024 x 2048) put the relative Frobenius error of O at up to
// 1.2e-2 after 5 steps, 1.6e-2 after 6, 1.8e-2 after 7 and 2.1e-2 after 8.
// Beyond DION2_DIRECT_MAX_STEPS AUTO takes the GRAM form, which carries the
// iteration in hi / lo pairs, and a forced DIRECT is refused.
constexpr int kDirectMaxSteps = DION2_DIRECT_MAX_STEPS;
static_assert(kChainMaxSteps == DION2_MAX_NS_STEPS, "the fused chain's coefficient table");

// own_sq = false leaves out the s x s buffers (a grouped call carves them
// once for every group of a shared Newton-Schulz chain).
int make_plan(int batch, int64_t rows, int64_t cols, float alpha, int axis, int ns_form, int ns_steps,
              Plan* p, bool own_sq = true, bool master = false, bool random_rule = false) {
    if (batch < 1 || batch > 65535) return fail(DION2_ERR_INVALID_ARG, "batch %d not in [1, 65535]", batch);
    if (rows < 1 || cols < 1)
        return fail(DION2_ERR_INVALID_ARG, "rows (%lld) and cols (%lld) must be >= 1",
                    (long long)rows, (long long)cols);
    if (rows > kMaxDim || cols > kMaxDim || rows * cols >= (int64_t(1) << 31))
        return fail(DION2_ERR_UNSUPPORTED, "matrix %lld x %lld exceeds the supported size",
                    (long long)rows, (long long)cols);
    if (!std::isfinite(alpha) || !(alpha > 0.f) || alpha > 1.f)
        return fail(DION2_ERR_INVALID_ARG, "alpha %g not in (0, 1]", (double)alpha);
    if (axis != DION2_AXIS_AUTO && axis != DION2_AXIS_ROWS && axis != DION2_AXIS_COLS)
        return fail(DION2_ERR_INVALID_ARG, "axis %d is not AUTO, ROWS or COLS", axis);
    if (ns_form != DION2_NS_AUTO && ns_form != DION2_NS_DIRECT && ns_form != DION2_NS_GRAM)
        return fail(DION2_ERR_INVALID_ARG, "ns_form %d is not AUTO, DIRECT or GRAM", ns_form);
    if (ns_form == DION2_NS_DIRECT && ns_steps > kDirectMaxSteps)
        return fail(DION2_ERR_UNSUPPORTED,
                    "ns_form DIRECT takes at most %d Newton-Schulz steps (%d given): its bf16 "
                    "rounding of X after every step grows past the 2e-2 accuracy bound",
                    kDirectMaxSteps, ns_steps);
    Plan& P = *p;
    P.axis = axis == DION2_AXIS_AUTO ? (rows <= cols ? 0 : 1) : axis;
    P.rows = rows;
    P.cols = cols;
    P.d_sel = P.axis == 0 ? rows : cols;
    P.d_oth = P.axis == 0 ? cols : rows;
    int64_t k = (int64_t)std::ceil((double)alpha * (double)P.d_sel);
    P.k = k < 1 ? 1 : (k > P.d_sel ? P.d_sel : k);
    P.kpad = round_up(P.k, kTile);
    P.opad = round_up(P.d_oth, kTile);
    P.z_is_L = P.k <= P.d_oth;
    P.s_pad = P.z_is_L ? P.kpad : P.opad;
    P.l_pad = P.z_is_L ? P.opad : P.kpad;
    // Every s x s matrix of either form is block diagonal, the s x s block
    // and the padding (Z's padding rows are zero; only Q's a I reaches the
    // padding's diagonal), so a product whose inner dimension is s or l
    // sums only to the real side, rounded up to the 32-deep K slice: the
    // terms left out are exact zeros in every real entry. (MoE experts:
    // s = 352 padded to 384, one slice in twelve.)
    P.s_k = round_up(P.z_is_L ? P.k : P.d_oth, kSliceK);
    P.l_k = round_up(P.z_is_L ? P.d_oth : P.k, kSliceK);
    // With a compact matrix of one tile a side the DIRECT form's bf16
    // rounding of X after every step lands on a few directions: an emulation
    // of its arithmetic put O up to 3.6e-2 from the exact iteration after 5
    // steps (s = 3) and 2.2e-2 after 6 (s = 32), against 1.4e-2 from s = 128
    // on. AUTO takes GRAM there at the same cost; a forced DIRECT is refused.
    if (ns_form == DION2_NS_DIRECT && P.s_pad <= kTile)
        return fail(DION2_ERR_UNSUPPORTED,
                    "ns_form DIRECT needs a compact matrix of more than %d lines a side (s = %lld): on "
                    "one tile its bf16 rounding of X after every step can exceed the 2e-2 accuracy "
                    "bound; the GRAM form, which AUTO takes there, costs the same",
                    kTile, (long long)(P.z_is_L ? P.k : P.d_oth));
    // The GRAM form trades 2 (s x l) GEMMs and the X traffic of every step
    // for about four three-pass s x s products; it pays once X is wide. With
    // a single tile a side (s <= 128) both forms cost a few microseconds of
    // launches, and GRAM, which keeps the iterate in hi / lo pairs, is the
    // more accurate one.
    P.gram = ns_form == DION2_NS_GRAM ||
             (ns_form == DION2_NS_AUTO &&
              (P.l_pad >= 3 * P.s_pad || P.s_pad <= kTile || ns_steps > kDirectMaxSteps));
    // the fp32 master runs in the GRAM order (its caller rejects a forced DIRECT)
    P.master = master;
    if (master) P.gram = true;
    // DIRECT's update B X on the plain-read 256-row tiles needs X^T as rows;
    // it pays from s = 2048 (below, the transposes cost more than they save)
    P.xrows = !P.gram && P.s_pad >= 2048 && P.s_pad % 256 == 0;
    // The Random rule draws K before M is read, so column selection can form
    // M + G, decay and gather in one pass instead of a norm pass and a second
    // read; the compact matrix is normalised once every row is in.
    P.colpass = random_rule && P.axis == 1 && !P.master && ns_steps > 0;
    P.batch = batch;
    P.nrb = P.axis == 1 ? (int)momentum_col_blocks(rows, &P.rb_rows) : 0;
    if (P.axis == 0) P.rb_rows = 0;

    const size_t B = (size_t)batch;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    P.o_l1 = take(B * P.d_sel * 8);
    P.o_sq = take(B * P.d_sel * 8);
    P.o_part = take(P.axis == 1 ? B * P.nrb * 3 * (size_t)cols * 8 : 0);
    P.o_sel = take(B * P.k * 4);
    P.o_rank = take(P.axis == 1 ? B * (size_t)(P.d_sel + 1) * 4 : 0);
    P.o_scale = take(B * 8);
    const size_t comp = B * (size_t)P.kpad * (size_t)P.opad * 2;
    P.o_Z = take(comp);
    P.o_Z1 = take(P.gram && !P.master ? 0 : comp);   // DIRECT's ping-pong copy, or the lo half of X
    P.o_ZT = take(P.xrows ? 2 * comp : 0);            // DIRECT's X^T, ping-pong
    P.o_sqp = take(P.colpass ? B * (size_t)(P.opad / 64) * (size_t)P.kpad * 8 : 0);
    P.S_bytes = align256(B * (size_t)P.s_pad * (size_t)P.s_pad * 2);
    P.o_S = take(own_sq ? P.S_bytes * (P.gram ? SQ_GRAM_COUNT : SQ_DIRECT_COUNT) : 0);
    P.o_O = take(B * (size_t)P.kpad * (size_t)P.opad * 4);
    P.o_tables = take(3 * B * sizeof(void*));
    P.total = off;
    return DION2_OK;
}

// ------------------------------------------------------------- workspaces

// Pinned host staging for one call's pointer tables. The copy to the device
// reads it after the call has returned, so a slot is reused only once the
// event recorded behind that copy has completed.
struct TableSlot {
    void** host = nullptr;
    size_t count = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
};
constexpr int kTableSlots = 8;

struct Workspace {
    void* dev = nullptr;
    size_t bytes = 0;
    TableSlot slots[kTableSlots];  // pointer-table staging, used round-robin
    int next_slot = 0;
    std::vector<hipStream_t> aux;  // grouped calls: streams the groups run on
    std::vector<hipEvent_t> ev;    // grouped calls: fork / dependency / join events
    std::mutex use;                // serialises host threads sharing a stream
};

// At least n auxiliary streams (default priority) and m events.
int ensure_aux(Workspace* w, int n, int m) {
    while ((int)w->aux.size() < n) {
        hipStream_t s = nullptr;
        hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "hipStreamCreateWithFlags");
        w->aux.push_back(s);
    }
    while ((int)w->ev.size() < m) {
        hipEvent_t ev = nullptr;
        hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
        w->ev.push_back(ev);
    }
    return DION2_OK;
}

std::mutex g_ws_mutex;
std::map<std::pair<int, hipStream_t>, Workspace*> g_ws;

Workspace* workspace_for(int dev, hipStream_t s) {
    std::lock_guard<std::mutex> lk(g_ws_mutex);
    auto& w = g_ws[{dev, s}];
    if (!w) w = new Workspace();
    return w;
}

int ensure_device(Workspace* w, size_t bytes) {
    if (w->bytes >= bytes) return DION2_OK;
    if (w->dev) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize before workspace growth");
        e = hipFree(w->dev);
        w->dev = nullptr;
        w->bytes = 0;
        if (e != hipSuccess) return hip_fail(e, "hipFree(workspace)");
    }
    hipError_t e = hipMalloc(&w->dev, bytes);
    if (e != hipSuccess) {
        w->dev = nullptr;
        return fail(DION2_ERR_WORKSPACE, "hipMalloc of %zu workspace bytes failed: %s", bytes,
                    hipGetErrorString(e));
    }
    w->bytes = bytes;
    return DION2_OK;
}

// -------------------------------------------------------------- profiler

struct ProfRecord {
    int phase;
    hipEvent_t start, stop;
    double flops, bytes;
    int launches;
};

struct Profiler {
    std::mutex mu;
    bool on = false;
    std::vector<ProfRecord> pending;
    std::vector<hipEvent_t> pool;
    double ms[DION2_PHASE_COUNT] = {};
    int64_t calls[DION2_PHASE_COUNT] = {};
    int64_t launches[DION2_PHASE_COUNT] = {};
    double flops[DION2_PHASE_COUNT] = {};
    double bytes[DION2_PHASE_COUNT] = {};

    hipEvent_t get() {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
};

Profiler g_prof;

// Set for the duration of an allocation-free call: its phases are not timed
// (the hooks create HIP events on demand).
thread_local bool t_no_alloc = false;

// Brackets one kernel phase with events when the hooks are on.
class PhaseTimer {
  public:
    PhaseTimer(int phase, double flops, double bytes, int launches, hipStream_t s) : s_(s) {
        if (t_no_alloc) return;
        std::lock_guard<std::mutex> lk(g_prof.mu);
        if (!g_prof.on) return;
        rec_.phase = phase;
        rec_.flops = flops;
        rec_.bytes = bytes;
        rec_.launches = launches;
        rec_.start = g_prof.get();
        rec_.stop = g_prof.get();
        if (rec_.start && rec_.stop && hipEventRecord(rec_.start, s) == hipSuccess) active_ = true;
    }
    void finish(bool ok) {
        if (!active_) return;
        std::lock_guard<std::mutex> lk(g_prof.mu);
        if (ok && hipEventRecord(rec_.stop, s_) == hipSuccess) {
            g_prof.pending.push_back(rec_);
        } else {
            g_prof.pool.push_back(rec_.start);
            g_prof.pool.push_back(rec_.stop);
        }
        active_ = false;
    }

  private:
    hipStream_t s_;
    ProfRecord rec_{};
    bool active_ = false;
};

template <typename F>
hipError_t timed(int phase, double flops, double bytes, int launches, hipStream_t s, F&& fn) {
    PhaseTimer t(phase, flops, bytes, launches, s);
    hipError_t e = fn();
    t.finish(e == hipSuccess);
    return e;
}

// ------------------------------------------------------ Newton-Schulz

// Storage of the GRAM form's s x s matrices. Every one of them is a
// polynomial in A_0 = Z Z^T, so its eigenvalues follow the scalar iteration
// x_{t+1} = x_t q_t(x_t)^2, q_t(x) = a + b x + c x^2, from A_0's
// eigenvalues, which lie in [0, ||Z||_F^2] = [0, 1] up to rounding; an entry
// of a symmetric matrix is at most its spectral norm. Scanning x_0 over
// [0, 1.0625] bounds A_t, Q_t = q_t(A_t), T_t = Q_t A_t and the partial
// products P_t = Q_{t-1} ... Q_0. In the fp16 form each kind is stored as
// fp16(2^e X), e chosen so that its bound lands at 2^14 or below: four times
// under fp16's largest finite value, and entries down to 2^-28 of the bound
// stay clear of fp16's subnormal range.
struct ChainFmt {
    bool f16 = false;
    int eA = 0, eQ = 0, eT = 0, eP = 0;
};

bool chain_bounds(const float* coeffs, int ns_steps, ChainFmt* f) {
    double mA = 1.0625, mQ = 0.0, mT = 0.0, mP = 0.0;
    constexpr int kGrid = 2048;
    for (int i = 0; i <= kGrid; ++i) {
        double x = 1.0625 * i / kGrid, p = 1.0;
        for (int t = 0; t < ns_steps; ++t) {
            const float* cf = coeffs ? coeffs + 3 * t : kMuonQuintic;
            const double q = (double)cf[0] + (double)cf[1] * x + (double)cf[2] * x * x;
            mQ = std::fmax(mQ, std::fabs(q));
            mT = std::fmax(mT, std::fabs(q * x));
            p *= q;
            x *= q * q;
            if (t + 1 < ns_steps) {   // the last P is written as a hi / lo pair
                mP = std::fmax(mP, std::fabs(p));
                mA = std::fmax(mA, std::fabs(x));
            }
        }
    }
    auto expo = [](double m, int* e) {
        if (!std::isfinite(m) || m > 0x1p40) return false;
        *e = m < 0x1p-26 ? 40 : (int)std::floor(std::log2(16384.0 / m));
        return true;
    };
    return expo(mA, &f->eA) && expo(mQ, &f->eQ) && expo(mT, &f->eT) && expo(mP, &f->eP);
}

// The DIRECT form keeps A_t = X_t X_t^T in fp16, as fp16(2^e A_t). A_t is
// positive semidefinite, so its entries are bounded by its largest
// eigenvalue x_t, the squared largest singular value of X_t; that follows
// x_{t+1} = x_t q_t(x_t)^2 from x_0 in [0, 1.0625] (X_0 is the bf16 rounding
// of a matrix of unit Frobenius norm). e puts the bound of every A_t at or
// below 2^14, a quarter of fp16's largest value, which leaves room for
// rounding; A_t^2 then accumulates in fp32 at scale 2^(2e). false when the
// coefficients take the bound beyond 2^40: the form then keeps A as a bf16
// hi / lo pair with three passes for A^2.
bool direct_a_exp_scan(const float* coeffs, int ns_steps, int* e) {
    double mA = 1.0625;
    constexpr int kGrid = 2048;
    for (int i = 0; i <= kGrid; ++i) {
        double x = 1.0625 * i / kGrid;
        for (int t = 0; t + 1 < ns_steps; ++t) {
            const float* cf = coeffs ? coeffs + 3 * t : kMuonQuintic;
            const double q = (double)cf[0] + (double)cf[1] * x + (double)cf[2] * x * x;
            x *= q * q;
            mA = std::fmax(mA, std::fabs(x));
        }
    }
    if (!std::isfinite(mA) || mA > 0x1p40) return false;
    *e = (int)std::floor(std::log2(16384.0 / mA));
    return true;
}

bool direct_a_exp(const float* coeffs, int ns_steps, int* e) {
    if (coeffs) return direct_a_exp_scan(coeffs, ns_steps, e);
    static const std::vector<int> tab = [] {
        std::vector<int> v(DION2_MAX_NS_STEPS + 1, 0);
        for (int n = 0; n <= DION2_MAX_NS_STEPS; ++n) direct_a_exp_scan(nullptr, n, &v[n]);
        return v;
    }();
    *e = tab[ns_steps];
    return true;
}

// dion2_options.ns_chain resolved for a call: fp16 for chains of two or more
// steps when asked for.
int chain_format(const dion2_options& opt, int ns_steps, ChainFmt* f) {
    *f = ChainFmt{};
    if (opt.ns_chain != DION2_CHAIN_HILO && opt.ns_chain != DION2_CHAIN_F16)
        return fail(DION2_ERR_INVALID_ARG, "ns_chain %d is not HILO or F16", opt.ns_chain);
    if (opt.ns_chain != DION2_CHAIN_F16 || ns_steps < 2) return DION2_OK;
    ChainFmt g;
    if (opt.ns_coeffs) {
        if (!chain_bounds(opt.ns_coeffs, ns_steps, &g))
            return fail(DION2_ERR_UNSUPPORTED,
                        "ns_chain F16: these coefficients take the chain's values beyond fp16's range");
    } else {
        static const std::vector<ChainFmt> tab = [] {
            std::vector<ChainFmt> v(DION2_MAX_NS_STEPS + 1);
            for (int n = 0; n <= DION2_MAX_NS_STEPS; ++n) chain_bounds(nullptr, n, &v[n]);
            return v;
        }();
        g = tab[ns_steps];
    }
    g.f16 = true;
    *f = g;
    return DION2_OK;
}

// Z is the wide orientation [s_pad][l_pad] of the compact matrix; O receives
// the result in the L layout [kpad][opad] (the transpose when Z is L^T).

double sym_flops(double s, double inner) { return s * (s + 1.0) * inner; }

GemmArgs gram_args(const Plan& P, const uint16_t* Z, uint16_t* hi, uint16_t* lo) {
    GemmArgs g{};
    g.batch = P.batch;
    g.A0 = g.B0 = Z;
    g.sA = g.sB = P.s_pad * P.l_pad;
    g.M = g.N = (int)P.s_pad;
    g.K = (int)P.l_k;
    g.lda = g.ldb = (int)P.l_pad;
    g.out0 = hi;
    g.out1 = lo;
    g.sOut0 = g.sOut1 = P.s_pad * P.s_pad;
    g.ldo0 = g.ldo1 = (int)P.s_pad;
    return g;
}

// Three-pass symmetric s x s product C = X Y (Y symmetric, given by rows),
// both operands as hi / lo pairs.
GemmArgs sym3_args(const Plan& P, const uint16_t* xh, const uint16_t* xl, const uint16_t* yh,
                   const uint16_t* yl, void* oh, void* ol) {
    GemmArgs q{};
    q.batch = P.batch;
    q.A0 = xh;
    q.A1 = xl;
    q.B0 = yh;
    q.B1 = yl;
    q.sA = q.sB = P.s_pad * P.s_pad;
    q.M = q.N = (int)P.s_pad;
    q.K = (int)P.s_k;
    q.lda = q.ldb = (int)P.s_pad;
    q.out0 = oh;
    q.out1 = ol;
    q.sOut0 = q.sOut1 = P.s_pad * P.s_pad;
    q.ldo0 = q.ldo1 = (int)P.s_pad;
    return q;
}

// C = X Z with X [s][s] by rows and Z [s][l] as the B operand ([K][N]).
GemmArgs right_args(const Plan& P, const uint16_t* xh, const uint16_t* xl, const uint16_t* Z) {
    GemmArgs x{};
    x.batch = P.batch;
    x.A0 = xh;
    x.A1 = xl;
    x.B0 = Z;
    x.sA = P.s_pad * P.s_pad;
    x.sB = P.s_pad * P.l_pad;
    x.M = (int)P.s_pad;
    x.N = (int)P.l_pad;
    x.K = (int)P.s_k;
    x.lda = (int)P.s_pad;
    x.ldb = (int)P.l_pad;
    return x;
}

// The final Newton-Schulz product either stores O for the apply pass, in the
// layout that pass reads along W's rows (L [kpad][opad] for row selection,
// L^T [opad][kpad] for columns), or, for row selection with O in the L
// layout and bf16 W, applies the update step itself (EPI_APPLY).
struct FinalSpec {
    bool fuse;          // EPI_APPLY instead of EPI_FINAL + K5
    MatSet ms;
    const int32_t* sel;
    double lr_eff;
    float* dbg;
};

GemmEpi final_output(const Plan& P, GemmArgs& x, float* O, const FinalSpec& f) {
    const bool want_lt = P.axis == 1;
    x.out_transposed = P.z_is_L == want_lt ? 1 : 0;   // Z's natural layout is L iff z_is_L
    if (f.fuse) {
        x.out_transposed = 0;
        x.ms = f.ms;
        x.sel = f.sel;
        x.k = (int)P.k;
        x.d_oth = (int)P.d_oth;
        x.cols = P.cols;
        x.lr_eff = f.lr_eff;
        x.dbg = f.dbg;
        return EPI_APPLY;
    }
    x.out0 = O;
    x.sOut0 = P.kpad * P.opad;
    x.ldo0 = (int)(want_lt ? P.kpad : P.opad);
    return EPI_FINAL;
}

// DIRECT: per step A = Z Z^T (fp16, scaled by 2^eA; or a bf16 hi / lo pair
// when the coefficients leave fp16's range), B = b A + c A^2, Z <- a Z + B Z.
// With P.xrows the update reads Z^T (ZT[cur]) as rows and writes Z'^T beside
// Z'; Z_0^T comes from one transpose.
hipError_t ns_direct(const Plan& P, uint16_t* Z0, uint16_t* Z1, uint16_t* const* ZT, uint16_t* const* sq,
                     float* O, int ns_steps, const dion2_options& opt, const FinalSpec& fin,
                     hipStream_t stream) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);   // unpadded sides
    const double l_r = (double)(P.k < P.d_oth ? P.d_oth : P.k);
    const double nb = (double)P.batch;
    int eA = 0;
    const bool a16 = direct_a_exp(opt.ns_coeffs, ns_steps, &eA);
    // Z in, A out (fp16, or hi + lo)
    const double gram_bytes = (2.0 * s_r * l_r + (a16 ? 2.0 : 4.0) * s_r * s_r) * nb;
    uint16_t* zbuf[2] = {Z0, Z1};
    const bool xrows = P.xrows && ns_steps > 0;
    if (xrows) {
        hipError_t e = timed(DION2_PHASE_NS_UPDATE, 0.0, 4.0 * s_r * l_r * nb, 1, stream, [&] {
            return launch_transpose_bf16(Z0, ZT[0], P.s_pad, P.l_pad, P.batch, P.s_pad * P.l_pad, stream);
        });
        if (e != hipSuccess) return e;
    }
    int cur = 0;
    for (int t = 0; t < ns_steps; ++t) {
        const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
        uint16_t* Z = zbuf[cur];
        GemmArgs g = gram_args(P, Z, sq[SQ_AHI], a16 ? nullptr : sq[SQ_ALO]);
        if (a16) g.oexp = eA;
        hipError_t e = timed(DION2_PHASE_NS_GRAM, sym_flops(s_r, l_r) * nb, gram_bytes, 1, stream,
                             [&] { return launch_gemm(g, a16 ? EPI_H16 : EPI_SPLIT, 1, stream); });
        if (e != hipSuccess) return e;

        GemmArgs q = sym3_args(P, sq[SQ_AHI], sq[SQ_ALO], sq[SQ_AHI], sq[SQ_ALO], sq[SQ_B], nullptr);
        q.cb = cf[1];
        q.cc = cf[2];
        q.E0 = sq[SQ_AHI];
        q.E1 = sq[SQ_ALO];
        q.sE = P.s_pad * P.s_pad;
        q.lde = (int)P.s_pad;
        if (a16) {
            // one fp16 pass: C = 2^(2 eA) A^2, E0 = 2^eA A
            q.A1 = q.B1 = q.E1 = nullptr;
            q.f16 = 1;
            q.oexp = -2 * eA;
            q.eexp = -eA;
            e = timed(DION2_PHASE_NS_POLY, sym_flops(s_r, s_r) * nb, 4.0 * s_r * s_r * nb, 1, stream,
                      [&] { return launch_gemm(q, EPI_POLY_H16, 1, stream); });
        } else {
            e = timed(DION2_PHASE_NS_POLY, 3.0 * sym_flops(s_r, s_r) * nb, 6.0 * s_r * s_r * nb, 1, stream,
                      [&] { return launch_gemm(q, EPI_POLY, 3, stream); });
        }
        if (e != hipSuccess) return e;

        // Z' = a Z + B Z (a Z added in the epilogue)
        GemmArgs x = right_args(P, sq[SQ_B], nullptr, Z);
        x.ca = cf[0];
        x.E0 = Z;
        x.sE = P.s_pad * P.l_pad;
        x.lde = (int)P.l_pad;
        if (xrows) {   // Z^T [l_pad][s_pad] as the B operand's rows
            x.B0 = ZT[cur];
            x.ldb = (int)P.s_pad;
            x.b_rows = 1;
        }
        const bool last = t + 1 == ns_steps;
        GemmEpi epi = EPI_UPDATE;
        if (!last) {
            x.out0 = zbuf[1 - cur];
            x.sOut0 = P.s_pad * P.l_pad;
            x.ldo0 = (int)P.l_pad;
            if (xrows) {
                x.out1 = ZT[1 - cur];
                x.sOut1 = P.s_pad * P.l_pad;
                x.ldo1 = (int)P.s_pad;
            }
        } else {
            epi = final_output(P, x, O, fin);
        }
        const double ubytes = (2.0 * s_r * s_r + (last ? 6.0 : (xrows ? 6.0 : 4.0)) * s_r * l_r) * nb;
        e = timed(DION2_PHASE_NS_UPDATE, 2.0 * s_r * s_r * l_r * nb, ubytes, 1, stream,
                  [&] { return launch_gemm(x, epi, 1, stream); });
        if (e != hipSuccess) return e;
        cur = 1 - cur;
    }
    return hipSuccess;
}

// GRAM: A_0 = Z Z^T; per step Q_t = a I + b A_t + c A_t^2, P <- Q_t P and
// A_{t+1} = Q_t (Q_t A_t); finally O = P Z. Every s x s matrix is a
// polynomial in A_0, hence symmetric, and all of them commute. The three
// parts are separate so that a grouped call can run the chain of s x s
// products once for several groups of the same padded size.

// A_0 = Z Z^T as a hi / lo pair, or in fp16 (scaled) for the fp16 chain.
// With Zlo (the fp32 master) Z is the pair Z + Zlo: three passes.
hipError_t gram_a0(const Plan& P, const uint16_t* Z, const uint16_t* Zlo, uint16_t* Ah, uint16_t* Al,
                   const ChainFmt& fmt, hipStream_t stream) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);
    const double l_r = (double)(P.k < P.d_oth ? P.d_oth : P.k);
    const double nb = (double)P.batch;
    const int npass = Zlo ? 3 : 1;
    // Z in (hi, and lo), A out (hi + lo, or fp16)
    const double gram_bytes = ((Zlo ? 4.0 : 2.0) * s_r * l_r + (fmt.f16 ? 2.0 : 4.0) * s_r * s_r) * nb;
    GemmArgs g = gram_args(P, Z, Ah, fmt.f16 ? nullptr : Al);
    if (fmt.f16) g.oexp = fmt.eA;
    if (Zlo) g.A1 = g.B1 = Zlo;
    return timed(DION2_PHASE_NS_GRAM, npass * sym_flops(s_r, l_r) * nb, gram_bytes, 1, stream,
                 [&] { return launch_gemm(g, fmt.f16 ? EPI_H16 : EPI_SPLIT, npass, stream); });
}

// Work of one group's s x s products, for the profiler. Per step: Q_t (from
// A: hi + lo in and out, 8 s^2 bytes), P <- Q_t P and T = Q_t A (one dual
// launch when both are due; each product two hi/lo operands in and one out,
// 12 s^2, less the shared Q_t's 4 s^2 when fused), A <- Q_t T (12 s^2). The
// fp16 chain runs one pass per product on 2-byte entries, and its last
// P product writes the 4-byte hi / lo pair.
struct ChainCost {
    double flops = 0.0, bytes = 0.0;
};
int chain_products(int ns_steps) { return ns_steps + 3 * (ns_steps - 1); }
int chain_launches(int ns_steps) { return ns_steps == 1 ? 1 : 3 * ns_steps - 1; }
ChainCost chain_cost(const Plan& P, int ns_steps, const ChainFmt& fmt, bool fused) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);
    const double nb = (double)P.batch;
    const int nprod = chain_products(ns_steps);
    const int ndual = ns_steps >= 3 ? ns_steps - 2 : 0;
    const double per = (8.0 * ns_steps + 12.0 * (nprod - ns_steps) - 4.0 * ndual);
    ChainCost c;
    c.flops = (fmt.f16 && !fused ? 1.0 : 3.0) * sym_flops(s_r, s_r) * nb * nprod;
    // fused (in LDS): only A_0 in and P_T out, hi / lo pairs
    c.bytes = (fused ? 8.0 : fmt.f16 ? per / 2.0 + 2.0 : per) * s_r * s_r * nb;
    return c;
}

// A GRAM chain whose compact matrices have s <= 64 runs in one launch with
// its matrices in LDS (launch_chain_small), unless the caller asks for one
// launch per product; its Gram matrix then comes as a hi / lo pair.
bool fused_chain(int64_t s_k, const dion2_options& opt) {
    return !opt.ns_chain_per_product && s_k <= kSmallChainS;
}
// The fp16 chain (ns_chain F16) is taken only where it pays and holds: a
// chain of launches on a compact matrix at least four times as long as it
// is high (l >= 4 s, real sides). On near-square ones the Gram matrix
// squares a condition number that fp16's 11 bits cannot carry (randomly
// drawn calls measured O 0.13-0.41 from the exact iteration), and with
// l / s just under 3 (235 x 664, log-normal row scales) one reached 2.3e-2,
// so the chain stays in hi / lo there, as it does in LDS.
bool f16_chain(const ChainFmt& fmt, bool fused, const Plan& P) {
    const int64_t s = P.z_is_L ? P.k : P.d_oth, l = P.z_is_L ? P.d_oth : P.k;
    return fmt.f16 && !fused && l >= 4 * s;
}
ChainFmt chain_fmt_for(const ChainFmt& fmt, bool f16) {
    ChainFmt f = fmt;
    f.f16 = f16;
    return f;
}

// The s x s products of `batch` matrices of padded side s_pad (buffers sq,
// each [batch][s_pad][s_pad], A_0 in sq[SQ_AHI / SQ_ALO]). *cur_out tells
// which P pair holds the product of the Q_t: SQ_P0* (0) or SQ_P1* (1).
// The chain in fp16: the same products, one pass each, every matrix kept as
// fp16(2^e X) with the exponents of ChainFmt (the host tracks which one each
// buffer carries); the last P product writes the hi / lo pair the final
// product reads.
hipError_t chain_f16(const Plan& C, uint16_t* const* sq, int ns_steps, const dion2_options& opt,
                     const ChainFmt& f, hipStream_t stream, int* cur_out) {
    const int64_t s2 = C.s_pad * C.s_pad;
    uint16_t* A = sq[SQ_AHI];
    uint16_t* T = sq[SQ_THI];
    uint16_t* Ph[2] = {sq[SQ_P0HI], sq[SQ_P1HI]};
    uint16_t* Pl[2] = {sq[SQ_P0LO], sq[SQ_P1LO]};
    auto prod = [&](const uint16_t* x, const uint16_t* y, void* out, int oexp) {
        GemmArgs g = sym3_args(C, x, nullptr, y, nullptr, out, nullptr);
        g.f16 = 1;
        g.oexp = oexp;
        return g;
    };
    int cur = 0, pexp = 0;
    for (int t = 0; t < ns_steps; ++t) {
        const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
        // Q_t; the first one is P itself
        uint16_t* q = t == 0 ? Ph[0] : sq[SQ_QHI];
        GemmArgs g = prod(A, A, q, -2 * f.eA);
        g.ca = cf[0];
        g.cb = cf[1];
        g.cc = cf[2];
        g.E0 = A;
        g.sE = s2;
        g.lde = (int)C.s_pad;
        g.eexp = -f.eA;
        g.sexp = f.eQ;
        hipError_t r = launch_gemm(g, EPI_QPOLY_H16, 1, stream);
        if (r != hipSuccess) return r;
        if (t == 0) pexp = f.eQ;
        const bool do_p = t > 0, do_t = t + 1 < ns_steps;
        if (!do_t) {   // the last step: P_T = Q_t P as the hi / lo pair
            GemmArgs u = prod(q, Ph[cur], Ph[1 - cur], -f.eQ - pexp);
            u.out1 = Pl[1 - cur];
            r = launch_gemm(u, EPI_SPLIT, 1, stream);
            if (r != hipSuccess) return r;
            cur = 1 - cur;
            break;
        }
        // P <- Q_t P (t > 0) and T = Q_t A in one dual launch, then A <- Q_t T
        GemmArgs u = do_p ? prod(q, Ph[cur], Ph[1 - cur], f.eP - f.eQ - pexp)
                          : prod(q, A, T, f.eT - f.eQ - f.eA);
        if (do_p) {
            u.dual = 1;
            u.B0x = A;
            u.out0x = T;
            u.oexpx = f.eT - f.eQ - f.eA;
        }
        r = launch_gemm(u, EPI_H16, 1, stream);
        if (r != hipSuccess) return r;
        if (do_p) {
            cur = 1 - cur;
            pexp = f.eP;
        }
        r = launch_gemm(prod(q, T, A, f.eA - f.eQ - f.eT), EPI_H16, 1, stream);
        if (r != hipSuccess) return r;
    }
    *cur_out = cur;
    return hipSuccess;
}

hipError_t gram_chain(int batch, int64_t s_pad, int64_t s_k, uint16_t* const* sq, int ns_steps,
                      const dion2_options& opt, const ChainFmt& fmt, const ChainCost& cost,
                      hipStream_t stream, int* cur_out, bool fused) {
    Plan C{};
    C.batch = batch;
    C.s_pad = s_pad;
    C.s_k = s_k;
    if (fused) {
        // P_T lands where the launch-per-product chain leaves it
        const int cur = (ns_steps - 1) & 1;
        SmallChainArgs c{};
        c.Ah = sq[SQ_AHI];
        c.Al = sq[SQ_ALO];
        c.Ph = sq[cur ? SQ_P1HI : SQ_P0HI];
        c.Pl = sq[cur ? SQ_P1LO : SQ_P0LO];
        c.s_pad = s_pad;
        c.s_k = (int)s_k;
        c.ns_steps = ns_steps;
        c.batch = batch;
        for (int t = 0; t < ns_steps; ++t) {
            const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
            for (int i = 0; i < 3; ++i) c.cf[t][i] = cf[i];
        }
        *cur_out = cur;
        return timed(DION2_PHASE_NS_POLY, cost.flops, cost.bytes, 1, stream,
                     [&] { return launch_chain_small(c, stream); });
    }
    if (fmt.f16)
        return timed(DION2_PHASE_NS_POLY, cost.flops, cost.bytes, chain_launches(ns_steps), stream,
                     [&] { return chain_f16(C, sq, ns_steps, opt, fmt, stream, cur_out); });
    uint16_t* Ah = sq[SQ_AHI];
    uint16_t* Al = sq[SQ_ALO];
    uint16_t* Ph[2] = {sq[SQ_P0HI], sq[SQ_P1HI]};
    uint16_t* Pl[2] = {sq[SQ_P0LO], sq[SQ_P1LO]};
    int cur = 0;
    // the products run back to back and are timed as one span
    hipError_t e = timed(DION2_PHASE_NS_POLY, cost.flops, cost.bytes, chain_launches(ns_steps), stream,
                         [&]() -> hipError_t {
        for (int t = 0; t < ns_steps; ++t) {
            const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
            // Q_t; the first one is P itself
            uint16_t* qh = t == 0 ? Ph[0] : sq[SQ_QHI];
            uint16_t* ql = t == 0 ? Pl[0] : sq[SQ_QLO];
            GemmArgs q = sym3_args(C, Ah, Al, Ah, Al, qh, ql);
            q.ca = cf[0];
            q.cb = cf[1];
            q.cc = cf[2];
            q.E0 = Ah;
            q.E1 = Al;
            q.sE = C.s_pad * C.s_pad;
            q.lde = (int)C.s_pad;
            hipError_t r = launch_gemm(q, EPI_QPOLY, 3, stream);
            if (r != hipSuccess) return r;
            // P <- Q_t P (t > 0) and T = Q_t A (t < T - 1) share Q_t: one
            // launch when both are due
            const bool do_p = t > 0, do_t = t + 1 < ns_steps;
            if (do_p || do_t) {
                GemmArgs u = do_p ? sym3_args(C, qh, ql, Ph[cur], Pl[cur], Ph[1 - cur], Pl[1 - cur])
                                  : sym3_args(C, qh, ql, Ah, Al, sq[SQ_THI], sq[SQ_TLO]);
                if (do_p && do_t) {
                    u.dual = 1;
                    u.B0x = Ah;
                    u.B1x = Al;
                    u.out0x = sq[SQ_THI];
                    u.out1x = sq[SQ_TLO];
                }
                r = launch_gemm(u, EPI_SPLIT, 3, stream);
                if (r != hipSuccess) return r;
                if (do_p) cur = 1 - cur;
            }
            if (do_t) {   // A <- Q_t T
                GemmArgs v = sym3_args(C, qh, ql, sq[SQ_THI], sq[SQ_TLO], Ah, Al);
                r = launch_gemm(v, EPI_SPLIT, 3, stream);
                if (r != hipSuccess) return r;
            }
        }
        return hipSuccess;
    });
    *cur_out = cur;
    return e;
}

// O = (P_hi + P_lo) Z, or the update step applied in the epilogue; with Zlo
// (the fp32 master) Z is the pair Z + Zlo and the product takes three passes.
hipError_t gram_final(const Plan& P, const uint16_t* Ph, const uint16_t* Pl, const uint16_t* Z,
                      const uint16_t* Zlo, float* O, const FinalSpec& fin, hipStream_t stream) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);
    const double l_r = (double)(P.k < P.d_oth ? P.d_oth : P.k);
    const double nb = (double)P.batch;
    GemmArgs x = right_args(P, Ph, Pl, Z);
    if (Zlo) x.B1 = Zlo;
    const GemmEpi epi = final_output(P, x, O, fin);
    const int npass = Zlo ? 3 : 2;
    // P hi + lo and Z (hi, and lo) in, O (or W's selected lines, read and written) out
    const double fbytes = (4.0 * s_r * s_r + (Zlo ? 8.0 : 6.0) * s_r * l_r) * nb;
    return timed(DION2_PHASE_NS_UPDATE, 2.0 * npass * s_r * s_r * l_r * nb, fbytes, 1, stream,
                 [&] { return launch_gemm(x, epi, npass, stream); });
}

hipError_t ns_gram(const Plan& P, const uint16_t* Z, const uint16_t* Zlo, uint16_t* const* sq, float* O,
                   int ns_steps, const dion2_options& opt, const ChainFmt& fmt, const FinalSpec& fin,
                   hipStream_t stream) {
    const bool fused = fused_chain(P.s_k, opt);
    const ChainFmt cf = chain_fmt_for(fmt, f16_chain(fmt, fused, P));
    hipError_t e = gram_a0(P, Z, Zlo, sq[SQ_AHI], sq[SQ_ALO], cf, stream);
    if (e != hipSuccess) return e;
    int cur = 0;
    e = gram_chain(P.batch, P.s_pad, P.s_k, sq, ns_steps, opt, cf, chain_cost(P, ns_steps, cf, fused), stream,
                   &cur, fused);
    if (e != hipSuccess) return e;
    return gram_final(P, cur ? sq[SQ_P1HI] : sq[SQ_P0HI], cur ? sq[SQ_P1LO] : sq[SQ_P0LO], Z, Zlo, O,
                      fin, stream);
}

// ------------------------------------------------------------------ step

// Device buffers of one group's step, carved from its workspace region.
struct Bufs {
    double* l1;
    double* sq;
    int32_t* sel;
    int32_t* rank;
    double* scale;
    uint16_t* Z0;   // compact matrix in its wide orientation: L [kpad][opad] or L^T [opad][kpad]
    uint16_t* Z1;
    uint16_t* ZT[2];   // DIRECT with xrows: X^T [l_pad][s_pad], ping-pong
    double* sqp;       // colpass: per-block sums of squares of the selected columns
    uint16_t* sbuf[SQ_GRAM_COUNT];   // s x s buffers (null when a shared chain owns them)
    float* O;
    double* part;
};

Bufs carve(const Plan& P, char* ws) {
    Bufs b{};
    b.l1 = reinterpret_cast<double*>(ws + P.o_l1);
    b.sq = reinterpret_cast<double*>(ws + P.o_sq);
    b.sel = reinterpret_cast<int32_t*>(ws + P.o_sel);
    b.rank = P.axis == 1 ? reinterpret_cast<int32_t*>(ws + P.o_rank) : nullptr;
    b.scale = reinterpret_cast<double*>(ws + P.o_scale);
    b.Z0 = reinterpret_cast<uint16_t*>(ws + P.o_Z);
    b.Z1 = reinterpret_cast<uint16_t*>(ws + P.o_Z1);
    b.ZT[0] = P.xrows ? reinterpret_cast<uint16_t*>(ws + P.o_ZT) : nullptr;
    b.ZT[1] = P.xrows ? b.ZT[0] + (size_t)P.batch * (size_t)P.s_pad * (size_t)P.l_pad : nullptr;
    b.sqp = P.colpass ? reinterpret_cast<double*>(ws + P.o_sqp) : nullptr;
    for (int i = 0; i < SQ_GRAM_COUNT; ++i)
        b.sbuf[i] = reinterpret_cast<uint16_t*>(ws + P.o_S + (size_t)i * P.S_bytes);
    b.O = reinterpret_cast<float*>(ws + P.o_O);
    b.part = reinterpret_cast<double*>(ws + P.o_part);
    return b;
}

// Bytes each phase must move as designed. Rows: K1 reads M, G and writes M;
// K3 reads and writes the selected rows of M and writes the compact bf16
// copy; K5 reads O and reads and writes the selected rows of W. Columns
// (selected columns touch every cache line of a row): K1 only reads M and
// G; K3 reads M, G and writes M whole, plus the compact copy; K5 reads O and
// reads and writes W whole.
struct PhaseBytes {
    double k1, k3, k5;
};
PhaseBytes phase_bytes(const Plan& P, const dion2_options& opt) {
    const double n_el = (double)P.batch * (double)P.rows * (double)P.cols;
    const double g_bytes = opt.g_dtype == DION2_DTYPE_BF16 ? 2.0 : 4.0;
    const double w_bytes = opt.w_dtype == DION2_DTYPE_BF16 ? 2.0 : 4.0;
    const double sel_el = (double)P.batch * (double)P.k * (double)P.d_oth;
    const bool cm = P.axis == 1;
    PhaseBytes pb;
    pb.k1 = n_el * ((cm ? 4.0 : 8.0) + g_bytes);
    pb.k3 = (cm ? n_el * (8.0 + g_bytes) : sel_el * 8.0) + sel_el * 2.0;
    if (cm && P.colpass && !opt.dbg_norms) {
        pb.k1 = 0.0;                   // no norm pass
        pb.k3 += sel_el * 8.0;         // the unscaled fp32 copy written and read back
    }
    pb.k5 = (cm ? n_el : sel_el) * 2.0 * w_bytes + sel_el * 4.0;
    return pb;
}

// K1 momentum and line norms, K2 selection, K3 gather and decay.
int front(const Plan& P, const MatSet& ms, const Bufs& b, float mu, int ns_steps,
          const dion2_options& opt, hipStream_t stream) {
    const PhaseBytes pb = phase_bytes(P, opt);
    const bool cm = P.axis == 1;
    // columns under the Random rule: no norm pass (the debug l1 norms need it)
    const bool colpass = P.colpass && !opt.dbg_norms;
    MomentumArgs ma{};
    ma.ms = ms;
    ma.rows = P.rows;
    ma.cols = P.cols;
    ma.batch = P.batch;
    ma.l1 = b.l1;
    ma.sq = b.sq;
    ma.part = b.part;
    ma.rb_rows = P.rb_rows;
    ma.nrb = P.nrb;
    ma.mu = mu;
    hipError_t e = hipSuccess;
    if (!colpass) {
        e = timed(DION2_PHASE_MOMENTUM, 0.0, pb.k1, P.axis == 0 ? 1 : 2, stream,
                  [&] { return launch_momentum(ma, P.axis, opt.g_dtype == DION2_DTYPE_BF16, stream); });
        if (e != hipSuccess) return hip_fail(e, "launch K1 momentum");
    }

    SelectArgs sa{};
    sa.l1 = b.l1;
    sa.sq = colpass ? nullptr : b.sq;   // the single pass computes the scale itself
    sa.d_sel = (int)P.d_sel;
    sa.k = (int)P.k;
    sa.batch = P.batch;
    sa.eps = (double)opt.ns_eps;
    sa.sel = b.sel;
    sa.scale = b.scale;
    sa.rank = b.rank;
    sa.rule = opt.select_rule;
    sa.seed = opt.rand_seed;
    sa.step = opt.rand_step;
    sa.matrix0 = opt.rand_matrix0;
    e = timed(DION2_PHASE_SELECT, 0.0, (double)P.batch * (double)P.d_sel * 16.0, 1, stream,
              [&] { return launch_select(sa, stream); });
    if (e != hipSuccess) return hip_fail(e, "launch K2 select");

    GatherArgs ga{};
    ga.ms = ms;
    ga.rows = P.rows;
    ga.cols = P.cols;
    ga.batch = P.batch;
    ga.k = (int)P.k;
    ga.d_oth = (int)P.d_oth;
    ga.kpad = (int)P.kpad;
    ga.opad = (int)P.opad;
    ga.sel = b.sel;
    ga.rank = b.rank;
    ga.scale = b.scale;
    ga.mu = mu;
    // rows: selective decay here, decay-all by its own pass; columns: both here
    ga.decay = cm ? (opt.decay_all ? 2 : 1) : (opt.decay_all ? 0 : 1);
    ga.L = P.z_is_L ? b.Z0 : nullptr;
    ga.LT = P.z_is_L ? nullptr : b.Z0;
    if (P.master && ns_steps > 0) {   // the lo half of X beside it
        ga.Llo = P.z_is_L ? b.Z1 : nullptr;
        ga.LTlo = P.z_is_L ? nullptr : b.Z1;
    }
    ga.O = ns_steps == 0 ? b.O : nullptr;
    if (colpass) {   // unscaled columns into O (free until the final product), then normalised
        ga.L = ga.LT = nullptr;
        ga.O = b.O;
        ga.sq_part = b.sqp;
    }
    e = timed(DION2_PHASE_GATHER, 0.0, pb.k3, colpass ? 3 : 1, stream, [&] {
        hipError_t r = launch_gather(ga, P.axis, opt.g_dtype == DION2_DTYPE_BF16, stream);
        if (r != hipSuccess || !colpass) return r;
        ColpassArgs ca{};
        ca.Ot = b.O;
        ca.sq_part = b.sqp;
        ca.scale = b.scale;
        ca.L = P.z_is_L ? b.Z0 : nullptr;
        ca.LT = P.z_is_L ? nullptr : b.Z0;
        ca.batch = P.batch;
        ca.k = (int)P.k;
        ca.kpad = (int)P.kpad;
        ca.opad = (int)P.opad;
        ca.eps = (double)opt.ns_eps;
        return launch_colpass_finish(ca, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "launch K3 gather");
    // the debug copies of X, before Newton-Schulz overwrites the DIRECT form's buffer
    for (int h = 0; h < 2; ++h) {
        uint16_t* dst = h == 0 ? opt.dbg_compact : opt.dbg_compact_lo;
        if (!dst) continue;
        CompactCopyArgs ca{h == 0 ? b.Z0 : b.Z1, dst, P.batch, (int)P.k, (int)P.d_oth,
                           (int)P.kpad, (int)P.opad, P.z_is_L ? 0 : 1};
        e = launch_copy_compact(ca, stream);
        if (e != hipSuccess) return hip_fail(e, "launch debug copy of X");
    }
    if (opt.decay_all && !cm) {
        DecayAllArgs da{ms, P.rows, P.cols, P.batch, mu};
        e = launch_decay_all(da, stream);
        if (e != hipSuccess) return hip_fail(e, "launch decay-all");
    }
    return DION2_OK;
}

// Whether the final Newton-Schulz product applies the update itself (row
// selection with O in the L layout and bf16 W), and its operands.
FinalSpec make_final(const Plan& P, const MatSet& ms, const Bufs& b, float lr, int ns_steps,
                     const dion2_options& opt) {
    FinalSpec fin{};
    fin.lr_eff = (double)lr * std::sqrt((double)P.rows / (double)P.cols);
    fin.fuse = ns_steps > 0 && P.axis == 0 && P.z_is_L && opt.w_dtype == DION2_DTYPE_BF16 &&
               P.cols % 8 == 0 && P.cols >= 16;
    fin.ms = ms;
    fin.sel = b.sel;
    fin.dbg = opt.dbg_update;
    return fin;
}

// K5 (unless fused into the final product) and the debug copies.
int back(const Plan& P, const MatSet& ms, const Bufs& b, const FinalSpec& fin,
         const dion2_options& opt, hipStream_t stream) {
    hipError_t e;
    if (!fin.fuse) {
        ApplyArgs aa{};
        aa.ms = ms;
        aa.rows = P.rows;
        aa.cols = P.cols;
        aa.batch = P.batch;
        aa.k = (int)P.k;
        aa.d_oth = (int)P.d_oth;
        aa.kpad = (int)P.kpad;
        aa.opad = (int)P.opad;
        aa.sel = b.sel;
        aa.rank = b.rank;
        aa.O = b.O;
        aa.lr_eff = fin.lr_eff;
        aa.dbg = opt.dbg_update;
        e = timed(DION2_PHASE_APPLY, 0.0, phase_bytes(P, opt).k5, 1, stream,
                  [&] { return launch_apply(aa, P.axis, opt.w_dtype == DION2_DTYPE_BF16, stream); });
        if (e != hipSuccess) return hip_fail(e, "launch K5 apply");
    }
    if (opt.dbg_sel_idx) {
        e = hipMemcpyAsync(opt.dbg_sel_idx, b.sel, (size_t)P.batch * P.k * 4, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "copy dbg_sel_idx");
    }
    if (opt.dbg_norms) {
        e = hipMemcpyAsync(opt.dbg_norms, b.l1, (size_t)P.batch * P.d_sel * 8, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "copy dbg_norms");
    }
    return DION2_OK;
}

struct Tables {
    void* const* W;
    float* const* M;
    const void* const* G;
};

int run_step(const Plan& P, void* W, float* M, const void* G, const Tables* tabs,
             float mu, float lr, int ns_steps, const dion2_options& opt, const ChainFmt& fmt,
             hipStream_t stream) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");

    Workspace* w = nullptr;
    std::unique_lock<std::mutex> use_lock;
    char* ws;
    if (opt.workspace) {
        ws = static_cast<char*>(opt.workspace);
    } else {
        w = workspace_for(dev, stream);
        use_lock = std::unique_lock<std::mutex>(w->use);
        int st = ensure_device(w, P.total);
        if (st != DION2_OK) return st;
        ws = static_cast<char*>(w->dev);
    }

    MatSet ms{};
    ms.stride = P.rows * P.cols;
    if (tabs) {
        // stage the host pointer tables and copy them to the device workspace
        void** dst = reinterpret_cast<void**>(ws + P.o_tables);
        const size_t n = 3 * (size_t)P.batch;
        void** staging = nullptr;
        TableSlot* slot = nullptr;
        if (w) {
            // The first slot whose earlier copy has completed (checked with
            // hipEventQuery, which does not block). Only with all slots'
            // copies still queued -- more than kTableSlots table calls in
            // flight on this stream -- does the host wait, for the oldest.
            for (int i = 0; i < kTableSlots && !slot; ++i) {
                TableSlot& c = w->slots[(w->next_slot + i) % kTableSlots];
                if (c.pending) {
                    e = hipEventQuery(c.done);
                    if (e == hipErrorNotReady) continue;
                    if (e != hipSuccess) return hip_fail(e, "hipEventQuery(tables)");
                    c.pending = false;
                }
                slot = &c;
            }
            if (!slot) {
                slot = &w->slots[w->next_slot];
                e = hipEventSynchronize(slot->done);
                if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(tables)");
                slot->pending = false;
            }
            w->next_slot = (int)(slot - w->slots + 1) % kTableSlots;
            if (slot->count < n) {
                if (slot->host) (void)hipHostFree(slot->host);   // a failed free only leaks
                slot->host = nullptr;
                slot->count = 0;
                e = hipHostMalloc(reinterpret_cast<void**>(&slot->host), n * sizeof(void*));
                if (e != hipSuccess) return hip_fail(e, "hipHostMalloc(pointer tables)");
                slot->count = n;
            }
            if (!slot->done) {
                e = hipEventCreateWithFlags(&slot->done, hipEventDisableTiming);
                if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
            }
            staging = slot->host;
        }
        void* tmp_local[3 * 64];
        if (!staging) staging = n <= 3 * 64 ? tmp_local : nullptr;
        if (!staging) {
            return fail(DION2_ERR_UNSUPPORTED,
                        "pointer tables of more than 64 matrices need the library workspace");
        }
        for (int b = 0; b < P.batch; ++b) {
            staging[b] = tabs->W[b];
            staging[P.batch + b] = tabs->M[b];
            staging[2 * P.batch + b] = const_cast<void*>(tabs->G[b]);
        }
        e = hipMemcpyAsync(dst, staging, n * sizeof(void*), hipMemcpyHostToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(pointer tables)");
        if (slot) {
            e = hipEventRecord(slot->done, stream);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(tables)");
            slot->pending = true;
        } else {
            e = hipStreamSynchronize(stream);   // tmp_local goes out of scope
            if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize(tables)");
        }
        ms.Wt = dst;
        ms.Mt = reinterpret_cast<float* const*>(dst + P.batch);
        ms.Gt = reinterpret_cast<const void* const*>(dst + 2 * P.batch);
    } else {
        ms.W = W;
        ms.M = M;
        ms.G = G;
    }

    Bufs b = carve(P, ws);
    int st = front(P, ms, b, mu, ns_steps, opt, stream);
    if (st != DION2_OK) return st;
    const FinalSpec fin = make_final(P, ms, b, lr, ns_steps, opt);
    if (ns_steps > 0) {   // with no step the gather has written O
        e = P.gram ? ns_gram(P, b.Z0, P.master ? b.Z1 : nullptr, b.sbuf, b.O, ns_steps, opt, fmt, fin, stream)
                   : ns_direct(P, b.Z0, b.Z1, b.ZT, b.sbuf, b.O, ns_steps, opt, fin, stream);
        if (e != hipSuccess) return hip_fail(e, "launch K4 Newton-Schulz");
    }
    return back(P, ms, b, fin, opt, stream);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int validate_common(float mu, float lr, int ns_steps, const dion2_options& opt) {
    if (!std::isfinite(mu)) return fail(DION2_ERR_INVALID_ARG, "mu is not finite");
    if (!std::isfinite(lr)) return fail(DION2_ERR_INVALID_ARG, "lr is not finite");
    if (ns_steps < 0 || ns_steps > DION2_MAX_NS_STEPS)
        return fail(DION2_ERR_INVALID_ARG, "ns_steps %d not in [0, %d]", ns_steps, DION2_MAX_NS_STEPS);
    if (opt.w_dtype != DION2_DTYPE_F32 && opt.w_dtype != DION2_DTYPE_BF16)
        return fail(DION2_ERR_INVALID_ARG, "w_dtype %d is not F32 or BF16", opt.w_dtype);
    if (opt.g_dtype != DION2_DTYPE_F32 && opt.g_dtype != DION2_DTYPE_BF16)
        return fail(DION2_ERR_INVALID_ARG, "g_dtype %d is not F32 or BF16", opt.g_dtype);
    if (!std::isfinite(opt.ns_eps) || opt.ns_eps < 0.f)
        return fail(DION2_ERR_INVALID_ARG, "ns_eps must be finite and >= 0");
    if (opt.decay_all != 0 && opt.decay_all != 1)
        return fail(DION2_ERR_INVALID_ARG, "decay_all must be 0 or 1");
    if (opt.select_rule != DION2_SELECT_L1 && opt.select_rule != DION2_SELECT_RANDOM)
        return fail(DION2_ERR_INVALID_ARG, "select_rule %d is not L1 or RANDOM", opt.select_rule);
    if (opt.ns_master != DION2_MASTER_BF16 && opt.ns_master != DION2_MASTER_FP32)
        return fail(DION2_ERR_INVALID_ARG, "ns_master %d is not BF16 or FP32", opt.ns_master);
    if (opt.ns_master == DION2_MASTER_FP32 && opt.ns_chain == DION2_CHAIN_F16)
        return fail(DION2_ERR_INVALID_ARG, "ns_master FP32 keeps the s x s chain in hi / lo pairs (ns_chain F16 given)");
    if (opt.ns_master == DION2_MASTER_FP32 && opt.ns_form == DION2_NS_DIRECT)
        return fail(DION2_ERR_UNSUPPORTED, "ns_master FP32 runs in the GRAM order (ns_form DIRECT given)");
    if (opt.dbg_compact_lo && (opt.ns_master != DION2_MASTER_FP32 || ns_steps < 1))
        return fail(DION2_ERR_INVALID_ARG, "dbg_compact_lo needs ns_master FP32 and ns_steps >= 1");
    if (opt.ns_coeffs) {
        for (int i = 0; i < 3 * ns_steps; ++i)
            if (!std::isfinite(opt.ns_coeffs[i]))
                return fail(DION2_ERR_INVALID_ARG, "ns_coeffs[%d] is not finite", i);
    }
    return DION2_OK;
}

// ------------------------------------------------- allocation-free calls
// The workspace of dion2_step_noalloc: a fixed device array that every GPU
// the library runs on holds until the process ends. In host code `scratch`
// names a host-side stand-in, not device memory; the device address of each
// GPU's copy comes from hipGetSymbolAddress, taken once per device with that
// device current, and only that address is ever handed to a kernel.
constexpr size_t kScratchBytes = DION2_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;   // device -> address of its scratch

int scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it == g_scratch_ptr.end()) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(DION2_ERR_HIP, "hipGetSymbolAddress(scratch) gave a null address");
        it = g_scratch_ptr.emplace(dev, ptr).first;
    }
    *out = it->second;
    return DION2_OK;
}

int step_impl(void* W, float* M, const void* G, const Tables* tabs, int batch, int64_t rows,
              int64_t cols, float alpha, float mu, float lr, int ns_steps, int axis,
              const dion2_options* opt_in, void* stream, bool no_alloc = false) {
    dion2_options opt;
    if (opt_in) opt = *opt_in;
    else dion2_options_init(&opt);
    int st = validate_common(mu, lr, ns_steps, opt);
    if (st != DION2_OK) return st;
    Plan P;
    st = make_plan(batch, rows, cols, alpha, axis, opt.ns_form, ns_steps, &P, true,
                   opt.ns_master == DION2_MASTER_FP32, opt.select_rule == DION2_SELECT_RANDOM);
    if (st != DION2_OK) return st;
    ChainFmt fmt;
    st = chain_format(opt, ns_steps, &fmt);
    if (st != DION2_OK) return st;
    if (opt.select_rule == DION2_SELECT_RANDOM &&
        (opt.rand_matrix0 < 0 || opt.rand_matrix0 + batch > (int64_t(1) << 32)))
        return fail(DION2_ERR_INVALID_ARG, "rand_matrix0 %lld with batch %d leaves [0, 2^32)",
                    (long long)opt.rand_matrix0, batch);
    if (tabs) {
        if (!tabs->W || !tabs->M || !tabs->G)
            return fail(DION2_ERR_INVALID_ARG, "pointer tables must not be NULL");
        for (int b = 0; b < batch; ++b) {
            if (!tabs->W[b] || !tabs->M[b] || !tabs->G[b])
                return fail(DION2_ERR_INVALID_ARG, "matrix %d has a NULL pointer", b);
            if (!aligned16(tabs->W[b]) || !aligned16(tabs->M[b]) || !aligned16(tabs->G[b]))
                return fail(DION2_ERR_INVALID_ARG, "matrix %d is not 16-byte aligned", b);
        }
    } else {
        if (!W || !M || !G) return fail(DION2_ERR_INVALID_ARG, "W, M and G must not be NULL");
        if (!aligned16(W) || !aligned16(M) || !aligned16(G))
            return fail(DION2_ERR_INVALID_ARG, "W, M and G must be 16-byte aligned");
    }
    if (no_alloc) {
        if (opt.workspace)
            return fail(DION2_ERR_INVALID_ARG,
                        "dion2_step_noalloc uses its own scratch (opt->workspace must be NULL)");
        if (P.total > kScratchBytes)
            return fail(DION2_ERR_WORKSPACE,
                        "this call needs %zu bytes of scratch; dion2_step_noalloc holds %zu "
                        "(DION2_NOALLOC_SCRATCH_BYTES): use a smaller batch or dion2_step_ex",
                        P.total, kScratchBytes);
        void* ptr = nullptr;
        st = scratch_address(&ptr);
        if (st != DION2_OK) return st;
        opt.workspace = ptr;
        opt.workspace_bytes = kScratchBytes;
        t_no_alloc = true;
        st = run_step(P, W, M, G, tabs, mu, lr, ns_steps, opt, fmt, static_cast<hipStream_t>(stream));
        t_no_alloc = false;
        return st;
    }
    if (opt.workspace) {
        if ((reinterpret_cast<uintptr_t>(opt.workspace) & 255u) != 0)
            return fail(DION2_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
        if (opt.workspace_bytes < P.total)
            return fail(DION2_ERR_WORKSPACE, "workspace of %zu bytes is below the %zu needed",
                        opt.workspace_bytes, P.total);
    }
    return run_step(P, W, M, G, tabs, mu, lr, ns_steps, opt, fmt, static_cast<hipStream_t>(stream));
}

// Several same-shape groups in one call. Each group runs K1-K3 in its own
// workspace region; the groups in the GRAM form are gathered into chains by
// padded s (one chain per size) whose s x s buffers hold all their matrices
// back to back, so every product of the chain is one launch for all of
// them; then each group's final product and K5 run. DIRECT groups run
// whole in the first pass. Per matrix the arithmetic is that of a call per
// group (every kernel treats the matrices of a batch independently).
constexpr int kMaxGroups = 64;
constexpr int kMaxGroupStreams = 8;
constexpr int kDefaultGroupStreams = 4;
// Groups share a chain only while one product of theirs has fewer output
// tiles than this (half the compute units). Sharing makes the chain wait for
// every member's first half, so groups big enough to keep half the chip
// busy do better on their own stream, overlapping the others: the three
// groups of the 1B stack at alpha = 0.25 (160 to 640 tiles) measured 40 us
// per step slower with the two small ones sharing.
constexpr int64_t kChainShareTiles = 128;

int groups_impl(const dion2_group* groups, int ngroups, float alpha, float mu, float lr,
                int ns_steps, const dion2_options* opt_in, hipStream_t stream) {
    dion2_options opt;
    if (opt_in) opt = *opt_in;
    else dion2_options_init(&opt);
    if (!groups) return fail(DION2_ERR_INVALID_ARG, "groups must not be NULL");
    if (ngroups < 1 || ngroups > kMaxGroups)
        return fail(DION2_ERR_INVALID_ARG, "ngroups %d not in [1, %d]", ngroups, kMaxGroups);
    if (opt.workspace)
        return fail(DION2_ERR_INVALID_ARG, "grouped calls use the library workspace (workspace must be NULL)");
    if (opt.dbg_sel_idx || opt.dbg_norms || opt.dbg_update || opt.dbg_compact || opt.dbg_compact_lo)
        return fail(DION2_ERR_INVALID_ARG, "grouped calls take no debug outputs");
    if (opt.group_streams < 0 || opt.group_streams > kMaxGroupStreams)
        return fail(DION2_ERR_INVALID_ARG, "group_streams %d not in [0, %d]", opt.group_streams,
                    kMaxGroupStreams);
    int st = validate_common(mu, lr, ns_steps, opt);
    if (st != DION2_OK) return st;
    ChainFmt fmt;
    st = chain_format(opt, ns_steps, &fmt);
    if (st != DION2_OK) return st;

    struct Chain {
        int64_t s_pad, s_k = 0;
        bool fused = false;   // one launch, in LDS (every member has s <= 64)
        bool f16 = false;     // the fp16 chain (every member wide)
        int batch = 0;
        size_t off = 0, S_bytes = 0;
    };
    std::vector<Plan> plans(ngroups);
    std::vector<int> chain_of(ngroups, -1);
    std::vector<int> chain_pos(ngroups, 0);   // first matrix of the group in its chain
    std::vector<Chain> chains;
    int64_t total_batch = 0;
    for (int g = 0; g < ngroups; ++g) {
        const dion2_group& G = groups[g];
        Plan P;
        const bool master = opt.ns_master == DION2_MASTER_FP32;
        st = make_plan(G.batch, G.rows, G.cols, alpha, G.axis, opt.ns_form, ns_steps, &P, true, master,
                       opt.select_rule == DION2_SELECT_RANDOM);
        if (st != DION2_OK) return fail(st, "group %d: %s", g, g_last_error.c_str());
        if (!G.W || !G.M || !G.G) return fail(DION2_ERR_INVALID_ARG, "group %d: W, M and G must not be NULL", g);
        if (!aligned16(G.W) || !aligned16(G.M) || !aligned16(G.G))
            return fail(DION2_ERR_INVALID_ARG, "group %d: W, M and G must be 16-byte aligned", g);
        // A group whose s x s products alone fill the chip keeps its own
        // chain (and can overlap the other groups); smaller ones share.
        const int64_t st_tiles = P.s_pad / kTile;
        const bool small = (int64_t)P.batch * st_tiles * (st_tiles + 1) / 2 < kChainShareTiles;
        if (P.gram && ns_steps > 0 && small) {
            const bool fused = fused_chain(P.s_k, opt);
            const bool f16 = f16_chain(fmt, fused, P);
            int c = 0;
            while (c < (int)chains.size() &&
                   (chains[c].s_pad != P.s_pad || chains[c].fused != fused || chains[c].f16 != f16))
                ++c;
            if (c == (int)chains.size()) {
                chains.push_back(Chain{});
                chains[c].s_pad = P.s_pad;
                chains[c].fused = fused;
                chains[c].f16 = f16;
            }
            // the shared products sum to the widest member's real side
            chains[c].s_k = std::max(chains[c].s_k, P.s_k);
            chain_of[g] = c;
            chain_pos[g] = chains[c].batch;
            chains[c].batch += P.batch;
            make_plan(G.batch, G.rows, G.cols, alpha, G.axis, opt.ns_form, ns_steps, &P, false, master,
                      opt.select_rule == DION2_SELECT_RANDOM);
        }
        plans[g] = P;
        total_batch += G.batch;
    }
    if (opt.select_rule == DION2_SELECT_RANDOM &&
        (opt.rand_matrix0 < 0 || opt.rand_matrix0 + total_batch > (int64_t(1) << 32)))
        return fail(DION2_ERR_INVALID_ARG, "rand_matrix0 %lld with %lld matrices leaves [0, 2^32)",
                    (long long)opt.rand_matrix0, (long long)total_batch);
    for (const Chain& c : chains)
        if (c.batch > 65535) return fail(DION2_ERR_INVALID_ARG, "more than 65535 matrices share one chain");

    // one workspace: the groups' regions, then the chains' s x s buffers
    std::vector<size_t> goff(ngroups);
    size_t total = 0;
    for (int g = 0; g < ngroups; ++g) {
        goff[g] = total;
        total += align256(plans[g].total);
    }
    for (Chain& c : chains) {
        c.S_bytes = align256((size_t)c.batch * (size_t)c.s_pad * (size_t)c.s_pad * 2);
        c.off = total;
        total += c.S_bytes * SQ_GRAM_COUNT;
    }

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Workspace* w = workspace_for(dev, stream);
    std::unique_lock<std::mutex> use_lock(w->use);
    st = ensure_device(w, total);
    if (st != DION2_OK) return st;
    char* ws = static_cast<char*>(w->dev);

    auto chain_buf = [&](int c, int i) {
        return reinterpret_cast<uint16_t*>(ws + chains[c].off + (size_t)i * chains[c].S_bytes);
    };
    // Streams: with one, everything goes on `stream` in order. Otherwise the
    // groups (and chains) are dealt round-robin to auxiliary streams forked
    // from `stream`; a chain waits for its groups' A_0, a group's final
    // product for its chain, and `stream` for every auxiliary stream.
    const int want = opt.group_streams == 0 ? kDefaultGroupStreams : opt.group_streams;
    const int nS = want < ngroups ? want : ngroups;
    const int nchain = (int)chains.size();
    std::vector<hipStream_t> strm(nS, stream);
    hipEvent_t fork = nullptr;
    std::vector<hipEvent_t> ev_a0(ngroups, nullptr), ev_chain(nchain, nullptr), ev_join(nS, nullptr);
    // Once forked, `stream` waits for every auxiliary stream on every way out
    // (an error return included), so later work on it never overlaps this
    // call's kernels.
    struct Join {
        int n;
        const std::vector<hipStream_t>& from;
        const std::vector<hipEvent_t>& ev;
        hipStream_t to;
        hipError_t run() {
            hipError_t first = hipSuccess;
            for (int i = 0; i < n; ++i) {
                hipError_t e = hipEventRecord(ev[i], from[i]);
                if (e == hipSuccess) e = hipStreamWaitEvent(to, ev[i], 0);
                if (e != hipSuccess && first == hipSuccess) first = e;
            }
            n = 0;
            return first;
        }
        ~Join() { (void)run(); }   // error paths: the status is already set
    } join{0, strm, ev_join, stream};
    if (nS > 1) {
        st = ensure_aux(w, nS, 1 + ngroups + nchain + nS);
        if (st != DION2_OK) return st;
        int ei = 0;
        fork = w->ev[ei++];
        for (int g = 0; g < ngroups; ++g) ev_a0[g] = w->ev[ei++];
        for (int c = 0; c < nchain; ++c) ev_chain[c] = w->ev[ei++];
        for (int i = 0; i < nS; ++i) ev_join[i] = w->ev[ei++];
        for (int i = 0; i < nS; ++i) strm[i] = w->aux[i];
        join.n = nS;   // from here on every exit joins
        e = hipEventRecord(fork, stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(fork)");
        for (int i = 0; i < nS; ++i) {
            e = hipStreamWaitEvent(strm[i], fork, 0);
            if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(fork)");
        }
    }
    auto stream_of = [&](int i) { return strm[i % nS]; };

    std::vector<Bufs> bufs(ngroups);
    std::vector<MatSet> sets(ngroups);
    std::vector<dion2_options> gopt(ngroups, opt);
    std::vector<FinalSpec> fins(ngroups);
    int64_t matrix0 = opt.rand_matrix0;
    // pass 1: K1-K3 of every group; DIRECT groups complete, GRAM groups put
    // A_0 into their chain
    for (int g = 0; g < ngroups; ++g) {
        const Plan& P = plans[g];
        const hipStream_t s = stream_of(g);
        MatSet ms{};
        ms.stride = P.rows * P.cols;
        ms.W = groups[g].W;
        ms.M = groups[g].M;
        ms.G = groups[g].G;
        sets[g] = ms;
        gopt[g].rand_matrix0 = matrix0;
        matrix0 += P.batch;
        Bufs b = carve(P, ws + goff[g]);
        const int c = chain_of[g];
        if (c >= 0) {
            const size_t m0 = (size_t)chain_pos[g] * (size_t)P.s_pad * (size_t)P.s_pad;
            for (int i = 0; i < SQ_GRAM_COUNT; ++i) b.sbuf[i] = chain_buf(c, i) + m0;
        }
        bufs[g] = b;
        st = front(P, ms, b, mu, ns_steps, gopt[g], s);
        if (st != DION2_OK) return st;
        fins[g] = make_final(P, ms, b, lr, ns_steps, gopt[g]);
        if (c >= 0) {
            e = gram_a0(P, b.Z0, P.master ? b.Z1 : nullptr, b.sbuf[SQ_AHI], b.sbuf[SQ_ALO],
                        chain_fmt_for(fmt, chains[c].f16), s);
            if (e != hipSuccess) return hip_fail(e, "launch K4 Gram");
            if (nS > 1) {
                e = hipEventRecord(ev_a0[g], s);
                if (e != hipSuccess) return hip_fail(e, "hipEventRecord(A_0)");
            }
            continue;
        }
        if (ns_steps > 0) {
            e = P.gram ? ns_gram(P, b.Z0, P.master ? b.Z1 : nullptr, b.sbuf, b.O, ns_steps, gopt[g], fmt, fins[g], s)
                       : ns_direct(P, b.Z0, b.Z1, b.ZT, b.sbuf, b.O, ns_steps, gopt[g], fins[g], s);
            if (e != hipSuccess) return hip_fail(e, "launch K4 Newton-Schulz");
        }
        st = back(P, ms, b, fins[g], gopt[g], s);
        if (st != DION2_OK) return st;
    }
    // pass 2: each chain's s x s products, all its matrices per launch
    std::vector<int> chain_cur(nchain, 0);
    for (int c = 0; c < nchain; ++c) {
        int first = 0;   // the chain runs on the stream of its first group
        while (chain_of[first] != c) ++first;
        const hipStream_t s = stream_of(first);
        ChainCost cost;
        for (int g = 0; g < ngroups; ++g) {
            if (chain_of[g] != c) continue;
            const ChainCost cg = chain_cost(plans[g], ns_steps, chain_fmt_for(fmt, chains[c].f16), chains[c].fused);
            cost.flops += cg.flops;
            cost.bytes += cg.bytes;
            if (nS > 1) {
                e = hipStreamWaitEvent(s, ev_a0[g], 0);
                if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(A_0)");
            }
        }
        uint16_t* sq[SQ_GRAM_COUNT];
        for (int i = 0; i < SQ_GRAM_COUNT; ++i) sq[i] = chain_buf(c, i);
        e = gram_chain(chains[c].batch, chains[c].s_pad, chains[c].s_k, sq, ns_steps, opt,
                       chain_fmt_for(fmt, chains[c].f16), cost, s, &chain_cur[c], chains[c].fused);
        if (e != hipSuccess) return hip_fail(e, "launch K4 s x s products");
        if (nS > 1) {
            e = hipEventRecord(ev_chain[c], s);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(chain)");
        }
    }
    // pass 3: final products and K5 of the chained groups
    for (int g = 0; g < ngroups; ++g) {
        const int c = chain_of[g];
        if (c < 0) continue;
        const hipStream_t s = stream_of(g);
        if (nS > 1) {
            e = hipStreamWaitEvent(s, ev_chain[c], 0);
            if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(chain)");
        }
        const Plan& P = plans[g];
        const Bufs& b = bufs[g];
        const int cur = chain_cur[c];
        e = gram_final(P, cur ? b.sbuf[SQ_P1HI] : b.sbuf[SQ_P0HI], cur ? b.sbuf[SQ_P1LO] : b.sbuf[SQ_P0LO],
                       b.Z0, P.master ? b.Z1 : nullptr, b.O, fins[g], s);
        if (e != hipSuccess) return hip_fail(e, "launch K4 final product");
        st = back(P, sets[g], b, fins[g], gopt[g], s);
        if (st != DION2_OK) return st;
    }
    e = join.run();
    if (e != hipSuccess) return hip_fail(e, "joining the group streams");
    return DION2_OK;
}

}  // namespace

extern "C" {

void dion2_options_init(dion2_options* opt) {
    if (!opt) return;
    std::memset(opt, 0, sizeof *opt);
    opt->w_dtype = DION2_DTYPE_BF16;
    opt->g_dtype = DION2_DTYPE_BF16;
    opt->ns_coeffs = nullptr;
    opt->ns_eps = 1e-7f;
    opt->decay_all = 0;
    opt->ns_form = DION2_NS_AUTO;
    opt->select_rule = DION2_SELECT_L1;
    opt->rand_seed = 0;
    opt->rand_step = 0;
    opt->rand_matrix0 = 0;
    opt->group_streams = 0;
    opt->ns_chain = DION2_CHAIN_HILO;
    opt->ns_master = DION2_MASTER_BF16;
}

int dion2_step(void* W, float* M, const void* G, int64_t rows, int64_t cols, float alpha,
               float mu, float lr, int ns_steps, int axis, void* stream) {
    return step_impl(W, M, G, nullptr, 1, rows, cols, alpha, mu, lr, ns_steps, axis, nullptr,
                     stream);
}

int dion2_step_strided(void* W, float* M, const void* G, int batch, int64_t rows, int64_t cols,
                       float alpha, float mu, float lr, int ns_steps, int axis, void* stream) {
    return step_impl(W, M, G, nullptr, batch, rows, cols, alpha, mu, lr, ns_steps, axis, nullptr,
                     stream);
}

int dion2_step_batched(void* const* W, float* const* M, const void* const* G, int batch,
                       int64_t rows, int64_t cols, float alpha, float mu, float lr, int ns_steps,
                       int axis, void* stream) {
    Tables t{W, M, G};
    return step_impl(nullptr, nullptr, nullptr, &t, batch, rows, cols, alpha, mu, lr, ns_steps,
                     axis, nullptr, stream);
}

int dion2_step_ex(void* W, float* M, const void* G, int batch, int64_t rows, int64_t cols,
                  float alpha, float mu, float lr, int ns_steps, int axis,
                  const dion2_options* opt, void* stream) {
    return step_impl(W, M, G, nullptr, batch, rows, cols, alpha, mu, lr, ns_steps, axis, opt,
                     stream);
}

int dion2_step_noalloc(void* W, float* M, const void* G, int batch, int64_t rows, int64_t cols,
                       float alpha, float mu, float lr, int ns_steps, int axis,
                       const dion2_options* opt, void* stream) {
    return step_impl(W, M, G, nullptr, batch, rows, cols, alpha, mu, lr, ns_steps, axis, opt,
                     stream, true);
}

int dion2_step_groups(const dion2_group* groups, int ngroups, float alpha, float mu, float lr,
                      int ns_steps, const dion2_options* opt, void* stream) {
    return groups_impl(groups, ngroups, alpha, mu, lr, ns_steps, opt, static_cast<hipStream_t>(stream));
}

size_t dion2_workspace_size(int batch, int64_t rows, int64_t cols, float alpha, int axis) {
    // the largest plan any options take: the GRAM order with the fp32 master
    // (X's lo half beside it and every s x s buffer), or DIRECT (X's
    // ping-pong copy and, from s = 2048, X^T twice) or GRAM with the Random
    // rule's column partials
    struct Case {
        int form;
        bool master, random;
    };
    const Case cases[] = {{DION2_NS_GRAM, true, false}, {DION2_NS_GRAM, false, true}, {DION2_NS_DIRECT, false, true}};
    const std::string saved = g_last_error;   // a size query leaves the last error alone
    size_t best = 0;
    for (const Case& c : cases) {
        Plan P;
        const int st = make_plan(batch, rows, cols, alpha, axis, c.form, 1, &P, true, c.master, c.random);
        if (st == DION2_ERR_UNSUPPORTED && c.form == DION2_NS_DIRECT) continue;   // one tile: no DIRECT
        if (st != DION2_OK) {
            g_last_error = saved;
            return 0;
        }
        best = P.total > best ? P.total : best;
    }
    g_last_error = saved;
    return best;
}

size_t dion2_workspace_size_ex(int batch, int64_t rows, int64_t cols, float alpha, int axis,
                               int ns_steps, const dion2_options* opt_in) {
    dion2_options opt;
    if (opt_in) opt = *opt_in;
    else dion2_options_init(&opt);
    const std::string saved = g_last_error;   // a size query leaves the last error alone
    Plan P;
    const bool ok = validate_common(0.f, 0.f, ns_steps, opt) == DION2_OK &&
                    make_plan(batch, rows, cols, alpha, axis, opt.ns_form, ns_steps, &P, true,
                              opt.ns_master == DION2_MASTER_FP32,
                              opt.select_rule == DION2_SELECT_RANDOM) == DION2_OK;
    g_last_error = saved;
    return ok ? P.total : 0;
}

int dion2_plan_info(int64_t rows, int64_t cols, float alpha, int axis, int64_t* k_out,
                    int* axis_out) {
    Plan P;
    int st = make_plan(1, rows, cols, alpha, axis, DION2_NS_AUTO, 0, &P);
    if (st != DION2_OK) return st;
    if (k_out) *k_out = P.k;
    if (axis_out) *axis_out = P.axis;
    return DION2_OK;
}

int dion2_plan_form(int batch, int64_t rows, int64_t cols, float alpha, int axis, int ns_steps,
                    const dion2_options* opt_in, int* form_out, int* chain_out, int* fused_out) {
    dion2_options opt;
    if (opt_in) opt = *opt_in;
    else dion2_options_init(&opt);
    int st = validate_common(0.f, 0.f, ns_steps, opt);
    if (st != DION2_OK) return st;
    Plan P;
    st = make_plan(batch, rows, cols, alpha, axis, opt.ns_form, ns_steps, &P, true,
                   opt.ns_master == DION2_MASTER_FP32, opt.select_rule == DION2_SELECT_RANDOM);
    if (st != DION2_OK) return st;
    ChainFmt fmt;
    st = chain_format(opt, ns_steps, &fmt);
    if (st != DION2_OK) return st;
    const bool fused = P.gram && ns_steps > 0 && fused_chain(P.s_k, opt);
    if (form_out) *form_out = P.gram ? DION2_NS_GRAM : DION2_NS_DIRECT;
    if (chain_out) *chain_out = P.gram && f16_chain(fmt, fused, P) ? DION2_CHAIN_F16 : DION2_CHAIN_HILO;
    if (fused_out) *fused_out = fused ? 1 : 0;
    return DION2_OK;
}

void dion2_release_workspaces(void) {
    std::lock_guard<std::mutex> lk(g_ws_mutex);
    int prev = -1;
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    for (auto& kv : g_ws) {
        Workspace* w = kv.second;
        std::lock_guard<std::mutex> use(w->use);
        // best effort: a failure here leaves memory to the process's end
        if (hipSetDevice(kv.first.first) == hipSuccess) (void)hipDeviceSynchronize();
        if (w->dev) (void)hipFree(w->dev);
        for (TableSlot& c : w->slots) {
            if (c.host) (void)hipHostFree(c.host);
            if (c.done) (void)hipEventDestroy(c.done);
            c = TableSlot{};
        }
        w->next_slot = 0;
        for (hipStream_t a : w->aux) (void)hipStreamDestroy(a);
        for (hipEvent_t ev : w->ev) (void)hipEventDestroy(ev);
        w->aux.clear();
        w->ev.clear();
        w->dev = nullptr;
        w->bytes = 0;
    }
    if (prev >= 0) (void)hipSetDevice(prev);
}

int dion2_profile_enable(int on) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    const int prev = g_prof.on ? 1 : 0;
    g_prof.on = on != 0;
    return prev;
}

int dion2_profile_read(double* ms, int64_t* calls, int64_t* launches, double* flops,
                       double* bytes, int n) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    for (const ProfRecord& r : g_prof.pending) {
        hipError_t e = hipEventSynchronize(r.stop);
        float t = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, r.start, r.stop);
        if (e != hipSuccess) {
            g_prof.pending.clear();
            return hip_fail(e, "reading profiling events");
        }
        g_prof.ms[r.phase] += t;
        g_prof.calls[r.phase] += 1;
        g_prof.launches[r.phase] += r.launches;
        g_prof.flops[r.phase] += r.flops;
        g_prof.bytes[r.phase] += r.bytes;
        g_prof.pool.push_back(r.start);
        g_prof.pool.push_back(r.stop);
    }
    g_prof.pending.clear();
    if (n < 0) return fail(DION2_ERR_INVALID_ARG, "n must be >= 0");
    if (n > DION2_PHASE_COUNT) n = DION2_PHASE_COUNT;
    for (int i = 0; i < n; ++i) {
        if (ms) ms[i] = g_prof.ms[i];
        if (calls) calls[i] = g_prof.calls[i];
        if (launches) launches[i] = g_prof.launches[i];
        if (flops) flops[i] = g_prof.flops[i];
        if (bytes) bytes[i] = g_prof.bytes[i];
    }
    return DION2_OK;
}

void dion2_profile_reset(void) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    for (const ProfRecord& r : g_prof.pending) {
        (void)hipEventSynchronize(r.stop);   // the events are reused; their times are dropped
        g_prof.pool.push_back(r.start);
        g_prof.pool.push_back(r.stop);
    }
    g_prof.pending.clear();
    for (int i = 0; i < DION2_PHASE_COUNT; ++i) {
        g_prof.ms[i] = 0.0;
        g_prof.calls[i] = 0;
        g_prof.launches[i] = 0;
        g_prof.flops[i] = 0.0;
        g_prof.bytes[i] = 0.0;
    }
}

const char* dion2_status_string(int status) {
    switch (status) {
        case DION2_OK: return "DION2_OK";
        case DION2_ERR_INVALID_ARG: return "DION2_ERR_INVALID_ARG: invalid argument";
        case DION2_ERR_UNSUPPORTED: return "DION2_ERR_UNSUPPORTED: outside what this build handles";
        case DION2_ERR_WORKSPACE: return "DION2_ERR_WORKSPACE: workspace too small or allocation failed";
        case DION2_ERR_HIP: return "DION2_ERR_HIP: a HIP runtime call failed";
        default: return "unknown dion2 status";
    }
}

const char* dion2_last_error(void) { return g_last_error.c_str(); }

int dion2_version(void) { return DION2_VERSION; }

}  // extern "C"
