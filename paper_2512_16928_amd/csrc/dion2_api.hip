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
    int batch;
    int nrb, rb_rows;         // column-mode reduction blocking
    bool gram;                // Newton-Schulz on s x s matrices (DION2_NS_GRAM)
    // workspace offsets
    size_t o_l1, o_sq, o_part, o_sel, o_rank, o_scale, o_Z, o_Z1, o_S, S_bytes, o_O, o_tables, total;
};

// s x s buffers of the two Newton-Schulz forms (bf16 [batch][s_pad][s_pad])
enum { SQ_AHI, SQ_ALO, SQ_B, SQ_DIRECT_COUNT = 3 };
enum { SQ_QHI = 2, SQ_QLO, SQ_THI, SQ_TLO, SQ_P0HI, SQ_P0LO, SQ_P1HI, SQ_P1LO, SQ_GRAM_COUNT };

int make_plan(int batch, int64_t rows, int64_t cols, float alpha, int axis, int ns_form, Plan* p) {
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
    // The GRAM form trades 2 (s x l) GEMMs and the X traffic of every step
    // for about four three-pass s x s products; it pays once X is wide.
    P.gram = ns_form == DION2_NS_GRAM || (ns_form == DION2_NS_AUTO && P.l_pad >= 3 * P.s_pad);
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
    P.o_Z1 = take(P.gram ? 0 : comp);
    P.S_bytes = align256(B * (size_t)P.s_pad * (size_t)P.s_pad * 2);
    P.o_S = take(P.S_bytes * (P.gram ? SQ_GRAM_COUNT : SQ_DIRECT_COUNT));
    P.o_O = take(B * (size_t)P.kpad * (size_t)P.opad * 4);
    P.o_tables = take(3 * B * sizeof(void*));
    P.total = off;
    return DION2_OK;
}

// ------------------------------------------------------------- workspaces

struct Workspace {
    void* dev = nullptr;
    size_t bytes = 0;
    void** pinned = nullptr;       // staging for pointer tables
    size_t pinned_count = 0;
    hipEvent_t tables_done = nullptr;
    bool tables_pending = false;
    std::mutex use;                // serialises host threads sharing a stream
};

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

// Brackets one kernel phase with events when the hooks are on.
class PhaseTimer {
  public:
    PhaseTimer(int phase, double flops, double bytes, int launches, hipStream_t s) : s_(s) {
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

// Z is the wide orientation [s_pad][l_pad] of the compact matrix; O receives
// the result in the L layout [kpad][opad] (the transpose when Z is L^T).

double sym_flops(double s, double inner) { return s * (s + 1.0) * inner; }

GemmArgs gram_args(const Plan& P, const uint16_t* Z, uint16_t* hi, uint16_t* lo) {
    GemmArgs g{};
    g.batch = P.batch;
    g.A0 = g.B0 = Z;
    g.sA = g.sB = P.s_pad * P.l_pad;
    g.M = g.N = (int)P.s_pad;
    g.K = (int)P.l_pad;
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
    q.M = q.N = q.K = (int)P.s_pad;
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
    x.K = (int)P.s_pad;
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

// DIRECT: per step A = Z Z^T (hi / lo), B = b A + c A^2, Z <- a Z + B Z.
hipError_t ns_direct(const Plan& P, uint16_t* Z0, uint16_t* Z1, uint16_t* const* sq, float* O,
                     int ns_steps, const dion2_options& opt, const FinalSpec& fin, hipStream_t stream) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);   // unpadded sides
    const double l_r = (double)(P.k < P.d_oth ? P.d_oth : P.k);
    const double nb = (double)P.batch;
    const double gram_bytes = (2.0 * s_r * l_r + 4.0 * s_r * s_r) * nb;   // Z in, A hi + lo out
    uint16_t* zbuf[2] = {Z0, Z1};
    int cur = 0;
    for (int t = 0; t < ns_steps; ++t) {
        const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
        uint16_t* Z = zbuf[cur];
        GemmArgs g = gram_args(P, Z, sq[SQ_AHI], sq[SQ_ALO]);
        hipError_t e = timed(DION2_PHASE_NS_GRAM, sym_flops(s_r, l_r) * nb, gram_bytes, 1, stream,
                             [&] { return launch_gemm(g, EPI_SPLIT, 1, stream); });
        if (e != hipSuccess) return e;

        GemmArgs q = sym3_args(P, sq[SQ_AHI], sq[SQ_ALO], sq[SQ_AHI], sq[SQ_ALO], sq[SQ_B], nullptr);
        q.cb = cf[1];
        q.cc = cf[2];
        q.E0 = sq[SQ_AHI];
        q.E1 = sq[SQ_ALO];
        q.sE = P.s_pad * P.s_pad;
        q.lde = (int)P.s_pad;
        e = timed(DION2_PHASE_NS_POLY, 3.0 * sym_flops(s_r, s_r) * nb, 6.0 * s_r * s_r * nb, 1, stream,
                  [&] { return launch_gemm(q, EPI_POLY, 3, stream); });
        if (e != hipSuccess) return e;

        // Z' = a Z + B Z (a Z added in the epilogue)
        GemmArgs x = right_args(P, sq[SQ_B], nullptr, Z);
        x.ca = cf[0];
        x.E0 = Z;
        x.sE = P.s_pad * P.l_pad;
        x.lde = (int)P.l_pad;
        const bool last = t + 1 == ns_steps;
        GemmEpi epi = EPI_UPDATE;
        if (!last) {
            x.out0 = zbuf[1 - cur];
            x.sOut0 = P.s_pad * P.l_pad;
            x.ldo0 = (int)P.l_pad;
        } else {
            epi = final_output(P, x, O, fin);
        }
        const double ubytes = (2.0 * s_r * s_r + (last ? 6.0 : 4.0) * s_r * l_r) * nb;
        e = timed(DION2_PHASE_NS_UPDATE, 2.0 * s_r * s_r * l_r * nb, ubytes, 1, stream,
                  [&] { return launch_gemm(x, epi, 1, stream); });
        if (e != hipSuccess) return e;
        cur = 1 - cur;
    }
    return hipSuccess;
}

// GRAM: A_0 = Z Z^T; per step Q_t = a I + b A_t + c A_t^2, P <- Q_t P and
// A_{t+1} = Q_t (Q_t A_t); finally O = P Z. Every s x s matrix is a
// polynomial in A_0, hence symmetric, and all of them commute.
hipError_t ns_gram(const Plan& P, const uint16_t* Z, uint16_t* const* sq, float* O, int ns_steps,
                   const dion2_options& opt, const FinalSpec& fin, hipStream_t stream) {
    const double s_r = (double)(P.k < P.d_oth ? P.k : P.d_oth);
    const double l_r = (double)(P.k < P.d_oth ? P.d_oth : P.k);
    const double nb = (double)P.batch;
    const double f3 = 3.0 * sym_flops(s_r, s_r) * nb;
    const double gram_bytes = (2.0 * s_r * l_r + 4.0 * s_r * s_r) * nb;
    uint16_t* Ah = sq[SQ_AHI];
    uint16_t* Al = sq[SQ_ALO];
    uint16_t* Ph[2] = {sq[SQ_P0HI], sq[SQ_P1HI]};
    uint16_t* Pl[2] = {sq[SQ_P0LO], sq[SQ_P1LO]};
    int cur = 0;

    GemmArgs g = gram_args(P, Z, Ah, Al);
    hipError_t e = timed(DION2_PHASE_NS_GRAM, sym_flops(s_r, l_r) * nb, gram_bytes, 1, stream,
                         [&] { return launch_gemm(g, EPI_SPLIT, 1, stream); });
    if (e != hipSuccess) return e;
    // The s x s products run back to back and are timed as one span. Per
    // step: Q_t (from A: hi + lo in and out, 8 s^2 bytes), P <- Q_t P and
    // T = Q_t A (one dual launch when both are due; each product two hi/lo
    // operands in and one out, 12 s^2, less the shared Q_t's 4 s^2 when
    // fused), A <- Q_t T (12 s^2).
    const int nprod = ns_steps + 3 * (ns_steps - 1);
    const int ndual = ns_steps >= 3 ? ns_steps - 2 : 0;
    const int nlaunch = ns_steps == 1 ? 1 : 3 * ns_steps - 1;
    const double sq_bytes =
        (8.0 * ns_steps + 12.0 * (nprod - ns_steps) - 4.0 * ndual) * s_r * s_r * nb;
    e = timed(DION2_PHASE_NS_POLY, f3 * nprod, sq_bytes, nlaunch, stream, [&]() -> hipError_t {
        for (int t = 0; t < ns_steps; ++t) {
            const float* cf = opt.ns_coeffs ? opt.ns_coeffs + 3 * t : kMuonQuintic;
            // Q_t; the first one is P itself
            uint16_t* qh = t == 0 ? Ph[0] : sq[SQ_QHI];
            uint16_t* ql = t == 0 ? Pl[0] : sq[SQ_QLO];
            GemmArgs q = sym3_args(P, Ah, Al, Ah, Al, qh, ql);
            q.ca = cf[0];
            q.cb = cf[1];
            q.cc = cf[2];
            q.E0 = Ah;
            q.E1 = Al;
            q.sE = P.s_pad * P.s_pad;
            q.lde = (int)P.s_pad;
            hipError_t r = launch_gemm(q, EPI_QPOLY, 3, stream);
            if (r != hipSuccess) return r;
            // P <- Q_t P (t > 0) and T = Q_t A (t < T - 1) share Q_t: one
            // launch when both are due
            const bool do_p = t > 0, do_t = t + 1 < ns_steps;
            if (do_p || do_t) {
                GemmArgs u = do_p ? sym3_args(P, qh, ql, Ph[cur], Pl[cur], Ph[1 - cur], Pl[1 - cur])
                                  : sym3_args(P, qh, ql, Ah, Al, sq[SQ_THI], sq[SQ_TLO]);
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
                GemmArgs v = sym3_args(P, qh, ql, sq[SQ_THI], sq[SQ_TLO], Ah, Al);
                r = launch_gemm(v, EPI_SPLIT, 3, stream);
                if (r != hipSuccess) return r;
            }
        }
        return hipSuccess;
    });
    if (e != hipSuccess) return e;
    // O = (P_hi + P_lo) Z
    GemmArgs x = right_args(P, Ph[cur], Pl[cur], Z);
    const GemmEpi epi = final_output(P, x, O, fin);
    // P hi + lo and Z in, O (or W's selected lines, read and written) out
    const double fbytes = (4.0 * s_r * s_r + 6.0 * s_r * l_r) * nb;
    return timed(DION2_PHASE_NS_UPDATE, 4.0 * s_r * s_r * l_r * nb, fbytes, 1, stream,
                 [&] { return launch_gemm(x, epi, 2, stream); });
}

// ------------------------------------------------------------------ step

struct Tables {
    void* const* W;
    float* const* M;
    const void* const* G;
};

int run_step(const Plan& P, void* W, float* M, const void* G, const Tables* tabs,
             float mu, float lr, int ns_steps, const dion2_options& opt, hipStream_t stream) {
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
        if (w) {
            if (w->tables_pending) {
                e = hipEventSynchronize(w->tables_done);
                if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(tables)");
                w->tables_pending = false;
            }
            if (w->pinned_count < n) {
                if (w->pinned) hipHostFree(w->pinned);
                w->pinned = nullptr;
                w->pinned_count = 0;
                e = hipHostMalloc(reinterpret_cast<void**>(&w->pinned), n * sizeof(void*));
                if (e != hipSuccess) return hip_fail(e, "hipHostMalloc(pointer tables)");
                w->pinned_count = n;
            }
            if (!w->tables_done) {
                e = hipEventCreateWithFlags(&w->tables_done, hipEventDisableTiming);
                if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
            }
            staging = w->pinned;
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
        if (w) {
            e = hipEventRecord(w->tables_done, stream);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(tables)");
            w->tables_pending = true;
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

    double* l1 = reinterpret_cast<double*>(ws + P.o_l1);
    double* sq = reinterpret_cast<double*>(ws + P.o_sq);
    int32_t* sel = reinterpret_cast<int32_t*>(ws + P.o_sel);
    int32_t* rank = P.axis == 1 ? reinterpret_cast<int32_t*>(ws + P.o_rank) : nullptr;
    double* scale = reinterpret_cast<double*>(ws + P.o_scale);
    // compact matrix in its wide orientation: L [kpad][opad] or L^T [opad][kpad]
    uint16_t* Z0 = reinterpret_cast<uint16_t*>(ws + P.o_Z);
    uint16_t* Z1 = reinterpret_cast<uint16_t*>(ws + P.o_Z1);
    uint16_t* sbuf[SQ_GRAM_COUNT];
    for (int i = 0; i < SQ_GRAM_COUNT; ++i)
        sbuf[i] = reinterpret_cast<uint16_t*>(ws + P.o_S + (size_t)i * P.S_bytes);
    float* O = reinterpret_cast<float*>(ws + P.o_O);

    // K1
    MomentumArgs ma{};
    ma.ms = ms;
    ma.rows = P.rows;
    ma.cols = P.cols;
    ma.batch = P.batch;
    ma.l1 = l1;
    ma.sq = sq;
    ma.part = reinterpret_cast<double*>(ws + P.o_part);
    ma.rb_rows = P.rb_rows;
    ma.nrb = P.nrb;
    ma.mu = mu;
    const double n_el = (double)P.batch * (double)P.rows * (double)P.cols;
    const double g_bytes = opt.g_dtype == DION2_DTYPE_BF16 ? 2.0 : 4.0;
    const double w_bytes = opt.w_dtype == DION2_DTYPE_BF16 ? 2.0 : 4.0;
    const double sel_el = (double)P.batch * (double)P.k * (double)P.d_oth;
    // Bytes each phase must move as designed. Rows: K1 reads M, G and writes
    // M; K3 reads and writes the selected rows of M and writes the compact
    // bf16 copy; K5 reads O and reads and writes the selected rows of W.
    // Columns (selected columns touch every cache line of a row): K1 only
    // reads M and G; K3 reads M, G and writes M whole, plus the compact copy;
    // K5 reads O and reads and writes W whole.
    const bool cm = P.axis == 1;
    const double k1_bytes = n_el * ((cm ? 4.0 : 8.0) + g_bytes);
    const double k3_bytes = (cm ? n_el * (8.0 + g_bytes) : sel_el * 8.0) + sel_el * 2.0;
    const double k5_bytes = (cm ? n_el : sel_el) * 2.0 * w_bytes + sel_el * 4.0;
    e = timed(DION2_PHASE_MOMENTUM, 0.0, k1_bytes, P.axis == 0 ? 1 : 2, stream,
              [&] { return launch_momentum(ma, P.axis, opt.g_dtype == DION2_DTYPE_BF16, stream); });
    if (e != hipSuccess) return hip_fail(e, "launch K1 momentum");

    // K2
    SelectArgs sa{};
    sa.l1 = l1;
    sa.sq = sq;
    sa.d_sel = (int)P.d_sel;
    sa.k = (int)P.k;
    sa.batch = P.batch;
    sa.eps = (double)opt.ns_eps;
    sa.sel = sel;
    sa.scale = scale;
    sa.rank = rank;
    sa.rule = opt.select_rule;
    sa.seed = opt.rand_seed;
    sa.step = opt.rand_step;
    sa.matrix0 = opt.rand_matrix0;
    e = timed(DION2_PHASE_SELECT, 0.0, (double)P.batch * (double)P.d_sel * 16.0, 1, stream,
              [&] { return launch_select(sa, stream); });
    if (e != hipSuccess) return hip_fail(e, "launch K2 select");

    // K3
    GatherArgs ga{};
    ga.ms = ms;
    ga.rows = P.rows;
    ga.cols = P.cols;
    ga.batch = P.batch;
    ga.k = (int)P.k;
    ga.d_oth = (int)P.d_oth;
    ga.kpad = (int)P.kpad;
    ga.opad = (int)P.opad;
    ga.sel = sel;
    ga.rank = rank;
    ga.scale = scale;
    ga.mu = mu;
    // rows: selective decay here, decay-all by its own pass; columns: both here
    ga.decay = cm ? (opt.decay_all ? 2 : 1) : (opt.decay_all ? 0 : 1);
    ga.L = P.z_is_L ? Z0 : nullptr;
    ga.LT = P.z_is_L ? nullptr : Z0;
    ga.O = ns_steps == 0 ? O : nullptr;
    e = timed(DION2_PHASE_GATHER, 0.0, k3_bytes, 1, stream,
              [&] { return launch_gather(ga, P.axis, opt.g_dtype == DION2_DTYPE_BF16, stream); });
    if (e != hipSuccess) return hip_fail(e, "launch K3 gather");
    if (opt.decay_all && !cm) {
        DecayAllArgs da{ms, P.rows, P.cols, P.batch, mu};
        e = launch_decay_all(da, stream);
        if (e != hipSuccess) return hip_fail(e, "launch decay-all");
    }

    // K4: Newton-Schulz
    FinalSpec fin{};
    fin.lr_eff = (double)lr * std::sqrt((double)P.rows / (double)P.cols);
    fin.fuse = ns_steps > 0 && P.axis == 0 && P.z_is_L && opt.w_dtype == DION2_DTYPE_BF16 &&
               P.cols % 8 == 0 && P.cols >= 16;
    fin.ms = ms;
    fin.sel = sel;
    fin.dbg = opt.dbg_update;
    if (ns_steps > 0) {   // with no step the gather has written O
        e = P.gram ? ns_gram(P, Z0, sbuf, O, ns_steps, opt, fin, stream)
                   : ns_direct(P, Z0, Z1, sbuf, O, ns_steps, opt, fin, stream);
    }
    if (e != hipSuccess) return hip_fail(e, "launch K4 Newton-Schulz");

    // K5
    ApplyArgs aa{};
    aa.ms = ms;
    aa.rows = P.rows;
    aa.cols = P.cols;
    aa.batch = P.batch;
    aa.k = (int)P.k;
    aa.d_oth = (int)P.d_oth;
    aa.kpad = (int)P.kpad;
    aa.opad = (int)P.opad;
    aa.sel = sel;
    aa.rank = rank;
    aa.O = O;
    aa.lr_eff = fin.lr_eff;
    aa.dbg = opt.dbg_update;
    if (!fin.fuse) {   // otherwise the final Newton-Schulz product has applied it
        e = timed(DION2_PHASE_APPLY, 0.0, k5_bytes, 1, stream,
                  [&] { return launch_apply(aa, P.axis, opt.w_dtype == DION2_DTYPE_BF16, stream); });
        if (e != hipSuccess) return hip_fail(e, "launch K5 apply");
    }

    if (opt.dbg_sel_idx) {
        e = hipMemcpyAsync(opt.dbg_sel_idx, sel, (size_t)P.batch * P.k * 4, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "copy dbg_sel_idx");
    }
    if (opt.dbg_norms) {
        e = hipMemcpyAsync(opt.dbg_norms, l1, (size_t)P.batch * P.d_sel * 8, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "copy dbg_norms");
    }
    return DION2_OK;
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
    if (opt.ns_coeffs) {
        for (int i = 0; i < 3 * ns_steps; ++i)
            if (!std::isfinite(opt.ns_coeffs[i]))
                return fail(DION2_ERR_INVALID_ARG, "ns_coeffs[%d] is not finite", i);
    }
    return DION2_OK;
}

int step_impl(void* W, float* M, const void* G, const Tables* tabs, int batch, int64_t rows,
              int64_t cols, float alpha, float mu, float lr, int ns_steps, int axis,
              const dion2_options* opt_in, void* stream) {
    dion2_options opt;
    if (opt_in) opt = *opt_in;
    else dion2_options_init(&opt);
    Plan P;
    int st = make_plan(batch, rows, cols, alpha, axis, opt.ns_form, &P);
    if (st != DION2_OK) return st;
    st = validate_common(mu, lr, ns_steps, opt);
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
    if (opt.workspace) {
        if ((reinterpret_cast<uintptr_t>(opt.workspace) & 255u) != 0)
            return fail(DION2_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
        if (opt.workspace_bytes < P.total)
            return fail(DION2_ERR_WORKSPACE, "workspace of %zu bytes is below the %zu needed",
                        opt.workspace_bytes, P.total);
    }
    return run_step(P, W, M, G, tabs, mu, lr, ns_steps, opt, static_cast<hipStream_t>(stream));
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

size_t dion2_workspace_size(int batch, int64_t rows, int64_t cols, float alpha, int axis) {
    Plan P;
    if (make_plan(batch, rows, cols, alpha, axis, DION2_NS_AUTO, &P) != DION2_OK) return 0;
    return P.total;
}

int dion2_plan_info(int64_t rows, int64_t cols, float alpha, int axis, int64_t* k_out,
                    int* axis_out) {
    Plan P;
    int st = make_plan(1, rows, cols, alpha, axis, DION2_NS_AUTO, &P);
    if (st != DION2_OK) return st;
    if (k_out) *k_out = P.k;
    if (axis_out) *axis_out = P.axis;
    return DION2_OK;
}

void dion2_release_workspaces(void) {
    std::lock_guard<std::mutex> lk(g_ws_mutex);
    int prev = -1;
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    for (auto& kv : g_ws) {
        Workspace* w = kv.second;
        std::lock_guard<std::mutex> use(w->use);
        if (hipSetDevice(kv.first.first) == hipSuccess) hipDeviceSynchronize();
        if (w->dev) hipFree(w->dev);
        if (w->pinned) hipHostFree(w->pinned);
        if (w->tables_done) hipEventDestroy(w->tables_done);
        w->dev = nullptr;
        w->bytes = 0;
        w->pinned = nullptr;
        w->pinned_count = 0;
        w->tables_done = nullptr;
        w->tables_pending = false;
    }
    if (prev >= 0) hipSetDevice(prev);
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
        hipEventSynchronize(r.stop);
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
