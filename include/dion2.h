/*
 * dion2.h -- C ABI of the Dion2 optimizer step for AMD Instinct MI355X (gfx950).
 *
 * The step is Algorithm 1 of "Dion2: A Simple Method to Shrink Matrix in
 * Muon" (Ahn, Amsel, Langford), applied to every matrix of a batch of
 * same-shape weight matrices W (rows x cols = fan-out x fan-in, y = W x):
 *
 *   M <- M + G                              accumulate
 *   K <- Select_alpha(M)                    k = ceil(alpha * d_sel) lines of
 *                                           largest l1 norm (Default rule)
 *   O <- NewtonSchulz(M[K, :])              only the selected submatrix
 *   M[K, :] <- mu * M[K, :]                 selective decay, eq. (2)
 *   W[K, :] <- W[K, :] - lr*sqrt(rows/cols)*O   sparse update, eq. (1)
 *
 * (rows shown; with axis = columns the same is done on M[:, K], W[:, K]).
 *
 * Numerical contract:
 *   - M is fp32; the accumulate and the decay are single IEEE fp32 RNE
 *     operations (bitwise reproducible).
 *   - The l1 norm of each line is accumulated in double-double from the fp32
 *     values of M and rounded once to fp64, in an order fixed by the shape,
 *     so selection does not depend on scheduling. It equals the exact sum of
 *     |M_ij| rounded once to fp64, except when that exact sum S lies within
 *     about n^2 2^-106 S (n the line's length) of a point halfway between
 *     two adjacent fp64 values: there the low word's own rounding can move
 *     the result by one unit. Ties go to the lower index; NaN ranks as
 *     +inf. K is ascending. (dion2_options.select_rule selects the Random
 *     rule.)
 *   - Newton-Schulz: X = M[K,:] / (||M[K,:]||_F + eps), then per step
 *     A = X X^T, B = b A + c A^2, X <- a X + B X on the orientation with the
 *     smaller Gram matrix (s x s, X is s x l, s <= l); X is rounded once to
 *     bf16 and every product runs on bf16 MFMA operands with fp32
 *     accumulation. Two evaluation orders give the same result in exact
 *     arithmetic (dion2_options.ns_form):
 *       DIRECT  the steps as written, X kept in bf16 between steps, A kept
 *               in fp16 with a power-of-two scale bounded from the
 *               coefficients (fp16 MFMA, one pass for A^2), or, for
 *               coefficients that take A beyond fp16's range, as a bf16
 *               hi/lo pair with three passes for A^2;
 *       GRAM    the iteration carried on s x s matrices: with
 *               Q_t = a I + b A_t + c A_t^2 one has X_{t+1} = Q_t X_t and
 *               A_{t+1} = Q_t A_t Q_t, so X_T = (Q_{T-1} ... Q_0) X_0, and X
 *               is read only twice. The s x s matrices are kept either as
 *               bf16 hi/lo pairs (three MFMA passes per product) or in fp16
 *               with a power-of-two scale per kind of matrix, derived from
 *               the coefficients so that no value overflows or falls into
 *               fp16's subnormal range (one pass, less accurate on
 *               ill-conditioned inputs; dion2_options.ns_chain).
 *               The final product takes P_T as a bf16 hi/lo pair (two
 *               passes).
 *     With dion2_options.ns_master = DION2_MASTER_FP32, X itself is kept as
 *     a bf16 hi/lo pair (about 16 significant bits) instead of being rounded
 *     once to bf16: the Gram matrix and the final product take three passes,
 *     and the iteration runs in the GRAM order.
 *     Default coefficients are Muon's quintic (3.4445, -4.7750, 2.0315) at
 *     every step, eps = 1e-7.
 *   - The weight update is computed in fp64 from the fp32 O and rounded once
 *     (RNE) to W's storage type. Unselected lines of W are not written.
 *
 * Conventions shared by every entry point:
 *   - W, M, G are DEVICE pointers to row-major, contiguous matrices, owned
 *     by the caller; the library never frees or keeps them. Each base
 *     pointer must be 16-byte aligned. W and M are updated in place; G is
 *     read-only. Matrices of one call must not overlap.
 *   - stream is a hipStream_t (NULL = the default stream). Calls are
 *     asynchronous: nothing is synchronised and no result returns to the
 *     host. Calls on one stream are serialised by the stream.
 *   - Arguments are validated before anything is launched or allocated; on
 *     any error nothing is modified and a negative dion2_status is returned.
 *     dion2_last_error() gives a message for the calling thread.
 *   - Without a caller workspace the library keeps one internal workspace
 *     per (device, stream) and grows it with hipMalloc when needed (the
 *     growth synchronises the device). Concurrent calls on different
 *     streams use different workspaces; concurrent calls on one stream
 *     from several host threads are serialised by a lock.
 *   - Limits: 1 <= rows, cols; rows * cols < 2^31; 1 <= batch <= 65535;
 *     0 < alpha <= 1; 0 <= ns_steps <= DION2_MAX_NS_STEPS; mu, lr finite.
 */
#ifndef DION2_H
#define DION2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DION2_VERSION 1
/* Accuracy and step count: with Muon's quintic, the stated 2e-2 bound on O
   holds at its 5 steps (on compact matrices of a few lines the 16-bit s x s
   chain has reached 2.1e-2 to 2.8e-2: 3 x 3 to 9 x 6 with ns_eps 1e-3). The quintic has no attracting fixed point (its slope
   inside the band reaches about 1.58), so each further step enlarges the
   bf16 rounding of the normalised input: the exact iteration on that rounded
   input can already lie more than 2e-2 from the exact result after 6 to 16
   steps on compact matrices of a few lines, and near-square ones drift past
   it after about 12. Longer schedules keep the bound when their steps after
   the fifth contract toward 1, e.g. cubic Newton-Schulz (1.5, -0.5, 0)
   through ns_coeffs, on compact matrices at least three times as long as
   high (l >= 3 s). Past DION2_DIRECT_MAX_STEPS every call runs the GRAM
   form, whose s x s matrices resolve singular values down to about 2^-8 of
   the largest; near-square compact matrices have many below that, and a
   schedule that lifts them toward 1 moves O by up to 7e-2 there. On compact
   matrices of deficient or nearly deficient rank (low rank plus a little
   noise, repeated lines) the GRAM form's rounding can leave A's eigenvalues
   in the null space slightly negative, and every step multiplies those by
   more than a^2 (a = 3.4445 for the quintic): from about 8 steps the chain
   can diverge and O overflow. Such momentum stays at the paper's 5 steps. */
#define DION2_MAX_NS_STEPS 16

typedef enum dion2_status {
    DION2_OK = 0,
    DION2_ERR_INVALID_ARG = -1, /* a bad pointer, size or hyperparameter      */
    DION2_ERR_UNSUPPORTED = -2, /* valid but outside what this build handles  */
    DION2_ERR_WORKSPACE = -3,   /* caller workspace too small / alloc failure */
    DION2_ERR_HIP = -4          /* a HIP runtime call failed                  */
} dion2_status;

typedef enum dion2_axis {
    DION2_AXIS_AUTO = -1, /* the shorter dimension; square selects rows (Sec. 4) */
    DION2_AXIS_ROWS = 0,  /* select rows:    M[K, :], W[K, :]                     */
    DION2_AXIS_COLS = 1   /* select columns: M[:, K], W[:, K]                     */
} dion2_axis;

typedef enum dion2_dtype {
    DION2_DTYPE_F32 = 0,
    DION2_DTYPE_BF16 = 1
} dion2_dtype;

typedef enum dion2_select_rule {
    DION2_SELECT_L1 = 0,     /* the k lines of largest l1 norm (default)         */
    DION2_SELECT_RANDOM = 1  /* k lines uniformly at random: the k smallest of
                                Philox-4x32-10 keys, see dion2_options          */
} dion2_select_rule;

typedef enum dion2_ns_form {
    DION2_NS_AUTO = 0,   /* GRAM when l >= 3 s or s <= 128 (padded sides) or
                            ns_steps > DION2_DIRECT_MAX_STEPS, else DIRECT     */
    DION2_NS_DIRECT = 1, /* iterate on X (s x l). X is rounded to bf16 after
                            every step, so the error grows with the step
                            count and is largest where few directions carry
                            it: at most DION2_DIRECT_MAX_STEPS steps, and
                            only for s > 128 (more than one tile a side);
                            other calls return DION2_ERR_UNSUPPORTED        */
    DION2_NS_GRAM = 2    /* iterate on s x s matrices, X read twice            */
} dion2_ns_form;

/* The most Newton-Schulz steps the DIRECT form runs. An emulation of its
   bf16 arithmetic on near-square compact matrices puts the relative
   Frobenius error of O at about 1.6e-2 after 6 steps and 2.1e-2 after 8,
   against 1.2e-2 after the default 5; the GRAM form stays at its 5-step
   error. On compact matrices of one tile a side (s <= 128) the same
   emulation reached 3.6e-2 after 5 steps (s = 3) and 2.2e-2 after 6
   (s = 32), so DIRECT is refused there; AUTO takes GRAM on them anyway. */
#define DION2_DIRECT_MAX_STEPS 6

typedef enum dion2_ns_chain {
    DION2_CHAIN_HILO = 0, /* GRAM s x s matrices as bf16 hi/lo pairs (default)  */
    DION2_CHAIN_F16 = 1   /* GRAM s x s matrices in scaled fp16: one MFMA pass
                             per product instead of three. The Gram matrix
                             squares Z's condition number, and fp16 keeps 11
                             significant bits, so accuracy drops for inputs
                             whose spectrum is dominated by a few directions
                             (kappa(Z)^2 beyond about 2^11); balanced wide
                             inputs stay within 2x of HILO. Taken only on
                             compact matrices at least four times as long
                             as high (l >= 4 s) with s > 64; elsewhere
                             (near-square ones, where it measured up to 0.4
                             from the exact iteration, 2.3e-2 at l = 2.8 s,
                             and the one-launch chains of s <= 64) the chain
                             stays in HILO. With ns_coeffs that take the
                             chain's values beyond 2^40 the call fails with
                             DION2_ERR_UNSUPPORTED; a chain of one step
                             (ns_steps = 1) uses HILO.                        */
} dion2_ns_chain;

typedef enum dion2_ns_master {
    DION2_MASTER_BF16 = 0, /* X rounded once to bf16 (default)                 */
    DION2_MASTER_FP32 = 1  /* X as a bf16 hi/lo pair through every product: the
                              GRAM order with hi/lo s x s matrices, three-pass
                              Gram and final products. Needs ns_form AUTO or
                              GRAM (DIRECT: DION2_ERR_UNSUPPORTED) and ns_chain
                              HILO (F16: DION2_ERR_INVALID_ARG). Costs three
                              times the Gram products and 1.5 times the final
                              one; on wide compact matrices the result is 10
                              to 70 times closer to the exact iteration. On
                              near-square ones the GRAM order squares their
                              condition number and the hi/lo chain limits it
                              (1.2e-2 measured at 78 x 90), still within the
                              2e-2 bound. Where X is of low rank plus a little
                              noise, rounding it once to bf16 moves even the
                              exact iteration by about 0.1 (rank 32 plus 1e-2
                              noise, 128 x 2048): the default lands there, the
                              master within 2e-2                              */
} dion2_ns_master;

/* Full-control options for dion2_step_ex. Fill with dion2_options_init. */
typedef struct dion2_options {
    int w_dtype;             /* storage type of W (default DION2_DTYPE_BF16)        */
    int g_dtype;             /* storage type of G (default DION2_DTYPE_BF16)        */
    const float* ns_coeffs;  /* HOST array [ns_steps][3] of (a, b, c) per step;
                                NULL = Muon's quintic at every step                */
    float ns_eps;            /* Frobenius-normalisation eps (default 1e-7), >= 0   */
    int decay_all;           /* 0 = selective decay, eq. (2) (default);
                                1 = decay all of M (the ablation of Sec. 4.2)      */
    void* workspace;         /* DEVICE scratch of workspace_bytes, 256-B aligned,
                                or NULL for the library-managed workspace          */
    size_t workspace_bytes;  /* >= dion2_workspace_size(...) when workspace set    */
    int32_t* dbg_sel_idx;    /* optional DEVICE out [batch][k]: K, ascending       */
    double* dbg_norms;       /* optional DEVICE out [batch][d_sel]: l1 norms       */
    float* dbg_update;       /* optional DEVICE out [batch][k][d_oth]: O, one
                                selected line per row (row k of O^T for columns),
                                before the lr*sqrt(rows/cols) scale                 */
    int ns_form;             /* dion2_ns_form (default DION2_NS_AUTO)               */
    int select_rule;         /* dion2_select_rule (default DION2_SELECT_L1).
                                RANDOM (Algorithm 1, selection step; Sec. 3.1):
                                line i of matrix b gets the 64-bit key made of the
                                first two output words (high first) of
                                Philox-4x32-10 with counter (i, rand_matrix0 + b,
                                rand_step low, rand_step high) and key (rand_seed
                                low, rand_seed high); the k smallest keys are
                                selected, ties to the lower index             */
    uint64_t rand_seed;      /* RANDOM: generator key (default 0)                   */
    uint64_t rand_step;      /* RANDOM: optimizer step, so each step draws anew     */
    int64_t rand_matrix0;    /* RANDOM: index of the batch's first matrix; >= 0 and
                                rand_matrix0 + batch <= 2^32                       */
    int group_streams;       /* dion2_step_groups: how many streams the groups may
                                run on at once (0 = the library's choice, 1 = all
                                on the call's stream, at most 8)                   */
    int ns_chain;            /* dion2_ns_chain (default DION2_CHAIN_HILO)           */
    int ns_master;           /* dion2_ns_master (default DION2_MASTER_BF16)         */
    uint16_t* dbg_compact;   /* optional DEVICE out [batch][k][d_oth] bf16 bits: X,
                                the normalised submatrix Newton-Schulz starts from
                                (Algorithm 1, orthonormalisation step), selected
                                line p in row p; each entry is
                                bf16(fl32(M[K] * fl32(1 / (||M[K]||_F + eps))))
                                from the accumulated momentum, the hi half with
                                DION2_MASTER_FP32. Written with ns_steps 0 too  */
    uint16_t* dbg_compact_lo;/* optional DEVICE out, same layout: the lo halves
                                bf16(x - hi) of X's fp32 values; only with
                                DION2_MASTER_FP32 and ns_steps >= 1, else the
                                call returns DION2_ERR_INVALID_ARG              */
    int ns_chain_per_product;/* GRAM form: 0 (default) runs the chain of s x s
                                products of a compact matrix with s <= 64 in one
                                launch, its matrices kept in LDS as hi / lo pairs
                                whatever ns_chain says; nonzero gives every
                                product its own launch. Bitwise the same result */
} dion2_options;

/* Defaults: bf16 W and G, Muon quintic, eps 1e-7, selective decay, internal
   workspace, no debug outputs, Newton-Schulz form chosen by shape with a
   hi/lo s x s chain and X rounded once to bf16, l1 rule. */
void dion2_options_init(dion2_options* opt);

/* One matrix. W, G: bf16 [rows][cols]; M: fp32 [rows][cols]. Algorithm 1. */
int dion2_step(void* W, float* M, const void* G, int64_t rows, int64_t cols,
               float alpha, float mu, float lr, int ns_steps, int axis,
               void* stream);

/* A batch of same-shape matrices as contiguous stacks: W, G bf16
   [batch][rows][cols]; M fp32 [batch][rows][cols]. Every matrix gets its own
   selection and Newton-Schulz (Algorithm 1 per matrix); the kernels are
   batched across the stack. */
int dion2_step_strided(void* W, float* M, const void* G, int batch,
                       int64_t rows, int64_t cols, float alpha, float mu,
                       float lr, int ns_steps, int axis, void* stream);

/* A batch of same-shape matrices given by HOST arrays of DEVICE pointers
   (W[i], G[i] bf16, M[i] fp32, each [rows][cols]): the step of Algorithm 1
   for every matrix, each with its own selection and Newton-Schulz, as in
   dion2_step_strided. The tables are read into pinned staging before the
   call returns, so the caller may reuse them at once; the copy to the device
   is queued on `stream`. The host does not wait for the device, except when
   more than 8 calls with pointer tables are still queued on one stream (it
   then waits for the oldest one's table copy). The batch must not exceed 64
   matrices when the tables cannot be staged (no library workspace). */
int dion2_step_batched(void* const* W, float* const* M, const void* const* G,
                       int batch, int64_t rows, int64_t cols, float alpha,
                       float mu, float lr, int ns_steps, int axis,
                       void* stream);

/* Strided stacks with full control; opt == NULL means defaults. Per matrix
   this is Algorithm 1 with the choices the options expose:
     - selection by the Default (l1) rule or the Random rule (Algorithm 1,
       selection step; Sec. 3.1), select_rule;
     - the selective decay of eq. (2) (Algorithm 1, decay step), or the
       decay of all of M, the ablation of Sec. 4.2 (decay_all);
     - the Newton-Schulz iteration of Algorithm 1's orthonormalisation step
       (Sec. 1) with a per-step coefficient table, eps, evaluation order and
       precision (ns_coeffs, ns_eps, ns_form, ns_chain, ns_master);
     - the storage types of W and G, a caller workspace and debug outputs.
   Errors as for every entry point; in addition DION2_ERR_UNSUPPORTED for
   ns_form DIRECT with more than DION2_DIRECT_MAX_STEPS steps or a compact
   matrix of at most 128 lines a side, and
   DION2_ERR_WORKSPACE for a caller workspace smaller than
   dion2_workspace_size_ex gives for the same arguments. */
int dion2_step_ex(void* W, float* M, const void* G, int batch, int64_t rows,
                  int64_t cols, float alpha, float mu, float lr, int ns_steps,
                  int axis, const dion2_options* opt, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc): the step
   of dion2_step_ex, bitwise the same results, with the workspace taken from
   a fixed device array of DION2_NOALLOC_SCRATCH_BYTES that each GPU the
   library runs on holds until the process ends. The call allocates no
   device memory (no hipMalloc, hipFree or allocating library routine) and
   takes strided stacks only. opt->workspace must be NULL
   (DION2_ERR_INVALID_ARG otherwise); a call whose workspace
   (dion2_workspace_size_ex) exceeds the array fails with DION2_ERR_WORKSPACE
   before anything runs. Every call on one GPU uses that GPU's one array, and
   nothing in it needs to start at zero: calls whose kernels overlap on one
   GPU (on different streams, say) race and give wrong results; calls queued
   on one stream, or otherwise ordered, are safe. The measurement hooks do
   not time its phases. */
#define DION2_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int dion2_step_noalloc(void* W, float* M, const void* G, int batch,
                       int64_t rows, int64_t cols, float alpha, float mu,
                       float lr, int ns_steps, int axis,
                       const dion2_options* opt, void* stream);

/* One same-shape group for dion2_step_groups: contiguous DEVICE stacks W
   and G [batch][rows][cols] in the storage types of the options, M fp32
   [batch][rows][cols], each 16-byte aligned, and the group's selection axis
   (DION2_AXIS_*). */
typedef struct dion2_group {
    void* W;
    float* M;
    const void* G;
    int batch;
    int64_t rows, cols;
    int axis;
} dion2_group;

/* The step of Algorithm 1 for several same-shape groups in one call on one
   stream, with shared hyper-parameters and options (a model's whole layer
   stack, say; every matrix is stepped independently, as Algorithm 1 is per
   matrix, with the options' meaning as in dion2_step_ex). The result is bitwise that of dion2_step_ex called for each
   group in order; for the RANDOM rule group g's matrix indices start at
   rand_matrix0 plus the batches of groups 0 .. g-1. Groups whose
   Newton-Schulz runs in the GRAM form with the same padded s x s size share
   one batched chain of s x s products, launched once for all of them.
   groups is a HOST array of ngroups entries, read before the call returns.
   The groups are independent until their chains, so they may run
   concurrently on internal streams of default priority (opt->group_streams);
   those fork from `stream` and are joined back into it before the call
   returns: work queued on `stream` before the call is done before any of
   it starts, and work queued after waits for all of it.
   The workspace is the library's (opt->workspace must be NULL) and the debug
   outputs must be NULL. Errors: DION2_ERR_INVALID_ARG for ngroups outside
   [1, 64], a NULL array or stack pointer, an unaligned stack, a set
   workspace or debug output, group_streams outside [0, 8]; the status
   dion2_step_ex would return for an argument it rejects for some group
   (nothing is modified in either case); DION2_ERR_HIP if an internal stream
   or event cannot be created. */
int dion2_step_groups(const dion2_group* groups, int ngroups, float alpha,
                      float mu, float lr, int ns_steps,
                      const dion2_options* opt, void* stream);

/* Bytes of device workspace (for dion2_options.workspace) that suffice for
   a call with these arguments under any options and step count: the
   largest of the GRAM order with DION2_MASTER_FP32, and the GRAM and DIRECT
   orders under the Random rule (whose column selection keeps per-block
   partial sums; DIRECT only where it is accepted, s > 128). Returns 0 for
   invalid arguments. */
size_t dion2_workspace_size(int batch, int64_t rows, int64_t cols,
                            float alpha, int axis);

/* Bytes of device workspace a dion2_step_ex call with exactly these
   arguments and options needs (opt == NULL: defaults; the options'
   workspace and debug pointers are ignored). Returns 0 where dion2_step_ex
   would reject the arguments or options. */
size_t dion2_workspace_size_ex(int batch, int64_t rows, int64_t cols,
                               float alpha, int axis, int ns_steps,
                               const dion2_options* opt);

/* Number of selected lines k = ceil(alpha * d_sel) clamped to [1, d_sel]
   and the resolved axis (DION2_AXIS_ROWS / _COLS), for sizing debug
   outputs. Returns DION2_OK or DION2_ERR_INVALID_ARG. */
int dion2_plan_info(int64_t rows, int64_t cols, float alpha, int axis,
                    int64_t* k_out, int* axis_out);

/* How a dion2_step_ex call with these arguments would evaluate the
   Newton-Schulz iteration of Algorithm 1 (orthonormalisation step), for
   callers that check or log the choice: *form_out receives DION2_NS_DIRECT or
   DION2_NS_GRAM (what AUTO resolves to), *chain_out the storage the GRAM
   chain takes (DION2_CHAIN_F16 only where ns_chain asks for it and the
   compact matrix qualifies; DION2_CHAIN_HILO otherwise and for DIRECT), and
   *fused_out 1 where the GRAM chain runs as one launch (s <= 64 and
   ns_chain_per_product 0), else 0. Host-only: no GPU call, nothing
   allocated, W, M and G not needed. opt may be NULL (defaults); any output
   pointer may be NULL. Returns what the call's own validation of the shape,
   alpha, ns_steps and options would return (e.g. DION2_ERR_UNSUPPORTED for a
   forced DIRECT on one tile), leaving the outputs unset on error. */
int dion2_plan_form(int batch, int64_t rows, int64_t cols, float alpha,
                    int axis, int ns_steps, const dion2_options* opt,
                    int* form_out, int* chain_out, int* fused_out);

/* ---- Measurement hooks ---------------------------------------------------
 * While enabled, every kernel phase of subsequent calls is bracketed by HIP
 * events recorded on the call's stream (the Newton-Schulz s x s products of
 * the GRAM form, which run back to back, as one span), and the phase's
 * algorithmic work is added to per-phase totals, as flops and as bytes:
 *   bytes: what the phase must move as designed. MOMENTUM: M and G read, M
 *     written (rows) or M and G read (columns). GATHER: the selected lines of
 *     M read and written and the compact bf16 copy written (rows), or M and
 *     G read and M written whole plus the compact copy (columns). APPLY: O
 *     read and the selected lines of W read and written (rows), or W read
 *     and written whole (columns). Newton-Schulz: each product's distinct
 *     operands read and its result written (the Gram matrix: X in, A hi/lo
 *     or fp16 out; an s x s product: two hi/lo or fp16 operands in, one
 *     out; the final product: X in, O (or W's selected lines, read and
 *     written) out).
 *   flops: MFMA flops of the Newton-Schulz GEMMs, every bf16 hi/lo pass
 *     included, a product with a symmetric result counted at s (s + 1) per
 *     inner index (the half it computes) instead of 2 s^2: the Gram matrix
 *     s (s + 1) l, a three-pass s x s product 3 s (s + 1) s, the update B X
 *     2 s^2 l and the two-pass final product of the GRAM form 4 s^2 l (s <= l
 *     are the compact matrix's unpadded sides); 0 for the other phases.
 * The events cost a little time, so the step time is measured with the
 * hooks off. */
typedef enum dion2_phase {
    DION2_PHASE_MOMENTUM = 0,  /* K1: M += G and line norms         */
    DION2_PHASE_SELECT = 1,    /* K2: top-k selection               */
    DION2_PHASE_GATHER = 2,    /* K3: compact gather + decay        */
    DION2_PHASE_NS_GRAM = 3,   /* K4: A = X X^T (hi/lo or fp16)     */
    DION2_PHASE_NS_POLY = 4,   /* K4: the s x s products            */
    DION2_PHASE_NS_UPDATE = 5, /* K4: X <- a X + B X, or O = P X_0  */
    DION2_PHASE_APPLY = 6,     /* K5: scatter-apply into W          */
    DION2_PHASE_COUNT = 7
} dion2_phase;

/* on != 0 enables the hooks, 0 disables them; returns the previous state. */
int dion2_profile_enable(int on);

/* Waits for the recorded events and writes, for the first n phases, the
   summed kernel milliseconds, the number of spans timed, the kernel launches
   and the summed algorithmic flops and bytes (as above). Any output pointer
   may be NULL. Totals accumulate until dion2_profile_reset. */
int dion2_profile_read(double* ms, int64_t* calls, int64_t* launches, double* flops,
                       double* bytes, int n);

void dion2_profile_reset(void);

/* Frees the library-managed workspaces (synchronises each device first). */
void dion2_release_workspaces(void);

/* Static description of a status code. */
const char* dion2_status_string(int status);

/* Message describing the last error returned on the calling thread. */
const char* dion2_last_error(void);

int dion2_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DION2_H */
