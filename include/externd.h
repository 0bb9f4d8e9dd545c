/*
 * externd.h -- C ABI of the MI355X (gfx950) ExTernD factorizer.
 *
 * ExTernD approximates a matrix A (m x n) as A ~= B diag(D) C with ternary
 * factors B in {-1,0,1}^{m x k}, C in {-1,0,1}^{k x n} and real scales D,
 * k = mu * min(m, n) (paper: "ExTernD: Expanded-Rank Ternary
 * Decomposition", Sec. 2.1, Eq. (1)).  Components are extracted by greedy
 * alternating least squares with sequential deflation (Sec. 2.3), in blocks
 * of b components with decorrelated least-squares targets (Sec. 2.4,
 * Eq. (3)) and a joint exact scale solve (Eq. (4)); optionally with
 * per-column importance weights (Sec. 2.5; lambda = 0, or any lambda >= 0
 * through externd_factorize_ex).
 *
 * Conventions for every entry point:
 *  - "device" pointers are HIP device memory on the current device (for
 *    example torch.cuda tensor data pointers); "host" pointers are ordinary
 *    CPU memory.
 *  - Matrices are row-major and dense (leading dimension = column count).
 *  - The caller owns every buffer.  The library keeps no pointer to a
 *    caller buffer after a call returns and allocates no device memory;
 *    calls on distinct workspaces and streams are independent.  Calls
 *    sharing a workspace must be ordered (same stream or synchronised by the
 *    caller).  The one piece of global state is the fixed device scratch of
 *    externd_apply_noalloc (below), one copy per device.
 *  - `stream` is a hipStream_t (NULL = the default stream).  All device work
 *    is enqueued on it.
 *  - Errors are returned as negative status codes; no exception crosses the
 *    ABI.  Argument errors are detected on the host before any device work
 *    is enqueued.  On error the contents of output buffers are unspecified
 *    (host energy outputs are set to NaN where given).
 *
 * Packed trit format (B and C outputs): 2 bits per element, element j of a
 * row in byte (j >> 2) at bits 2*(j & 3) .. 2*(j & 3)+1; bit 0 = nonzero,
 * bit 1 = negative: 00 -> 0, 01 -> +1, 11 -> -1 (10 is never written).
 * Each row is padded to a whole byte with zero bits.
 */
#ifndef EXTERND_H
#define EXTERND_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EXTERND_OK            0
#define EXTERND_EINVAL       -1  /* bad scalar argument or NULL required pointer        */
#define EXTERND_ENONFINITE   -2  /* NaN/Inf in A (detected on the device)               */
#define EXTERND_EWORKSPACE   -3  /* workspace smaller than externd_workspace_bytes()    */
#define EXTERND_EHIP         -4  /* HIP runtime or launch failure                       */
#define EXTERND_EUNSUPPORTED -5  /* shape outside the supported range                   */
#define EXTERND_ESYNC        -6  /* a bounded wait between the workgroups of one kernel
                                    launch ran out (the U-step's row groups and the
                                    V-step's last row group of each column tile wait at
                                    most 20 ms for the inverse Gram of the same launch);
                                    the factors of such a call are not to be used       */
#define EXTERND_ESCRATCH     -7  /* the call needs more than the fixed device scratch of
                                    an allocation-free entry point                       */

/* Largest effective block width the kernels handle (four quarters of 64
 * components; the paper's default b = 256, Sec. 2.4).  A call whose
 * effective width (externd_effective_block) exceeds it returns
 * EXTERND_EUNSUPPORTED before any device work; nothing is clamped.
 * Effective widths above 64 run the block as quarters coupled through
 * their Gram inverses and the joint solve; refinement sweeps and the
 * safeguard accept effective widths up to 64 only.                      */
#define EXTERND_MAX_BLOCK 256

/* Ridge of the decorrelated targets, Eq. (3): eps = EXTERND_RIDGE_REL *
 * trace(G) / bb for each Gram matrix G of a block of bb components.      */
#define EXTERND_RIDGE_REL 1e-6
/* Guard of the joint scale solve, Eq. (4): (M + delta I) d = g with
 * delta = EXTERND_SCALE_GUARD_REL * trace(M) / bb.                       */
#define EXTERND_SCALE_GUARD_REL 1e-12

/* Human-readable name of a status code (static string). */
const char* externd_strerror(int status);

/* Inner rank k = floor(mu * min(m, n) + 0.5) (Sec. 2.1); -1 if k < 1 or
 * the arguments are invalid.                                             */
int64_t externd_rank(int64_t m, int64_t n, double mu);

/* Block width actually used: min(block, floor(min(m, n) / 8)), at least
 * 1 (Sec. 2.4 caps b at min(m, n) / 8).  The factorizing entry points
 * return EXTERND_EUNSUPPORTED when it exceeds EXTERND_MAX_BLOCK.  -1 on
 * invalid arguments.                                                     */
int32_t externd_effective_block(int64_t m, int64_t n, int32_t block);

/* Device workspace, in bytes, for an m x n matrix and inner rank k:
 * k = externd_rank(m, n, mu) for externd_factorize, k = 0 for the step
 * entry points.  Independent of block and of whether weights are given:
 * sized for blocks of EXTERND_MAX_BLOCK components, 4 m n bytes for the
 * fp32 residual plus about 5.5 kB per row and (2 + 2 gv) kB per column
 * (gv <= 8 row groups of the V-step's partial contractions) and under
 * 16 MB of fixed buffers.  0 on invalid arguments or unsupported shapes. */
size_t externd_workspace_bytes(int64_t m, int64_t n, int64_t k);

/*
 * externd_factorize -- full greedy block-ALS factorization (Sec. 2.3-2.5).
 *
 *  A          device, fp32 m x n, read only.
 *  m, n       1 <= m <= 2^26, 1 <= n <= 2^20, and with both rounded up to
 *             multiples of 32 their product below 2^31 (else
 *             EXTERND_EUNSUPPORTED).
 *  mu         inner-rank multiplier, k = externd_rank(m, n, mu) >= 1.
 *  tau        threshold scale of T_tau, Eq. (2); finite, >= 0.
 *  block      requested block width b >= 1 (see externd_effective_block;
 *             block = 1 is the sequential algorithm of Sec. 2.3).  An
 *             effective width above EXTERND_MAX_BLOCK (256) is
 *             EXTERND_EUNSUPPORTED.
 *  iters      ALS iterations per block, >= 1; one iteration is a V-step
 *             followed by a U-step (Sec. 2.3 order).
 *  importance device fp32[n] per-column weights h (finite, >= 0, max > 0),
 *             or NULL for the plain Frobenius objective.  h~ = h / max(h).
 *  B_packed   device, m rows of ceil(k/4) bytes (packed trits, B[:, i]).
 *  C_packed   device, k rows of ceil(n/4) bytes (packed trits, C[i, :]).
 *  D          device fp32[k].
 *  energy     host, out: E = 1 - ||A - B diag(D) C||^2 / ||A||^2 (Sec. 2.1)
 *             as tracked on the device residual.
 *  energy_w   host, out (may be NULL): weighted energy
 *             1 - sum_j h~_j ||R_:j||^2 / sum_j h~_j ||A_:j||^2;
 *             equals energy when importance is NULL.
 *  energy_curve, energy_w_curve
 *             host, out (may be NULL): E (resp. weighted E) after each
 *             block, ceil(k / b_eff) doubles.
 *  workspace  device, >= externd_workspace_bytes(m, n, k) bytes, 256-byte
 *             aligned.
 *  stream     hipStream_t or NULL.
 *
 * Enqueues all work on `stream` and synchronises that stream before
 * returning (energies are host outputs).  Deterministic: identical inputs
 * give bit-identical outputs.
 */
int externd_factorize(const float* A, int64_t m, int64_t n, double mu, double tau,
                      int32_t block, int32_t iters, const float* importance,
                      uint8_t* B_packed, uint8_t* C_packed, float* D,
                      double* energy, double* energy_w,
                      double* energy_curve, double* energy_w_curve,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * externd_factorize_ex -- externd_factorize with the two options of the
 * method that the plain call fixes: the lambda of the importance weights
 * and the single-entry safeguard.
 *
 *  lambda     finite, >= 0: h~ = h / max(h) + lambda (Sec. 2.5; lambda
 *             interpolates between the importance-weighted objective at 0
 *             and the plain one as it grows).  Ignored when importance is
 *             NULL.  lambda = 0 gives externd_factorize's result bit for bit.
 *  safeguard  0 or 1.  1: the block form of Proposition 2's augmented step
 *             (Appendix A).  After each block's Eq. (4) solve, the objective
 *             the block removes, 2 d^T g - d^T M d, is compared with the
 *             largest squared residual entry R_ij^2 (the first in row-major
 *             order on ties); when the entry is strictly larger the block
 *             becomes u = e_i, v = sign(R_ij) e_j, d = |R_ij| followed by
 *             zero components, which removes R_ij exactly.  Every block then
 *             removes at least ||R||^2 / (m n).  Plain objective only:
 *             safeguard = 1 with importance != NULL is EXTERND_EINVAL.  When
 *             it never fires the outputs equal those of externd_factorize.
 *  safeguard_fired  host, out (may be NULL): blocks replaced.
 * Other arguments, workspace size, status codes and synchronisation as
 * externd_factorize.
 */
int externd_factorize_ex(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block, int32_t iters,
                         const float* importance, double lambda, int32_t safeguard, uint8_t* B_packed,
                         uint8_t* C_packed, float* D, double* energy, double* energy_w, double* energy_curve,
                         double* energy_w_curve, int64_t* safeguard_fired, void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * externd_factorize_to_energy -- the factorization stopped at an energy
 * target (the paper chooses mu per matrix so that a target accuracy is met
 * exactly, Sec. 1 and Sec. 3; greedy deflation makes every prefix of the
 * components the same as in a longer run, Sec. 2.1).
 *
 *  mu_max         k_max = externd_rank(m, n, mu_max) components at most.
 *  target_energy  finite; after each block the energy E (or, with
 *                 importance, the weighted energy E_w) is compared with
 *                 it, and extraction stops at the first block that
 *                 reaches it (or at k_max).
 *  k_used         host, out: components extracted, a multiple of the
 *                 effective block width, or k_max.
 *  B_packed, C_packed, D, workspace: sized for k_max as in
 *                 externd_factorize; components past k_used are zero.
 *  energy, energy_w: after k_used components.  energy_curve,
 *                 energy_w_curve (may be NULL): room for ceil(k_max / b)
 *                 entries, the first ceil(k_used / b) are written.
 * Other arguments, status codes and synchronisation as externd_factorize.
 * Each block adds one small device-to-host read of the energy history.
 */
int externd_factorize_to_energy(const float* A, int64_t m, int64_t n, double mu_max, double target_energy,
                                double tau, int32_t block, int32_t iters, const float* importance,
                                uint8_t* B_packed, uint8_t* C_packed, float* D, int64_t* k_used, double* energy,
                                double* energy_w, double* energy_curve, double* energy_w_curve, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * externd_factorize_refined -- externd_factorize followed by refinement
 * sweeps (Sec. 2.4: after extraction each block is added back to the
 * residual, fitted again and deflated again, which raises energy
 * monotonically).
 *
 * A sweep revisits the blocks in extraction order.  A revisit forms
 * R' = R + U diag(d) V^T, runs `iters` V-step/U-step iterations of Eq. (3)
 * warm-started from the block's current U, and solves Eq. (4) for the new
 * scales d'.  The new block replaces the old one (in B_packed, C_packed
 * and D) only when the objective it removes from R', 2 d'^T g' - d'^T M' d'
 * (weighted when importance is given), exceeds what the old block removes,
 * ||R'||^2 - ||R||^2; otherwise the old block is deflated again and the
 * outputs keep it.  No revisit therefore increases the objective beyond the
 * rounding of the fp32 residual.
 *
 *  sweeps          >= 0 (0 gives the result of externd_factorize).
 *  energy, energy_w  host, out: after the last sweep.
 *  energy_curve, energy_w_curve  host, out (may be NULL): the extraction's
 *                  per-block curve, as in externd_factorize.
 *  sweep_energy, sweep_energy_w  host, out (may be NULL): E and weighted E
 *                  after each sweep (`sweeps` doubles each).
 *  accepted        host, out (may be NULL): revisits that replaced their
 *                  block, out of sweeps * ceil(k / b_eff).
 * Other arguments, workspace size, status codes and synchronisation as
 * externd_factorize.  Each sweep adds one small device-to-host read.
 */
int externd_factorize_refined(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block,
                              int32_t iters, int32_t sweeps, const float* importance, uint8_t* B_packed,
                              uint8_t* C_packed, float* D, double* energy, double* energy_w, double* energy_curve,
                              double* energy_w_curve, double* sweep_energy, double* sweep_energy_w,
                              int64_t* accepted, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Inference with a factorization (Sec. 2.6 cost model): for each of nb
 * input vectors x (rows of X), y = B (diag(D) (C x)), computed on the packed
 * trits in a fixed order (deterministic).
 *  - One vector with n, k <= 10240: integer matrix cores.  x and the
 *    intermediate t = diag(D) C x enter as 48-bit fixed-point vectors (one
 *    power-of-two scale each: x's from max |x|, t's from the bound
 *    max |D| sum_j |x_j|), so every product and sum is exact; the error is
 *    that of the two conversions and the final rounding: at most
 *    u |y| + 2^-46 [ (|B| (|D| (|C| 1))) max|x| + (|B| 1) max|D| sum|x| ]
 *    per output, u = 2^-24 (entries of x within 2^22 of max |x| convert
 *    exactly).  A NaN or infinite entry of x or D makes every output NaN.
 *  - Otherwise one vector runs on fp32 FMA and two or more on bf16 matrix
 *    cores with exact operands (trits are exact in bf16; every fp32 vector
 *    entry is split exactly into three bf16 parts), with fp32 sums: at most
 *    (n + k + 4) u (|B| (|D| (|C| |x|))) per output, for finite inputs whose
 *    nonzero entries are fp32 normals.
 *
 *  B_packed   device, m rows of ceil(k/4) bytes; C_packed device, k rows of
 *             ceil(n/4) bytes; D device fp32[k] -- as written by
 *             externd_factorize (or _to_energy, whose zero components
 *             contribute nothing).  On the matrix-core path, rows of a
 *             multiple of 8 bytes (nb <= 5) or 16 bytes (nb >= 6) at an
 *             aligned base take whole-word loads.
 *  X          device fp32, nb x n row-major.  Y device fp32, nb x m
 *             row-major (out).
 *  nb         1 <= nb <= EXTERND_APPLY_MAX_BATCH.
 *  workspace  device, >= externd_apply_workspace_bytes(m, n, k, nb) bytes,
 *             256-byte aligned.  nb = 1: the intermediate diag(D) C x
 *             (n, k <= 10240: its six 8-bit digit planes, 1536 bytes per
 *             256 entries, and an exponent word; else 4 k bytes).  nb >= 2: its bf16 parts (6 nb k bytes) and
 *             partial sums over slices of the contracted dimensions (at
 *             most nb max(n, m) k / 32 bytes, rounded up to whole row
 *             groups).
 * Asynchronous on `stream`.  m, n, k <= 2^31 (else EXTERND_EUNSUPPORTED).
 */
#define EXTERND_APPLY_MAX_BATCH 8
size_t externd_apply_workspace_bytes(int64_t m, int64_t n, int64_t k, int32_t nb);  /* 0 on invalid arguments */
int externd_apply(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                  int64_t k, const float* X, int32_t nb, float* Y, void* workspace, size_t workspace_bytes,
                  void* stream);

/*
 * externd_apply without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, arithmetic, results
 * (bit for bit) and status codes as externd_apply, with the workspace held
 * in a fixed device array of the library instead:
 *  - at most EXTERND_APPLY_NOALLOC_MAX_BYTES, i.e.
 *    externd_apply_workspace_bytes(m, n, k, nb) <= that bound (m = 9728,
 *    n = 2560, k = 7680 takes 5.0 MB at nb = 8, 31 kB at nb = 1); larger
 *    calls return EXTERND_ESCRATCH before any device work;
 *  - the array is per device: the current device's copy is used, and the
 *    stream must belong to the current device.  Each device keeps its copy
 *    until the process ends.  The first call on a device looks up the
 *    array's address (hipGetSymbolAddress); no call allocates or frees
 *    device memory;
 *  - every call on a device shares that device's array: calls that overlap
 *    on one device (concurrent streams, or several host threads without
 *    ordering) race and give unspecified results.  Calls ordered on one
 *    stream are safe; nothing needs to be cleared between calls (every
 *    entry a call reads is written earlier in the same call).
 */
#define EXTERND_APPLY_NOALLOC_MAX_BYTES (8u << 20)
int externd_apply_noalloc(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                          int64_t k, const float* X, int32_t nb, float* Y, void* stream);

/* Kernel classes timed by externd_factorize_timed. */
#define EXTERND_KCLASS_VSTEP   0  /* V-step contraction P = U^T R (+ Gram of U, inverse) */
#define EXTERND_KCLASS_USTEP   1  /* U-step contraction Q = R diag(h~) V (+ Gram of V)  */
#define EXTERND_KCLASS_DEFLATE 2  /* deflation R -= U diag(d) V^T (+ column energies)   */
#define EXTERND_KCLASS_VTARGET 3  /* V-step target Y = G_U^{-1} P and its statistics    */
#define EXTERND_KCLASS_UTARGET 4  /* U-step target Z = Q G_V^{-1} and its statistics    */
#define EXTERND_KCLASS_SEQ     5  /* the one-launch sequential path (block width 1 on a
                                     small matrix: every launch is timed)              */
#define EXTERND_KCLASS_TERNV   6  /* V = T_tau(Y^T) per component, Eq. (2)            */
#define EXTERND_KCLASS_TERNU   7  /* U = T_tau(Z) per component, Eq. (2) (+ g = diag(U^T Q)
                                     in the last U-step of a block)                     */
#define EXTERND_KCLASS_COUNT   8

typedef struct {
  double total_ms[EXTERND_KCLASS_COUNT];  /* summed durations of the timed launches */
  int64_t launches[EXTERND_KCLASS_COUNT]; /* number of timed launches of each class */
  int64_t issued[EXTERND_KCLASS_COUNT];   /* number of launches of each class       */
} externd_kernel_times;

/* Launches of each class timed by externd_factorize_timed: one in every
 * EXTERND_TIMING_STRIDE, evenly spread over the call.                    */
#define EXTERND_TIMING_STRIDE 16

/* externd_factorize with HIP events recorded on `stream` around a sample
 * of the launches of the kernel classes above (every
 * EXTERND_TIMING_STRIDE-th launch of a class; the events are created
 * without system-scope fences, so a timed launch ends without an L2
 * write-back, and add a small host-side cost per timed launch).  `times`
 * (host, required) receives the summed durations, the number of timed
 * launches and the number of all launches of each class.  Same outputs and
 * status codes as externd_factorize.                                     */
int externd_factorize_timed(const float* A, int64_t m, int64_t n, double mu, double tau,
                            int32_t block, int32_t iters, const float* importance,
                            uint8_t* B_packed, uint8_t* C_packed, float* D,
                            double* energy, double* energy_w,
                            double* energy_curve, double* energy_w_curve,
                            void* workspace, size_t workspace_bytes, void* stream,
                            externd_kernel_times* times);

/*
 * Step entry points: one step each of the block ALS on caller-given state,
 * for per-step parity checks.  They share the kernels of
 * externd_factorize.  Block matrices are row-major with bb columns:
 * U is m x bb int8 in {-1,0,1}, V is n x bb int8.  1 <= bb <= EXTERND_MAX_BLOCK.
 * Every pointer except `h` / `*_or_null` outputs is required.  These calls
 * are asynchronous on `stream`.
 */

/* Initial U of a block (paper silent; reading: the residual columns with
 * the bb largest h~_j ||R_:j||^2, ties to the smaller index, are
 * ternarized with T_tau, Eq. (2)).  J_out: device int32[bb], the chosen
 * column indices in descending order of weighted energy.                 */
int externd_step_init(const float* R, int64_t m, int64_t n, const float* h, int32_t bb,
                      double tau, int8_t* U_out, int32_t* J_out,
                      void* workspace, size_t workspace_bytes, void* stream);

/* V-step of Eq. (3): Y = (U^T U + eps I)^{-1} U^T R, V[:, c] = T_tau(Y[c, :]).
 * V_out device int8 n x bb; Y_out_or_null device fp64 bb x n.            */
int externd_step_vstep(const float* R, int64_t m, int64_t n, const int8_t* U, int32_t bb,
                       double tau, int8_t* V_out, double* Y_out_or_null,
                       void* workspace, size_t workspace_bytes, void* stream);

/* U-step of Eq. (3) with the weighting of Sec. 2.5:
 * Q = R diag(h~) V, Z = Q (V^T diag(h~) V + eps I)^{-1}, U[:, c] = T_tau(Z[:, c]).
 * h may be NULL (h~ = 1).  U_out device int8 m x bb; Q_out_or_null and
 * Z_out_or_null device fp64 m x bb.                                      */
int externd_step_ustep(const float* R, int64_t m, int64_t n, const int8_t* V, int32_t bb,
                       double tau, const float* h, int8_t* U_out,
                       double* Q_out_or_null, double* Z_out_or_null,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Joint scale solve, Eq. (4): [(U^T U) o (V^T diag(h~) V) + delta I] d =
 * diag(U^T Q) with Q = R diag(h~) V (device fp64 m x bb, as returned by
 * externd_step_ustep).  d_out device fp64[bb].                           */
int externd_step_scale(const int8_t* U, const int8_t* V, const double* Q, int64_t m,
                       int64_t n, int32_t bb, const float* h, double* d_out,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Block deflation R <- R - U diag(d) V^T (Sec. 2.4), in place on the
 * device fp32 m x n matrix R, with d rounded to fp32 (as stored in D).
 * colnorm2_out device fp64[n] (may be NULL): ||R_:j||^2 after the update;
 * fro2_out device fp64[1] (may be NULL): ||R||_F^2 after the update.    */
int externd_step_deflate(float* R, int64_t m, int64_t n, const int8_t* U, const int8_t* V,
                         const double* d, int32_t bb, double* colnorm2_out, double* fro2_out,
                         void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EXTERND_H */
