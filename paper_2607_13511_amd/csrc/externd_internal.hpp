// Internal declarations shared by the kernels and the host orchestration.
// Not part of the public ABI (see include/externd.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "externd.h"

namespace externd {

// Components of a block are padded to BBP; rows and columns of the residual
// are padded to multiples of TILE (zero padding, never touched by updates).
constexpr int BBP = 64;
constexpr int TILE = 32;
// Wide blocks (Sec. 2.4 allows b up to min(m, n) / 8; the paper's default is
// 256): up to NQMAX quarters of BBP components.  Every per-component buffer
// holds BMAX components, quarter q at component 64 q; the kernels above run
// per quarter on a view of the workspace (quarter_view), and the coupling
// between quarters (the Gram matrices of Eq. (3), the joint solve of
// Eq. (4)) runs on BMAX x BMAX fp64 matrices in blocks of 64.
constexpr int NQMAX = 4;
constexpr int BMAX = NQMAX * BBP;
constexpr int NPAIR_MAX = NQMAX * (NQMAX + 1) / 2;  // quarter pairs q <= q'
// Workgroups that build integer Gram matrices (int8 MFMA), beside a
// contraction or in a launch of their own.
constexpr int NSIDE_INT = 8;   // integer-Gram workgroups of the scale solve
constexpr int NSIDE_GRAM = 16; // workgroups of the integer Gram launch
constexpr int NSIDE_MAX = 16;
constexpr int GV_MAX = 8;      // row groups of the V-step contraction
// Workgroups of the contraction kernels resident at once: two per CU on
// 256 CUs (LDS and register budgets of k_vstep / k_ustep).
constexpr int USTEP_SLOTS = 512;
// The same for the deflation kernel (240 VGPRs: two workgroups per CU).
constexpr int DEFLATE_SLOTS = 512;
// Threads per workgroup for all kernels except the selection kernel.
constexpr int NT = 256;
// Weighted Grams on int8 MFMA: the weights h~_j / max h~ as integers of at
// most WSHIFT_MAX bits, split into WDIG digit planes of WDIG_BITS bits.
constexpr int WDIG = 6;
constexpr int WDIG_BITS = 7;
constexpr int WSHIFT_MAX = WDIG * WDIG_BITS;
constexpr int NT_SELECT = 1024;
// Ternarization: workgroups per component (each takes a 32-aligned chunk
// of about TERN_CHUNK entries; at most TERN_SPLIT_MAX per component).
constexpr int TERN_SPLIT_MAX = 8;
constexpr int TERN_CHUNK = 640;

// Index of counters in Ws::counters (each used by one kernel family, reset
// to zero by the workgroup that consumes it).
// CNT_DECISION: the last refinement revisit kept its new block (1) or not;
// CNT_ACCEPTED: revisits of the call that kept the new block.
// CNT_SAFEGUARD: blocks replaced by the single-entry step; CNT_SG_*: the
// last block's single-entry decision (fired, row, column, negative sign);
// CNT_SEQ_USED: components extracted by the persistent sequential path.
// CNT_GINV_V: set to 1 by the U-step's side path once G_V^{-1} is stored
// (the row groups of the same launch wait for it); cleared by k_tern_u.
// CNT_GINV_U: the same for the V-step's G_U^{-1}; cleared by k_tern_v.
enum Counter {
  CNT_GRAM_U = 0, CNT_GRAM_V = 1, CNT_SCALE = 2,
  CNT_DECISION = 5, CNT_ACCEPTED = 6, CNT_SAFEGUARD = 7,
  CNT_SG_FIRE = 8, CNT_SG_ROW = 9, CNT_SG_COL = 10, CNT_SG_NEG = 11, CNT_SEQ_USED = 12, CNT_GINV_V = 13,
  CNT_GINV_U = 14, CNT_COUNT = 16
};
// Flags written by the device, read by the host.
enum Flag { FLAG_NONFINITE = 0, FLAG_BADWEIGHT = 1, FLAG_SYNC = 2, FLAG_COUNT = 4 };

// Device workspace carved out of the caller's buffer.
struct Ws {
  int64_t m, n, m_pad, n_pad;
  int nblk_cap;          // capacity of the per-block arrays (k + 2)
  int gv;                // row groups of the V-step contraction
  int gd;                // row groups of the deflation / staging passes
  int urows, ntu;        // U-step: rows per workgroup (<= 32) and number of row groups
  int nsu, nsv;          // ternarization workgroups per U / V component
  int64_t ntmax;         // statistics tiles per component (the larger of the U and V sides)

  float* R;              // m_pad x n_pad residual, fp32, row-major
  int8_t* Ut;            // BBP x m_pad, U transposed (component-major)
  int8_t* Ur;            // m_pad x BBP, U row-major
  unsigned short* Ub;    // m_pad x BBP, U row-major as bf16 bits (deflation operand)
  int8_t* Vt;            // BBP x n_pad
  int8_t* Vr;            // n_pad x BBP
  int8_t* Umf;           // BBP x m_pad bytes, U in the MFMA-ready operand layout
  int8_t* Vmf;           // BBP x n_pad bytes, V in the MFMA-ready operand layout
  double* tps;           // BBP x tiles: per-32-index-tile sum |x| of a target component
  double* tpm;           // BBP x tiles: per-tile max |x|
  int* tpi;              // BBP x tiles: per-tile smallest index attaining the max
  int* gacc;             // 2 x 4096: integer Gram accumulators of the V-step (U) and U-step (V)
  double* Q;             // BBP x m_pad, Q = R diag(h) V  (component-major)
  double* Z;             // BBP x m_pad, U-step target
  long long* Pp;         // gv x BBP x n_pad, V-step partial contractions
  double* Y;             // BBP x n_pad, V-step target
  double* ginvU;         // BBP x BBP
  double* ginvV;         // BBP x BBP
  double* gramV;         // BBP x BBP raw V^T H V (no ridge)
  int* gparti;           // NSIDE_MAX x BBP x BBP partial integer Grams
  double* colE_part;     // gd x n_pad partial column energies
  double* hw;            // n_pad: h~ (fp64), 1 when unweighted
  double* gvec;          // BBP x TERN_SPLIT_MAX: diag(U^T Q) in per-split partial sums
  double* dvec;          // BBP: joint scales (fp64)
  float* dF;             // BBP: joint scales rounded to fp32
  int* J;                // BBP: init columns
  float* rowb;           // m_pad: upper bound on max_j |R_ij| h~_j per row (h~ = 1 unweighted): the
                         // U-step's fixed-point exponent of row i; measured by every U-step, raised
                         // by every deflation
  float* rowb_part;      // (n_pad/32) x m_pad: per-column-strip row maxima from staging
  double* hwmax;         // 2: max_j h~_j (1 + lambda with weights, 1 without), then the unit of the
                         // weighted integer Grams (max h~ 2^-wshift)
  int* cshift;           // n_pad: the V-step's fixed-point exponent of column j, from ||R_:j||^2
                         // (written with the energy reduction after staging and each deflation)
  unsigned long long* argkey;  // nblk_cap: (max|R| bits << 32) | (2^32 - 1 - first row-major index), safeguard only
  int8_t* hdig;          // WDIG x n_pad: digit planes of the quantized weights (weighted Grams)
  int8_t* Wmf;           // WDIG x BMAX x n_pad: V with row j scaled by digit d of the weight, plane d
                         // at d BMAX n_pad, each plane in the layout of Vmf
  long long* gacc64;     // 4096: weighted Gram accumulator of the U-step (V^T diag(H) V)
  // wide blocks
  int* gaccW;            // NPAIR_MAX x 4096: integer Gram blocks X_q^T X_q' (q <= q') of a factor (int32;
                         // int64 for the weighted Grams of V)
  double* gramVW;        // BMAX x BMAX raw V^T H V (row-major), for the joint solve
  double* wA0;           // BMAX x BMAX: the matrix being swept (ping)
  double* wA1;           // BMAX x BMAX: (pong)
  double* ginvUW;        // NQMAX x NQMAX blocks of 4096 (fp64 MFMA operand order): (U^T U + eps I)^{-1}
  double* ginvVW;        // the same for (V^T H V + eps I)^{-1}
  int* wflag;            // 1: the swept matrix had zero trace
  unsigned* vtcnt;       // n_pad / 32 arrival counters of the V-step's column tiles (zero between launches)
  double* fro2_hist;     // nblk_cap: ||R||^2 before each block, then after the last
  double* fro2w_hist;    // nblk_cap: weighted ||R||^2
  unsigned* counters;    // CNT_COUNT
  int* flags;            // FLAG_COUNT
};

// The workspace as seen by one quarter of a wide block: every per-component
// buffer offset to component 64 q (the shared buffers unchanged).
Ws quarter_view(const Ws& w, int q);

// Optional per-kernel-class event timing (host side).  begin/end record a
// pair of events on the stream around one launch; collect() sums the
// elapsed times after the stream has been synchronised.
struct Timer {
  hipStream_t stream = nullptr;
  struct Mark { hipEvent_t a, b; int cls; };
  Mark* marks = nullptr;
  int n = 0, cap = 0;
  int64_t seen[EXTERND_KCLASS_COUNT] = {};
  // Whether this launch of class cls is one of the sampled ones (every
  // EXTERND_TIMING_STRIDE-th, from the middle of the first stride on).
  // The one-launch sequential path is always timed.
  bool sample(int cls) {
    return (seen[cls]++ % EXTERND_TIMING_STRIDE) == EXTERND_TIMING_STRIDE / 2 || cls == EXTERND_KCLASS_SEQ;
  }
  // The event pair of the next timed launch (created on first use).
  hipError_t take(int cls, hipEvent_t* a, hipEvent_t* b);
  hipError_t collect(double* total_ms, int64_t* launches, int ncls);
  ~Timer();
};
// Launch `kernel`; when `t` is non-null, every EXTERND_TIMING_STRIDE-th
// launch of the class carries start/stop events that the runtime stamps at
// the kernel's own start and end (hipExtLaunchKernelGGL), so the measured
// time excludes dispatch gaps; sampling keeps the host-side cost of the
// events from slowing the launch stream it measures.
#define EXTERND_LAUNCH_TIMED(t, cls, kernel, grid, block, shm, s, ...)          \
  do {                                                                        \
    if ((t) && (t)->sample(cls)) {                                            \
      hipEvent_t _a, _b;                                                      \
      hipError_t _e = (t)->take(cls, &_a, &_b);                               \
      if (_e != hipSuccess) return _e;                                        \
      hipExtLaunchKernelGGL(kernel, grid, block, shm, s, _a, _b, 0, __VA_ARGS__); \
    } else {                                                                  \
      hipLaunchKernelGGL(kernel, grid, block, shm, s, __VA_ARGS__);           \
    }                                                                         \
  } while (0)

size_t workspace_bytes(int64_t m, int64_t n, int64_t k);
bool carve(Ws& w, void* base, size_t bytes, int64_t m, int64_t n, int64_t k);

// ---- launchers (all asynchronous on `s`) ----
// lam: h~ = h / max(h) + lam (Sec. 2.5).
hipError_t launch_prep(const Ws& w, const float* h, hipStream_t s, double lam = 0.0);
// track: also the position of the largest |R| entry (argkey slot 0).
hipError_t launch_stage(const Ws& w, const float* A, int64_t lda, hipStream_t s, bool track = false);
hipError_t launch_select(const Ws& w, int blk, int bb, hipStream_t s);
hipError_t launch_finish(const Ws& w, int blk, hipStream_t s);
hipError_t launch_init(const Ws& w, int bb, double tau, hipStream_t s);
// The contraction launches build the Gram of their factor themselves (side
// workgroups; weighted U-step: V^T diag(H) V from the weights' digit
// planes); launch_gram_acc serves the scale solve.
// weighted: the V-step also writes the digit-scaled planes of V (Wmf) for
// the weighted Gram of the next U-step.
hipError_t launch_vstep(const Ws& w, int blk, int bb, double tau, hipStream_t s, Timer* t = nullptr,
                        bool weighted = false);
// final: the last U-step of a block, which also forms g = diag(U^T Q) for
// the scale solve.
// keep_q: store Q also when the step is not the block's last (the step API
// returns it).
hipError_t launch_ustep(const Ws& w, int blk, int bb, double tau, bool weighted, bool final, hipStream_t s,
                        Timer* t = nullptr, bool keep_q = false);
hipError_t launch_scale(const Ws& w, int bb, hipStream_t s);
// Wide blocks (64 < bb <= BMAX): the same steps over the quarters of the
// block, coupled through the BMAX x BMAX Gram inverses and joint solve.
hipError_t launch_init_wide(const Ws& w, int bb, double tau, hipStream_t s);
hipError_t launch_vstep_wide(const Ws& w, int blk, int bb, double tau, hipStream_t s, Timer* t = nullptr,
                             bool weighted = false);
hipError_t launch_ustep_wide(const Ws& w, int blk, int bb, double tau, bool weighted, bool final, hipStream_t s,
                             Timer* t = nullptr);
hipError_t launch_scale_wide(const Ws& w, int bb, float* D_block, hipStream_t s);
hipError_t launch_gram_wide_raw(const Ws& w, int bb, bool weighted, hipStream_t s);
hipError_t launch_block_out_wide(const Ws& w, int64_t c0, int bb, int64_t k, uint8_t* Bp, uint8_t* Cp, float* D,
                                 hipStream_t s);
hipError_t launch_deflate_wide(const Ws& w, int blk, int bb, bool transposes, hipStream_t s, Timer* t = nullptr);
// The end of a block: scale solve, row-major factor copies, packed B and C, D.
// revisit: the scales were settled by launch_revisit_decide, whose decision
// selects the new block (written out) or the old one (operands rebuilt from
// the packed outputs).
// safeguard: the scales were settled by launch_safeguard, and a block it
// replaced is written out as its single entry.
hipError_t launch_block_out(const Ws& w, int64_t c0, int bb, int64_t k, uint8_t* Bp, uint8_t* Cp, float* D,
                            hipStream_t s, bool revisit = false, bool safeguard = false, bool solve = true);
// Joint scale solve of the block before slot blk's residual is deflated,
// with the single-entry option of Proposition 2 (D_block: D + c0).
hipError_t launch_safeguard(const Ws& w, int blk, int bb, float* D_block, hipStream_t s);
// transposes: rebuild the row-major factor copies from Ut/Vt first (step
// entry point).  Writes max|R| of the result into slot blk + 1.
// track: also the position of the largest |R| entry (argkey of the slot).
hipError_t launch_deflate(const Ws& w, int blk, bool transposes, hipStream_t s, Timer* t = nullptr,
                          bool track = false);
hipError_t launch_deflate_slot(const Ws& w, int out_slot, hipStream_t s, Timer* t = nullptr, bool track = false);
// Refinement revisit of the block at columns c0 .. c0+bb-1: decode it from
// the packed outputs (clearing residual-bound slots slot1 and slot2), and
// after the fit choose between the new and the old block by the objective
// each removes (history slots slot_prev: before the add-back, slot_added:
// after it).
hipError_t launch_revisit_load(const Ws& w, const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t c0, int bb,
                               int64_t k, int slot1, int slot2, hipStream_t s);
hipError_t launch_revisit_decide(const Ws& w, int bb, float* D_block, bool weighted, int slot_prev, int slot_added,
                                 hipStream_t s);
// step-entry helpers
// X: len x bb int8 with leading dimension ld (0: bb).
hipError_t launch_load_factor(int8_t* Xt, int8_t* Xr, int8_t* Xmf, const int8_t* X, int64_t len, int64_t len_pad,
                              int bb, hipStream_t s, int ld = 0);
hipError_t launch_store_factor(int8_t* X, const int8_t* Xt, int64_t len, int64_t len_pad, int bb, hipStream_t s);
hipError_t launch_store_cm(double* X, const double* Xcm, int64_t len, int64_t len_pad, int bb,
                           hipStream_t s);
hipError_t launch_load_cm(double* Xcm, const double* X, int64_t len, int64_t len_pad, int bb,
                          hipStream_t s);
hipError_t launch_unstage(const Ws& w, float* A, hipStream_t s);
hipError_t launch_colnorms(const Ws& w, int blk, double* colnorm2, double* fro2, hipStream_t s);
hipError_t launch_gram_only(const Ws& w, int bb, bool weighted, hipStream_t s);
// The digit-scaled planes of a V loaded from the caller (Wmf), for the
// weighted Gram of the step entry points.
hipError_t launch_vweight(const Ws& w, int bb, hipStream_t s);
hipError_t launch_gvec(const Ws& w, int bb, hipStream_t s);
// X^T X of the factor in Umf (which = 0) or Vmf (which = 1) into its Gram accumulator.
hipError_t launch_gram_acc(const Ws& w, int which, hipStream_t s);
hipError_t launch_set_scales(const Ws& w, const double* d, int bb, hipStream_t s);
// Persistent single-workgroup sequential path (block width 1) for small
// shapes: the whole extraction in one launch (staging included; weights
// from launch_prep).  target: NaN, or stop after the first component whose
// energy reaches it (components extracted in counters[CNT_SEQ_USED]).
bool seq_supported(int64_t m, int64_t n);
hipError_t launch_seq(const Ws& w, const float* A, int64_t k, double tau, int iters, bool weighted, bool safeguard,
                      double target, uint8_t* Bp, uint8_t* Cp, float* D, hipStream_t s, Timer* t = nullptr);

}  // namespace externd
