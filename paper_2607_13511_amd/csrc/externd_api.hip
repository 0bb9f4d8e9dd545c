// C-ABI entry points of the ExTernD factorizer (declared in include/externd.h).
//
// Host orchestration of the greedy block ALS (paper Sec. 2.3-2.5): argument
// validation, workspace carving, the sequential loop over blocks
// (deflation across blocks is sequential, Sec. 2.4), and the read-back of
// the energy history.  All arithmetic runs in the kernels of
// externd_kernels.hip.
#include "externd.h"
#include "externd_internal.hpp"

#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>
#include <vector>

namespace externd {

static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
static inline int64_t round_up(int64_t x, int64_t q) { return (x + q - 1) / q * q; }
static inline int clampi(int64_t v, int64_t lo, int64_t hi) { return (int)(v < lo ? lo : (v > hi ? hi : v)); }

struct Layout {
  int64_t m_pad, n_pad;
  int gv, gd, nblk_cap;
  int urows, ntu, nsu, nsv;
  size_t off[48];
  size_t total;
};

static int64_t stat_tiles(int64_t nrt, int64_t nct, int64_t ntu) {
  const int64_t a = nrt > 2 * nct ? nrt : 2 * nct;
  return a > ntu ? a : ntu;
}

static Layout make_layout(int64_t m, int64_t n, int64_t k) {
  Layout L{};
  L.m_pad = round_up(m, TILE);
  L.n_pad = round_up(n, TILE);
  const int64_t nct = L.n_pad / TILE, nrt = L.m_pad / TILE;
  // V-step: about 480 column-tile x row-group workgroups.  Deflation and
  // staging: as many row groups as keep the whole deflation grid resident
  // in one pass (a second, partial pass leaves its CUs moving 1.5 shares of
  // the residual while the others idle).
  L.gv = clampi((480 + nct - 1) / nct, 1, nrt < GV_MAX ? nrt : GV_MAX);
  L.gd = clampi(DEFLATE_SLOTS / nct, 1, nrt < 64 ? nrt : 64);
  // U-step: equal row groups of at most 32 rows, as many as fit beside the
  // side workgroups in one pass of USTEP_SLOTS resident workgroups, so
  // that every CU streams the same share of R.  NSIDE_MAX more slots stay
  // empty: those that the dispatcher places beside the side workgroups
  // (ntu counts them; the launch maps them out).
  L.urows = clampi((L.m_pad + (USTEP_SLOTS - 2 * NSIDE_MAX) - 1) / (USTEP_SLOTS - 2 * NSIDE_MAX), 1, TILE);
  L.ntu = (int)((L.m_pad + L.urows - 1) / L.urows) + NSIDE_MAX;
  L.nsu = clampi((L.m_pad + TERN_CHUNK - 1) / TERN_CHUNK, 1, TERN_SPLIT_MAX);
  L.nsv = clampi((L.n_pad + TERN_CHUNK - 1) / TERN_CHUNK, 1, TERN_SPLIT_MAX);
  L.nblk_cap = (int)(k + 2);  // fro2 before every block and after the last; one spare
  // statistics tiles: 32-row tiles (initial gather, wide U-steps) or the
  // U-step's row groups on the U side, 16-column tiles on the V side
  const int64_t ntmax = stat_tiles(nrt, nct, L.ntu);
  const size_t sizes[] = {
      sizeof(float) * (size_t)(L.m_pad * L.n_pad),     // 0 R
      (size_t)(BMAX * L.m_pad),                        // 1 Ut
      (size_t)(BMAX * L.m_pad),                        // 2 Ur
      (size_t)(BMAX * L.n_pad),                        // 3 Vt
      (size_t)(BMAX * L.n_pad),                        // 4 Vr
      sizeof(double) * (size_t)(BMAX * L.m_pad),       // 5 Q
      sizeof(double) * (size_t)(BMAX * L.m_pad),       // 6 Z
      sizeof(long long) * (size_t)(L.gv * BMAX * L.n_pad),  // 7 Pp
      sizeof(double) * (size_t)(BMAX * L.n_pad),       // 8 Y
      sizeof(double) * 4096,                           // 9 ginvU
      sizeof(double) * 4096,                           // 10 ginvV
      sizeof(double) * 4096,                           // 11 gramV
      sizeof(long long) * 4096,                        // 12 gacc64
      sizeof(int) * 4096 * NSIDE_MAX,                  // 13 gparti
      sizeof(double) * (size_t)(L.gd * L.n_pad),       // 14 colE_part
      sizeof(double) * (size_t)L.n_pad,                // 15 hw
      sizeof(double) * BMAX * TERN_SPLIT_MAX,          // 16 gvec
      sizeof(double) * BMAX,                           // 17 dvec
      sizeof(float) * BMAX,                            // 18 dF
      sizeof(int) * BMAX,                              // 19 J
      sizeof(float) * (size_t)L.m_pad,                 // 20 rowb
      sizeof(double) * (size_t)L.nblk_cap,             // 21 fro2_hist
      sizeof(double) * (size_t)L.nblk_cap,             // 22 fro2w_hist
      sizeof(unsigned) * CNT_COUNT,                    // 23 counters
      sizeof(int) * FLAG_COUNT,                        // 24 flags
      sizeof(float) * (size_t)(nct * L.m_pad),         // 25 rowb_part
      (size_t)(BMAX * L.m_pad),                        // 26 Umf
      (size_t)(BMAX * L.n_pad),                        // 27 Vmf
      sizeof(double) * (size_t)(BMAX * ntmax),         // 28 tps
      sizeof(double) * (size_t)(BMAX * ntmax),         // 29 tpm
      sizeof(int) * (size_t)(BMAX * ntmax),            // 30 tpi
      sizeof(unsigned short) * (size_t)(BMAX * L.m_pad),  // 31 Ub
      sizeof(unsigned long long) * (size_t)L.nblk_cap, // 32 argkey
      sizeof(int) * 2 * 4096,                          // 33 gacc
      (size_t)(WDIG * L.n_pad),                        // 34 hdig
      sizeof(double) * 2,                              // 35 hwmax
      sizeof(int) * (size_t)L.n_pad,                   // 36 cshift
      sizeof(long long) * 4096 * NPAIR_MAX,            // 37 gaccW (int32 Grams, int64 weighted Grams)
      sizeof(double) * BMAX * BMAX,                    // 38 gramVW
      sizeof(double) * BMAX * BMAX,                    // 39 wA0
      sizeof(double) * BMAX * BMAX,                    // 40 wA1
      (size_t)(WDIG * BMAX * L.n_pad),                 // 41 Wmf
      sizeof(double) * BMAX * BMAX,                    // 42 ginvUW
      sizeof(double) * BMAX * BMAX,                    // 43 ginvVW
      sizeof(unsigned) * (size_t)(L.n_pad / TILE),    // 44 vtcnt
      sizeof(int) * 64,                                // 45 wflag
  };
  size_t o = 0;
  for (size_t i = 0; i < sizeof(sizes) / sizeof(sizes[0]); ++i) {
    L.off[i] = o;
    o += align256(sizes[i]);
  }
  L.total = o;
  return L;
}

size_t workspace_bytes(int64_t m, int64_t n, int64_t k) { return make_layout(m, n, k).total; }

bool carve(Ws& w, void* base, size_t bytes, int64_t m, int64_t n, int64_t k) {
  const Layout L = make_layout(m, n, k);
  if (bytes < L.total || base == nullptr || ((uintptr_t)base & 255u) != 0) return false;
  char* b = (char*)base;
  w.m = m;
  w.n = n;
  w.m_pad = L.m_pad;
  w.n_pad = L.n_pad;
  w.nblk_cap = L.nblk_cap;
  w.gv = L.gv;
  w.gd = L.gd;
  w.urows = L.urows;
  w.ntu = L.ntu;
  w.nsu = L.nsu;
  w.nsv = L.nsv;
  w.R = (float*)(b + L.off[0]);
  w.Ut = (int8_t*)(b + L.off[1]);
  w.Ur = (int8_t*)(b + L.off[2]);
  w.Vt = (int8_t*)(b + L.off[3]);
  w.Vr = (int8_t*)(b + L.off[4]);
  w.Q = (double*)(b + L.off[5]);
  w.Z = (double*)(b + L.off[6]);
  w.Pp = (long long*)(b + L.off[7]);
  w.Y = (double*)(b + L.off[8]);
  w.ginvU = (double*)(b + L.off[9]);
  w.ginvV = (double*)(b + L.off[10]);
  w.gramV = (double*)(b + L.off[11]);
  w.gparti = (int*)(b + L.off[13]);
  w.colE_part = (double*)(b + L.off[14]);
  w.hw = (double*)(b + L.off[15]);
  w.gvec = (double*)(b + L.off[16]);
  w.dvec = (double*)(b + L.off[17]);
  w.dF = (float*)(b + L.off[18]);
  w.J = (int*)(b + L.off[19]);
  w.rowb = (float*)(b + L.off[20]);
  w.fro2_hist = (double*)(b + L.off[21]);
  w.fro2w_hist = (double*)(b + L.off[22]);
  w.counters = (unsigned*)(b + L.off[23]);
  w.flags = (int*)(b + L.off[24]);
  w.rowb_part = (float*)(b + L.off[25]);
  w.Umf = (int8_t*)(b + L.off[26]);
  w.Vmf = (int8_t*)(b + L.off[27]);
  w.tps = (double*)(b + L.off[28]);
  w.tpm = (double*)(b + L.off[29]);
  w.tpi = (int*)(b + L.off[30]);
  w.Ub = (unsigned short*)(b + L.off[31]);
  w.argkey = (unsigned long long*)(b + L.off[32]);
  w.gacc = (int*)(b + L.off[33]);
  w.hdig = (int8_t*)(b + L.off[34]);
  w.Wmf = (int8_t*)(b + L.off[41]);
  w.gacc64 = (long long*)(b + L.off[12]);
  w.hwmax = (double*)(b + L.off[35]);
  w.cshift = (int*)(b + L.off[36]);
  w.gaccW = (int*)(b + L.off[37]);
  w.gramVW = (double*)(b + L.off[38]);
  w.wA0 = (double*)(b + L.off[39]);
  w.wA1 = (double*)(b + L.off[40]);
  w.ginvUW = (double*)(b + L.off[42]);
  w.ginvVW = (double*)(b + L.off[43]);
  w.wflag = (int*)(b + L.off[45]);
  w.vtcnt = (unsigned*)(b + L.off[44]);
  const int64_t nrt = L.m_pad / TILE, nct = L.n_pad / TILE;
  w.ntmax = stat_tiles(nrt, nct, L.ntu);
  return true;
}

Ws quarter_view(const Ws& w, int q) {
  Ws v = w;
  const int64_t c0 = (int64_t)BBP * q;
  v.Ut = w.Ut + c0 * w.m_pad;
  v.Ur = w.Ur + c0 * w.m_pad;
  v.Ub = w.Ub + c0 * w.m_pad;
  v.Umf = w.Umf + c0 * w.m_pad;
  v.Q = w.Q + c0 * w.m_pad;
  v.Z = w.Z + c0 * w.m_pad;
  v.Vt = w.Vt + c0 * w.n_pad;
  v.Vr = w.Vr + c0 * w.n_pad;
  v.Vmf = w.Vmf + c0 * w.n_pad;
  v.Wmf = w.Wmf + c0 * w.n_pad;
  v.Y = w.Y + c0 * w.n_pad;
  v.Pp = w.Pp + c0 * w.gv * w.n_pad;
  v.tps = w.tps + c0 * w.ntmax;
  v.tpm = w.tpm + c0 * w.ntmax;
  v.tpi = w.tpi + c0 * w.ntmax;
  v.gvec = w.gvec + c0 * TERN_SPLIT_MAX;
  v.dvec = w.dvec + c0;
  v.dF = w.dF + c0;
  v.J = w.J + c0;
  return v;
}

hipError_t Timer::take(int cls, hipEvent_t* a, hipEvent_t* b) {
  if (n == cap) {
    const int ncap = cap ? 2 * cap : 1024;
    Mark* nm = new Mark[ncap];
    for (int i = 0; i < n; ++i) nm[i] = marks[i];
    delete[] marks;
    marks = nm;
    for (int i = cap; i < ncap; ++i) {
      marks[i].a = nullptr;
      marks[i].b = nullptr;
    }
    cap = ncap;
  }
  Mark& mk = marks[n];
  if (!mk.a) {
    // timing only: no system-scope fence (no L2 write-back at the timed
    // kernel's end, which would lengthen the very launch being measured)
    hipError_t e = hipEventCreateWithFlags(&mk.a, hipEventDisableSystemFence);
    if (e != hipSuccess) return e;
    e = hipEventCreateWithFlags(&mk.b, hipEventDisableSystemFence);
    if (e != hipSuccess) return e;
  }
  mk.cls = cls;
  *a = mk.a;
  *b = mk.b;
  ++n;
  return hipSuccess;
}

hipError_t Timer::collect(double* total_ms, int64_t* launches, int ncls) {
  for (int c = 0; c < ncls; ++c) {
    total_ms[c] = 0.0;
    launches[c] = 0;
  }
  for (int i = 0; i < n; ++i) {
    float ms = 0.0f;
    hipError_t e = hipEventElapsedTime(&ms, marks[i].a, marks[i].b);
    if (e != hipSuccess) return e;
    if (marks[i].cls >= 0 && marks[i].cls < ncls) {
      total_ms[marks[i].cls] += ms;
      launches[marks[i].cls] += 1;
    }
  }
  return hipSuccess;
}

Timer::~Timer() {
  for (int i = 0; i < cap; ++i) {
    if (marks[i].a) (void)hipEventDestroy(marks[i].a);
    if (marks[i].b) (void)hipEventDestroy(marks[i].b);
  }
  delete[] marks;
}

}  // namespace externd

using namespace externd;

// ---------------------------------------------------------------------------
// validation helpers
// ---------------------------------------------------------------------------
static const int64_t kMaxDim = (int64_t)1 << 26;

static bool shape_ok(int64_t m, int64_t n) {
  if (m < 1 || n < 1 || m > kMaxDim || n > ((int64_t)1 << 20)) return false;
  const int64_t mp = (m + TILE - 1) / TILE * TILE, np = (n + TILE - 1) / TILE * TILE;
  return mp * np < ((int64_t)1 << 31);
}

#define HIP_TRY(expr)                               \
  do {                                              \
    hipError_t _e = (expr);                         \
    if (_e != hipSuccess) return EXTERND_EHIP;      \
  } while (0)

extern "C" {

const char* externd_strerror(int status) {
  switch (status) {
    case EXTERND_OK: return "ok";
    case EXTERND_EINVAL: return "invalid argument";
    case EXTERND_ENONFINITE: return "non-finite value in the input matrix";
    case EXTERND_EWORKSPACE: return "workspace too small or misaligned";
    case EXTERND_EHIP: return "HIP runtime or launch failure";
    case EXTERND_EUNSUPPORTED: return "unsupported shape";
    case EXTERND_ESYNC: return "device-side synchronisation between workgroups timed out";
    case EXTERND_ESCRATCH: return "call exceeds the fixed device scratch of an allocation-free entry point";
    default: return "unknown status";
  }
}

int64_t externd_rank(int64_t m, int64_t n, double mu) {
  if (m < 1 || n < 1 || !(mu > 0.0) || !isfinite(mu)) return -1;
  const double kk = floor(mu * (double)(m < n ? m : n) + 0.5);
  if (kk < 1.0 || kk > 9.0e15) return -1;
  return (int64_t)kk;
}

int32_t externd_effective_block(int64_t m, int64_t n, int32_t block) {
  if (m < 1 || n < 1 || block < 1) return -1;
  int64_t cap = (m < n ? m : n) / 8;
  if (cap < 1) cap = 1;
  int64_t b = block;
  if (b > cap) b = cap;
  return (int32_t)b;
}

size_t externd_workspace_bytes(int64_t m, int64_t n, int64_t k) {
  if (!shape_ok(m, n) || k < 0) return 0;
  return externd::workspace_bytes(m, n, k);
}

// Refinement sweeps after extraction (Sec. 2.4): every block in turn is
// added back to R, fitted again from its current U, and the better of the
// old and the new block (by the objective removed from R + U diag(d) V^T)
// is deflated.  The per-pass history slots (residual bound, ||R||^2) are
// used as a ring of nblk_cap >= 3 entries from slot S on; the extraction's
// energy curve has been read before.
struct SweepOut {
  double* energy;     // host, sweeps entries (may be null)
  double* energy_w;   // host, sweeps entries (may be null)
  double fro2_last, fro2w_last;
};
static hipError_t run_sweeps(const Ws& w, int64_t k, int b_eff, double tau, int32_t iters, int32_t sweeps,
                             bool weighted, uint8_t* B_packed, uint8_t* C_packed, float* D, int S, double a2,
                             double a2w, SweepOut& out, hipStream_t s, Timer* tm) {
  const int64_t nblk = (k + b_eff - 1) / b_eff;
  const int cap = w.nblk_cap;
  hipError_t e;
#define SWEEP_TRY(expr)          \
  do {                           \
    e = (expr);                  \
    if (e != hipSuccess) return e; \
  } while (0)
  for (int sw = 0; sw < sweeps; ++sw) {
    for (int64_t blk = 0; blk < nblk; ++blk) {
      const int64_t c0 = blk * b_eff;
      const int bb = (int)((k - c0) < b_eff ? (k - c0) : b_eff);
      const int S1 = (S + 1) % cap, S2 = (S + 2) % cap;
      SWEEP_TRY(launch_revisit_load(w, B_packed, C_packed, D, c0, bb, k, S1, S2, s));
      SWEEP_TRY(launch_deflate_slot(w, S1, s, tm));  // R' = R + U diag(d) V^T
      SWEEP_TRY(launch_finish(w, S1, s));
      for (int it = 0; it < iters; ++it) {
        SWEEP_TRY(launch_vstep(w, S1, bb, tau, s, tm, weighted));
        SWEEP_TRY(launch_ustep(w, S1, bb, tau, weighted, it == iters - 1, s, tm));
      }
      SWEEP_TRY(launch_gram_acc(w, 0, s));
      SWEEP_TRY(launch_revisit_decide(w, bb, D + c0, weighted, S, S1, s));
      SWEEP_TRY(launch_block_out(w, c0, bb, k, B_packed, C_packed, D, s, true));
      SWEEP_TRY(launch_deflate_slot(w, S2, s, tm));
      SWEEP_TRY(launch_finish(w, S2, s));
      S = S2;
    }
    double f[2];
    SWEEP_TRY(hipMemcpyAsync(&f[0], w.fro2_hist + S, sizeof(double), hipMemcpyDeviceToHost, s));
    SWEEP_TRY(hipMemcpyAsync(&f[1], w.fro2w_hist + S, sizeof(double), hipMemcpyDeviceToHost, s));
    SWEEP_TRY(hipStreamSynchronize(s));
    out.fro2_last = f[0];
    out.fro2w_last = f[1];
    if (out.energy) out.energy[sw] = a2 == 0.0 ? 1.0 : 1.0 - f[0] / a2;
    if (out.energy_w) out.energy_w[sw] = a2w == 0.0 ? 1.0 : 1.0 - f[1] / a2w;
  }
#undef SWEEP_TRY
  return hipSuccess;
}

// target: NaN for the full run; else stop after the first block whose
// energy (E, or E_w with weights) reaches it, reporting *k_used.
// sweeps: refinement sweeps after a full run (0 = none).
// lam: h~ = h / max(h) + lam (Sec. 2.5).  safeguard: the single-entry
// option of Proposition 2 per block (plain objective), counted in *fired.
static int factorize_impl(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block, int32_t iters,
                          const float* importance, uint8_t* B_packed, uint8_t* C_packed, float* D, double* energy,
                          double* energy_w, double* energy_curve, double* energy_w_curve, void* workspace,
                          size_t workspace_bytes, void* stream, externd_kernel_times* times,
                          double target = NAN, int64_t* k_used = nullptr, int32_t sweeps = 0,
                          double* sweep_energy = nullptr, double* sweep_energy_w = nullptr,
                          int64_t* accepted = nullptr, double lam = 0.0, bool safeguard = false,
                          int64_t* fired = nullptr) {
  if (energy) *energy = NAN;
  if (energy_w) *energy_w = NAN;
  if (!A || !B_packed || !C_packed || !D || !energy || !workspace) return EXTERND_EINVAL;
  if (m < 1 || n < 1 || !isfinite(tau) || tau < 0.0 || block < 1 || iters < 1 || sweeps < 0) return EXTERND_EINVAL;
  if (!isfinite(lam) || lam < 0.0 || (safeguard && importance)) return EXTERND_EINVAL;
  const bool stop_at_target = !isnan(target);
  if (stop_at_target && (!isfinite(target) || !k_used || sweeps > 0)) return EXTERND_EINVAL;
  const int64_t k = externd_rank(m, n, mu);
  if (k < 1) return EXTERND_EINVAL;
  if (!shape_ok(m, n)) return EXTERND_EUNSUPPORTED;
  const int b_eff = externd_effective_block(m, n, block);
  // the kernels hold at most EXTERND_MAX_BLOCK components of a block; wide
  // blocks (more than 64) run without refinement sweeps and the safeguard
  if (b_eff > EXTERND_MAX_BLOCK) return EXTERND_EUNSUPPORTED;
  const bool wide = b_eff > BBP;
  if (wide && (sweeps > 0 || safeguard)) return EXTERND_EUNSUPPORTED;
  const int64_t nblk = (k + b_eff - 1) / b_eff;
  Ws w{};
  if (!carve(w, workspace, workspace_bytes, m, n, k)) return EXTERND_EWORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  const bool weighted = importance != nullptr;
  Timer timer;
  timer.stream = s;
  Timer* tm = times ? &timer : nullptr;

  // Block width 1 on a small matrix: the whole extraction in one launch.
  const bool one_launch = b_eff == 1 && sweeps == 0 && seq_supported(m, n);
  int flags[FLAG_COUNT];
  HIP_TRY(launch_prep(w, importance, s, lam));
  if (stop_at_target) {
    // components past the stop stay zero
    HIP_TRY(hipMemsetAsync(B_packed, 0, (size_t)m * (size_t)((k + 3) / 4), s));
    HIP_TRY(hipMemsetAsync(C_packed, 0, (size_t)k * (size_t)((n + 3) / 4), s));
    HIP_TRY(hipMemsetAsync(D, 0, sizeof(float) * (size_t)k, s));
  }
  int64_t nblk_done = nblk;
  if (one_launch) {
    HIP_TRY(launch_seq(w, A, k, tau, iters, weighted, safeguard, stop_at_target ? target : NAN, B_packed, C_packed,
                       D, s, tm));
    unsigned used = 0;
    HIP_TRY(hipMemcpyAsync(flags, w.flags, sizeof(flags), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(&used, w.counters + CNT_SEQ_USED, sizeof(unsigned), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (flags[FLAG_BADWEIGHT]) return EXTERND_EINVAL;
    if (flags[FLAG_NONFINITE]) return EXTERND_ENONFINITE;
    nblk_done = (int64_t)used;
  } else {
    HIP_TRY(launch_stage(w, A, n, s, safeguard));
    HIP_TRY(hipMemcpyAsync(flags, w.flags, sizeof(flags), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (flags[FLAG_BADWEIGHT]) return EXTERND_EINVAL;
    if (flags[FLAG_NONFINITE]) return EXTERND_ENONFINITE;
    for (int64_t blk = 0; blk < nblk; ++blk) {
      const int64_t c0 = blk * b_eff;
      const int bb = (int)((k - c0) < b_eff ? (k - c0) : b_eff);
      HIP_TRY(launch_select(w, (int)blk, bb, s));
      if (bb > BBP) {
        // a wide block: its quarters coupled through the Gram inverses
        HIP_TRY(launch_init_wide(w, bb, tau, s));
        for (int it = 0; it < iters; ++it) {
          HIP_TRY(launch_vstep_wide(w, (int)blk, bb, tau, s, tm, weighted));
          HIP_TRY(launch_ustep_wide(w, (int)blk, bb, tau, weighted, it == iters - 1, s, tm));
        }
        HIP_TRY(launch_block_out_wide(w, c0, bb, k, B_packed, C_packed, D, s));
        HIP_TRY(launch_deflate_wide(w, (int)blk, bb, false, s, tm));
      } else {
        HIP_TRY(launch_init(w, bb, tau, s));
        for (int it = 0; it < iters; ++it) {
          HIP_TRY(launch_vstep(w, (int)blk, bb, tau, s, tm, weighted));
          HIP_TRY(launch_ustep(w, (int)blk, bb, tau, weighted, it == iters - 1, s, tm));
        }
        HIP_TRY(launch_gram_acc(w, 0, s));  // U^T U of the final U, for the scale solve
        if (safeguard) HIP_TRY(launch_safeguard(w, (int)blk, bb, D + c0, s));
        HIP_TRY(launch_block_out(w, c0, bb, k, B_packed, C_packed, D, s, false, safeguard));
        HIP_TRY(launch_deflate(w, (int)blk, false, s, tm, safeguard));
      }
      if (stop_at_target && blk + 1 < nblk) {
        // energy after this block (||R||^2 history entries 0 and blk + 1)
        HIP_TRY(launch_finish(w, (int)blk + 1, s));
        double h2[2][2];
        HIP_TRY(hipMemcpyAsync(&h2[0][0], w.fro2_hist, sizeof(double), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(&h2[0][1], w.fro2_hist + blk + 1, sizeof(double), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(&h2[1][0], w.fro2w_hist, sizeof(double), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(&h2[1][1], w.fro2w_hist + blk + 1, sizeof(double), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        const double* hv = weighted ? h2[1] : h2[0];
        const double e = hv[0] == 0.0 ? 1.0 : 1.0 - hv[1] / hv[0];
        if (e >= target) {
          nblk_done = blk + 1;
          break;
        }
      }
    }
    if (nblk_done == nblk) HIP_TRY(launch_finish(w, (int)nblk, s));
  }

  std::vector<double> f2((size_t)nblk_done + 1), f2w((size_t)nblk_done + 1);
  HIP_TRY(hipMemcpyAsync(f2.data(), w.fro2_hist, sizeof(double) * (nblk_done + 1), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipMemcpyAsync(f2w.data(), w.fro2w_hist, sizeof(double) * (nblk_done + 1), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  SweepOut so{sweep_energy, sweep_energy_w, f2[(size_t)nblk_done], f2w[(size_t)nblk_done]};
  if (sweeps > 0)
    HIP_TRY(run_sweeps(w, k, b_eff, tau, iters, sweeps, weighted, B_packed, C_packed, D, (int)nblk, f2[0], f2w[0], so,
                       s, tm));
  unsigned n_acc = 0, n_fired = 0;
  HIP_TRY(hipMemcpyAsync(&n_acc, w.counters + CNT_ACCEPTED, sizeof(unsigned), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipMemcpyAsync(&n_fired, w.counters + CNT_SAFEGUARD, sizeof(unsigned), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipMemcpyAsync(flags, w.flags, sizeof(flags), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (flags[FLAG_SYNC]) return EXTERND_ESYNC;
  if (accepted) *accepted = (int64_t)n_acc;
  if (fired) *fired = (int64_t)n_fired;
  if (tm) {
    HIP_TRY(tm->collect(times->total_ms, times->launches, EXTERND_KCLASS_COUNT));
    for (int c = 0; c < EXTERND_KCLASS_COUNT; ++c) times->issued[c] = tm->seen[c];
  }
  const double a2 = f2[0], a2w = f2w[0];
  auto E = [&](int64_t b) { return a2 == 0.0 ? 1.0 : 1.0 - f2[(size_t)b] / a2; };
  auto Ew = [&](int64_t b) { return a2w == 0.0 ? 1.0 : 1.0 - f2w[(size_t)b] / a2w; };
  *energy = a2 == 0.0 ? 1.0 : 1.0 - so.fro2_last / a2;
  if (energy_w) *energy_w = a2w == 0.0 ? 1.0 : 1.0 - so.fro2w_last / a2w;
  for (int64_t b = 0; b < nblk_done; ++b) {
    if (energy_curve) energy_curve[b] = E(b + 1);
    if (energy_w_curve) energy_w_curve[b] = Ew(b + 1);
  }
  if (k_used) *k_used = nblk_done * b_eff < k ? nblk_done * b_eff : k;
  return EXTERND_OK;
}

int externd_factorize(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block, int32_t iters,
                      const float* importance, uint8_t* B_packed, uint8_t* C_packed, float* D, double* energy,
                      double* energy_w, double* energy_curve, double* energy_w_curve, void* workspace,
                      size_t workspace_bytes, void* stream) {
  return factorize_impl(A, m, n, mu, tau, block, iters, importance, B_packed, C_packed, D, energy, energy_w,
                        energy_curve, energy_w_curve, workspace, workspace_bytes, stream, nullptr);
}

int externd_factorize_to_energy(const float* A, int64_t m, int64_t n, double mu_max, double target_energy,
                                double tau, int32_t block, int32_t iters, const float* importance,
                                uint8_t* B_packed, uint8_t* C_packed, float* D, int64_t* k_used, double* energy,
                                double* energy_w, double* energy_curve, double* energy_w_curve, void* workspace,
                                size_t workspace_bytes, void* stream) {
  if (k_used) *k_used = 0;
  if (isnan(target_energy)) {
    if (energy) *energy = NAN;
    return EXTERND_EINVAL;
  }
  return factorize_impl(A, m, n, mu_max, tau, block, iters, importance, B_packed, C_packed, D, energy, energy_w,
                        energy_curve, energy_w_curve, workspace, workspace_bytes, stream, nullptr, target_energy,
                        k_used);
}

int externd_factorize_refined(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block,
                              int32_t iters, int32_t sweeps, const float* importance, uint8_t* B_packed,
                              uint8_t* C_packed, float* D, double* energy, double* energy_w, double* energy_curve,
                              double* energy_w_curve, double* sweep_energy, double* sweep_energy_w,
                              int64_t* accepted, void* workspace, size_t workspace_bytes, void* stream) {
  return factorize_impl(A, m, n, mu, tau, block, iters, importance, B_packed, C_packed, D, energy, energy_w,
                        energy_curve, energy_w_curve, workspace, workspace_bytes, stream, nullptr, NAN, nullptr,
                        sweeps, sweep_energy, sweep_energy_w, accepted);
}

int externd_factorize_ex(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block, int32_t iters,
                         const float* importance, double lambda, int32_t safeguard, uint8_t* B_packed,
                         uint8_t* C_packed, float* D, double* energy, double* energy_w, double* energy_curve,
                         double* energy_w_curve, int64_t* safeguard_fired, void* workspace, size_t workspace_bytes,
                         void* stream) {
  if (safeguard_fired) *safeguard_fired = 0;
  if (safeguard != 0 && safeguard != 1) {
    if (energy) *energy = NAN;
    return EXTERND_EINVAL;
  }
  return factorize_impl(A, m, n, mu, tau, block, iters, importance, B_packed, C_packed, D, energy, energy_w,
                        energy_curve, energy_w_curve, workspace, workspace_bytes, stream, nullptr, NAN, nullptr, 0,
                        nullptr, nullptr, nullptr, lambda, safeguard == 1, safeguard_fired);
}

int externd_factorize_timed(const float* A, int64_t m, int64_t n, double mu, double tau, int32_t block,
                            int32_t iters, const float* importance, uint8_t* B_packed, uint8_t* C_packed, float* D,
                            double* energy, double* energy_w, double* energy_curve, double* energy_w_curve,
                            void* workspace, size_t workspace_bytes, void* stream, externd_kernel_times* times) {
  if (!times) {
    if (energy) *energy = NAN;
    return EXTERND_EINVAL;
  }
  return factorize_impl(A, m, n, mu, tau, block, iters, importance, B_packed, C_packed, D, energy, energy_w,
                        energy_curve, energy_w_curve, workspace, workspace_bytes, stream, times);
}

// ---------------------------------------------------------------------------
// step entry points
// ---------------------------------------------------------------------------
// A caller's factor (len x bb int8, row-major) into the component-major,
// row-major and MFMA-ready copies of U (which = 0) or V (which = 1), one
// quarter of 64 components at a time.
static hipError_t load_factor_quarters(const Ws& w, int which, const int8_t* X, int64_t len, int32_t bb,
                                       hipStream_t s) {
  for (int q = 0; q * BBP < bb; ++q) {
    const Ws v = quarter_view(w, q);
    const int bq = bb - BBP * q < BBP ? bb - BBP * q : BBP;
    const hipError_t e = which ? launch_load_factor(v.Vt, v.Vr, v.Vmf, X + BBP * q, len, w.n_pad, bq, s, bb)
                               : launch_load_factor(v.Ut, v.Ur, v.Umf, X + BBP * q, len, w.m_pad, bq, s, bb);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

static int step_prologue(Ws& w, const float* R, int64_t m, int64_t n, int32_t bb, void* ws, size_t ws_bytes) {
  if (!R || !ws || m < 1 || n < 1 || bb < 1 || bb > BMAX) return EXTERND_EINVAL;
  if (!shape_ok(m, n)) return EXTERND_EUNSUPPORTED;
  if (!carve(w, ws, ws_bytes, m, n, 0)) return EXTERND_EWORKSPACE;
  return EXTERND_OK;
}

int externd_step_init(const float* R, int64_t m, int64_t n, const float* h, int32_t bb, double tau, int8_t* U_out,
                      int32_t* J_out, void* ws, size_t ws_bytes, void* stream) {
  Ws w{};
  int st = step_prologue(w, R, m, n, bb, ws, ws_bytes);
  if (st) return st;
  if (!U_out || !J_out || !isfinite(tau) || tau < 0.0 || bb > n) return EXTERND_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_prep(w, h, s));
  HIP_TRY(launch_stage(w, R, n, s));
  HIP_TRY(launch_select(w, 0, bb, s));
  HIP_TRY(bb > BBP ? launch_init_wide(w, bb, tau, s) : launch_init(w, bb, tau, s));
  HIP_TRY(launch_store_factor(U_out, w.Ut, m, w.m_pad, bb, s));
  HIP_TRY(hipMemcpyAsync(J_out, w.J, sizeof(int32_t) * bb, hipMemcpyDeviceToDevice, s));
  return EXTERND_OK;
}

int externd_step_vstep(const float* R, int64_t m, int64_t n, const int8_t* U, int32_t bb, double tau, int8_t* V_out,
                       double* Y_out_or_null, void* ws, size_t ws_bytes, void* stream) {
  Ws w{};
  int st = step_prologue(w, R, m, n, bb, ws, ws_bytes);
  if (st) return st;
  if (!U || !V_out || !isfinite(tau) || tau < 0.0) return EXTERND_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_prep(w, nullptr, s));
  HIP_TRY(launch_stage(w, R, n, s));
  HIP_TRY(launch_finish(w, 0, s));  // column energies -> the V-step's per-column exponents
  HIP_TRY(load_factor_quarters(w, 0, U, m, bb, s));
  HIP_TRY(bb > BBP ? launch_vstep_wide(w, 0, bb, tau, s) : launch_vstep(w, 0, bb, tau, s));
  HIP_TRY(launch_store_factor(V_out, w.Vt, n, w.n_pad, bb, s));
  if (Y_out_or_null) {
    // Y is bb x n: row c of the component-major buffer, pitch n_pad -> n
    HIP_TRY(hipMemcpy2DAsync(Y_out_or_null, sizeof(double) * n, w.Y, sizeof(double) * w.n_pad, sizeof(double) * n,
                             bb, hipMemcpyDeviceToDevice, s));
  }
  return EXTERND_OK;
}

int externd_step_ustep(const float* R, int64_t m, int64_t n, const int8_t* V, int32_t bb, double tau, const float* h,
                       int8_t* U_out, double* Q_out_or_null, double* Z_out_or_null, void* ws, size_t ws_bytes,
                       void* stream) {
  Ws w{};
  int st = step_prologue(w, R, m, n, bb, ws, ws_bytes);
  if (st) return st;
  if (!V || !U_out || !isfinite(tau) || tau < 0.0) return EXTERND_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_prep(w, h, s));
  HIP_TRY(launch_stage(w, R, n, s));
  HIP_TRY(load_factor_quarters(w, 1, V, n, bb, s));
  if (h) HIP_TRY(launch_vweight(w, bb, s));
  HIP_TRY(bb > BBP ? launch_ustep_wide(w, 0, bb, tau, h != nullptr, false, s)
                   : launch_ustep(w, 0, bb, tau, h != nullptr, false, s, nullptr, true));
  HIP_TRY(launch_store_factor(U_out, w.Ut, m, w.m_pad, bb, s));
  if (Q_out_or_null) HIP_TRY(launch_store_cm(Q_out_or_null, w.Q, m, w.m_pad, bb, s));
  if (Z_out_or_null) HIP_TRY(launch_store_cm(Z_out_or_null, w.Z, m, w.m_pad, bb, s));
  return EXTERND_OK;
}

int externd_step_scale(const int8_t* U, const int8_t* V, const double* Q, int64_t m, int64_t n, int32_t bb,
                       const float* h, double* d_out, void* ws, size_t ws_bytes, void* stream) {
  if (!U || !V || !Q || !d_out || !ws || m < 1 || n < 1 || bb < 1 || bb > BMAX) return EXTERND_EINVAL;
  if (!shape_ok(m, n)) return EXTERND_EUNSUPPORTED;
  Ws w{};
  if (!carve(w, ws, ws_bytes, m, n, 0)) return EXTERND_EWORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_prep(w, h, s));
  HIP_TRY(load_factor_quarters(w, 0, U, m, bb, s));
  HIP_TRY(load_factor_quarters(w, 1, V, n, bb, s));
  if (h) HIP_TRY(launch_vweight(w, bb, s));
  HIP_TRY(launch_load_cm(w.Q, Q, m, w.m_pad, bb, s));
  HIP_TRY(launch_gvec(w, bb, s));
  if (bb > BBP) {
    HIP_TRY(launch_gram_wide_raw(w, bb, h != nullptr, s));  // raw V^T H V
    HIP_TRY(launch_scale_wide(w, bb, nullptr, s));
  } else {
    HIP_TRY(launch_gram_only(w, bb, h != nullptr, s));
    HIP_TRY(launch_gram_acc(w, 0, s));
    HIP_TRY(launch_scale(w, bb, s));
  }
  HIP_TRY(hipMemcpyAsync(d_out, w.dvec, sizeof(double) * bb, hipMemcpyDeviceToDevice, s));
  return EXTERND_OK;
}

int externd_step_deflate(float* R, int64_t m, int64_t n, const int8_t* U, const int8_t* V, const double* d,
                         int32_t bb, double* colnorm2_out, double* fro2_out, void* ws, size_t ws_bytes,
                         void* stream) {
  Ws w{};
  int st = step_prologue(w, R, m, n, bb, ws, ws_bytes);
  if (st) return st;
  if (!U || !V || !d) return EXTERND_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_prep(w, nullptr, s));
  HIP_TRY(launch_stage(w, R, n, s));
  HIP_TRY(load_factor_quarters(w, 0, U, m, bb, s));
  HIP_TRY(load_factor_quarters(w, 1, V, n, bb, s));
  HIP_TRY(launch_set_scales(w, d, bb, s));
  HIP_TRY(bb > BBP ? launch_deflate_wide(w, 0, bb, true, s) : launch_deflate(w, 0, true, s));
  HIP_TRY(launch_unstage(w, R, s));
  if (colnorm2_out || fro2_out) HIP_TRY(launch_colnorms(w, 0, colnorm2_out, fro2_out, s));
  return EXTERND_OK;
}

}  // extern "C"
