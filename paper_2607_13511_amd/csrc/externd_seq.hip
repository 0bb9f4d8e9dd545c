// Persistent single-workgroup path of the sequential greedy ALS (block
// width 1, Sec. 2.3) for small matrices: the whole factorization runs in one
// launch of one 512-thread workgroup, with the residual held in registers.
//
// Thread (wave w of 8, lane l) holds R[w + 8 r][l + 64 c] for r < NR,
// c < NC (NR * NC = 128 fp32 values, zero outside m x n), so m <= 8 NR and
// n <= 64 NC: up to 256 x 256, or 128 x 512.  Vectors over the rows or the
// columns are distributed one entry per thread (entry t in thread t).
// Per component (Sec. 2.3, with the readings of the block path at b = 1):
//   init    j* = argmax_j h~_j ||R_:j||^2 (smaller j on ties), u = T(R[:, j*])
//   iters   v = T(R^T u); u = T(R diag(h~) v)       (Eq. (3) at b = 1: the
//           ridge and Gram factors are positive scalars, which T ignores)
//   scale   d = g / (M + delta), g = u^T R diag(h~) v, M = ||u||^2 v^T diag(h~) v,
//           delta = 1e-12 M (Eq. (4) at b = 1); optionally the single-entry
//           option of Proposition 2
//   deflate R -= fp32(d) u v^T, column energies, ||R||^2, weighted ||R||^2
// Contractions: each thread sums its own terms in fp32 (NR rows, or NC
// columns), and the partial sums are combined across threads in fp64 in a
// fixed order: through LDS across the waves for R^T u, through an LDS
// transpose inside each wave for R v.  Block reductions: DPP within a wave
// (result in lane 63), then the 8 wave results in wave order, read by every
// thread, so every thread holds bit-identical values and every branch is
// uniform.  Thresholds, scales and energies are fp64.  Deterministic.
#include "externd_dpp.hpp"
#include "externd_internal.hpp"

#include <limits.h>

namespace externd {

constexpr int SEQ_NT = 512;
constexpr int SEQ_WAVES = SEQ_NT / 64;
constexpr int SEQ_P2_PITCH = 68;  // floats per row of the R v transpose (16-byte rows, banks spread)

// Wave results of the block reductions, double-buffered: a reduction writes
// one buffer and the next the other, so a buffer is rewritten only after
// every thread has passed the barrier of the reduction in between.
struct SeqRed {
  double v[2][SEQ_WAVES][4];
  int i[2][SEQ_WAVES];
};

// Sum of the 8 wave results of slot q as a fixed tree.
__device__ __forceinline__ double tree8(const double (&v)[SEQ_WAVES][4], int q) {
  return ((v[0][q] + v[1][q]) + (v[2][q] + v[3][q])) + ((v[4][q] + v[5][q]) + (v[6][q] + v[7][q]));
}

// Block reduction of NSUM (<= 3) fp64 sums s[0 .. NSUM) and, with ARG, one
// (max, first index) pair; every thread receives the same results.
template <int NSUM, bool ARG>
__device__ __forceinline__ void block_reduce(double* s, double& mv, int& mi, SeqRed& R, int& buf) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
#pragma unroll
  for (int q = 0; q < NSUM; ++q) wave_sum63(s[q]);
  if (ARG) wave_argmax63(mv, mi);
  if (l == 63) {
#pragma unroll
    for (int q = 0; q < NSUM; ++q) R.v[buf][w][q] = s[q];
    if (ARG) {
      R.v[buf][w][3] = mv;
      R.i[buf][w] = mi;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NSUM; ++q) s[q] = tree8(R.v[buf], q);
  if (ARG) {
    mv = R.v[buf][0][3];
    mi = R.i[buf][0];
#pragma unroll
    for (int x = 1; x < SEQ_WAVES; ++x) dpp_argmax_combine(mv, mi, R.v[buf][x][3], R.i[buf][x]);
  }
  buf ^= 1;
}

// T_tau (Eq. (2)) of a vector of length L held one entry per thread (entry
// t in thread t, `valid` = t < L): theta = tau * sum|x| / L, strict ">",
// and when no entry passes, the largest |x_t| (smallest t) keeps its sign;
// zero stays zero.  Returns this thread's trit as a float.
__device__ __forceinline__ float seq_ternarize(double xv, bool valid, int L, double tau, SeqRed& R, int& buf) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const double a = valid ? fabs(xv) : 0.0;
  double s = a, mx = valid ? a : -1.0;
  wave_sum63(s);
  wave_max63(mx);
  if (l == 63) {
    R.v[buf][w][0] = s;
    R.v[buf][w][1] = mx;
  }
  __syncthreads();
  s = tree8(R.v[buf], 0);
  {
    const double(&v)[SEQ_WAVES][4] = R.v[buf];
    mx = fmax(fmax(fmax(v[0][1], v[1][1]), fmax(v[2][1], v[3][1])), fmax(fmax(v[4][1], v[5][1]), fmax(v[6][1], v[7][1])));
  }
  buf ^= 1;
  const double theta = tau * (s / (double)L);
  if (mx > theta) return (valid && a > theta) ? (xv > 0.0 ? 1.0f : -1.0f) : 0.0f;
  if (!(mx > 0.0)) return 0.0f;
  // no entry passes: the first entry of largest magnitude keeps its sign
  int first = (valid && a == mx) ? (int)threadIdx.x : INT_MAX;
  wave_imin63(first);
  if (l == 63) R.i[buf][w] = first;
  __syncthreads();
  int f = R.i[buf][0];
#pragma unroll
  for (int x = 1; x < SEQ_WAVES; ++x) f = min(f, R.i[buf][x]);
  buf ^= 1;
  return (int)threadIdx.x == f ? (xv > 0.0 ? 1.0f : -1.0f) : 0.0f;
}

template <int NR, int NC>
struct SeqLds {
  static constexpr int MP = SEQ_WAVES * NR, NP = 64 * NC, XL = MP > NP ? MP : NP;
  union {
    double part[SEQ_WAVES][NP];             // per-wave column partial sums
    float p2[SEQ_WAVES][NR][SEQ_P2_PITCH];  // per-lane row partial sums (R v)
  } u;
  double x[XL];      // a gathered column, or q = R diag(h~) v by row
  double colE[NP];   // ||R_:j||^2
  double hw[NP];     // h~_j (zero past n)
  float uf[MP];      // current u
  float vf[NP];      // current v
  int8_t uh[4][MP];  // the last four u's (one packed byte of B per row)
  SeqRed red;
};

// Column energies of the residual in registers, ||R||^2, the weighted
// ||R||^2 and, with track, the largest |R_ij| with key 2 (i n + j) + [R_ij < 0]
// (the first in row-major order on ties).
template <int NR, int NC>
__device__ __forceinline__ void seq_energies(const float (&Rr)[NR][NC], int n, bool track, SeqLds<NR, NC>& S,
                                             int& buf, double& fro2, double& fro2w, double& gmax, int& gkey) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  double ce[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) ce[c] = 0.0;
  float tmax = 0.0f;
  int tkey = INT_MAX;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float v = Rr[r][c];
      ce[c] = fma((double)v, (double)v, ce[c]);
      if (track && fabsf(v) > tmax) {
        tmax = fabsf(v);
        tkey = 2 * ((w + SEQ_WAVES * r) * n + (l + 64 * c)) + (v < 0.0f ? 1 : 0);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) S.u.part[w][l + 64 * c] = ce[c];
  __syncthreads();
  double cj = 0.0;
  if (t < SeqLds<NR, NC>::NP) {
#pragma unroll
    for (int q = 0; q < SEQ_WAVES; ++q) cj += S.u.part[q][t];
    if (t >= n) cj = 0.0;
    S.colE[t] = cj;
  }
  double s[2] = {cj, t < SeqLds<NR, NC>::NP ? S.hw[t] * cj : 0.0};
  double mv = tmax > 0.0f ? (double)tmax : -1.0;
  int mi = tmax > 0.0f ? tkey : INT_MAX;
  if (track)
    block_reduce<2, true>(s, mv, mi, S.red, buf);
  else
    block_reduce<2, false>(s, mv, mi, S.red, buf);
  fro2 = s[0];
  fro2w = s[1];
  gmax = track && mv > 0.0 ? mv : 0.0;
  gkey = mi;
}

__device__ __forceinline__ unsigned seq_trit_code(float t) { return t == 0.0f ? 0u : (t > 0.0f ? 1u : 3u); }

// Shapes the persistent path holds in registers, tried in this order.
template <int NR, int NC>
static bool seq_fits(int64_t m, int64_t n) {
  return m <= SEQ_WAVES * NR && n <= 64 * NC;
}

template <int NR, int NC>
__global__ __launch_bounds__(SEQ_NT) void k_seq(const float* __restrict__ A, int64_t m, int64_t n, int64_t k,
                                                double tau, int iters, const double* __restrict__ hw, int weighted,
                                                int safeguard, double target, uint8_t* __restrict__ Bp,
                                                uint8_t* __restrict__ Cp, float* __restrict__ D,
                                                double* __restrict__ fro2_hist, double* __restrict__ fro2w_hist,
                                                unsigned* counters, int* flags) {
  constexpr int MP = SeqLds<NR, NC>::MP, NP = SeqLds<NR, NC>::NP;
  constexpr int LPR = 64 / NR;  // lanes per row in the R v transpose
  constexpr int PER = 64 / LPR; // partials each of them sums
  static_assert(NR * NC == 128 && (LPR == 2 || LPR == 4), "register layouts of 128 values, 2 or 4 lanes per row");
  __shared__ SeqLds<NR, NC> S;
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  if (flags[FLAG_BADWEIGHT]) return;  // invalid weights: the host reports it
  const bool track = safeguard != 0;
  const bool has_target = !isnan(target);
  const int64_t pitchB = (k + 3) >> 2, pitchC = (n + 3) >> 2;
  const int mi = (int)m, ni = (int)n;
  int buf = 0;

  float hwf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int j = l + 64 * c;
    hwf[c] = j < ni ? (float)hw[j] : 0.0f;
  }
  const double hw_t = t < ni ? hw[t] : 0.0;
  if (t < NP) S.hw[t] = hw_t;

  // stage: R <- A (zero outside m x n), non-finite check
  float Rr[NR][NC];
  int bad = 0;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int i = w + SEQ_WAVES * r;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int j = l + 64 * c;
      float v = 0.0f;
      if (i < mi && j < ni) v = A[(int64_t)i * n + j];
      if (!isfinite(v)) {
        bad = 1;
        v = 0.0f;
      }
      Rr[r][c] = v;
    }
  }
  {
    double s[1] = {(double)bad}, mv = 0.0;
    int mx = 0;
    block_reduce<1, false>(s, mv, mx, S.red, buf);
    if (s[0] != 0.0) {
      if (t == 0) flags[FLAG_NONFINITE] = 1;
      return;
    }
  }
  double fro2, fro2w, gmax;
  int gkey;
  seq_energies<NR, NC>(Rr, ni, track, S, buf, fro2, fro2w, gmax, gkey);
  const double a2 = fro2, a2w = fro2w;
  if (t == 0) {
    fro2_hist[0] = fro2;
    fro2w_hist[0] = fro2w;
  }
  int64_t used = k;
  unsigned fired = 0;
  for (int64_t comp = 0; comp < k; ++comp) {
    // init (reading R1): the column with the largest weighted energy
    int js;
    {
      double kv = t < ni ? S.hw[t] * S.colE[t] : -1.0;
      int ki = t < ni ? t : INT_MAX;
      block_reduce<0, true>(nullptr, kv, ki, S.red, buf);
      js = ki;
    }
    if (l == (js & 63)) {
      const int cs = js >> 6;
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        float v = 0.0f;
#pragma unroll
        for (int c = 0; c < NC; ++c)
          if (c == cs) v = Rr[r][c];
        S.x[w + SEQ_WAVES * r] = (double)v;
      }
    }
    __syncthreads();
    float u_t = seq_ternarize(t < mi ? S.x[t] : 0.0, t < mi, mi, tau, S.red, buf);
    if (t < MP) S.uf[t] = u_t;
    __syncthreads();
    float v_t = 0.0f;
    double q_t = 0.0;
    for (int it = 0; it < iters; ++it) {
      // V-step: y = R^T u, v = T(y)
      {
        // two independent accumulation chains per column (rows r < NR/2, r >= NR/2)
        float p[2][NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) p[0][c] = p[1][c] = 0.0f;
#pragma unroll
        for (int r = 0; r < NR / 2; ++r) {
          const float u0 = S.uf[w + SEQ_WAVES * r], u1 = S.uf[w + SEQ_WAVES * (r + NR / 2)];
#pragma unroll
          for (int c = 0; c < NC; ++c) {
            p[0][c] = fmaf(Rr[r][c], u0, p[0][c]);
            p[1][c] = fmaf(Rr[r + NR / 2][c], u1, p[1][c]);
          }
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) S.u.part[w][l + 64 * c] = (double)p[0][c] + (double)p[1][c];
      }
      __syncthreads();
      double y = 0.0;
      if (t < NP) {
        const double(&pp)[SEQ_WAVES][NP] = S.u.part;
        y = ((pp[0][t] + pp[1][t]) + (pp[2][t] + pp[3][t])) + ((pp[4][t] + pp[5][t]) + (pp[6][t] + pp[7][t]));
      }
      v_t = seq_ternarize(y, t < ni, ni, tau, S.red, buf);
      if (t < NP) S.vf[t] = v_t;
      __syncthreads();
      // U-step: q = R diag(h~) v, u = T(q)
      {
        float hv[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) hv[c] = hwf[c] * S.vf[l + 64 * c];
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          float s = 0.0f;
#pragma unroll
          for (int c = 0; c < NC; ++c) s = fmaf(Rr[r][c], hv[c], s);
          S.u.p2[w][r][l] = s;
        }
        // each wave reads back only what it wrote itself
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // lane l sums PER partials of row l / LPR, then the LPR lanes of a row combine
        const int rr = l / LPR, pp = l % LPR;
        const float4* src = (const float4*)&S.u.p2[w][rr][pp * PER];
        double a4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int e = 0; e < PER / 4; ++e) {
          const float4 f = src[e];
          a4[0] += (double)f.x;
          a4[1] += (double)f.y;
          a4[2] += (double)f.z;
          a4[3] += (double)f.w;
        }
        double acc = (a4[0] + a4[1]) + (a4[2] + a4[3]);
        acc += dpp_f64<DPP_QUAD_XOR1, 0xF>(0.0, acc);
        if (LPR == 4) acc += dpp_f64<DPP_QUAD_XOR2, 0xF>(0.0, acc);
        if (pp == 0) S.x[w + SEQ_WAVES * rr] = acc;
      }
      __syncthreads();
      q_t = t < mi ? S.x[t] : 0.0;
      u_t = seq_ternarize(q_t, t < mi, mi, tau, S.red, buf);
      if (t < MP) S.uf[t] = u_t;
      __syncthreads();
    }
    // joint scale (Eq. (4) at b = 1) from the last U-step's q
    double d, delta;
    {
      double s[3] = {(double)u_t * q_t, (double)(u_t * u_t), hw_t * (double)(v_t * v_t)};
      double mv = 0.0;
      int mx = 0;
      block_reduce<3, false>(s, mv, mx, S.red, buf);
      const double g = s[0], M = s[1] * s[2];
      d = 0.0;
      delta = 0.0;
      if (M != 0.0) {
        delta = EXTERND_SCALE_GUARD_REL * M;
        d = g / (M + delta);
      }
      // single-entry option of Proposition 2: removed objective d g + delta d^2
      if (track && gmax > 0.0 && gmax * gmax > d * g + delta * d * d) {
        const int flat = gkey >> 1;
        const int gi = flat / ni, gj = flat % ni;
        d = gmax;
        if (t < MP) S.uf[t] = t == gi ? 1.0f : 0.0f;
        if (t < NP) S.vf[t] = t == gj ? ((gkey & 1) ? -1.0f : 1.0f) : 0.0f;
        ++fired;
        __syncthreads();
      }
    }
    const float dF = (float)d;
    // outputs: D, row comp of C, the packed byte of B every fourth component
    if (t == 0) D[comp] = dF;
    if (t < pitchC) {
      unsigned byte = 0;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int j = 4 * t + s;
        if (j < ni) byte |= seq_trit_code(S.vf[j]) << (2 * s);
      }
      Cp[comp * pitchC + t] = (uint8_t)byte;
    }
    if (t < MP) S.uh[comp & 3][t] = (int8_t)S.uf[t];
    // deflation R -= fp32(d) u v^T (u v is an exact ternary product)
    {
      float vv[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) vv[c] = S.vf[l + 64 * c];
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const float u = S.uf[w + SEQ_WAVES * r];
#pragma unroll
        for (int c = 0; c < NC; ++c) Rr[r][c] -= (u * vv[c]) * dF;
      }
    }
    // (the barrier in seq_energies also orders the uh writes before the B write)
    seq_energies<NR, NC>(Rr, ni, track, S, buf, fro2, fro2w, gmax, gkey);
    if (t == 0) {
      fro2_hist[comp + 1] = fro2;
      fro2w_hist[comp + 1] = fro2w;
    }
    // energy target (E, or E_w with weights): stop after this component
    bool stop = false;
    if (has_target && comp + 1 < k) {
      const double e = weighted ? (a2w == 0.0 ? 1.0 : 1.0 - fro2w / a2w) : (a2 == 0.0 ? 1.0 : 1.0 - fro2 / a2);
      stop = e >= target;
    }
    if ((comp & 3) == 3 || comp == k - 1 || stop) {
      if (t < mi) {
        unsigned byte = 0;
        const int top = (int)(comp & 3);
        for (int s = 0; s <= top; ++s) byte |= seq_trit_code((float)S.uh[s][t]) << (2 * s);
        Bp[(int64_t)t * pitchB + (comp >> 2)] = (uint8_t)byte;
      }
    }
    if (stop) {
      used = comp + 1;
      break;
    }
  }
  if (t == 0) {
    counters[CNT_SEQ_USED] = (unsigned)used;
    counters[CNT_SAFEGUARD] = fired;
  }
}

bool seq_supported(int64_t m, int64_t n) { return seq_fits<32, 4>(m, n) || seq_fits<16, 8>(m, n); }

hipError_t launch_seq(const Ws& w, const float* A, int64_t k, double tau, int iters, bool weighted, bool safeguard,
                      double target, uint8_t* Bp, uint8_t* Cp, float* D, hipStream_t s, Timer* tm) {
  const int64_t m = w.m, n = w.n;
#define SEQ_LAUNCH(NR, NC)                                                                                  \
  EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_SEQ, (k_seq<NR, NC>), dim3(1), dim3(SEQ_NT), 0, s, A, m, n, k, tau, \
                       iters, (const double*)w.hw, weighted ? 1 : 0, safeguard ? 1 : 0, target, Bp, Cp, D,    \
                       w.fro2_hist, w.fro2w_hist, w.counters, w.flags)
  if (seq_fits<32, 4>(m, n))
    SEQ_LAUNCH(32, 4);
  else if (seq_fits<16, 8>(m, n))
    SEQ_LAUNCH(16, 8);
  else
    return hipErrorInvalidValue;
#undef SEQ_LAUNCH
  return hipGetLastError();
}

}  // namespace externd
