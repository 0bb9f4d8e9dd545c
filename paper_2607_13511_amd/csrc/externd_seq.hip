// Persistent single-workgroup path of the sequential greedy ALS (block
// width 1, Sec. 2.3) for small matrices: the whole factorization runs in one
// launch of one 512-thread workgroup, with the residual held in registers.
//
// Thread (wave w of 8, lane l) holds R[w + 8 r][l + 64 c] for r < NR,
// c < NC (NR * NC = 128 fp32 values, zero outside m x n), so m <= 8 NR and
// n <= 64 NC: up to 256 x 256, or 128 x 512.  Per component (Sec. 2.3, with the readings of the block
// path at b = 1):
//   init   j* = argmax_j h~_j ||R_:j||^2 (smaller j on ties), u = T(R[:, j*])
//   iters  v = T(R^T u); u = T(R diag(h~) v)       (Eq. (3) at b = 1: the
//          ridge and Gram factors are positive scalars, which T ignores)
//   scale  d = g / (M + delta), g = u^T R diag(h~) v, M = ||u||^2 v^T diag(h~) v,
//          delta = 1e-12 M (Eq. (4) at b = 1); optionally the single-entry
//          option of Proposition 2
//   deflate R -= fp32(d) u v^T, column energies, ||R||^2, weighted ||R||^2
// Contractions: each thread sums its own terms in fp32 (at most 64), the
// partial sums are combined across threads in fp64 in a fixed order.
// Thresholds, scales and energies are fp64.  Deterministic.
#include "externd_internal.hpp"

namespace externd {

constexpr int SEQ_NT = 512;
constexpr int SEQ_WAVES = SEQ_NT / 64;

// (value, index) pairs: larger value first, then smaller index.
__device__ __forceinline__ void seq_argmax_combine(double& v, int& i, double ov, int oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

// Block-wide sum of three fp64 values and (max, first index) of one more;
// every thread receives the same results (xor butterflies are symmetric,
// the 16 wave results are combined in wave order by every thread).
struct SeqShared {
  double s[SEQ_WAVES][4];
  int i[SEQ_WAVES];
};
__device__ __forceinline__ void seq_reduce(double& a, double& b, double& c, double& mx, int& ix, SeqShared& sh) {
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_xor(a, o, 64);
    b += __shfl_xor(b, o, 64);
    c += __shfl_xor(c, o, 64);
    const double om = __shfl_xor(mx, o, 64);
    const int oi = __shfl_xor(ix, o, 64);
    seq_argmax_combine(mx, ix, om, oi);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh.s[w][0] = a;
    sh.s[w][1] = b;
    sh.s[w][2] = c;
    sh.s[w][3] = mx;
    sh.i[w] = ix;
  }
  __syncthreads();
  a = sh.s[0][0];
  b = sh.s[0][1];
  c = sh.s[0][2];
  mx = sh.s[0][3];
  ix = sh.i[0];
  for (int q = 1; q < SEQ_WAVES; ++q) {
    a += sh.s[q][0];
    b += sh.s[q][1];
    c += sh.s[q][2];
    seq_argmax_combine(mx, ix, sh.s[q][3], sh.i[q]);
  }
  __syncthreads();
}

// T_tau (Eq. (2)) of x[0 .. L) into out[0 .. Lpad) as floats in {-1, 0, 1}:
// theta = tau * sum|x| / L, strict ">", and when no entry passes the
// largest |x_i| (smallest i) keeps its sign; zero stays zero.  L <= SEQ_NT.
__device__ __forceinline__ void seq_ternarize(const double* x, int L, int Lpad, double tau, float* out,
                                              SeqShared& sh) {
  const int t = threadIdx.x;
  const double xv = t < L ? x[t] : 0.0;
  double s = fabs(xv), z0 = 0.0, z1 = 0.0, mx = t < L ? fabs(xv) : -1.0;
  int ix = t;
  seq_reduce(s, z0, z1, mx, ix, sh);
  const double theta = tau * (s / (double)L);
  if (t < Lpad) {
    float o = 0.0f;
    if (t < L) {
      const bool keep = mx > theta ? fabs(xv) > theta : (t == ix && mx > 0.0);
      if (keep) o = xv > 0.0 ? 1.0f : -1.0f;
    }
    out[t] = o;
  }
  __syncthreads();
}

template <int NR, int NC>
struct SeqLds {
  static constexpr int MP = SEQ_WAVES * NR, NP = 64 * NC, XL = MP > NP ? MP : NP;
  double part[SEQ_WAVES][NP];   // per-wave column partial sums
  double x[XL];                 // the vector being ternarized (targets), then q of the last U-step
  double colE[NP];              // ||R_:j||^2
  double hw[NP];                // h~_j (zero past n)
  float uf[MP];                 // current u
  float vf[NP];                 // current v
  int8_t uh[4][MP];             // the last four u's (one packed byte of B per row)
  SeqShared red;
};

// Column energies of the residual in registers (and, with track, its largest
// |R_ij|: value, first row-major index i * n + j, sign), the plain and the
// weighted ||R||^2.
template <int NR, int NC>
__device__ __forceinline__ void seq_energies(const float (&Rr)[NR][NC], int64_t n, bool track, SeqLds<NR, NC>& S,
                                             double& fro2, double& fro2w, double& gmax, int& gidx, float& gval) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  double ce[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) ce[c] = 0.0;
  float tmax = 0.0f, tval = 0.0f;
  int tidx = 0x7FFFFFFF;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float v = Rr[r][c];
      ce[c] = fma((double)v, (double)v, ce[c]);
      if (track && fabsf(v) > tmax) {
        tmax = fabsf(v);
        tval = v;
        tidx = (int)((int64_t)(w + SEQ_WAVES * r) * n + (l + 64 * c));
      }
    }
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) S.part[w][l + 64 * c] = ce[c];
  __syncthreads();
  double cj = 0.0;
  if (t < SeqLds<NR, NC>::NP) {
    for (int q = 0; q < SEQ_WAVES; ++q) cj += S.part[q][t];
    if (t >= n) cj = 0.0;
    S.colE[t] = cj;
  }
  double a = cj, b = t < SeqLds<NR, NC>::NP ? S.hw[t] * cj : 0.0, z = 0.0;
  double mx = track ? (double)tmax : 0.0;
  int ix = tidx;
  // the signed value travels with the index: recover it from the owner
  seq_reduce(a, b, z, mx, ix, S.red);
  fro2 = a;
  fro2w = b;
  if (track) {
    gmax = mx;
    gidx = ix;
    // the thread that holds the winning entry publishes its sign
    if (tidx == ix && (double)tmax == mx && mx > 0.0) S.red.s[0][0] = (double)tval;
    __syncthreads();
    gval = mx > 0.0 ? (float)S.red.s[0][0] : 0.0f;
    __syncthreads();
  }
}

// Sum over the 64 lanes of a wave of each of p[0 .. NR): recursive halving
// (a lane keeps one half of its values and adds its partner's copy of that
// half), after which lane l holds the sum of p[l >> (6 - log2 NR)].
template <int K, int MASK, int NR>
struct SeqHalve {
  static __device__ __forceinline__ void run(double (&p)[NR], int l) {
    if constexpr (K > 1) {
      const bool hi = (l & MASK) != 0;
#pragma unroll
      for (int i = 0; i < K / 2; ++i) {
        const double keep = hi ? p[i + K / 2] : p[i];
        const double send = hi ? p[i] : p[i + K / 2];
        p[i] = keep + __shfl_xor(send, MASK, 64);
      }
      SeqHalve<K / 2, MASK / 2, NR>::run(p, l);
    } else if constexpr (MASK > 0) {
      p[0] += __shfl_xor(p[0], MASK, 64);
      SeqHalve<1, MASK / 2, NR>::run(p, l);
    }
  }
};
template <int NR>
__device__ __forceinline__ double seq_lane_reduce_scatter(double (&p)[NR]) {
  SeqHalve<NR, 32, NR>::run(p, threadIdx.x & 63);
  return p[0];
}

template <int NR>
struct Log2 {
  static constexpr int v = NR <= 1 ? 0 : 1 + Log2<NR / 2>::v;
};
template <>
struct Log2<1> {
  static constexpr int v = 0;
};

__device__ __forceinline__ unsigned seq_trit_code(float t) { return t == 0.0f ? 0u : (t > 0.0f ? 1u : 3u); }

// Shapes the persistent path holds in registers, tried in this order.
template <int NR, int NC>
static bool seq_fits(int64_t m, int64_t n) {
  return m <= SEQ_WAVES * NR && n <= 64 * NC;
}

template <int NR, int NC>
__global__ __launch_bounds__(SEQ_NT) void k_seq(const float* __restrict__ A, int64_t m, int64_t n, int64_t k,
                                                double tau, int iters, const double* __restrict__ hw, int weighted,
                                                int safeguard, double target, uint8_t* __restrict__ Bp, uint8_t* __restrict__ Cp,
                                                float* __restrict__ D, double* __restrict__ fro2_hist,
                                                double* __restrict__ fro2w_hist, unsigned* counters, int* flags) {
  constexpr int MP = SeqLds<NR, NC>::MP, NP = SeqLds<NR, NC>::NP;
  constexpr int RC = NR < 4 ? NR : 4;  // rows per lane reduction (bounds the registers it holds)
  constexpr int LG = Log2<RC>::v;
  __shared__ SeqLds<NR, NC> S;
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  if (flags[FLAG_BADWEIGHT]) return;  // invalid weights: the host reports it
  const bool track = safeguard != 0;
  const bool has_target = !isnan(target);
  const int64_t pitchB = (k + 3) >> 2, pitchC = (n + 3) >> 2;

  float hwf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int j = l + 64 * c;
    hwf[c] = j < n ? (float)hw[j] : 0.0f;
  }
  if (t < NP) S.hw[t] = t < n ? hw[t] : 0.0;

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
      if (i < m && j < n) v = A[(int64_t)i * n + j];
      if (!isfinite(v)) {
        bad = 1;
        v = 0.0f;
      }
      Rr[r][c] = v;
    }
  }
  {
    double a = (double)bad, z0 = 0.0, z1 = 0.0, mx = 0.0;
    int ix = 0;
    seq_reduce(a, z0, z1, mx, ix, S.red);
    if (a != 0.0) {
      if (t == 0) flags[FLAG_NONFINITE] = 1;
      return;
    }
  }
  double fro2, fro2w, gmax = 0.0;
  int gidx = 0;
  float gval = 0.0f;
  seq_energies<NR, NC>(Rr, n, track, S, fro2, fro2w, gmax, gidx, gval);
  const double a2 = fro2, a2w = fro2w;
  if (t == 0) {
    fro2_hist[0] = fro2;
    fro2w_hist[0] = fro2w;
  }
  int64_t used = k;
  unsigned fired = 0;
  for (int64_t comp = 0; comp < k; ++comp) {
    // init (reading R1): column with the largest weighted energy
    int js;
    {
      double z0 = 0.0, z1 = 0.0, z2 = 0.0;
      double kv = (t < n) ? S.hw[t] * S.colE[t] : -1.0;
      int ki = t;
      seq_reduce(z0, z1, z2, kv, ki, S.red);
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
    seq_ternarize(S.x, (int)m, MP, tau, S.uf, S.red);
    for (int it = 0; it < iters; ++it) {
      // V-step: y = R^T u, v = T(y)
      {
        float p[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) p[c] = 0.0f;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float u = S.uf[w + SEQ_WAVES * r];
#pragma unroll
          for (int c = 0; c < NC; ++c) p[c] = fmaf(Rr[r][c], u, p[c]);
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) S.part[w][l + 64 * c] = (double)p[c];
      }
      __syncthreads();
      if (t < NP) {
        double y = 0.0;
        for (int q = 0; q < SEQ_WAVES; ++q) y += S.part[q][t];
        S.x[t] = y;
      }
      __syncthreads();
      seq_ternarize(S.x, (int)n, NP, tau, S.vf, S.red);
      // U-step: q = R diag(h~) v, u = T(q)
      {
        float hv[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) hv[c] = hwf[c] * S.vf[l + 64 * c];
#pragma unroll
        for (int ch = 0; ch < NR / RC; ++ch) {
          double p[RC];
#pragma unroll
          for (int r = 0; r < RC; ++r) {
            float s = 0.0f;
#pragma unroll
            for (int c = 0; c < NC; ++c) s = fmaf(Rr[ch * RC + r][c], hv[c], s);
            p[r] = (double)s;
          }
          const double q = seq_lane_reduce_scatter<RC>(p);
          if ((l & ((64 >> LG) - 1)) == 0) S.x[w + SEQ_WAVES * (ch * RC + (l >> (6 - LG)))] = q;
        }
      }
      __syncthreads();
      seq_ternarize(S.x, (int)m, MP, tau, S.uf, S.red);
    }
    // joint scale (Eq. (4) at b = 1) from the last U-step's q
    double d, delta;
    {
      double g = t < m ? (double)S.uf[t] * S.x[t] : 0.0;
      double nu = t < m ? (double)(S.uf[t] * S.uf[t]) : 0.0;
      double vh = t < n ? S.hw[t] * (double)(S.vf[t] * S.vf[t]) : 0.0;
      double z = 0.0;
      int zi = 0;
      seq_reduce(g, nu, vh, z, zi, S.red);
      const double M = nu * vh;
      d = 0.0;
      delta = 0.0;
      if (M != 0.0) {
        delta = EXTERND_SCALE_GUARD_REL * M;
        d = g / (M + delta);
      }
      // single-entry option of Proposition 2: removed objective d g + delta d^2
      if (track && gmax > 0.0 && gmax * gmax > d * g + delta * d * d) {
        const int gi = (int)(gidx / n), gj = (int)(gidx % n);
        d = gmax;
        if (t < MP) S.uf[t] = t == gi ? 1.0f : 0.0f;
        if (t < NP) S.vf[t] = t == gj ? (gval < 0.0f ? -1.0f : 1.0f) : 0.0f;
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
        if (j < n) byte |= seq_trit_code(S.vf[j]) << (2 * s);
      }
      Cp[comp * pitchC + t] = (uint8_t)byte;
    }
    if (t < MP) S.uh[comp & 3][t] = (int8_t)S.uf[t];
    // deflation R -= fp32(d) u v^T (the ternary product is exact)
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const float u = S.uf[w + SEQ_WAVES * r];
#pragma unroll
      for (int c = 0; c < NC; ++c) Rr[r][c] -= (u * S.vf[l + 64 * c]) * dF;
    }
    __syncthreads();  // uh written, uf / vf read
    seq_energies<NR, NC>(Rr, n, track, S, fro2, fro2w, gmax, gidx, gval);
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
      if (t < m) {
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

}  // namespace externd

namespace externd {

bool seq_supported(int64_t m, int64_t n) {
  return seq_fits<32, 4>(m, n) || seq_fits<16, 8>(m, n);
}

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
