// HIP kernels (gfx950) for the ExTernD greedy block-ALS factorization.
//
// Method (paper "ExTernD: Expanded-Rank Ternary Decomposition"):
//   * T_tau ternarization, Eq. (2), Sec. 2.2;
//   * block ALS with decorrelated targets, Eq. (3), Sec. 2.4, weighted per
//     Sec. 2.5 (U-step on R diag(h~), V-step on the plain residual);
//   * joint exact scale solve, Eq. (4);
//   * block deflation R <- R - U diag(d) V^T, Sec. 2.4.
//
// Arithmetic design:
//   * The two residual contractions (P = U^T R and Q = R diag(h~) V) run on
//     int8 MFMA (v_mfma_i32_32x32x32_i8).  Each fp32 residual entry is
//     scaled by a power of two and rounded to a 32-bit integer, which is
//     split into four signed 8-bit digits; the ternary operand is exact in
//     int8.  The exponent follows the index the contraction keeps: column j
//     in the V-step (P[:, j] only involves column j of R; 2^s_j bounds
//     ||R_:j|| / 2^30, from the fused column energies), row i in the U-step
//     (Q[i, :] only involves row i; 2^s_i bounds max_j |R_ij h~_j| / 2^30,
//     measured by the previous U-step and raised by each deflation), so a
//     large entry costs resolution only in its own column or row.  The four
//     digit planes accumulate separately in int32 and are combined in
//     int64, so each contraction is exact for the fixed-point residual and
//     independent of summation order.
//   * Gram matrices of ternary factors are exact integers (int8 MFMA); the
//     weighted Gram V^T diag(h~) V and all solves are fp64.
//   * Targets Y, Z and the T_tau thresholds are fp64.
//   * Deflation runs on bf16 MFMA: the ternary factors are exact in bf16
//     and each fp32 scale d_c is split exactly into three bf16 parts;
//     products accumulate in fp32.
#include "externd.h"
#include "externd_dpp.hpp"
#include "externd_internal.hpp"

#include <hip/hip_runtime.h>
#include <math.h>

namespace externd {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef short v8s __attribute__((ext_vector_type(8)));
typedef double v4d __attribute__((ext_vector_type(4)));
typedef double v2d __attribute__((ext_vector_type(2)));
typedef long long v2l __attribute__((ext_vector_type(2)));
constexpr int GV_ONE = 6;  // V-step row groups summed in one round of loads
typedef float v4f __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// Fixed-point exponent of a row from its bound b >= max_j |R_ij h~_j|:
// b < 2^e  =>  s = 30 - e, so |x 2^s| < 2^30.
__device__ __forceinline__ int fx_shift(float b) {
  int e = 0;
  if (b > 0.0f) frexpf(b, &e);
  return 30 - e;
}
// Fixed-point exponent of column j from its energy S = sum_i R_ij^2 (the
// fused column energies, row-group partials added in group order): every
// |R_ij| <= sqrt(S) (a sum of non-negative terms never rounds below its
// largest term), and S < 2^E gives |R_ij| < 2^ceil(E/2).  Computed once per
// residual by the kernel that reduces the energies (cshift), read by the
// V-step contraction and its target.
__device__ __forceinline__ int col_shift(double S) {
  int E = 0;
  if (S > 0.0) frexp(S, &E);
  return 30 - ((E + 1) >> 1);
}

// x 2^s rounded to the nearest int32 (unbiased, so rounding errors do not
// accumulate along fitted signs), biased so that every byte is a digit + 128
// (bytes 0..2) or the signed top digit (byte 3).
__device__ __forceinline__ unsigned fx_biased(float x, int s) {
  return (unsigned)(int)__builtin_rintf(__builtin_amdgcn_ldexpf(x, s)) + 0x00808080u;
}
// The same with the power of two 2^s given as a factor (x 2^s is exact).
__device__ __forceinline__ unsigned fx_biased_m(float x, float p2s) {
  return (unsigned)(int)__builtin_rintf(x * p2s) + 0x00808080u;
}
// Weighted: x hw 2^s rounded to the nearest integer (ties to even) in one
// step, with c = 1.5 2^(52 - s) (weighted_round_const).  Adding c inside
// the fma rounds the exact product x hw at spacing 2^-s, so for
// |x hw 2^s| < 2^31 the low word of the result is that integer in two's
// complement.
__device__ __forceinline__ unsigned fx_biased_w(float x, double hw, double c) {
  const double t = __builtin_fma((double)x, hw, c);
  return (unsigned)__double2loint(t) + 0x00808080u;
}
__device__ __forceinline__ double weighted_round_const(int s) { return ldexp(1.5, 52 - s); }

// Upper bound (fp32) on |v| * hw for the weighted fixed-point scale: the
// fp64 product rounded to fp32, inflated by 2^-20 so that rounding can never
// make the bound smaller than the true value.
__device__ __forceinline__ float weighted_abs_bound(float v, double hw) {
  return (float)((double)fabsf(v) * hw) * 1.000001f;
}

// Byte-transpose four biased words into four digit planes:
// plane p holds byte p of (y0, y1, y2, y3); planes 0..2 are re-centred
// (xor 0x80 turns an unsigned digit+128 into the signed digit).
__device__ __forceinline__ void planes4(unsigned y0, unsigned y1, unsigned y2, unsigned y3,
                                        int& p0, int& p1, int& p2, int& p3) {
  unsigned t0 = __builtin_amdgcn_perm(y1, y0, 0x05010400u);  // y0b0 y1b0 y0b1 y1b1
  unsigned t1 = __builtin_amdgcn_perm(y1, y0, 0x07030602u);  // y0b2 y1b2 y0b3 y1b3
  unsigned t2 = __builtin_amdgcn_perm(y3, y2, 0x05010400u);
  unsigned t3 = __builtin_amdgcn_perm(y3, y2, 0x07030602u);
  p0 = (int)(__builtin_amdgcn_perm(t2, t0, 0x05040100u) ^ 0x80808080u);
  p1 = (int)(__builtin_amdgcn_perm(t2, t0, 0x07060302u) ^ 0x80808080u);
  p2 = (int)(__builtin_amdgcn_perm(t3, t1, 0x05040100u) ^ 0x80808080u);
  p3 = (int)__builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

// 16 biased words (K slots 0..15 of one lane) -> 4 planes of 16 int8.
__device__ __forceinline__ void make_planes(const unsigned (&y)[16], v4i (&P)[4]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    int a, b, c, d;
    planes4(y[4 * g], y[4 * g + 1], y[4 * g + 2], y[4 * g + 3], a, b, c, d);
    P[0][g] = a;
    P[1][g] = b;
    P[2][g] = c;
    P[3][g] = d;
  }
}

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

// MFMA-ready layout of a ternary factor X (BBP components x L): for K step
// ks (32 indices) and component half t, the 64 lanes' 16-byte operands of
// v_mfma_i32_32x32x32_i8 are contiguous, lane l holding
// X[32 t + l % 32][32 ks + 16 (l / 32) .. + 16).  Both operands of the
// integer Gram and the ternary operand of either contraction load from it
// with one fully coalesced 1 KB read per wave.
__device__ __forceinline__ int64_t mf_offset(int c, int64_t i) {
  return ((i >> 5) * 2 + (c >> 5)) * 1024 + ((c & 31) + 32 * ((i >> 4) & 1)) * 16 + (i & 15);
}

typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ unsigned lds_addr(const void* p) { return (unsigned)(uintptr_t)(const lds_void*)p; }

// Four 16-byte LDS reads after waiting until at most VM vector-memory
// operations of this wave are outstanding.  Direct-to-LDS loads
// (global_load_lds) complete in issue order with the other vector loads,
// so VM = the number of direct loads issued after the ones being read
// makes their data visible.  Written as one asm block because the
// compiler otherwise waits for every outstanding direct load before any
// LDS read.
template <int VM>
__device__ __forceinline__ void lds_read4_after(unsigned a0, unsigned a1, unsigned a2, unsigned a3, v4f& x0, v4f& x1,
                                                v4f& x2, v4f& x3) {
  asm volatile(
      "s_waitcnt vmcnt(%8)\n\tds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\t"
      "ds_read_b128 %3, %7\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(x0), "=&v"(x1), "=&v"(x2), "=&v"(x3)
      : "v"(a0), "v"(a1), "v"(a2), "v"(a3), "n"(VM)
      : "memory");
}
// One 4-byte LDS read after waiting until at most VM vector-memory
// operations of this wave are outstanding (see lds_read4_after).
template <int VM>
__device__ __forceinline__ float lds_read1_after(unsigned a) {
  float x;
  asm volatile("s_waitcnt vmcnt(%1)\n\tds_read_b32 %0, %2\n\ts_waitcnt lgkmcnt(0)" : "=&v"(x) : "n"(VM), "v"(a) : "memory");
  return x;
}
// Eight 16-byte LDS reads (no vector-memory wait: issue after
// lds_read4_after on the same stage).
__device__ __forceinline__ void lds_read8(unsigned a, v2d (&x)[8]) {
  asm volatile(
      "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:16\n\tds_read_b128 %2, %8 offset:32\n\t"
      "ds_read_b128 %3, %8 offset:48\n\tds_read_b128 %4, %8 offset:64\n\tds_read_b128 %5, %8 offset:80\n\t"
      "ds_read_b128 %6, %8 offset:96\n\tds_read_b128 %7, %8 offset:112\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(x[4]), "=&v"(x[5]), "=&v"(x[6]), "=&v"(x[7])
      : "v"(a)
      : "memory");
}

// Planes of one wave's accumulators combined exactly into int64.
__device__ __forceinline__ long long combine_acc(const v16i (&acc)[2][4], int t, int r) {
  return (long long)acc[t][0][r] + ((long long)acc[t][1][r] << 8) + ((long long)acc[t][2][r] << 16) +
         ((long long)acc[t][3][r] << 24);
}

// Planes folded in pairs, lo = a0 + 2^8 a1 and hi = a2 + 2^8 a3, so that the
// tile entry is lo + 2^16 hi.  Every product of a digit (|d| <= 128) and a
// trit is at most 2^7, a K step adds 32 of them, so after k K steps over all
// waves |lo|, |hi| <= k 2^12 257: the folded sums stay exact in int32 for
// k <= FOLD_KMAX.
constexpr int FOLD_KMAX = 2039;  // floor((2^31 - 1) / (2^12 257))
__device__ __forceinline__ int2 fold_acc(const v16i (&acc)[2][4], int t, int r) {
  return make_int2(acc[t][0][r] + acc[t][1][r] * 256, acc[t][2][r] + acc[t][3][r] * 256);
}

// Sum of the 4 waves' contraction tiles (2 tiles of 32x32, MFMA output
// layout) through LDS (red: 8192 int64 = 64 KB).  Wave w finishes slots
// 8w .. 8w + 7; out(t, M, N, v) receives every entry once, M the tile row
// and N the tile column.  Integer sums: exact and order-free.  With `fold`
// (at most FOLD_KMAX K steps summed in the workgroup) the planes travel as
// int32 pairs and only the final entries are widened, a quarter of the
// 64-bit work of widening every wave's planes.
template <typename Out>
__device__ __forceinline__ void reduce_waves(long long* red, const v16i (&acc)[2][4], bool fold, Out out) {
  const int lane = lane_id(), wave = wave_id();
  long long v[8];
  if (fold) {
    int2* r2 = (int2*)red;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) r2[(wave * 32 + t * 16 + r) * 64 + lane] = fold_acc(acc, t, r);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int slot = wave * 8 + i;
      const int2 a = r2[slot * 64 + lane], b = r2[(32 + slot) * 64 + lane];
      const int2 c = r2[(64 + slot) * 64 + lane], d = r2[(96 + slot) * 64 + lane];
      v[i] = (long long)((a.x + b.x) + (c.x + d.x)) + (long long)((a.y + b.y) + (c.y + d.y)) * 65536;
    }
  } else {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(wave * 32 + t * 16 + r) * 64 + lane] = combine_acc(acc, t, r);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int slot = wave * 8 + i;
      v[i] = red[slot * 64 + lane] + red[(32 + slot) * 64 + lane] + red[(64 + slot) * 64 + lane] +
             red[(96 + slot) * 64 + lane];
    }
  }
  __syncthreads();  // red may be reused by out()
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int slot = wave * 8 + i;
    const int t = slot >> 4, r = slot & 15;
    out(t, 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3), lane & 31, v[i]);
  }
}

// Deterministic reductions: fixed shuffle tree, lane 0 holds the result.
// Wave sum on DPP (lane 63), read back so that every lane holds it.
__device__ __forceinline__ double wave_sum_d(double v) {
  wave_sum63(v);
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)b, 63), hi = __builtin_amdgcn_readlane((int)(b >> 32), 63);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
__device__ __forceinline__ long long wave_sum_ll(long long v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, 64);
  return v;
}
// max |x| with the smallest index on ties
__device__ __forceinline__ void argmax_merge(double& v, long long& i, double v2, long long i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}
__device__ __forceinline__ void wave_argmax(double& v, long long& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    double v2 = __shfl_down(v, o, 64);
    long long i2 = __shfl_down(i, o, 64);
    argmax_merge(v, i, v2, i2);
  }
}

// Block-wide sum over NT threads, result broadcast to all threads.
__device__ __forceinline__ double block_sum_d(double v, double* sh /* >= NT/64 */) {
  v = wave_sum_d(v);
  if (lane_id() == 0) sh[wave_id()] = v;
  __syncthreads();
  double r = 0.0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) r += sh[w];
  __syncthreads();
  return r;
}
__device__ __forceinline__ int block_sum_i(int v, int* sh) {
  v = wave_sum_i(v);
  if (lane_id() == 0) sh[wave_id()] = v;
  __syncthreads();
  int r = 0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) r += sh[w];
  __syncthreads();
  return r;
}
__device__ __forceinline__ void block_argmax(double& v, long long& i, double* shv, long long* shi) {
  wave_argmax(v, i);
  if (lane_id() == 0) {
    shv[wave_id()] = v;
    shi[wave_id()] = i;
  }
  __syncthreads();
  double bv = shv[0];
  long long bi = shi[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) argmax_merge(bv, bi, shv[w], shi[w]);
  __syncthreads();
  v = bv;
  i = bi;
}

// ---------------------------------------------------------------------------
// 64x64 SPD inverse: block sweep operator (block Gauss-Jordan without
// pivoting, stable for SPD) with 4x4 pivot blocks and fp64 MFMA updates.
// A: LDS 64x64 row-major, in: matrix, out: inverse.  pbuf: LDS 1024 doubles.
// Requires blockDim.x == 256.
//
// The matrix is first scaled exactly by powers of two, A~ = S A S with
// S = diag(2^-e_i), so that every diagonal entry lies in [0.5, 2); then
// A^{-1} = S A~^{-1} S.  Sweeping the pivot block K (4 indices) with
// P = A~_KK maps A_ij -> A_ij - A_iK P^{-1} A_Kj (i, j outside K),
// A_iK -> A_iK P^{-1}, A_Kj -> P^{-1} A_Kj, A_KK -> -P^{-1}; after all 16
// blocks the matrix is -A~^{-1}.  With C = A~[:, K] - E_K all four cases
// are the single rank-4 update A -= (C P^{-1}) C^T, except the diagonal of
// the pivot block, which needs a further -2.
//
// Wave w holds tile row w of A in v_mfma_f64_16x16x4f64 accumulators
// (lane l, register r, tile nt <-> A[16 w + l/16 + 4 r][16 nt + l%16]);
// the sweep keeps A symmetric, so C^T is the pivot rows minus E_K^T, held
// by one wave: it publishes them through LDS, every lane forms P^{-1}
// (closed form by 2x2 Schur blocks) and its entry of W = -C P^{-1}, and
// each wave applies W C^T to its four tiles with four MFMAs.  One barrier
// per step (the published rows are double-buffered).
// ---------------------------------------------------------------------------
__device__ __forceinline__ v4d mfma_f64(double a, double b, v4d c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// 1 / x for the pivots of the sweep below: the hardware estimate refined by
// two Newton steps r <- r (2 - x r) (error ~ 1 ulp).  The sweep works on a
// matrix scaled to a unit-order diagonal, so x is far from the denormal and
// overflow ranges that the full IEEE division sequence guards against.
__device__ __forceinline__ double recip_nr(double x) {
  double r = __builtin_amdgcn_rcp(x);
  r = r * fma(-x, r, 2.0);
  r = r * fma(-x, r, 2.0);
  return r;
}

// Inverse of the symmetric 4x4 block [[A, B], [B^T, D]] (2x2 blocks) by the
// Schur complement S = D - B^T A^{-1} B; uses the upper triangle of P.
__device__ __forceinline__ void spd_inverse4(const double (&P)[4][4], double (&Pi)[4][4]) {
  const double ra = recip_nr(P[0][0] * P[1][1] - P[0][1] * P[0][1]);
  const double a00 = P[1][1] * ra, a01 = -P[0][1] * ra, a11 = P[0][0] * ra;
  // X = A^{-1} B
  const double x00 = a00 * P[0][2] + a01 * P[1][2], x01 = a00 * P[0][3] + a01 * P[1][3];
  const double x10 = a01 * P[0][2] + a11 * P[1][2], x11 = a01 * P[0][3] + a11 * P[1][3];
  // S = D - B^T X
  const double s00 = P[2][2] - (P[0][2] * x00 + P[1][2] * x10);
  const double s01 = P[2][3] - (P[0][2] * x01 + P[1][2] * x11);
  const double s11 = P[3][3] - (P[0][3] * x01 + P[1][3] * x11);
  const double rs = recip_nr(s00 * s11 - s01 * s01);
  const double t00 = s11 * rs, t01 = -s01 * rs, t11 = s00 * rs;
  // Y = X S^{-1}
  const double y00 = x00 * t00 + x01 * t01, y01 = x00 * t01 + x01 * t11;
  const double y10 = x10 * t00 + x11 * t01, y11 = x10 * t01 + x11 * t11;
  Pi[0][0] = a00 + (y00 * x00 + y01 * x01);
  Pi[0][1] = a01 + (y00 * x10 + y01 * x11);
  Pi[1][0] = Pi[0][1];
  Pi[1][1] = a11 + (y10 * x10 + y11 * x11);
  Pi[0][2] = -y00; Pi[0][3] = -y01;
  Pi[1][2] = -y10; Pi[1][3] = -y11;
  Pi[2][0] = -y00; Pi[3][0] = -y01;
  Pi[2][1] = -y10; Pi[3][1] = -y11;
  Pi[2][2] = t00; Pi[2][3] = t01;
  Pi[3][2] = t01; Pi[3][3] = t11;
}

template <typename T>
__device__ __forceinline__ T load_coherent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void store_coherent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A 64 x 64 inverse shared between workgroups is stored in the operand
// order of the fp64 MFMA (A operand, 16x16x4): wave w, K step ks and lane
// (li = lane % 16, lk = lane / 16) read element [16 w + li][4 ks + lk] at
// (16 w + ks) * 64 + lane, so each load instruction of a wave reads 512
// contiguous bytes.  The inverses are symmetric, so the same array serves
// the transposed operand (Z^T = G^{-1} Q^T).
__device__ __forceinline__ int ginv_index(int row, int col) {
  return (((row >> 4) * 16 + (col >> 2)) << 6) + (col & 3) * 16 + (row & 15);
}
// The consumers run in a later launch than the producer, so plain loads
// see the inverse, and after the first workgroup of an XCD they hit in its
// L2 (coherent loads would go past the L2 for every workgroup).
__device__ __forceinline__ void load_ginv(const double* ginv, double (&a)[16]) {
  const double* p = ginv + wave_id() * 1024 + lane_id();
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) a[ks] = p[ks * 64];
}
// A consumer in the producer's launch loads it the same way once the flag
// below is seen: the producer wrote it through to memory, and no workgroup
// of the launch reads those lines before the flag, so no L2 holds an older
// copy (each launch starts with clean caches); the first workgroup of each
// XCD fetches them from memory and the others hit in its L2.

// A flag between the workgroups of one launch.  The producer's stores are
// coherent (written through); once every one of them has completed
// (s_waitcnt, then the barrier) one thread sets the flag.  The waiting side
// polls it with coherent loads for at most SYNC_TICKS of the 100 MHz wall
// clock (20 ms, against a few microseconds expected); past that it raises
// FLAG_SYNC, which the host reports as EXTERND_ESYNC, and goes on.
constexpr unsigned long long SYNC_TICKS = 2000000ull;
__device__ __forceinline__ void ginv_ready(unsigned* ready) {
  if (!ready) return;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) store_coherent(ready, 1u);
}
__device__ __forceinline__ void await_flag(unsigned* ready, int* flags) {
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  while (load_coherent(ready) == 0u) {
    if (__builtin_amdgcn_s_memrealtime() - t0 > SYNC_TICKS) {
      store_coherent(flags + FLAG_SYNC, 1);
      return;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// nk: pivot blocks to sweep, ceil(bb / 4) for a block of bb real components
// whose padding is the identity.  A pivot block made only of padding has
// A - I exactly zero in its rows (the padding diagonal is exactly 1 before
// and after the power-of-two scaling, and no earlier step touches rows
// that are zero in every real column), so its step would add exactly zero:
// stopping after nk blocks gives the same inverse bit for bit.
__device__ __forceinline__ void spd_inverse64(double* A, double* pbuf, int nk, double* out = nullptr) {
  __shared__ int sexp[64];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int lr = lane >> 4, lc = lane & 15;
  if (t < 64) {
    int E = 0;
    frexp(A[t * 65], &E);
    sexp[t] = E >> 1;  // floor(E / 2)
  }
  __syncthreads();
  int er[4], ec[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    er[q] = sexp[16 * w + lr + 4 * q];
    ec[q] = sexp[16 * q + lc];
  }
  v4d acc[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      acc[nt][r] = ldexp(A[(16 * w + lr + 4 * r) * 64 + 16 * nt + lc], -(er[r] + ec[nt]));
  const double m0 = lr == 0, m1 = lr == 1, m2 = lr == 2, m3 = lr == 3;
  // The loop over the owner waves stays rolled: the sweep runs once per
  // launch, and its code is fetched cold while the streaming workgroups
  // load the memory system, so a 4x smaller body is faster.
#pragma unroll 1
  for (int ntK = 0; ntK < 4 && 4 * ntK < nk; ++ntK)
#pragma unroll
  for (int rK = 0; rK < 4; ++rK) {
    const int K = 4 * ntK + rK;
    if (K >= nk) break;
    // The sweep keeps A symmetric, so the pivot column block equals the
    // pivot rows: their owner (wave K / 4, register K % 4) publishes
    // C^T[c][j] = A[4K + c][j] - delta(j, 4K + c) and every wave builds
    // its own operands from it.  Double-buffered: one barrier per step.
    double* Rb = pbuf + (rK & 1) * 256;
    if (w == ntK) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int col = 16 * nt + lc;
        Rb[lr * 64 + col] = acc[nt][rK] - (col == 4 * K + lr ? 1.0 : 0.0);
      }
    }
    __syncthreads();
    double P[4][4], Pi[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = a; b < 4; ++b) {
        P[a][b] = Rb[a * 64 + 4 * K + b] + (a == b ? 1.0 : 0.0);
        P[b][a] = P[a][b];
      }
    double cw[4], bop[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) cw[c] = Rb[c * 64 + 16 * w + lc];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) bop[nt] = Rb[lr * 64 + 16 * nt + lc];
    spd_inverse4(P, Pi);
    // A operand: W[16 w + lc][lr] = -(C P^{-1})[16 w + lc][lr]; column lr
    // of P^{-1} picked by exact 0/1 weights (no divergent selects)
    double wc[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) wc[b] = cw[0] * Pi[0][b] + cw[1] * Pi[1][b] + cw[2] * Pi[2][b] + cw[3] * Pi[3][b];
    const double aop = -(wc[0] * m0 + wc[1] * m1 + wc[2] * m2 + wc[3] * m3);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma_f64(aop, bop[nt], acc[nt]);
  }
  // Each step also takes 2 off its pivot block's diagonal.  A pivot row is
  // published only in its own step and no later step reads the diagonal
  // entry, so all these corrections are applied here at once (the
  // accumulators stay in the MFMA registers during the sweep).
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (16 * w + lr + 4 * r == 16 * nt + lc) acc[nt][r] -= 2.0;
  // the inverse goes back to A (LDS, row-major), or to out (global, in the
  // fp64 MFMA operand order of ginv_index, for the target kernel of the
  // next launch; written through)
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * w + lr + 4 * r, col = 16 * nt + lc;
      const double v = -ldexp(acc[nt][r], -(er[r] + ec[nt]));
      if (out) store_coherent(out + ginv_index(row, col), v);
      else A[row * 64 + col] = v;
    }
  __syncthreads();
}

// Turn the raw Gram (LDS, 64x64) of a block with bb real components into
// (G + eps I) on the real block and the identity on the padding, invert,
// and write the inverse.  Zero trace -> zero inverse on the real block
// (every component is zero, Eq. (3) target is zero).
__device__ __forceinline__ void ridge_invert_store(double* G, double* colbuf, int bb, double* ginv_out) {
  // The raw Gram of the zero padding components is exactly zero, so only
  // the diagonal changes: + eps on the real block, 1 on the padding.
  __shared__ double s_tr;
  const int t = threadIdx.x;
  if (t < 64) {
    const double tr = wave_sum_d(t < bb ? G[t * 65] : 0.0);
    const double trb = __shfl(tr, 0);
    if (t == 0) s_tr = trb;
    const double eps = EXTERND_RIDGE_REL * trb / (double)bb;
    G[t * 65] = (t < bb) ? G[t * 65] + eps : 1.0;
  }
  __syncthreads();
  if (s_tr == 0.0) {
    for (int e = t; e < 4096; e += blockDim.x) {
      const int r = e >> 6, c = e & 63;
      store_coherent(ginv_out + ginv_index(r, c), (r >= bb || c >= bb) ? ((r == c) ? 1.0 : 0.0) : 0.0);
    }
    return;
  }
  spd_inverse64(G, colbuf, (bb + 3) >> 2, ginv_out);
}

// ---------------------------------------------------------------------------
// Gram matrices of a ternary factor, built by `nside` workgroups
// ---------------------------------------------------------------------------
// Partial integer Gram of X (BBP x L int8, MFMA-ready layout) over this
// workgroup's share of K steps, on int8 MFMA; all four wave results are
// summed in LDS (integer adds, order-free) and written to gparti[side].
// Returns true in the last of the nside workgroups to finish, with the
// complete Gram in G (LDS, fp64).
__device__ __forceinline__ bool side_gram_int(const v4i* __restrict__ Xmf, int64_t L, int side, int nside, int* gparti,
                              unsigned* counter, double* G, int* ired /* LDS 4096 */) {
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  const int nks = (int)(L / TILE);
  const int ks0 = (int)((long long)side * nks / nside), ks1 = (int)((long long)(side + 1) * nks / nside);
  v16i acc00 = {}, acc01 = {}, acc10 = {}, acc11 = {};
  int ks = ks0 + wave;
  // four K steps per round, loads issued before the MFMAs
  for (; ks + 12 < ks1; ks += 16) {
    v4i a[4][2];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a[u][0] = Xmf[(int64_t)(ks + 4 * u) * 128 + lane];
      a[u][1] = Xmf[(int64_t)(ks + 4 * u) * 128 + 64 + lane];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc00 = mfma_i8(a[u][0], a[u][0], acc00);
      acc01 = mfma_i8(a[u][0], a[u][1], acc01);
      acc10 = mfma_i8(a[u][1], a[u][0], acc10);
      acc11 = mfma_i8(a[u][1], a[u][1], acc11);
    }
  }
  for (; ks < ks1; ks += 4) {
    const v4i a0 = Xmf[(int64_t)ks * 128 + lane];
    const v4i a1 = Xmf[(int64_t)ks * 128 + 64 + lane];
    acc00 = mfma_i8(a0, a0, acc00);
    acc01 = mfma_i8(a0, a1, acc01);
    acc10 = mfma_i8(a1, a0, acc10);
    acc11 = mfma_i8(a1, a1, acc11);
  }
  for (int e = threadIdx.x; e < 4096; e += blockDim.x) ired[e] = 0;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int M = 8 * (r >> 2) + 4 * h + (r & 3);
    const int N = l32;
    atomicAdd(&ired[M * 64 + N], acc00[r]);
    atomicAdd(&ired[M * 64 + 32 + N], acc01[r]);
    atomicAdd(&ired[(32 + M) * 64 + N], acc10[r]);
    atomicAdd(&ired[(32 + M) * 64 + 32 + N], acc11[r]);
  }
  __syncthreads();
  int* mine = gparti + (size_t)side * 4096;
  for (int e = threadIdx.x; e < 4096; e += blockDim.x) mine[e] = ired[e];
  __threadfence();
  __syncthreads();
  __shared__ int s_last;
  if (threadIdx.x == 0) {
    const unsigned old = atomicAdd(counter, 1u);
    s_last = (old == (unsigned)(nside - 1));
  }
  __syncthreads();
  if (!s_last) return false;
  __threadfence();
  // all nside x 4 loads of a thread are independent and issued together
  // (nside <= NSIDE_INT, blockDim == NT): one round of memory latency
  int4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = make_int4(0, 0, 0, 0);
#pragma unroll
  for (int q = 0; q < NSIDE_INT; ++q) {
    const int qq = q < nside ? q : nside - 1;
    const int keep = q < nside;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int4 v = ((const int4*)(gparti + (size_t)qq * 4096))[threadIdx.x + NT * j];
      acc[j].x += keep * v.x;
      acc[j].y += keep * v.y;
      acc[j].z += keep * v.z;
      acc[j].w += keep * v.w;
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e4 = threadIdx.x + NT * j;
    G[4 * e4] = (double)acc[j].x;
    G[4 * e4 + 1] = (double)acc[j].y;
    G[4 * e4 + 2] = (double)acc[j].z;
    G[4 * e4 + 3] = (double)acc[j].w;
  }
  if (threadIdx.x == 0) *counter = 0u;
  __syncthreads();
  return true;
}

// ---------------------------------------------------------------------------
// Integer Gram of a ternary factor, computed by a small launch right after
// the factor is made (no residual stream to compete with): NSIDE_GRAM
// workgroups add X^T X (MFMA-ready layout) into the accumulator gacc
// (4096 int32) with integer atomics, exact and independent of order.  The
// launch that needs G^{-1} takes the accumulated Gram and clears gacc.
// ---------------------------------------------------------------------------
// Partial Gram over the K steps [ks0, ks1) of X, added into gacc.  Wave w
// of the first four forms the 32 x 32 block (w / 2, w % 2) of X^T X over
// all the K steps (operands: the two halves of each K step, up to GRAM_KB
// K steps of loads in flight) and adds it into gacc with integer atomics
// straight from its accumulator: no LDS, no barrier (blockDim: any
// multiple of 256).
constexpr int GRAM_KB = 20;
__device__ __forceinline__ void gram_accumulate(const v4i* __restrict__ Xmf, int ks0, int ks1, int* gacc, int* red) {
  (void)red;
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  if (wave >= 4) return;
  const int bx = wave >> 1, by = wave & 1;
  v16i acc = {};
  for (int ks = ks0; ks < ks1; ks += GRAM_KB) {
    v4i ax[GRAM_KB], ay[GRAM_KB];
#pragma unroll
    for (int u = 0; u < GRAM_KB; ++u) {
      const int kc = ks + u < ks1 ? ks + u : ks1 - 1;
      ax[u] = Xmf[(int64_t)kc * 128 + 64 * bx + lane];
      ay[u] = Xmf[(int64_t)kc * 128 + 64 * by + lane];
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first MFMA
#pragma unroll
    for (int u = 0; u < GRAM_KB; ++u) {
      const bool in = ks + u < ks1;
      acc = mfma_i8(in ? ax[u] : v4i{}, in ? ay[u] : v4i{}, acc);
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int M = 8 * (r >> 2) + 4 * h + (r & 3);
    const int v = acc[r];
    if (v) __hip_atomic_fetch_add(gacc + (32 * bx + M) * 64 + 32 * by + l32, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Side workgroup `side` of `nside` adds its share of the K steps of X^T X
// into gacc; the last to arrive (arrival counter, reset by it) takes the
// accumulated Gram into G (LDS, fp64) with coherent loads, as the atomics
// of the other side workgroups belong to the same launch, and clears gacc
// for the next accumulation.  red: LDS, 4 x 4096 int32 (may alias G).
__device__ __forceinline__ bool side_gram_acc(const v4i* __restrict__ Xmf, int64_t L_pad, int side, int nside,
                                              int* gacc, unsigned* counter, double* G, int* red) {
  const int nks = (int)(L_pad / TILE);
  gram_accumulate(Xmf, (int)((long long)side * nks / nside), (int)((long long)(side + 1) * nks / nside), gacc, red);
  __builtin_amdgcn_s_waitcnt(0);  // this wave's atomics have been performed
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned old = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (old == (unsigned)(nside - 1));
  }
  __syncthreads();
  if (!s_last) return false;
  if (threadIdx.x == 0) store_coherent(counter, 0u);
  int v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = load_coherent(gacc + threadIdx.x + NT * j);
#pragma unroll
  for (int j = 0; j < 16; ++j) G[threadIdx.x + NT * j] = (double)v[j];
#pragma unroll
  for (int j = 0; j < 16; ++j) gacc[threadIdx.x + NT * j] = 0;
  __syncthreads();
  return true;
}

// ---------------------------------------------------------------------------
// Weighted Gram X_a^T diag(h~) X_b of ternary factors (Sec. 2.5) on int8
// MFMA.  The weights enter as the integers
//   H_j = min(rint(h~_j / max h~ 2^w), 2^w - 1),  w = min(WSHIFT_MAX, 61 - ceil(log2 n_pad)),
// split into WDIG planes of WDIG_BITS-bit digits (hdig[d * n_pad + j], digit d
// of H_j, least significant first; written once per call by k_prep), so that
//   sum_j H_j x_jc y_jc' = sum_d 128^d sum_j dig_d(j) x_jc y_jc'
// is an exact integer below 2^61: every product digit x trit lies in
// [-127, 127] and is itself an int8 MFMA operand.  The Gram is that integer
// times the unit max h~ 2^-w.  With w = 42 (n_pad <= 2^19) each weight
// differs from h~_j by at most 2^-43 max h~, the order of the rounding of
// an fp64 sum over the n weights.  The operands dig_d(j) y_jc are formed
// where V is made (Wmf: plane d at d * wstride, the MFMA-ready layout of
// V), so that the Gram itself is loads and MFMAs only.
// ---------------------------------------------------------------------------
// Bytes t (trits: 0x00, 0x01, 0xFF) times bytes d (digits 0..127), byte by
// byte: d where t = 1, -d where t = -1 (two's complement ~d + 1, the + 1
// added below bit 7 of each byte, so no carry crosses a byte), 0 where t = 0.
__device__ __forceinline__ int trit_times_digit(int t, int d) {
  const unsigned tu = (unsigned)t;
  const unsigned one = tu & 0x01010101u;         // 1 in the bytes where t != 0
  const unsigned neg = (tu >> 7) & 0x01010101u;  // 1 in the bytes where t < 0
  const unsigned y = ((unsigned)d & (one * 0xFFu)) ^ (neg * 0xFFu);
  return (int)(((y & 0x7F7F7F7Fu) + neg) ^ (y & 0x80808080u));
}

// The accumulator blocks of a 64 x 64 int8-MFMA Gram (00, 01, 10, 11; SAME:
// 10 = 01^T is neither formed nor stored) to mine (4096 int32, row-major).
template <bool SAME>
__device__ __forceinline__ void store_gram_blocks(const v16i* acc, int* mine) {
  const int lane = lane_id();
  const int h = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int M = 8 * (r >> 2) + 4 * h + (r & 3);
    const int N = l32;
    mine[M * 64 + N] = acc[0][r];
    mine[M * 64 + 32 + N] = acc[1][r];
    if (!SAME) mine[(32 + M) * 64 + N] = acc[2][r];
    mine[(32 + M) * 64 + 32 + N] = acc[SAME ? 2 : 3][r];
  }
}

// X_a^T diag(H) X_b over the K steps [ks0, ks1) (MFMA-ready layouts: Xa,
// and Wb = the digit-scaled planes of X_b, plane stride wstride bytes;
// SAME: X_b = X_a, a symmetric Gram of which the lower-left 32 x 32 block
// is left out), added into g64 (int64 atomics on the nonzero entries:
// exact, order-free).  Wave w forms plane w over all the K steps (A) and
// plane 4 + w / 2 over half of them (B).  The planes are added through LDS
// in two rounds, A then B, into int64 per entry (every partial sum stays
// below 2^42 * 32 (ks1 - ks0)).  blockDim == NT.  red: LDS, 4 x 4096 int32.
static_assert(WDIG == 6 && NT == 256, "planes 0-3 on the four waves, 4-5 on wave pairs");
template <bool SAME>
__device__ __forceinline__ void gram_w_accumulate(const v4i* Xa, const int8_t* Wb, int64_t wstride, int ks0,
                                                  int ks1, long long* g64, int* red) {
  constexpr int KR = SAME ? 4 : 2;  // K steps of loads in flight (register budget of two waves per SIMD)
  constexpr int NB = SAME ? 3 : 4;
  const int lane = lane_id(), wave = wave_id();
  const int kmid = ks0 + (ks1 - ks0 + 1) / 2;
  const int kb0 = (wave & 1) ? kmid : ks0, kb1 = (wave & 1) ? ks1 : kmid;
  const v4i* WA = (const v4i*)(Wb + (int64_t)wave * wstride);
  const v4i* WB = (const v4i*)(Wb + (int64_t)(4 + (wave >> 1)) * wstride);
  v16i accA[NB], accB[NB];
#pragma unroll
  for (int q = 0; q < NB; ++q) accA[q] = accB[q] = v16i{};
  for (int ks = ks0; ks < ks1; ks += KR) {
    v4i a[KR][2], wa[KR][2], wb[KR][2];
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      // every load from a clamped K step (a load under a branch would be
      // waited for before the next one is issued); the steps past ks1 are
      // skipped below
      const int64_t kk = ks + u < ks1 ? ks + u : ks0;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        a[u][t] = Xa[kk * 128 + 64 * t + lane];
        wa[u][t] = WA[kk * 128 + 64 * t + lane];
        wb[u][t] = WB[kk * 128 + 64 * t + lane];
      }
    }
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      const int kk = ks + u;
      if (kk < ks1) {  // uniform over the wave
        accA[0] = mfma_i8(a[u][0], wa[u][0], accA[0]);
        accA[1] = mfma_i8(a[u][0], wa[u][1], accA[1]);
        if (!SAME) accA[2] = mfma_i8(a[u][1], wa[u][0], accA[2]);
        accA[NB - 1] = mfma_i8(a[u][1], wa[u][1], accA[NB - 1]);
        if (kk >= kb0 && kk < kb1) {  // uniform over the wave
          accB[0] = mfma_i8(a[u][0], wb[u][0], accB[0]);
          accB[1] = mfma_i8(a[u][0], wb[u][1], accB[1]);
          if (!SAME) accB[2] = mfma_i8(a[u][1], wb[u][0], accB[2]);
          accB[NB - 1] = mfma_i8(a[u][1], wb[u][1], accB[NB - 1]);
        }
      }
    }
  }
  constexpr int PER = 4096 / NT;
  long long v[PER];
  store_gram_blocks<SAME>(accA, red + wave * 4096);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = threadIdx.x + NT * j;
    const long long r0 = red[e], r1 = red[4096 + e], r2 = red[8192 + e], r3 = red[12288 + e];
    v[j] = r0 + (r1 << WDIG_BITS) + (r2 << (2 * WDIG_BITS)) + (r3 << (3 * WDIG_BITS));
  }
  __syncthreads();  // red is rewritten by round B
  store_gram_blocks<SAME>(accB, red + wave * 4096);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = threadIdx.x + NT * j;
    const long long r0 = red[e], r1 = red[4096 + e], r2 = red[8192 + e], r3 = red[12288 + e];
    v[j] += ((r0 + r1) << (4 * WDIG_BITS)) + ((r2 + r3) << (5 * WDIG_BITS));
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = threadIdx.x + NT * j;
    const bool stored = !SAME || (e >> 6) < 32 || (e & 63) >= 32;  // SAME: no lower-left block
    if (stored && v[j]) __hip_atomic_fetch_add(g64 + e, v[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The symmetric weighted Gram X^T diag(H) X over the K steps [ks0, ks1) by
// blocks: wave w in {0, 1, 3} forms block (w / 2, w % 2) over all six
// digit planes (operands: half w / 2 of each K step of X and half w % 2 of
// each digit-scaled plane, GRAMW_KB K steps of loads issued before their
// MFMAs), combines the planes into int64 per entry (sum_d 128^d plane_d)
// and adds the block into g64 with integer atomics straight from its
// accumulators: no LDS, no barrier.  The lower-left block is the transpose
// of the upper-right one and is not formed.
constexpr int GRAMW_KB = 4;
__device__ __forceinline__ void gram_w_blocks(const v4i* __restrict__ Xa, const int8_t* __restrict__ Wb,
                                              int64_t wstride, int ks0, int ks1, long long* g64) {
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  if (wave >= 4 || wave == 2) return;
  const int bx = wave >> 1, by = wave & 1;
  v16i acc[WDIG];
#pragma unroll
  for (int d = 0; d < WDIG; ++d) acc[d] = v16i{};
  for (int ks = ks0; ks < ks1; ks += GRAMW_KB) {
    v4i a[GRAMW_KB], wv[GRAMW_KB][WDIG];
#pragma unroll
    for (int u = 0; u < GRAMW_KB; ++u) {
      const int64_t kc = ks + u < ks1 ? ks + u : ks0;
      a[u] = Xa[kc * 128 + 64 * bx + lane];
#pragma unroll
      for (int d = 0; d < WDIG; ++d)
        wv[u][d] = ((const v4i*)(Wb + (int64_t)d * wstride))[kc * 128 + 64 * by + lane];
    }
    __builtin_amdgcn_sched_barrier(0);  // every load issued before the first MFMA
#pragma unroll
    for (int u = 0; u < GRAMW_KB; ++u) {
      const v4i x = ks + u < ks1 ? a[u] : v4i{};
#pragma unroll
      for (int d = 0; d < WDIG; ++d) acc[d] = mfma_i8(x, wv[u][d], acc[d]);
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int M = 8 * (r >> 2) + 4 * h + (r & 3);
    long long v = 0;
#pragma unroll
    for (int d = 0; d < WDIG; ++d) v += (long long)acc[d][r] * (1ll << (WDIG_BITS * d));
    if (v) __hip_atomic_fetch_add(g64 + (32 * bx + M) * 64 + 32 * by + l32, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The symmetric weighted Gram from its accumulator (upper-left, upper-right
// and lower-right blocks; the lower-left one is the transpose of the
// upper-right): G (LDS, fp64) = g64 * unit, with coherent loads (the
// atomics of the other workgroups belong to the same launch); g64 is
// cleared for the next accumulation.
__device__ __forceinline__ void take_gram_w(long long* g64, double unit, double* G) {
  constexpr int PER = 4096 / NT;
  long long v[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int e = threadIdx.x + NT * j, r = e >> 6, c = e & 63;
    v[j] = load_coherent(g64 + ((r >= 32 && c < 32) ? c * 64 + r : e));
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) G[threadIdx.x + NT * j] = (double)v[j] * unit;
  __syncthreads();  // every entry has been read before any is cleared
#pragma unroll
  for (int j = 0; j < PER; ++j) g64[threadIdx.x + NT * j] = 0;
  __syncthreads();
}

// Side workgroup `side` of `nside` adds its share of the K steps of
// V^T diag(H) V (V and its digit-scaled planes Wmf) into g64; the last to
// arrive (arrival counter, reset by it)
// takes the weighted Gram into G.  red: LDS, 4 x 4096 int32 (may alias G).
__device__ __forceinline__ bool side_gram_w(const v4i* __restrict__ Vmf, const int8_t* __restrict__ Wmf,
                                            int64_t wstride, int64_t n_pad, int side, int nside, long long* g64,
                                            double unit, unsigned* counter, double* G, int* red) {
  const int nks = (int)(n_pad / TILE);
  (void)red;
  gram_w_blocks(Vmf, Wmf, wstride, (int)((long long)side * nks / nside), (int)((long long)(side + 1) * nks / nside),
                g64);
  __builtin_amdgcn_s_waitcnt(0);  // this wave's atomics have been performed
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned old = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (old == (unsigned)(nside - 1));
  }
  __syncthreads();
  if (!s_last) return false;
  if (threadIdx.x == 0) store_coherent(counter, 0u);
  take_gram_w(g64, unit, G);
  return true;
}

// Consumer (a later launch than the producer, so plain accesses suffice):
// the accumulated Gram into G (LDS, fp64); gacc is cleared for the next
// accumulation.  blockDim == NT: 16 entries per thread, loaded in one round.
__device__ __forceinline__ void take_gram(int* gacc, double* G) {
  int4 v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = ((const int4*)gacc)[threadIdx.x + NT * j];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * (threadIdx.x + NT * j);
    G[e] = (double)v[j].x;
    G[e + 1] = (double)v[j].y;
    G[e + 2] = (double)v[j].z;
    G[e + 3] = (double)v[j].w;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) ((int4*)gacc)[threadIdx.x + NT * j] = make_int4(0, 0, 0, 0);
}


// ---------------------------------------------------------------------------
// Targets on fp64 MFMA (v_mfma_f64_16x16x4f64), one 32-index tile at a
// time, plus the per-tile statistics of |x| that T_tau needs (Eq. (2)):
// the sum, the max and the smallest index attaining it (indices < L only),
// written component-major as ps/pm/pi[c * ntile + tile].
// Wave w computes components 16 w .. 16 w + 15 of both 16-index halves:
// lane l, register r <-> component 16 w + l/16 + 4 r, index 16 h + l%16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void tile_stats(const v4d (&x)[2], int w, int64_t i0, int64_t L, int ntile, int tile,
                                           double* __restrict__ ps, double* __restrict__ pm, int* __restrict__ pi) {
  const int lane = lane_id();
  const int li = lane & 15, lk = lane >> 4;
  const int64_t ia = i0 + li, ib = i0 + 16 + li;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const double a0 = ia < L ? fabs(x[0][r]) : 0.0, a1 = ib < L ? fabs(x[1][r]) : 0.0;
    double s = a0 + a1;
    // invalid indices never win the max; the 16 lanes of a row (one
    // component) are reduced on DPP into lane 15 of the row
    double mv = ia < L ? a0 : -1.0;
    long long mi = ia;
    argmax_merge(mv, mi, ib < L ? a1 : -1.0, ib);
    int mi32 = (int)mi;
    row_sum15(s);
    row_argmax15(mv, mi32);
    mi = mi32;
    if (li == 15) {
      const int c = 16 * w + lk + 4 * r;
      ps[(int64_t)c * ntile + tile] = s;
      pm[(int64_t)c * ntile + tile] = mv;
      pi[(int64_t)c * ntile + tile] = (int)mi;
    }
  }
}

// ---------------------------------------------------------------------------
// V-step contraction P = U^T R  (Eq. (3), first half; the target
// Y = G_U^{-1} P follows in k_vtarget)
// grid: nside side WGs (the U Gram U^T U on int8 MFMA over K slices, then
//       in the last of them the ridge and inverse G_U^{-1}) followed by
//       (n_pad/32 column tiles) x gv row groups, each storing its exact
//       int64 partial of the P tile.
// Each WG owns 32 columns and a contiguous range of 32-row K steps, split
// over its 4 waves; A = U (MFMA-ready layout), B = R digit planes.  Lane
// (j, h) loads column j, rows 16h .. 16h+15 of the K step: every load
// instruction reads two full 128-byte row segments.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_vstep(const float* __restrict__ R, const v4i* __restrict__ Umf,
                                              long long* __restrict__ Pp, const int* __restrict__ cshift,
                                              int64_t m_pad, int64_t n_pad, int gv, int bb, int* gacc,
                                              unsigned* gcounter, double* ginvU, int nside, double* __restrict__ Y,
                                              double* ps, double* pm, int* pi, int64_t n, unsigned* tcnt,
                                              unsigned* ready, int* flags) {
  // side path: ired 16 KB | G 32 KB | inverse scratch 8 KB; contraction:
  // 64 KB wave reduction
  __shared__ __attribute__((aligned(16))) long long smem[8192];
  if ((int)blockIdx.x < nside) {
    // the side path is the launch's critical path: its waves win issue
    // arbitration against the streaming waves sharing their SIMDs
    __builtin_amdgcn_s_setprio(3);
    double* Gs = (double*)(smem + 2048);
    double* pbuf = Gs + 4096;
    if (!side_gram_acc(Umf, m_pad, blockIdx.x, nside, gacc, gcounter, Gs, (int*)smem)) return;
    ridge_invert_store(Gs, pbuf, bb, ginvU);
    ginv_ready(ready);
    return;
  }
  // as in the U-step, the second workgroups on the side workgroups' CUs
  // (grid indices 256 .. 256 + nside - 1) stay empty
  const int b0 = blockIdx.x - nside;
  if (nside && b0 >= 256 - nside && b0 < 256) return;
  const int b = (nside && b0 >= 256) ? b0 - nside : b0;
  const int nct = (int)(n_pad / TILE);
  if (b >= nct * gv) return;
  const int ct = b % nct, g = b / nct;
  const int nks = (int)(m_pad / TILE);
  const int ks0 = (int)((long long)g * nks / gv), ks1 = (int)((long long)(g + 1) * nks / gv);
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  // lane (j, h) converts column ct * 32 + j only: its own exponent
  const int s = cshift[(int64_t)ct * TILE + l32];
  v16i acc[2][4];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int p = 0; p < 4; ++p) acc[t][p] = v16i{};
  const float* Rc = R + (int64_t)ct * TILE + l32;
  // software pipeline: the loads of K step ks + 4 are in flight while
  // step ks is converted and multiplied
  float xn[16];
  v4i an0 = {}, an1 = {};
  int ks = ks0 + wave;
  if (ks < ks1) {
    const int64_t i0 = (int64_t)ks * TILE + 16 * h;
    an0 = Umf[(int64_t)ks * 128 + lane];
    an1 = Umf[(int64_t)ks * 128 + 64 + lane];
#pragma unroll
    for (int q = 0; q < 16; ++q) xn[q] = Rc[(i0 + q) * n_pad];
  }
  for (; ks < ks1; ks += 4) {
    unsigned y[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) y[q] = fx_biased(xn[q], s);
    const v4i a0 = an0, a1 = an1;
    const int ksn = ks + 4;
    if (ksn < ks1) {
      const int64_t i0 = (int64_t)ksn * TILE + 16 * h;
      an0 = Umf[(int64_t)ksn * 128 + lane];
      an1 = Umf[(int64_t)ksn * 128 + 64 + lane];
#pragma unroll
      for (int q = 0; q < 16; ++q) xn[q] = Rc[(i0 + q) * n_pad];
    }
    v4i P[4];
    make_planes(y, P);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      acc[0][p] = mfma_i8(a0, P[p], acc[0][p]);
      acc[1][p] = mfma_i8(a1, P[p], acc[1][p]);
    }
  }
  // out[t][M = component][N = column]: this row group's partial P tile, at
  // the column's fixed-point scale
  long long* Pg = Pp + ((int64_t)g * BBP) * n_pad + (int64_t)ct * TILE;
  if (!Y) {
    reduce_waves(smem, acc, ks1 - ks0 <= FOLD_KMAX,
                 [&](int t, int M, int N, long long v) { Pg[(int64_t)(32 * t + M) * n_pad + N] = v; });
    return;
  }
  // The partials go out written through, and the last of the column tile's
  // gv row groups to arrive forms its targets Y = G_U^{-1} P (Eq. (3) first
  // half) and their T_tau statistics (one 32-column tile).
  reduce_waves(smem, acc, ks1 - ks0 <= FOLD_KMAX,
               [&](int t, int M, int N, long long v) { store_coherent(Pg + (int64_t)(32 * t + M) * n_pad + N, v); });
  __builtin_amdgcn_s_waitcnt(0);
  __shared__ int s_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned old = __hip_atomic_fetch_add(tcnt + ct, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = old == (unsigned)(gv - 1);
  }
  __syncthreads();
  if (!s_last) return;
  if (threadIdx.x == 0) store_coherent(tcnt + ct, 0u);
  // P = sum of the partials (exact int64), at the column's scale 2^-s:
  // Ps[c * 33 + j], thread (c = e / 32, j = e % 32) for e = tid + 256 i
  double* Ps = (double*)smem;
  const int64_t j0 = (int64_t)ct * TILE;
  // gv <= 6 (the usual case): thread t takes columns j0 + jp, jp + 1
  // (jp = 2 (t % 16)) of components t / 16 + 16 i, i < 4, with the gv
  // partials of its four pairs all in flight at once, as 16-byte plain
  // loads from clamped row groups (masked in the sum).  Plain loads see the
  // written-through partials: no workgroup of this launch reads these lines
  // before the arrival count shows them complete, and each launch starts
  // with clean caches.
  if (gv <= GV_ONE) {
    const int jp = 2 * (threadIdx.x & 15), cq = threadIdx.x >> 4;
    v2l v[4][GV_ONE];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int gg = 0; gg < GV_ONE; ++gg) {
        const int gc = gg < gv ? gg : 0;
        v[i][gg] = *(const v2l*)(Pp + ((int64_t)gc * BBP + cq + 16 * i) * n_pad + j0 + jp);
      }
    const int sh0 = cshift[j0 + jp], sh1 = cshift[j0 + jp + 1];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      long long s0 = 0, s1 = 0;
#pragma unroll
      for (int gg = 0; gg < GV_ONE; ++gg) {
        s0 += gg < gv ? v[i][gg].x : 0ll;
        s1 += gg < gv ? v[i][gg].y : 0ll;
      }
      const int c = cq + 16 * i;
      Ps[c * 33 + jp] = ldexp((double)s0, -sh0);
      Ps[c * 33 + jp + 1] = ldexp((double)s1, -sh1);
    }
  } else {
    // thread (c = e / 32, j = e % 32) for e = tid + 256 i, in two rounds of
    // four entries: the gv partials of each entry, all in flight at once
  #pragma unroll
    for (int half = 0; half < 2; ++half) {
      long long v[4][GV_MAX];
  #pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = threadIdx.x + NT * (4 * half + i), c = e >> 5, j = e & 31;
  #pragma unroll
        for (int gg = 0; gg < GV_MAX; ++gg)
          v[i][gg] = gg < gv ? load_coherent(Pp + ((int64_t)gg * BBP + c) * n_pad + j0 + j) : 0ll;
      }
  #pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = threadIdx.x + NT * (4 * half + i), c = e >> 5, j = e & 31;
        long long sum = 0;
  #pragma unroll
        for (int gg = 0; gg < GV_MAX; ++gg) sum += v[i][gg];
        Ps[c * 33 + j] = ldexp((double)sum, -cshift[j0 + j]);
      }
    }
  }
  if (threadIdx.x == 0) await_flag(ready, flags);
  __syncthreads();
  double a[16];
  load_ginv(ginvU, a);
  const int li = lane & 15, lk = lane >> 4;
  v4d y[2] = {v4d{}, v4d{}};
  // A = G^{-1}[16 w + li][4 ks + lk], B = P[4 ks + lk][li (+16)] (LDS)
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    y[0] = mfma_f64(a[ks], Ps[(4 * ks + lk) * 33 + li], y[0]);
    y[1] = mfma_f64(a[ks], Ps[(4 * ks + lk) * 33 + 16 + li], y[1]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    double* row = Y + (int64_t)(16 * wave + lk + 4 * r) * n_pad + j0;
    row[li] = y[0][r];
    row[16 + li] = y[1][r];
  }
  tile_stats(y, wave, j0, n, (int)(n_pad / TILE), ct, ps, pm, pi);
}

// V-step target Y = G_U^{-1} P (Eq. (3) first half) and its T_tau
// statistics, after the contraction launch: P is the sum of the gv row
// groups' exact partials, G_U^{-1} comes from the contraction's side path.
// grid: n_pad / 16 tiles of 16 columns (statistics per 16-column tile).
template <int GV>
__device__ __forceinline__ void vtarget_sum16(const long long* __restrict__ Pp, int s, int64_t n_pad, int64_t j0,
                                              double* Ps) {
  long long v[GV][4];
#pragma unroll
  for (int g = 0; g < GV; ++g)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = threadIdx.x + q * NT, c = e >> 4, jj = e & 15;
      v[g][q] = Pp[((int64_t)g * BBP + c) * n_pad + j0 + jj];
    }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    long long acc = 0;
#pragma unroll
    for (int g = 0; g < GV; ++g) acc += v[g][q];
    const int e = threadIdx.x + q * NT;
    Ps[(e >> 4) * 17 + (e & 15)] = ldexp((double)acc, -s);  // column j0 + (e & 15) = j0 + (tid & 15)
  }
}

// WIDE (a block of nq > 1 quarters, Sec. 2.4 with b up to BMAX): the
// quarter's targets Y_q = sum_q' G^{-1}[q][q'] P_q', with ginvU the block
// row q of the nq x nq blocks (block q' at ginvU + 4096 q') and Pp the
// partials of quarter 0 (quarter q' at Pp + q' pq_stride); Y, ps, pm, pi are
// the quarter's.
template <bool WIDE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_vtarget(const long long* __restrict__ Pp, const int* __restrict__ cshift,
                                                int64_t n_pad, int gv, const double* __restrict__ ginvU,
                                                double* __restrict__ Y, int64_t n, double* ps, double* pm, int* pi,
                                                int nq, int64_t pq_stride) {
  __shared__ double Ps[64 * 17];
  const int tile = blockIdx.x;
  const int ntile = (int)(n_pad / 16);
  const int64_t j0 = (int64_t)tile * 16;
  const int lane = lane_id(), w = wave_id();
  const int li = lane & 15, lk = lane >> 4;
  // the contraction's exponent of the one column this thread sums
  const int s = cshift[j0 + (threadIdx.x & 15)];
  double a[16];
  v4d y[2] = {v4d{}, v4d{}};
  static_assert(GV_MAX == 8, "one case per group count");
  for (int q2 = 0; q2 < (WIDE ? nq : 1); ++q2) {
    load_ginv(ginvU + (WIDE ? (int64_t)q2 * 4096 : 0), a);
    const long long* Pq = Pp + (WIDE ? q2 * pq_stride : 0);
    if (WIDE && q2 > 0) __syncthreads();  // Ps of the previous quarter consumed
    switch (gv) {
      case 1: vtarget_sum16<1>(Pq, s, n_pad, j0, Ps); break;
      case 2: vtarget_sum16<2>(Pq, s, n_pad, j0, Ps); break;
      case 3: vtarget_sum16<3>(Pq, s, n_pad, j0, Ps); break;
      case 4: vtarget_sum16<4>(Pq, s, n_pad, j0, Ps); break;
      case 5: vtarget_sum16<5>(Pq, s, n_pad, j0, Ps); break;
      case 6: vtarget_sum16<6>(Pq, s, n_pad, j0, Ps); break;
      case 7: vtarget_sum16<7>(Pq, s, n_pad, j0, Ps); break;
      default: vtarget_sum16<8>(Pq, s, n_pad, j0, Ps); break;
    }
    __syncthreads();
    // A = G^{-1}[16 w + li][4 ks + lk] (a), B = P[4 ks + lk][li] (LDS)
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) y[0] = mfma_f64(a[ks], Ps[(4 * ks + lk) * 17 + li], y[0]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) Y[(int64_t)(16 * w + lk + 4 * r) * n_pad + j0 + li] = y[0][r];
  // the second half of the 32-wide statistics tile lies past the limit
  tile_stats(y, w, j0, (j0 + 16 < n ? j0 + 16 : n), ntile, tile, ps, pm, pi);
}
// ---------------------------------------------------------------------------
// U-step Q = R diag(h~) V  (Eq. (3) second half, Sec. 2.5); the target
// Z = Q G_V^{-1} follows in k_utarget
// grid: nside side WGs (V^T V on int8 MFMA over K slices, weighted
//       V^T diag(H) V from the weights' digit planes; the last of them adds
//       the ridge and inverts; the raw Gram is kept for the scale solve)
//       followed by ntile row groups of `rows` <= 32 rows, sized so
//       that the whole grid is resident at two workgroups per CU and every
//       CU streams the same share of R; each row group stores Q, waits for
//       G_V^{-1} and writes its Z rows and T_tau statistics.
// Each WG owns `rows` full rows (one 32-row MFMA tile; rows past `rows`
// are neither loaded nor stored); its 4 waves interleave 32-column K steps.
// A = R digit planes (rows x columns), B = V (MFMA-ready layout).  Each
// wave streams its 32 x 32 residual tiles into LDS with direct loads
// (8 lanes per 128-byte row segment, 16-byte chunks XOR-swizzled by row)
// NST_U tiles ahead, then reads them back in operand order (lane (i, h):
// row i, columns 16h .. 16h+15).  The weighted variant stages the 32
// weights of the K step beside each tile.
// ---------------------------------------------------------------------------
constexpr int NST_U = 3;
constexpr int USTAGE_B = 4096 + 256;  // bytes per staged K step: tile + weights
// LDS of k_ustep: the staging area (4 waves x NST_U K steps), which the
// 64 KB wave reduction reuses afterwards
constexpr int USTEP_SMEM_LL = (4 * NST_U * USTAGE_B + 7) / 8 > 8192 ? (4 * NST_U * USTAGE_B + 7) / 8 : 8192;

template <bool WEIGHTED>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_ustep(const float* __restrict__ R, const v4i* __restrict__ Vmf,
                                              const int8_t* __restrict__ Vr, const double* __restrict__ hw,
                                              double* __restrict__ Q, float* __restrict__ rowb,
                                              int64_t m_pad, int64_t n_pad, int bb, int* gacc, unsigned* counter,
                                              double* ginvV, double* gramV, int nside, int rows,
                                              const int8_t* __restrict__ Wmf, long long* gacc64,
                                              const double* __restrict__ hwmax, double* __restrict__ Z, double* ps,
                                              double* pm, int* pi, int64_t m, unsigned* ready, int* flags,
                                              int storeQ) {
  // side path: ired 16 KB | G 32 KB | inverse scratch 8 KB; contraction:
  // 4 waves x NST_U staged K steps (52 KB), then the 64 KB wave reduction
  __shared__ __attribute__((aligned(16))) long long smem[USTEP_SMEM_LL];
  if ((int)blockIdx.x < nside) {
    // critical path of the launch (see k_vstep)
    __builtin_amdgcn_s_setprio(3);
    double* Gs = (double*)(smem + 2048);
    double* pbuf = Gs + 4096;
    if (WEIGHTED) {
      // V^T diag(H) V on int8 MFMA from the digit-scaled planes of V; the last
      // side workgroup keeps the raw Gram for the scale solve, adds the
      // ridge and inverts
      if (side_gram_w(Vmf, Wmf, (int64_t)BMAX * n_pad, n_pad, blockIdx.x, nside, gacc64, hwmax[1], counter, Gs,
                      (int*)smem)) {
        for (int e = threadIdx.x; e < 4096; e += NT) gramV[e] = Gs[e];
        __syncthreads();
        ridge_invert_store(Gs, pbuf, bb, ginvV);
        ginv_ready(ready);
      }
      return;
    }
    if (side_gram_acc(Vmf, n_pad, blockIdx.x, nside, gacc, counter, Gs, (int*)smem)) {
      for (int e = threadIdx.x; e < 4096; e += NT) gramV[e] = Gs[e];
      __syncthreads();
      ridge_invert_store(Gs, pbuf, bb, ginvV);
      ginv_ready(ready);
    }
    return;
  }
  // The workgroups are dispatched one per CU first (the side workgroups
  // take the first nside CUs), then a second one per CU; the second ones
  // on the side workgroups' CUs (indices 256 .. 256 + nside - 1 of the
  // grid) are left empty so that the inverse sweep has its CU to itself,
  // and the row groups after them shift down.  Were the placement
  // different, those slots would only cost their share of the stream.
  const int rt0 = blockIdx.x - nside;
  if (nside && rt0 >= 256 - nside && rt0 < 256) return;
  const int rt = (nside && rt0 >= 256) ? rt0 - nside : rt0;
  const int64_t i0 = (int64_t)rt * rows;
  if (i0 >= m_pad) return;  // the slots counted for the empty ones, past the last row group
  const int valid = (int)(m_pad - i0 < rows ? m_pad - i0 : rows);
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  // lane (i, h) converts row i0 + i only: its own exponent, from the row's
  // bound (rows past `valid` read the last valid row's; their results are
  // discarded)
  __shared__ int s_row[TILE];
  __shared__ int s_rmax[4][64];

  // the row's largest |x h~_j| seen by this lane: fp32 |x| unweighted, the
  // extreme biased fixed-point words weighted (|x h~_j 2^s| <= |q| + 1/2)
  float rmax = 0.0f;
  int ymin = 0x00808080, ymax = 0x00808080;  // q = 0: also right for a wave without K steps
  v16i acc[2][4];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int p = 0; p < 4; ++p) acc[t][p] = v16i{};
  const int nks = (int)(n_pad / TILE);
  char* wst = (char*)smem + wave * (NST_U * USTAGE_B);
  // loader mapping: lane -> row 8 q + lane / 8, 16-byte chunk lane % 8,
  // stored at chunk position (lane % 8) ^ (row % 8); rows >= valid are
  // not loaded (their staging rows hold stale values; the MFMA output rows
  // they feed are discarded), so a stage issues between 1 and 4 direct
  // loads.  The operand reads wait until at most NLD * (NST_U - 1) loads are
  // outstanding; even with one direct load per stage at least that many
  // follow the stage read (its two factor loads, then NST_U - 1 stages of
  // >= 3 loads each; weighted >= 4), so the bound holds for NST_U = 3.
  static_assert(NST_U == 3, "vmcnt bound of the operand reads assumes three stages");
  const int lrow = lane >> 3;
  const float* Rld = R + (i0 + lrow) * n_pad + (((lane & 7) ^ lrow) * 4);
  constexpr int NLD = WEIGHTED ? 5 : 4;  // direct loads per staged K step
  v4i bn[NST_U][2];
  // stage st <- K step kk (< nks); nothing is loaded past the last K step
  auto issue = [&](int kk, int st) {
    char* dst = wst + st * USTAGE_B;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (8 * q + lrow < valid)
        __builtin_amdgcn_global_load_lds(Rld + (int64_t)8 * q * n_pad + (int64_t)kk * TILE,
                                         (lds_void*)(dst + q * 1024), 16, 0, 0);
    if (WEIGHTED)
      __builtin_amdgcn_global_load_lds((const float*)(hw + (int64_t)kk * TILE) + lane, (lds_void*)(dst + 4096), 4, 0,
                                       0);
    bn[st][0] = Vmf[(int64_t)kk * 128 + lane];
    bn[st][1] = Vmf[(int64_t)kk * 128 + 64 + lane];
  };
  // The rows' bounds go to LDS with a direct load issued before the first
  // stages and are read back behind an explicit wait: a register-destined
  // load here makes the compiler drain every stage of the stream loop.
  // Lane l of each wave stages the bound of row min(l % 32, valid - 1).
  __shared__ float s_rbw[4][64];
  __builtin_amdgcn_global_load_lds(rowb + i0 + (l32 < valid ? l32 : valid - 1), (lds_void*)&s_rbw[wave][0], 4, 0, 0);
#pragma unroll
  for (int d = 0; d < NST_U - 1; ++d)
    if (wave + 4 * d < nks) issue(wave + 4 * d, d);
  // with both first stages issued (nks >= 8) at least 2 x 3 loads follow
  // the bound's (one direct residual load and two factor loads per stage)
  const unsigned rba = lds_addr(&s_rbw[wave][lane]);
  const float rbound = nks >= 4 * (NST_U - 1) ? lds_read1_after<2 * 3>(rba) : lds_read1_after<0>(rba);
  const int s = fx_shift(rbound);
  const float p2s = __builtin_amdgcn_ldexpf(1.0f, s);  // x 2^s = x * p2s exactly
  const double cw = weighted_round_const(s);
  // operand read: row l32, logical chunks 4h .. 4h+3
  const unsigned sw = (unsigned)(l32 & 7);
  const unsigned o0 = l32 * 128 + ((4 * h + 0) ^ sw) * 16, o1 = l32 * 128 + ((4 * h + 1) ^ sw) * 16;
  const unsigned o2 = l32 * 128 + ((4 * h + 2) ^ sw) * 16, o3 = l32 * 128 + ((4 * h + 3) ^ sw) * 16;
  const unsigned wbase = lds_addr(wst);
  for (int ks = wave; ks < nks; ks += 4 * NST_U) {
#pragma unroll
    for (int u = 0; u < NST_U; ++u) {
      const int kk = ks + 4 * u, kn = kk + 4 * (NST_U - 1);
      if (kn < nks) issue(kn, (u + NST_U - 1) % NST_U);
      if (kk < nks) {
        const unsigned b = wbase + u * USTAGE_B;
        v4f x[4];
        // with the following stages issued, at least NLD * (NST_U - 1)
        // loads follow this stage's; near the end the wait drains
        if (kn < nks) lds_read4_after<NLD * (NST_U - 1)>(b + o0, b + o1, b + o2, b + o3, x[0], x[1], x[2], x[3]);
        else lds_read4_after<0>(b + o0, b + o1, b + o2, b + o3, x[0], x[1], x[2], x[3]);
        unsigned y[16];
        if (WEIGHTED) {
          v2d wv[8];
          lds_read8(b + 4096 + 128 * h, wv);
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              y[4 * q + e] = fx_biased_w(x[q][e], wv[(4 * q + e) >> 1][e & 1], cw);
              ymin = min(ymin, (int)y[4 * q + e]);
              ymax = max(ymax, (int)y[4 * q + e]);
            }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              y[4 * q + e] = fx_biased_m(x[q][e], p2s);
              rmax = fmaxf(rmax, fabsf(x[q][e]));
            }
        }
        v4i P[4];
        make_planes(y, P);
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          acc[0][p] = mfma_i8(P[p], bn[u][0], acc[0][p]);
          acc[1][p] = mfma_i8(P[p], bn[u][1], acc[1][p]);
        }
      }
    }
  }
  // the row's measured bound replaces the one it was converted with (R does
  // not change until the next deflation, which raises it again)
  if (threadIdx.x < TILE) s_row[threadIdx.x] = s;
  if (WEIGHTED) {
    constexpr int BIAS = 0x00808080;
    s_rmax[wave][lane] = max(ymax - BIAS, BIAS - ymin);  // max |q| over this lane's words
  } else {
    s_rmax[wave][lane] = __float_as_int(rmax);            // non-negative floats order like ints
  }
  // every direct load has landed before the staging area is reused
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x < valid) {
    const int i = threadIdx.x;
    int r = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) r = max(r, max(s_rmax[q][i], s_rmax[q][i + 32]));
    rowb[i0 + i] = WEIGHTED ? __int2float_ru(r + 1) * __builtin_amdgcn_ldexpf(1.0f, -s_row[i]) : __int_as_float(r);
  }
  // out[t][M = row][N = component] -> Q[32 t + N][row], via a transposed
  // LDS tile for coalesced stores
  double* tq = (double*)smem;
  reduce_waves(smem, acc, nks <= FOLD_KMAX,
               [&](int t, int M, int N, long long v) { tq[(32 * t + N) * 32 + M] = ldexp((double)v, -s_row[M]); });
  __syncthreads();
  if (storeQ)
    for (int e = threadIdx.x; e < 2048; e += NT)
      if ((e & 31) < valid) Q[(int64_t)(e >> 5) * m_pad + i0 + (e & 31)] = tq[e];
  if (!Z) return;
  // The target rows Z = Q G_V^{-1} of this row group (Eq. (3) second half)
  // and their T_tau statistics, once the side path has stored G_V^{-1}.
  if (threadIdx.x == 0) await_flag(ready, flags);
  __syncthreads();
  double a[16];
  load_ginv(ginvV, a);
  const int li = lane & 15, lk = lane >> 4;
  v4d z[2] = {v4d{}, v4d{}};
  // A = G^{-1}[16 w + li][4 ks + lk], B = Q^T[4 ks + lk][li (+16)] (LDS)
#pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    z[0] = mfma_f64(a[ks], tq[(4 * ks + lk) * 32 + li], z[0]);
    z[1] = mfma_f64(a[ks], tq[(4 * ks + lk) * 32 + 16 + li], z[1]);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    double* row = Z + (int64_t)(16 * wave + lk + 4 * r) * m_pad + i0;
    if (li < valid) row[li] = z[0][r];
    if (16 + li < valid) row[16 + li] = z[1][r];
  }
  const int64_t iend = i0 + valid < m ? i0 + valid : m;
  tile_stats(z, wave, i0, iend, (int)gridDim.x - 2 * nside, rt, ps, pm, pi);
}

// U-step target rows Z = Q G_V^{-1} (Eq. (3) second half) and their T_tau
// statistics, after the contraction launch (G_V^{-1} from its side path).
// grid: m_pad / 32 row tiles (statistics per tile).  Rows past m hold
// Q = 0 (zero residual padding), so their targets are zero.
// WIDE: Z_q^T = sum_q' G^{-1}[q][q'] Q_q'^T, with ginvV the block row q
// (block q' at + 4096 q') and Q the contraction of quarter 0 (quarter q' at
// Q + q' 64 m_pad); Z, ps, pm, pi are the quarter's.
template <bool WIDE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_utarget(const double* __restrict__ Q, const double* __restrict__ ginvV,
                                                double* __restrict__ Z, int64_t m, int64_t m_pad, double* ps,
                                                double* pm, int* pi, int nq) {
  const int nrt = (int)(m_pad / TILE);
  const int lane = lane_id(), w = wave_id();
  const int li = lane & 15, lk = lane >> 4;
  double a[16];
  {
    const int rt = (int)blockIdx.x;
    const int64_t i0 = (int64_t)rt * TILE;
    v4d z[2] = {v4d{}, v4d{}};
    for (int q2 = 0; q2 < (WIDE ? nq : 1); ++q2) {
      load_ginv(ginvV + (WIDE ? (int64_t)q2 * 4096 : 0), a);
      // B = Q[4 ks + lk][i0 + li (+16)], straight from memory
      const double* Qq = Q + (WIDE ? (int64_t)q2 * BBP * m_pad : 0);
      double b0[16], b1[16];
#pragma unroll
      for (int ks = 0; ks < 16; ++ks) {
        const double* qr = Qq + (int64_t)(4 * ks + lk) * m_pad + i0 + li;
        b0[ks] = qr[0];
        b1[ks] = qr[16];
      }
#pragma unroll
      for (int ks = 0; ks < 16; ++ks) {
        z[0] = mfma_f64(a[ks], b0[ks], z[0]);
        z[1] = mfma_f64(a[ks], b1[ks], z[1]);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      double* row = Z + (int64_t)(16 * w + lk + 4 * r) * m_pad + i0;
      row[li] = z[0][r];
      row[16 + li] = z[1][r];
    }
    tile_stats(z, w, i0, m, nrt, rt, ps, pm, pi);
  }
}
// ---------------------------------------------------------------------------
// T_tau of target components from their per-tile statistics (Eq. (2)):
// theta = tau * (sum |x|) / L, strict ">", and when no entry exceeds theta
// (max |x| <= theta) only the largest |x| (smallest index) is kept.
// Workgroup (c, split) handles entries [i0, i1) of component c: every split
// reduces the same statistics with the same arithmetic, so all splits of a
// component apply the identical threshold.  The statistics loads are
// issued before the chunk's targets so that the reduction overlaps them.
// Writes the trits component-major (dst) and into the MFMA-ready layout
// mf, zero beyond L, and hands each (index, trit) to emit; with q it
// returns this chunk's sum_i t_i q_i (fp64, fixed reduction order).
// blockDim.x = NT.
// ---------------------------------------------------------------------------
constexpr int TERN_SP = 2;  // statistics tiles per thread loaded up front
constexpr int TERN_XS = 8;  // chunk entries per thread kept in registers

// Sum and max over the workgroup (DPP within each wave, then the waves in
// order); every thread receives both.  m: values >= -1.
__device__ __forceinline__ void block_sum_max(double& s, double& m, double* sh /* >= 8 */) {
  wave_sum63(s);
  wave_max63(m);
  const int w = wave_id();
  if (lane_id() == 63) {
    sh[w] = s;
    sh[4 + w] = m;
  }
  __syncthreads();
  s = ((sh[0] + sh[1]) + sh[2]) + sh[3];
  m = fmax(fmax(sh[4], sh[5]), fmax(sh[6], sh[7]));
}

template <typename Emit>
__device__ __forceinline__ double tern_chunk(const double* __restrict__ x, const double* __restrict__ q, int64_t L,
                                             int64_t i0, int64_t i1, int ntile, const double* __restrict__ ps,
                                             const double* __restrict__ pm, const int* __restrict__ pi, double tau,
                                             int8_t* __restrict__ dst, int8_t* __restrict__ mf, int c, Emit emit) {
  __shared__ double shd[8];
  __shared__ int shi[4];
  const int tid = threadIdx.x;
  double psr[TERN_SP], pmr[TERN_SP];
  // loads from clamped indices, masked afterwards: a load under a branch
  // would be waited for at the join before the next one is issued
#pragma unroll
  for (int k = 0; k < TERN_SP; ++k) {
    const int t = tid + k * NT, tc = t < ntile ? t : 0;
    psr[k] = ps[tc];
    pmr[k] = pm[tc];
  }
#pragma unroll
  for (int k = 0; k < TERN_SP; ++k) {
    const bool ok = tid + k * NT < ntile;
    psr[k] = ok ? psr[k] : 0.0;
    pmr[k] = ok ? pmr[k] : -1.0;
  }
  double xc[TERN_XS], qc[TERN_XS];
#pragma unroll
  for (int k = 0; k < TERN_XS; ++k) {
    const int64_t i = i0 + tid + (int64_t)k * NT;
    xc[k] = (i < i1 && i < L) ? x[i] : 0.0;
    qc[k] = (q && i < i1 && i < L) ? q[i] : 0.0;
  }
  double S = 0.0, M = -1.0;
#pragma unroll
  for (int k = 0; k < TERN_SP; ++k) {
    S += psr[k];
    M = fmax(M, pmr[k]);
  }
  for (int t = tid + TERN_SP * NT; t < ntile; t += NT) {
    S += ps[t];
    M = fmax(M, pm[t]);
  }
  block_sum_max(S, M, shd);
  const double theta = tau * (S / (double)L);
  const bool keep_max = !(M > theta);  // uniform over the workgroup
  int mi = 0;
  if (keep_max) {
    // the smallest index attaining the maximum: the smallest tile argmax
    // among the tiles whose maximum is M
    int best = 0x7fffffff;
    for (int t = tid; t < ntile; t += NT)
      if (pm[t] == M) best = min(best, pi[t]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) best = min(best, __shfl_xor(best, o, 64));
    if (lane_id() == 0) shi[wave_id()] = best;
    __syncthreads();
    mi = min(min(shi[0], shi[1]), min(shi[2], shi[3]));
  }
  auto decide = [&](int64_t i, double xv) -> int8_t {
    if (i >= L) return 0;
    const bool on = keep_max ? (i == mi) : (fabs(xv) > theta);
    return on ? ((xv > 0.0) ? 1 : ((xv < 0.0) ? -1 : 0)) : 0;
  };
  double g = 0.0;
#pragma unroll
  for (int k = 0; k < TERN_XS; ++k) {
    const int64_t i = i0 + tid + (int64_t)k * NT;
    if (i < i1) {
      const int8_t t = decide(i, xc[k]);
      g += (double)t * qc[k];
      dst[i] = t;
      mf[mf_offset(c, i)] = t;
      emit(i, t);
    }
  }
  for (int64_t i = i0 + tid + (int64_t)TERN_XS * NT; i < i1; i += NT) {
    const double xv = i < L ? x[i] : 0.0;
    const int8_t t = decide(i, xv);
    if (q && i < L) g += (double)t * q[i];
    dst[i] = t;
    mf[mf_offset(c, i)] = t;
    emit(i, t);
  }
  if (!q) return 0.0;
  double dummy = 0.0;
  __syncthreads();  // shd reuse
  block_sum_max(g, dummy, shd);
  return g;
}

// Split `sp` of `ns` of a length-L_pad component: [i0, i1), 32-aligned.
__device__ __forceinline__ void tern_range(int64_t L_pad, int sp, int ns, int64_t& i0, int64_t& i1) {
  const int64_t chunk = ((L_pad + ns - 1) / ns + TILE - 1) / TILE * TILE;
  i0 = (int64_t)sp * chunk;
  i1 = i0 + chunk < L_pad ? i0 + chunk : L_pad;
}

// V <- T_tau(Y[c, :]) for c < bb; zero components beyond bb.  Weighted
// (Wmf given): also the digit-scaled planes of V for the weighted Gram,
// Wmf[d * wstride + mf_offset(c, j)] = dig_d(j) v_jc.
// grid: BBP x ns (component c = blockIdx.x / ns, split blockIdx.x % ns).
__global__ __launch_bounds__(NT) void k_tern_v(const double* __restrict__ Y, int64_t n, int64_t n_pad, int bb, double tau,
                                               const double* __restrict__ ps, const double* __restrict__ pm,
                                               const int* __restrict__ pi, int ntile, int ns, int8_t* __restrict__ Vt,
                                               int8_t* __restrict__ Vmf, const int8_t* __restrict__ hdig,
                                               int8_t* __restrict__ Wmf, int64_t wstride, unsigned* ready) {
  const int c = blockIdx.x / ns, sp = blockIdx.x % ns;
  if (ready && blockIdx.x == 0 && threadIdx.x == 0) *ready = 0u;  // the V-step's G_U^{-1} flag
  int64_t i0, i1;
  tern_range(n_pad, sp, ns, i0, i1);
  int8_t* dst = Vt + (int64_t)c * n_pad;
  auto emit = [&](int64_t j, int8_t t) {
    if (Wmf) {  // uniform
      int8_t dg[WDIG];
#pragma unroll
      for (int d = 0; d < WDIG; ++d) dg[d] = hdig[(int64_t)d * n_pad + j];
      const int64_t o = mf_offset(c, j);
#pragma unroll
      for (int d = 0; d < WDIG; ++d) Wmf[(int64_t)d * wstride + o] = (int8_t)(t * dg[d]);
    }
  };
  if (c >= bb) {
    for (int64_t j = i0 + threadIdx.x; j < i1; j += NT) {
      dst[j] = 0;
      Vmf[mf_offset(c, j)] = 0;
      emit(j, (int8_t)0);
    }
    return;
  }
  const int64_t o = (int64_t)c * ntile;
  tern_chunk(Y + (int64_t)c * n_pad, nullptr, n, i0, i1, ntile, ps + o, pm + o, pi + o, tau, dst, Vmf, c, emit);
}

// U <- T_tau(Z[:, c]).  With Q (the last U-step of a block), also the
// split's share of g_c = sum_i U_ic Q_ic = diag(U^T R H V)_c for the joint
// scale solve (Eq. (4)): gpart[c * TERN_SPLIT_MAX + sp], unused slots 0.
// ps/pm/pi: statistics of ntile row groups (the U-step's groups, or 32-row
// tiles after the initial gather).  grid: BBP x ns as k_tern_v.
__global__ __launch_bounds__(NT) void k_tern_u(const double* __restrict__ Z, const double* __restrict__ Q, int64_t m,
                                               int64_t m_pad, int bb, double tau, const double* __restrict__ ps,
                                               const double* __restrict__ pm, const int* __restrict__ pi, int ntile,
                                               int ns, int8_t* __restrict__ Ut, int8_t* __restrict__ Umf,
                                               double* __restrict__ gpart, unsigned* ready) {
  const int c = blockIdx.x / ns, sp = blockIdx.x % ns;
  if (ready && blockIdx.x == 0 && threadIdx.x == 0) *ready = 0u;  // the U-step's G_V^{-1} flag
  int64_t i0, i1;
  tern_range(m_pad, sp, ns, i0, i1);
  int8_t* dst = Ut + (int64_t)c * m_pad;
  double g = 0.0;
  if (c >= bb) {
    for (int64_t i = i0 + threadIdx.x; i < i1; i += NT) {
      dst[i] = 0;
      Umf[mf_offset(c, i)] = 0;
    }
  } else {
    const int64_t o = (int64_t)c * ntile;
    const double* qrow = Q ? Q + (int64_t)c * m_pad : nullptr;
    g = tern_chunk(Z + (int64_t)c * m_pad, qrow, m, i0, i1, ntile, ps + o, pm + o, pi + o, tau, dst, Umf, c,
                   [](int64_t, int8_t) {});
  }
  if (Q && threadIdx.x == 0) {
    gpart[c * TERN_SPLIT_MAX + sp] = g;
    if (sp == 0)
      for (int k = ns; k < TERN_SPLIT_MAX; ++k) gpart[c * TERN_SPLIT_MAX + k] = 0.0;
  }
}

// Block initialisation (paper silent; reading: U[:, c] = T_tau(R[:, J_c])).
// Gathers the bb selected residual columns into X (component-major fp64,
// 64 x m_pad; zero for c >= bb) with the per-32-row-tile statistics of
// |x| that T_tau needs; k_tern_u then thresholds them like a U target.
// grid: m_pad/32 row tiles; thread (c = tid % 64, g = tid / 64) takes rows
// 8 g .. 8 g + 7 of the tile for component c.
__global__ __launch_bounds__(NT) void k_init_gather(const float* __restrict__ R, const int* __restrict__ J, int64_t m,
                                                    int64_t m_pad, int64_t n_pad, int bb, double* __restrict__ X,
                                                    double* __restrict__ ps, double* __restrict__ pm,
                                                    int* __restrict__ pi) {
  __shared__ double s_sum[4][BBP], s_max[4][BBP];
  __shared__ int s_idx[4][BBP];
  const int rt = blockIdx.x, ntile = (int)gridDim.x;
  const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int64_t i0 = (int64_t)rt * TILE + 8 * g;
  int jc = c < bb ? J[c] : 0;
  jc = jc < 0 ? 0 : (jc >= n_pad ? (int)(n_pad - 1) : jc);  // J comes from k_select; keep reads in bounds
  // all eight loads in flight together: clamped rows, masked afterwards
  float f[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int64_t i = i0 + r < m ? i0 + r : m - 1;
    f[r] = R[i * n_pad + jc];
  }
  double v[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) v[r] = (c < bb && i0 + r < m) ? (double)f[r] : 0.0;
  double s = 0.0, mv = -1.0;
  long long mi = i0;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    X[(int64_t)c * m_pad + i0 + r] = v[r];
    if (i0 + r < m) {
      s += fabs(v[r]);
      argmax_merge(mv, mi, fabs(v[r]), i0 + r);
    }
  }
  s_sum[g][c] = s;
  s_max[g][c] = mv;
  s_idx[g][c] = (int)mi;
  __syncthreads();
  if (g == 0) {
    double S = s_sum[0][c], M = s_max[0][c];
    long long I = s_idx[0][c];
#pragma unroll
    for (int q = 1; q < 4; ++q) {
      S += s_sum[q][c];
      argmax_merge(M, I, s_max[q][c], s_idx[q][c]);
    }
    ps[(int64_t)c * ntile + rt] = S;
    pm[(int64_t)c * ntile + rt] = M;
    pi[(int64_t)c * ntile + rt] = (int)I;
  }
}

// Xt (BBP x L int8, component-major) -> Xr (L x BBP, row-major) and, when
// Xb is given, the same trits as bf16 (0, +-1.0; L x BBP).
// grid: L/32 chunks.
__global__ __launch_bounds__(NT) void k_transpose8(const int8_t* __restrict__ Xt, int8_t* __restrict__ Xr,
                                                   int64_t L, unsigned short* __restrict__ Xb) {
  __shared__ int8_t tile[32][BBP + 4];
  const int64_t j0 = (int64_t)blockIdx.x * 32;
  for (int e = threadIdx.x; e < BBP * 32; e += NT) {
    const int c = e >> 5, jj = e & 31;
    tile[jj][c] = Xt[(int64_t)c * L + j0 + jj];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < BBP * 32; e += NT) {
    const int jj = e >> 6, c = e & 63;
    const int8_t t = tile[jj][c];
    Xr[(j0 + jj) * BBP + c] = t;
    if (Xb) Xb[(j0 + jj) * BBP + c] = t == 0 ? 0 : (t > 0 ? 0x3F80u : 0xBF80u);
  }
}

// ---------------------------------------------------------------------------
// Joint scale solve, Eq. (4): M = (U^T U) o (V^T H V) (+ delta I),
// d = M^{-1} g.  grid: one WG; U^T U is the accumulated Gram of the block's
// final U.
// ---------------------------------------------------------------------------
// Returns (want_gain, all threads) the objective the block removes from
// the residual, 2 d^T g - d^T M d, which equals d^T g + delta ||d||^2 when
// (M + delta I) d = g.
__device__ __forceinline__ double scale_solve(int* gacc, int bb, const double* __restrict__ gramV,
                                              const double* __restrict__ gvec, double* dvec, float* dF, float* Dout,
                                              double* Gs /* LDS 4096 */, double* colbuf /* LDS 1024 */,
                                              bool want_gain = false) {
  __shared__ double s_trb[16];
  const int t = threadIdx.x;
  // V^T H V issued with the U Gram's loads, all in one round
  double gv[4096 / NT];
#pragma unroll
  for (int j = 0; j < 4096 / NT; ++j) gv[j] = gramV[t + NT * j];
  take_gram(gacc, Gs);
#pragma unroll
  for (int j = 0; j < 4096 / NT; ++j) {
    const int e = t + NT * j, r = e >> 6, c = e & 63;
    Gs[e] = (r < bb && c < bb) ? Gs[e] * gv[j] : ((r == c) ? 1.0 : 0.0);
  }
  __syncthreads();
  const double tr = block_sum_d((t < bb) ? Gs[t * 64 + t] : 0.0, s_trb);
  if (tr == 0.0) {
    if (t < BBP) {
      dvec[t] = 0.0;
      dF[t] = 0.0f;
      if (Dout && t < bb) Dout[t] = 0.0f;
    }
    return 0.0;
  }
  const double delta = EXTERND_SCALE_GUARD_REL * tr / (double)bb;
  if (t < bb) Gs[t * 64 + t] += delta;
  __syncthreads();
  spd_inverse64(Gs, colbuf, (bb + 3) >> 2);
  // g_c: the per-split partial sums in split order
  __shared__ double s_g[BBP];
  if (t < BBP) {
    double g = 0.0;
#pragma unroll
    for (int k = 0; k < TERN_SPLIT_MAX; ++k) g += gvec[t * TERN_SPLIT_MAX + k];
    s_g[t] = t < bb ? g : 0.0;
  }
  __syncthreads();
  // d = M^{-1} g: row t / 4, the quarter t % 4 of its columns in registers,
  // the quarters added pairwise in a fixed order
  double dq = 0.0;
  {
    const int r = t >> 2, q = t & 3;
#pragma unroll
    for (int c = 0; c < 16; ++c) dq += Gs[r * 64 + 16 * q + c] * s_g[16 * q + c];
    dq += __shfl_xor(dq, 1, 64);
    dq += __shfl_xor(dq, 2, 64);
    if (q == 0) colbuf[r] = (r < bb) ? dq : 0.0;
  }
  __syncthreads();
  double gain = 0.0;
  if (t < BBP) {
    const double d = colbuf[t];
    dvec[t] = d;
    dF[t] = (float)d;
    if (Dout && t < bb) Dout[t] = (float)d;
    gain = d * s_g[t] + delta * d * d;
  }
  return want_gain ? block_sum_d(gain, s_trb) : 0.0;
}

__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_scale(int* gacc, int bb, const double* __restrict__ gramV,
                                              const double* __restrict__ gvec, double* dvec, float* dF, float* Dout) {
  __shared__ double Gs[4096];
  __shared__ double colbuf[1024];
  scale_solve(gacc, bb, gramV, gvec, dvec, dF, Dout, Gs, colbuf);
}

// ---------------------------------------------------------------------------
// Deflation R <- R - U diag(d) V^T on bf16 MFMA (Sec. 2.4), fused with the
// column energies ||R_:j||^2 (fp64 partials per row group) and max|R|.
// grid: (n_pad/32 column strips) x gd row groups; each wave takes 32-row
// tiles of its WG's group.  B = d-weighted V (3 exact bf16 parts of d),
// A = U (exact bf16).
// TRACK: also the largest |R| entry with its first row-major position, as
// one 64-bit key per slot (see argmax_key), for the single-entry option of
// Proposition 2.
// ---------------------------------------------------------------------------
// Key ordering the entries of R by |R| (fp32 bits, monotone for values
// >= 0), then by the smaller row-major index i * n + j.
__device__ __forceinline__ unsigned long long argmax_key(float absval, unsigned flat) {
  return ((unsigned long long)__float_as_uint(absval) << 32) | (unsigned long long)(0xFFFFFFFFu - flat);
}
// (value, index) pairs of a wave combined towards lane 0: larger value,
// then smaller index.
__device__ __forceinline__ void wave_argmax(float& v, unsigned& idx) {
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_down(v, o, 64);
    const unsigned oi = __shfl_down(idx, o, 64);
    if (ov > v || (ov == v && oi < idx)) {
      v = ov;
      idx = oi;
    }
  }
}

__device__ __forceinline__ unsigned short bf16_bits_trunc(float x) { return (unsigned short)(__float_as_uint(x) >> 16); }
__device__ __forceinline__ float bf16_to_f(unsigned short b) { return __uint_as_float((unsigned)b << 16); }
__device__ __forceinline__ short tern_bf16(int8_t t, unsigned short mag) {
  // t in {-1, 0, 1}: 0 -> +0, 1 -> mag, -1 -> mag with the sign bit flipped
  return (short)(t == 0 ? 0 : (t > 0 ? mag : (unsigned short)(mag ^ 0x8000u)));
}

template <bool TRACK>
__global__ __launch_bounds__(NT) void k_deflate(float* __restrict__ R, const v8s* __restrict__ Ub,
                                                const int8_t* __restrict__ Vr, const float* __restrict__ dF,
                                                double* __restrict__ colE_part, float* __restrict__ rowb,
                                                const int8_t* __restrict__ Ur, const double* __restrict__ hwmax,
                                                int64_t m_pad, int64_t n_pad, int gd,
                                                unsigned long long* __restrict__ argkey_next, int64_t n) {
  __shared__ double colsum[4][32];
  __shared__ float amax[4];
  __shared__ unsigned aidx[4];
  const int nct = (int)(n_pad / TILE);
  const int ct = blockIdx.x % nct, g = blockIdx.x / nct;
  const int nrt = (int)(m_pad / TILE);
  const int rt0 = (int)((long long)g * nrt / gd), rt1 = (int)((long long)(g + 1) * nrt / gd);
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  const int64_t col = (int64_t)ct * TILE + l32;
  // Row bounds of the U-step's fixed-point exponents: |R'_ij h~_j| <=
  // (|R_ij| + sum_c |U_ic d_c| |V_jc|) h~_j <= rowb_i + max h~ sum_c |U_ic| |d_c|,
  // inflated for the fp32 rounding of the update (< 2^-12 relative even for
  // the worst-case accumulation of the 3 x 64 MFMA terms).  The nct
  // workgroups of a row group share its rows, each row has one owner; the
  // first row of a thread is loaded here (clamped index, masked use) with
  // the B fragments, so the update adds no round of latency.
  const int64_t rg0 = (int64_t)rt0 * TILE, rg1 = (int64_t)rt1 * TILE;
  const int64_t rchunk = (rg1 - rg0 + nct - 1) / nct;
  const int64_t rb0 = rg0 + (int64_t)ct * rchunk, rb1 = rb0 + rchunk < rg1 ? rb0 + rchunk : rg1;
  const int64_t ib = rb0 + threadIdx.x;
  const int64_t ibc = ib < m_pad ? ib : m_pad - 1;
  int4 ur4[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) ur4[q] = ((const int4*)(Ur + ibc * BBP))[q];
  const float rbv = rowb[ibc];
  // B fragments: lane (h, col) holds components 16 ks + 8 h + e.
  v8s Bf[3][4];
  {
    const int8_t* vrow = Vr + col * BBP;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = 16 * ks + 8 * h + e;
        const float d = dF[c];
        const unsigned short hi = bf16_bits_trunc(d);
        const float r1 = d - bf16_to_f(hi);
        const unsigned short mi = bf16_bits_trunc(r1);
        const float r2 = r1 - bf16_to_f(mi);
        const unsigned short lo = bf16_bits_trunc(r2);
        const int8_t v = vrow[c];
        Bf[0][ks][e] = tern_bf16(v, hi);
        Bf[1][ks][e] = tern_bf16(v, mi);
        Bf[2][ks][e] = tern_bf16(v, lo);
      }
    }
  }
  {
    const double hmax = *hwmax;
    auto row_update = [&](int64_t i, const int4 (&u4)[4], float rb) {
      double sd = 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int8_t* ub = (const int8_t*)&u4[q];
#pragma unroll
        for (int e = 0; e < 16; ++e) sd += (ub[e] != 0 ? 1.0 : 0.0) * fabs((double)dF[16 * q + e]);
      }
      rowb[i] = __double2float_ru(((double)rb + hmax * sd) * (1.0 + 0x1p-12));
    };
    if (ib < rb1) row_update(ib, ur4, rbv);
    for (int64_t i = ib + NT; i < rb1; i += NT) {  // more than NT rows per workgroup: very tall matrices
      int4 u4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) u4[q] = ((const int4*)(Ur + i * BBP))[q];
      row_update(i, u4, rowb[i]);
    }
  }
  double csum = 0.0;
  // TRACK: this lane's first (smallest row) largest |R|; zero entries
  // (including the padding) never replace the start value
  float tmax = 0.0f;
  unsigned tidx = 0xFFFFFFFFu;
  // software pipeline: the residual values and U fragments of the wave's
  // next row tile (rt + 4, other rows) are loaded before this tile is
  // updated and stored
  float xn[16];
  v8s un[4];
  auto load_tile = [&](int rt) {
    const int64_t i0 = (int64_t)rt * TILE;
    // A fragments: row i0 + l32, components 16 ks + 8 h .. + 8 (bf16)
    const v8s* urow = Ub + (i0 + l32) * (BBP / 8);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) un[ks] = urow[2 * ks + h];
#pragma unroll
    for (int r = 0; r < 16; ++r) xn[r] = R[(i0 + 8 * (r >> 2) + 4 * h + (r & 3)) * n_pad + col];
  };
  if (rt0 + wave < rt1) load_tile(rt0 + wave);
  for (int rt = rt0 + wave; rt < rt1; rt += 4) {
    const int64_t i0 = (int64_t)rt * TILE;
    float x[16];
    v8s uu[4];
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = xn[r];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) uu[ks] = un[ks];
    if (rt + 4 < rt1) load_tile(rt + 4);
    v16f acc = {};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int p = 0; p < 3; ++p)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, uu[ks]), __builtin_bit_cast(v8bf, Bf[p][ks]),
                                                      acc, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 8 * (r >> 2) + 4 * h + (r & 3);
      const float v = x[r] - acc[r];
      R[(i0 + row) * n_pad + col] = v;
      csum += (double)v * (double)v;
      if (TRACK && fabsf(v) > tmax) {
        tmax = fabsf(v);
        tidx = (unsigned)((i0 + row) * n + col);
      }
    }
  }
  // combine the two half-waves (same column), then the 4 waves in order
  csum += __shfl_down(csum, 32, 64);
  if (TRACK) wave_argmax(tmax, tidx);
  if (h == 0) colsum[wave][l32] = csum;
  if (TRACK && lane == 0) {
    amax[wave] = tmax;
    aidx[wave] = tidx;
  }
  __syncthreads();
  if (threadIdx.x < 32) {
    const double s = ((colsum[0][threadIdx.x] + colsum[1][threadIdx.x]) + colsum[2][threadIdx.x]) + colsum[3][threadIdx.x];
    colE_part[(int64_t)g * n_pad + (int64_t)ct * TILE + threadIdx.x] = s;
  }
  if (threadIdx.x == 0) {
    if (TRACK) {
      unsigned long long key = 0ull;
      for (int q = 0; q < 4; ++q) {
        const unsigned long long kq = argmax_key(amax[q], aidx[q]);
        key = kq > key ? kq : key;
      }
      atomicMax(argkey_next, key);
    }
  }
}

// ---------------------------------------------------------------------------
// Staging: R <- A (zero padded), column energies (fp64 partials), max|A|,
// non-finite detection.  grid: (n_pad/32) x gd; thread (row lane, column).
// ---------------------------------------------------------------------------
template <bool TRACK>
__global__ __launch_bounds__(NT) void k_stage(const float* __restrict__ A, int64_t lda, int64_t m, int64_t n,
                                              float* __restrict__ R, double* __restrict__ colE_part,
                                              float* __restrict__ rowb_part, const double* __restrict__ hw,
                                              int* flags, int64_t m_pad, int64_t n_pad, int gd,
                                              unsigned long long* __restrict__ argkey0) {
  __shared__ double colsum[8][32];
  __shared__ float amax[NT / 64];
  __shared__ unsigned aidx[NT / 64];
  const int nct = (int)(n_pad / TILE);
  const int ct = blockIdx.x % nct, g = blockIdx.x / nct;
  const int64_t r0 = (int64_t)g * m_pad / gd, r1 = (int64_t)(g + 1) * m_pad / gd;
  const int cl = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int64_t j = (int64_t)ct * TILE + cl;
  double cs = 0.0;
  float tmax = 0.0f;            // TRACK: first (smallest row) largest |A| of this thread
  unsigned tidx = 0xFFFFFFFFu;
  int bad = 0;
  const double hwj = hw[j];
  for (int64_t i = r0 + rl; i < r1; i += 8) {
    float v = 0.0f;
    if (i < m && j < n) v = A[i * lda + j];
    if (!isfinite(v)) {
      bad = 1;
      v = 0.0f;
    }
    R[i * n_pad + j] = v;
    cs += (double)v * (double)v;
    if (TRACK && fabsf(v) > tmax) {
      tmax = fabsf(v);
      tidx = (unsigned)(i * n + j);
    }
    // this strip's share of the row bound max_j |R_ij| h~_j: the 32 lanes
    // of row i (a half-wave) reduced to lane cl = 0
    float b = weighted_abs_bound(v, hwj);
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) b = fmaxf(b, __shfl_xor(b, o, 32));
    if (cl == 0) rowb_part[(int64_t)ct * m_pad + i] = b;
  }
  colsum[rl][cl] = cs;
  if (TRACK) wave_argmax(tmax, tidx);
  if (TRACK && lane_id() == 0) {
    amax[wave_id()] = tmax;
    aidx[wave_id()] = tidx;
  }
  if (bad) flags[FLAG_NONFINITE] = 1;
  __syncthreads();
  if (threadIdx.x < 32) {
    double s = 0.0;
    for (int q = 0; q < 8; ++q) s += colsum[q][threadIdx.x];
    colE_part[(int64_t)g * n_pad + j] = s;
  }
  if (threadIdx.x == 0) {
    if (TRACK) {
      unsigned long long key = 0ull;
      for (int w = 0; w < NT / 64; ++w) {
        const unsigned long long kw = argmax_key(amax[w], aidx[w]);
        key = kw > key ? kw : key;
      }
      atomicMax(argkey0, key);
    }
  }
}

// Row bounds after staging: rowb_i = max over the column strips' partials.
// grid: ceil(m_pad / NT).
__global__ __launch_bounds__(NT) void k_rowb_init(const float* __restrict__ rowb_part, int nct, int64_t m_pad,
                                                  float* __restrict__ rowb) {
  const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (i >= m_pad) return;
  float b = 0.0f;
  for (int c = 0; c < nct; ++c) b = fmaxf(b, rowb_part[(int64_t)c * m_pad + i]);
  rowb[i] = b;
}

// R (padded) -> A (m x n, row-major)
__global__ __launch_bounds__(NT) void k_unstage(const float* __restrict__ R, float* __restrict__ A, int64_t m,
                                                int64_t n, int64_t n_pad) {
  const int64_t total = m * n;
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < total; e += (int64_t)gridDim.x * NT) {
    const int64_t i = e / n, j = e % n;
    A[e] = R[i * n_pad + j];
  }
}

// Bits of the weighted Grams' integer weights: w = min(WSHIFT_MAX,
// 61 - ceil(log2 n_pad)), so that sum_j H_j < n_pad 2^w <= 2^61.
__device__ __forceinline__ int weight_bits(int64_t n_pad) {
  int c = 0;
  while (((int64_t)1 << c) < n_pad) ++c;
  return 61 - c < WSHIFT_MAX ? 61 - c : WSHIFT_MAX;
}
// Digit planes of the weight r = h~_j / max h~ in [0, 1]:
// H_j = min(rint(r 2^wb), 2^wb - 1), digit d of H_j in hdig[d * n_pad + j].
__device__ __forceinline__ void put_weight_digits(int8_t* hdig, int64_t n_pad, int64_t j, double r, int wb) {
  const double q = rint(ldexp(r, wb));
  const long long top = ((long long)1 << wb) - 1;
  const long long H = q < (double)top ? (long long)q : top;
#pragma unroll
  for (int d = 0; d < WDIG; ++d)
    hdig[(int64_t)d * n_pad + j] = (int8_t)((H >> (WDIG_BITS * d)) & ((1 << WDIG_BITS) - 1));
}

// Weights and bookkeeping (1 WG): h~ = h / max(h) + lam in fp64 (Sec. 2.5;
// ones when no weights), zero padding; clear counters, flags and the
// per-block arrays.
__global__ __launch_bounds__(NT) void k_prep(const float* __restrict__ h, int64_t n, int64_t n_pad,
                                             double* __restrict__ hw, double* __restrict__ hwmax,
                                             double* fro2_hist, double* fro2w_hist, int nblk_cap,
                                             unsigned* counters, int* flags, int* gacc, double lam,
                                             unsigned long long* argkey, int* gaccW, long long* gacc64,
                                             int8_t* __restrict__ hdig, unsigned* vtcnt) {
  __shared__ float smax[NT / 64];
  __shared__ int sbad[NT / 64];
  for (int64_t e = threadIdx.x; e < n_pad / TILE; e += NT) vtcnt[e] = 0u;
  for (int e = threadIdx.x; e < nblk_cap; e += NT) {
    fro2_hist[e] = 0.0;
    fro2w_hist[e] = 0.0;
    argkey[e] = 0ull;
  }
  if (threadIdx.x < CNT_COUNT) counters[threadIdx.x] = 0u;
  for (int e = threadIdx.x; e < 2 * 4096; e += NT) gacc[e] = 0;
  for (int e = threadIdx.x; e < 2 * NPAIR_MAX * 4096; e += NT) gaccW[e] = 0;
  for (int e = threadIdx.x; e < 4096; e += NT) gacc64[e] = 0;
  if (threadIdx.x < FLAG_COUNT) flags[threadIdx.x] = 0;
  if (!h) {
    for (int64_t j = threadIdx.x; j < n_pad; j += NT) hw[j] = (j < n) ? 1.0 : 0.0;
    if (threadIdx.x == 0) {
      hwmax[0] = 1.0;
      hwmax[1] = ldexp(1.0, -weight_bits(n_pad));
    }
    return;
  }
  float mx = 0.0f;
  int bad = 0;
  for (int64_t j = threadIdx.x; j < n; j += NT) {
    const float v = h[j];
    if (!isfinite(v) || v < 0.0f) bad = 1;
    else mx = fmaxf(mx, v);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_down(mx, o, 64));
    bad |= __shfl_down(bad, o, 64);
  }
  if (lane_id() == 0) {
    smax[wave_id()] = mx;
    sbad[wave_id()] = bad;
  }
  __syncthreads();
  float gmx = 0.0f;
  int gbad = 0;
  for (int w = 0; w < NT / 64; ++w) {
    gmx = fmaxf(gmx, smax[w]);
    gbad |= sbad[w];
  }
  if (!(gmx > 0.0f)) gbad = 1;
  if (gbad) {
    if (threadIdx.x == 0) {
      flags[FLAG_BADWEIGHT] = 1;
      *hwmax = 1.0;
    }
    const int wb = weight_bits(n_pad);
    for (int64_t j = threadIdx.x; j < n_pad; j += NT) {
      hw[j] = (j < n) ? 1.0 : 0.0;
      put_weight_digits(hdig, n_pad, j, hw[j], wb);
    }
    if (threadIdx.x == 0) hwmax[1] = ldexp(1.0, -wb);
    return;
  }
  const double dm = (double)gmx;
  // the largest weight is exactly max(h) / max(h) + lam
  const double hmax = 1.0 + lam;
  const int wb = weight_bits(n_pad);
  for (int64_t j = threadIdx.x; j < n_pad; j += NT) {
    const double v = (j < n) ? (double)h[j] / dm + lam : 0.0;
    hw[j] = v;
    put_weight_digits(hdig, n_pad, j, v / hmax, wb);
  }
  if (threadIdx.x == 0) {
    hwmax[0] = hmax;
    hwmax[1] = ldexp(hmax, -wb);
  }
}

// ---------------------------------------------------------------------------
// Column energies -> ||R||^2 history and the top-bb selection (1 WG,
// NT_SELECT threads).  key_j = h~_j ||R_:j||^2 (fp64, >= 0, so its bit
// pattern orders like the value); exact radix select of the bb-th largest
// key, ties broken towards the smaller column index.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void reduce_colE(const double* __restrict__ colE_part, int gd, int64_t n, int64_t n_pad,
                            const double* __restrict__ hw, double* colE, double* out_fro2, double* out_fro2w,
                            double* shd, int* cshift) {
  double s = 0.0, sw = 0.0;
  for (int64_t j = threadIdx.x; j < n_pad; j += blockDim.x) {
    double c = 0.0;
#pragma unroll 8
    for (int g = 0; g < gd; ++g) c += colE_part[(int64_t)g * n_pad + j];
    if (j >= n) c = 0.0;
    if (colE && j < n) colE[j] = c;
    cshift[j] = col_shift(c);
    s += c;
    sw += hw[j] * c;
  }
  s = block_sum_d(s, shd);
  sw = block_sum_d(sw, shd);
  if (threadIdx.x == 0) {
    *out_fro2 = s;
    if (out_fro2w) *out_fro2w = sw;
  }
}

constexpr int SELECT_CACHE = 8;  // keys per thread kept in registers (n <= SELECT_CACHE * NT_SELECT without memory passes)

// Column energies of the NQ columns j = tid + q st of this thread: the gd
// row-group partials summed in row-group order, GU row groups a round with
// all their loads issued together (clamped indices, masked afterwards).
template <int NQ>
__device__ __forceinline__ void select_energies(const double* __restrict__ colE_part, int gd, int64_t n_pad,
                                                int64_t st, double (&e)[SELECT_CACHE]) {
  constexpr int GU = NQ >= 16 ? 1 : 16 / NQ;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q) e[q] = 0.0;
  for (int g0 = 0; g0 < gd; g0 += GU) {
    double v[GU][NQ];
#pragma unroll
    for (int u = 0; u < GU; ++u) {
      const int g = g0 + u < gd ? g0 + u : gd - 1;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int64_t j = tid + q * st;
        v[u][q] = colE_part[(int64_t)g * n_pad + (j < n_pad ? j : 0)];
      }
    }
#pragma unroll
    for (int u = 0; u < GU; ++u)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        if (g0 + u < gd) e[q] += v[u][q];
  }
}

__global__ __launch_bounds__(NT_SELECT) void k_select(const double* __restrict__ colE_part, int gd, int64_t n,
                                                      int64_t n_pad, const double* __restrict__ hw,
                                                      double* keys /* n_pad scratch */, double* fro2_out,
                                                      double* fro2w_out, int bb, int* __restrict__ J,
                                                      int* __restrict__ cshift) {
  __shared__ double wred[4][NT_SELECT / 64];
  __shared__ unsigned hist[256];
  __shared__ unsigned long long s_prefix;
  __shared__ int s_need, s_exact, s_hi;
  __shared__ int s_cnt;
  __shared__ unsigned long long cand_key[BMAX];
  __shared__ int cand_idx[BMAX];
  __shared__ int s_scan[NT_SELECT / 64];
  __shared__ int s_rank[BMAX];
  const int tid = threadIdx.x;
  const int64_t st = blockDim.x;
  const int nw = (int)(blockDim.x >> 6);
  if (tid < BMAX) {
    cand_key[tid] = 0ull;
    cand_idx[tid] = 0;
  }
  // Column energies ||R_:j||^2 of this thread's columns; the keys
  // h~_j ||R_:j||^2 stay in registers, columns beyond SELECT_CACHE st (very
  // wide matrices only) go through `keys`.  Every global store of the
  // kernel (exponents, norms, the selection) is issued at its end, so that
  // no barrier waits for one.
  double hq[SELECT_CACHE];
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q) {
    const int64_t j = tid + q * st;
    hq[q] = hw[j < n_pad ? j : 0];
  }
  double e[SELECT_CACHE];
  const int64_t nq = (n_pad + st - 1) / st;
  if (nq <= 1) select_energies<1>(colE_part, gd, n_pad, st, e);
  else if (nq <= 2) select_energies<2>(colE_part, gd, n_pad, st, e);
  else if (nq <= 3) select_energies<3>(colE_part, gd, n_pad, st, e);
  else if (nq <= 4) select_energies<4>(colE_part, gd, n_pad, st, e);
  else select_energies<SELECT_CACHE>(colE_part, gd, n_pad, st, e);
  double s = 0.0, sw = 0.0;
  unsigned long long kc[SELECT_CACHE];
  int csh[SELECT_CACHE];
  double kmax = 0.0, kmin = INFINITY;
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q) {
    const int64_t j = tid + q * st;
    const double c = j < n ? e[q] : 0.0;
    csh[q] = col_shift(c);
    s += c;
    sw += hq[q] * c;
    const double key = hq[q] * c;
    kc[q] = j < n ? (unsigned long long)__double_as_longlong(key) : 0ull;
    if (j < n) {
      kmax = fmax(kmax, key);
      kmin = fmin(kmin, key);
    }
  }
  for (int64_t j = tid + SELECT_CACHE * st; j < n_pad; j += st) {
    double c = 0.0;
    for (int g = 0; g < gd; ++g) c += colE_part[(int64_t)g * n_pad + j];
    if (j >= n) c = 0.0;
    cshift[j] = col_shift(c);
    s += c;
    sw += hw[j] * c;
    if (j < n) {
      const double key = hw[j] * c;
      keys[j] = key;
      kmax = fmax(kmax, key);
      kmin = fmin(kmin, key);
    }
  }
  // one block reduction for the two norms and the key range (DPP within
  // each wave, then the waves in order)
  kmin = -kmin;
  wave_sum63(s);
  wave_sum63(sw);
  wave_max63(kmax);
  wave_max63(kmin);
  if (lane_id() == 63) {
    wred[0][wave_id()] = s;
    wred[1][wave_id()] = sw;
    wred[2][wave_id()] = kmax;
    wred[3][wave_id()] = kmin;
  }
  __syncthreads();
  double f2 = 0.0, f2w = 0.0;
  if (tid == 0) {
    double a = 0.0, b = -INFINITY;
    for (int w = 0; w < nw; ++w) {
      f2 += wred[0][w];
      f2w += wred[1][w];
      a = fmax(a, wred[2][w]);
      b = fmax(b, wred[3][w]);
    }
    // the radix passes start below the leading bits that every key shares
    // (non-negative doubles order like their bit patterns)
    const unsigned long long ka = (unsigned long long)__double_as_longlong(a);
    const unsigned long long kb = (unsigned long long)__double_as_longlong(-b);
    const unsigned long long d = ka ^ kb;
    const int hi = d ? 64 - __clzll((long long)d) : 0;
    s_hi = hi;
    s_prefix = hi < 64 ? (ka & (~0ull << hi)) : 0ull;
    s_need = bb;
    s_exact = 0;
  }
  __syncthreads();
  // Radix select of the bb-th largest key over 8-bit windows [lo, hi) from
  // the first bit where keys differ down to bit 0.  The passes stop early
  // once the window bin holding the bb-th largest key holds exactly the
  // keys still needed: then the selection is every key >= that bin's lower
  // bound.  (All keys equal: hi = 0, no pass, T = that key.)
  for (int hi = s_hi; hi > 0;) {
    const int lo = hi > 8 ? hi - 8 : 0;
    const unsigned dmask = (1u << (hi - lo)) - 1u;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    const unsigned long long prefix = s_prefix;
    const unsigned long long hmask = hi < 64 ? (~0ull << hi) : 0ull;
#pragma unroll
    for (int q = 0; q < SELECT_CACHE; ++q) {
      const int64_t j = tid + q * st;
      if (j < n && (kc[q] & hmask) == prefix) atomicAdd(&hist[(unsigned)(kc[q] >> lo) & dmask], 1u);
    }
    for (int64_t j = tid + SELECT_CACHE * st; j < n; j += st) {
      const unsigned long long kb = (unsigned long long)__double_as_longlong(keys[j]);
      if ((kb & hmask) == prefix) atomicAdd(&hist[(unsigned)(kb >> lo) & dmask], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // wave 0: lane l holds digits 255-4l .. 252-4l (descending); the
      // first lane whose inclusive count reaches `need` holds the digit.
      const int lane = tid;
      const int need = s_need;
      int c[4], tot = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = (int)hist[255 - 4 * lane - q];
        tot += c[q];
      }
      // inclusive scan over the wave on DPP: within rows, then across rows
      int incl = tot;
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_SHR1, 0xF, 0xF, false);
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_SHR2, 0xF, 0xF, false);
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_SHR4, 0xF, 0xF, false);
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_SHR8, 0xF, 0xF, false);
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_BCAST15, 0xA, 0xF, false);
      incl += __builtin_amdgcn_update_dpp(0, incl, DPP_ROW_BCAST31, 0xC, 0xF, false);
      const unsigned long long hit = __ballot(incl >= need);
      const int first = hit ? (__ffsll((long long)hit) - 1) : 63;
      if (lane == first) {
        int run = incl - tot, d = 0, nn = need;
        bool found = false;
        int cd = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (!found && run + c[q] >= need) {
            d = 255 - 4 * lane - q;
            nn = need - run;
            cd = c[q];
            found = true;
          }
          if (!found) run += c[q];
        }
        if (!found) {
          d = 0;
          nn = need - run;
        }
        s_need = nn;
        s_prefix = prefix | ((unsigned long long)d << lo);
        s_exact = found && cd == nn;
      }
    }
    __syncthreads();
    if (s_exact) break;
    hi = lo;
  }
  // T = s_prefix: either the exact key of the bb-th largest (keys > T all
  // selected, then the s_need smallest indices with key == T), or, after an
  // early stop, the lower bound of a bin whose keys are all selected (keys
  // >= T, nothing left to tie-break).
  const bool ge = s_exact != 0;
  const unsigned long long T = s_prefix;
  const int need_eq = ge ? 0 : s_need;
  auto above = [&](unsigned long long kb) { return ge ? kb >= T : kb > T; };
  if (tid == 0) s_cnt = 0;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q) {
    const int64_t j = tid + q * st;
    if (j < n && above(kc[q])) {
      const int slot = atomicAdd(&s_cnt, 1);
      if (slot < BMAX) {
        cand_key[slot] = kc[q];
        cand_idx[slot] = (int)j;
      }
    }
  }
  for (int64_t j = tid + SELECT_CACHE * st; j < n; j += st) {
    const unsigned long long kb = (unsigned long long)__double_as_longlong(keys[j]);
    if (above(kb)) {
      const int slot = atomicAdd(&s_cnt, 1);
      if (slot < BMAX) {
        cand_key[slot] = kb;
        cand_idx[slot] = (int)j;
      }
    }
  }
  __syncthreads();
  // keys equal to T, in index order: block-wide exclusive scans over
  // consecutive rounds of blockDim indices (the round count and the stop
  // condition are uniform across the block)
  int carry = 0;
  const int base = s_cnt;
  const int rounds = (int)((n + st - 1) / st);
  bool done = need_eq == 0;
  auto scan_round = [&](int64_t j, unsigned long long kb) {
    const int f = (j < n && kb == T) ? 1 : 0;
    int v = f;
    const int lane = lane_id();
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(v, o, 64);
      if (lane >= o) v += u;
    }
    if (lane == 63) s_scan[wave_id()] = v;
    __syncthreads();
    int woff = 0, tot = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      if (w < wave_id()) woff += s_scan[w];
      tot += s_scan[w];
    }
    const int pos = carry + woff + v - f;
    if (f && pos < need_eq && base + pos < BMAX) {
      cand_key[base + pos] = T;
      cand_idx[base + pos] = (int)j;
    }
    carry += tot;
    __syncthreads();
    done = carry >= need_eq;
  };
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q)
    if (!done && q < rounds) scan_round(tid + q * st, kc[q]);
  for (int q = SELECT_CACHE; !done && q < rounds; ++q) {
    const int64_t j = tid + q * st;
    scan_round(j, j < n ? (unsigned long long)__double_as_longlong(keys[j]) : 0ull);
  }
  __syncthreads();
  // order the bb winners by (key desc, index asc): TPW threads per winner
  // each compare it with every TPW-th other, summed over the TPW lanes
  {
    constexpr int TPW = NT_SELECT / BMAX;
    static_assert(TPW == 4, "four threads per winner");
    const int a = tid / TPW, b = tid % TPW;
    int r = 0;
    if (a < bb) {
      const unsigned long long k0 = cand_key[a];
      const int i0 = cand_idx[a];
#pragma unroll 8
      for (int q = b; q < bb; q += TPW) {
        const unsigned long long k1 = cand_key[q];
        const int i1 = cand_idx[q];
        r += (k1 > k0) || (k1 == k0 && i1 < i0);
      }
    }
    r += __shfl_xor(r, 1, 64);
    r += __shfl_xor(r, 2, 64);
    if (b == 0 && a < bb) s_rank[a] = r;
  }
  __syncthreads();
  if (tid < bb) J[s_rank[tid]] = cand_idx[tid];
  if (tid == 0) {
    *fro2_out = f2;
    *fro2w_out = f2w;
  }
#pragma unroll
  for (int q = 0; q < SELECT_CACHE; ++q) {
    const int64_t j = tid + q * st;
    if (j < n_pad) cshift[j] = csh[q];
  }
}

// ||R||^2 after the last block (1 WG).
__global__ __launch_bounds__(NT_SELECT) void k_finish(const double* __restrict__ colE_part, int gd, int64_t n,
                                                      int64_t n_pad, const double* __restrict__ hw,
                                                      double* colE_out, double* fro2_out, double* fro2w_out,
                                                      int* __restrict__ cshift) {
  __shared__ double shd[16];
  reduce_colE(colE_part, gd, n, n_pad, hw, colE_out, fro2_out, fro2w_out, shd, cshift);
}

// ---------------------------------------------------------------------------
// Emit a block into the packed outputs (2-bit trits: 00 = 0, 01 = +1,
// 11 = -1; element j of a row at byte j>>2, bits 2(j&3)).
// ---------------------------------------------------------------------------
__device__ __forceinline__ unsigned trit_code(int8_t t) { return t == 0 ? 0u : (t > 0 ? 1u : 3u); }

// ---------------------------------------------------------------------------
// End of a block, one launch: the joint scale solve (Eq. (4)) in WG 0,
// writing d to the output D; then 32-index tiles of U and V: their
// row-major copies for the deflation (U also as bf16) and the block's trits
// packed into the rows of B and C (Eq. (1); 2-bit codes, element j at byte
// j>>2, bits 2(j&3); B bytes shared with neighbouring blocks are
// read-modified-written, padding bits beyond k cleared).
// grid: 1 + m_pad/32 (U tiles) + n_pad/32 (V tiles).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int8_t trit_decode(unsigned byte, int64_t pos) {
  const unsigned code = (byte >> (2 * (int)(pos & 3))) & 3u;
  return (int8_t)(code == 1u ? 1 : (code == 3u ? -1 : 0));
}

// decision: null during extraction.  In a refinement revisit it is the
// device word set by k_revisit_decide: WG 0 then does nothing (the scales
// are settled), and when the old block is kept (decision 0) the tiles
// rebuild the deflation operands from the packed B and C, which stay as
// they are.
// sg: null unless the single-entry option is on; then the scales were
// settled by k_safeguard, and when it fired (sg[0]) the block written out
// is u = e_row, v = (+-1) e_col in component 0 and zero components after.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_block_out(int* gacc, int bb, const double* __restrict__ gramV,
                                                  const double* __restrict__ gvec, double* dvec, float* dF,
                                                  float* Dout, const int8_t* __restrict__ Ut, int8_t* __restrict__ Ur,
                                                  unsigned short* __restrict__ Ub, int64_t m, int64_t m_pad,
                                                  int64_t c0, int64_t k, uint8_t* __restrict__ Bp,
                                                  const int8_t* __restrict__ Vt, int8_t* __restrict__ Vr, int64_t n,
                                                  int64_t n_pad, uint8_t* __restrict__ Cp,
                                                  const unsigned* __restrict__ decision,
                                                  const unsigned* __restrict__ sg, int solve) {
  __shared__ double Gs[4096];
  __shared__ double colbuf[1024];
  if (blockIdx.x == 0) {
    if (solve && !decision && !sg) scale_solve(gacc, bb, gramV, gvec, dvec, dF, Dout, Gs, colbuf);
    return;
  }
  int8_t (*tile)[BBP + 4] = (int8_t (*)[BBP + 4])Gs;  // 32 x 68 bytes
  const int nut = (int)(m_pad / TILE);
  const bool isU = (int)blockIdx.x <= nut;
  const int64_t L = isU ? m_pad : n_pad;
  const int8_t* Xt = isU ? Ut : Vt;
  const int64_t j0 = (int64_t)(isU ? blockIdx.x - 1 : blockIdx.x - 1 - nut) * 32;
  const bool keep_old = decision && *decision == 0u;
  const bool single = sg && sg[0] != 0u;
  if (single) {
    const int64_t at = isU ? (int64_t)sg[1] : (int64_t)sg[2];
    const int8_t one = (!isU && sg[3]) ? (int8_t)-1 : (int8_t)1;
    for (int e = threadIdx.x; e < BBP * 32; e += NT) {
      const int c = e >> 5, jj = e & 31;
      tile[jj][c] = (c == 0 && j0 + jj == at) ? one : (int8_t)0;
    }
  } else if (keep_old) {
    const int64_t pitchB = (k + 3) >> 2, pitchC = (n + 3) >> 2;
    for (int e = threadIdx.x; e < BBP * 32; e += NT) {
      const int c = e >> 5, jj = e & 31;
      const int64_t j = j0 + jj;
      int8_t t = 0;
      if (c < bb) {
        if (isU) {
          if (j < m) t = trit_decode(Bp[j * pitchB + ((c0 + c) >> 2)], c0 + c);
        } else if (j < n) {
          t = trit_decode(Cp[(c0 + c) * pitchC + (j >> 2)], j);
        }
      }
      tile[jj][c] = t;
    }
  } else {
    for (int e = threadIdx.x; e < BBP * 32; e += NT) {
      const int c = e >> 5, jj = e & 31;
      tile[jj][c] = Xt[(int64_t)c * L + j0 + jj];
    }
  }
  __syncthreads();
  int8_t* Xr = isU ? Ur : Vr;
  for (int e = threadIdx.x; e < BBP * 32; e += NT) {
    const int jj = e >> 6, c = e & 63;
    const int8_t t = tile[jj][c];
    Xr[(j0 + jj) * BBP + c] = t;
    if (isU) Ub[(j0 + jj) * BBP + c] = t == 0 ? 0 : (t > 0 ? 0x3F80u : 0xBF80u);
  }
  if (keep_old) return;
  if (isU) {
    // rows j0 .. j0+31 of B, byte range covering columns [c0, c0 + bb)
    const int64_t pitch = (k + 3) >> 2;
    const int64_t q0 = c0 >> 2, q1 = (c0 + bb - 1) >> 2;
    const int nq = (int)(q1 - q0 + 1);
    for (int e = threadIdx.x; e < 32 * nq; e += NT) {
      const int jj = e / nq;
      const int64_t i = j0 + jj, q = q0 + e % nq;
      if (i >= m) continue;
      uint8_t* dst = Bp + i * pitch + q;
      unsigned byte = *dst;
      for (int s = 0; s < 4; ++s) {
        const int64_t p = 4 * q + s;
        if (p >= k) byte &= ~(3u << (2 * s));
        else if (p >= c0 && p < c0 + bb) {
          byte &= ~(3u << (2 * s));
          byte |= trit_code(tile[jj][p - c0]) << (2 * s);
        }
      }
      *dst = (uint8_t)byte;
    }
  } else {
    // columns j0 .. j0+31 of C rows c0 .. c0+bb-1: 8 whole bytes per row
    const int64_t pitch = (n + 3) >> 2;
    for (int e = threadIdx.x; e < bb * 8; e += NT) {
      const int c = e >> 3, qq = e & 7;
      const int64_t q = (j0 >> 2) + qq;
      if (q >= pitch) continue;
      unsigned byte = 0;
      for (int s = 0; s < 4; ++s) {
        const int64_t j = 4 * q + s;
        if (j < n) byte |= trit_code(tile[4 * qq + s][c]) << (2 * s);
      }
      Cp[(c0 + c) * pitch + q] = (uint8_t)byte;
    }
  }
}

// ---------------------------------------------------------------------------
// Refinement sweeps (Sec. 2.4): a revisit adds the block back to R, fits it
// again from its current U and deflates the better of the old and the new
// block.
// ---------------------------------------------------------------------------
// Start of a revisit: the block's factors decoded from the packed B and C
// into the workspace layouts (U as the warm start and, with V, as the
// add-back operands), add-back scales -D, and the residual-bound slots the
// revisit's two deflations write cleared.
// grid: 1 + m_pad/32 (U tiles) + n_pad/32 (V tiles).
__global__ __launch_bounds__(NT) void k_revisit_load(const uint8_t* __restrict__ Bp, const uint8_t* __restrict__ Cp,
                                                     const float* __restrict__ D, int64_t c0, int bb, int64_t k,
                                                     int64_t m, int64_t m_pad, int64_t n, int64_t n_pad,
                                                     int8_t* __restrict__ Ut, int8_t* __restrict__ Ur,
                                                     unsigned short* __restrict__ Ub, int8_t* __restrict__ Umf,
                                                     int8_t* __restrict__ Vt, int8_t* __restrict__ Vr,
                                                     int8_t* __restrict__ Vmf, float* __restrict__ dF) {
  if (blockIdx.x == 0) {
    if (threadIdx.x < BBP) dF[threadIdx.x] = (int)threadIdx.x < bb ? -D[c0 + threadIdx.x] : 0.0f;
    return;
  }
  const int nut = (int)(m_pad / TILE);
  const bool isU = (int)blockIdx.x <= nut;
  const int64_t j0 = (int64_t)(isU ? blockIdx.x - 1 : blockIdx.x - 1 - nut) * 32;
  const int64_t pitchB = (k + 3) >> 2, pitchC = (n + 3) >> 2;
  for (int e = threadIdx.x; e < 32 * BBP; e += NT) {
    const int jj = e >> 6, c = e & 63;
    const int64_t j = j0 + jj;
    int8_t t = 0;
    if (c < bb) {
      if (isU) {
        if (j < m) t = trit_decode(Bp[j * pitchB + ((c0 + c) >> 2)], c0 + c);
      } else if (j < n) {
        t = trit_decode(Cp[(c0 + c) * pitchC + (j >> 2)], j);
      }
    }
    if (isU) {
      Ut[(int64_t)c * m_pad + j] = t;
      Ur[j * BBP + c] = t;
      Ub[j * BBP + c] = t == 0 ? 0 : (t > 0 ? 0x3F80u : 0xBF80u);
      Umf[mf_offset(c, j)] = t;
    } else {
      Vt[(int64_t)c * n_pad + j] = t;
      Vr[j * BBP + c] = t;
      Vmf[mf_offset(c, j)] = t;
    }
  }
}

// After the fit: the joint scale solve of the new block (Eq. (4)) and the
// choice between it and the old block.  The new block is kept when the
// objective it removes from R' exceeds what the old block removes,
// fro2_added - fro2_prev (both from the fused column energies: R before the
// add-back and R' after it).  Kept: D <- fp32(d) and the new scales go to
// the deflation.  Otherwise the deflation takes the old scales D and the
// outputs stay.  *decision = 1 / 0; *accepted counts the kept new blocks.
// grid: one WG.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_revisit_decide(int* gacc, int bb, const double* __restrict__ gramV,
                                                       const double* __restrict__ gvec, double* dvec, float* dF,
                                                       float* D, const double* fro2_prev,
                                                       const double* fro2_added, unsigned* decision,
                                                       unsigned* accepted) {
  __shared__ double Gs[4096];
  __shared__ double colbuf[1024];
  const double gain = scale_solve(gacc, bb, gramV, gvec, dvec, dF, nullptr, Gs, colbuf, true);
  const double old_gain = *fro2_added - *fro2_prev;
  const bool take_new = gain > old_gain;
  const int t = threadIdx.x;
  // thread t wrote dF[t] in the solve
  if (t < BBP) {
    if (take_new) {
      if (t < bb) D[t] = dF[t];
    } else {
      dF[t] = t < bb ? D[t] : 0.0f;
    }
  }
  if (t == 0) {
    *decision = take_new ? 1u : 0u;
    if (take_new) *accepted += 1u;
  }
}

// ---------------------------------------------------------------------------
// Single-entry option of Proposition 2 for a block (plain objective): after
// the Eq. (4) solve, the objective the block removes, 2 d^T g - d^T M d
// (= d^T g + delta ||d||^2 for the guarded solve), is compared with the
// largest squared residual entry R_ij^2 (first in row-major order on
// ties).  When the entry is strictly larger the block becomes the single
// component u = e_i, v = sign(R_ij) e_j, d = |R_ij| followed by zero
// components; k_block_out writes it out and the deflation removes R_ij
// exactly.  sg receives (fired, i, j, R_ij < 0); *fired counts the blocks.
// grid: one WG.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_safeguard(int* gacc, int bb, const double* __restrict__ gramV,
                                                  const double* __restrict__ gvec, double* dvec, float* dF,
                                                  float* Dout, const float* __restrict__ R, int64_t n, int64_t n_pad,
                                                  const unsigned long long* __restrict__ argkey, unsigned* sg,
                                                  unsigned* fired) {
  __shared__ double Gs[4096];
  __shared__ double colbuf[1024];
  const double gain = scale_solve(gacc, bb, gramV, gvec, dvec, dF, Dout, Gs, colbuf, true);
  const unsigned long long key = *argkey;
  const float rmax = __uint_as_float((unsigned)(key >> 32));
  const bool fire = rmax > 0.0f && (double)rmax * (double)rmax > gain;
  const int t = threadIdx.x;
  // thread t wrote dvec[t], dF[t] and Dout[t] in the solve
  if (fire && t < BBP) {
    const float dv = t == 0 ? rmax : 0.0f;
    dvec[t] = (double)dv;
    dF[t] = dv;
    if (t < bb) Dout[t] = dv;
  }
  if (t == 0) {
    unsigned i = 0u, j = 0u, neg = 0u;
    if (fire) {
      const unsigned flat = 0xFFFFFFFFu - (unsigned)(key & 0xFFFFFFFFull);
      i = (unsigned)(flat / (unsigned long long)n);
      j = (unsigned)(flat % (unsigned long long)n);
      neg = R[(int64_t)i * n_pad + j] < 0.0f ? 1u : 0u;
      *fired += 1u;
    }
    sg[0] = fire ? 1u : 0u;
    sg[1] = i;
    sg[2] = j;
    sg[3] = neg;
  }
}

// ---------------------------------------------------------------------------
// step-entry helpers: caller layouts <-> workspace layouts
// ---------------------------------------------------------------------------
// X: len x bb row-major int8 -> Xt (BBP x len_pad) and Xr (len_pad x BBP), zero padded.
__global__ __launch_bounds__(NT) void k_load_factor(int8_t* Xt, int8_t* Xr, int8_t* Xmf, const int8_t* X, int64_t len,
                                                    int64_t len_pad, int bb, int ld) {
  const int64_t total = len_pad * BBP;
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < total; e += (int64_t)gridDim.x * NT) {
    const int64_t i = e / BBP;
    const int c = (int)(e % BBP);
    const int8_t v = (i < len && c < bb) ? X[i * ld + c] : (int8_t)0;
    Xr[e] = v;
    Xt[(int64_t)c * len_pad + i] = v;
    Xmf[mf_offset(c, i)] = v;
  }
}
__global__ __launch_bounds__(NT) void k_store_factor(int8_t* X, const int8_t* Xt, int64_t len, int64_t len_pad,
                                                     int bb) {
  const int64_t total = len * bb;
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < total; e += (int64_t)gridDim.x * NT) {
    const int64_t i = e / bb;
    const int c = (int)(e % bb);
    X[e] = Xt[(int64_t)c * len_pad + i];
  }
}
// component-major (BBP x len_pad) <-> row-major (len x bb)
__global__ __launch_bounds__(NT) void k_store_cm(double* X, const double* Xcm, int64_t len, int64_t len_pad,
                                                 int bb) {
  const int64_t total = len * bb;
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < total; e += (int64_t)gridDim.x * NT) {
    const int64_t i = e / bb;
    const int c = (int)(e % bb);
    X[e] = Xcm[(int64_t)c * len_pad + i];
  }
}
__global__ __launch_bounds__(NT) void k_load_cm(double* Xcm, const double* X, int64_t len, int64_t len_pad,
                                                int bb) {
  const int64_t total = len_pad * (bb > BBP ? BMAX : BBP);
  for (int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x; e < total; e += (int64_t)gridDim.x * NT) {
    const int c = (int)(e / len_pad);
    const int64_t i = e % len_pad;
    Xcm[e] = (i < len && c < bb) ? X[i * bb + c] : 0.0;
  }
}


// Weighted Gram of V alone (raw V^T diag(H) V into gramV), for the scale
// step entry point: the arithmetic of the U-step's side path in a launch of
// its own.  grid: NSIDE_GRAM.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_gram_vw(
    const v4i* __restrict__ Vmf, const int8_t* __restrict__ Wmf, int64_t n_pad, long long* gacc64,
    const double* __restrict__ hwmax, unsigned* counter, double* gramV) {
  __shared__ __attribute__((aligned(16))) int red[4 * 4096];
  __shared__ double Gs[4096];
  if (!side_gram_w(Vmf, Wmf, (int64_t)BMAX * n_pad, n_pad, blockIdx.x, (int)gridDim.x, gacc64, hwmax[1], counter, Gs,
                   red))
    return;
  for (int e = threadIdx.x; e < 4096; e += NT) gramV[e] = Gs[e];
}

// The digit-scaled planes of a V given by the caller (step entry points;
// in a factorization k_tern_v writes them with V): Wmf[d * wstride + o] =
// dig_d(j) v_jc for the MFMA-ready byte o of (c, j), for the nq quarters.
// grid: (n_pad / 32 K steps, nq); thread t < 128 takes the 16 bytes
// (K step, t) of the quarter.
__global__ __launch_bounds__(128) void k_vweight(const v4i* __restrict__ Vmf, const int8_t* __restrict__ hdig,
                                                 int64_t n_pad, int8_t* __restrict__ Wmf, int64_t wstride) {
  const int64_t ks = blockIdx.x, q = blockIdx.y;
  const int t = threadIdx.x, h = (t & 63) >> 5;
  const int64_t e = q * 4 * n_pad + ks * 128 + t;  // v4i index within Vmf
  const v4i x = Vmf[e];
#pragma unroll
  for (int d = 0; d < WDIG; ++d) {
    const v4i dg = *(const v4i*)(hdig + (int64_t)d * n_pad + ks * TILE + 16 * h);
    v4i r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = trit_times_digit(x[k], dg[k]);
    ((v4i*)(Wmf + (int64_t)d * wstride))[e] = r;
  }
}

// Integer Gram of V alone (raw V^T V and its ridge inverse), for the scale
// step entry point; the weighted Gram comes from k_gram_vw.
// grid: NSIDE_INT.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_gram_v(const v4i* __restrict__ Vmf, int64_t n_pad, int bb, int* gparti,
                                               unsigned* counter, double* ginvV, double* gramV) {
  __shared__ __attribute__((aligned(16))) int red[4096];
  __shared__ double Gs[4096];
  __shared__ double colbuf[1024];
  if (!side_gram_int(Vmf, n_pad, blockIdx.x, (int)gridDim.x, gparti, counter, Gs, red)) return;
  for (int e = threadIdx.x; e < 4096; e += NT) gramV[e] = Gs[e];
  __syncthreads();
  ridge_invert_store(Gs, colbuf, bb, ginvV);
}

// Integer Gram of a factor given by the caller (step entry points): adds
// X^T X into gacc.  grid: NSIDE_GRAM WGs over the K steps.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_gram_acc(const v4i* __restrict__ Xmf, int64_t L_pad, int* gacc) {
  const int nks = (int)(L_pad / TILE);
  gram_accumulate(Xmf, (int)((long long)blockIdx.x * nks / gridDim.x), (int)((long long)(blockIdx.x + 1) * nks / gridDim.x),
                  gacc, nullptr);
}

// g_c = sum_i U_ic Q_ic (fp64), in slot 0 of the per-split partial sums.
// grid: BBP.
__global__ __launch_bounds__(NT) void k_gvec(const int8_t* __restrict__ Ut, const double* __restrict__ Q, int64_t m,
                                             int64_t m_pad, int bb, double* __restrict__ gvec) {
  __shared__ double shd[16];
  const int c = blockIdx.x;
  double acc = 0.0;
  if (c < bb)
    for (int64_t i = threadIdx.x; i < m; i += NT) acc += (double)Ut[(int64_t)c * m_pad + i] * Q[(int64_t)c * m_pad + i];
  acc = block_sum_d(acc, shd);
  if (threadIdx.x < TERN_SPLIT_MAX) gvec[c * TERN_SPLIT_MAX + threadIdx.x] = threadIdx.x == 0 ? acc : 0.0;
}

// Scales given by the caller: dvec = d, dF = fp32(d), zero beyond bb.
__global__ void k_set_scales(const double* __restrict__ d, int bb, double* dvec, float* dF) {
  const int c = threadIdx.x;
  if (c < BMAX) {
    const double v = (c < bb) ? d[c] : 0.0;
    dvec[c] = v;
    dF[c] = (float)v;
  }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Wide blocks (bb up to BMAX = NQMAX x 64 components, Sec. 2.4): the Gram
// matrices of Eq. (3) and the matrix of the joint solve of Eq. (4) couple
// the quarters of a block; they are formed here as BMAX x BMAX fp64 matrices
// (64 x 64 blocks, quarter pairs q <= q') and inverted by a blocked sweep.
// ---------------------------------------------------------------------------
// quarter pair p <-> (q, q') with q <= q' < nq, in row order
__device__ __forceinline__ void pair_of(int p, int nq, int& q, int& q2) {
  q = 0;
  while (p >= nq - q) {
    p -= nq - q;
    ++q;
  }
  q2 = q + p;
}
__host__ __device__ __forceinline__ int pair_index(int q, int q2, int nq) {
  return q * nq - q * (q - 1) / 2 + (q2 - q);
}

// Integer Gram blocks X_q^T X_q' of a ternary factor (MFMA-ready layout,
// quarter q at byte 64 q L_pad) for every pair q <= q' < nq, on int8 MFMA,
// added into gaccW[pair] with integer atomics (exact, order-free); the
// sweep's first pivot launch clears gaccW again.
// grid: npairs x nslice workgroups, workgroup (pair, slice) takes a slice of
// the K steps.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_gram_pairs(
    const v4i* __restrict__ Xmf, int64_t L_pad, int nq, int nslice, int* __restrict__ gaccW) {
  __shared__ int red[4 * 4096];
  const int p = blockIdx.x / nslice, sl = blockIdx.x % nslice;
  int q, q2;
  pair_of(p, nq, q, q2);
  const int nks = (int)(L_pad / TILE);
  const int ks0 = (int)((long long)sl * nks / nslice), ks1 = (int)((long long)(sl + 1) * nks / nslice);
  const v4i* Xa = Xmf + (int64_t)q * 4 * L_pad;
  const v4i* Xb = Xmf + (int64_t)q2 * 4 * L_pad;
  constexpr int KR = 4;
  const int lane = lane_id(), wave = wave_id();
  const int h = lane >> 5, l32 = lane & 31;
  v16i acc00 = {}, acc01 = {}, acc10 = {}, acc11 = {};
  for (int ks = ks0 + wave; ks < ks1; ks += 4 * KR) {
    v4i a[KR][2], b[KR][2];
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      const int kk = ks + 4 * u;
      if (kk < ks1) {
        a[u][0] = Xa[(int64_t)kk * 128 + lane];
        a[u][1] = Xa[(int64_t)kk * 128 + 64 + lane];
        b[u][0] = Xb[(int64_t)kk * 128 + lane];
        b[u][1] = Xb[(int64_t)kk * 128 + 64 + lane];
      } else {
        a[u][0] = a[u][1] = b[u][0] = b[u][1] = v4i{};
      }
    }
#pragma unroll
    for (int u = 0; u < KR; ++u) {
      acc00 = mfma_i8(a[u][0], b[u][0], acc00);
      acc01 = mfma_i8(a[u][0], b[u][1], acc01);
      acc10 = mfma_i8(a[u][1], b[u][0], acc10);
      acc11 = mfma_i8(a[u][1], b[u][1], acc11);
    }
  }
  int* mine = red + wave * 4096;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int M = 8 * (r >> 2) + 4 * h + (r & 3);
    const int N = l32;
    mine[M * 64 + N] = acc00[r];
    mine[M * 64 + 32 + N] = acc01[r];
    mine[(32 + M) * 64 + N] = acc10[r];
    mine[(32 + M) * 64 + 32 + N] = acc11[r];
  }
  __syncthreads();
  int* g = gaccW + (int64_t)p * 4096;
  for (int e = threadIdx.x; e < 4096; e += NT) {
    const int v = red[e] + red[4096 + e] + red[8192 + e] + red[12288 + e];
    if (v) __hip_atomic_fetch_add(g + e, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Weighted Gram blocks V_q^T diag(H) V_q' of V (Sec. 2.5) for every pair
// q <= q' < nq on int8 MFMA from the digit-scaled planes of V (the
// arithmetic of gram_w_accumulate), added into g64[pair] (int64 atomics, exact and
// order-free); the sweep's first pivot launch clears g64 again.
// grid: npairs x nslice workgroups, workgroup (pair, slice) takes a slice of
// the K steps.
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void k_gram_pairs_w(
    const v4i* __restrict__ Vmf, const int8_t* __restrict__ Wmf, int64_t n_pad, int nq, int nslice,
    long long* __restrict__ g64) {
  __shared__ int red[4 * 4096];
  const int p = blockIdx.x / nslice, sl = blockIdx.x % nslice;
  int q, q2;
  pair_of(p, nq, q, q2);
  const int nks = (int)(n_pad / TILE);
  const int ks0 = (int)((long long)sl * nks / nslice), ks1 = (int)((long long)(sl + 1) * nks / nslice);
  gram_w_accumulate<false>(Vmf + (int64_t)q * 4 * n_pad, Wmf + (int64_t)q2 * BBP * n_pad, (int64_t)BMAX * n_pad, ks0,
                           ks1, g64 + (int64_t)p * 4096, red);
}

// The matrix to sweep, A (BMAX-stride row-major, nq x nq blocks), from one
// pair block per workgroup (both triangles):
//   mode 0: (G + eps I) from the integer Gram blocks gaccW, the raw Gram
//           also into raw (if given);
//   mode 1: (G + eps I) from the weighted integer Gram blocks g64 times
//           their unit (hwmax[1]), the raw Gram into raw;
//   mode 2: (G_U o G_V + delta I) from gaccW (G_U) and raw (G_V), Eq. (4);
// with eps or delta = rel * trace / bb over the bb real components and the
// identity on the padding components.  A zero trace sets wflag[0] (the
// result is then zero targets, or zero scales) and leaves the identity in A.
// grid: npairs.
__global__ __launch_bounds__(NT) void k_wide_prep(int mode, const int* __restrict__ gaccW,
                                                  const double* __restrict__ hwmax, double* raw, int bb, int nq,
                                                  double rel, double* __restrict__ A, int* __restrict__ wflag) {
  __shared__ double shd[NT / 64];
  const int p = blockIdx.x;
  int q, q2;
  pair_of(p, nq, q, q2);
  // trace over the real components, the same arithmetic in every workgroup
  double dv = 0.0;
  const int c = threadIdx.x;  // BMAX == NT: one diagonal entry per thread
  if (c < bb) {
    const int qc = c / BBP, cl = c % BBP, pd = pair_index(qc, qc, nq);
    if (mode == 0) dv = (double)gaccW[(int64_t)pd * 4096 + cl * 65];
    else if (mode == 1)
      dv = (double)((const long long*)gaccW)[(int64_t)pd * 4096 + cl * 65] * hwmax[1];
    else
      dv = (double)gaccW[(int64_t)pd * 4096 + cl * 65] * raw[(int64_t)c * BMAX + c];
  }
  const double tr = block_sum_d(dv, shd);
  const bool zero = tr == 0.0;
  if (p == 0 && threadIdx.x == 0) *wflag = zero ? 1 : 0;
  const double ridge = zero ? 0.0 : rel * tr / (double)bb;
  // The block's values first, every load issued before any is used (a loop
  // that stores each value would wait for each load in turn).
  constexpr int PER = 4096 / NT;
  double vals[PER];
  if (mode == 1) {
    const double unit = hwmax[1];
    long long gv[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) gv[u] = ((const long long*)gaccW)[(int64_t)p * 4096 + threadIdx.x + NT * u];
#pragma unroll
    for (int u = 0; u < PER; ++u) vals[u] = (double)gv[u] * unit;
  } else if (mode == 2) {
    int gv[PER];
    double rv[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + NT * u;
      gv[u] = gaccW[(int64_t)p * 4096 + e];
      rv[u] = raw[(int64_t)(BBP * q + (e >> 6)) * BMAX + BBP * q2 + (e & 63)];
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) vals[u] = (double)gv[u] * rv[u];
  } else {
    int gv[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) gv[u] = gaccW[(int64_t)p * 4096 + threadIdx.x + NT * u];
#pragma unroll
    for (int u = 0; u < PER; ++u) vals[u] = (double)gv[u];
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + NT * u;
    const int r = e >> 6, cc = e & 63;
    const int gi = BBP * q + r, gj = BBP * q2 + cc;
    const bool real = gi < bb && gj < bb;
    double v = vals[u];
    if (!real) v = 0.0;
    if (raw && mode != 2) {
      raw[(int64_t)gi * BMAX + gj] = v;
      raw[(int64_t)gj * BMAX + gi] = v;
    }
    double a = (gi == gj) ? (real && !zero ? v + ridge : 1.0) : (zero ? 0.0 : v);
    A[(int64_t)gi * BMAX + gj] = a;
    A[(int64_t)gj * BMAX + gi] = a;
  }
}

// C (64 x 64 block of this workgroup, rows 16 w .. of wave w) += X Y for
// 64 x 64 operands with leading dimensions ldx, ldy, on fp64 MFMA:
// acc[nt][r] <-> row 16 w + lane / 16 + 4 r, column 16 nt + lane % 16.
__device__ __forceinline__ void gemm64(const double* X, int64_t ldx, const double* Y, int64_t ldy, v4d (&acc)[4]) {
  const int lane = lane_id(), w = wave_id();
  const int li = lane & 15, lk = lane >> 4;
#pragma unroll 4
  for (int ks = 0; ks < 16; ++ks) {
    const double a = X[(int64_t)(16 * w + li) * ldx + 4 * ks + lk];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma_f64(a, Y[(int64_t)(4 * ks + lk) * ldy + 16 * nt + li], acc[nt]);
  }
}

// C += X Y for 64 x 64 operands in LDS, both stored K-major: XT[kk][row]
// (XT = X^T) and Y[kk][col], row strides ldx and ldy (80 doubles: lanes
// 0..31 of a read then cover all 64 banks); the accumulator layout of
// gemm64.
__device__ __forceinline__ void gemm64_kmajor(const double* XT, int ldx, const double* Y, int ldy, v4d (&acc)[4]) {
  const int lane = lane_id(), w = wave_id();
  const int li = lane & 15, lk = lane >> 4;
#pragma unroll 4
  for (int ks = 0; ks < 16; ++ks) {
    const double a = XT[(4 * ks + lk) * ldx + 16 * w + li];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma_f64(a, Y[(4 * ks + lk) * ldy + 16 * nt + li], acc[nt]);
  }
}

// One step of the blocked sweep as one launch: every workgroup inverts the
// pivot block itself (the same arithmetic in each, so all hold the same
// P = A_kk^{-1}) and updates its own block, A -> B:
//   B_kk = -P, B_kj = P A_kj, B_ik = A_ik P, B_ij = A_ij - (A_ik P) A_kj.
// The swept matrix stays symmetric, so A_ik^T is the stored block A_ki and
// P^T = P.  All operand blocks are loaded into LDS at once (one memory
// latency) and the products read LDS.  nk: 4 x 4 pivots holding real
// components; step 0 also clears the integer Gram blocks (nclear entries,
// split over the workgroups) for the next accumulation.  grid: nq x nq.
constexpr int SWEEP_LD = 80;
__global__ __launch_bounds__(NT) void k_wide_step(const double* __restrict__ A, double* __restrict__ B, int k,
                                                  int nq, int nk, int* gaccW, int nclear) {
  __shared__ double Gs[4096];                   // the pivot block, then P (row stride 64)
  __shared__ double pbuf[1024];
  __shared__ double XT[BBP * SWEEP_LD];         // A_ki = A_ik^T, then (A_ik P)^T
  __shared__ double Ys[BBP * SWEEP_LD];         // A_kj
  const int i = blockIdx.x / nq, j = blockIdx.x % nq;
  const int lane = lane_id(), w = wave_id();
  const int li = lane & 15, lk = lane >> 4;
  if (nclear) {
    const int per = (nclear + (int)gridDim.x - 1) / (int)gridDim.x;
    const int e0 = per * (int)blockIdx.x, e1 = e0 + per < nclear ? e0 + per : nclear;
    for (int e = e0 + threadIdx.x; e < e1; e += NT) gaccW[e] = 0;
  }
  const double* Akk = A + (int64_t)BBP * k * BMAX + BBP * k;
  const double* Aki = A + (int64_t)BBP * k * BMAX + BBP * i;
  const double* Akj = A + (int64_t)BBP * k * BMAX + BBP * j;
  const double* Aij = A + (int64_t)BBP * i * BMAX + BBP * j;
  double* Bij = B + (int64_t)BBP * i * BMAX + BBP * j;
  const bool gen = i != k && j != k;
  // A_ij for the general blocks, in the accumulator layout (issued first)
  double aij[4][4];
  if (gen) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) aij[nt][r] = Aij[(int64_t)(16 * w + lk + 4 * r) * BMAX + 16 * nt + li];
  }
  // every load of the three blocks issued before the first LDS store (a
  // loop that stores each value would wait for each load in turn); blocks
  // a workgroup does not use read the pivot block again
  constexpr int PER = 4096 / NT;
  const double* Xsrc = (j == k || gen) ? Aki : Akk;
  const double* Ysrc = (i == k || gen) ? Akj : Akk;
  double gv[PER], xv[PER], yv[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = threadIdx.x + NT * q;
    const int64_t o = (int64_t)(e >> 6) * BMAX + (e & 63);
    gv[q] = Akk[o];
    xv[q] = Xsrc[o];
    yv[q] = Ysrc[o];
  }
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = threadIdx.x + NT * q;
    const int r = e >> 6, c = e & 63;
    Gs[e] = gv[q];
    XT[r * SWEEP_LD + c] = xv[q];
    Ys[r * SWEEP_LD + c] = yv[q];
  }
  __syncthreads();
  spd_inverse64(Gs, pbuf, nk);  // Gs = P (ends with a barrier)
  v4d acc[4] = {v4d{}, v4d{}, v4d{}, v4d{}};
  double sgn = 1.0;
  if (i == k && j == k) {
    for (int e = threadIdx.x; e < 4096; e += NT) Bij[(int64_t)(e >> 6) * BMAX + (e & 63)] = -Gs[e];
    return;
  } else if (i == k) {
    gemm64_kmajor(Gs, BBP, Ys, SWEEP_LD, acc);  // P A_kj (P^T = P)
  } else if (j == k) {
    gemm64_kmajor(XT, SWEEP_LD, Gs, BBP, acc);  // A_ik P
  } else {
    gemm64_kmajor(XT, SWEEP_LD, Gs, BBP, acc);  // T = A_ik P
    __syncthreads();                            // every wave is done with A_ki
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) XT[(16 * nt + li) * SWEEP_LD + 16 * w + lk + 4 * r] = acc[nt][r];  // T^T
    __syncthreads();
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = v4d{};
    gemm64_kmajor(XT, SWEEP_LD, Ys, SWEEP_LD, acc);
    sgn = -1.0;
  }
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t o = (int64_t)(16 * w + lk + 4 * r) * BMAX + 16 * nt + li;
      Bij[o] = (sgn < 0.0 ? aij[nt][r] : 0.0) + sgn * acc[nt][r];
    }
}

// G^{-1} = -S (S: the fully swept matrix) into nq x nq blocks in the fp64
// MFMA operand order of the target kernels (block (q, q') at
// ginvW + (q NQMAX + q') 4096); with zero trace (wflag) the inverse is zero
// on the real components and the identity on the padding.  grid: nq x nq.
__global__ __launch_bounds__(NT) void k_wide_ginv(const double* __restrict__ S, int nq, int bb,
                                                  const int* __restrict__ wflag, double* __restrict__ ginvW) {
  const int i = blockIdx.x / nq, j = blockIdx.x % nq;
  const bool zero = *wflag != 0;
  double* out = ginvW + (int64_t)(i * NQMAX + j) * 4096;
  constexpr int PER = 4096 / NT;
  double sv[PER];  // every load before the first store
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + NT * u;
    sv[u] = S[(int64_t)(BBP * i + (e >> 6)) * BMAX + BBP * j + (e & 63)];
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + NT * u;
    const int r = e >> 6, c = e & 63;
    const int gi = BBP * i + r, gj = BBP * j + c;
    double v;
    if (zero) v = (gi >= bb || gj >= bb) ? (gi == gj ? 1.0 : 0.0) : 0.0;
    else v = -sv[u];
    out[ginv_index(r, c)] = v;
  }
}

// Joint scales of a wide block, d = M^{-1} g (Eq. (4)) with M^{-1} = -S and
// g_c = diag(U^T Q)_c (the per-split partial sums in split order); zero
// trace: d = 0.  d into dvec, dF (fp32) and D (the block's output).
// One workgroup; row c of the product by thread c (columns in order).
__global__ __launch_bounds__(NT) void k_wide_scales(const double* __restrict__ S, const double* __restrict__ gvec,
                                                    int bb, const int* __restrict__ wflag, double* dvec, float* dF,
                                                    float* Dout) {
  __shared__ double g[BMAX];
  const int c = threadIdx.x;  // BMAX == NT
  double gc = 0.0;
  if (c < bb)
#pragma unroll
    for (int k = 0; k < TERN_SPLIT_MAX; ++k) gc += gvec[c * TERN_SPLIT_MAX + k];
  g[c] = gc;
  __syncthreads();
  double d = 0.0;
  if (c < bb && *wflag == 0) {
    for (int c2 = 0; c2 < bb; ++c2) d += -S[(int64_t)c * BMAX + c2] * g[c2];
  }
  dvec[c] = d;
  dF[c] = (float)d;
  if (Dout && c < bb) Dout[c] = (float)d;
}

static inline unsigned grid_for(int64_t total) {
  int64_t g = (total + NT - 1) / NT;
  if (g < 1) g = 1;
  if (g > 8192) g = 8192;
  return (unsigned)g;
}

hipError_t launch_prep(const Ws& w, const float* h, hipStream_t s, double lam) {
  hipLaunchKernelGGL(k_prep, dim3(1), dim3(NT), 0, s, h, w.n, w.n_pad, w.hw, w.hwmax, w.fro2_hist,
                     w.fro2w_hist, w.nblk_cap, w.counters, w.flags, w.gacc, lam, w.argkey, w.gaccW, w.gacc64,
                     w.hdig, w.vtcnt);
  return hipGetLastError();
}

hipError_t launch_stage(const Ws& w, const float* A, int64_t lda, hipStream_t s, bool track) {
  const unsigned grid = (unsigned)((w.n_pad / TILE) * w.gd);
  if (track)
    hipLaunchKernelGGL(k_stage<true>, dim3(grid), dim3(NT), 0, s, A, lda, w.m, w.n, w.R, w.colE_part, w.rowb_part,
                       (const double*)w.hw, w.flags, w.m_pad, w.n_pad, w.gd, w.argkey);
  else
    hipLaunchKernelGGL(k_stage<false>, dim3(grid), dim3(NT), 0, s, A, lda, w.m, w.n, w.R, w.colE_part, w.rowb_part,
                       (const double*)w.hw, w.flags, w.m_pad, w.n_pad, w.gd, (unsigned long long*)nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rowb_init, dim3((unsigned)((w.m_pad + NT - 1) / NT)), dim3(NT), 0, s,
                     (const float*)w.rowb_part, (int)(w.n_pad / TILE), w.m_pad, w.rowb);
  return hipGetLastError();
}

hipError_t launch_unstage(const Ws& w, float* A, hipStream_t s) {
  hipLaunchKernelGGL(k_unstage, dim3(grid_for(w.m * w.n)), dim3(NT), 0, s, w.R, A, w.m, w.n, w.n_pad);
  return hipGetLastError();
}

hipError_t launch_select(const Ws& w, int blk, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_select, dim3(1), dim3(NT_SELECT), 0, s, w.colE_part, w.gd, w.n, w.n_pad, w.hw, w.Y,
                     w.fro2_hist + blk, w.fro2w_hist + blk, bb, w.J, w.cshift);
  return hipGetLastError();
}

hipError_t launch_finish(const Ws& w, int blk, hipStream_t s) {
  hipLaunchKernelGGL(k_finish, dim3(1), dim3(NT_SELECT), 0, s, w.colE_part, w.gd, w.n, w.n_pad, w.hw,
                     (double*)nullptr, w.fro2_hist + blk, w.fro2w_hist + blk, w.cshift);
  return hipGetLastError();
}

hipError_t launch_colnorms(const Ws& w, int blk, double* colnorm2, double* fro2, hipStream_t s) {
  hipLaunchKernelGGL(k_finish, dim3(1), dim3(NT_SELECT), 0, s, w.colE_part, w.gd, w.n, w.n_pad, w.hw, colnorm2,
                     fro2 ? fro2 : (w.fro2_hist + blk), w.fro2w_hist + blk, w.cshift);
  return hipGetLastError();
}

hipError_t launch_init(const Ws& w, int bb, double tau, hipStream_t s) {
  hipLaunchKernelGGL(k_init_gather, dim3((unsigned)(w.m_pad / TILE)), dim3(NT), 0, s, w.R, w.J, w.m, w.m_pad, w.n_pad,
                     bb, w.Z, w.tps, w.tpm, w.tpi);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_tern_u, dim3(BBP * w.nsu), dim3(NT), 0, s, w.Z, (const double*)nullptr, w.m, w.m_pad, bb, tau,
                     w.tps, w.tpm, w.tpi, (int)(w.m_pad / TILE), w.nsu, w.Ut, w.Umf, w.gvec, (unsigned*)nullptr);
  return hipGetLastError();
}

// One launch forms P = U^T R (gv row-group partials per column tile),
// G_U^{-1} (side path) and, in the last row group of each column tile, the
// targets Y = G_U^{-1} P with their statistics (one tile per 32 columns).
hipError_t launch_vstep(const Ws& w, int blk, int bb, double tau, hipStream_t s, Timer* tm, bool weighted) {
  const int nsb = (int)((w.n_pad / TILE) * w.gv);  // streaming workgroups, plus the empty slots past 256
  const unsigned grid = (unsigned)(NSIDE_GRAM + nsb + (nsb > 256 - NSIDE_GRAM ? NSIDE_GRAM : 0));
  unsigned* ready = w.counters + CNT_GINV_U;
  EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_VSTEP, k_vstep, dim3(grid), dim3(NT), 0, s, w.R, (const v4i*)w.Umf, w.Pp, (const int*)w.cshift, w.m_pad,
                                   w.n_pad, w.gv, bb, w.gacc, w.counters + CNT_GRAM_U, w.ginvU, NSIDE_GRAM, w.Y,
                                   w.tps, w.tpm, w.tpi, w.n, w.vtcnt, ready, w.flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_TERNV, k_tern_v, dim3(BBP * w.nsv), dim3(NT), 0, s, (const double*)w.Y, w.n,
                       w.n_pad, bb, tau, (const double*)w.tps, (const double*)w.tpm, (const int*)w.tpi,
                       (int)(w.n_pad / TILE), w.nsv, w.Vt, w.Vmf, (const int8_t*)w.hdig, weighted ? w.Wmf : nullptr,
                       (int64_t)BMAX * w.n_pad, ready);
  return hipGetLastError();
}

// One launch forms Q = R diag(h~) V, G_V^{-1} (side path) and the targets
// Z = Q G_V^{-1} with their statistics (one tile per row group); Q is
// stored only where it is read afterwards (g of the last U-step of a block,
// the step API).
hipError_t launch_ustep(const Ws& w, int blk, int bb, double tau, bool weighted, bool final, hipStream_t s,
                        Timer* tm, bool keep_q) {
  hipError_t e;
  static_assert(NSIDE_GRAM == NSIDE_MAX, "the empty row-group slots match the side workgroups");
  const unsigned nside = NSIDE_GRAM;
  const unsigned grid = (unsigned)(nside + w.ntu);
  unsigned* ready = w.counters + CNT_GINV_V;
  const int storeQ = (final || keep_q) ? 1 : 0;
  if (weighted)
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_USTEP, (k_ustep<true>), dim3(grid), dim3(NT), 0, s, w.R, (const v4i*)w.Vmf, w.Vr, w.hw, w.Q,
                                     w.rowb, w.m_pad, w.n_pad, bb, w.gacc + 4096,
                                     w.counters + CNT_GRAM_V, w.ginvV, w.gramV, (int)nside, w.urows,
                                     (const int8_t*)w.Wmf, w.gacc64, (const double*)w.hwmax, w.Z, w.tps, w.tpm,
                                     w.tpi, w.m, ready, w.flags, storeQ);
  else
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_USTEP, (k_ustep<false>), dim3(grid), dim3(NT), 0, s, w.R, (const v4i*)w.Vmf, w.Vr, w.hw, w.Q,
                                     w.rowb, w.m_pad, w.n_pad, bb, w.gacc + 4096,
                                     w.counters + CNT_GRAM_V, w.ginvV, w.gramV, (int)nside, w.urows,
                                     (const int8_t*)nullptr, (long long*)nullptr, (const double*)nullptr, w.Z,
                                     w.tps, w.tpm, w.tpi, w.m, ready, w.flags, storeQ);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_TERNU, k_tern_u, dim3(BBP * w.nsu), dim3(NT), 0, s, (const double*)w.Z,
                       final ? (const double*)w.Q : nullptr, w.m, w.m_pad, bb, tau, (const double*)w.tps,
                       (const double*)w.tpm, (const int*)w.tpi, w.ntu - (int)NSIDE_MAX, w.nsu, w.Ut, w.Umf, w.gvec,
                       ready);
  return hipGetLastError();
}

// ---- wide blocks (nq = ceil(bb / 64) > 1 quarters) ----
static int nq_of(int bb) { return (bb + BBP - 1) / BBP; }
static int bb_of_quarter(int bb, int q) { return bb - BBP * q < BBP ? bb - BBP * q : BBP; }
constexpr int GRAM_PAIR_SLICES = 16;  // K slices per quarter pair of the integer Gram

// Blocked sweep of the matrix prepared in wA0 (nq quarters): one launch
// per pivot block (k_wide_step: every workgroup inverts the pivot and
// updates its block); *out receives the buffer holding -A^{-1}.  The first
// step clears the integer Gram blocks.
static hipError_t wide_sweep(const Ws& w, int bb, hipStream_t s, const double** out, bool clear64 = false) {
  const int nq = nq_of(bb), npairs = nq * (nq + 1) / 2;
  const int nclear = (clear64 ? 2 : 1) * npairs * 4096;  // int32 words of the Gram blocks used
  double* A = w.wA0;
  double* B = w.wA1;
  for (int k = 0; k < nq; ++k) {
    const int bq = bb_of_quarter(bb, k);
    hipLaunchKernelGGL(k_wide_step, dim3((unsigned)(nq * nq)), dim3(NT), 0, s, (const double*)A, B, k, nq,
                       (bq + 3) / 4, w.gaccW, k == 0 ? nclear : 0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    double* t = A;
    A = B;
    B = t;
  }
  *out = A;
  return hipSuccess;
}

// (X^T diag(h~) X + eps I)^{-1} of the block's U (which = 0) or V (which = 1,
// weighted with h~ when `weighted`) into ginvUW / ginvVW; for V the raw Gram
// is kept in gramVW for the joint solve.
static hipError_t wide_gram_inverse(const Ws& w, int which, bool weighted, int bb, hipStream_t s) {
  static_assert(BMAX == NT, "one diagonal entry per thread in the wide preparation");
  const int nq = nq_of(bb), npairs = nq * (nq + 1) / 2;
  hipError_t e;
  if (which == 1 && weighted) {
    hipLaunchKernelGGL(k_gram_pairs_w, dim3((unsigned)(npairs * GRAM_PAIR_SLICES)), dim3(NT), 0, s,
                       (const v4i*)w.Vmf, (const int8_t*)w.Wmf, w.n_pad, nq, GRAM_PAIR_SLICES, (long long*)w.gaccW);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_wide_prep, dim3((unsigned)npairs), dim3(NT), 0, s, 1, (const int*)w.gaccW,
                       (const double*)w.hwmax, w.gramVW, bb, nq, EXTERND_RIDGE_REL, w.wA0, w.wflag);
  } else {
    const v4i* X = (const v4i*)(which ? w.Vmf : w.Umf);
    hipLaunchKernelGGL(k_gram_pairs, dim3((unsigned)(npairs * GRAM_PAIR_SLICES)), dim3(NT), 0, s, X,
                       which ? w.n_pad : w.m_pad, nq, GRAM_PAIR_SLICES, w.gaccW);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_wide_prep, dim3((unsigned)npairs), dim3(NT), 0, s, 0, (const int*)w.gaccW,
                       (const double*)w.hwmax, which ? w.gramVW : (double*)nullptr, bb, nq, EXTERND_RIDGE_REL,
                       w.wA0, w.wflag);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const double* S = nullptr;
  e = wide_sweep(w, bb, s, &S, which == 1 && weighted);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_wide_ginv, dim3((unsigned)(nq * nq)), dim3(NT), 0, s, S, nq, bb, (const int*)w.wflag,
                     which ? w.ginvVW : w.ginvUW);
  return hipGetLastError();
}

hipError_t launch_init_wide(const Ws& w, int bb, double tau, hipStream_t s) {
  for (int q = 0; q < nq_of(bb); ++q) {
    const hipError_t e = launch_init(quarter_view(w, q), bb_of_quarter(bb, q), tau, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_vstep_wide(const Ws& w, int blk, int bb, double tau, hipStream_t s, Timer* tm, bool weighted) {
  const int nq = nq_of(bb);
  hipError_t e;
  // P_q = U_q^T R per quarter (contraction launches without a side path)
  for (int q = 0; q < nq; ++q) {
    const Ws v = quarter_view(w, q);
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_VSTEP, k_vstep, dim3((unsigned)((w.n_pad / TILE) * w.gv)), dim3(NT), 0,
                         s, w.R, (const v4i*)v.Umf, v.Pp, (const int*)w.cshift, w.m_pad, w.n_pad, w.gv,
                         bb_of_quarter(bb, q), w.gacc, w.counters + CNT_GRAM_U, w.ginvU, 0, (double*)nullptr,
                         (double*)nullptr, (double*)nullptr, (int*)nullptr, w.n, (unsigned*)nullptr,
                         (unsigned*)nullptr, (int*)nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  e = wide_gram_inverse(w, 0, false, bb, s);
  if (e != hipSuccess) return e;
  for (int q = 0; q < nq; ++q) {
    const Ws v = quarter_view(w, q);
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_VTARGET, k_vtarget<true>, dim3((unsigned)(w.n_pad / 16)), dim3(NT), 0, s,
                         (const long long*)w.Pp, (const int*)w.cshift, w.n_pad, w.gv,
                         (const double*)(w.ginvUW + (int64_t)q * NQMAX * 4096), v.Y, w.n, v.tps, v.tpm, v.tpi, nq,
                         (int64_t)BBP * w.gv * w.n_pad);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_TERNV, k_tern_v, dim3(BBP * w.nsv), dim3(NT), 0, s, (const double*)v.Y,
                         w.n, w.n_pad, bb_of_quarter(bb, q), tau, (const double*)v.tps, (const double*)v.tpm,
                         (const int*)v.tpi, (int)(w.n_pad / 16), w.nsv, v.Vt, v.Vmf, (const int8_t*)w.hdig,
                         weighted ? v.Wmf : nullptr, (int64_t)BMAX * w.n_pad, (unsigned*)nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_ustep_wide(const Ws& w, int blk, int bb, double tau, bool weighted, bool final, hipStream_t s,
                             Timer* tm) {
  const int nq = nq_of(bb);
  hipError_t e;
  // Q_q = R diag(h~) V_q per quarter (contraction launches without a side path)
  for (int q = 0; q < nq; ++q) {
    const Ws v = quarter_view(w, q);
    const int bq = bb_of_quarter(bb, q);
    if (weighted)
      EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_USTEP, (k_ustep<true>), dim3((unsigned)w.ntu), dim3(NT), 0, s, w.R,
                           (const v4i*)v.Vmf, v.Vr, w.hw, v.Q, w.rowb, w.m_pad, w.n_pad, bq, w.gacc + 4096,
                           w.counters + CNT_GRAM_V, w.ginvV, w.gramV, 0, w.urows, (const int8_t*)nullptr,
                           (long long*)nullptr, (const double*)nullptr, (double*)nullptr, (double*)nullptr,
                           (double*)nullptr, (int*)nullptr, w.m, (unsigned*)nullptr, (int*)nullptr, 1);
    else
      EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_USTEP, (k_ustep<false>), dim3((unsigned)w.ntu), dim3(NT), 0, s, w.R,
                           (const v4i*)v.Vmf, v.Vr, w.hw, v.Q, w.rowb, w.m_pad, w.n_pad, bq, w.gacc + 4096,
                           w.counters + CNT_GRAM_V, w.ginvV, w.gramV, 0, w.urows, (const int8_t*)nullptr,
                           (long long*)nullptr, (const double*)nullptr, (double*)nullptr, (double*)nullptr,
                           (double*)nullptr, (int*)nullptr, w.m, (unsigned*)nullptr, (int*)nullptr, 1);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  e = wide_gram_inverse(w, 1, weighted, bb, s);
  if (e != hipSuccess) return e;
  for (int q = 0; q < nq; ++q) {
    const Ws v = quarter_view(w, q);
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_UTARGET, k_utarget<true>, dim3((unsigned)(w.m_pad / TILE)), dim3(NT), 0,
                         s, (const double*)w.Q, (const double*)(w.ginvVW + (int64_t)q * NQMAX * 4096), v.Z, w.m,
                         w.m_pad, v.tps, v.tpm, v.tpi, nq);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_TERNU, k_tern_u, dim3(BBP * w.nsu), dim3(NT), 0, s, (const double*)v.Z,
                         final ? (const double*)v.Q : nullptr, w.m, w.m_pad, bb_of_quarter(bb, q), tau,
                         (const double*)v.tps, (const double*)v.tpm, (const int*)v.tpi, (int)(w.m_pad / TILE), w.nsu,
                         v.Ut, v.Umf, v.gvec, (unsigned*)nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The raw V^T H V of a wide block into gramVW (the step entry point of the
// joint solve; the factorization leaves it from its last U-step).
hipError_t launch_gram_wide_raw(const Ws& w, int bb, bool weighted, hipStream_t s) {
  return wide_gram_inverse(w, 1, weighted, bb, s);
}

// Joint scales of a wide block (Eq. (4)): [(U^T U) o (V^T H V) + delta I]
// d = g with the raw V^T H V of the last U-step, d into dvec, dF and D_block.
hipError_t launch_scale_wide(const Ws& w, int bb, float* D_block, hipStream_t s) {
  const int nq = nq_of(bb), npairs = nq * (nq + 1) / 2;
  hipLaunchKernelGGL(k_gram_pairs, dim3((unsigned)(npairs * GRAM_PAIR_SLICES)), dim3(NT), 0, s, (const v4i*)w.Umf,
                     w.m_pad, nq, GRAM_PAIR_SLICES, w.gaccW);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_wide_prep, dim3((unsigned)npairs), dim3(NT), 0, s, 2, (const int*)w.gaccW,
                     (const double*)nullptr, w.gramVW, bb, nq, EXTERND_SCALE_GUARD_REL, w.wA0, w.wflag);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const double* S = nullptr;
  e = wide_sweep(w, bb, s, &S);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_wide_scales, dim3(1), dim3(NT), 0, s, S, (const double*)w.gvec, bb, (const int*)w.wflag,
                     w.dvec, w.dF, D_block);
  return hipGetLastError();
}

// Block end of a wide block: joint scales, then per quarter the row-major
// factor copies and the packed outputs (columns c0 + 64 q ..).
hipError_t launch_block_out_wide(const Ws& w, int64_t c0, int bb, int64_t k, uint8_t* Bp, uint8_t* Cp, float* D,
                                 hipStream_t s) {
  hipError_t e = launch_scale_wide(w, bb, D + c0, s);
  if (e != hipSuccess) return e;
  for (int q = 0; q < nq_of(bb); ++q) {
    e = launch_block_out(quarter_view(w, q), c0 + (int64_t)BBP * q, bb_of_quarter(bb, q), k, Bp, Cp, D, s, false,
                         false, false);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// R <- R - sum_q U_q diag(d_q) V_q^T, one deflation launch per quarter (the
// column energies and the residual bound of the last one are the block's).
hipError_t launch_deflate_wide(const Ws& w, int blk, int bb, bool transposes, hipStream_t s, Timer* tm) {
  for (int q = 0; q < nq_of(bb); ++q) {
    const hipError_t e = launch_deflate(quarter_view(w, q), blk, transposes, s, tm, false);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_scale(const Ws& w, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_scale, dim3(1), dim3(NT), 0, s, w.gacc, bb, w.gramV, w.gvec, w.dvec, w.dF, (float*)nullptr);
  return hipGetLastError();
}

hipError_t launch_block_out(const Ws& w, int64_t c0, int bb, int64_t k, uint8_t* Bp, uint8_t* Cp, float* D,
                           hipStream_t s, bool revisit, bool safeguard, bool solve) {
  const unsigned grid = (unsigned)(1 + w.m_pad / TILE + w.n_pad / TILE);
  hipLaunchKernelGGL(k_block_out, dim3(grid), dim3(NT), 0, s, w.gacc, bb, w.gramV, w.gvec, w.dvec, w.dF, D + c0,
                     w.Ut, w.Ur, w.Ub, w.m, w.m_pad, c0, k, Bp, w.Vt, w.Vr, w.n, w.n_pad, Cp,
                     revisit ? (const unsigned*)(w.counters + CNT_DECISION) : nullptr,
                     safeguard ? (const unsigned*)(w.counters + CNT_SG_FIRE) : nullptr, solve ? 1 : 0);
  return hipGetLastError();
}
hipError_t launch_safeguard(const Ws& w, int blk, int bb, float* D_block, hipStream_t s) {
  hipLaunchKernelGGL(k_safeguard, dim3(1), dim3(NT), 0, s, w.gacc, bb, w.gramV, w.gvec, w.dvec, w.dF, D_block,
                     (const float*)w.R, w.n, w.n_pad, (const unsigned long long*)(w.argkey + blk),
                     w.counters + CNT_SG_FIRE, w.counters + CNT_SAFEGUARD);
  return hipGetLastError();
}
hipError_t launch_revisit_load(const Ws& w, const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t c0, int bb,
                               int64_t k, int slot1, int slot2, hipStream_t s) {
  const unsigned grid = (unsigned)(1 + w.m_pad / TILE + w.n_pad / TILE);
  hipLaunchKernelGGL(k_revisit_load, dim3(grid), dim3(NT), 0, s, Bp, Cp, D, c0, bb, k, w.m, w.m_pad, w.n, w.n_pad,
                     w.Ut, w.Ur, w.Ub, w.Umf, w.Vt, w.Vr, w.Vmf, w.dF);
  return hipGetLastError();
}
hipError_t launch_revisit_decide(const Ws& w, int bb, float* D_block, bool weighted, int slot_prev, int slot_added,
                                 hipStream_t s) {
  const double* hist = weighted ? w.fro2w_hist : w.fro2_hist;
  hipLaunchKernelGGL(k_revisit_decide, dim3(1), dim3(NT), 0, s, w.gacc, bb, w.gramV, w.gvec, w.dvec, w.dF, D_block,
                     hist + slot_prev, hist + slot_added, w.counters + CNT_DECISION, w.counters + CNT_ACCEPTED);
  return hipGetLastError();
}

hipError_t launch_deflate(const Ws& w, int blk, bool transposes, hipStream_t s, Timer* tm, bool track) {
  hipError_t e;
  if (transposes) {
    hipLaunchKernelGGL(k_transpose8, dim3((unsigned)(w.m_pad / 32)), dim3(NT), 0, s, w.Ut, w.Ur, w.m_pad, w.Ub);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_transpose8, dim3((unsigned)(w.n_pad / 32)), dim3(NT), 0, s, w.Vt, w.Vr, w.n_pad,
                       (unsigned short*)nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_deflate_slot(w, blk + 1, s, tm, track);
}
hipError_t launch_deflate_slot(const Ws& w, int out_slot, hipStream_t s, Timer* tm, bool track) {
  const unsigned grid = (unsigned)((w.n_pad / TILE) * w.gd);
  if (track)
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_DEFLATE, k_deflate<true>, dim3(grid), dim3(NT), 0, s, w.R, (const v8s*)w.Ub,
                         w.Vr, w.dF, w.colE_part, w.rowb, (const int8_t*)w.Ur, (const double*)w.hwmax, w.m_pad, w.n_pad,
                         w.gd, w.argkey + out_slot, w.n);
  else
    EXTERND_LAUNCH_TIMED(tm, EXTERND_KCLASS_DEFLATE, k_deflate<false>, dim3(grid), dim3(NT), 0, s, w.R,
                         (const v8s*)w.Ub, w.Vr, w.dF, w.colE_part, w.rowb, (const int8_t*)w.Ur, (const double*)w.hwmax,
                         w.m_pad, w.n_pad, w.gd, (unsigned long long*)nullptr, w.n);
  return hipGetLastError();
}

hipError_t launch_load_factor(int8_t* Xt, int8_t* Xr, int8_t* Xmf, const int8_t* X, int64_t len, int64_t len_pad,
                              int bb, hipStream_t s, int ld) {
  hipLaunchKernelGGL(k_load_factor, dim3(grid_for(len_pad * BBP)), dim3(NT), 0, s, Xt, Xr, Xmf, X, len, len_pad, bb,
                     ld > 0 ? ld : bb);
  return hipGetLastError();
}
hipError_t launch_store_factor(int8_t* X, const int8_t* Xt, int64_t len, int64_t len_pad, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_store_factor, dim3(grid_for(len * bb)), dim3(NT), 0, s, X, Xt, len, len_pad, bb);
  return hipGetLastError();
}
hipError_t launch_store_cm(double* X, const double* Xcm, int64_t len, int64_t len_pad, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_store_cm, dim3(grid_for(len * bb)), dim3(NT), 0, s, X, Xcm, len, len_pad, bb);
  return hipGetLastError();
}
hipError_t launch_load_cm(double* Xcm, const double* X, int64_t len, int64_t len_pad, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_load_cm, dim3(grid_for(len_pad * BBP)), dim3(NT), 0, s, Xcm, X, len, len_pad, bb);
  return hipGetLastError();
}

hipError_t launch_vweight(const Ws& w, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_vweight, dim3((unsigned)(w.n_pad / TILE), (unsigned)nq_of(bb)), dim3(128), 0, s,
                     (const v4i*)w.Vmf, (const int8_t*)w.hdig, w.n_pad, w.Wmf, (int64_t)BMAX * w.n_pad);
  return hipGetLastError();
}
hipError_t launch_gram_only(const Ws& w, int bb, bool weighted, hipStream_t s) {
  if (weighted) {
    hipLaunchKernelGGL(k_gram_vw, dim3(NSIDE_GRAM), dim3(NT), 0, s, (const v4i*)w.Vmf, (const int8_t*)w.Wmf,
                       w.n_pad, w.gacc64, (const double*)w.hwmax, w.counters + CNT_GRAM_V, w.gramV);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_gram_v, dim3(NSIDE_INT), dim3(NT), 0, s, (const v4i*)w.Vmf, w.n_pad, bb, w.gparti,
                     w.counters + CNT_GRAM_V, w.ginvV, w.gramV);
  return hipGetLastError();
}
hipError_t launch_gram_acc(const Ws& w, int which, hipStream_t s) {
  const v4i* X = (const v4i*)(which ? w.Vmf : w.Umf);
  hipLaunchKernelGGL(k_gram_acc, dim3(NSIDE_GRAM), dim3(NT), 0, s, X, which ? w.n_pad : w.m_pad, w.gacc + 4096 * which);
  return hipGetLastError();
}

hipError_t launch_gvec(const Ws& w, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_gvec, dim3(bb > BBP ? BMAX : BBP), dim3(NT), 0, s, w.Ut, w.Q, w.m, w.m_pad, bb, w.gvec);
  return hipGetLastError();
}
hipError_t launch_set_scales(const Ws& w, const double* d, int bb, hipStream_t s) {
  hipLaunchKernelGGL(k_set_scales, dim3(1), dim3(BMAX), 0, s, d, bb, w.dvec, w.dF);
  return hipGetLastError();
}

}  // namespace externd
