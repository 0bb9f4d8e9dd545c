// Inference with a factorization: Y = X (B diag(D) C)^T, i.e. for each input
// vector x the product y = B (diag(D) (C x)) (paper, Sec. 2.6 cost model),
// computed directly on the packed 2-bit trits written by externd_factorize.
//
// Trit code (include/externd.h): 00 -> 0, 01 -> +1, 11 -> -1, element j of a
// row in byte j >> 2 at bits 2 (j & 3).
//
// Two paths, chosen by the batch size nb.
//
// One vector (a matrix-vector product), k_apply_vec_c then k_apply_vec_b:
// fp32 FMA on the vector ALUs.  The signed 2-bit field extract (v_bfe_i32)
// of a code is the trit itself (01 -> 1, 11 -> -1, 00 -> 0).  A workgroup
// takes VEC_RPW consecutive rows; lane l of wave w takes byte
// p = 64 w + l + 256 i of the rows (elements 4p .. 4p+3), so the vector
// entries a wave needs are contiguous and each loaded slice serves all
// VEC_RPW rows from registers.  Each wave sums its lanes with a fixed
// shuffle tree and the four waves are added in wave order through LDS.  For
// one vector the matrix-core path below spends more on decoding trits and
// staging than this path spends on arithmetic; from two vectors on it is
// the faster one.
//
// Two or more vectors: both products run on bf16 MFMA with fp32 accumulation and
// exact operands:
//  * the trits are exact in bf16; a 16-entry table in LDS turns each 4-bit
//    pair of codes into two bf16 trits (one dword); the 16 entries lie in
//    16 different banks, so the lookups never conflict;
//  * every fp32 vector entry v is split exactly into three bf16 parts,
//    v = hi + mid + lo (each part the truncation of what the previous ones
//    leave: 8 + 8 + 8 significand bits, all of the same sign), so every
//    product trit x part is exact and only the fp32 sums round.  Column
//    3 b + p of the MFMA's B operand holds part p of vector b, and an
//    output's three part sums are added in a fixed order.
// Two MFMA shapes: for 3 nb <= 16, v_mfma_f32_16x16x32_bf16 (16 columns,
// four 16-row tiles per wave); otherwise v_mfma_f32_32x32x16_bf16 (32
// columns, two 32-row tiles).  The narrower shape halves the matrix-core
// work of the small batches.
//
// A product (k_apply_prod) splits its rows into groups of 256 (64 per wave)
// and its contracted dimension into KS slices of SL 128-component chunks;
// a workgroup takes one (row group, slice).  It first issues every trit
// load of its waves (one memory latency for the whole slice), stages the
// slice's vector parts in LDS (the C side splits x on the fly, the B side
// copies the parts of T), then runs the products with the B operand read
// from LDS; columns past 3 nb read a zero row.  Each wave adds the parts of
// its 64 rows and writes one partial sum per (slice, row, vector).  Small
// launches then add the slices in slice order: k_apply_tsum forms
// T = diag(D) (sum) and its parts, k_apply_ysum forms Y.  With a single
// slice the product writes its result directly.  No workgroup depends on
// another within a launch; every result is deterministic.
//
// K order inside a chunk: a 128-component chunk of a row is 32 packed
// bytes.  With the 16-row shape, lane (row r, group g = lane / 16) loads
// bytes 8 g .. 8 g + 7 (components 32 g .. 32 g + 31) and feeds K step s
// (0..3) with components 32 g + 8 s + e, e < 8, as the A operand's K index
// 8 g + e; with the 32-row shape, lane (row r, half g = lane / 32) loads
// bytes 16 g .. 16 g + 15 and feeds K step s (0..7) with components
// 64 g + 8 s + e as K index 8 g + e.  The B operand's lane (column, g)
// holds the same components of the vectors at the same K index, so the sum
// runs over every component exactly once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "externd.h"
#include "externd_internal.hpp"

namespace externd {

typedef __bf16 v8bf_a __attribute__((ext_vector_type(8)));
typedef float v16f_a __attribute__((ext_vector_type(16)));
typedef float v4f_a __attribute__((ext_vector_type(4)));
typedef unsigned v4u_a __attribute__((ext_vector_type(4)));
typedef unsigned v2u_a __attribute__((ext_vector_type(2)));

constexpr int NT_AP = 256;                // threads per workgroup (4 waves)
constexpr int AP_WROWS = 64;              // rows per wave
constexpr int AP_GROUP = 4 * AP_WROWS;    // rows per workgroup
constexpr int AP_CHUNK = 128;             // components per 32-byte row chunk
constexpr int AP_SLMAX = 4;               // chunks per slice at most
constexpr int AP_VEC_MAX = 1;             // batches up to this size take the vector-ALU path
constexpr int VEC_RPW = 8;                // vector-ALU path: rows per workgroup
constexpr int AP_COLS = 3 * EXTERND_APPLY_MAX_BATCH;  // vector-part columns at most

// The two MFMA shapes (TM = rows of a tile).
template <int TM>
struct Shape {
  static constexpr int tiles = AP_WROWS / TM;       // tiles per wave
  static constexpr int cols = TM;                   // MFMA columns
  static constexpr int steps = TM == 16 ? 4 : 8;    // K steps per chunk
  static constexpr int bytes = TM == 16 ? 8 : 16;   // trit bytes per lane and chunk
  typedef typename std::conditional<TM == 16, v2u_a, v4u_a>::type word;
  typedef typename std::conditional<TM == 16, v4f_a, v16f_a>::type accum;
};

__device__ __forceinline__ unsigned short bf16_trunc(float x) { return (unsigned short)(__float_as_uint(x) >> 16); }
__device__ __forceinline__ float bf16_val(unsigned short b) { return __uint_as_float((unsigned)b << 16); }

// Part p of v = hi + mid + lo (exact for normal fp32 v).
__device__ __forceinline__ unsigned short bf16_part(float v, int p) {
  const unsigned short hi = bf16_trunc(v);
  const float r1 = v - bf16_val(hi);
  const unsigned short mi = bf16_trunc(r1);
  const float r2 = r1 - bf16_val(mi);
  return p == 0 ? hi : (p == 1 ? mi : bf16_trunc(r2));
}

// bf16 of a trit code (00 -> 0, 01 -> +1, 11 -> -1; 10 is never written).
__device__ __forceinline__ unsigned tritcode_bf16(unsigned c) { return c == 1u ? 0x3F80u : (c == 3u ? 0xBF80u : 0u); }

// One trit-matrix x vectors product.  P: rows x rb packed bytes over nch
// chunks (the contracted length rounded up to AP_CHUNK); KS slices of SL
// chunks.  C side: the vectors are X (nb x len fp32, split on the fly);
// B side: the parts VS[(3 b + p) * vstride + c] of T.
struct ProdArgs {
  const uint8_t* P;
  int64_t rows, rb, nch;
  int nb, KS;
  const float* X;             // C side
  int64_t len;                // C side: length of the vectors (n)
  const unsigned short* VS;   // B side
  int64_t vstride;            // B side: kp
  float* part;                // KS > 1: part[(slice * prow + row) * nb + b]
  int64_t prow;               // rows rounded up to AP_GROUP
  // KS == 1, C side: T = diag(D) (C X^T) into parts TS[(3 b + p) * tstride + c] (zero for rows..tstride)
  const float* D;
  unsigned short* TS;
  int64_t tstride;
  // KS == 1, B side: Y[b * rows + i]
  float* Y;
};

// The parts of T_c = D_c v (zero past the real rows).
__device__ __forceinline__ void store_t(const float* D, unsigned short* TS, int64_t tstride, int64_t rows, int64_t c,
                                        int b, float v) {
  const float t = c < rows ? D[c] * v : 0.0f;
#pragma unroll
  for (int p = 0; p < 3; ++p) TS[(int64_t)(3 * b + p) * tstride + c] = bf16_part(t, p);
}

// grid: ceil(rows / AP_GROUP) row groups x KS slices, the slice fastest.
// AL: whole-word trit loads (rows of a multiple of the word's bytes, aligned
// base).
template <bool AL, bool CSIDE, int TM, int SL>
__global__ __launch_bounds__(NT_AP) void k_apply_prod(ProdArgs a) {
  typedef Shape<TM> S;
  // LDS: the staged vector parts (rows of SL chunks + 16 bytes; row
  // AP_COLS holds zeros) until the products are done, then the waves'
  // tiles.
  constexpr int VSTR = SL * AP_CHUNK + 8;
  constexpr int VS_BYTES = (AP_COLS + 1) * VSTR * 2;
  constexpr int SM_BYTES = 4 * AP_WROWS * (S::cols + 1) * 4;
  __shared__ unsigned lut[16];
  __shared__ __attribute__((aligned(16))) unsigned char lds[VS_BYTES > SM_BYTES ? VS_BYTES : SM_BYTES];
  unsigned short (*vs)[VSTR] = (unsigned short (*)[VSTR])lds;
  float (*sm)[AP_WROWS][S::cols + 1] = (float (*)[AP_WROWS][S::cols + 1])lds;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane % TM, g = lane / TM;
  const int rgrp = (int)(blockIdx.x / a.KS), ks = (int)(blockIdx.x % a.KS);
  const int64_t row0 = (int64_t)rgrp * AP_GROUP + w * AP_WROWS;
  const int64_t ch0 = (int64_t)ks * SL;
  const int ncol = 3 * a.nb;
  const int SLC = SL * AP_CHUNK;

  // 1. The vector loads of the staging (issued first: a wait for them does
  //    not wait for the trit loads issued after them).
  constexpr int XQ = (SL * AP_CHUNK + NT_AP - 1) / NT_AP;  // C side: components per thread and vector
  float xv[CSIDE ? XQ * EXTERND_APPLY_MAX_BATCH : 1];
  constexpr int VQ = (AP_COLS * SL * AP_CHUNK / 8 + NT_AP - 1) / NT_AP;  // B side: 16-byte pieces per thread
  v4u_a tv[CSIDE ? 1 : VQ];
  if constexpr (CSIDE) {
#pragma unroll
    for (int b = 0; b < EXTERND_APPLY_MAX_BATCH; ++b)
#pragma unroll
      for (int q = 0; q < XQ; ++q) {
        const int j = threadIdx.x + q * NT_AP;
        const int64_t c = ch0 * AP_CHUNK + j;
        xv[b * XQ + q] = (b < a.nb && j < SLC && c < a.len) ? a.X[(int64_t)b * a.len + c] : 0.0f;
      }
  } else {
#pragma unroll
    for (int q = 0; q < VQ; ++q) {
      const int e = threadIdx.x + q * NT_AP;  // piece: column e / (SLC / 8), offset 8 (e % (SLC / 8))
      const int col = e / (SLC / 8), off = 8 * (e % (SLC / 8));
      const int64_t c = ch0 * AP_CHUNK + off;
      v4u_a v = {0u, 0u, 0u, 0u};
      if (col < ncol && c < a.vstride) v = *(const v4u_a*)(a.VS + (int64_t)col * a.vstride + c);
      tv[q] = v;
    }
  }

  // 2. Every trit load of the wave's slice.
  typename S::word wd[SL][S::tiles];
#pragma unroll
  for (int j = 0; j < SL; ++j) {
    const int64_t ch = ch0 + j;
    const int64_t b0 = (ch < a.nch ? ch : 0) * (AP_CHUNK / 4) + S::bytes * g;
    const bool ok = ch < a.nch && b0 < a.rb;
#pragma unroll
    for (int t = 0; t < S::tiles; ++t) {
      int64_t row = row0 + TM * t + lr;
      row = row < a.rows ? row : a.rows - 1;
      if (AL) {
        // out of range: the row's first bytes, against zero vector parts
        wd[j][t] = *(const typename S::word*)(a.P + row * a.rb + (ok ? b0 : 0));
      } else {
        unsigned u[4] = {0u, 0u, 0u, 0u};
        if (ok)
          for (int q = 0; q < S::bytes; ++q)
            if (b0 + q < a.rb) u[q >> 2] |= (unsigned)a.P[row * a.rb + b0 + q] << (8 * (q & 3));
        typename S::word v;
#pragma unroll
        for (int q = 0; q < S::bytes / 4; ++q) v[q] = u[q];
        wd[j][t] = v;
      }
    }
  }

  // 3. The table, the zero row and the slice's vector parts into LDS
  //    (zero past the vectors' length).
  if (threadIdx.x < 16) lut[threadIdx.x] = tritcode_bf16(threadIdx.x & 3u) | (tritcode_bf16(threadIdx.x >> 2) << 16);
  for (int e = threadIdx.x; e < SLC / 8; e += NT_AP) *(v4u_a*)&vs[AP_COLS][8 * e] = v4u_a{0u, 0u, 0u, 0u};
  if constexpr (CSIDE) {
#pragma unroll
    for (int b = 0; b < EXTERND_APPLY_MAX_BATCH; ++b) {
      if (b >= a.nb) break;
#pragma unroll
      for (int q = 0; q < XQ; ++q) {
        const int j = threadIdx.x + q * NT_AP;
        if (j < SLC) {
#pragma unroll
          for (int p = 0; p < 3; ++p) vs[3 * b + p][j] = bf16_part(xv[b * XQ + q], p);
        }
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < VQ; ++q) {
      const int e = threadIdx.x + q * NT_AP;
      const int col = e / (SLC / 8), off = 8 * (e % (SLC / 8));
      if (col < ncol) *(v4u_a*)&vs[col][off] = tv[q];
    }
  }
  __syncthreads();

  // 4. The products.
  typename S::accum acc[S::tiles];
#pragma unroll
  for (int t = 0; t < S::tiles; ++t) acc[t] = typename S::accum{};
  const unsigned short* vrow = &vs[lr < ncol ? lr : AP_COLS][0];
#pragma unroll
  for (int j = 0; j < SL; ++j) {
#pragma unroll
    for (int s = 0; s < S::steps; ++s) {
      const v4u_a bv = *(const v4u_a*)(vrow + j * AP_CHUNK + 4 * S::bytes * g + 8 * s);
#pragma unroll
      for (int t = 0; t < S::tiles; ++t) {
        const unsigned two = (wd[j][t][s >> 1] >> (16 * (s & 1))) & 0xFFFFu;  // the step's 8 components
        v4u_a av;
        av[0] = lut[two & 15u];
        av[1] = lut[(two >> 4) & 15u];
        av[2] = lut[(two >> 8) & 15u];
        av[3] = lut[two >> 12];
        if constexpr (TM == 16)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf_a, av),
                                                           __builtin_bit_cast(v8bf_a, bv), acc[t], 0, 0, 0);
        else
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf_a, av),
                                                           __builtin_bit_cast(v8bf_a, bv), acc[t], 0, 0, 0);
      }
    }
  }

  __syncthreads();  // every wave is done with the staged parts

  // 5. The wave's tiles into its LDS area (16x16 D: lane l, register i ->
  //    row 4 (l / 16) + i, column l % 16; 32x32 D: register r -> row
  //    8 (r / 4) + 4 (l / 32) + r % 4, column l % 32), then lane = row: the
  //    parts as (hi + mid) + lo.
  if (lr < ncol) {
#pragma unroll
    for (int t = 0; t < S::tiles; ++t) {
      if constexpr (TM == 16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) sm[w][16 * t + 4 * g + i][lr] = acc[t][i];
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) sm[w][32 * t + 8 * (r >> 2) + 4 * g + (r & 3)][lr] = acc[t][r];
      }
    }
  }
  __syncthreads();
  const int64_t row = row0 + lane;
  const float* my = &sm[w][lane][0];
  float v[EXTERND_APPLY_MAX_BATCH];
#pragma unroll
  for (int b = 0; b < EXTERND_APPLY_MAX_BATCH; ++b) v[b] = b < a.nb ? (my[3 * b] + my[3 * b + 1]) + my[3 * b + 2] : 0.0f;
  if (a.KS == 1) {
#pragma unroll
    for (int b = 0; b < EXTERND_APPLY_MAX_BATCH; ++b) {
      if (b >= a.nb) break;
      if (CSIDE) {
        if (row < a.tstride) store_t(a.D, a.TS, a.tstride, a.rows, row, b, v[b]);
      } else if (row < a.rows) {
        a.Y[(int64_t)b * a.rows + row] = v[b];
      }
    }
    return;
  }
  // the slices are added by k_apply_tsum / k_apply_ysum
#pragma unroll
  for (int b = 0; b < EXTERND_APPLY_MAX_BATCH; ++b)
    if (b < a.nb) a.part[((int64_t)ks * a.prow + row) * a.nb + b] = v[b];
}

// sum_q p[q * stride], q < KS, in order; the loads of 8 slices at a time are
// issued together (slices past KS reload the last one and add nothing).
__device__ __forceinline__ float sum_slices(const float* __restrict__ p, int KS, int64_t stride) {
  float s = 0.0f;
  for (int q0 = 0; q0 < KS; q0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(q0 + u < KS ? q0 + u : KS - 1) * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (q0 + u < KS) s += v[u];
  }
  return s;
}

// T from the C side's slices: TS[(3 b + p) * kp + c] = part p of
// D_c sum_s part[(s * prow + c) * nb + b] (slices in order; zero for
// k <= c < kp).  grid: ceil(kp nb / NT_AP).
__global__ __launch_bounds__(NT_AP) void k_apply_tsum(const float* __restrict__ part, int KS, int64_t prow, int nb,
                                                      const float* __restrict__ D, int64_t k, int64_t kp,
                                                      unsigned short* __restrict__ TS) {
  const int64_t e = (int64_t)blockIdx.x * NT_AP + threadIdx.x;
  if (e >= kp * nb) return;
  const int64_t c = e / nb;
  const int b = (int)(e - c * nb);
  store_t(D, TS, kp, k, c, b, sum_slices(part + c * nb + b, KS, prow * nb));
}

// Y from the B side's slices: Y[b * m + i] = sum_s part[(s * prow + i) * nb + b]
// (slices in order).  grid: ceil(m nb / NT_AP).
__global__ __launch_bounds__(NT_AP) void k_apply_ysum(const float* __restrict__ part, int KS, int64_t prow, int nb,
                                                      int64_t m, float* __restrict__ Y) {
  const int64_t e = (int64_t)blockIdx.x * NT_AP + threadIdx.x;
  if (e >= m * nb) return;
  const int64_t i = e / nb;
  const int b = (int)(e - i * nb);
  Y[(int64_t)b * m + i] = sum_slices(part + i * nb + b, KS, prow * nb);
}

// ---- vector-ALU path (nb <= AP_VEC_MAX) ----

__device__ __forceinline__ float trit_of(unsigned byte, int t) {
  // the builtin is declared unsigned; its v_bfe_i32 result is the signed trit
  return (float)(int)__builtin_amdgcn_sbfe((int)byte, 2 * t, 2);
}

// Rows r0 .. r0 + VEC_RPW - 1 of the packed matrix P (rows x len trits)
// times the nb vectors V (V[b * vs + j], j < len), summed over the
// workgroup: dst[(r0 + r) + b * b_stride] = scale[r0 + r] * sum.
template <int NB, bool ALIGNED>
__device__ __forceinline__ void rows_times_vectors(const uint8_t* __restrict__ P, int64_t rows, int64_t len,
                                                   int64_t r0, const float* __restrict__ V, int64_t vs, int nb,
                                                   const float* scale, float* dst, int64_t b_stride) {
  __shared__ float part[4][VEC_RPW * NB];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t rb = (len + 3) >> 2;
  float acc[VEC_RPW][NB];
#pragma unroll
  for (int r = 0; r < VEC_RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.0f;
  for (int64_t p = 64 * w + lane; p < rb; p += NT_AP) {
    unsigned byte[VEC_RPW];
#pragma unroll
    for (int r = 0; r < VEC_RPW; ++r) byte[r] = r0 + r < rows ? P[(r0 + r) * rb + p] : 0u;
    const int64_t j = 4 * p;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b >= nb) continue;
      float v[4];
      if (ALIGNED) {
        const float4 q = *(const float4*)(V + b * vs + j);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = j + t < len ? V[b * vs + j + t] : 0.0f;
      }
#pragma unroll
      for (int r = 0; r < VEC_RPW; ++r)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[r][b] = fmaf(trit_of(byte[r], t), v[t], acc[r][b]);
    }
  }
#pragma unroll
  for (int r = 0; r < VEC_RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) acc[r][b] += __shfl_xor(acc[r][b], o, 64);
      if (lane == 0) part[w][r * NB + b] = acc[r][b];
    }
  __syncthreads();
  if (threadIdx.x < VEC_RPW * NB) {
    const int r = threadIdx.x / NB, b = threadIdx.x % NB;
    if (r0 + r < rows && b < nb) {
      const float v = ((part[0][threadIdx.x] + part[1][threadIdx.x]) + part[2][threadIdx.x]) + part[3][threadIdx.x];
      dst[(r0 + r) + b * b_stride] = (scale ? scale[r0 + r] : 1.0f) * v;
    }
  }
}

// T[b * kq + c] = D[c] sum_j C[c][j] X[b][j] (kq = k rounded up to 4; the
// padding entries are zero: B's padding trits are zero, and 0 times an
// unset float could be NaN).  grid: ceil(k / VEC_RPW).
template <int NB>
__global__ __launch_bounds__(NT_AP) void k_apply_vec_c(const uint8_t* __restrict__ Cp, const float* __restrict__ D,
                                                        int64_t n, int64_t k, int64_t kq,
                                                        const float* __restrict__ X, int nb, float* __restrict__ T) {
  if (blockIdx.x == 0 && threadIdx.x < NB * (kq - k)) {
    const int pad = (int)(kq - k);
    T[(threadIdx.x / pad) * kq + k + threadIdx.x % pad] = 0.0f;
  }
  rows_times_vectors<NB, false>(Cp, k, n, (int64_t)blockIdx.x * VEC_RPW, X, n, nb, D, T, kq);
}

// Y[b * m + i] = sum_c B[i][c] T[b * kq + c].  grid: ceil(m / VEC_RPW).
template <int NB>
__global__ __launch_bounds__(NT_AP) void k_apply_vec_b(const uint8_t* __restrict__ Bp, int64_t m, int64_t k,
                                                        int64_t kq, const float* __restrict__ T, int nb,
                                                        float* __restrict__ Y) {
  rows_times_vectors<NB, true>(Bp, m, k, (int64_t)blockIdx.x * VEC_RPW, T, kq, nb, nullptr, Y, m);
}

// ---- one vector on integer matrix cores (nb = 1, n and k <= GV_MAX_LEN) ----
//
// A product y = P v (P: rows x len packed trits, v: len fp32) as an exact
// integer sum.  v enters as the 48-bit fixed-point vector q = rint(v 2^s),
// one exponent per vector, in six balanced base-256 digit planes
// (q = sum_p 256^p d_p, d_p in [-128, 127]); every fp32 entry within 2^22
// of the largest |v| is exact in it.  The trits enter through bit masks of
// the packed bytes: for trit position i of a byte (bits 2i, 2i + 1), the
// byte & (1 << 2i) is 4^i bit0 and the byte & (2 << 2i) is 2 4^i bit1 (for
// i = 3 the latter reads as the int8 -128), with t = bit0 - 2 bit1.  On
// v_mfma_i32_16x16x64_i8 (A: 16 rows x 64 masked bytes, B: the digit planes
// of the components at trit position i of those bytes in columns 0..5)
// every product and every int32 sum is exact, so per plane
//   sum_c t_c d_p,c = sum_{i<3} (acc_i,0 - acc_i,1) / 4^i + (acc_3,0 + acc_3,1) / 64
// (exact divisions) and y = 2^-s sum_p 256^p (...) in int64.  No table
// lookups and no data-dependent control flow: the decode is eight ANDs per
// 16 packed bytes.
//
// Layout.  A super-step covers 256 components, 64 packed bytes of a row;
// lane (rr = lane % 16, g = lane / 16) of a wave holds the 16 bytes
// [64 ss + 16 g, + 16) of row rr of the wave's 16-row tile, i.e. components
// c = 256 ss + 64 g + 4 e + i (byte e, trit position i).  The digit planes
// of the vector live in LDS as [ss][i][g][p][e] (16 bytes per (ss, i, g, p);
// lane (p, g) reads its B operand as one 16-byte read, the 24 lanes p < 6
// of a super-step position contiguous; lanes p >= 6 read a zero block).
// A workgroup holds GV_TILES tiles of 16 rows and the whole vector; the
// super-steps of a tile are split between GV_KSPLIT waves, whose int32
// plane sums are added through LDS at the end.  Each workgroup covers the
// whole contracted dimension, so no partial sums leave it and no workgroup
// depends on another.
//
// The C side (t = diag(D) C x) converts x itself (every workgroup the same
// arithmetic) and writes t already in digit planes, in the layout above, to
// the workspace; their common exponent comes from a bound every workgroup
// forms identically, |t_c| <= max|D| sum_j |x_j|, so no workgroup waits for
// another's result.  The B side copies those planes into LDS.  A non-finite
// entry of x or D makes every entry of y NaN.
constexpr int GV_TILES = 2;                       // 16-row tiles per workgroup
constexpr int GV_KSPLIT = 4;                      // waves per tile (quarters of the super-steps)
constexpr int GV_NT = 64 * GV_TILES * GV_KSPLIT;  // threads per workgroup
constexpr int GV_ROWS = 16 * GV_TILES;            // rows per workgroup
constexpr int GV_SS = 256;                        // components per super-step
constexpr int GV_PLANES = 6;
constexpr int GV_SSB = 4 * 4 * GV_PLANES * 16;    // digit bytes per super-step (= 6 x 256)
constexpr int GV_MAX_LEN = 10240;                 // longest vector held in LDS
constexpr int GV_MAX_SS = GV_MAX_LEN / GV_SS;
constexpr int GV_NONFINITE = 0x7fffffff;          // exponent word: a non-finite input
static_assert(GV_SSB == GV_PLANES * GV_SS, "digit bytes per super-step");

typedef int v4i_g __attribute__((ext_vector_type(4)));

// Byte offset of the digit of plane p of component c in the [ss][i][g][p][e]
// layout.
__device__ __forceinline__ int64_t gv_digit_offset(int64_t c, int p) {
  const int64_t ss = c >> 8;
  const int g = (int)(c >> 6) & 3, e = (int)(c >> 2) & 15, i = (int)c & 3;
  return ss * GV_SSB + (((i * 4 + g) * GV_PLANES + p) << 4) + e;
}

// Balanced base-256 digits of q, |q| < 2^47: q = sum_{p<6} 256^p d_p with
// d_0..d_4 in [-128, 127] (bytes of q + 0x8080808080 re-centred) and
// d_5 = (q + 0x8080808080) >> 40 in [-128, 127].
__device__ __forceinline__ void gv_digits(long long q, int8_t (&d)[GV_PLANES]) {
  const long long u = q + 0x8080808080ll;
#pragma unroll
  for (int p = 0; p < GV_PLANES - 1; ++p) d[p] = (int8_t)((((unsigned long long)u >> (8 * p)) & 0xFFu) ^ 0x80u);
  d[GV_PLANES - 1] = (int8_t)(u >> 40);
}

// 48-bit fixed point: s = 46 - e for a magnitude bound b < 2^e (every |v| <=
// b gives |v 2^s| < 2^46).
__device__ __forceinline__ int gv_shift(double b) {
  int e = 0;
  if (b > 0.0) frexp(b, &e);
  return 46 - e;
}

// Sum (fp64) and two maxima over the workgroup, the same tree in every
// workgroup: butterfly within each wave, then the waves in order.
// sh: >= 3 x waves.
__device__ __forceinline__ void gv_sum_max2(double& sum, double& m1, double& m2, double* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sum += __shfl_xor(sum, o, 64);
    m1 = fmax(m1, __shfl_xor(m1, o, 64));
    m2 = fmax(m2, __shfl_xor(m2, o, 64));
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh[3 * w] = sum;
    sh[3 * w + 1] = m1;
    sh[3 * w + 2] = m2;
  }
  __syncthreads();
  sum = 0.0;
  m1 = m2 = 0.0;
  for (int q = 0; q < GV_NT / 64; ++q) {
    sum += sh[3 * q];
    m1 = fmax(m1, sh[3 * q + 1]);
    m2 = fmax(m2, sh[3 * q + 2]);
  }
}

// The 16 packed bytes of lane (rr, g) for super-step ss of row `row` (rb
// bytes per row).  ALIGNED: rb and the base are multiples of 16, so a chunk
// lies wholly inside or wholly past the row; a chunk past it is loaded from
// the row's start and zeroed where it is used (gv_tile: masking it here
// would wait for the load).  Else byte loads, zero past the row.
template <bool ALIGNED>
__device__ __forceinline__ v4i_g gv_load(const uint8_t* __restrict__ row, int64_t rb, int64_t ss, int g) {
  const int64_t o = ss * 64 + 16 * g;
  if (ALIGNED) return *(const v4i_g*)(row + (o < rb ? o : 0));
  uint8_t b[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) b[e] = row[o + e < rb ? o + e : 0];
  unsigned w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    w[q] = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[q] |= (o + 4 * q + e < rb ? (unsigned)b[4 * q + e] : 0u) << (8 * e);
  }
  return v4i_g{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

// The wave's share of a tile: super-steps [s0, s1) of row `row` (rows past
// the matrix read its last row; their results are discarded).
struct GvWave {
  const uint8_t* row;
  int s0, s1;
};
__device__ __forceinline__ GvWave gv_wave(const uint8_t* __restrict__ P, int64_t rows, int64_t rb, int nss,
                                          int64_t r0) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int tile = w / GV_KSPLIT, kh = w % GV_KSPLIT;
  const int half = (nss + GV_KSPLIT - 1) / GV_KSPLIT;
  const int64_t rr = r0 + 16 * tile + (lane & 15);
  GvWave v;
  v.row = P + (rr < rows ? rr : rows - 1) * rb;
  v.s0 = kh * half < nss ? kh * half : nss;
  v.s1 = (kh + 1) * half < nss ? (kh + 1) * half : nss;
  return v;
}

// Super-steps per wave at most (the wave's share of the longest vector),
// and the steps of trit loads a wave keeps in flight.
constexpr int GV_NSTEP = (GV_MAX_SS + GV_KSPLIT - 1) / GV_KSPLIT;
constexpr int GV_PF = 6;

// The wave's trit chunk of step j (super-step s0 + j; a step past s1 loads
// super-step s0 again, its result unused).
template <bool ALIGNED>
__device__ __forceinline__ v4i_g gv_step_load(const GvWave& v, int64_t rb, int j) {
  const int g = (threadIdx.x & 63) >> 4;
  return gv_load<ALIGNED>(v.row, rb, v.s0 + j < v.s1 ? v.s0 + j : v.s0, g);
}

// The first GV_PF steps' trit loads (issued before the vector is staged, so
// that they are in flight meanwhile).
template <bool ALIGNED>
__device__ __forceinline__ void gv_prefetch(const GvWave& v, int64_t rb, v4i_g (&buf)[GV_NSTEP]) {
#pragma unroll
  for (int j = 0; j < GV_PF; ++j) buf[j] = gv_step_load<ALIGNED>(v, rb, j);
}

// One wave's int32 plane sums over its super-steps; out[r] = sum over the
// wave's components of t_c d_p,c for tile row 4 g + r and plane
// p = lane % 16 (zero for p >= 6).  dig: the digit planes in LDS; zero16: a
// zeroed 16-byte LDS block; buf: the wave's trit chunks, the first GV_PF
// loaded by gv_prefetch.  Unrolled over GV_NSTEP steps, without branches (a
// loop would carry the loads in flight in registers that its back edge
// copies, and a branch would make the compiler wait for them at its entry):
// step j issues the load of step j + GV_PF before its own work.
template <bool ALIGNED>
__device__ __forceinline__ void gv_tile(const GvWave& v, int64_t rb, v4i_g (&buf)[GV_NSTEP], const uint8_t* dig,
                                        const uint8_t* zero16, int (&out)[4]) {
  const int lane = threadIdx.x & 63, p = lane & 15, g = lane >> 4;
  v4i_g acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i][0] = acc[i][1] = v4i_g{0, 0, 0, 0};
  const int boff = ((g * GV_PLANES + p) << 4);  // lane's 16 bytes within an (ss, i) group of 384
  const uint8_t* bsrc = p < GV_PLANES ? dig + (int64_t)v.s0 * GV_SSB + boff : zero16;
  const int bstep = p < GV_PLANES ? GV_SSB : 0;
#pragma unroll
  for (int j = 0; j < GV_NSTEP; ++j) {
    if (j + GV_PF < GV_NSTEP) buf[j + GV_PF] = gv_step_load<ALIGNED>(v, rb, j + GV_PF);
    // keep the load here: scheduled after the step's MFMAs it would leave
    // the memory system idle meanwhile
    __builtin_amdgcn_sched_barrier(0);
    // no branch: a step past the wave's share (or a chunk past the row)
    // multiplies zero trits, its B operands read at a clamped address
    const int cur = v.s0 + j;
    const bool live = cur < v.s1 && (!ALIGNED || (int64_t)cur * 64 + 16 * g < rb);
    const int jb = cur < v.s1 ? j : 0;
    v4i_g bo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) bo[i] = *(const v4i_g*)(bsrc + jb * bstep + i * (4 * GV_PLANES * 16));
    const v4i_g w = live ? buf[j] : v4i_g{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m0 = 0x01010101 << (2 * i), m1 = 0x02020202 << (2 * i);
      const v4i_g a0 = w & m0, a1 = w & m1;
      acc[i][0] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0, bo[i], acc[i][0], 0, 0, 0);
      acc[i][1] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1, bo[i], acc[i][1], 0, 0, 0);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
    out[r] = ((acc[0][0][r] - acc[0][1][r])) + ((acc[1][0][r] - acc[1][1][r]) >> 2) +
             ((acc[2][0][r] - acc[2][1][r]) >> 4) + ((acc[3][0][r] + acc[3][1][r]) >> 6);
}

// The tile's plane sums of both K halves added and the planes combined into
// int64: for lane l < 16 of the first wave of each tile, the exact
// sum_c t_c q_c of tile row l.
__device__ __forceinline__ long long gv_combine(const int (&out)[4], int (*xch)[64][4]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int r = 0; r < 4; ++r) xch[w][lane][r] = out[r];
  __syncthreads();
  long long y = 0;
  if (w % GV_KSPLIT == 0 && lane < 16) {
    const int g = lane >> 2, r = lane & 3;
#pragma unroll
    for (int p = GV_PLANES - 1; p >= 0; --p) {
      long long sp = 0;
#pragma unroll
      for (int h = 0; h < GV_KSPLIT; ++h) sp += xch[w + h][16 * g + p][r];
      y = y * 256 + sp;
    }
  }
  return y;
}

// C side: T (digit planes of t = diag(D) C x, layout above, 256 nss_t
// components, zero past k) and the exponent word *sT (GV_NONFINITE for a
// non-finite x or D).  grid: ceil(k / GV_ROWS).
constexpr int GV_XPT = (GV_MAX_LEN + GV_NT - 1) / GV_NT;  // vector entries per thread at most (x, D)
template <bool ALIGNED>
__global__ __launch_bounds__(GV_NT) void k_gemv_c(const uint8_t* __restrict__ Cp, const float* __restrict__ D,
                                                  const float* __restrict__ X, int64_t n, int64_t k, int nss_t,
                                                  uint8_t* __restrict__ T, int* __restrict__ sT) {
  __shared__ __attribute__((aligned(16))) uint8_t dig[GV_MAX_SS * GV_SSB];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  __shared__ int xch[GV_NT / 64][64][4];
  __shared__ double sh[3 * (GV_NT / 64)];
  const int tid = threadIdx.x;
  const int nss = (int)((n + GV_SS - 1) / GV_SS);
  const int64_t rb = (n + 3) >> 2;
  const int64_t r0 = (int64_t)blockIdx.x * GV_ROWS;
  // every load of the prologue in one round (component tid + GV_NT j of x
  // and D); clamped indices, masked below
  float xv[GV_XPT], dv[GV_XPT];
#pragma unroll
  for (int j = 0; j < GV_XPT; ++j) {
    const int64_t c = tid + (int64_t)GV_NT * j;
    xv[j] = X[c < n ? c : 0];
    dv[j] = D[c < k ? c : 0];
  }
  // the trit prefetch after them (a wait for x and D then does not wait for it)
  __builtin_amdgcn_sched_barrier(0);
  const GvWave v = gv_wave(Cp, k, rb, nss, r0);
  v4i_g buf[GV_NSTEP];
  gv_prefetch<ALIGNED>(v, rb, buf);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < 4) ((int*)zero16)[tid] = 0;
  // statistics of x and D: the same arithmetic in every workgroup
  double sx = 0.0, mx = 0.0, md = 0.0;
  bool bad = false;
#pragma unroll
  for (int j = 0; j < GV_XPT; ++j) {
    const int64_t c = tid + (int64_t)GV_NT * j;
    const double a = c < n ? fabs((double)xv[j]) : 0.0;
    const double b = c < k ? fabs((double)dv[j]) : 0.0;
    bad |= !(a <= 1.0e300) || !(b <= 1.0e300);
    sx += a;
    mx = fmax(mx, a);
    md = fmax(md, b);
  }
  if (bad) mx = INFINITY;
  gv_sum_max2(sx, mx, md, sh);
  const bool finite = mx < INFINITY;
  const int s_x = gv_shift(mx);
  const int s_t = gv_shift(md * sx);
  // x in digit planes (zero past n)
#pragma unroll
  for (int j = 0; j < GV_XPT; ++j) {
    const int64_t c = tid + (int64_t)GV_NT * j;
    if (c < (int64_t)nss * GV_SS) {
      const float x = (c < n && finite) ? xv[j] : 0.0f;
      int8_t d[GV_PLANES];
      gv_digits((long long)rint(ldexp((double)x, s_x)), d);
#pragma unroll
      for (int p = 0; p < GV_PLANES; ++p) dig[gv_digit_offset(c, p)] = (uint8_t)d[p];
    }
  }
  __syncthreads();
  int out[4];
  gv_tile<ALIGNED>(v, rb, buf, dig, zero16, out);
  const long long y = gv_combine(out, xch);
  const int lane = tid & 63, w = tid >> 6;
  if (w % GV_KSPLIT == 0 && lane < 16) {
    const int64_t c = r0 + 16 * (w / GV_KSPLIT) + lane;
    if (c < (int64_t)nss_t * GV_SS) {
      long long q = 0;
      if (c < k && finite) q = (long long)rint(ldexp((double)y, s_t - s_x) * (double)D[c]);
      int8_t d[GV_PLANES];
      gv_digits(q, d);
#pragma unroll
      for (int p = 0; p < GV_PLANES; ++p) T[gv_digit_offset(c, p)] = (uint8_t)d[p];
    }
  }
  // the padding components past the last workgroup's rows
  if (blockIdx.x == gridDim.x - 1) {
    for (int64_t c = (int64_t)gridDim.x * GV_ROWS + tid; c < (int64_t)nss_t * GV_SS; c += GV_NT)
#pragma unroll
      for (int p = 0; p < GV_PLANES; ++p) T[gv_digit_offset(c, p)] = 0;
  }
  if (blockIdx.x == 0 && tid == 0) *sT = finite ? s_t : GV_NONFINITE;
}

// B side: Y[i] = sum_c B_ic t_c from the digit planes of t.  grid:
// ceil(m / GV_ROWS).
template <bool ALIGNED>
__global__ __launch_bounds__(GV_NT) __attribute__((amdgpu_waves_per_eu(4))) void k_gemv_b(const uint8_t* __restrict__ Bp, const uint8_t* __restrict__ T,
                                                  const int* __restrict__ sT, int64_t m, int64_t k,
                                                  float* __restrict__ Y) {
  __shared__ __attribute__((aligned(16))) uint8_t dig[GV_MAX_SS * GV_SSB];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  __shared__ int xch[GV_NT / 64][64][4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int nss = (int)((k + GV_SS - 1) / GV_SS);
  const int64_t rb = (k + 3) >> 2;
  const int64_t r0 = (int64_t)blockIdx.x * GV_ROWS;
  // the digit planes of t: every load in one round (16 bytes per piece,
  // clamped indices), then the trit prefetch, then the LDS stores (the wait
  // for the pieces leaves the prefetch in flight)
  constexpr int NCP = (GV_MAX_SS * GV_SSB / 16 + GV_NT - 1) / GV_NT;
  const int ncp = nss * GV_SSB / 16;
  v4i_g cp[NCP];
#pragma unroll
  for (int j = 0; j < NCP; ++j) {
    const int e = tid + GV_NT * j;
    cp[j] = ((const v4i_g*)T)[e < ncp ? e : 0];
  }
  const int s_t = *sT;
  __builtin_amdgcn_sched_barrier(0);
  const GvWave v = gv_wave(Bp, m, rb, nss, r0);
  v4i_g buf[GV_NSTEP];
  gv_prefetch<ALIGNED>(v, rb, buf);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < 4) ((int*)zero16)[tid] = 0;
#pragma unroll
  for (int j = 0; j < NCP; ++j) {
    const int e = tid + GV_NT * j;
    if (e < ncp) ((v4i_g*)dig)[e] = cp[j];
  }
  __syncthreads();
  int out[4];
  gv_tile<ALIGNED>(v, rb, buf, dig, zero16, out);
  const long long y = gv_combine(out, xch);
  if (wv % GV_KSPLIT == 0 && lane < 16) {
    const int64_t i = r0 + 16 * (wv / GV_KSPLIT) + lane;
    if (i < m) Y[i] = s_t == GV_NONFINITE ? NAN : (float)ldexp((double)y, -s_t);
  }
}

// ---- matrix-core path ----

// Chunks per slice for nch chunks over nrg row groups: the most (a power of
// two up to AP_SLMAX) that still give every CU a workgroup.
static int slice_chunks(int64_t nch, int64_t nrg) {
  for (int sl = AP_SLMAX; sl > 1; sl /= 2)
    if (nrg * ((nch + sl - 1) / sl) >= 256) return sl;
  return 1;
}

struct ApplyLayout {
  int64_t kp, prow_c, prow_b;
  int sl_c, sl_b, ks_c, ks_b;
  size_t ts, part, total;
};

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace (offsets 256-byte aligned): the parts of T (3 nb columns of
// kp) and the partial sums (shared by the two products, which run one
// after the other).
// One vector with both sides short enough for the vector's digit planes to
// fit in LDS: the integer matrix-core path (k_gemv_c, k_gemv_b).
static bool gemv_fits(int64_t n, int64_t k, int nb) { return nb == 1 && n <= GV_MAX_LEN && k <= GV_MAX_LEN; }

static ApplyLayout apply_layout(int64_t m, int64_t n, int64_t k, int nb) {
  ApplyLayout L{};
  if (gemv_fits(n, k, nb)) {
    // the digit planes of t (256-component super-steps) and the exponent word
    L.ts = al256((size_t)((k + GV_SS - 1) / GV_SS) * GV_SSB);
    L.total = L.ts + 256;
    return L;
  }
  if (nb <= AP_VEC_MAX) {
    // vector-ALU path: T, nb x kq floats (kq = k rounded up to 4)
    L.total = al256(sizeof(float) * (size_t)nb * (size_t)((k + 3) & ~(int64_t)3));
    return L;
  }
  const int64_t nch_c = (n + AP_CHUNK - 1) / AP_CHUNK, nch_b = (k + AP_CHUNK - 1) / AP_CHUNK;
  L.kp = nch_b * AP_CHUNK;
  const int64_t nrg_c = (L.kp + AP_GROUP - 1) / AP_GROUP, nrg_b = (m + AP_GROUP - 1) / AP_GROUP;
  L.prow_c = nrg_c * AP_GROUP;
  L.prow_b = nrg_b * AP_GROUP;
  L.sl_c = slice_chunks(nch_c, nrg_c);
  L.sl_b = slice_chunks(nch_b, nrg_b);
  L.ks_c = (int)((nch_c + L.sl_c - 1) / L.sl_c);
  L.ks_b = (int)((nch_b + L.sl_b - 1) / L.sl_b);
  const size_t part_c = L.ks_c > 1 ? (size_t)L.ks_c * (size_t)L.prow_c * nb : 0;
  const size_t part_b = L.ks_b > 1 ? (size_t)L.ks_b * (size_t)L.prow_b * nb : 0;
  size_t o = 0;
  L.ts = o;
  o += al256(sizeof(unsigned short) * 3 * (size_t)nb * (size_t)L.kp);
  L.part = o;
  o += al256(sizeof(float) * (part_c > part_b ? part_c : part_b));
  L.total = o;
  return L;
}

template <bool AL, bool CSIDE, int TM>
static void launch_prod_sl(const ProdArgs& a, int sl, const dim3& grid, hipStream_t s) {
  if (sl == 4)
    hipLaunchKernelGGL((k_apply_prod<AL, CSIDE, TM, 4>), grid, dim3(NT_AP), 0, s, a);
  else if (sl == 2)
    hipLaunchKernelGGL((k_apply_prod<AL, CSIDE, TM, 2>), grid, dim3(NT_AP), 0, s, a);
  else
    hipLaunchKernelGGL((k_apply_prod<AL, CSIDE, TM, 1>), grid, dim3(NT_AP), 0, s, a);
}

template <bool CSIDE, int TM>
static void launch_prod_tm(const ProdArgs& a, int sl, hipStream_t s) {
  const dim3 grid((unsigned)(((a.rows + AP_GROUP - 1) / AP_GROUP) * a.KS));
  const int wb = Shape<TM>::bytes;
  if (a.rb % wb == 0 && ((uintptr_t)a.P % wb) == 0)
    launch_prod_sl<true, CSIDE, TM>(a, sl, grid, s);
  else
    launch_prod_sl<false, CSIDE, TM>(a, sl, grid, s);
}

template <bool CSIDE>
static void launch_prod(const ProdArgs& a, int sl, hipStream_t s) {
  if (3 * a.nb <= 16)
    launch_prod_tm<CSIDE, 16>(a, sl, s);
  else
    launch_prod_tm<CSIDE, 32>(a, sl, s);
}

template <int NB>
static hipError_t run_vec(const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t m, int64_t n, int64_t k,
                          const float* X, int nb, float* Y, float* T, hipStream_t s) {
  const int64_t kq = (k + 3) & ~(int64_t)3;
  hipLaunchKernelGGL(k_apply_vec_c<NB>, dim3((unsigned)((k + VEC_RPW - 1) / VEC_RPW)), dim3(NT_AP), 0, s, Cp, D, n, k,
                     kq, X, nb, T);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_apply_vec_b<NB>, dim3((unsigned)((m + VEC_RPW - 1) / VEC_RPW)), dim3(NT_AP), 0, s, Bp, m, k,
                     kq, (const float*)T, nb, Y);
  return hipGetLastError();
}

static hipError_t run_gemv(const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t m, int64_t n, int64_t k,
                           const float* X, float* Y, char* ws, hipStream_t s) {
  const ApplyLayout L = apply_layout(m, n, k, 1);
  uint8_t* T = (uint8_t*)ws;
  int* sT = (int*)(ws + L.ts);
  const int nss_t = (int)((k + GV_SS - 1) / GV_SS);
  const int64_t rbc = (n + 3) / 4, rbb = (k + 3) / 4;
  const dim3 gc((unsigned)((k + GV_ROWS - 1) / GV_ROWS)), gb((unsigned)((m + GV_ROWS - 1) / GV_ROWS));
  if (rbc % 16 == 0 && ((uintptr_t)Cp % 16) == 0)
    hipLaunchKernelGGL(k_gemv_c<true>, gc, dim3(GV_NT), 0, s, Cp, D, X, n, k, nss_t, T, sT);
  else
    hipLaunchKernelGGL(k_gemv_c<false>, gc, dim3(GV_NT), 0, s, Cp, D, X, n, k, nss_t, T, sT);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (rbb % 16 == 0 && ((uintptr_t)Bp % 16) == 0)
    hipLaunchKernelGGL(k_gemv_b<true>, gb, dim3(GV_NT), 0, s, Bp, (const uint8_t*)T, (const int*)sT, m, k, Y);
  else
    hipLaunchKernelGGL(k_gemv_b<false>, gb, dim3(GV_NT), 0, s, Bp, (const uint8_t*)T, (const int*)sT, m, k, Y);
  return hipGetLastError();
}

static hipError_t run_apply_kernels(const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t m, int64_t n,
                                    int64_t k, const float* X, int nb, float* Y, char* ws, hipStream_t s) {
  if (gemv_fits(n, k, nb)) return run_gemv(Bp, Cp, D, m, n, k, X, Y, ws, s);
  if (nb <= AP_VEC_MAX) return run_vec<AP_VEC_MAX>(Bp, Cp, D, m, n, k, X, nb, Y, (float*)ws, s);
  const ApplyLayout L = apply_layout(m, n, k, nb);
  unsigned short* TS = (unsigned short*)(ws + L.ts);
  float* part = (float*)(ws + L.part);

  ProdArgs c{};
  c.P = Cp;
  c.rows = k;
  c.rb = (n + 3) / 4;
  c.nch = (n + AP_CHUNK - 1) / AP_CHUNK;
  c.nb = nb;
  c.KS = L.ks_c;
  c.X = X;
  c.len = n;
  c.part = part;
  c.prow = L.prow_c;
  c.D = D;
  c.TS = TS;
  c.tstride = L.kp;  // the row groups cover kp: rows k .. kp - 1 of T are written as zeros
  launch_prod<true>(c, L.sl_c, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (L.ks_c > 1) {
    hipLaunchKernelGGL(k_apply_tsum, dim3((unsigned)((L.kp * nb + NT_AP - 1) / NT_AP)), dim3(NT_AP), 0, s,
                       (const float*)part, L.ks_c, L.prow_c, nb, D, k, L.kp, TS);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  ProdArgs b{};
  b.P = Bp;
  b.rows = m;
  b.rb = (k + 3) / 4;
  b.nch = L.kp / AP_CHUNK;
  b.nb = nb;
  b.KS = L.ks_b;
  b.VS = TS;
  b.vstride = L.kp;
  b.part = part;
  b.prow = L.prow_b;
  b.Y = Y;
  launch_prod<false>(b, L.sl_b, s);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (L.ks_b > 1) {
    hipLaunchKernelGGL(k_apply_ysum, dim3((unsigned)((m * nb + NT_AP - 1) / NT_AP)), dim3(NT_AP), 0, s,
                       (const float*)part, L.ks_b, L.prow_b, nb, m, Y);
    e = hipGetLastError();
  }
  return e;
}

// Allocation-free variant: the workspace lives in a file-scope device array
// of a fixed size.  Each device that runs the code object holds its own copy
// until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns on that device (the array's name in host code
// is a stand-in, not a device address).
static __device__ __align__(256) float scratch[EXTERND_APPLY_NOALLOC_MAX_BYTES / sizeof(float)];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static char* g_scratch_ptr[kMaxDevices];

// The scratch array's device address on the current device, looked up once
// per device with that device current.
static int scratch_on_current_device(char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return EXTERND_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return EXTERND_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return EXTERND_EHIP;
    g_scratch_ptr[dev] = (char*)p;
  }
  *out = g_scratch_ptr[dev];
  return EXTERND_OK;
}

static bool apply_sizes_ok(int64_t m, int64_t n, int64_t k, int32_t nb) {
  return m >= 1 && n >= 1 && k >= 1 && nb >= 1 && nb <= EXTERND_APPLY_MAX_BATCH;
}
static bool apply_sizes_supported(int64_t m, int64_t n, int64_t k) {
  return m <= ((int64_t)1 << 31) && n <= ((int64_t)1 << 31) && k <= ((int64_t)1 << 31);
}

static int check_apply_args(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                            int64_t k, const float* X, int32_t nb, float* Y) {
  if (!B_packed || !C_packed || !D || !X || !Y) return EXTERND_EINVAL;
  if (!apply_sizes_ok(m, n, k, nb)) return EXTERND_EINVAL;
  if (!apply_sizes_supported(m, n, k)) return EXTERND_EUNSUPPORTED;
  return EXTERND_OK;
}

}  // namespace externd

using namespace externd;

extern "C" {

size_t externd_apply_workspace_bytes(int64_t m, int64_t n, int64_t k, int32_t nb) {
  if (!apply_sizes_ok(m, n, k, nb) || !apply_sizes_supported(m, n, k)) return 0;
  return apply_layout(m, n, k, nb).total;
}

int externd_apply(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n, int64_t k,
                  const float* X, int32_t nb, float* Y, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_apply_args(B_packed, C_packed, D, m, n, k, X, nb, Y);
  if (st != EXTERND_OK) return st;
  if (!workspace) return EXTERND_EINVAL;
  const size_t need = externd_apply_workspace_bytes(m, n, k, nb);
  if (need == 0 || workspace_bytes < need || ((uintptr_t)workspace & 255u)) return EXTERND_EWORKSPACE;
  const hipError_t e = run_apply_kernels(B_packed, C_packed, D, m, n, k, X, nb, Y, (char*)workspace,
                                         (hipStream_t)stream);
  return e == hipSuccess ? EXTERND_OK : EXTERND_EHIP;
}

int externd_apply_noalloc(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                          int64_t k, const float* X, int32_t nb, float* Y, void* stream) {
  int st = check_apply_args(B_packed, C_packed, D, m, n, k, X, nb, Y);
  if (st != EXTERND_OK) return st;
  const size_t need = externd_apply_workspace_bytes(m, n, k, nb);
  if (need == 0 || need > (size_t)EXTERND_APPLY_NOALLOC_MAX_BYTES) return EXTERND_ESCRATCH;
  char* ws = nullptr;
  st = scratch_on_current_device(&ws);
  if (st != EXTERND_OK) return st;
  const hipError_t e = run_apply_kernels(B_packed, C_packed, D, m, n, k, X, nb, Y, ws, (hipStream_t)stream);
  return e == hipSuccess ? EXTERND_OK : EXTERND_EHIP;
}

}  // extern "C"
