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
static ApplyLayout apply_layout(int64_t m, int64_t n, int64_t k, int nb) {
  ApplyLayout L{};
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

static hipError_t run_apply_kernels(const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t m, int64_t n,
                                    int64_t k, const float* X, int nb, float* Y, char* ws, hipStream_t s) {
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
