// Inference with a factorization: Y = X (B diag(D) C)^T, i.e. for each input
// vector x the product y = B (diag(D) (C x)) (paper, Sec. 2.6 cost model),
// computed directly on the packed 2-bit trits written by externd_factorize.
//
// Trit code (include/externd.h): 00 -> 0, 01 -> +1, 11 -> -1, element j of a
// row in byte j >> 2 at bits 2 (j & 3); the signed 2-bit field extract
// (v_bfe_i32) of a pair is the trit itself (01 -> 1, 11 -> -1, 00 -> 0).
//
// Two launches: k_apply_c forms T = diag(D) C X^T (nb x k, batch-major,
// row stride kp = k rounded up to 4, in the workspace), k_apply_b forms
// Y = B T.  A workgroup takes RPW consecutive rows; lane l of wave w takes
// byte p = 64 w + l + 256 i of the rows (elements 4p .. 4p+3), so the vector
// entries a wave needs are contiguous and each loaded vector slice serves
// all RPW rows from registers.  fp32 accumulation; each wave sums its lanes
// with a fixed shuffle tree and the four waves are added in wave order
// through LDS (deterministic).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "externd.h"
#include "externd_internal.hpp"

namespace externd {

constexpr int NT_APPLY = 256;
constexpr int RPW = 8;  // rows per workgroup

__device__ __forceinline__ float trit_of(unsigned byte, int t) {
  // the builtin is declared unsigned; its v_bfe_i32 result is the signed trit
  return (float)(int)__builtin_amdgcn_sbfe((int)byte, 2 * t, 2);
}

// Rows r0 .. r0+RPW-1 of the packed matrix P (rows x len trits) times the
// nb vectors V (V[b * vs + j], j < len), summed over the workgroup:
// dst[(r0 + r) * row_stride + b * b_stride] = scale[r0 + r] * sum.
template <int NB, bool ALIGNED>
__device__ __forceinline__ void rows_times_vectors(const uint8_t* __restrict__ P, int64_t rows, int64_t len,
                                                   int64_t r0, const float* __restrict__ V, int64_t vs, int nb,
                                                   const float* scale, float* dst, int64_t row_stride,
                                                   int64_t b_stride) {
  __shared__ float part[4][RPW * NB];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t rb = (len + 3) >> 2;
  float acc[RPW][NB];
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.0f;
  for (int64_t p = 64 * w + lane; p < rb; p += NT_APPLY) {
    unsigned byte[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) byte[r] = r0 + r < rows ? P[(r0 + r) * rb + p] : 0u;
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
      for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[r][b] = fmaf(trit_of(byte[r], t), v[t], acc[r][b]);
    }
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) acc[r][b] += __shfl_xor(acc[r][b], o, 64);
      if (lane == 0) part[w][r * NB + b] = acc[r][b];
    }
  __syncthreads();
  if (threadIdx.x < RPW * NB) {
    const int r = threadIdx.x / NB, b = threadIdx.x % NB;
    if (r0 + r < rows && b < nb) {
      const float v = ((part[0][threadIdx.x] + part[1][threadIdx.x]) + part[2][threadIdx.x]) + part[3][threadIdx.x];
      dst[(r0 + r) * row_stride + b * b_stride] = (scale ? scale[r0 + r] : 1.0f) * v;
    }
  }
}

// T[b * kp + c] = D[c] * sum_j C[c][j] X[b][j].  grid: ceil(k / RPW).
template <int NB>
__global__ __launch_bounds__(NT_APPLY) void k_apply_c(const uint8_t* __restrict__ Cp, const float* __restrict__ D,
                                                       int64_t n, int64_t k, int64_t kp, const float* __restrict__ X,
                                                       int nb, float* __restrict__ T) {
  // the padding entries k .. kp-1 of each vector are zero (B's padding
  // trits are zero, and 0 times an unset float could be NaN)
  if (blockIdx.x == 0 && threadIdx.x < NB * (kp - k)) {
    const int pad = (int)(kp - k);
    T[(threadIdx.x / pad) * kp + k + threadIdx.x % pad] = 0.0f;
  }
  const int64_t r0 = (int64_t)blockIdx.x * RPW;
  rows_times_vectors<NB, false>(Cp, k, n, r0, X, n, nb, D, T, 1, kp);
}

// Y[b * m + i] = sum_c B[i][c] T[b * kp + c].  grid: ceil(m / RPW).
template <int NB>
__global__ __launch_bounds__(NT_APPLY) void k_apply_b(const uint8_t* __restrict__ Bp, int64_t m, int64_t k, int64_t kp,
                                                       const float* __restrict__ T, int nb, float* __restrict__ Y) {
  const int64_t r0 = (int64_t)blockIdx.x * RPW;
  rows_times_vectors<NB, true>(Bp, m, k, r0, T, kp, nb, nullptr, Y, 1, m);
}

template <int NB>
static hipError_t launch_apply_nb(const uint8_t* Bp, const uint8_t* Cp, const float* D, int64_t m, int64_t n,
                                  int64_t k, const float* X, int nb, float* Y, float* T, hipStream_t s) {
  const int64_t kp = (k + 3) & ~(int64_t)3;
  const int64_t rows_per_wg = RPW;
  hipLaunchKernelGGL(k_apply_c<NB>, dim3((unsigned)((k + rows_per_wg - 1) / rows_per_wg)), dim3(NT_APPLY), 0, s, Cp,
                     D, n, k, kp, X, nb, T);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_apply_b<NB>, dim3((unsigned)((m + rows_per_wg - 1) / rows_per_wg)), dim3(NT_APPLY), 0, s, Bp,
                     m, k, kp, (const float*)T, nb, Y);
  return hipGetLastError();
}

// The intermediate holds apply_slots(nb) x kp floats.
static int apply_slots(int nb) { return nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : 8; }

// Allocation-free variant: the k x nb intermediate lives in a file-scope
// device array of a fixed size.  Each device that runs the code object holds
// its own copy until the process ends; host code reaches it only through the
// address hipGetSymbolAddress returns on that device (the array's name in
// host code is a stand-in, not a device address).
static __device__ __align__(256) float scratch[EXTERND_APPLY_NOALLOC_MAX_BYTES / sizeof(float)];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static float* g_scratch_ptr[kMaxDevices];

// The scratch array's device address on the current device, looked up once
// per device with that device current.
static int scratch_on_current_device(float** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return EXTERND_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return EXTERND_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return EXTERND_EHIP;
    g_scratch_ptr[dev] = (float*)p;
  }
  *out = g_scratch_ptr[dev];
  return EXTERND_OK;
}

static int check_apply_args(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                            int64_t k, const float* X, int32_t nb, float* Y) {
  if (!B_packed || !C_packed || !D || !X || !Y) return EXTERND_EINVAL;
  if (m < 1 || n < 1 || k < 1 || nb < 1 || nb > EXTERND_APPLY_MAX_BATCH) return EXTERND_EINVAL;
  if (m > ((int64_t)1 << 31) || n > ((int64_t)1 << 31) || k > ((int64_t)1 << 31)) return EXTERND_EUNSUPPORTED;
  return EXTERND_OK;
}

static int run_apply(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                     int64_t k, const float* X, int32_t nb, float* Y, float* T, hipStream_t s) {
  hipError_t e;
  switch (apply_slots(nb)) {
    case 1: e = launch_apply_nb<1>(B_packed, C_packed, D, m, n, k, X, nb, Y, T, s); break;
    case 2: e = launch_apply_nb<2>(B_packed, C_packed, D, m, n, k, X, nb, Y, T, s); break;
    case 4: e = launch_apply_nb<4>(B_packed, C_packed, D, m, n, k, X, nb, Y, T, s); break;
    default: e = launch_apply_nb<8>(B_packed, C_packed, D, m, n, k, X, nb, Y, T, s); break;
  }
  return e == hipSuccess ? EXTERND_OK : EXTERND_EHIP;
}

}  // namespace externd

using namespace externd;

extern "C" {

size_t externd_apply_workspace_bytes(int64_t k, int32_t nb) {
  if (k < 1 || nb < 1 || nb > EXTERND_APPLY_MAX_BATCH || k > ((int64_t)1 << 40)) return 0;
  return sizeof(float) * (size_t)((k + 3) & ~(int64_t)3) * (size_t)apply_slots(nb);
}

int externd_apply(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n, int64_t k,
                  const float* X, int32_t nb, float* Y, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_apply_args(B_packed, C_packed, D, m, n, k, X, nb, Y);
  if (st != EXTERND_OK) return st;
  if (!workspace) return EXTERND_EINVAL;
  const size_t need = externd_apply_workspace_bytes(k, nb);
  if (need == 0 || workspace_bytes < need || ((uintptr_t)workspace & 15u)) return EXTERND_EWORKSPACE;
  return run_apply(B_packed, C_packed, D, m, n, k, X, nb, Y, (float*)workspace, (hipStream_t)stream);
}

int externd_apply_noalloc(const uint8_t* B_packed, const uint8_t* C_packed, const float* D, int64_t m, int64_t n,
                          int64_t k, const float* X, int32_t nb, float* Y, void* stream) {
  int st = check_apply_args(B_packed, C_packed, D, m, n, k, X, nb, Y);
  if (st != EXTERND_OK) return st;
  const size_t need = externd_apply_workspace_bytes(k, nb);
  if (need == 0 || need > (size_t)EXTERND_APPLY_NOALLOC_MAX_BYTES) return EXTERND_ESCRATCH;
  float* T = nullptr;
  st = scratch_on_current_device(&T);
  if (st != EXTERND_OK) return st;
  return run_apply(B_packed, C_packed, D, m, n, k, X, nb, Y, T, (hipStream_t)stream);
}

}  // extern "C"
