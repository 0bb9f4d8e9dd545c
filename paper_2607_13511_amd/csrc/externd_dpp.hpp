// Wavefront reductions on DPP (data-parallel primitives: a VALU operand
// read from another lane of the same row of 16, or broadcast across rows),
// shared by the block path and the one-launch path.  Results land in lane
// 63 of the wave (whole-wave reductions) or lane 15 of each row (row
// reductions); the combination order is fixed, so results are
// deterministic.
#pragma once

#include <hip/hip_runtime.h>
#include <limits.h>

namespace externd {

// DPP controls (row = 16 lanes): shift right by 1, 2, 4, 8 within a row;
// broadcast lane 15 of each row to the next row; broadcast lane 31 to the
// upper half; quad permutations swapping neighbours / pairs.
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114, DPP_ROW_SHR8 = 0x118;
constexpr int DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;
constexpr int DPP_QUAD_XOR1 = 0xB1, DPP_QUAD_XOR2 = 0x4E;

// One DPP move of a 64-bit value; lanes whose source lies outside the
// pattern, or whose row ROWMASK excludes, receive `old`.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ double dpp_f64(double old, double src) {
  const unsigned long long o = (unsigned long long)__double_as_longlong(old);
  const unsigned long long v = (unsigned long long)__double_as_longlong(src);
  const int lo = __builtin_amdgcn_update_dpp((int)(unsigned)o, (int)(unsigned)v, CTRL, ROWMASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(unsigned)(o >> 32), (int)(unsigned)(v >> 32), CTRL, ROWMASK, 0xF,
                                             false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// (value, index) pairs: larger value first, then smaller index.
__device__ __forceinline__ void dpp_argmax_combine(double& v, int& i, double ov, int oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

template <int CTRL, int ROWMASK>
__device__ __forceinline__ void dpp_sum_step(double& x) {
  x += dpp_f64<CTRL, ROWMASK>(0.0, x);
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ void dpp_argmax_step(double& v, int& i) {
  const double ov = dpp_f64<CTRL, ROWMASK>(-1.0, v);
  const int oi = __builtin_amdgcn_update_dpp(INT_MAX, i, CTRL, ROWMASK, 0xF, false);
  dpp_argmax_combine(v, i, ov, oi);
}
// Wave sum; lane 63 receives the total (rows by shifts, then across rows).
__device__ __forceinline__ void wave_sum63(double& x) {
  dpp_sum_step<DPP_ROW_SHR1, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR2, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR4, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR8, 0xF>(x);
  dpp_sum_step<DPP_ROW_BCAST15, 0xA>(x);
  dpp_sum_step<DPP_ROW_BCAST31, 0xC>(x);
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ void dpp_max_step(double& x) {
  x = fmax(x, dpp_f64<CTRL, ROWMASK>(-1.0, x));
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ void dpp_imin_step(int& x) {
  x = min(x, __builtin_amdgcn_update_dpp(INT_MAX, x, CTRL, ROWMASK, 0xF, false));
}
// Wave max of values >= 0 (identity -1); lane 63.
__device__ __forceinline__ void wave_max63(double& x) {
  dpp_max_step<DPP_ROW_SHR1, 0xF>(x);
  dpp_max_step<DPP_ROW_SHR2, 0xF>(x);
  dpp_max_step<DPP_ROW_SHR4, 0xF>(x);
  dpp_max_step<DPP_ROW_SHR8, 0xF>(x);
  dpp_max_step<DPP_ROW_BCAST15, 0xA>(x);
  dpp_max_step<DPP_ROW_BCAST31, 0xC>(x);
}
// Wave minimum of ints (identity INT_MAX); lane 63.
__device__ __forceinline__ void wave_imin63(int& x) {
  dpp_imin_step<DPP_ROW_SHR1, 0xF>(x);
  dpp_imin_step<DPP_ROW_SHR2, 0xF>(x);
  dpp_imin_step<DPP_ROW_SHR4, 0xF>(x);
  dpp_imin_step<DPP_ROW_SHR8, 0xF>(x);
  dpp_imin_step<DPP_ROW_BCAST15, 0xA>(x);
  dpp_imin_step<DPP_ROW_BCAST31, 0xC>(x);
}
// Wave (max, first index); values >= 0, identity (-1, INT_MAX); lane 63.
__device__ __forceinline__ void wave_argmax63(double& v, int& i) {
  dpp_argmax_step<DPP_ROW_SHR1, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR2, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR4, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR8, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_BCAST15, 0xA>(v, i);
  dpp_argmax_step<DPP_ROW_BCAST31, 0xC>(v, i);
}

// Row (16-lane) reductions; lane 15 of each row receives the result.
__device__ __forceinline__ void row_sum15(double& x) {
  dpp_sum_step<DPP_ROW_SHR1, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR2, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR4, 0xF>(x);
  dpp_sum_step<DPP_ROW_SHR8, 0xF>(x);
}
__device__ __forceinline__ void row_argmax15(double& v, int& i) {
  dpp_argmax_step<DPP_ROW_SHR1, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR2, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR4, 0xF>(v, i);
  dpp_argmax_step<DPP_ROW_SHR8, 0xF>(v, i);
}

}  // namespace externd
