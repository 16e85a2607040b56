// Wave-wide (64-lane) reductions for the gfx950 kernels, built from DPP row
// operations and readlanes, with no LDS round trips.  Internal to the
// library; every function is inline and wave-uniform in its result.
#pragma once

#include <hip/hip_runtime.h>

namespace precog {
namespace {

// Wave-wide reductions with DPP row operations (no LDS round trips): swap
// neighbours, swap pairs, rotate the row by 4 then by 8, so every lane holds
// its 16-lane row's result; the four rows' results are combined from
// readlanes, so the value is wave-uniform.
template <int kCtrl>
__device__ __forceinline__ int dpp(int v) {
  return __builtin_amdgcn_update_dpp(0, v, kCtrl, 0xf, 0xf, false);
}
template <int kCtrl>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, dpp<kCtrl>(__builtin_bit_cast(int, v)));
}
constexpr int kQuadSwap1 = 0xB1;  // quad_perm [1, 0, 3, 2]
constexpr int kQuadSwap2 = 0x4E;  // quad_perm [2, 3, 0, 1]
constexpr int kRowRor4 = 0x124;
constexpr int kRowRor8 = 0x128;

__device__ __forceinline__ int readlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float readlane(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
  v = op(v, dpp<kQuadSwap1>(v));
  v = op(v, dpp<kQuadSwap2>(v));
  v = op(v, dpp<kRowRor4>(v));
  v = op(v, dpp<kRowRor8>(v));
  return op(op(readlane(v, 0), readlane(v, 16)), op(readlane(v, 32), readlane(v, 48)));
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ int wave_min(int v) {
  return wave_reduce(v, [](int a, int b) { return a < b ? a : b; });
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}
// fp64 sum over the wave in the same pattern (the halves move together)
template <int kCtrl>
__device__ __forceinline__ double dpp_d(double v) {
  const int lo = dpp<kCtrl>(static_cast<int>(__double2loint(v)));
  const int hi = dpp<kCtrl>(static_cast<int>(__double2hiint(v)));
  return __hiloint2double(hi, lo);
}
__device__ __forceinline__ double readlane_d(double v, int l) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(__double2loint(v)), l);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(__double2hiint(v)), l);
  return __hiloint2double(hi, lo);
}
__device__ __forceinline__ double wave_sum_d(double v) {
  v += dpp_d<kQuadSwap1>(v);
  v += dpp_d<kQuadSwap2>(v);
  v += dpp_d<kRowRor4>(v);
  v += dpp_d<kRowRor8>(v);
  return (readlane_d(v, 0) + readlane_d(v, 16)) + (readlane_d(v, 32) + readlane_d(v, 48));
}

}  // namespace
}  // namespace precog
