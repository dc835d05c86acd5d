// Static min-max calibration and symmetrization factors (OutlierTune
// Sec. 3.2: z = (max + min) / 2 per activation channel; App. A: min-max
// calibration of the activation scale, offline).
//
// Device layout of the running state: minmax[0, K) = per-channel minima,
// minmax[K, 2K) = maxima, both fp32 (the inputs are fp16, so exact).
// Minimum and maximum are order-independent, so the state is the same
// whatever the launch shape and however the rows are split across calls.
#include <math.h>

#include "ot_common.h"

namespace ot {
namespace detail {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = 64;

// Float atomics through the integer order of IEEE bit patterns: for
// non-negative floats the signed-int order is the float order, for negative
// floats the unsigned order is the reverse of it.  -0 must be mapped to +0
// by the caller.
__device__ inline void atomic_min_f32(float *addr, float v) {
  if (v >= 0.0f)
    atomicMin(reinterpret_cast<int *>(addr), __float_as_int(v));
  else
    atomicMax(reinterpret_cast<unsigned int *>(addr), __float_as_uint(v));
}

__device__ inline void atomic_max_f32(float *addr, float v) {
  if (v >= 0.0f)
    atomicMax(reinterpret_cast<int *>(addr), __float_as_int(v));
  else
    atomicMin(reinterpret_cast<unsigned int *>(addr), __float_as_uint(v));
}

// A quiet NaN whose bit pattern, read as a signed int, is above every finite
// float and +inf: once stored into a maximum slot no later update replaces it.
constexpr int kPoison = 0x7FC00000;

__global__ __launch_bounds__(kThreads) void calib_reset_kernel(float *minmax, int64_t K) {
  const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (k < K) {
    minmax[k] = INFINITY;
    minmax[K + k] = -INFINITY;
  }
}

// grid.x: channel blocks of kThreads channels, grid.y: row blocks (strided
// when there are more than 4096).  Each thread owns one channel and scans
// blocks of kRowsPerBlock rows (coalesced: a wave
// reads 64 consecutive fp16 of a row), then publishes one atomic min and max.
__global__ __launch_bounds__(kThreads) void calib_minmax_kernel(const uint16_t *__restrict__ x,
                                                                int64_t rows, int64_t K,
                                                                float *__restrict__ minmax) {
  const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (k >= K) return;
  float lo = INFINITY, hi = -INFINITY;
  bool bad = false;
  for (int64_t r0 = (int64_t)blockIdx.y * kRowsPerBlock; r0 < rows;
       r0 += (int64_t)gridDim.y * kRowsPerBlock) {
    const int64_t r1 = r0 + kRowsPerBlock < rows ? r0 + kRowsPerBlock : rows;
    for (int64_t r = r0; r < r1; ++r) {
      const float v = half_bits_to_float(x[r * K + k]) + 0.0f;  // -0 -> +0
      bad |= !isfinite(v);
      lo = fminf(lo, v);
      hi = fmaxf(hi, v);
    }
  }
  if (bad) {
    atomicMax(reinterpret_cast<int *>(&minmax[K + k]), kPoison);
    return;
  }
  atomic_min_f32(&minmax[k], lo);
  atomic_max_f32(&minmax[K + k], hi);
}

// z, s, inv_s from the state, in fp64 with one rounding to fp32 each.
// symmetrize != 0: Sec. 3.2's z = (hi + lo) / 2, s = ((hi - lo) / 2) / qa.
// symmetrize == 0 (the ablation of Sec. 4.4): z = 0, s = max(|lo|, |hi|) / qa.
__global__ __launch_bounds__(kThreads) void calib_finalize_kernel(const float *__restrict__ minmax,
                                                                  int64_t K, int qa,
                                                                  int symmetrize,
                                                                  float *__restrict__ z,
                                                                  float *__restrict__ s,
                                                                  float *__restrict__ inv_s) {
  const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (k >= K) return;
  const double lo = (double)minmax[k];
  const double hi = (double)minmax[K + k];
  // exact: both are fp16 values
  const double half = symmetrize ? (hi - lo) / 2.0 : fmax(fabs(lo), fabs(hi));
  float sk = (float)(half / (double)qa);
  if (sk == 0.0f) sk = 1.0f;
  z[k] = symmetrize ? (float)((hi + lo) / 2.0) : 0.0f;
  s[k] = sk;
  inv_s[k] = (float)(1.0 / (double)sk);
}

unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace detail

using namespace detail;

hipError_t launch_calib_reset(float *minmax, int64_t K, hipStream_t st) {
  calib_reset_kernel<<<blocks_for(K, kThreads), kThreads, 0, st>>>(minmax, K);
  return hipGetLastError();
}

hipError_t launch_calib_minmax(const uint16_t *x, int64_t rows, int64_t K, float *minmax,
                               hipStream_t st) {
  unsigned gy = blocks_for(rows, kRowsPerBlock);
  dim3 grid(blocks_for(K, kThreads), gy < 4096 ? gy : 4096);
  calib_minmax_kernel<<<grid, kThreads, 0, st>>>(x, rows, K, minmax);
  return hipGetLastError();
}

hipError_t launch_calib_finalize(const float *minmax, int64_t K, int qa, int symmetrize, float *z,
                                 float *s, float *inv_s, hipStream_t st) {
  calib_finalize_kernel<<<blocks_for(K, kThreads), kThreads, 0, st>>>(minmax, K, qa, symmetrize, z,
                                                                      s, inv_s);
  return hipGetLastError();
}

}  // namespace ot
