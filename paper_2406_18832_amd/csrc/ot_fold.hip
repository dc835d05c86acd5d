// Offline weight and bias transform of OutlierTune:
//   Sec. 3.1 Eq. (e):  W_s[n, k] = W[n, k] * s_k   (activation scale folded
//                      into the weights along the input channels)
//   Eq. (f):           per-output-channel quantization of W_s with a
//                      min-max scale sW_n = max_k |W_s[n, k]| / qw
//   Sec. 3.2 Eq. (g):  compensated bias b'_n = sum_k z_k W[n, k] + b_n
//   Implementation paragraph: done once, before inference.
// and, for the per-token linears (out, fc2; Eq. (c), (h)), the same
// per-output-channel quantization of W itself with the bias b + z.
//
// One workgroup per output channel n.  Pass 1 reduces max |W_s| and the
// bias sum in fp64 (each product is exact in fp64: 24 x 11 significand
// bits); pass 2 writes the codes with a correctly rounded fp64 division.
// The max is order-free, so sW and Wq are exact; the fp64 bias sum is a
// fixed tree, so b' is deterministic but may differ from a sequential sum in
// its last fp32 place.
#include <math.h>

#include "ot_common.h"

namespace ot {
namespace detail {

constexpr int kThreads = 256;

// s == nullptr means s = 1 (no activation scale to fold: the per-token
// path), z == nullptr means z = 0; zres (nullable, [N]) is added to the bias
// (Eq. (h): the shift of a symmetrized residual stream).
__global__ __launch_bounds__(kThreads) void fold_kernel(const uint16_t *__restrict__ W,
                                                        const uint16_t *__restrict__ b,
                                                        const float *__restrict__ zres,
                                                        int64_t K, int qw,
                                                        const float *__restrict__ z,
                                                        const float *__restrict__ s,
                                                        int8_t *__restrict__ Wq,
                                                        float *__restrict__ sW,
                                                        float *__restrict__ bprime) {
  __shared__ double red_max[kThreads];
  __shared__ double red_sum[kThreads];
  __shared__ int red_bad[kThreads];
  __shared__ double row_scale;

  const int64_t n = blockIdx.x;
  const uint16_t *w = W + n * K;
  const int t = threadIdx.x;

  double m = 0.0, acc = 0.0;
  int bad = 0;
  for (int64_t k = t; k < K; k += kThreads) {
    const double wk = (double)half_bits_to_float(w[k]);
    bad |= !isfinite(wk);
    const double ws = s ? (double)s[k] * wk : wk;  // Eq. (e), exact
    m = fmax(m, fabs(ws));
    if (z) acc += (double)z[k] * wk;  // exact product, fp64 sum
  }
  red_max[t] = m;
  red_sum[t] = acc;
  red_bad[t] = bad;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if (t < off) {
      red_max[t] = fmax(red_max[t], red_max[t + off]);
      red_sum[t] = red_sum[t] + red_sum[t + off];
      red_bad[t] |= red_bad[t + off];
    }
    __syncthreads();
  }
  if (t == 0) {
    float sw = (float)(red_max[0] / (double)qw);
    if (sw == 0.0f) sw = 1.0f;
    const double bn = b ? (double)half_bits_to_float(b[n]) : 0.0;
    sW[n] = red_bad[0] ? __builtin_nanf("") : sw;  // the host checks sW
    bprime[n] = (float)(red_sum[0] + bn + (zres ? (double)zres[n] : 0.0));
    row_scale = (double)sw;
  }
  __syncthreads();
  const double sc = row_scale;
  const double lim = (double)qw;
  int8_t *q = Wq + n * K;
  for (int64_t k = t; k < K; k += kThreads) {
    const double wk = (double)half_bits_to_float(w[k]);
    const double ws = s ? (double)s[k] * wk : wk;
    const double r = fmin(fmax(rint(ws / sc), -lim), lim);
    q[k] = (int8_t)(int)r;
  }
}

// Asymmetric weights (the "Int8" setting): per output channel n of W_s,
//   lo, hi = min(min_k W_s, 0), max(max_k W_s, 0);  sW = fp32((hi - lo) / L)
//   zW = clip(rne(-lo / sW), 0, L);  c = clip(rne(W_s / sW) + zW, 0, L)
// with L = 2^bits - 1 (Eq. (a) with a zero point).  Codes and zero point
// are stored shifted by 2^(bits-1) (signed int8 for the matrix cores).
__global__ __launch_bounds__(kThreads) void fold_asym_kernel(
    const uint16_t *__restrict__ W, const uint16_t *__restrict__ b, int64_t K, int w_bits,
    const float *__restrict__ z, const float *__restrict__ s, int8_t *__restrict__ Wq,
    float *__restrict__ sW, int32_t *__restrict__ zW, float *__restrict__ bprime) {
  __shared__ double red_min[kThreads];
  __shared__ double red_max[kThreads];
  __shared__ double red_sum[kThreads];
  __shared__ int red_bad[kThreads];
  __shared__ double row_scale, row_zero;

  const int64_t n = blockIdx.x;
  const uint16_t *w = W + n * K;
  const int t = threadIdx.x;
  const double L = (double)((1 << w_bits) - 1);
  const int half = 1 << (w_bits - 1);

  double lo = 0.0, hi = 0.0, acc = 0.0;  // the range always holds 0
  int bad = 0;
  for (int64_t k = t; k < K; k += kThreads) {
    const double wk = (double)half_bits_to_float(w[k]);
    bad |= !isfinite(wk);
    const double ws = (double)s[k] * wk;  // Eq. (e), exact
    lo = fmin(lo, ws);
    hi = fmax(hi, ws);
    acc += (double)z[k] * wk;  // exact product, fp64 sum
  }
  red_min[t] = lo;
  red_max[t] = hi;
  red_sum[t] = acc;
  red_bad[t] = bad;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if (t < off) {
      red_min[t] = fmin(red_min[t], red_min[t + off]);
      red_max[t] = fmax(red_max[t], red_max[t + off]);
      red_sum[t] = red_sum[t] + red_sum[t + off];
      red_bad[t] |= red_bad[t + off];
    }
    __syncthreads();
  }
  if (t == 0) {
    float sw = (float)((red_max[0] - red_min[0]) / L);
    if (sw == 0.0f) sw = 1.0f;
    const double zp = fmin(fmax(rint(-red_min[0] / (double)sw), 0.0), L);
    const double bn = b ? (double)half_bits_to_float(b[n]) : 0.0;
    sW[n] = red_bad[0] ? __builtin_nanf("") : sw;  // the host checks sW
    zW[n] = (int32_t)zp - half;
    bprime[n] = (float)(red_sum[0] + bn);
    row_scale = (double)sw;
    row_zero = zp;
  }
  __syncthreads();
  const double sc = row_scale, zp = row_zero;
  int8_t *q = Wq + n * K;
  for (int64_t k = t; k < K; k += kThreads) {
    const double ws = (double)s[k] * (double)half_bits_to_float(w[k]);
    const double c = fmin(fmax(rint(ws / sc) + zp, 0.0), L);
    q[k] = (int8_t)((int)c - half);
  }
}

}  // namespace detail

using namespace detail;

hipError_t launch_fold(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K, int qw,
                       const float *z, const float *s, int8_t *Wq, float *sW, float *bprime,
                       hipStream_t st) {
  fold_kernel<<<(unsigned)N, kThreads, 0, st>>>(W, b, nullptr, K, qw, z, s, Wq, sW, bprime);
  return hipGetLastError();
}

// Per-token linear (Eq. (c), (h)): sW_n = max_k |W[n, k]| / qw, codes of W
// itself, b'_n = b_n + zres_n.
hipError_t launch_fold_per_token(const uint16_t *W, const uint16_t *b, const float *zres,
                                 int64_t N, int64_t K, int qw, int8_t *Wq, float *sW,
                                 float *bprime, hipStream_t st) {
  fold_kernel<<<(unsigned)N, kThreads, 0, st>>>(W, b, zres, K, qw, nullptr, nullptr, Wq, sW,
                                                bprime);
  return hipGetLastError();
}

hipError_t launch_fold_asym(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K,
                            int w_bits, const float *z, const float *s, int8_t *Wq, float *sW,
                            int32_t *zW, float *bprime, hipStream_t st) {
  fold_asym_kernel<<<(unsigned)N, kThreads, 0, st>>>(W, b, K, w_bits, z, s, Wq, sW, zW, bprime);
  return hipGetLastError();
}

}  // namespace ot
