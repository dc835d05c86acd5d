// LayerNorm fused with symmetrization and per-channel quantization
// (OutlierTune Sec. 3.2: the shift z is taken into the LayerNorm's bias and
// the quantization of Eq. (g) is fused with the LayerNorm that precedes the
// linear, so the fp16 activation never goes to memory).
//
// Per row h [K] (fp16), with c = h_0 and d_k = h_k - c (exact in float64):
//   mean = c + sum_k d_k / K                            float64
//   var  = sum_k d_k^2 / K - (sum_k d_k / K)^2          (population variance)
//   rstd = 1 / sqrt(var + eps)                          float64
//   mu32 = fp32(mean), r32 = fp32(rstd)
// and per element (fp32 operations, round to nearest even, no contraction):
//   y = ((fp32(h_k) - mu32) * r32) * gamma_k + (beta_k - z_k)
//   q = clip(rne(y * inv_s_k), -qa, qa)
//
// The float64 sums run in a fixed order (each thread's chunks in order, a
// fixed butterfly across a wave, waves in order), so the result does not
// change from run to run.  Their relative error, a few units of the 53rd
// bit (times (mean - c)^2 / var for the variance), is far below fp32's 24
// bits: mu32 and r32 are the fp32 roundings of the exact mean and rstd
// except when those lie that close to an fp32 rounding boundary.
//
// HBM-bound: 2 bytes in, 1 byte out per element.  A workgroup of T threads
// takes R rows; thread t owns the 8-channel chunks t, t + T, ... (CPT of
// them, 16-byte coalesced loads) and holds its R x CPT chunks in registers
// from the statistics to the normalize pass (one HBM read).
// The per-channel gamma, beta - z and inv_s (L2-resident) are read once per
// chunk and applied to all R rows.
#include "ot_common.h"

namespace ot {
namespace detail {

__device__ inline float half_lo(uint32_t w) { return half_bits_to_float((uint16_t)w); }
__device__ inline float half_hi(uint32_t w) { return half_bits_to_float((uint16_t)(w >> 16)); }

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <int CPT, int R, int MAXT>
__global__ __launch_bounds__(MAXT) void ln_quantize_kernel(
    const uint16_t *__restrict__ h, int64_t M, int K, const uint16_t *__restrict__ gamma,
    const uint16_t *__restrict__ beta, double eps, float qa, const float *__restrict__ z,
    const float *__restrict__ inv_s, int8_t *__restrict__ Xq) {
  __shared__ double red[2][16][R];  // per wave partial sums of d and d^2
  const int T = blockDim.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, nwaves = T >> 6;
  const int nchunks = K / 8;
  const int64_t row0 = (int64_t)blockIdx.x * R;

  // load the rows (zeros outside the matrix contribute nothing to the sums)
  uint4 x[R][CPT];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int ch = t + j * T;
      const int64_t row = row0 + r;
      x[r][j] = (ch < nchunks && row < M)
                    ? *reinterpret_cast<const uint4 *>(h + row * K + (int64_t)ch * 8)
                    : make_uint4(0, 0, 0, 0);
    }

  // statistics, one pass: sums of d = h - c and d^2 with c = h[row, 0]
  // (d is exact in float64; the shift keeps the variance free of the
  // cancellation that sum h^2 - K mean^2 suffers when |mean| >> std)
  double cs[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row0 + r;
    cs[r] = row < M ? (double)half_bits_to_float(h[row * K]) : 0.0;
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      if (t + j * T >= nchunks) continue;
      const uint32_t w[4] = {x[r][j].x, x[r][j].y, x[r][j].z, x[r][j].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double d0 = (double)half_lo(w[i]) - cs[r];
        const double d1 = (double)half_hi(w[i]) - cs[r];
        s1 += d0;
        s1 += d1;
        s2 = fma(d0, d0, s2);
        s2 = fma(d1, d1, s2);
      }
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    if (lane == 0) {
      red[0][wave][r] = s1;
      red[1][wave][r] = s2;
    }
  }
  __syncthreads();
  float mu32[R], r32[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    double s1 = 0.0, s2 = 0.0;
    for (int w = 0; w < nwaves; ++w) {
      s1 += red[0][w][r];
      s2 += red[1][w][r];
    }
    const double dm = s1 / (double)K;  // mean - c
    const double var = fmax(s2 / (double)K - dm * dm, 0.0);
    mu32[r] = (float)(cs[r] + dm);
    r32[r] = (float)(1.0 / sqrt(var + eps));
  }

  // normalize, shifted affine, quantize; each chunk's gamma,
  // beta - z and inv_s are loaded once and applied to all R rows
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int ch = t + j * T;
    if (ch >= nchunks) continue;
    const uint4 gv = *reinterpret_cast<const uint4 *>(gamma + ch * 8);
    const uint4 bv = *reinterpret_cast<const uint4 *>(beta + ch * 8);
    const float4 z0 = reinterpret_cast<const float4 *>(z + ch * 8)[0];
    const float4 z1 = reinterpret_cast<const float4 *>(z + ch * 8)[1];
    const float4 i0 = reinterpret_cast<const float4 *>(inv_s + ch * 8)[0];
    const float4 i1 = reinterpret_cast<const float4 *>(inv_s + ch * 8)[1];
    const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w}, bw[4] = {bv.x, bv.y, bv.z, bv.w};
    const float zz[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
    const float is[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
    float g[8], c[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      g[e] = (e & 1) ? half_hi(gw[e >> 1]) : half_lo(gw[e >> 1]);
      c[e] = ((e & 1) ? half_hi(bw[e >> 1]) : half_lo(bw[e >> 1])) - zz[e];
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t row = row0 + r;
      if (row >= M) continue;
      const uint32_t w[4] = {x[r][j].x, x[r][j].y, x[r][j].z, x[r][j].w};
      uint32_t code[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float hv = (e & 1) ? half_hi(w[e >> 1]) : half_lo(w[e >> 1]);
        const float d = hv - mu32[r];
        const float n = d * r32[r];
        const float gg = n * g[e];
        const float y = gg + c[e];
        const float u = y * is[e];
        // clamp, then round to nearest even by adding 1.5 * 2^23: for
        // |v| <= 127 the sum's unit is 1, so its low byte is the code
        const float v = __builtin_amdgcn_fmed3f(u, -qa, qa);
        code[e] = __float_as_uint(v + 12582912.0f);
      }
      const uint32_t lo = __builtin_amdgcn_perm(code[1], code[0], 0x0c0c0400u) |
                          __builtin_amdgcn_perm(code[3], code[2], 0x04000c0cu);
      const uint32_t hi = __builtin_amdgcn_perm(code[5], code[4], 0x0c0c0400u) |
                          __builtin_amdgcn_perm(code[7], code[6], 0x04000c0cu);
      *reinterpret_cast<uint2 *>(Xq + row * K + (int64_t)ch * 8) = make_uint2(lo, hi);
    }
  }
}

// MAXT bounds the workgroup (and so frees registers for larger CPT)
template <int CPT, int R, int MAXT = 1024>
hipError_t launch_lnq(const uint16_t *h, int64_t M, int64_t K, const uint16_t *gamma,
                      const uint16_t *beta, float eps, int qa, const float *z, const float *inv_s,
                      int8_t *Xq, hipStream_t st) {
  static_assert(MAXT % 64 == 0 && MAXT <= 1024, "workgroup size");
  const int64_t nchunks = K / 8;
  const int threads = (int)((nchunks + CPT * 64 - 1) / (CPT * 64)) * 64;
  if (threads > MAXT) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((M + R - 1) / R);
  ln_quantize_kernel<CPT, R, MAXT><<<grid, threads, 0, st>>>(h, M, (int)K, gamma, beta,
                                                             (double)eps, (float)qa, z, inv_s, Xq);
  return hipGetLastError();
}

}  // namespace detail

using namespace detail;

hipError_t launch_ln_quantize_act(const uint16_t *h, int64_t M, int64_t K, const uint16_t *gamma,
                                  const uint16_t *beta, float eps, int qa, const float *z,
                                  const float *inv_s, int8_t *Xq, hipStream_t st) {
  // one row per workgroup, 4 chunks of 8 channels per thread up to
  // K = 2048 and 8 beyond (a workgroup of at most 1024 threads covers
  // K = 65536); measured on K = 768 ... 32768 against 2 to 32 chunks per
  // thread, 1 or 2 rows per workgroup and two launch bounds (8 chunks is
  // 10 % faster than 4 at K = 4096 and within 2 % of the best from 3072 to
  // 9216)
  if (K <= 2048) return launch_lnq<4, 1>(h, M, K, gamma, beta, eps, qa, z, inv_s, Xq, st);
  return launch_lnq<8, 1>(h, M, K, gamma, beta, eps, qa, z, inv_s, Xq, st);
}

}  // namespace ot
