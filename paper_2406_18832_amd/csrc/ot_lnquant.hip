// LayerNorm fused with symmetrization and per-channel quantization
// (OutlierTune Sec. 3.2: the shift z is taken into the LayerNorm's bias and
// the quantization of Eq. (g) is fused with the LayerNorm that precedes the
// linear, so the fp16 activation never goes to memory).
//
// Row statistics, exactly as defined: every fp16 value is an integer
// multiple of 2^-24, so a_k = h_k 2^24 is an integer (|a_k| < 2^40) and the
// sums S1 = sum a_k and S2 = sum a_k^2 are exact integers.  Then, each step
// rounded to nearest in float64,
//   mean = fl(fl(S1) / K) 2^-24
//   var  = fl(fl(K S2 - S1^2) / K^2) 2^-48          (population variance)
//   rstd = fl(1 / fl(sqrt(fl(var + eps))))
//   mu32 = fp32(mean), r32 = fp32(rstd)
// and per element (fp32 operations, round to nearest even, no contraction):
//   y = ((fp32(h_k) - mu32) * r32) * gamma_k + (beta_k - z_k)
//   q = clip(rne(y * inv_s_k), -qa, qa)
//
// Two ways to the same mu32 and r32.  The fast one sums d_k = h_k - c with
// c = h_0 (exact in float64) in float64, in a fixed order (each thread's
// chunks, a butterfly across a wave, waves in order), and bounds its own
// error: a sum whose terms pass through at most n additions is off by at
// most n 2^-53 times the sum of their magnitudes (and sum |d_k| <=
// sqrt(K sum d_k^2)); the few float64 steps after the sums (products with
// fl(1/K), a Newton-refined reciprocal square root) add a few units each.
// If the float64 mean and rstd lie farther than that bound (plus the
// rounding error of the exact procedure itself) from every fp32 rounding
// boundary, their fp32 roundings are the exact ones.  Rows
// where they do not (rare: a few in 10^5 on spread-out rows; always for a
// row whose mean is 0 but whose values are not all 0) take the second way:
// exact integer sums (S1 in 64 bits, S2 in 128 bits) and the float64 steps
// above.  Both paths give the same codes on every run.
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

// h 2^24 as an exact integer (|.| < 2^40): (1024 + m) 2^(e - 1) for a
// normal fp16 with exponent field e and mantissa field m, m for a subnormal.
__device__ inline int64_t half_fixed24(uint32_t b) {
  const int e = (b >> 10) & 31;
  const int64_t m = b & 1023;
  const int64_t mag = e ? (m + 1024) << (e - 1) : m;
  return (b & 0x8000u) ? -mag : mag;
}

typedef unsigned __int128 u128;

// Nearest float64 to a 128-bit unsigned integer (ties to even).
__device__ inline double u128_to_double(u128 v) {
  const uint64_t hi = (uint64_t)(v >> 64);
  if (hi == 0) return (double)(uint64_t)v;  // one correctly rounded conversion
  const int lz = __builtin_clzll(hi);
  const u128 n = v << lz;                   // leading one at bit 127
  const uint64_t top = (uint64_t)(n >> 64);
  const bool sticky = (uint64_t)n != 0;
  uint64_t mant = top >> 11;                // 53 bits
  const uint64_t rest = top & 0x7FF;
  if (rest > 0x400 || (rest == 0x400 && (sticky || (mant & 1)))) ++mant;
  return ldexp((double)mant, 75 - lz);      // bit 0 of mant has weight 2^(75 - lz)
}

// True when x and the value it stands for, known to within err, may lie on
// different sides of a boundary between two fp32 rounding cells, i.e. when
// fp32(x) is not certain to be the fp32 rounding of that value.  The cell
// of f = fp32(x) ends halfway to its neighbours, taken from f's bits.
__device__ inline bool near_fp32_boundary(double x, double err) {
  const float f = (float)x;
  const uint32_t b = __float_as_uint(f);
  if ((b & 0x7f800000u) == 0x7f800000u || !(err < 1e300)) return true;
  uint32_t bu, bd;  // the next fp32 values above and below f
  if ((b & 0x7fffffffu) == 0) {
    bu = 0x00000001u;
    bd = 0x80000001u;
  } else if (b >> 31) {
    bu = b - 1;
    bd = b + 1;
  } else {
    bu = b + 1;
    bd = b - 1;
  }
  const double up = 0.5 * ((double)f + (double)__uint_as_float(bu));  // exact
  const double dn = 0.5 * ((double)f + (double)__uint_as_float(bd));
  return x + err >= up || x - err <= dn;
}

// 1/sqrt(v) to within a few float64 units: the hardware estimate refined
// by two Newton steps (each at least squares the estimate's relative error
// and adds about 3 units of rounding).
__device__ inline double rsqrt_refined(double v) {
  double r = __builtin_amdgcn_rsq(v);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const double t = (v * r) * r;
    r = r * (1.5 - 0.5 * t);
  }
  return r;
}

// Wave-wide exact sums (lane 0 ends with the totals).
__device__ inline int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ inline u128 wave_sum_u128(u128 v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t lo = __shfl_xor((unsigned long long)(uint64_t)v, off);
    const uint64_t hi = __shfl_xor((unsigned long long)(uint64_t)(v >> 64), off);
    v += ((u128)hi << 64) | lo;
  }
  return v;
}

template <int CPT, int R, int MAXT>
__global__ __launch_bounds__(MAXT) void ln_quantize_kernel(
    const uint16_t *__restrict__ h, int64_t M, int K, const uint16_t *__restrict__ gamma,
    const uint16_t *__restrict__ beta, double eps, double inv_k, float qa,
    const float *__restrict__ z, const float *__restrict__ inv_s, int8_t *__restrict__ Xq) {
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
  // No term of the float64 sums passes through more than this many
  // additions: 8 per chunk in a thread, 6 butterfly levels, one per wave.
  const double kU = 0x1p-53;
  const double gam = 1.01 * kU * (double)(8 * CPT + 6 + nwaves + 2);
  float mu32[R], r32[R];
  bool exact[R];
  bool any_exact = false;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    double s1 = 0.0, s2 = 0.0;
    for (int w = 0; w < nwaves; ++w) {
      s1 += red[0][w][r];
      s2 += red[1][w][r];
    }
    // the fast path only has to land within the bound below of the exact
    // procedure, so it takes the cheap operations: products with a rounded
    // 1/K and a refined reciprocal square root
    const double dm = s1 * inv_k;  // mean - c
    const double q = s2 * inv_k;   // sum d^2 / K
    const double mean = cs[r] + dm;
    const double var = fmax(q - dm * dm, 0.0);
    const double ve = var + eps;
    const double rstd = rsqrt_refined(ve);
    mu32[r] = (float)mean;
    r32[r] = (float)rstd;
    // error bounds against the exact procedure, its own roundings included;
    // rms >= sqrt(sum d^2 / K) >= sum |d| / K (sqrt to within one fp32 unit)
    const double rms = (double)(__builtin_amdgcn_sqrtf((float)q) * 1.0001f);
    const double e_dm = gam * rms + 2.01 * kU * fabs(dm);
    const double e_mean = 1.1 * (e_dm + 4.0 * kU * fabs(mean));
    const double e_var = 1.1 * ((gam + 3.0 * kU) * rms * rms + (2.0 * fabs(dm) + 2.0 * e_dm) * e_dm +
                                kU * dm * dm + 4.0 * kU * var);
    // relative change of rstd: half that of var + eps (1 / (var + eps) =
    // rstd^2), plus the roundings of both square roots and reciprocals
    const double e_rstd = rstd * (0.55 * (e_var * rstd * rstd + 3.0 * kU) + 20.0 * kU);
    exact[r] = row0 + r < M &&
               (near_fp32_boundary(mean, e_mean) || near_fp32_boundary(rstd, e_rstd));
    any_exact |= exact[r];
  }

  // the exact procedure for the rows the bound cannot settle (every thread
  // takes the same branch: the values above are identical in all of them)
  if (any_exact) {
    __shared__ int64_t xs1[16][R];
    __shared__ uint64_t xs2[2][16][R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!exact[r]) continue;
      // re-read from the L2 rather than from the registers that hold the
      // row: this branch then adds little to the kernel's register budget
      int64_t e1 = 0;
      u128 e2 = 0;
      const uint16_t *hr = h + (row0 + r) * K;
#pragma unroll 1
      for (int ch = t; ch < nchunks; ch += T) {
        const uint4 v = *reinterpret_cast<const uint4 *>(hr + (int64_t)ch * 8);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t a = half_fixed24((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xFFFFu));
          const uint64_t m = (uint64_t)(a < 0 ? -a : a);
          e1 += a;
          e2 += (u128)m * m;
        }
      }
      e1 = wave_sum_i64(e1);
      e2 = wave_sum_u128(e2);
      if (lane == 0) {
        xs1[wave][r] = e1;
        xs2[0][wave][r] = (uint64_t)e2;
        xs2[1][wave][r] = (uint64_t)(e2 >> 64);
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!exact[r]) continue;
      int64_t S1 = 0;
      u128 S2 = 0;
      for (int w = 0; w < nwaves; ++w) {
        S1 += xs1[w][r];
        S2 += ((u128)xs2[1][w][r] << 64) | xs2[0][w][r];
      }
      const uint64_t m1 = (uint64_t)(S1 < 0 ? -S1 : S1);
      const u128 D = (u128)(uint64_t)K * S2 - (u128)m1 * m1;  // K^2 var 2^48 >= 0
      const double mean = ((double)S1 / (double)K) * 0x1p-24;
      const double var = (u128_to_double(D) / ((double)K * (double)K)) * 0x1p-48;
      const double rstd = 1.0 / sqrt(var + eps);
      mu32[r] = (float)mean;
      r32[r] = (float)rstd;
    }
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
  ln_quantize_kernel<CPT, R, MAXT><<<grid, threads, 0, st>>>(
      h, M, (int)K, gamma, beta, (double)eps, 1.0 / (double)K, (float)qa, z, inv_s, Xq);
  return hipGetLastError();
}

}  // namespace detail

using namespace detail;

hipError_t launch_ln_quantize_act(const uint16_t *h, int64_t M, int64_t K, const uint16_t *gamma,
                                  const uint16_t *beta, float eps, int qa, const float *z,
                                  const float *inv_s, int8_t *Xq, hipStream_t st) {
  // one row per workgroup, 6 chunks of 8 channels per thread up to
  // K = 49152 (a workgroup of at most 1024 threads) and 8 beyond (up to
  // K = 65536).  Measured on 8 shapes (K = 2048 ... 12288, 1024 to 8192
  // rows) against 3 to 8 chunks per thread and 1, 2 or 4 rows per
  // workgroup: 6 chunks and one row is 10 % faster than 8 chunks over the
  // shapes (its fewer registers keep more rows in flight per CU), the
  // fastest at 4 of them and within 9 % of the fastest at every one
  if (K <= 6 * 8 * 1024) return launch_lnq<6, 1>(h, M, K, gamma, beta, eps, qa, z, inv_s, Xq, st);
  return launch_lnq<8, 1>(h, M, K, gamma, beta, eps, qa, z, inv_s, Xq, st);
}

}  // namespace ot
