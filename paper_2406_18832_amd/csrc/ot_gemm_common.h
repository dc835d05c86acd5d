// Device helpers shared by the quantized-linear GEMM kernels (prefill and
// decode): the dequantizing epilogue and LDS/wait primitives.
//
// The quantized linear of OutlierTune: the integer GEMM of Eq. (f)'s
// right-hand side (no scale inside the sum once s^X is folded into W) and
// the dequantizing epilogue of Eq. (g):
//
//   acc[m, n] = sum_k Xq[m, k] * Wq[n, k]                  (exact int32)
//   Y[m, n]   = fp16(fp32(fp32(acc[m, n]) * sW[n]) + b'[n])
//
// Both operands are K-contiguous ("NT"), which is the layout the int8 matrix
// cores want for both sides, so no transposition is needed anywhere.
//
// Operand roles.  The MFMA's A side (the rows of its 32x32 or 16x16 output
// block) takes weight rows n, the B side takes token rows m.  Each lane then
// holds four consecutive output channels n of one token m, which the
// epilogue scales and stores as one 8-byte fp16 vector.
//
// K order inside an MFMA.  An MFMA sums over its K positions; which byte of
// which lane the hardware assigns to which position does not matter as long
// as the A and B lanes that meet use the same assignment.  Every lane here
// loads 16 contiguous K bytes for its row, picked identically on both sides,
// so the product is the plain dot product whatever the hardware's order.
#pragma once

#include "ot_common.h"

namespace ot {
namespace detail {

// ---------------------------------------------------------------------------
// Epilogue helpers
// ---------------------------------------------------------------------------
__device__ inline uint16_t dequant(int a, float sw, float bp) {
  const float v = (float)a;  // int32 -> fp32, round to nearest even
  const float p = v * sw;    // fp32, RNE (contraction is off)
  const float y = p + bp;    // fp32, RNE
  return float_to_half_bits(y);
}

// Per-token path, Eq. (c): y = fp16(fp32(fp32(fp32(acc) * sX_m) * sW_n) + b'_n).
__device__ inline uint16_t dequant_pt(int a, float sx, float sw, float bp) {
  const float v = (float)a;
  const float t = v * sx;
  const float p = t * sw;
  const float y = p + bp;
  return float_to_half_bits(y);
}

// Epilogue flavours
//   kEpiChannel  per-channel path, Eq. (g): scale per output channel
//   kEpiToken    per-token path, Eq. (c): token scale sx as well
//   kEpiAsym     asymmetric weights, Eq. (a): the integer sum becomes
//                acc - zW[n] * rowsum(Xq[m]) before the per-channel scale
constexpr int kEpiChannel = 0, kEpiToken = 1, kEpiAsym = 2;

template <int EPI>
__device__ inline uint16_t dequant_x(int a, float sx, float sw, float bp) {
  if constexpr (EPI == kEpiToken) return dequant_pt(a, sx, sw, bp);
  else return dequant(a, sw, bp);
}

// Four consecutive weight zero points n..n+3 (zeros past N; unused unless
// EPI == kEpiAsym).
template <int EPI>
__device__ inline int4 load_zw4(const int32_t *__restrict__ zW, int64_t n, int64_t N) {
  if constexpr (EPI != kEpiAsym) {
    return make_int4(0, 0, 0, 0);
  } else {
    if (n + 3 < N && (N & 3) == 0) return *reinterpret_cast<const int4 *>(zW + n);
    return make_int4(n < N ? zW[n] : 0, n + 1 < N ? zW[n + 1] : 0, n + 2 < N ? zW[n + 2] : 0,
                     n + 3 < N ? zW[n + 3] : 0);
  }
}

// Scale, bias and (asymmetric weights) zero point of the four consecutive
// channels n..n+3 (zeros past N).
template <int EPI>
__device__ inline void load_epi4(const float *__restrict__ sW, const float *__restrict__ bp,
                                 const int32_t *__restrict__ zW, int64_t n, int64_t N, float4 &s4,
                                 float4 &b4, int4 &z4) {
  if (n + 3 < N && (N & 3) == 0) {
    s4 = *reinterpret_cast<const float4 *>(sW + n);
    b4 = *reinterpret_cast<const float4 *>(bp + n);
  } else {
    s4 = make_float4(0.f, 0.f, 0.f, 0.f);
    b4 = s4;
    if (n + 0 < N) { s4.x = sW[n + 0]; b4.x = bp[n + 0]; }
    if (n + 1 < N) { s4.y = sW[n + 1]; b4.y = bp[n + 1]; }
    if (n + 2 < N) { s4.z = sW[n + 2]; b4.z = bp[n + 2]; }
    if (n + 3 < N) { s4.w = sW[n + 3]; b4.w = bp[n + 3]; }
  }
  z4 = load_zw4<EPI>(zW, n, N);
}

// Writes four consecutive channels n..n+3 of token m, given their scale,
// bias and zero point.  sx is the token's scale (kEpiToken), rs its code
// sum (kEpiAsym); acc_out receives the integer sum the epilogue scales.
template <int EPI>
__device__ inline void store4_pre(uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out,
                                  float4 s4, float4 b4, int4 z4, float sx, int rs, int64_t m,
                                  int64_t n, int64_t M, int64_t N, int a0, int a1, int a2, int a3) {
  if (m >= M) return;
  if constexpr (EPI == kEpiAsym) {
    a0 -= z4.x * rs;
    a1 -= z4.y * rs;
    a2 -= z4.z * rs;
    a3 -= z4.w * rs;
  }
  const int64_t base = m * N + n;
  if (n + 3 < N && (N & 3) == 0) {
    uint2 o;
    o.x = (uint32_t)dequant_x<EPI>(a0, sx, s4.x, b4.x) |
          ((uint32_t)dequant_x<EPI>(a1, sx, s4.y, b4.y) << 16);
    o.y = (uint32_t)dequant_x<EPI>(a2, sx, s4.z, b4.z) |
          ((uint32_t)dequant_x<EPI>(a3, sx, s4.w, b4.w) << 16);
    *reinterpret_cast<uint2 *>(Y + base) = o;
    if (acc_out) *reinterpret_cast<int4 *>(acc_out + base) = make_int4(a0, a1, a2, a3);
  } else {
    const int a[4] = {a0, a1, a2, a3};
    const float s[4] = {s4.x, s4.y, s4.z, s4.w}, b[4] = {b4.x, b4.y, b4.z, b4.w};
    for (int i = 0; i < 4; ++i) {
      if (n + i < N) {
        Y[base + i] = dequant_x<EPI>(a[i], sx, s[i], b[i]);
        if (acc_out) acc_out[base + i] = a[i];
      }
    }
  }
}

// Writes four consecutive channels n..n+3 of token m (loading their scale,
// bias and zero point).
template <int EPI>
__device__ inline void store4(uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out,
                              const float *__restrict__ sW, const float *__restrict__ bp,
                              const int32_t *__restrict__ zW, float sx, int rs, int64_t m,
                              int64_t n, int64_t M, int64_t N, int a0, int a1, int a2, int a3) {
  if (m >= M) return;
  float4 s4, b4;
  int4 z4;
  load_epi4<EPI>(sW, bp, zW, n, N, s4, b4, z4);
  store4_pre<EPI>(Y, acc_out, s4, b4, z4, sx, rs, m, n, M, N, a0, a1, a2, a3);
}

// Sum of the 16 signed bytes of a fragment (one dot-product instruction per
// 4 bytes against all-ones).
__device__ inline int byte_sum16(v4i f, int acc) {
  acc = __builtin_amdgcn_sdot4(f[0], 0x01010101, acc, false);
  acc = __builtin_amdgcn_sdot4(f[1], 0x01010101, acc, false);
  acc = __builtin_amdgcn_sdot4(f[2], 0x01010101, acc, false);
  return __builtin_amdgcn_sdot4(f[3], 0x01010101, acc, false);
}

typedef __attribute__((address_space(3))) void lds_void;

// Workgroup barrier without the memory fence of __syncthreads() (which would
// drain every outstanding global load): the callers wait for exactly the
// loads they need first.  The clobber keeps the compiler from moving LDS
// accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt (gfx9 encoding) waiting until at most N vector-memory operations
// are outstanding, leaving the other counters unconstrained.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  constexpr int kImm = (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);
  __builtin_amdgcn_s_waitcnt(kImm);
}

}  // namespace detail
}  // namespace ot
