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

// Epilogue flavours: PT = false is the per-channel path (one scale per
// output channel), PT = true the per-token path (token scale sx as well).
template <bool PT>
__device__ inline uint16_t dequant_x(int a, float sx, float sw, float bp) {
  if constexpr (PT) return dequant_pt(a, sx, sw, bp);
  else return dequant(a, sw, bp);
}

// Writes four consecutive channels n..n+3 of token m (token scale sx, used
// when PT).
template <bool PT>
__device__ inline void store4(uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out,
                              const float *__restrict__ sW, const float *__restrict__ bp,
                              float sx, int64_t m, int64_t n, int64_t M, int64_t N, int a0,
                              int a1, int a2, int a3) {
  if (m >= M) return;
  const int64_t base = m * N + n;
  if (n + 3 < N && (N & 3) == 0) {
    const float4 s4 = *reinterpret_cast<const float4 *>(sW + n);
    const float4 b4 = *reinterpret_cast<const float4 *>(bp + n);
    uint2 o;
    o.x = (uint32_t)dequant_x<PT>(a0, sx, s4.x, b4.x) |
          ((uint32_t)dequant_x<PT>(a1, sx, s4.y, b4.y) << 16);
    o.y = (uint32_t)dequant_x<PT>(a2, sx, s4.z, b4.z) |
          ((uint32_t)dequant_x<PT>(a3, sx, s4.w, b4.w) << 16);
    *reinterpret_cast<uint2 *>(Y + base) = o;
    if (acc_out) *reinterpret_cast<int4 *>(acc_out + base) = make_int4(a0, a1, a2, a3);
  } else {
    const int a[4] = {a0, a1, a2, a3};
    for (int i = 0; i < 4; ++i) {
      if (n + i < N) {
        Y[base + i] = dequant_x<PT>(a[i], sx, sW[n + i], bp[n + i]);
        if (acc_out) acc_out[base + i] = a[i];
      }
    }
  }
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
