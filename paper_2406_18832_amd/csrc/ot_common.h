// Internal declarations shared by libot's translation units (not installed).
//
// Every translation unit is compiled for gfx950 only, with floating-point
// contraction off: the method's roundings are specified step by step, and
// a fused multiply-add would skip one of them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ot.h"

namespace ot {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// Word 3 of a raw (untyped) buffer resource on gfx9-family GPUs.
constexpr uint32_t kRsrcWord3 = 0x00020000u;
// A byte offset no buffer here reaches: a load from it returns zeros.
constexpr uint32_t kOobOffset = 0x80000000u;

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)nbytes,
                                           (int)kRsrcWord3);
}

__device__ inline float half_bits_to_float(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// fp32 -> fp16, round to nearest even, +-inf on overflow.
__device__ inline uint16_t float_to_half_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// Compute units of the current device (queried once per device; 256 if the
// query fails).  The GEMM launchers size their grids by it.
int device_cus();

// Launchers: each validates nothing (the C ABI layer does) and returns the
// launch status.
hipError_t launch_calib_reset(float *minmax, int64_t K, hipStream_t st);
hipError_t launch_calib_minmax(const uint16_t *x, int64_t rows, int64_t K, float *minmax,
                               hipStream_t st);
hipError_t launch_calib_finalize(const float *minmax, int64_t K, int qa, int symmetrize, float *z,
                                 float *s, float *inv_s, hipStream_t st);
hipError_t launch_fold(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K, int qw,
                       const float *z, const float *s, int8_t *Wq, float *sW, float *bprime,
                       hipStream_t st);
hipError_t launch_quantize_act(const uint16_t *x, int64_t M, int64_t K, int qa, const float *z,
                               const float *inv_s, int8_t *Xq, hipStream_t st);
hipError_t launch_ln_quantize_act(const uint16_t *h, int64_t M, int64_t K, const uint16_t *gamma,
                                  const uint16_t *beta, float eps, int qa, const float *z,
                                  const float *inv_s, int8_t *Xq, hipStream_t st);
// packed: Wq holds micro-tiles from launch_pack_weights instead of [N x K].
hipError_t launch_qgemm_decode(const int8_t *Xq, const int8_t *Wq, const float *sX,
                               const int32_t *zW, const float *sW, const float *bprime,
                               int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                               void *workspace, bool packed, hipStream_t st);
// Decode micro-tile layout of the weight codes (bytes; the packing).
size_t packed_weights_bytes(int64_t N, int64_t K);
hipError_t launch_pack_weights(const int8_t *Wq, int64_t N, int64_t K, int8_t *Wp,
                               hipStream_t st);
// Scratch bytes the decode kernels use for split-K partial sums (0: none).
size_t qgemm_decode_workspace_bytes(int64_t M, int64_t N, int64_t K);
// The prefill tile launch_qgemm_prefill picks ("prefill 320x256", ...).
const char *prefill_tile_name(int64_t M, int64_t N, int64_t K);
// The decode configuration launch_qgemm_decode picks, as text.
void describe_decode(int64_t M, int64_t N, int64_t K, bool packed, bool workspace, char *buf,
                     size_t len);
hipError_t launch_qgemm_prefill(const int8_t *Xq, const int8_t *Wq, const float *sX,
                                const int32_t *zW, const float *sW, const float *bprime,
                                int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                                hipStream_t st);
// Epilogue: sX != nullptr per-token scales (Eq. (c)); zW != nullptr
// asymmetric weight zero points (Eq. (a)); neither, per-channel (Eq. (g)).
// workspace: nullptr, or at least qgemm_workspace_bytes(M, N, K) bytes.
hipError_t launch_qgemm(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                        const float *sW, const float *bprime, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y, int32_t *acc_out, void *workspace, hipStream_t st);
size_t qgemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_fold_asym(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K,
                            int w_bits, const float *z, const float *s, int8_t *Wq, float *sW,
                            int32_t *zW, float *bprime, hipStream_t st);
hipError_t launch_quantize_act_per_token(const uint16_t *x, int64_t M, int64_t K, int qa,
                                         int8_t *Xq, float *sX, hipStream_t st);
hipError_t launch_fold_per_token(const uint16_t *W, const uint16_t *b, const float *zres,
                                 int64_t N, int64_t K, int qw, int8_t *Wq, float *sW,
                                 float *bprime, hipStream_t st);

}  // namespace ot
