// C ABI of libot (declared in include/ot.h): argument checks on the host,
// then kernel launches on the caller's stream.  Nothing here allocates
// device memory or keeps state between calls.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "ot_common.h"

namespace {

// Largest K the kernels' 32-bit in-tile offsets cover (a tile of at most
// 320 K-byte rows must stay below 2^31 bytes).
constexpr int64_t kMaxK = int64_t(1) << 22;
constexpr int64_t kMaxLnK = int64_t(1) << 16;  // LayerNorm width (exact sums, one workgroup per row)
constexpr int64_t kMaxRows = (int64_t(1) << 31) - 1;
// Prefill workgroups of the smallest tile (128 tokens by 256 channels): the
// grid must fit a 32-bit count.
bool grid_ok(int64_t M, int64_t N) { return (M + 127) / 128 * ((N + 255) / 256) <= kMaxRows; }

bool bits_ok(int bits) { return bits >= 2 && bits <= 8; }
int qmax(int bits) { return (1 << (bits - 1)) - 1; }
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

ot_status hip_status(hipError_t e) { return e == hipSuccess ? OT_OK : OT_EHIP; }

bool all_finite(const std::vector<float> &v) {
  for (float f : v)
    if (!isfinite(f)) return false;
  return true;
}

}  // namespace

extern "C" {

const char *ot_strerror(int status) {
  switch (status) {
    case OT_OK: return "ok";
    case OT_EINVAL: return "invalid argument (null or misaligned pointer, bits outside [2, 8], negative size)";
    case OT_ESHAPE: return "unsupported shape (K must be a positive multiple of 16 within limits; sizes must be nonzero where required)";
    case OT_ERANGE: return "K * qa * qw >= 2^31: the int32 accumulator could overflow";
    case OT_ENONFINITE: return "non-finite value (NaN or infinity) in calibration data or weights";
    case OT_EHIP: return "HIP runtime error";
    case OT_ENOSCRATCH: return "these sizes need more scratch than ot_qlinear_noalloc's fixed array holds (use ot_qlinear with a workspace)";
    default: return "unknown status";
  }
}

int ot_abi_version(void) { return 1; }

#ifndef OT_SOURCES_SHA256
#define OT_SOURCES_SHA256 "unknown"
#endif
#define OT_STR2(x) #x
#define OT_STR(x) OT_STR2(x)

const char *ot_build_info(void) {
  return "sources_sha256=" OT_SOURCES_SHA256 ";arch=gfx950;hip=" OT_STR(HIP_VERSION_MAJOR) "." OT_STR(
      HIP_VERSION_MINOR) "." OT_STR(HIP_VERSION_PATCH);
}

ot_status ot_calibrate(const uint16_t *x, int64_t rows, int64_t K, int a_bits, int first,
                       float *minmax, float *z, float *s, float *inv_s, void *stream) {
  if (!x || !minmax || !z || !s || !inv_s) return OT_EINVAL;
  if (!bits_ok(a_bits) || rows < 0 || K < 0) return OT_EINVAL;
  if (rows == 0 || K == 0 || rows > kMaxRows || K > kMaxRows) return OT_ESHAPE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  ot_status rc;
  if (first && (rc = hip_status(ot::launch_calib_reset(minmax, K, st))) != OT_OK) return rc;
  if ((rc = hip_status(ot::launch_calib_minmax(x, rows, K, minmax, st))) != OT_OK) return rc;
  std::vector<float> state((size_t)(2 * K));
  if ((rc = hip_status(hipMemcpyAsync(state.data(), minmax, sizeof(float) * 2 * K,
                                      hipMemcpyDeviceToHost, st))) != OT_OK)
    return rc;
  if ((rc = hip_status(hipStreamSynchronize(st))) != OT_OK) return rc;
  if (!all_finite(state)) return OT_ENONFINITE;
  if ((rc = hip_status(ot::launch_calib_finalize(minmax, K, qmax(a_bits), 1, z, s, inv_s, st))) !=
      OT_OK)
    return rc;
  return hip_status(hipStreamSynchronize(st));
}

ot_status ot_scales_from_minmax(const float *minmax, int64_t K, int a_bits, int symmetrize,
                                float *z, float *s, float *inv_s, void *stream) {
  if (!bits_ok(a_bits) || K < 0) return OT_EINVAL;
  if (K == 0 || K > kMaxRows) return OT_ESHAPE;
  if (!minmax || !z || !s || !inv_s) return OT_EINVAL;
  return hip_status(ot::launch_calib_finalize(minmax, K, qmax(a_bits), symmetrize ? 1 : 0, z, s,
                                              inv_s, static_cast<hipStream_t>(stream)));
}

// Reads sW and b' back (synchronously): a NaN scale marks non-finite weights,
// a non-finite b' non-finite bias or shift.
static ot_status fold_outputs_finite(const float *sW, const float *bprime, int64_t N,
                                     hipStream_t st) {
  ot_status rc;
  std::vector<float> scale((size_t)N), bias((size_t)N);
  if ((rc = hip_status(hipMemcpyAsync(scale.data(), sW, sizeof(float) * N, hipMemcpyDeviceToHost,
                                      st))) != OT_OK ||
      (rc = hip_status(hipMemcpyAsync(bias.data(), bprime, sizeof(float) * N,
                                      hipMemcpyDeviceToHost, st))) != OT_OK)
    return rc;
  if ((rc = hip_status(hipStreamSynchronize(st))) != OT_OK) return rc;
  if (!all_finite(scale) || !all_finite(bias)) return OT_ENONFINITE;
  return OT_OK;
}

ot_status ot_fold_weights(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K, int w_bits,
                          const float *z, const float *s, int8_t *Wq, float *sW, float *bprime,
                          void *stream) {
  if (!W || !z || !s || !Wq || !sW || !bprime) return OT_EINVAL;
  if (!bits_ok(w_bits) || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K == 0 || N > kMaxRows || K > kMaxRows) return OT_ESHAPE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  ot_status rc;
  if ((rc = hip_status(ot::launch_fold(W, b, N, K, qmax(w_bits), z, s, Wq, sW, bprime, st))) !=
      OT_OK)
    return rc;
  return fold_outputs_finite(sW, bprime, N, st);
}

ot_status ot_quantize_act(const uint16_t *x, int64_t M, int64_t K, int a_bits, const float *z,
                          const float *inv_s, int8_t *Xq, void *stream) {
  if (!bits_ok(a_bits) || M < 0 || K < 0) return OT_EINVAL;
  if (K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows) return OT_ESHAPE;
  if (M == 0) return OT_OK;
  if (!x || !z || !inv_s || !Xq) return OT_EINVAL;
  if (!aligned16(x) || !aligned16(z) || !aligned16(inv_s) || !aligned16(Xq)) return OT_EINVAL;
  return hip_status(ot::launch_quantize_act(x, M, K, qmax(a_bits), z, inv_s, Xq,
                                            static_cast<hipStream_t>(stream)));
}

ot_status ot_ln_quantize_act(const uint16_t *h, int64_t M, int64_t K, const uint16_t *gamma,
                             const uint16_t *beta, float eps, int a_bits, const float *z,
                             const float *inv_s, int8_t *Xq, void *stream) {
  if (!bits_ok(a_bits) || M < 0 || K < 0 || !(eps >= 0.f) || eps > 3.4e38f) return OT_EINVAL;
  if (K < 16 || K % 16 != 0 || K > kMaxLnK || M > kMaxRows) return OT_ESHAPE;
  if (M == 0) return OT_OK;
  if (!h || !gamma || !beta || !z || !inv_s || !Xq) return OT_EINVAL;
  if (!aligned16(h) || !aligned16(gamma) || !aligned16(beta) || !aligned16(z) ||
      !aligned16(inv_s) || !aligned16(Xq))
    return OT_EINVAL;
  return hip_status(ot::launch_ln_quantize_act(h, M, K, gamma, beta, eps, qmax(a_bits), z, inv_s,
                                               Xq, static_cast<hipStream_t>(stream)));
}

ot_status ot_qlinear(const int8_t *Xq, const int8_t *Wq, const float *sW, const float *bprime,
                     int64_t M, int64_t N, int64_t K, int a_bits, int w_bits, uint16_t *Y,
                     int32_t *acc_out, void *workspace, void *stream) {
  if (!bits_ok(a_bits) || !bits_ok(w_bits) || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows || N > kMaxRows)
    return OT_ESHAPE;
  if (!grid_ok(M, N)) return OT_ESHAPE;
  if (K * qmax(a_bits) * qmax(w_bits) >= (int64_t(1) << 31)) return OT_ERANGE;
  if (M == 0) return OT_OK;
  if (!Xq || !Wq || !sW || !bprime || !Y) return OT_EINVAL;
  if (!aligned16(Xq) || !aligned16(Wq) || !aligned16(sW) || !aligned16(bprime) || !aligned16(Y) ||
      (acc_out && !aligned16(acc_out)) ||
      (workspace && !aligned16(workspace)))
    return OT_EINVAL;
  return hip_status(ot::launch_qgemm(Xq, Wq, nullptr, nullptr, sW, bprime, M, N, K, Y, acc_out,
                                     workspace, static_cast<hipStream_t>(stream)));
}

ot_status ot_quantize_act_per_token(const uint16_t *x, int64_t M, int64_t K, int a_bits,
                                    int8_t *Xq, float *sX, void *stream) {
  if (!bits_ok(a_bits) || M < 0 || K < 0) return OT_EINVAL;
  if (K < 16 || K % 16 != 0 || K > kMaxLnK || M > kMaxRows) return OT_ESHAPE;
  if (M == 0) return OT_OK;
  if (!x || !Xq || !sX) return OT_EINVAL;
  if (!aligned16(x) || !aligned16(Xq) || !aligned16(sX)) return OT_EINVAL;
  return hip_status(ot::launch_quantize_act_per_token(x, M, K, qmax(a_bits), Xq, sX,
                                                      static_cast<hipStream_t>(stream)));
}

ot_status ot_fold_weights_per_token(const uint16_t *W, const uint16_t *b, const float *zres,
                                    int64_t N, int64_t K, int w_bits, int8_t *Wq, float *sW,
                                    float *bprime, void *stream) {
  if (!bits_ok(w_bits) || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K == 0 || N > kMaxRows || K > kMaxRows) return OT_ESHAPE;
  if (!W || !Wq || !sW || !bprime) return OT_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  ot_status rc;
  if ((rc = hip_status(ot::launch_fold_per_token(W, b, zres, N, K, qmax(w_bits), Wq, sW, bprime,
                                                 st))) != OT_OK)
    return rc;
  return fold_outputs_finite(sW, bprime, N, st);
}

ot_status ot_qlinear_per_token(const int8_t *Xq, const int8_t *Wq, const float *sX,
                               const float *sW, const float *bprime, int64_t M, int64_t N,
                               int64_t K, int a_bits, int w_bits, uint16_t *Y, int32_t *acc_out,
                               void *workspace, void *stream) {
  if (!bits_ok(a_bits) || !bits_ok(w_bits) || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows || N > kMaxRows)
    return OT_ESHAPE;
  if (!grid_ok(M, N)) return OT_ESHAPE;
  if (K * qmax(a_bits) * qmax(w_bits) >= (int64_t(1) << 31)) return OT_ERANGE;
  if (M == 0) return OT_OK;
  if (!Xq || !Wq || !sX || !sW || !bprime || !Y) return OT_EINVAL;
  if (!aligned16(Xq) || !aligned16(Wq) || !aligned16(sW) || !aligned16(bprime) || !aligned16(Y) ||
      (acc_out && !aligned16(acc_out)) ||
      (workspace && !aligned16(workspace)))
    return OT_EINVAL;
  return hip_status(ot::launch_qgemm(Xq, Wq, sX, nullptr, sW, bprime, M, N, K, Y, acc_out,
                                     workspace, static_cast<hipStream_t>(stream)));
}

ot_status ot_fold_weights_asym(const uint16_t *W, const uint16_t *b, int64_t N, int64_t K,
                               int w_bits, const float *z, const float *s, int8_t *Wq, float *sW,
                               int32_t *zW, float *bprime, void *stream) {
  if (!W || !z || !s || !Wq || !sW || !zW || !bprime) return OT_EINVAL;
  if (!bits_ok(w_bits) || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K == 0 || N > kMaxRows || K > kMaxRows) return OT_ESHAPE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  ot_status rc;
  if ((rc = hip_status(ot::launch_fold_asym(W, b, N, K, w_bits, z, s, Wq, sW, zW, bprime, st))) !=
      OT_OK)
    return rc;
  return fold_outputs_finite(sW, bprime, N, st);
}

ot_status ot_qlinear_asym(const int8_t *Xq, const int8_t *Wq, const float *sW, const int32_t *zW,
                          const float *bprime, int64_t M, int64_t N, int64_t K, int a_bits,
                          int w_bits, uint16_t *Y, int32_t *acc_out, void *workspace,
                          void *stream) {
  if (!bits_ok(a_bits) || !bits_ok(w_bits) || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows || N > kMaxRows)
    return OT_ESHAPE;
  if (!grid_ok(M, N)) return OT_ESHAPE;
  // |Xq| <= qa against stored codes and zero points of magnitude <= 2^(w_bits-1):
  // every partial sum stays below K qa 2^w_bits
  if (K * qmax(a_bits) * (int64_t(1) << w_bits) >= (int64_t(1) << 31)) return OT_ERANGE;
  if (M == 0) return OT_OK;
  if (!Xq || !Wq || !sW || !zW || !bprime || !Y) return OT_EINVAL;
  if (!aligned16(Xq) || !aligned16(Wq) || !aligned16(sW) || !aligned16(zW) ||
      !aligned16(bprime) || !aligned16(Y) || (acc_out && !aligned16(acc_out)) ||
      (workspace && !aligned16(workspace)))
    return OT_EINVAL;
  return hip_status(ot::launch_qgemm(Xq, Wq, nullptr, zW, sW, bprime, M, N, K, Y, acc_out,
                                     workspace, static_cast<hipStream_t>(stream)));
}

size_t ot_packed_weights_size(int64_t N, int64_t K) {
  if (N <= 0 || K < 16 || K % 16 != 0 || N > kMaxRows || K > kMaxK) return 0;
  return ot::packed_weights_bytes(N, K);
}

ot_status ot_pack_weights(const int8_t *Wq, int64_t N, int64_t K, int8_t *Wp, void *stream) {
  if (N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || N > kMaxRows) return OT_ESHAPE;
  if (!Wq || !Wp || !aligned16(Wq) || !aligned16(Wp)) return OT_EINVAL;
  return hip_status(ot::launch_pack_weights(Wq, N, K, Wp, static_cast<hipStream_t>(stream)));
}

ot_status ot_qlinear_packed(const int8_t *Xq, const int8_t *Wp, const float *sW,
                            const float *bprime, int64_t M, int64_t N, int64_t K, int a_bits,
                            int w_bits, uint16_t *Y, int32_t *acc_out, void *workspace,
                            void *stream) {
  if (!bits_ok(a_bits) || !bits_ok(w_bits) || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (M > 64 || N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || N > kMaxRows) return OT_ESHAPE;
  if (K * qmax(a_bits) * qmax(w_bits) >= (int64_t(1) << 31)) return OT_ERANGE;
  if (M == 0) return OT_OK;
  if (!Xq || !Wp || !sW || !bprime || !Y) return OT_EINVAL;
  if (!aligned16(Xq) || !aligned16(Wp) || !aligned16(sW) || !aligned16(bprime) || !aligned16(Y) ||
      (acc_out && !aligned16(acc_out)) || (workspace && !aligned16(workspace)))
    return OT_EINVAL;
  return hip_status(ot::launch_qgemm_decode(Xq, Wp, nullptr, nullptr, sW, bprime, M, N, K, Y,
                                            acc_out, workspace, true,
                                            static_cast<hipStream_t>(stream)));
}

ot_status ot_qlinear_plan(int64_t M, int64_t N, int64_t K, int packed, int with_workspace,
                          char *buf, size_t len) {
  if (!buf || len == 0 || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows || N > kMaxRows ||
      !grid_ok(M, N) || (packed && M > 64))
    return OT_ESHAPE;
  if (M == 0)
    snprintf(buf, len, "none");
  else if (M <= 64)
    ot::describe_decode(M, N, K, packed != 0, with_workspace != 0, buf, len);
  else
    snprintf(buf, len, "%s", ot::prefill_tile_name(M, N, K));
  return OT_OK;
}

size_t ot_qlinear_workspace_size(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0 || M > kMaxRows || N > kMaxRows || K > kMaxK) return 0;
  return ot::qgemm_workspace_bytes(M, N, K);
}

}  // extern "C"
