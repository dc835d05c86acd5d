// The quantized linear of OutlierTune, Eq. (f) and (g): int8 GEMM over the
// folded operands plus the dequantizing epilogue (kernels in ot_prefill.hip
// and ot_decode.hip, shared helpers in ot_gemm_common.h).
#include "ot_common.h"

namespace ot {

// At most 64 tokens (decode) the GEMM streams the weights once and is bound
// by HBM bandwidth; beyond that (prefill) it is a tiled int8 MFMA GEMM.
// Epilogue: sX != nullptr the per-token scales of Eq. (c); zW != nullptr the
// asymmetric weight zero points of Eq. (a); neither, the per-channel
// epilogue of Eq. (g).
hipError_t launch_qgemm(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                        const float *sW, const float *bprime, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y, int32_t *acc_out, hipStream_t st) {
  if (M <= 64) return launch_qgemm_decode(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
  return launch_qgemm_prefill(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
}

}  // namespace ot
