// The quantized linear of OutlierTune, Eq. (f) and (g): int8 GEMM over the
// folded operands plus the dequantizing epilogue (kernels in ot_prefill.hip
// and ot_decode.hip, shared helpers in ot_gemm_common.h).
#include <atomic>

#include "ot_common.h"

namespace ot {

int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// At most 64 tokens (decode) the GEMM streams the weights once and is bound
// by HBM bandwidth; beyond that (prefill) it is a tiled int8 MFMA GEMM.
// Epilogue: sX != nullptr the per-token scales of Eq. (c); zW != nullptr the
// asymmetric weight zero points of Eq. (a); neither, the per-channel
// epilogue of Eq. (g).
// The prefill kernels use no scratch; the decode kernels use the workspace
// (when given) for split-K partial sums.
hipError_t launch_qgemm(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                        const float *sW, const float *bprime, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y, int32_t *acc_out, void *workspace, hipStream_t st) {
  if (M <= 64)
    return launch_qgemm_decode(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, workspace, false,
                               st);
  return launch_qgemm_prefill(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
}

size_t qgemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return M <= 64 ? qgemm_decode_workspace_bytes(M, N, K) : 0;
}

}  // namespace ot
