// ot_qlinear_noalloc: ot_qlinear for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).  The only scratch the quantized linear uses is
// the split-K decode's int32 partial sums (17..64 tokens, where the launch
// plan splits K); here they live in a fixed device array of this library
// instead of a caller workspace.  Prefill and unsplit decode launches use
// no scratch at all and run exactly as ot_qlinear does.
#include <atomic>
#include <mutex>

#include "ot_common.h"

namespace {

// The split-K partial sums [runs][M][N] and the tokens' partial code sums
// [runs][M] of the call in flight.  Every device the library runs on holds
// its own copy until the process ends.  Its contents need no clearing: a
// split launch writes every partial sum it later reads.  In host code the
// name stands for a host-side shadow, never the device memory: the device
// address comes from hipGetSymbolAddress below.
static __device__ __align__(256) int8_t scratch[OT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// The device address of this device's copy of the array, looked up once per
// device (with that device current) and kept; nullptr on failure.
void *scratch_on(int dev) {
  void *p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (p) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
  g_scratch[dev].store(p, std::memory_order_release);
  return p;
}

constexpr int64_t kMaxK = int64_t(1) << 22;
constexpr int64_t kMaxRows = (int64_t(1) << 31) - 1;
bool bits_ok(int bits) { return bits >= 2 && bits <= 8; }
int qmax(int bits) { return (1 << (bits - 1)) - 1; }
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" ot_status ot_qlinear_noalloc(const int8_t *Xq, const int8_t *Wq, const float *sW,
                                        const float *bprime, int64_t M, int64_t N, int64_t K,
                                        int a_bits, int w_bits, uint16_t *Y, int32_t *acc_out,
                                        void *stream) {
  // the checks of ot_qlinear, in the same order
  if (!bits_ok(a_bits) || !bits_ok(w_bits) || M < 0 || N < 0 || K < 0) return OT_EINVAL;
  if (N == 0 || K < 16 || K % 16 != 0 || K > kMaxK || M > kMaxRows || N > kMaxRows)
    return OT_ESHAPE;
  if ((M + 127) / 128 * ((N + 255) / 256) > kMaxRows) return OT_ESHAPE;
  if (K * qmax(a_bits) * qmax(w_bits) >= (int64_t(1) << 31)) return OT_ERANGE;
  if (M == 0) return OT_OK;
  if (!Xq || !Wq || !sW || !bprime || !Y) return OT_EINVAL;
  if (!aligned16(Xq) || !aligned16(Wq) || !aligned16(sW) || !aligned16(bprime) || !aligned16(Y) ||
      (acc_out && !aligned16(acc_out)))
    return OT_EINVAL;
  const size_t need = ot::qgemm_workspace_bytes(M, N, K);
  if (need > (size_t)OT_NOALLOC_SCRATCH_BYTES) return OT_ENOSCRATCH;
  void *ws = nullptr;
  if (need > 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return OT_EHIP;
    if ((ws = scratch_on(dev)) == nullptr) return OT_EHIP;
  }
  const hipError_t e = ot::launch_qgemm(Xq, Wq, nullptr, nullptr, sW, bprime, M, N, K, Y, acc_out,
                                        ws, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? OT_OK : OT_EHIP;
}
