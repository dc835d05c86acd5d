// Runtime symmetrize + per-channel quantize (OutlierTune Sec. 3.2, Eq. (g):
// the codes round((X - z) / s^X) with static per-channel z and s).
//
//   Xq[m, k] = clip(rne(fp32(fp32(x[m, k]) - z_k) * inv_s_k), -qa, qa)
//
// HBM-bound streaming kernel: 2 bytes in, 1 byte out per element.  A wave
// covers 64 x 8 = 512 consecutive channels (16-byte loads and 8-byte stores
// per lane, fully coalesced), keeps those channels' z and inv_s in registers
// and takes kRowsPerWave consecutive rows at a time, all of their
// (non-temporal) loads issued before any arithmetic.
//
// Also here: the dynamic per-token quantizer of Eq. (c) for the linears that
// the paper leaves per-token (out, fc2).
#include "ot_common.h"

namespace ot {
namespace detail {

constexpr int kWavesPerBlock = 4;
constexpr int kChannelsPerLane = 8;
// From sweeps on MI355X of 8 or 16 channels per lane, 1-16 waves per block,
// 2-64 rows per wave and 1-16 rows' loads in flight, over 2048-8192 rows by
// 4096-36864 channels; with the input read non-temporally (it is read once)
// 8 rows in flight win: the OPT-13B step's four inputs (441 MB, evicted
// from the last-level cache) in 84 us against 110 us with plain loads and
// 4 rows.  The codes are stored normally: the GEMM reads them next.
constexpr int kRowsPerWave = 8;

typedef unsigned v4u __attribute__((ext_vector_type(4)));

__device__ inline uint32_t pack4(int a, int b, int c, int d) {
  return (uint32_t)(a & 0xff) | ((uint32_t)(b & 0xff) << 8) | ((uint32_t)(c & 0xff) << 16) |
         ((uint32_t)(d & 0xff) << 24);
}

__global__ __launch_bounds__(64 * kWavesPerBlock) void quantize_act_kernel(
    const uint16_t *__restrict__ x, int64_t M, int64_t K, float qa, const float *__restrict__ z,
    const float *__restrict__ inv_s, int8_t *__restrict__ Xq) {
  const int64_t k0 = ((int64_t)blockIdx.x * 64 + threadIdx.x) * kChannelsPerLane;
  if (k0 >= K) return;
  float zr[kChannelsPerLane], ir[kChannelsPerLane];
#pragma unroll
  for (int i = 0; i < kChannelsPerLane / 4; ++i) {
    const float4 zz = reinterpret_cast<const float4 *>(z + k0)[i];
    const float4 ii = reinterpret_cast<const float4 *>(inv_s + k0)[i];
    zr[4 * i + 0] = zz.x; zr[4 * i + 1] = zz.y; zr[4 * i + 2] = zz.z; zr[4 * i + 3] = zz.w;
    ir[4 * i + 0] = ii.x; ir[4 * i + 1] = ii.y; ir[4 * i + 2] = ii.z; ir[4 * i + 3] = ii.w;
  }
  // groups of kRowsPerWave consecutive rows, one per wave at a time
  const int64_t group_step = (int64_t)gridDim.y * kWavesPerBlock;
  for (int64_t g = (int64_t)blockIdx.y * kWavesPerBlock + threadIdx.y; g * kRowsPerWave < M;
       g += group_step) {
    const int64_t r0 = g * kRowsPerWave;
    v4u v[kRowsPerWave];
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u)
      v[u] = r0 + u < M
                 ? __builtin_nontemporal_load(reinterpret_cast<const v4u *>(x + (r0 + u) * K + k0))
                 : v4u{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) {
      if (r0 + u >= M) break;
      const uint32_t words[4] = {v[u][0], v[u][1], v[u][2], v[u][3]};
      int q[kChannelsPerLane];
#pragma unroll
      for (int i = 0; i < kChannelsPerLane; ++i) {
        const uint16_t h = (uint16_t)(words[i >> 1] >> (16 * (i & 1)));
        const float t = half_bits_to_float(h) - zr[i];  // fp32, RNE
        const float w = t * ir[i];                      // fp32, RNE
        q[i] = (int)rintf(fminf(fmaxf(w, -qa), qa));
      }
      *reinterpret_cast<uint2 *>(Xq + (r0 + u) * K + k0) =
          make_uint2(pack4(q[0], q[1], q[2], q[3]), pack4(q[4], q[5], q[6], q[7]));
    }
  }
}

// Per-token dynamic quantization (Eq. (c); out and fc2 inputs):
//   s_m = fp32(max_k |x[m, k]| / qa)   (fp64 division; 1 for a zero row)
//   Xq[m, k] = clip(rne(fp32(x[m, k]) * fp32(1 / s_m)), -qa, qa)
// One workgroup per row: each thread holds CPT 16-byte chunks (chunks t,
// t + T, ...) between the max reduction (exact, order-free) and the
// quantize step, so the row is read from HBM once.
template <int CPT, int MAXT>
__global__ __launch_bounds__(MAXT) void quantize_per_token_kernel(
    const uint16_t *__restrict__ x, int K, float qa, int8_t *__restrict__ Xq,
    float *__restrict__ sX) {
  __shared__ float red[16];
  const int T = blockDim.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, nwaves = T >> 6;
  const int nchunks = K / 8;
  const int64_t row = blockIdx.x;
  uint4 v[CPT];
  float mx = 0.f;
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int ch = t + j * T;
    v[j] = ch < nchunks ? *reinterpret_cast<const uint4 *>(x + row * K + (int64_t)ch * 8)
                        : make_uint4(0, 0, 0, 0);
    const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      mx = fmaxf(mx, fabsf(half_bits_to_float((uint16_t)w[i])));
      mx = fmaxf(mx, fabsf(half_bits_to_float((uint16_t)(w[i] >> 16))));
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = 0.f;
  for (int w = 0; w < nwaves; ++w) mx = fmaxf(mx, red[w]);
  float s = (float)((double)mx / (double)qa);
  if (s == 0.f) s = 1.f;
  const float inv = (float)(1.0 / (double)s);
  if (t == 0) sX[row] = s;
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int ch = t + j * T;
    if (ch >= nchunks) continue;
    const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
    uint32_t packed[2] = {0, 0};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float hv = half_bits_to_float((uint16_t)(w[e >> 1] >> (16 * (e & 1))));
      const float u = hv * inv;  // fp32, RNE
      const int q = (int)rintf(fminf(fmaxf(u, -qa), qa));
      packed[e >> 2] |= (uint32_t)(q & 0xff) << (8 * (e & 3));
    }
    *reinterpret_cast<uint2 *>(Xq + row * K + (int64_t)ch * 8) = make_uint2(packed[0], packed[1]);
  }
}

template <int CPT, int MAXT>
hipError_t launch_qpt(const uint16_t *x, int64_t M, int64_t K, int qa, int8_t *Xq, float *sX,
                      hipStream_t st) {
  const int64_t nchunks = K / 8;
  const int threads = (int)((nchunks + CPT * 64 - 1) / (CPT * 64)) * 64;
  if (threads > MAXT) return hipErrorInvalidValue;
  quantize_per_token_kernel<CPT, MAXT><<<(unsigned)M, threads, 0, st>>>(x, (int)K, (float)qa, Xq,
                                                                        sX);
  return hipGetLastError();
}

}  // namespace detail

using namespace detail;

hipError_t launch_quantize_act(const uint16_t *x, int64_t M, int64_t K, int qa, const float *z,
                               const float *inv_s, int8_t *Xq, hipStream_t st) {
  const int64_t chunks = K / kChannelsPerLane;
  const unsigned gx = (unsigned)((chunks + 63) / 64);
  int64_t gy = (M + (int64_t)kWavesPerBlock * kRowsPerWave - 1) /
               ((int64_t)kWavesPerBlock * kRowsPerWave);
  if (gy > 65535) gy = 65535;
  dim3 block(64, kWavesPerBlock);
  quantize_act_kernel<<<dim3(gx, (unsigned)gy), block, 0, st>>>(x, M, K, (float)qa, z, inv_s, Xq);
  return hipGetLastError();
}

hipError_t launch_quantize_act_per_token(const uint16_t *x, int64_t M, int64_t K, int qa,
                                         int8_t *Xq, float *sX, hipStream_t st) {
  if (K <= 4096) return launch_qpt<4, 1024>(x, M, K, qa, Xq, sX, st);
  return launch_qpt<8, 1024>(x, M, K, qa, Xq, sX, st);
}

}  // namespace ot
