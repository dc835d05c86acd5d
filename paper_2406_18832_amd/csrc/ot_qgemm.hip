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

// Writes four consecutive channels n..n+3 of token m.
__device__ inline void store4(uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out,
                              const float *__restrict__ sW, const float *__restrict__ bp,
                              int64_t m, int64_t n, int64_t M, int64_t N, int a0, int a1, int a2,
                              int a3) {
  if (m >= M) return;
  const int64_t base = m * N + n;
  if (n + 3 < N && (N & 3) == 0) {
    const float4 s4 = *reinterpret_cast<const float4 *>(sW + n);
    const float4 b4 = *reinterpret_cast<const float4 *>(bp + n);
    uint2 o;
    o.x = (uint32_t)dequant(a0, s4.x, b4.x) | ((uint32_t)dequant(a1, s4.y, b4.y) << 16);
    o.y = (uint32_t)dequant(a2, s4.z, b4.z) | ((uint32_t)dequant(a3, s4.w, b4.w) << 16);
    *reinterpret_cast<uint2 *>(Y + base) = o;
    if (acc_out) *reinterpret_cast<int4 *>(acc_out + base) = make_int4(a0, a1, a2, a3);
  } else {
    const int a[4] = {a0, a1, a2, a3};
    for (int i = 0; i < 4; ++i) {
      if (n + i < N) {
        Y[base + i] = dequant(a[i], sW[n + i], bp[n + i]);
        if (acc_out) acc_out[base + i] = a[i];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Prefill: LDS-tiled int8 MFMA GEMM (v_mfma_i32_32x32x32_i8)
// ---------------------------------------------------------------------------
// Workgroup tile BN (weight rows) x BM (token rows), K step BK bytes, waves
// arranged WN x WM, each wave owning a (BN/WN) x (BM/WM) block of 32x32 MFMA
// tiles.  Global -> LDS traffic uses the buffer "load to LDS" path (no
// registers, no ds_write): one wave-wide 16-byte-per-lane load fills 1 KiB
// of LDS, i.e. 1024/BK whole rows of a tile.  Rows are stored with their
// 16-byte chunks XOR-swizzled by (row mod BK/16), so that the MFMA fragment
// reads (lanes 0..31 = 32 consecutive rows, same chunk) hit distinct banks.
// Buffer loads return zeros past the end of the resource, which pads ragged
// M and N tiles; a K tail is padded by aiming its lanes at an out-of-range
// offset.  Two LDS stages: the next K tile streams in while the current one
// feeds the matrix cores.
template <int BN, int BM, int BK, int WN, int WM>
struct PrefillCfg {
  static constexpr int kWaves = WN * WM;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kChunks = BK / 16;           // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 1024 / BK;    // rows per wave-wide load
  static constexpr int kTN = BN / WN, kTM = BM / WM;
  static constexpr int kFN = kTN / 32, kFM = kTM / 32;
  static constexpr int kABytes = BN * BK, kBBytes = BM * BK;
  static constexpr int kStage = kABytes + kBBytes;
  static constexpr int kLoadsA = kABytes / 1024 / kWaves;
  static constexpr int kLoadsB = kBBytes / 1024 / kWaves;
  static_assert(kChunks <= 8 && (kRowsPerLoad % kChunks) == 0, "swizzle period");
  static_assert(kLoadsA * 1024 * kWaves == kABytes && kLoadsB * 1024 * kWaves == kBBytes,
                "tile must split evenly into wave loads");
  static_assert(kTN % 32 == 0 && kTM % 32 == 0 && BK % 32 == 0, "MFMA tiling");
};

typedef __attribute__((address_space(3))) void lds_void;

// Issues one K tile of both operands into LDS stage `dst` (this wave's share).
template <int BN, int BM, int BK, int WN, int WM>
__device__ __forceinline__ void prefill_load_tile(
    __amdgpu_buffer_rsrc_t rsrc_a, __amdgpu_buffer_rsrc_t rsrc_b, const uint32_t *off_a,
    const uint32_t *off_b, int lchunk, int wave, int K, int k0, int8_t *dst) {
  using C = PrefillCfg<BN, BM, BK, WN, WM>;
  const bool in_k = k0 + lchunk * 16 < K;
  int8_t *sb = dst + C::kABytes;
#pragma unroll
  for (int j = 0; j < C::kLoadsA; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc_a, (lds_void *)(dst + (wave * C::kLoadsA + j) * 1024), 16,
        in_k ? off_a[j] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
#pragma unroll
  for (int j = 0; j < C::kLoadsB; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc_b, (lds_void *)(sb + (wave * C::kLoadsB + j) * 1024), 16,
        in_k ? off_b[j] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
}

template <int BN, int BM, int BK, int WN, int WM>
__global__ __launch_bounds__(64 * WN * WM, 1) void qgemm_prefill_kernel(
    const int8_t *__restrict__ Xq, const int8_t *__restrict__ Wq, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, int K, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out, int tiles_m, int tiles_n, int group_m) {
  using C = PrefillCfg<BN, BM, BK, WN, WM>;
  __shared__ __attribute__((aligned(1024))) int8_t smem[2 * C::kStage];

  // ---- tile schedule ------------------------------------------------------
  // The dispatcher deals workgroups to the 8 XCDs round-robin (id mod 8), and
  // each XCD has its own L2.  Renumber so that each XCD owns a contiguous
  // range of logical tiles, then walk the tiles in groups of group_m token
  // tiles so that concurrently running tiles share operand rows in that L2.
  const int nwg = gridDim.x;
  const int bid = blockIdx.x;
  const int xcd = bid & 7, local = bid >> 3;
  const int per = nwg >> 3, rem = nwg & 7;
  const int lid = (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + local;
  const int group_size = group_m * tiles_n;
  const int first_m = (lid / group_size) * group_m;
  const int gm = min(tiles_m - first_m, group_m);
  const int tm = first_m + (lid % group_size) % gm;
  const int tn = (lid % group_size) / gm;
  const int n0 = tn * BN, m0 = tm * BM;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wn = wave % WN, wm = wave / WN;

  // ---- global -> LDS addressing --------------------------------------------
  const int rows_a = min(BN, N - n0), rows_b = min(BM, M - m0);
  const __amdgpu_buffer_rsrc_t rsrc_a = make_rsrc(Wq + (int64_t)n0 * K, (uint32_t)(rows_a * K));
  const __amdgpu_buffer_rsrc_t rsrc_b = make_rsrc(Xq + (int64_t)m0 * K, (uint32_t)(rows_b * K));
  const int lrow = lane / C::kChunks;                               // row within a load
  const int lchunk = (lane % C::kChunks) ^ (lrow % C::kChunks);     // logical chunk it fetches
  uint32_t off_a[C::kLoadsA], off_b[C::kLoadsB];
#pragma unroll
  for (int j = 0; j < C::kLoadsA; ++j)
    off_a[j] = (uint32_t)(((wave * C::kLoadsA + j) * C::kRowsPerLoad + lrow) * K + lchunk * 16);
#pragma unroll
  for (int j = 0; j < C::kLoadsB; ++j)
    off_b[j] = (uint32_t)(((wave * C::kLoadsB + j) * C::kRowsPerLoad + lrow) * K + lchunk * 16);


  // ---- LDS -> register fragment addressing ----------------------------------
  const int fr = lane & 31, fh = lane >> 5;
  int frag_off[BK / 32];
#pragma unroll
  for (int s = 0; s < BK / 32; ++s) frag_off[s] = fr * BK + (((2 * s + fh) ^ (fr % C::kChunks)) * 16);
  const int a_base = wn * C::kTN * BK;
  const int b_base = C::kABytes + wm * C::kTM * BK;

  v16i acc[C::kFN][C::kFM];
#pragma unroll
  for (int f = 0; f < C::kFN; ++f)
#pragma unroll
    for (int g = 0; g < C::kFM; ++g) acc[f][g] = v16i{};

  const int KT = (K + BK - 1) / BK;
  prefill_load_tile<BN, BM, BK, WN, WM>(rsrc_a, rsrc_b, off_a, off_b, lchunk, wave, K, 0, smem);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT)
      prefill_load_tile<BN, BM, BK, WN, WM>(rsrc_a, rsrc_b, off_a, off_b, lchunk, wave, K,
                                            (kt + 1) * BK, smem + (cur ^ 1) * C::kStage);
    const int8_t *st = smem + cur * C::kStage;
#pragma unroll
    for (int s = 0; s < BK / 32; ++s) {
      v4i a[C::kFN], b[C::kFM];
#pragma unroll
      for (int f = 0; f < C::kFN; ++f)
        a[f] = *reinterpret_cast<const v4i *>(st + a_base + f * 32 * BK + frag_off[s]);
#pragma unroll
      for (int g = 0; g < C::kFM; ++g)
        b[g] = *reinterpret_cast<const v4i *>(st + b_base + g * 32 * BK + frag_off[s]);
#pragma unroll
      for (int f = 0; f < C::kFN; ++f)
#pragma unroll
        for (int g = 0; g < C::kFM; ++g)
          acc[f][g] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[f], b[g], acc[f][g], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // ---- epilogue ----------------------------------------------------------------
  // 32x32 output block, 16 values per lane: lane l holds column (l mod 32)
  // and rows 8*(r/4) + 4*(l/32) + (r mod 4) for register r.  Columns are
  // tokens here and rows are channels, so registers 4j..4j+3 are four
  // consecutive channels of one token.
#pragma unroll
  for (int f = 0; f < C::kFN; ++f)
#pragma unroll
    for (int g = 0; g < C::kFM; ++g) {
      const int64_t m = m0 + wm * C::kTM + g * 32 + fr;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t n = n0 + wn * C::kTN + f * 32 + 8 * j + 4 * fh;
        store4(Y, acc_out, sW, bp, m, n, M, N, acc[f][g][4 * j], acc[f][g][4 * j + 1],
               acc[f][g][4 * j + 2], acc[f][g][4 * j + 3]);
      }
    }
}

template <int BN, int BM, int BK, int WN, int WM>
hipError_t launch_prefill(const int8_t *Xq, const int8_t *Wq, const float *sW, const float *bp,
                          int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                          hipStream_t st) {
  const int tiles_m = (int)((M + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
  const int group_m = 8;
  const unsigned grid = (unsigned)(tiles_m * tiles_n);
  qgemm_prefill_kernel<BN, BM, BK, WN, WM><<<grid, 64 * WN * WM, 0, st>>>(
      Xq, Wq, sW, bp, (int)M, (int)N, (int)K, Y, acc_out, tiles_m, tiles_n, group_m);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Decode (M <= 64): weight-streaming GEMV-like kernel on v_mfma_i32_16x16x64_i8
// ---------------------------------------------------------------------------
// HBM-bound on the weight bytes.  A workgroup owns 16*RB weight rows and all
// tokens (MB blocks of 16, zero-padded), and its kWaves waves split K in
// 64-byte steps, interleaved, so that together they stream whole cache lines
// of each row.  Each lane loads 16 bytes of one weight row per step (a wave
// covers 16 rows x 64 contiguous bytes), and the matching 16 bytes of each
// token row, which stay in L2 across workgroups.  U steps are kept in flight
// per wave.  The partial accumulators of the waves are summed in LDS and the
// epilogue is fused.
constexpr int kDecWaves = 8;

template <int MB, int RB, int U>
__global__ __launch_bounds__(64 * kDecWaves) void qgemm_decode_kernel(
    const int8_t *__restrict__ Xq, const int8_t *__restrict__ Wq, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, int K, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out) {
  __shared__ v4i red[kDecWaves][RB][MB][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16 * RB;
  const int rows_w = min(16 * RB, N - n0);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(Wq + (int64_t)n0 * K, (uint32_t)(rows_w * K));
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(Xq, (uint32_t)(M * K));
  const int r16 = lane & 15, c4 = lane >> 4;
  // byte offsets of this lane's 16-byte piece within a 64-byte step
  uint32_t offw[RB], offx[MB];
#pragma unroll
  for (int i = 0; i < RB; ++i) offw[i] = (uint32_t)((i * 16 + r16) * K + c4 * 16);
#pragma unroll
  for (int i = 0; i < MB; ++i) offx[i] = (uint32_t)((i * 16 + r16) * K + c4 * 16);

  v4i acc[RB][MB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) acc[i][j] = v4i{};

  const int steps = (K + 63) / 64;
  for (int s0 = wave; s0 < steps; s0 += kDecWaves * U) {
    v4i w[U][RB], x[U][MB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u * kDecWaves;
      const int k = s * 64 + c4 * 16;
      const bool ok = s < steps && k < K;
#pragma unroll
      for (int i = 0; i < RB; ++i)
        w[u][i] = __builtin_amdgcn_raw_buffer_load_b128(rw, ok ? offw[i] + (uint32_t)(s * 64) : kOobOffset, 0, 0);
#pragma unroll
      for (int j = 0; j < MB; ++j)
        x[u][j] = __builtin_amdgcn_raw_buffer_load_b128(rx, ok ? offx[j] + (uint32_t)(s * 64) : kOobOffset, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(w[u][i], x[u][j], acc[i][j], 0, 0, 0);
  }

#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) red[wave][i][j][lane] = acc[i][j];
  __syncthreads();
  // 16x16 output block, 4 values per lane: lane l holds column (l mod 16) and
  // rows 4*(l/16) + r.  Rows are channels, columns tokens.
  for (int t = wave; t < RB * MB; t += kDecWaves) {
    const int i = t / MB, j = t % MB;
    v4i sum = v4i{};
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) sum += red[w][i][j][lane];
    const int64_t m = j * 16 + r16;
    const int64_t n = n0 + i * 16 + 4 * c4;
    store4(Y, acc_out, sW, bp, m, n, M, N, sum[0], sum[1], sum[2], sum[3]);
  }
}

template <int MB, int RB, int U>
hipError_t launch_decode(const int8_t *Xq, const int8_t *Wq, const float *sW, const float *bp,
                         int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                         hipStream_t st) {
  const unsigned grid = (unsigned)((N + 16 * RB - 1) / (16 * RB));
  qgemm_decode_kernel<MB, RB, U><<<grid, 64 * kDecWaves, 0, st>>>(
      Xq, Wq, sW, bp, (int)M, (int)N, (int)K, Y, acc_out);
  return hipGetLastError();
}

}  // namespace detail

using namespace detail;

hipError_t launch_qgemm(const int8_t *Xq, const int8_t *Wq, const float *sW, const float *bprime,
                        int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                        hipStream_t st) {
  if (M <= 16) return launch_decode<1, 1, 4>(Xq, Wq, sW, bprime, M, N, K, Y, acc_out, st);
  if (M <= 32) return launch_decode<2, 1, 4>(Xq, Wq, sW, bprime, M, N, K, Y, acc_out, st);
  if (M <= 64) return launch_decode<4, 1, 2>(Xq, Wq, sW, bprime, M, N, K, Y, acc_out, st);
  return launch_prefill<256, 256, 128, 2, 2>(Xq, Wq, sW, bprime, M, N, K, Y, acc_out, st);
}

}  // namespace ot
