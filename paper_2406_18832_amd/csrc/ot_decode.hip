// Decode GEMM of the quantized linear (at most 64 tokens), bound by
// streaming the weights from HBM.
#include <algorithm>

#include <stdio.h>

#include "ot_gemm_common.h"

namespace ot {
namespace detail {

// ---------------------------------------------------------------------------
// Shared-token ring: one LDS ring for tokens and (row-major) weights
// ---------------------------------------------------------------------------
// Loading the token fragments into every wave's registers would limit how
// far ahead a wave can fetch (and repeat the token loads per wave).  The
// NW = NR x NK waves of a workgroup step through K together over one ring of
// S stages (packed weights bypass it: decode_body_packed).  A stage
// holds the token tile [16*MB rows][BKD] and the workgroup's weight tile
// [16*RBW*NR rows][BKD], both filled by buffer load-to-LDS S-1 stages ahead
// with the loads spread evenly over all waves; one barrier per stage.  Wave
// (rg, kg) multiplies weight rows 16*RBW*rg.. by every token over the kg-th
// 1/NK of the stage's 64-byte K steps; the NK partial sums of a row group are
// added through LDS at the end (integer sums, so the order is immaterial).
// Chunk c of stage row r sits at chunk c ^ swz_rows(r), which keeps both the
// fragment reads and the DMA writes free of bank conflicts.
template <int MB, int NR, int NK, int RBW, int BKD, int S>
struct DecodeCfg {
  static constexpr int kWaves = NR * NK;
  static constexpr int kTokRows = 16 * MB;
  static constexpr int kWRows = 16 * RBW * NR;
  static constexpr int kRows = kTokRows + kWRows;
  static constexpr int kChunks = BKD / 16;
  static constexpr int kSteps = BKD / 64 / NK;  // 64-byte K steps per wave per stage
  static constexpr int kStage = kRows * BKD;
  static constexpr int kRowsPerLoad = 1024 / BKD;
  static constexpr int kLoads = kStage / 1024 / kWaves;  // per wave per stage
  static constexpr int kRed = (NK - 1) * NR * RBW * MB * 1024;  // partial sums, bytes
  static constexpr int kRedRs = (NK - 1) * MB * 64 * 4;         // token code sums, bytes
  static_assert(BKD == 128 || BKD == 256 || BKD == 512, "BKD");
  static_assert(kSteps >= 1 && kSteps * 64 * NK == BKD, "K steps split evenly over NK");
  static_assert(kTokRows % kRowsPerLoad == 0, "a load never straddles tokens and weights");
  static_assert(S >= 2, "stages");
  // packed weights: the LDS ring holds the token tile only
  static constexpr int kTokStage = kTokRows * BKD;
  static constexpr int kTokLoads = kTokStage / 1024 / kWaves;  // per wave per stage
  static constexpr int kLoadsPacked = kTokLoads + RBW * kSteps;
  static constexpr int kSmemPacked =
      S * kTokStage > kRed + kRedRs ? S * kTokStage : kRed + kRedRs;
  static constexpr int smem_bytes(bool packed) { return packed ? kSmemPacked : S * kStage; }
};

// cache-policy operand of a buffer load on gfx950: non-temporal
constexpr int kNonTemporal = 2;

// No memory access moves across this point at compile time (it emits no
// instruction).
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Packed weights (PACKED): Wq re-laid as 1 KiB micro-tiles of 16 rows by 64
// K bytes, [ceil(N/16)][ceil(K/64)][64 lanes][16 bytes], each in the lane
// order of the A operand of v_mfma_i32_16x16x64_i8 (lane l: row l mod 16,
// bytes 16 (l / 16) .. +15 of the 64), zeros past N and K.  A micro-tile is
// then one wave's A fragment and one contiguous 1 KiB load, so each wave
// streams its own weights straight into registers (no LDS round trip), and
// only the token tile, which all row groups share, goes through LDS.
constexpr int kMicroTile = 1024;

template <int kChunks>
__device__ __forceinline__ int swz_rows(int r) {
  if constexpr (kChunks == 8) return (r & 7) ^ ((r >> 3) & 1);
  else return r & 15;
}

// The epilogue's per-channel scale, bias and zero point (RBW groups of four
// channels per lane) and per-token scales (MB tokens per lane), loaded at
// the start of the kernel so that their latency passes during the K loop
// instead of after it.  Only the waves that run the epilogue (K group 0)
// load them; a split run has no epilogue.
template <int RBW, int MB>
struct EpiParams {
  float4 s4[RBW], b4[RBW];
  int4 z4[RBW];
  float sx[MB];
};

template <int MB, int RBW, int EPI, bool SPLIT>
__device__ __forceinline__ void epi_preload(EpiParams<RBW, MB> &ep, const float *__restrict__ sX,
                                            const int32_t *__restrict__ zW,
                                            const float *__restrict__ sW,
                                            const float *__restrict__ bp, int lane, int rg, int kg,
                                            int nwg0, int M, int N) {
  if constexpr (!SPLIT) {
    const int r16 = lane & 15, c4 = lane >> 4;
    if (kg == 0) {
#pragma unroll
      for (int i = 0; i < RBW; ++i)
        load_epi4<EPI>(sW, bp, zW, (int64_t)nwg0 + (rg * RBW + i) * 16 + 4 * c4, N, ep.s4[i],
                       ep.b4[i], ep.z4[i]);
#pragma unroll
      for (int j = 0; j < MB; ++j) {
        const int m = j * 16 + r16;
        ep.sx[j] = (EPI == kEpiToken && m < M) ? sX[m] : 0.f;
      }
    }
  }
}

// Keeps the compiler from sinking the preloads to their use after the K
// loop (it emits no instruction; the values are ready by then).
template <int RBW, int MB>
__device__ __forceinline__ void epi_pin(EpiParams<RBW, MB> &ep) {
#pragma unroll
  for (int i = 0; i < RBW; ++i) {
    asm volatile("" : "+v"(ep.s4[i].x), "+v"(ep.s4[i].y), "+v"(ep.s4[i].z), "+v"(ep.s4[i].w));
    asm volatile("" : "+v"(ep.b4[i].x), "+v"(ep.b4[i].y), "+v"(ep.b4[i].z), "+v"(ep.b4[i].w));
    asm volatile("" : "+v"(ep.z4[i].x), "+v"(ep.z4[i].y), "+v"(ep.z4[i].z), "+v"(ep.z4[i].w));
  }
#pragma unroll
  for (int j = 0; j < MB; ++j) asm volatile("" : "+v"(ep.sx[j]));
}

// After the K loop: the asymmetric-weight token code sums, the K groups'
// partial sums added through LDS, then either the epilogue (dequantize,
// bias, fp16 store) or, split, the run's int32 partial sums.
template <int MB, int NR, int NK, int RBW, int BKD, int S, int EPI, bool SPLIT>
__device__ __forceinline__ void decode_finish(
    int8_t *smem, v4i (&acc)[RBW][MB], int (&rs)[MB], const EpiParams<RBW, MB> &ep, int lane,
    int rg, int kg, int nwg0, int M, int N, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out, int32_t *__restrict__ part, int32_t *__restrict__ part_rs) {
  using C = DecodeCfg<MB, NR, NK, RBW, BKD, S>;
  const int r16 = lane & 15, c4 = lane >> 4;

  // asymmetric weights: token code sums over this wave's K slice (the four
  // 16-lane groups hold the four 16-byte parts of every 64-byte step)
  if constexpr (EPI == kEpiAsym) {
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      rs[j] += __shfl_xor(rs[j], 16);
      rs[j] += __shfl_xor(rs[j], 32);
    }
  }

  if constexpr (NK > 1) {
    lds_barrier();
    v4i *red = reinterpret_cast<v4i *>(smem);
    int *red_rs = reinterpret_cast<int *>(smem + C::kRed);  // [NK-1][MB][64]
    if (kg > 0) {
#pragma unroll
      for (int i = 0; i < RBW; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
          red[((((kg - 1) * NR + rg) * RBW + i) * MB + j) * 64 + lane] = acc[i][j];
      if (EPI == kEpiAsym && rg == 0) {
#pragma unroll
        for (int j = 0; j < MB; ++j) red_rs[((kg - 1) * MB + j) * 64 + lane] = rs[j];
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);
    lds_barrier();
    if (kg > 0) return;
#pragma unroll
    for (int g = 0; g < NK - 1; ++g) {
#pragma unroll
      for (int i = 0; i < RBW; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
          acc[i][j] += red[(((g * NR + rg) * RBW + i) * MB + j) * 64 + lane];
      if constexpr (EPI == kEpiAsym) {
#pragma unroll
        for (int j = 0; j < MB; ++j) rs[j] += red_rs[(g * MB + j) * 64 + lane];
      }
    }
  }

  // 16x16 output blocks: lane l holds token l%16 and channels 4*(l/16) + r
  if constexpr (SPLIT) {
    const int64_t slab = (int64_t)blockIdx.y * M;
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int m = j * 16 + r16;
      if (m >= M) continue;
#pragma unroll
      for (int i = 0; i < RBW; ++i) {
        const int64_t n = nwg0 + (rg * RBW + i) * 16 + 4 * c4;
        int32_t *dst = part + (slab + m) * N + n;
        if (n + 3 < N && (N & 3) == 0) {
          *reinterpret_cast<v4i *>(dst) = acc[i][j];
        } else {
          for (int e = 0; e < 4; ++e)
            if (n + e < N) dst[e] = acc[i][j][e];
        }
      }
      if (EPI == kEpiAsym && blockIdx.x == 0 && rg == 0 && c4 == 0) part_rs[slab + m] = rs[j];
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < MB; ++j) {
    const int m = j * 16 + r16;
#pragma unroll
    for (int i = 0; i < RBW; ++i) {
      const int64_t n = nwg0 + (rg * RBW + i) * 16 + 4 * c4;
      store4_pre<EPI>(Y, acc_out, ep.s4[i], ep.b4[i], ep.z4[i], ep.sx[j], rs[j], m, n, M, N,
                      acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
}


// Split K (SPLIT): workgroup (x, y) takes the y-th run of `per` stages of K
// and, instead of the epilogue, writes its integer partial sums to
// part[y][m][n] (and, for asymmetric weights, the tokens' partial code sums
// to part_rs[y][m] from the first row tile); decode_reduce_kernel adds the
// runs and applies the epilogue.
template <int MB, int NR, int NK, int RBW, int BKD, int S, int EPI, bool SPLIT>
__device__ __forceinline__ void decode_body(
    int8_t *smem, const int8_t *__restrict__ Xq, const int8_t *__restrict__ Wq,
    const float *__restrict__ sX, const int32_t *__restrict__ zW, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, int K, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out, int32_t *__restrict__ part, int32_t *__restrict__ part_rs,
    int per) {
  using C = DecodeCfg<MB, NR, NK, RBW, BKD, S>;
  static_assert(C::kLoads >= 1 && C::kLoads * 1024 * C::kWaves == C::kStage,
                "stage splits evenly over the waves");
  static_assert((S - 2) * C::kLoads <= 63, "vmcnt range");
  static_assert(C::kRed + C::kRedRs <= S * C::kStage, "partial sums fit in the ring");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rg = wave % NR, kg = wave / NR;
  const int nwg0 = blockIdx.x * C::kWRows;  // first weight row of the workgroup
  const int rows_w = min(C::kWRows, N - nwg0);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(Wq + (int64_t)nwg0 * K, (uint32_t)(rows_w * K));
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(Xq, (uint32_t)(M * K));
  const int r16 = lane & 15, c4 = lane >> 4;
  EpiParams<RBW, MB> ep{};  // zeros where this wave loads none
  epi_preload<MB, RBW, EPI, SPLIT>(ep, sX, zW, sW, bp, lane, rg, kg, nwg0, M, N);

  // this wave's j-th load of a stage fills 1 KiB block q = wave*kLoads + j:
  // stage rows q*kRowsPerLoad.. (tokens below kTokRows, then weights)
  uint32_t goff[C::kLoads];
  int gck[C::kLoads];
#pragma unroll
  for (int j = 0; j < C::kLoads; ++j) {
    const int q = wave * C::kLoads + j;
    const int row = q * C::kRowsPerLoad + lane / C::kChunks;
    const int ch = (lane % C::kChunks) ^ swz_rows<C::kChunks>(row);
    gck[j] = ch * 16;
    const int grow = row < C::kTokRows ? row : row - C::kTokRows;
    goff[j] = (uint32_t)(grow * K + ch * 16);
  }
  // stages [st0, st0 + nst) of K; a split never starts past the last stage
  int st0 = 0, nst = (K + BKD - 1) / BKD;
  if constexpr (SPLIT) {
    st0 = blockIdx.y * per;
    nst = min(nst - st0, per);
  }
  auto issue = [&](int st) {
    int8_t *dst = smem + (st % S) * C::kStage;
    const int k0 = (st0 + st) * BKD;  // stages past this split's run are loaded but unused
#pragma unroll
    for (int j = 0; j < C::kLoads; ++j) {
      const int q = wave * C::kLoads + j;  // wave-uniform
      const uint32_t off = (goff[j] + (uint32_t)k0) | ((uint32_t)(k0 + gck[j] >= K) << 31);
      // weights are read once: non-temporal ("nt") keeps them from evicting
      // the token rows, which every workgroup re-reads, from the caches
      if (q * C::kRowsPerLoad < C::kTokRows)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void *)(dst + q * 1024), 16, off, 0, 0, 0);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void *)(dst + q * 1024), 16, off, 0, 0,
                                                 kNonTemporal);
    }
  };
  // fragment offsets within a stage: lane (r16, c4) of step t reads logical
  // chunk 4*(kg*kSteps + t) + c4 of weight row (this wave's block i) or
  // token row (block j)
  int fragw[C::kSteps][RBW], fragx[C::kSteps][MB];
#pragma unroll
  for (int t = 0; t < C::kSteps; ++t) {
    const int c = 4 * (kg * C::kSteps + t) + c4;
#pragma unroll
    for (int i = 0; i < RBW; ++i) {
      const int row = C::kTokRows + (rg * RBW + i) * 16 + r16;
      fragw[t][i] = row * BKD + 16 * (c ^ swz_rows<C::kChunks>(row));
    }
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int row = j * 16 + r16;
      fragx[t][j] = row * BKD + 16 * (c ^ swz_rows<C::kChunks>(row));
    }
  }

  v4i acc[RBW][MB];
#pragma unroll
  for (int i = 0; i < RBW; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) acc[i][j] = v4i{};
  int rs[MB];
#pragma unroll
  for (int j = 0; j < MB; ++j) rs[j] = 0;

#pragma unroll
  for (int t = 0; t < S - 1; ++t) issue(t);
  wait_vmcnt<(S - 2) * C::kLoads>();
  lds_barrier();
  epi_pin(ep);
  issue(S - 1);
  for (int st = 0; st < nst; ++st) {
    const int8_t *src = smem + (st % S) * C::kStage;
#pragma unroll
    for (int t = 0; t < C::kSteps; ++t) {
      v4i wf[RBW], xf[MB];
#pragma unroll
      for (int i = 0; i < RBW; ++i) wf[i] = *reinterpret_cast<const v4i *>(src + fragw[t][i]);
#pragma unroll
      for (int j = 0; j < MB; ++j) xf[j] = *reinterpret_cast<const v4i *>(src + fragx[t][j]);
#pragma unroll
      for (int i = 0; i < RBW; ++i)
#pragma unroll
        for (int j = 0; j < MB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf[i], xf[j], acc[i][j], 0, 0, 0);
      if constexpr (EPI == kEpiAsym) {
#pragma unroll
        for (int j = 0; j < MB; ++j) rs[j] = byte_sum16(xf[j], rs[j]);
      }
    }
    // stage st+1 has landed once at most S-2 younger stages are in flight;
    // after the barrier every wave is done with stage st, whose slot takes st+S
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    wait_vmcnt<(S - 2) * C::kLoads>();
    lds_barrier();
    issue(st + S);
  }
  // the ring's last (zero-filling) loads must land before its bytes are reused
  wait_vmcnt<0>();
  decode_finish<MB, NR, NK, RBW, BKD, S, EPI, SPLIT>(smem, acc, rs, ep, lane, rg, kg, nwg0, M,
                                                     N, Y, acc_out, part, part_rs);
}

// Packed weights: wave (rg, kg) loads the micro-tiles of its RBW row blocks
// and its 1/NK of each stage's K steps into a register ring of S stages (the
// K loop is unrolled by S so that every ring slot is a fixed register set);
// the token tile takes the LDS ring as in decode_body.  Past the last stage
// of the run every load is out of range and returns zeros, so the loop runs
// whole groups of S stages and the extra ones add nothing.  The vmcnt waits
// are counted by hand over the program order of the loads, so the weight
// pointer carries no __restrict__ and a compiler fence closes each stage's
// group of loads: a register load from memory the compiler may not assume
// unchanged then stays between the fences and barriers (which clobber
// memory) around it, instead of moving past a wait.
template <int MB, int NR, int NK, int RBW, int BKD, int S, int EPI, bool SPLIT>
__device__ __forceinline__ void decode_body_packed(
    int8_t *smem, const int8_t *__restrict__ Xq, const int8_t *Wp,
    const float *__restrict__ sX, const int32_t *__restrict__ zW, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, int K, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out, int32_t *__restrict__ part, int32_t *__restrict__ part_rs,
    int per) {
  using C = DecodeCfg<MB, NR, NK, RBW, BKD, S>;
  constexpr int kTL = C::kTokLoads, kL = C::kLoadsPacked;
  static_assert(kTL >= 1 && kTL * 1024 * C::kWaves == C::kTokStage,
                "token tile splits evenly over the waves");
  static_assert((S - 2) * kL <= 63, "vmcnt range");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rg = wave % NR, kg = wave / NR;
  const int nwg0 = blockIdx.x * C::kWRows;  // first weight row of the workgroup
  constexpr int kMT = BKD / 64;              // micro-tiles per row group and stage
  const int KS = (K + 63) / 64;              // micro-tiles per row group
  const int groups_w = min(C::kWRows / 16, (N + 15) / 16 - nwg0 / 16);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(Wp + (int64_t)(nwg0 / 16) * KS * kMicroTile,
                                              (uint32_t)groups_w * (uint32_t)KS * kMicroTile);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(Xq, (uint32_t)(M * K));
  const int r16 = lane & 15, c4 = lane >> 4;
  EpiParams<RBW, MB> ep{};  // zeros where this wave loads none
  epi_preload<MB, RBW, EPI, SPLIT>(ep, sX, zW, sW, bp, lane, rg, kg, nwg0, M, N);

  // token loads: this wave's j-th fills 1 KiB block q = wave*kTL + j of the
  // stage's token rows
  uint32_t xoff[kTL];
  int xck[kTL];
#pragma unroll
  for (int j = 0; j < kTL; ++j) {
    const int row = (wave * kTL + j) * C::kRowsPerLoad + lane / C::kChunks;
    const int ch = (lane % C::kChunks) ^ swz_rows<C::kChunks>(row);
    xck[j] = ch * 16;
    xoff[j] = (uint32_t)(row * K + ch * 16);
  }
  // weight micro-tile (i, t): row group rg*RBW + i, K micro-tile kg*kSteps + t
  // of the stage
  uint32_t woff[RBW];
#pragma unroll
  for (int i = 0; i < RBW; ++i) woff[i] = (uint32_t)((rg * RBW + i) * KS) * kMicroTile + lane * 16;

  int st0 = 0, nst = (K + BKD - 1) / BKD;
  if constexpr (SPLIT) {
    st0 = blockIdx.y * per;
    nst = min(nst - st0, per);
  }
  v4i wr[S][RBW][C::kSteps];
  auto issue = [&](int st, int slot) {
    int8_t *dst = smem + slot * C::kTokStage;
    const uint32_t past = st >= nst ? 1u : 0u;  // wave-uniform: beyond this run
    const int k0 = (st0 + st) * BKD;
#pragma unroll
    for (int j = 0; j < kTL; ++j) {
      const uint32_t oob = past | (uint32_t)(k0 + xck[j] >= K);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void *)(dst + (wave * kTL + j) * 1024), 16,
                                               (xoff[j] + (uint32_t)k0) | (oob << 31), 0, 0, 0);
    }
    const int mt0 = (st0 + st) * kMT + kg * C::kSteps;
#pragma unroll
    for (int i = 0; i < RBW; ++i)
#pragma unroll
      for (int t = 0; t < C::kSteps; ++t) {
        const uint32_t oob = past | (uint32_t)(mt0 + t >= KS);
        const uint32_t off = (woff[i] + (uint32_t)(mt0 + t) * kMicroTile) | (oob << 31);
        wr[slot][i][t] = __builtin_bit_cast(
            v4i, __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, kNonTemporal));
      }
  };
  // token fragment offsets within a stage (as in decode_body)
  int fragx[C::kSteps][MB];
#pragma unroll
  for (int t = 0; t < C::kSteps; ++t) {
    const int c = 4 * (kg * C::kSteps + t) + c4;
#pragma unroll
    for (int j = 0; j < MB; ++j) {
      const int row = j * 16 + r16;
      fragx[t][j] = row * BKD + 16 * (c ^ swz_rows<C::kChunks>(row));
    }
  }

  v4i acc[RBW][MB];
#pragma unroll
  for (int i = 0; i < RBW; ++i)
#pragma unroll
    for (int j = 0; j < MB; ++j) acc[i][j] = v4i{};
  int rs[MB];
#pragma unroll
  for (int j = 0; j < MB; ++j) rs[j] = 0;

  // each issue() group stays between the fences: the hand-counted waits
  // below see the loads in stage order
#pragma unroll
  for (int t = 0; t < S - 1; ++t) {
    issue(t, t);
    compiler_fence();
  }
  wait_vmcnt<(S - 2) * kL>();
  lds_barrier();
  epi_pin(ep);
  issue(S - 1, S - 1);
  const int nrun = (nst + S - 1) / S * S;  // nst >= 1
  int base = 0;
  do {
#pragma unroll
    for (int slot = 0; slot < S; ++slot) {
      const int8_t *src = smem + slot * C::kTokStage;
#pragma unroll
      for (int t = 0; t < C::kSteps; ++t) {
        v4i xf[MB];
#pragma unroll
        for (int j = 0; j < MB; ++j) xf[j] = *reinterpret_cast<const v4i *>(src + fragx[t][j]);
#pragma unroll
        for (int i = 0; i < RBW; ++i)
#pragma unroll
          for (int j = 0; j < MB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wr[slot][i][t], xf[j], acc[i][j], 0,
                                                               0, 0);
        if constexpr (EPI == kEpiAsym) {
#pragma unroll
          for (int j = 0; j < MB; ++j) rs[j] = byte_sum16(xf[j], rs[j]);
        }
      }
      // stage base+slot+1 has landed once at most S-2 younger stages are in
      // flight; after the barrier every wave is done with this slot
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
      compiler_fence();
      wait_vmcnt<(S - 2) * kL>();
      lds_barrier();
      issue(base + slot + S, slot);
    }
    base += S;
  } while (base < nrun);
  // the last (zero-filling) loads must land before the ring is reused
  wait_vmcnt<0>();
  decode_finish<MB, NR, NK, RBW, BKD, S, EPI, SPLIT>(smem, acc, rs, ep, lane, rg, kg, nwg0, M,
                                                     N, Y, acc_out, part, part_rs);
}

template <int MB, int NR, int NK, int RBW, int BKD, int S, int EPI, bool PACKED>
__global__ __launch_bounds__(64 * NR * NK) void qgemm_decode_kernel(
    const int8_t *__restrict__ Xq, const int8_t *Wq, const float *__restrict__ sX,
    const int32_t *__restrict__ zW, const float *__restrict__ sW, const float *__restrict__ bp,
    int M, int N, int K, uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out) {
  __shared__ __attribute__((aligned(1024)))
  int8_t smem[DecodeCfg<MB, NR, NK, RBW, BKD, S>::smem_bytes(PACKED)];
  if constexpr (PACKED)
    decode_body_packed<MB, NR, NK, RBW, BKD, S, EPI, false>(smem, Xq, Wq, sX, zW, sW, bp, M, N, K,
                                                            Y, acc_out, nullptr, nullptr, 0);
  else
    decode_body<MB, NR, NK, RBW, BKD, S, EPI, false>(smem, Xq, Wq, sX, zW, sW, bp, M, N, K, Y,
                                                     acc_out, nullptr, nullptr, 0);
}

// Split-K partial sums (ROWSUM: also the token code sums of asymmetric weights).
template <int MB, int NR, int NK, int RBW, int BKD, int S, bool ROWSUM, bool PACKED>
__global__ __launch_bounds__(64 * NR * NK) void qgemm_decode_split_kernel(
    const int8_t *__restrict__ Xq, const int8_t *Wq, int M, int N, int K,
    int32_t *__restrict__ part, int32_t *__restrict__ part_rs, int per) {
  __shared__ __attribute__((aligned(1024)))
  int8_t smem[DecodeCfg<MB, NR, NK, RBW, BKD, S>::smem_bytes(PACKED)];
  constexpr int kE = ROWSUM ? kEpiAsym : kEpiChannel;
  if constexpr (PACKED)
    decode_body_packed<MB, NR, NK, RBW, BKD, S, kE, true>(smem, Xq, Wq, nullptr, nullptr, nullptr,
                                                          nullptr, M, N, K, nullptr, nullptr, part,
                                                          part_rs, per);
  else
    decode_body<MB, NR, NK, RBW, BKD, S, kE, true>(smem, Xq, Wq, nullptr, nullptr, nullptr,
                                                   nullptr, M, N, K, nullptr, nullptr, part,
                                                   part_rs, per);
}

// Adds the split runs' partial sums (integer sums, so any order gives the
// same result) and applies the epilogue: thread t takes channels
// 4 (t mod N4) .. +3 of token t / N4.  Every run's 16-byte partial is
// loaded before any is added (at most kMaxRuns runs), so the loads are in
// flight together.
constexpr int kMaxRuns = 8;

template <int EPI>
__global__ __launch_bounds__(256) void decode_reduce_kernel(
    const int32_t *__restrict__ part, const int32_t *__restrict__ part_rs, int splits,
    const float *__restrict__ sX, const int32_t *__restrict__ zW, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out) {
  const int n4 = (N + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)M * n4) return;
  const int m = (int)(t / n4), n = 4 * (int)(t % n4);
  const int64_t run_stride = (int64_t)M * N;
  const int32_t *src = part + (int64_t)m * N + n;
  int a[4] = {0, 0, 0, 0};
  int rs = 0;
  if (n + 3 < N && (N & 3) == 0) {
    v4i v[kMaxRuns];
#pragma unroll
    for (int s = 0; s < kMaxRuns; ++s)
      if (s < splits) v[s] = *reinterpret_cast<const v4i *>(src + s * run_stride);
#pragma unroll
    for (int s = 0; s < kMaxRuns; ++s)
      if (s < splits) {
        a[0] += v[s][0]; a[1] += v[s][1]; a[2] += v[s][2]; a[3] += v[s][3];
      }
  } else {
    for (int s = 0; s < splits; ++s)
      for (int e = 0; e < 4; ++e)
        if (n + e < N) a[e] += src[s * run_stride + e];
  }
  if constexpr (EPI == kEpiAsym) {
    for (int s = 0; s < splits; ++s) rs += part_rs[(int64_t)s * M + m];
  }
  const float sx = EPI == kEpiToken ? sX[m] : 0.f;
  store4<EPI>(Y, acc_out, sW, bp, zW, sx, rs, m, n, M, N, a[0], a[1], a[2], a[3]);
}

// At most `runs` runs of whole BKD-byte stages (fewer where the stages do
// not divide so; never an empty run).
template <int MB, int NR, int NK, int RBW, int BKD, int S, bool PACKED>
hipError_t launch_decode_split(const int8_t *Xq, const int8_t *Wq, const float *sX,
                               const int32_t *zW, const float *sW, const float *bp, int64_t M,
                               int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out, int runs,
                               int32_t *part, int32_t *part_rs, hipStream_t st) {
  constexpr int rows = 16 * RBW * NR;
  const int64_t nst = (K + BKD - 1) / BKD;
  const int per = (int)((nst + runs - 1) / runs);
  const int splits = (int)((nst + per - 1) / per);
  const dim3 grid((unsigned)((N + rows - 1) / rows), (unsigned)splits);
  const dim3 block(64 * NR * NK);
  if (zW)
    qgemm_decode_split_kernel<MB, NR, NK, RBW, BKD, S, true, PACKED><<<grid, block, 0, st>>>(
        Xq, Wq, (int)M, (int)N, (int)K, part, part_rs, per);
  else
    qgemm_decode_split_kernel<MB, NR, NK, RBW, BKD, S, false, PACKED><<<grid, block, 0, st>>>(
        Xq, Wq, (int)M, (int)N, (int)K, part, part_rs, per);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned rgrid = (unsigned)((M * ((N + 3) / 4) + 255) / 256);
  if (sX)
    decode_reduce_kernel<kEpiToken><<<rgrid, 256, 0, st>>>(part, part_rs, splits, sX, zW, sW, bp,
                                                            (int)M, (int)N, Y, acc_out);
  else if (zW)
    decode_reduce_kernel<kEpiAsym><<<rgrid, 256, 0, st>>>(part, part_rs, splits, sX, zW, sW, bp,
                                                           (int)M, (int)N, Y, acc_out);
  else
    decode_reduce_kernel<kEpiChannel><<<rgrid, 256, 0, st>>>(part, part_rs, splits, sX, zW, sW,
                                                              bp, (int)M, (int)N, Y, acc_out);
  return hipGetLastError();
}

// Epilogue by argument: sX != nullptr per-token scales sX [M]; zW != nullptr
// asymmetric weight zero points zW [N]; neither: per-channel.
template <int MB, int NR, int NK, int RBW, int BKD, int S, bool PACKED>
hipError_t launch_decode_t(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                           const float *sW, const float *bp, int64_t M, int64_t N, int64_t K,
                           uint16_t *Y, int32_t *acc_out, hipStream_t st) {
  constexpr int rows = 16 * RBW * NR;
  const unsigned grid = (unsigned)((N + rows - 1) / rows);
  const dim3 block(64 * NR * NK);
  if (sX)
    qgemm_decode_kernel<MB, NR, NK, RBW, BKD, S, kEpiToken, PACKED><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out);
  else if (zW)
    qgemm_decode_kernel<MB, NR, NK, RBW, BKD, S, kEpiAsym, PACKED><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out);
  else
    qgemm_decode_kernel<MB, NR, NK, RBW, BKD, S, kEpiChannel, PACKED><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out);
  return hipGetLastError();
}

// Weight layout by argument: packed micro-tiles or Wq [N x K].
template <int MB, int NR, int NK, int RBW, int BKD, int S>
hipError_t launch_decode(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                         const float *sW, const float *bp, int64_t M, int64_t N, int64_t K,
                         uint16_t *Y, int32_t *acc_out, bool packed, hipStream_t st) {
  if (packed)
    return launch_decode_t<MB, NR, NK, RBW, BKD, S, true>(Xq, Wq, sX, zW, sW, bp, M, N, K, Y,
                                                          acc_out, st);
  return launch_decode_t<MB, NR, NK, RBW, BKD, S, false>(Xq, Wq, sX, zW, sW, bp, M, N, K, Y,
                                                         acc_out, st);
}

// Packs Wq [N x K] into micro-tiles (see PACKED above): thread t writes the
// 16 bytes of lane t mod 64 of micro-tile t / 64.
__global__ __launch_bounds__(256) void pack_weights_kernel(const int8_t *__restrict__ Wq,
                                                           int64_t N, int64_t K, int64_t KS,
                                                           int64_t chunks,
                                                           int8_t *__restrict__ Wp) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= chunks) return;
  const int l = (int)(t & 63);
  const int64_t mt = t >> 6;  // micro-tile: row group mt / KS, K step mt mod KS
  const int64_t row = (mt / KS) * 16 + (l & 15);
  const int64_t col = (mt % KS) * 64 + 16 * (l >> 4);
  uint4 v = make_uint4(0, 0, 0, 0);
  if (row < N && col < K) v = *reinterpret_cast<const uint4 *>(Wq + row * K + col);
  reinterpret_cast<uint4 *>(Wp)[t] = v;
}

}  // namespace detail

using namespace detail;

// Launch plan for 17-64 tokens: the tile height (weight rows per workgroup)
// and the number of K runs (split K: each run writes int32 partial sums
// that a second kernel adds up).  Every candidate grid fits one pass over
// the CUs (the tiles are sized for one workgroup per CU); the plan with the
// least estimated time wins, and the same plan serves both weight layouts
// (so the workspace size does not depend on the layout).  The estimate, in microseconds, was fitted to
// every (tile height, runs) pair measured on MI355X for 13 layer shapes
// (N = 2048 .. 21504, K = 2048 .. 36864) at 24, 32, 48 and 64 tokens, and
// keeps the fit's physical reading:
//   each CU streams its weight rows plus the token rows (L2 hits, counted
//   half) of its K run at ~40 GB/s;
//   the whole chip streams the weights from HBM at ~6 TB/s, and weights
//   plus every tile's token re-read from L2 at ~10 TB/s;
//   a split adds ~2 us (the reduce launch) plus its runs x M x N int32
//   partial sums, written and read back at ~2 TB/s.
// Taller tiles re-read the token tile less (M / rows bytes per weight
// byte); splits fill CUs that short, wide-K layers would leave idle.
struct DecodePlan {
  int rows;  // 32, 64, 96 or 128
  int runs;  // K runs, at most; 1 = one kernel with the epilogue
};

static double plan_cost(int64_t M, int64_t N, int64_t K, int rows, int runs, int64_t cus) {
  const double chip = (double)cus / 256.0;  // bandwidths below are for 256 CUs
  const double kr = (double)K / runs;
  const double tiles = (double)((N + rows - 1) / rows);
  const double per_cu = (rows + 0.5 * M) * kr / 40e3;
  const double hbm = (double)N * K / (6e6 * chip);
  const double l2 = ((double)N * K + tiles * M * K) / (10e6 * chip);
  double t = std::max(per_cu, std::max(hbm, l2));
  if (runs > 1) t += 2.0 + (double)runs * M * N * 8 / (2e6 * chip);
  return t;
}

static DecodePlan decode_plan(int64_t M, int64_t N, int64_t K, int64_t cus, bool split) {
  // past 128 rows per CU no grid fits one pass: 64-row tiles keep the last
  // pass's tail short
  DecodePlan best{64, 1};
  double best_t = 0;
  const int64_t k256 = (K + 255) / 256;  // 256-byte K slices
  for (int rows : {32, 64, 96, 128}) {
    const int64_t tiles = (N + rows - 1) / rows;
    if (tiles > cus) continue;
    for (int runs = 1; runs <= (split ? kMaxRuns : 1) && tiles * runs <= cus; ++runs) {
      if (runs > 1 && k256 < 4 * runs) break;  // runs of at least 1 KiB of K
      const double t = plan_cost(M, N, K, rows, runs, cus);
      if (best_t == 0 || t < best_t) {
        best = DecodePlan{rows, runs};
        best_t = t;
      }
    }
  }
  return best;
}

size_t qgemm_decode_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M <= 16 || M > 64) return 0;
  const DecodePlan p = decode_plan(M, N, K, device_cus(), true);
  return p.runs > 1 ? (size_t)p.runs * (size_t)M * (size_t)(N + 1) * sizeof(int32_t) : 0;
}

size_t packed_weights_bytes(int64_t N, int64_t K) {
  return (size_t)((N + 15) / 16) * (size_t)((K + 63) / 64) * kMicroTile;
}

hipError_t launch_pack_weights(const int8_t *Wq, int64_t N, int64_t K, int8_t *Wp,
                               hipStream_t st) {
  const int64_t KS = (K + 63) / 64;
  const int64_t chunks = (N + 15) / 16 * KS * 64;
  pack_weights_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, st>>>(Wq, N, K, KS, chunks, Wp);
  return hipGetLastError();
}

// One tile configuration <token blocks, row groups, K groups, row blocks
// per wave, BKD, stages> per (17-32 or 33-64 tokens, tile height, weight
// layout), each the fastest in sweeps of the valid configurations on MI355X
// (row-major and packed weights load differently, so their best stage
// shapes differ).
template <int MB, int NR, int NK, int RBW, int BKD, int S, bool PACKED>
static hipError_t decode_tile(int runs, const int8_t *Xq, const int8_t *Wq, const float *sX,
                              const int32_t *zW, const float *sW, const float *bp, int64_t M,
                              int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out, int32_t *part,
                              int32_t *part_rs, hipStream_t st) {
  if (runs > 1)
    return launch_decode_split<MB, NR, NK, RBW, BKD, S, PACKED>(Xq, Wq, sX, zW, sW, bp, M, N, K, Y,
                                                                acc_out, runs, part, part_rs, st);
  return launch_decode_t<MB, NR, NK, RBW, BKD, S, PACKED>(Xq, Wq, sX, zW, sW, bp, M, N, K, Y,
                                                          acc_out, st);
}

template <bool PACKED>
static hipError_t decode_tiles(const DecodePlan &p, const int8_t *Xq, const int8_t *Wq,
                               const float *sX, const int32_t *zW, const float *sW,
                               const float *bp, int64_t M, int64_t N, int64_t K, uint16_t *Y,
                               int32_t *acc_out, int32_t *part, int32_t *part_rs, hipStream_t st) {
#define OT_TILE(MB, NR, NK, RBW, BKD, S)                                                       \
  return decode_tile<MB, NR, NK, RBW, BKD, S, PACKED>(p.runs, Xq, Wq, sX, zW, sW, bp, M, N, K, \
                                                      Y, acc_out, part, part_rs, st)
  if (M <= 32) {
    if constexpr (PACKED) {
      if (p.rows == 32) OT_TILE(2, 2, 1, 1, 128, 8);
      if (p.rows == 64) OT_TILE(2, 4, 1, 1, 128, 8);
      if (p.rows == 96) OT_TILE(2, 2, 2, 3, 128, 8);
      OT_TILE(2, 4, 1, 2, 128, 4);
    } else {
      if (p.rows == 32) OT_TILE(2, 2, 4, 1, 256, 4);
      if (p.rows == 64) OT_TILE(2, 4, 2, 1, 256, 4);
      if (p.rows == 96) OT_TILE(2, 2, 4, 3, 256, 3);
      OT_TILE(2, 4, 1, 2, 128, 4);
    }
  }
  if constexpr (PACKED) {
    if (p.rows == 32) OT_TILE(4, 2, 4, 1, 256, 4);
    if (p.rows == 64) OT_TILE(4, 4, 2, 1, 256, 4);
    // over all of K, 2 K groups with 4 stages; the split runs (shorter K)
    // keep the 4 K groups with 3 stages below
    if (p.rows == 96 && p.runs == 1) OT_TILE(4, 2, 2, 3, 256, 4);
  } else {
    if (p.rows == 32) OT_TILE(4, 2, 4, 1, 256, 3);
    if (p.rows == 64) OT_TILE(4, 4, 2, 1, 256, 3);
  }
  if (p.rows == 96) OT_TILE(4, 2, 4, 3, 256, 3);
  OT_TILE(4, 8, 1, 1, 128, 4);
#undef OT_TILE
}

void describe_decode(int64_t M, int64_t N, int64_t K, bool packed, bool workspace, char *buf,
                     size_t len) {
  const int64_t cus = device_cus();
  const char *layout = packed ? "packed" : "row-major";
  if (M <= 16) {
    const int rows = N <= 16 * cus ? 16 : (packed && N > 32 * cus && N <= 64 * cus) ? 64 : 32;
    snprintf(buf, len, "decode %s %d-row tiles", layout, rows);
    return;
  }
  const DecodePlan p = decode_plan(M, N, K, cus, workspace);
  if (p.runs > 1)
    snprintf(buf, len, "decode %s %d-row tiles split-K %d", layout, p.rows, p.runs);
  else
    snprintf(buf, len, "decode %s %d-row tiles", layout, p.rows);
}

// Wq: the weight codes [N x K], or (packed) their micro-tiles.
hipError_t launch_qgemm_decode(const int8_t *Xq, const int8_t *Wq, const float *sX,
                               const int32_t *zW, const float *sW, const float *bprime,
                               int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                               void *workspace, bool packed, hipStream_t st) {
  // Template arguments
  // <token blocks, row groups, K groups, row blocks per wave, BKD, stages>,
  // chosen from sweeps of every valid configuration on MI355X.
  // Up to 16 tokens: 32-row tiles.  Where they fill at most one pass over
  // the CUs, one 8-wave workgroup per CU streams 16 KiB of weights per stage
  // (512-byte K slices, 3 stages ahead); with more rows, 2-wave workgroups
  // with 128-byte slices run six to a CU.  Below 16 rows per CU, 16-row tiles
  // split over 4 K groups.
  // 17-64 tokens: the tile height and split from decode_plan, the tile
  // configuration from decode_tiles.
  const int64_t cus = device_cus();
  if (M <= 16 && packed) {
    // packed weights stream into registers and the LDS ring holds only the
    // token rows, so deeper rings win: from a sweep of 23 configurations on
    // 14 layer shapes (N = 4096 .. 36864) at 1, 8 and 16 tokens
    if (N <= 16 * cus)
      return launch_decode_t<1, 1, 4, 1, 256, 8, true>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
    if (N <= 32 * cus || N > 64 * cus)
      return launch_decode_t<1, 2, 1, 1, 128, 8, true>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
    return launch_decode_t<1, 2, 1, 2, 128, 6, true>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, st);
  }
  if (M <= 16) {
    if (N <= 16 * cus)
      return launch_decode<1, 1, 4, 1, 256, 4>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, packed, st);
    if (N <= 32 * cus)
      return launch_decode<1, 2, 4, 1, 512, 4>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, packed, st);
    return launch_decode<1, 2, 1, 1, 128, 4>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, packed, st);
  }
  // 17-64 tokens: the plan's tile height and K runs
  const DecodePlan p = decode_plan(M, N, K, cus, workspace != nullptr);
  int32_t *part = static_cast<int32_t *>(workspace);
  int32_t *part_rs = p.runs > 1 ? part + (int64_t)p.runs * M * N : nullptr;
  return packed ? decode_tiles<true>(p, Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, part,
                                     part_rs, st)
                : decode_tiles<false>(p, Xq, Wq, sX, zW, sW, bprime, M, N, K, Y, acc_out, part,
                                      part_rs, st);
}

}  // namespace ot
