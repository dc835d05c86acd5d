// Prefill GEMM of the quantized linear (more than 64 tokens).
#include "ot_gemm_common.h"

namespace ot {
namespace detail {

// ---------------------------------------------------------------------------
// Prefill: LDS-tiled int8 MFMA GEMM (v_mfma_i32_32x32x32_i8)
// ---------------------------------------------------------------------------
// Workgroup tile BN (weight rows) x BM (token rows), K tile BK bytes, waves
// arranged WN x WM, each wave owning a (BN/WN) x (BM/WM) block of 32x32 MFMA
// tiles, accumulated in the AGPR file.
//
// Global -> LDS: buffer "load to LDS" (no registers, no ds_write).  One
// wave-wide 16-byte-per-lane load fills 1 KiB of LDS, lane i landing at byte
// 16 i.  LDS holds each operand tile row-major ([rows][BK]) with the 16-byte
// chunks of each row permuted by swz() so that fragment reads are free of
// bank conflicts.  The permutation is applied on the global side: each lane
// fetches the (row, chunk) that belongs at its fixed LDS position.  Buffer loads return
// zeros past the end of the resource, which pads ragged M and N tiles; a K
// tail is padded by aiming its lanes at an out-of-range offset.
//
// Pipeline: S LDS stages form a ring, K tiles are prefetched S-1 ahead.  Each
// wave double-buffers its MFMA fragments in registers: while the matrix
// cores work on one 32-byte K step the fragments of the next are in flight.
// The one barrier per K tile sits between the last fragment reads of tile t
// and its last MFMAs; right after it the wave starts reading tile t+1 and
// refills tile t's stage with tile t+S.  The refill's loads are not issued
// in one burst: one follows every MPL-th MFMA, over the tile's last K step
// and the next tile's first ones.  Issued back to back after the barrier,
// the loads of both waves of a SIMD held its matrix core idle (a load
// instruction takes the wave's issue for tens of cycles); spread between
// the MFMAs their issue overlaps the matrix work.
template <int BN, int BM, int BK, int WN, int WM, int S>
struct PrefillCfg {
  static constexpr int kWaves = WN * WM;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kChunks = BK / 16;         // 16-byte chunks per row
  static constexpr int kTN = BN / WN, kTM = BM / WM;
  static constexpr int kFN = kTN / 32, kFM = kTM / 32;
  static constexpr int kKSteps = BK / 32;
  static constexpr int kABytes = BN * BK, kBBytes = BM * BK;
  static constexpr int kStage = kABytes + kBBytes;
  static constexpr int kLoadsA = kABytes / 1024 / kWaves;
  static constexpr int kLoadsB = kBBytes / 1024 / kWaves;
  static constexpr int kLoads = kLoadsA + kLoadsB;  // per wave per K tile
  static_assert(BK == 64 || BK == 128, "an even number of 32-byte K steps per tile");
  static_assert(kLoadsA * 1024 * kWaves == kABytes && kLoadsB * 1024 * kWaves == kBBytes,
                "tile must split evenly into wave loads");
  static_assert(kTN % 32 == 0 && kTM % 32 == 0, "MFMA tiling");
  static_assert(S >= 2 && (S - 2) * kLoads <= 63, "vmcnt range");
  static_assert(S * kStage <= 160 * 1024, "LDS");
  // the workgroup's fp16 output tile, which the epilogue stages whole in the
  // idle ring: where it is larger than the ring, the workgroup takes LDS for
  // it (up to the 160 KiB a workgroup can have)
  static constexpr int kOutBytes = BN * BM * 2;
  static constexpr int kSmem = kOutBytes > S * kStage && kOutBytes <= 160 * 1024
                                   ? kOutBytes
                                   : S * kStage;
};

// LDS swizzle of an operand tile [rows][BK]: chunk c (16 bytes) of row r is
// stored at chunk c ^ g(r) of that row.  A fragment read has 16 consecutive
// rows (lanes) fetch the same logical chunk; with g below those 16 reads
// cover 16 distinct 16-byte bank groups of a 256-byte window, and any 8 of
// them (rows 8i..8i+7) cover 8 distinct groups of a 128-byte window, so the
// read is conflict-free whether the LDS serves 8 or 16 lanes per cycle.
template <int kChunks>
__device__ __forceinline__ int swz(int r) {
  if constexpr (kChunks == 4) return ((r >> 1) & 3) ^ ((r >> 3) & 1);
  else return (r & 7) ^ ((r >> 3) & 1);
}

template <bool B>
struct BoolC {
  static constexpr bool value = B;
};

// The kernel body lives in a device function: hipcc drops the host stub of a
// kernel template whose body holds lambdas.
template <int BN, int BM, int BK, int WN, int WM, int S, int EPI, int MPL>
__device__ __forceinline__ void prefill_body(
    int8_t *smem, const int8_t *__restrict__ Xq, const int8_t *__restrict__ Wq,
    const float *__restrict__ sX, const int32_t *__restrict__ zW, const float *__restrict__ sW,
    const float *__restrict__ bp, int M, int N, int K, uint16_t *__restrict__ Y,
    int32_t *__restrict__ acc_out, int tiles_m, int tiles_n, int group_m) {
  using C = PrefillCfg<BN, BM, BK, WN, WM, S>;

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
  // Lane i of the j-th 1 KiB load lands at LDS slot 64 j' + i (j' = this
  // wave's load index in the tile), i.e. row (64 j' + i) / kChunks, physical
  // chunk i % kChunks; it fetches the logical chunk stored there.
  constexpr int kRowsPerLoad = 64 / C::kChunks;
  uint32_t off_a[C::kLoadsA], off_b[C::kLoadsB];
  int ck_a[C::kLoadsA], ck_b[C::kLoadsB];
#pragma unroll
  for (int j = 0; j < C::kLoadsA; ++j) {
    const int row = (wave * C::kLoadsA + j) * kRowsPerLoad + lane / C::kChunks;
    ck_a[j] = (lane % C::kChunks) ^ swz<C::kChunks>(row);
    off_a[j] = (uint32_t)(row * K + ck_a[j] * 16);
  }
#pragma unroll
  for (int j = 0; j < C::kLoadsB; ++j) {
    const int row = (wave * C::kLoadsB + j) * kRowsPerLoad + lane / C::kChunks;
    ck_b[j] = (lane % C::kChunks) ^ swz<C::kChunks>(row);
    off_b[j] = (uint32_t)(row * K + ck_b[j] * 16);
  }
  const int KT = (K + BK - 1) / BK;
  // Neighbouring tiles (a checkerboard over token x channel tiles) walk K
  // one tile apart, the odd ones starting at K tile 1 and wrapping round to
  // 0, so that the tiles sharing operand panels in an XCD's L2 do not all
  // ask for the same lines at once.  The accumulators are exact integer
  // sums, which do not depend on the order.
  const int phi = (tm + tn) & 1;

  auto issue_tile = [&](int kt) {
    int kr = kt;  // the K tile that iteration kt loads
    if (kt < KT) {
      kr = kt + phi;
      if (kr >= KT) kr -= KT;
    }
    const int k0 = kr * BK;  // iterations kt >= KT load only out-of-range chunks
    int8_t *sa = smem + (kt % S) * C::kStage;
    int8_t *sb = sa + C::kABytes;
#pragma unroll
    for (int j = 0; j < C::kLoadsA; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc_a, (lds_void *)(sa + (wave * C::kLoadsA + j) * 1024), 16,
          k0 + ck_a[j] * 16 < K ? off_a[j] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < C::kLoadsB; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc_b, (lds_void *)(sb + (wave * C::kLoadsB + j) * 1024), 16,
          k0 + ck_b[j] * 16 < K ? off_b[j] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
  };

  // ---- LDS -> register fragment addressing ----------------------------------
  // Lane (fr, fh) of a 32x32x32 MFMA reads row fr of a 32-row block, logical
  // chunk 2s + fh of K step s.  Blocks start at multiples of 32 rows and the
  // swizzle has period 16, so it depends on fr only.
  const int fr = lane & 31, fh = lane >> 5;
  int frag_off[C::kKSteps];
#pragma unroll
  for (int s = 0; s < C::kKSteps; ++s)
    frag_off[s] = fr * BK + 16 * ((2 * s + fh) ^ swz<C::kChunks>(fr));
  const int a_base = wn * C::kTN * BK;
  const int b_base = C::kABytes + wm * C::kTM * BK;

  v4i fa[2][C::kFN], fb[2][C::kFM];
  auto read_frags = [&](int kt, int s, int buf) {
    const int8_t *st = smem + (kt % S) * C::kStage;
#pragma unroll
    for (int f = 0; f < C::kFN; ++f)
      fa[buf][f] = *reinterpret_cast<const v4i *>(st + a_base + f * 32 * BK + frag_off[s]);
#pragma unroll
    for (int g = 0; g < C::kFM; ++g)
      fb[buf][g] = *reinterpret_cast<const v4i *>(st + b_base + g * 32 * BK + frag_off[s]);
  };

  v16i acc[C::kFN][C::kFM];
#pragma unroll
  for (int f = 0; f < C::kFN; ++f)
#pragma unroll
    for (int g = 0; g < C::kFM; ++g) acc[f][g] = v16i{};
  // asymmetric weights: the code sum of every token.  The WN waves that
  // share a token block split the work by K step (wave wn takes the steps s
  // with s mod WN = wn) and sum the token fragments they already hold (a
  // lane covers its token fr, half fh of the step); the partials meet in
  // LDS after the loop.
  static_assert(EPI != kEpiAsym || C::kKSteps % WN == 0, "K steps split over the WN waves");
  int rs[C::kFM];
#pragma unroll
  for (int g = 0; g < C::kFM; ++g) rs[g] = 0;
  // ---- main loop ----------------------------------------------------------------
  // One 1 KiB load of tile kt's stage: j < kLoadsA a weight load, else a
  // token load (the j-th of issue_tile's order).
  auto issue_one = [&](int kt, int j) {
    int kr = kt;
    if (kt < KT) {
      kr = kt + phi;
      if (kr >= KT) kr -= KT;
    }
    const int k0 = kr * BK;
    int8_t *sa = smem + (kt % S) * C::kStage;
    if (j < C::kLoadsA) {
      const int ja = j < C::kLoadsA ? j : 0;  // j is a constant once unrolled
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc_a, (lds_void *)(sa + (wave * C::kLoadsA + ja) * 1024), 16,
          k0 + ck_a[ja] * 16 < K ? off_a[ja] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
    } else {
      const int jb = j >= C::kLoadsA && j < C::kLoads ? j - C::kLoadsA : 0;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rsrc_b, (lds_void *)(sa + C::kABytes + (wave * C::kLoadsB + jb) * 1024), 16,
          k0 + ck_b[jb] * 16 < K ? off_b[jb] + (uint32_t)k0 : kOobOffset, 0, 0, 0);
    }
  };
  // A tile's last K step issues the first kLast loads of the tile S ahead
  // (whose stage the barrier before it has just freed), one after every
  // MPL-th MFMA; the next tile's first K steps issue the rest at the same
  // rate, all before the wait that precedes its last step.
  constexpr int kMfma = C::kFN * C::kFM;
  constexpr int kReads = C::kFN + C::kFM;
  constexpr int kPerStep = kMfma / MPL;
  constexpr int kLast = kPerStep < C::kLoads ? kPerStep : C::kLoads;
  static_assert(kPerStep >= 1, "at least one load per K step");
  static_assert(kLast + (C::kKSteps - 2) * kPerStep >= C::kLoads,
                "every load of a tile is issued before the wait for it");
  // One K step: the MFMAs of K step `step` on fragment buffer cb, the
  // fragment reads of tile rkt's K step rstep into buffer nb, and loads
  // j0 .. j0+nl-1 of tile lt, issued in that interleaved order (a read
  // before each MFMA while reads remain, a load after every MPL-th).
  auto kstep = [&](int cb, int step, int rkt, int rstep, int nb, int lt, int j0, int nl) {
    const int8_t *st = smem + (rkt % S) * C::kStage;
#pragma unroll
    for (int i = 0; i < kMfma; ++i) {
      if (i < C::kFN)
        fa[nb][i] = *reinterpret_cast<const v4i *>(st + a_base + i * 32 * BK + frag_off[rstep]);
      else if (i < kReads)
        fb[nb][i - C::kFN] =
            *reinterpret_cast<const v4i *>(st + b_base + (i - C::kFN) * 32 * BK + frag_off[rstep]);
      const int f = i / C::kFM, g = i % C::kFM;
      acc[f][g] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[cb][f], fb[cb][g], acc[f][g], 0, 0, 0);
      if (i % MPL == MPL - 1 && i / MPL < nl) issue_one(lt, j0 + i / MPL);
    }
    if constexpr (EPI == kEpiAsym) {
      if (step % WN == __builtin_amdgcn_readfirstlane(wn)) {
#pragma unroll
        for (int g = 0; g < C::kFM; ++g) rs[g] = byte_sum16(fb[cb][g], rs[g]);
      }
    }
    // keep that order through the scheduler
    constexpr int kMaskMfma = 0x008, kMaskVmemRead = 0x020, kMaskDsRead = 0x100;
#pragma unroll
    for (int i = 0; i < kMfma; ++i) {
      if (i < kReads) __builtin_amdgcn_sched_group_barrier(kMaskDsRead, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kMaskMfma, 1, 0);
      if (i % MPL == MPL - 1 && i / MPL < nl) __builtin_amdgcn_sched_group_barrier(kMaskVmemRead, 1, 0);
    }
  };

  // Tiles past the end of K are issued too, as out-of-range loads that land
  // zeros in a stage nobody reads: every iteration then has the same number
  // of loads in flight and one fixed wait, with no branches in the loop.
#pragma unroll
  for (int t = 0; t < S - 1; ++t) issue_tile(t);
  wait_vmcnt<(S - 2) * C::kLoads>();  // tile 0 has landed
  lds_barrier();
#pragma unroll
  for (int j = 0; j < kLast; ++j) issue_one(S - 1, j);
  read_frags(0, 0, 0);

  for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
    for (int s = 0; s + 1 < C::kKSteps; ++s) {
      const int j0 = kLast + s * kPerStep;
      const int nl = j0 >= C::kLoads ? 0 : (C::kLoads - j0 < kPerStep ? C::kLoads - j0 : kPerStep);
      kstep(s & 1, s, kt, s + 1, (s + 1) & 1, kt + S - 1, j0, nl);
    }
    // This wave's reads of tile kt are complete once lgkmcnt drains; tile
    // kt+1 has landed once at most S-2 younger tiles (kt+2 .. kt+S-1) are in
    // flight.  After the barrier every wave is past tile kt, so its stage
    // takes tile kt+S.  At kt = KT-1 the reads of "tile KT" are unused.
    // The scheduling fences keep every MFMA of the steps above ahead of the
    // wait, so the reads have that long to land.
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    wait_vmcnt<(S - 2) * C::kLoads>();
    lds_barrier();
    kstep(1, C::kKSteps - 1, kt + 1, 0, 0, kt + S, 0, kLast);
    __builtin_amdgcn_sched_barrier(0);
  }
  wait_vmcnt<0>();

  if constexpr (EPI == kEpiAsym) {
    // combine the two K halves of each step (lanes l and l ^ 32), then the
    // WN waves' step subsets through LDS (the ring is idle after the loop)
    int *part = reinterpret_cast<int *>(smem);  // [kWaves][kFM][32]
    static_assert(C::kWaves * C::kFM * 32 * 4 <= S * C::kStage, "partials fit the ring");
#pragma unroll
    for (int g = 0; g < C::kFM; ++g) rs[g] += __shfl_xor(rs[g], 32);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's last fragment reads
    lds_barrier();                        // every wave is done with the ring
    if (lane < 32) {
#pragma unroll
      for (int g = 0; g < C::kFM; ++g) part[(wave * C::kFM + g) * 32 + lane] = rs[g];
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);
    lds_barrier();
#pragma unroll
    for (int g = 0; g < C::kFM; ++g) {
      int t = 0;
#pragma unroll
      for (int w = 0; w < WN; ++w) t += part[((wm * WN + w) * C::kFM + g) * 32 + fr];
      rs[g] = t;
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);
    lds_barrier();  // the partials are read before the ring is reused
  }

  // ---- epilogue ----------------------------------------------------------------
  // 32x32 output block, 16 values per lane: lane l holds column (l mod 32)
  // and rows 8*(r/4) + 4*(l/32) + (r mod 4) for register r.  Columns are
  // tokens here and rows are channels, so registers 4j..4j+3 are four
  // consecutive channels of one token.
  // token scales of this lane's tokens (per-token path)
  float sx[C::kFM];
#pragma unroll
  for (int g = 0; g < C::kFM; ++g) {
    const int m = m0 + wm * C::kTM + g * 32 + fr;
    sx[g] = (EPI == kEpiToken && m < M) ? sX[m] : 0.f;
  }
  if (acc_out != nullptr) {  // test path: also stores the raw accumulators
#pragma unroll
    for (int f = 0; f < C::kFN; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t n = n0 + wn * C::kTN + f * 32 + 8 * j + 4 * fh;
#pragma unroll
        for (int g = 0; g < C::kFM; ++g) {
          const int64_t m = m0 + wm * C::kTM + g * 32 + fr;
          store4<EPI>(Y, acc_out, sW, bp, zW, sx[g], rs[g], m, n, M, N, acc[f][g][4 * j],
                      acc[f][g][4 * j + 1], acc[f][g][4 * j + 2], acc[f][g][4 * j + 3]);
        }
      }
    return;
  }
  // Dequantize into a wave-private fp16 staging tile in the now idle LDS
  // (the ring, and past it up to 160 KiB where the workgroup's output tile
  // needs more), then write whole token rows with 16-byte stores.  The tile
  // holds kSlab token rows by kTN channels: the wave's whole block when every
  // wave's block fits, else 32 tokens (one register block g) at a time.
  // In LDS the 8-byte unit u (4 channels) of staging row r sits at
  // unit u ^ h(r), h(r) < kSwz: the lanes that write one register group (32
  // tokens, same channels) then spread over the banks (h(r) = r mod 16 for
  // 128-byte rows, (r / 2) mod 8 for 320-byte rows, each checked
  // conflict-free for 32 and 64 banks).
  constexpr int kUnits = C::kTN / 4;                       // 8-byte units per row
  constexpr int kSwz = (kUnits % 16 == 0) ? 16 : 8;         // XOR group of the swizzle
  constexpr int kCpr = C::kTN / 8;                          // 16-byte chunks per row
  constexpr bool kWhole = C::kWaves * C::kTM * C::kTN * 2 <= C::kSmem;
  constexpr int kSlab = kWhole ? C::kTM : 32;               // token rows per staging pass
  constexpr int kSlabG = kSlab / 32;                        // register blocks per pass
  static_assert(kUnits % kSwz == 0, "the swizzle permutes whole groups of units");
  static_assert(C::kWaves * kSlab * C::kTN * 2 <= C::kSmem, "staging tile fits the LDS");
  static_assert((kSlab * kCpr) % 64 == 0, "row pass covers the slab in whole wave passes");
  auto stage_swz = [](int r) { return kSwz == 16 ? (r & 15) : ((r >> 1) & 7); };
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's last reads
  wait_vmcnt<0>();                     // the trailing out-of-range tiles
  lds_barrier();                        // every wave is done with the ring
  uint16_t *tile = reinterpret_cast<uint16_t *>(smem) + wave * (kSlab * C::kTN);
  const int nw0 = n0 + wn * C::kTN;   // first channel of this wave
  const int mw0 = m0 + wm * C::kTM;   // first token of this wave
  // The same steps with and without per-lane bounds checks: a tile inside
  // M x N whose output rows are whole 16-byte chunks needs none (measured:
  // 23 k against 16 k shader cycles per 320 x 256 tile).
  auto epilogue = [&](auto interior) {
    constexpr bool kIn = decltype(interior)::value;
#pragma unroll
    for (int g0 = 0; g0 < C::kFM; g0 += kSlabG) {
#pragma unroll
      for (int f = 0; f < C::kFN; ++f)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int nl = f * 32 + 8 * j + 4 * fh;  // channel within the wave tile
          const int n = nw0 + nl;
          float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f), b4 = s4;
          if (kIn || (n + 3 < N && (N & 3) == 0)) {
            s4 = *reinterpret_cast<const float4 *>(sW + n);
            b4 = *reinterpret_cast<const float4 *>(bp + n);
          } else {
            if (n + 0 < N) { s4.x = sW[n + 0]; b4.x = bp[n + 0]; }
            if (n + 1 < N) { s4.y = sW[n + 1]; b4.y = bp[n + 1]; }
            if (n + 2 < N) { s4.z = sW[n + 2]; b4.z = bp[n + 2]; }
            if (n + 3 < N) { s4.w = sW[n + 3]; b4.w = bp[n + 3]; }
          }
          const int4 z4 = load_zw4<EPI>(zW, n, N);
#pragma unroll
          for (int gs = 0; gs < kSlabG; ++gs) {
            const int g = g0 + gs;
            const int r = gs * 32 + fr;  // staging row
            uint2 h;
            const int a0 = acc[f][g][4 * j + 0] - z4.x * rs[g];
            const int a1 = acc[f][g][4 * j + 1] - z4.y * rs[g];
            const int a2 = acc[f][g][4 * j + 2] - z4.z * rs[g];
            const int a3 = acc[f][g][4 * j + 3] - z4.w * rs[g];
            h.x = (uint32_t)dequant_x<EPI>(a0, sx[g], s4.x, b4.x) |
                  ((uint32_t)dequant_x<EPI>(a1, sx[g], s4.y, b4.y) << 16);
            h.y = (uint32_t)dequant_x<EPI>(a2, sx[g], s4.z, b4.z) |
                  ((uint32_t)dequant_x<EPI>(a3, sx[g], s4.w, b4.w) << 16);
            const int unit = (nl >> 2) ^ stage_swz(r);
            *reinterpret_cast<uint2 *>(tile + r * C::kTN + unit * 4) = h;
          }
        }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the slab is in LDS
      __builtin_amdgcn_wave_barrier();
      // Row pass: lane c of the slab moves 16-byte chunk c mod kCpr (8
      // channels) of staging row c / kCpr; consecutive lanes write
      // consecutive chunks of a token row.
#pragma unroll 2
      for (int c0 = 0; c0 < kSlab * kCpr; c0 += 64) {
        const int c = c0 + lane;
        const int r = c / kCpr, cc = c % kCpr;
        const int x = stage_swz(r);
        const int pair = cc ^ (x >> 1);  // units 2cc and 2cc+1 sit in this aligned pair
        uint4 v = *reinterpret_cast<const uint4 *>(tile + r * C::kTN + pair * 8);
        if (x & 1) {  // the two 8-byte units of the pair are stored swapped
          const uint32_t t0 = v.x, t1 = v.y;
          v.x = v.z; v.y = v.w; v.z = t0; v.w = t1;
        }
        const int64_t m = mw0 + g0 * 32 + r;
        const int n = nw0 + cc * 8;
        if (kIn || m < M) {
          uint16_t *dst = Y + m * (int64_t)N + n;
          if (kIn || ((N & 7) == 0 && n + 7 < N)) {
            *reinterpret_cast<uint4 *>(dst) = v;
          } else {
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
            for (int i = 0; i < 8; ++i)
              if (n + i < N) dst[i] = (uint16_t)(w[i >> 1] >> (16 * (i & 1)));
          }
        }
      }
      if (g0 + kSlabG < C::kFM) {
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the slab is read before it is rewritten
        __builtin_amdgcn_wave_barrier();
      }
    }
  };
  if (n0 + BN <= N && m0 + BM <= M && (N & 7) == 0)
    epilogue(BoolC<true>{});
  else
    epilogue(BoolC<false>{});
}

template <int BN, int BM, int BK, int WN, int WM, int S, int MPL, int OCC, int EPI>
__global__ __launch_bounds__(64 * WN * WM, OCC) void qgemm_prefill_kernel(
    const int8_t *__restrict__ Xq, const int8_t *__restrict__ Wq, const float *__restrict__ sX,
    const int32_t *__restrict__ zW, const float *__restrict__ sW, const float *__restrict__ bp,
    int M, int N, int K, uint16_t *__restrict__ Y, int32_t *__restrict__ acc_out, int tiles_m,
    int tiles_n, int group_m) {
  __shared__ __attribute__((aligned(1024)))
  int8_t smem[PrefillCfg<BN, BM, BK, WN, WM, S>::kSmem];
  prefill_body<BN, BM, BK, WN, WM, S, EPI, MPL>(smem, Xq, Wq, sX, zW, sW, bp, M, N, K, Y, acc_out,
                                           tiles_m, tiles_n, group_m);
}

// Epilogue by argument: sX != nullptr per-token scales sX [M]; zW != nullptr
// asymmetric weight zero points zW [N]; neither: per-channel.
template <int BN, int BM, int BK, int WN, int WM, int S, int MPL, int OCC = 1>
hipError_t launch_prefill(const int8_t *Xq, const int8_t *Wq, const float *sX, const int32_t *zW,
                          const float *sW, const float *bp, int64_t M, int64_t N, int64_t K,
                          uint16_t *Y, int32_t *acc_out, hipStream_t st, int group_m = 8) {
  const int tiles_m = (int)((M + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
  const unsigned grid = (unsigned)(tiles_m * tiles_n);
  const dim3 block(64 * WN * WM);
  if (sX)
    qgemm_prefill_kernel<BN, BM, BK, WN, WM, S, MPL, OCC, kEpiToken><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out, tiles_m, tiles_n, group_m);
  else if (zW)
    qgemm_prefill_kernel<BN, BM, BK, WN, WM, S, MPL, OCC, kEpiAsym><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out, tiles_m, tiles_n, group_m);
  else
    qgemm_prefill_kernel<BN, BM, BK, WN, WM, S, MPL, OCC, kEpiChannel><<<grid, block, 0, st>>>(
        Xq, Wq, sX, zW, sW, bp, (int)M, (int)N, (int)K, Y, acc_out, tiles_m, tiles_n, group_m);
  return hipGetLastError();
}

}  // namespace detail

using namespace detail;

// Relative time of a launch with BN x BM tiles, one workgroup per CU: whole
// passes over the CUs, each as long as one tile.  A tile's time is
// proportional to its products over K plus its epilogue, which costs about
// as much as 820 more K steps, times a factor per tile shape for the operand
// bytes it stages per product: 0.97 for the wider tile (fewer bytes per
// product), 1.5 for the shorter one (1.5 times the bytes), 1.15 for the
// narrower one (1.17 times).  Measured on MI355X, per pass against 256 x 256
// at the OPT-6.7B, -13B and -66B layer shapes: 0.93-1.01, 1.3-1.6 and, for
// 192 x 256, the cheapest tile wherever the model picks it (2048 tokens by
// 12288 channels: 103.7 against 116.1 us; one-pass launches of 2000 tokens
// by 5000 channels: equal to 256 x 256 within 4 %).  Re-measured with the
// loads spread over the MFMAs (OPT-6.7B and -13B shapes): 1.01, 1.61 and
// 1.24, which pick the same tiles on those layers.
static double prefill_cost(int64_t M, int64_t N, int64_t K, int bn, int bm, int cus) {
  const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  const int64_t passes = (tiles + cus - 1) / cus;
  const double penalty = bn == 320 ? 0.97 : bn == 192 ? 1.15 : bm == 128 ? 1.5 : 1.0;
  return (double)passes * bn * bm * ((double)K + 820.0) * penalty;
}

// Four tile shapes, each one workgroup of 8 waves per CU with a 2-stage
// ring of BK = 128:
//   256 (channels) x 256 (tokens), waves 4 x 2 of 64 x 128 (128 KiB of LDS);
//   320 x 256, waves 2 x 4 of 160 x 64 (a 144 KiB ring in 160 KiB, which
//     holds the epilogue's whole output tile): lets layers whose tile
//     count leaves the last pass over the CUs mostly empty fill whole passes
//     (4096 tokens by 5120 or 15360 channels: 256 and 768 tiles against 320
//     and 960 of 256 x 256);
//   256 x 128, waves 4 x 2 of 64 x 64 (96 KiB): for launches that fill less
//     than one pass with 256 x 256 (2048 tokens by 4096 channels: 256 tiles
//     against 128);
//   192 x 256, waves 2 x 4 of 96 x 64 (112 KiB): the same for launches
//     whose last pass of 256 x 256 runs half empty (2048 tokens by 12288
//     channels: two full passes of 512 tiles against 1.5 of 384).
// The cheapest by prefill_cost runs; all give identical results.
enum class PrefillTile { k256x256, k320x256, k256x128, k192x256 };

static PrefillTile prefill_tile(int64_t M, int64_t N, int64_t K) {
  const int cus = device_cus();
  const double c0 = prefill_cost(M, N, K, 256, 256, cus);
  const double c1 = prefill_cost(M, N, K, 320, 256, cus);
  const double c2 = prefill_cost(M, N, K, 256, 128, cus);
  const double c3 = prefill_cost(M, N, K, 192, 256, cus);
  if (c1 < c0 && c1 <= c2 && c1 <= c3) return PrefillTile::k320x256;
  if (c3 < c0 && c3 <= c2) return PrefillTile::k192x256;
  if (c2 < c0) return PrefillTile::k256x128;
  return PrefillTile::k256x256;
}

const char *prefill_tile_name(int64_t M, int64_t N, int64_t K) {
  switch (prefill_tile(M, N, K)) {
    case PrefillTile::k320x256: return "prefill 320x256";
    case PrefillTile::k256x128: return "prefill 256x128";
    case PrefillTile::k192x256: return "prefill 192x256";
    default: return "prefill 256x256";
  }
}

hipError_t launch_qgemm_prefill(const int8_t *Xq, const int8_t *Wq, const float *sX,
                                const int32_t *zW, const float *sW, const float *bprime,
                                int64_t M, int64_t N, int64_t K, uint16_t *Y, int32_t *acc_out,
                                hipStream_t st) {
  switch (prefill_tile(M, N, K)) {
    case PrefillTile::k320x256:
      return launch_prefill<320, 256, 128, 2, 4, 2, 2>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y,
                                                    acc_out, st);
    case PrefillTile::k256x128:
      return launch_prefill<256, 128, 128, 4, 2, 2, 1>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y,
                                                    acc_out, st);
    case PrefillTile::k192x256:
      return launch_prefill<192, 256, 128, 2, 4, 2, 2>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y,
                                                    acc_out, st);
    default:
      return launch_prefill<256, 256, 128, 4, 2, 2, 2>(Xq, Wq, sX, zW, sW, bprime, M, N, K, Y,
                                                    acc_out, st);
  }
}

}  // namespace ot
