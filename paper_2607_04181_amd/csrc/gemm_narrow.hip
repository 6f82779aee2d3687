// Prefill GEMMs on 256-row tiles of TN columns (bf16 MFMA), each unsplit
// along K with its consumer's work in the epilogue.
//
//   acc[m][n] = sum_k A[m][k] * W[n][k]      A: [M][K], W: [N][K], both bf16
//
// A and W are in tile order (tile_off / pack_tile_order): every 16 rows x
// 32 k is one contiguous 1 KB block, laid out lane by lane as a
// v_mfma_f32_16x16x32_bf16 operand, so one 16-byte-per-lane load copies a
// block to LDS unchanged and one 16-byte LDS read per lane is a fragment.
//
// A 256 x 256 tile grid leaves the d-wide projections with d / 256 column
// tiles per 256 rows: 160 tiles for d = 5120 and a 2048-row chunk, on 256
// CUs. Here TN comes from N alone: 160 or 128 for the O and down projections
// (narrow_tile_n: d / TN <= 32 column tiles, so a 2048-row chunk is exactly
// 256 tiles for d = 5120 and 4096), 192 for gate/up, 224, 192 or 160 for
// QKV. Epilogue variants:
//   * residual (O projection): x1 = acc + residual row (fp32 out),
//     h = bf16(x1 * gamma) in tile order for the gate/up projection, and the
//     tile's row sums of x1^2 (RMSNorm_2's statistics, finished by the
//     gate/up epilogue);
//   * scatter (down projection): out[out_idx[m]] = bf16(x1 + acc), the layer
//     output written straight to its row of the full batch;
//   * SwiGLU (gate/up projection): each lane holds the gate and up values of
//     its outputs; h = silu(gate / rms) * up / rms in tile order;
//   * QKV: a tile holds whole RoPE pairs; queries are rotated into q, keys
//     rotated and values copied into the paged cache.
// gemm_narrow_swiglu_persistent_kernel runs the SwiGLU variant with one
// workgroup per CU walking several column tiles of one row tile.
// The main loop:
//   * 512 threads, eight waves as 4 (rows) x 2 (columns); each wave owns a
//     64 x TN/2 sub-tile as 4 x TN/32 accumulators of 16 x 16, two waves per
//     SIMD so one wave's MFMAs issue while the other reads LDS;
//   * 32-deep K stages of both tiles go straight from global memory to LDS
//     (global_load_lds, no register staging) into a ring of six slots (five
//     for TN > 160), all but one stage in flight (the loads come from L2, the
//     MALL or HBM, whose latency under this load is several stages of MFMA
//     work); wave w copies A blocks 2w, 2w + 1 and W block w, and for
//     TN > 128 a second W block (or a spare copy);
//   * one barrier per stage, which publishes stage st + 1 and guarantees
//     that the slot the next loads overwrite was read by every wave;
//   * workgroups are remapped so that the tiles sharing a W column slab run
//     on the same XCD (blockIdx % 8) and hit its L2.
// Every output element is one chain of MFMAs over k in ascending 32-steps,
// and the tile width depends on N only, so a row's result does not depend on
// M or on the other rows of the call.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kNM = 256;        // tile rows
constexpr int kNK = 32;         // k per stage
constexpr int kNThreads = 512;  // 8 waves, two per SIMD
constexpr int kNXCDs = 8;
constexpr int kNMaxTiles = 32;  // column tiles (the gate/up fold's limit)

typedef __attribute__((address_space(3))) void lds_void_t;

// LDS ring slots for a tile width: as many stages of 256 x 32 A and TN x 32
// W as fit beside the spare block in 160 KB.
constexpr int narrow_slots(int TN) { return TN <= 160 ? 6 : 5; }
// Stages per unrolled round of the main loop: fragment registers alternate
// with the stage's parity, so a round is an even number of stages.
constexpr int narrow_round(int TN) {
  return narrow_slots(TN) % 2 ? 2 * narrow_slots(TN) : narrow_slots(TN);
}

// kNarrowSwigluPlain: the SwiGLU epilogue without RMSNorm_2's 1/rms (the
// operand is already normalised).
enum { kNarrowResid = 0, kNarrowScatter = 1, kNarrowSwiglu = 2, kNarrowQkv = 3, kNarrowSwigluPlain = 4 };

template <int TN, int MODE>
__global__ __launch_bounds__(kNThreads) void gemm_narrow_kernel(const bf16_t* __restrict__ A,
                                                                 const bf16_t* __restrict__ W,
                                                                 int M, int N, int K,
                                                                 NarrowEpiArgs ea) {
  static_assert(TN % 32 == 0 && TN / 16 >= 8 && TN / 16 <= 16, "tile width");
  constexpr bool kSwi = MODE == kNarrowSwiglu || MODE == kNarrowSwigluPlain;
  static_assert(!kSwi || TN % 64 == 0, "SwiGLU pairs gate and up blocks");
  static_assert(MODE != kNarrowQkv || (TN >= 160 && TN <= 224), "QKV exchange areas");
  constexpr int WB = TN / 32;          // 16-column blocks per wave
  constexpr int kWBlocks = TN / 16;    // W blocks per stage
  constexpr int kExtra = kWBlocks - 8; // waves that copy a second W block
  // Loads per stage and wave. With a second W block (TN > 128) every wave
  // issues one: waves past kExtra copy their first block again into a spare
  // block that is never read, so all waves wait on the same counts and the
  // loop has no branch around a load.
  constexpr int kLoads = kExtra > 0 ? 4 : 3;
  constexpr int kBuf = narrow_slots(TN);
  constexpr int kAhead = kBuf - 1;  // stages in flight
  constexpr int kRound = narrow_round(TN);
  // One LDS object per ring slot, so the compiler tracks each slot's pending
  // direct loads on its own and never drains the ring before a fragment read.
  __shared__ __attribute__((aligned(16))) bf16_t sa0[kNM * kNK], sa1[kNM * kNK],
      sa2[kNM * kNK], sa3[kNM * kNK], sa4[kNM * kNK], sa5[kNM * kNK];
  __shared__ __attribute__((aligned(16))) bf16_t sw0[TN * kNK], sw1[TN * kNK], sw2[TN * kNK],
      sw3[TN * kNK], sw4[TN * kNK], sw5[TN * kNK];
  // Target of the loads that only keep the per-wave load count uniform
  // (never read; several waves may write it at once).
  __shared__ __attribute__((aligned(16))) bf16_t spare[512];
  bf16_t* const ta[6] = {sa0, sa1, sa2, sa3, sa4, sa5};
  bf16_t* const tw[6] = {sw0, sw1, sw2, sw3, sw4, sw5};

  const int tiles_m = (M + kNM - 1) / kNM;
  const int nb = gridDim.x;
  const int b = blockIdx.x;
  const int full = (nb / kNXCDs) * kNXCDs;
  const int lid = b < full ? (b % kNXCDs) * (nb / kNXCDs) + b / kNXCDs : b;
  const int m0 = (lid % tiles_m) * kNM;
  const int n0 = (lid / tiles_m) * TN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv & 3, wn = wv >> 2;  // 64-row quarter, column half
  const int c16 = lane & 15, j4 = lane >> 4;

  // W block (16 rows) of the tile's block b. SwiGLU: W is [W_g; W_u], [2F][K];
  // the tile holds outputs o0 .. o0 + TN/2 - 1, and the WB blocks of column
  // half h are the gate blocks of outputs o0 + TN/4 h + 16 q (q < WB/2), then
  // the matching up blocks, so a lane holds both factors of its outputs.
  const int F = N / 2, o0 = n0 / 2;
  auto w_block = [&](int blk) -> int {
    if constexpr (kSwi) {
      const int h = blk / WB, r = blk % WB;
      const int o = o0 + h * (TN / 4) + 16 * (r % (WB / 2));
      return ((r < WB / 2 ? 0 : F) + o) >> 4;
    }
    if constexpr (MODE == kNarrowQkv) {
      // Rotation pairs: pair p = 64 hh + j holds dims j and j + 64 of head hh.
      // The tile holds pairs TN/2 (n0/TN) .. + TN/2 - 1 as WB groups of 16;
      // column half 0 holds the j dims of group q in block q, half 1 the
      // j + 64 dims, so both dims of a pair sit in the same lane of the two
      // waves of a row quarter.
      const int h = blk / WB, q = blk % WB;
      const int p0 = 16 * ((n0 / TN) * WB + q);
      return ((p0 >> 6) * 128 + (p0 & 63) + 64 * h) >> 4;
    }
    return (n0 >> 4) + blk;
  };
  // This wave's sources: A blocks of row groups 2 wv, 2 wv + 1 of the tile
  // (groups past the last row read the last group; their rows are never
  // stored), W block wv and, for TN > 128, W block 8 + wv (waves below
  // kExtra) or a spare copy of block wv (the others).
  const int stages = K / kNK;
  const bf16_t* src_a[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ag = min((m0 + 32 * wv + 16 * h) >> 4, (M - 1) >> 4);
    src_a[h] = A + (int64_t)ag * (K / kNK) * 512 + lane * 8;
  }
  const bf16_t* src_w0 = W + (int64_t)w_block(wv) * (K / kNK) * 512 + lane * 8;
  const bf16_t* src_w1 =
      W + (int64_t)w_block(wv < kExtra ? 8 + wv : wv) * (K / kNK) * 512 + lane * 8;
  // Loads past the slice repeat its last stage (never multiplied).
  auto issue = [&](int st, int slot) {
    const int sc = min(st, stages - 1);
#pragma unroll
    for (int h = 0; h < 2; ++h)
      __builtin_amdgcn_global_load_lds(src_a[h] + sc * 512,
                                       (lds_void_t*)(ta[slot] + (2 * wv + h) * 512), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(src_w0 + sc * 512, (lds_void_t*)(tw[slot] + wv * 512), 16,
                                     0, 0);
    if constexpr (kExtra > 0)
      __builtin_amdgcn_global_load_lds(
          src_w1 + sc * 512, (lds_void_t*)(wv < kExtra ? tw[slot] + (8 + wv) * 512 : spare),
          16, 0, 0);
  };

  f32x4_t acc[4][WB];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < WB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  auto read_frags = [&](const bf16_t* la, const bf16_t* lw, bf16x8_t* a, bf16x8_t* w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(la + (wm * 4 + i) * 512 + lane * 8));
#pragma unroll
    for (int j = 0; j < WB; ++j)
      w[j] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lw + (wn * WB + j) * 512 + lane * 8));
  };
  auto mfma_step = [&](const bf16x8_t* a, const bf16x8_t* w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], w[j], acc[i][j], 0, 0, 0);
    // The stage's direct loads after the first four MFMAs (the MFMA pipe
    // restarts right after the barrier), then the fragment reads of the next
    // stage interleaved with these MFMAs.
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);       // MFMA
    __builtin_amdgcn_sched_group_barrier(0x020, kLoads, 0);  // VMEM read
    for (int g = 0; g < 4 + WB; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * WB - 8 - WB, 0);
  };

  // The epilogue's row of each tile row (residual and scatter variants) or
  // RMSNorm_2's per-tile sums of the row (SwiGLU: every thread loads those of
  // row m0 + tid % 256, all kNMaxTiles of them, tiles past n_ss repeating the
  // last one), loaded ahead of the ring with no branch around a load, so the
  // first stage wait below covers them.
  int erow = 0;
  u32x2_t rinfo = {0u, 0u};
  float ssv[kNMaxTiles];
  if constexpr (MODE == kNarrowQkv) {
    if (tid < kNM) rinfo = *(const u32x2_t*)(ea.row_info + 2 * min(m0 + tid, M - 1));
  } else if constexpr (MODE == kNarrowSwiglu) {
    const int m = min(m0 + (tid & (kNM - 1)), M - 1);
#pragma unroll
    for (int t = 0; t < kNMaxTiles; ++t) ssv[t] = ea.ss_in[(int64_t)min(t, ea.n_ss - 1) * M + m];
  } else if (tid < kNM) {
    const int m = min(m0 + tid, M - 1);
    const int32_t* idx = MODE == kNarrowResid ? ea.res_idx : ea.out_idx;
    erow = idx ? idx[m] : m;
  }

#pragma unroll
  for (int st = 0; st < kAhead; ++st) issue(st, st);
  wait_vmcnt<(kAhead - 1) * kLoads>();  // this wave's stage-0 loads are in LDS
  // SwiGLU: the row's 1/rms (sums in tile order). Its loads are older than
  // the stage-0 loads, so they are in too; nothing moves across this point.
  float rnorm = 1.f;
  if constexpr (MODE == kNarrowSwiglu) {
    __builtin_amdgcn_sched_barrier(0);
    float t2 = 0.f;
#pragma unroll
    for (int t = 0; t < kNMaxTiles; ++t) t2 += t < ea.n_ss ? ssv[t] : 0.f;
    rnorm = 1.0f / sqrtf(t2 / (float)K + ea.eps);
  }
  stage_barrier();  // every wave's stage-0 loads are in LDS
  bf16x8_t fa[2][4], fw[2][WB];
  read_frags(ta[0], tw[0], fa[0], fw[0]);
  // One unrolled round: stages st0 .. st0 + kRound - 1. In the last, partial
  // round (masked) stages past the end load the last stage again and multiply
  // nothing.
  auto ring_round = [&](int st0, auto masked) {
#pragma unroll
    for (int u = 0; u < kRound; ++u) {
      const int st = st0 + u;
      wait_vmcnt<(kAhead - 2) * kLoads>();  // this wave's loads of stage st + 1 are in LDS
      stage_barrier();  // every wave's: stage st + 1 published, stage st - 1 read
      issue(st + kAhead, (u + kAhead) % kBuf);
      read_frags(ta[(u + 1) % kBuf], tw[(u + 1) % kBuf], fa[(u + 1) & 1], fw[(u + 1) & 1]);
      if (!decltype(masked)::value || st < stages) mfma_step(fa[u & 1], fw[u & 1]);
    }
  };
  const int full_end = stages - stages % kRound;
  for (int st0 = 0; st0 < full_end; st0 += kRound) ring_round(st0, std::false_type{});
  if (full_end < stages) ring_round(full_end, std::true_type{});
  wait_vmcnt<0>();  // no direct load outlives the workgroup

  // Epilogues. The idle ring holds each tile row's epilogue value in slot 4
  // (its row of the residual or the output, SwiGLU: its 1/rms; QKV: its
  // (position clamped to the RoPE table, cache block)). The residual,
  // scatter and QKV epilogues work one row quarter at a time: the waves of
  // quarter p put their fp32 accumulators in LDS as rows of TN + 4 floats
  // (16-row groups in slots 0-3; the 4-float pad spreads the four rows a
  // wave store touches over all banks), then every thread takes 8-column
  // pieces of those 64 rows, so each load and store is 16 contiguous bytes
  // per lane.
  __syncthreads();  // every wave is done with the ring
  int* const g_nrow = (int*)sa4;
  u32x2_t* const slots = (u32x2_t*)sa4;
  if (tid < kNM) {
    if constexpr (MODE == kNarrowQkv)
      slots[tid] = rinfo;
    else
      g_nrow[tid] = kSwi ? __float_as_int(rnorm) : erow;
  }
  __syncthreads();
  constexpr int TNP = TN + 4;  // staged row stride (floats)
  static_assert(16 * TNP * 4 <= kNM * kNK * 2, "a 16-row group fits a slot");
  auto st_row = [&](int rq) -> float* {  // row rq (0..63) of the staged quarter
    const int g = rq >> 4;
    return (float*)(g == 0 ? sa0 : g == 1 ? sa1 : g == 2 ? sa2 : sa3) + (rq & 15) * TNP;
  };
  // Accumulator layout: lane (j4, c16) of block (i, j) holds rows
  // 16 (4 wm + i) + 4 j4 + r, r < 4, of column 16 (WB wn + j) + c16.
  auto stage_quarter = [&](int p) {
    if (wm == p) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float* const row = st_row(16 * i + 4 * j4 + r);
#pragma unroll
          for (int j = 0; j < WB; ++j) row[16 * (WB * wn + j) + c16] = acc[i][j][r];
        }
    }
  };
  constexpr int kCh = TN / 8;                                  // 8-column pieces per row
  constexpr int kPer = (64 * kCh + kNThreads - 1) / kNThreads;  // pieces per thread and quarter
  if constexpr (MODE == kNarrowResid) {
    // x1 = acc + residual row (fp32 out), h = bf16(x1 * gamma) in tile
    // order, and the row's sum of x1^2 over the tile: per piece in column
    // order, then the pieces in order (slot 4, after the row indices).
    float* const ssp = (float*)sa4 + kNM;
    // A thread's residual pieces of all four quarters and its gamma pieces
    // (the same columns in every quarter), for clamped pieces (no branch),
    // before the first quarter: one memory round trip for the epilogue.
    u32x4_t rv[4][kPer], gv[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int it = min(tid + u * kNThreads, 64 * kCh - 1);
      const int rq = it / kCh, ch = it - rq * kCh;
      gv[u] = *(const u32x4_t*)(ea.gamma + n0 + 8 * ch);
#pragma unroll
      for (int p = 0; p < 4; ++p)
        rv[p][u] = *(const u32x4_t*)(ea.res_x + (int64_t)g_nrow[64 * p + rq] * N + n0 + 8 * ch);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      stage_quarter(p);
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int it = tid + u * kNThreads;
        if (it >= 64 * kCh) continue;
        const int rq = it / kCh, ch = it - rq * kCh;
        const float* a = st_row(rq) + 8 * ch;
        const f32x4_t a0 = *(const f32x4_t*)a, a1 = *(const f32x4_t*)(a + 4);
        float x1[8], y[8];
        float sq = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x1[2 * e] = (e < 2 ? a0[2 * e] : a1[2 * e - 4]) + bf16_to_f32(rv[p][u][e] & 0xFFFFu);
          x1[2 * e + 1] = (e < 2 ? a0[2 * e + 1] : a1[2 * e - 3]) + bf16_to_f32(rv[p][u][e] >> 16);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sq += x1[e] * x1[e];
          y[e] = x1[e] * bf16_to_f32(e & 1 ? gv[u][e >> 1] >> 16 : gv[u][e >> 1] & 0xFFFFu);
        }
        ssp[rq * kCh + ch] = sq;
        const int m = m0 + 64 * p + rq;
        if (m < M) {
          float* xo = ea.x1 + (int64_t)m * N + n0 + 8 * ch;
          *(f32x4_t*)xo = f32x4_t{x1[0], x1[1], x1[2], x1[3]};
          *(f32x4_t*)(xo + 4) = f32x4_t{x1[4], x1[5], x1[6], x1[7]};
          *(u32x4_t*)(ea.h + tile_off(m, n0 + 8 * ch, N)) =
              u32x4_t{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                      pack_bf16x2(y[6], y[7])};
        }
      }
      __syncthreads();
      if (tid < 64 && m0 + 64 * p + tid < M) {
        float t = 0.f;
        for (int ch = 0; ch < kCh; ++ch) t += ssp[tid * kCh + ch];
        ea.ss_part[(int64_t)(n0 / TN) * M + m0 + 64 * p + tid] = t;
      }
      __syncthreads();  // the quarter's staging and sums are read
    }
  } else if constexpr (MODE == kNarrowScatter) {
    // out[out_idx[m]] = bf16(x1 + acc), 8 columns per piece. A thread's x1
    // pieces of all four quarters are loaded before the first quarter.
    f32x4_t xv[4][kPer][2];
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int it = min(tid + u * kNThreads, 64 * kCh - 1);
        const int rq = it / kCh, ch = it - rq * kCh;
        const float* xr = ea.x1_in + (int64_t)min(m0 + 64 * p + rq, M - 1) * N + n0 + 8 * ch;
        xv[p][u][0] = *(const f32x4_t*)xr;
        xv[p][u][1] = *(const f32x4_t*)(xr + 4);
      }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      stage_quarter(p);
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int it = tid + u * kNThreads;
        if (it >= 64 * kCh) continue;
        const int rq = it / kCh, ch = it - rq * kCh;
        const int m = m0 + 64 * p + rq;
        if (m >= M) continue;
        const float* a = st_row(rq) + 8 * ch;
        const f32x4_t a0 = *(const f32x4_t*)a, a1 = *(const f32x4_t*)(a + 4);
        const f32x4_t s0 = xv[p][u][0] + a0, s1 = xv[p][u][1] + a1;
        *(u32x4_t*)(ea.out + (int64_t)g_nrow[64 * p + rq] * N + n0 + 8 * ch) =
            u32x4_t{pack_bf16x2(s0[0], s0[1]), pack_bf16x2(s0[2], s0[3]),
                    pack_bf16x2(s1[0], s1[1]), pack_bf16x2(s1[2], s1[3])};
      }
      __syncthreads();  // the quarter's staging is read
    }
  } else if constexpr (MODE == kNarrowQkv) {
    // Column block q of half 0 holds dims j of pair group q, block WB + q
    // the dims j + 64, so a staged row has both halves of each pair. Per
    // quarter: queries and keys in pieces of 8 pairs (rotate-half RoPE with
    // the table's fp32 cos/sin of (position, j), then 16-byte stores of the 8
    // j dims and of the 8 j + 64 dims: q_out [M][Hq][128], or the key tile
    // of the row's cache slot); values (not rotated) as 8-byte runs of four
    // tokens (the value tile order) where four staged rows fill slots
    // 4a .. 4a + 3 of one block, element by element otherwise.
    constexpr int kHd = 128, kTile = kBlockTokens * kHd;
    const int g0 = (n0 / TN) * WB;  // first pair group of the tile
    constexpr int kQK = 64 * WB * 2;  // (row, group, 8-pair half) pieces per quarter
    constexpr int kQKPer = (kQK + kNThreads - 1) / kNThreads;
    // The (cos, sin) of 8 pairs per piece, one quarter ahead.
    f32x4_t cs[2][kQKPer][4];
    auto load_cs = [&](int p, f32x4_t (&dst)[kQKPer][4]) {
#pragma unroll
      for (int u = 0; u < kQKPer; ++u) {
        const int it = min(tid + u * kNThreads, kQK - 1);
        const int c8 = it & 1, q = (it >> 1) % WB, rq = (it >> 1) / WB;
        const int jd0 = 16 * ((g0 + q) & 3) + 8 * c8;
        const f32x4_t* t =
            (const f32x4_t*)(ea.rope + ((int64_t)slots[64 * p + rq].x * (kHd / 2) + jd0) * 2);
#pragma unroll
        for (int v = 0; v < 4; ++v) dst[u][v] = t[v];
      }
    };
    load_cs(0, cs[0]);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (p + 1 < 4) load_cs(p + 1, cs[(p + 1) & 1]);
      stage_quarter(p);
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kQKPer; ++u) {
        const int it = tid + u * kNThreads;
        if (it >= kQK) continue;
        const int c8 = it & 1, q = (it >> 1) % WB, rq = (it >> 1) / WB;
        const int hh = (g0 + q) >> 2;
        const int m = m0 + 64 * p + rq;
        if (m >= M || hh >= ea.Hq + ea.Hkv) continue;  // values below
        const float* lo = st_row(rq) + 16 * q + 8 * c8;
        const float* up = st_row(rq) + 16 * (WB + q) + 8 * c8;
        uint32_t wl[4], wu[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float rl[2], ru[2];
#pragma unroll
          for (int f = 0; f < 2; ++f) {
            const int k = 2 * e + f;  // pair k of the piece
            const float c = cs[p & 1][u][k >> 1][2 * (k & 1)];
            const float sn = cs[p & 1][u][k >> 1][2 * (k & 1) + 1];
            rl[f] = lo[k] * c - up[k] * sn;
            ru[f] = up[k] * c + lo[k] * sn;
          }
          wl[e] = pack_bf16x2(rl[0], rl[1]);
          wu[e] = pack_bf16x2(ru[0], ru[1]);
        }
        const int jd0 = 16 * ((g0 + q) & 3) + 8 * c8;
        const u32x4_t vl = {wl[0], wl[1], wl[2], wl[3]}, vu = {wu[0], wu[1], wu[2], wu[3]};
        if (hh < ea.Hq) {
          bf16_t* dst = ea.q_out + ((int64_t)m * ea.Hq + hh) * kHd + jd0;
          *(u32x4_t*)dst = vl;
          *(u32x4_t*)(dst + 64) = vu;
        } else {
          const u32x2_t sl = slots[64 * p + rq];
          const int slot = (int)sl.x % kBlockTokens;
          bf16_t* tile = ea.k_cache + ((int64_t)(int)sl.y * ea.Hkv + (hh - ea.Hq)) * kTile;
          *(u32x4_t*)(tile + k_tile_offset(slot, jd0)) = vl;
          *(u32x4_t*)(tile + k_tile_offset(slot, jd0 + 64)) = vu;
        }
      }
      // Values: (row quad, group, 32 dims), the dim fastest.
      constexpr int kV = 16 * WB * 32;
      for (int it = tid; it < kV; it += kNThreads) {
        const int d32 = it & 31, q = (it >> 5) % WB, quad = (it >> 5) / WB;
        const int hh = (g0 + q) >> 2;
        if (hh < ea.Hq + ea.Hkv) continue;  // queries and keys above
        const int dim = 64 * (d32 >> 4) + 16 * ((g0 + q) & 3) + (d32 & 15);
        const int col = 16 * ((d32 >> 4) * WB + q) + (d32 & 15);  // staged column
        const int lr0 = 64 * p + 4 * quad;
        bf16_t* const vbase = ea.v_cache + (int64_t)(hh - ea.Hq - ea.Hkv) * kTile;
        uint32_t e4[4];
        u32x2_t sl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          e4[e] = f32_to_bf16(st_row(4 * quad + e)[col]);
          sl[e] = slots[lr0 + e];
        }
        const int t0 = (int)sl[0].x % kBlockTokens;
        bool run = m0 + lr0 + 3 < M && t0 % 4 == 0;
#pragma unroll
        for (int e = 1; e < 4; ++e)
          run = run && sl[e].y == sl[0].y && (int)sl[e].x % kBlockTokens == t0 + e;
        if (run) {
          *(u32x2_t*)(vbase + (int64_t)(int)sl[0].y * ea.Hkv * kTile + v_tile_offset(t0, dim)) =
              u32x2_t{e4[0] | (e4[1] << 16), e4[2] | (e4[3] << 16)};
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (m0 + lr0 + e < M)
              vbase[(int64_t)(int)sl[e].y * ea.Hkv * kTile +
                    v_tile_offset((int)sl[e].x % kBlockTokens, dim)] = (bf16_t)e4[e];
        }
      }
      __syncthreads();  // the quarter's staging is read
    }
  } else if constexpr (kSwi) {
    // Gate in blocks q < WB/2, up in blocks WB/2 + q, of outputs
    // o0 + TN/4 wn + 16 q + c16; h = silu(gate) * up, staged in LDS (row
    // quarter wm in slot wm, rows padded to kSS) and written in tile order
    // [M][F] as whole 1 KB blocks, one per wave store.
    constexpr int kSO = TN / 2;   // outputs per tile row
    constexpr int kSS = kSO + 8;  // staged row stride: 16-byte rows, conflict-free reads
    static_assert(kSO % 32 == 0 && 64 * kSS <= kNM * kNK, "staged quarter fits a slot");
    auto stg = [&](int k) -> bf16_t* {  // k wave-uniform
      return k == 0 ? sa0 : k == 1 ? sa1 : k == 2 ? sa2 : sa3;
    };
    bf16_t* const mine = stg(wm);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rl = i * 16 + 4 * j4 + r;  // row within the quarter
        const float rs = __int_as_float(g_nrow[wm * 64 + rl]);
#pragma unroll
        for (int q = 0; q < WB / 2; ++q) {
          const float g = acc[i][q][r] * rs, u = acc[i][WB / 2 + q][r] * rs;
          mine[rl * kSS + wn * (TN / 4) + 16 * q + c16] =
              (bf16_t)f32_to_bf16(silu_mul(g, u));
        }
      }
    __syncthreads();
    // Block (16-row group, 32-output group); lane l holds chunk l: row
    // l % 16 of the group, outputs 8 (l / 16) .. + 7 of the block.
    constexpr int kBlocks = (kNM / 16) * (kSO / 32);
    for (int bi = wv; bi < kBlocks; bi += kNThreads / kWave) {
      const int rg = bi / (kSO / 32), kb = bi % (kSO / 32);
      const int row = rg * 16 + (lane & 15), oc = kb * 32 + (lane >> 4) * 8;
      const u32x4_t v = *(const u32x4_t*)(stg(row >> 6) + (row & 63) * kSS + oc);
      if (m0 + row < M) *(u32x4_t*)(ea.h + tile_off(m0 + row, o0 + oc, F)) = v;
    }
  }
}

// Persistent SwiGLU variant (gate/up projection with RMSNorm_2 folded in):
// one workgroup per CU keeps a row tile and walks a list of column tiles, so
// the direct-load ring streams on across tile boundaries (the next tile's
// first stages load while a tile's epilogue runs, and no workgroup starts
// cold after the first), and the rows' 1/rms are taken once. Same main loop,
// stage order and epilogue arithmetic as gemm_narrow_kernel's SwiGLU mode,
// so every output is bit-identical to it.
//   * Grid: 256 workgroups, 32 per XCD (blockIdx % 8). Workgroup k of XCD x
//     takes row tile k % tiles_m and the column tiles
//     x + 8 (k / tiles_m + ng s), s = 0, 1, ..., ng = 32 / tiles_m: at each
//     step the workgroups of one XCD share ng W tiles in its L2, each read by
//     tiles_m of them.
//   * The ring's slots are in use during an epilogue, so each wave stages its
//     SwiGLU outputs through a private 16-row buffer and writes them as
//     16-byte tile-order pieces. After an epilogue all vector memory
//     operations are waited for: the partial wait counts of the ring assume
//     that only its loads are outstanding.
template <int TN>
__global__ __launch_bounds__(kNThreads) void gemm_narrow_swiglu_persistent_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, int M, int F, int K,
    bf16_t* __restrict__ H, const float* __restrict__ ss_in, int n_ss, float eps) {
  static_assert(TN % 64 == 0 && TN / 16 >= 8 && TN / 16 <= 16, "tile width");
  constexpr int WB = TN / 32, kWBlocks = TN / 16, kExtra = kWBlocks - 8;
  constexpr int kLoads = kExtra > 0 ? 4 : 3;
  constexpr int kBuf = narrow_slots(TN);
  constexpr int kAhead = kBuf - 1;
  constexpr int kRound = narrow_round(TN);
  constexpr int kWO = TN / 4;  // outputs of a wave's column half
  static_assert(kWO % 8 == 0, "16-byte output pieces");
  __shared__ __attribute__((aligned(16))) bf16_t sa0[kNM * kNK], sa1[kNM * kNK],
      sa2[kNM * kNK], sa3[kNM * kNK], sa4[kNM * kNK], sa5[kNM * kNK];
  __shared__ __attribute__((aligned(16))) bf16_t sw0[TN * kNK], sw1[TN * kNK], sw2[TN * kNK],
      sw3[TN * kNK], sw4[TN * kNK], sw5[TN * kNK];
  __shared__ __attribute__((aligned(16))) bf16_t spare[512];
  __shared__ __attribute__((aligned(16))) bf16_t stg[8][16 * kWO];  // per-wave output rows
  __shared__ float rn[kNM];                                         // the rows' 1/rms
  bf16_t* const ta[6] = {sa0, sa1, sa2, sa3, sa4, sa5};
  bf16_t* const tw[6] = {sw0, sw1, sw2, sw3, sw4, sw5};

  const int N = 2 * F;
  const int tiles_m = (M + kNM - 1) / kNM;  // divides 32 (host check)
  const int tiles_n = N / TN;
  const int x = blockIdx.x % kNXCDs, kx = blockIdx.x / kNXCDs;
  const int ng = 32 / tiles_m;
  const int n_first = x + kNXCDs * (kx / tiles_m), n_step = kNXCDs * ng;
  const int T = n_first < tiles_n ? (tiles_n - 1 - n_first) / n_step + 1 : 0;
  if (T == 0) return;  // the whole workgroup leaves
  const int m0 = (kx % tiles_m) * kNM;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv & 3, wn = wv >> 2;
  const int c16 = lane & 15, j4 = lane >> 4;
  const int stages = K / kNK;

  // W block of the first tile's block blk (the gate/up pairing of
  // gemm_narrow_kernel); later tiles are n_step tiles further, a fixed
  // number of blocks.
  const int o_first = n_first * (TN / 2);
  auto w_block = [&](int blk) -> int {
    const int h = blk / WB, r = blk % WB;
    const int o = o_first + h * (TN / 4) + 16 * (r % (WB / 2));
    return ((r < WB / 2 ? 0 : F) + o) >> 4;
  };
  const int64_t blk_elems = (int64_t)(K / kNK) * 512;
  const int64_t w_step = (int64_t)n_step * (TN / 32) * blk_elems;
  const bf16_t* src_a[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ag = min((m0 + 32 * wv + 16 * h) >> 4, (M - 1) >> 4);
    src_a[h] = A + (int64_t)ag * blk_elems + lane * 8;
  }
  const bf16_t* src_w0 = W + (int64_t)w_block(wv) * blk_elems + lane * 8;
  const bf16_t* src_w1 = W + (int64_t)w_block(wv < kExtra ? 8 + wv : wv) * blk_elems + lane * 8;
  // Stage st of the tile whose W blocks are w_off past the first tile's.
  // The stage offsets pass through empty asm statements: the compiler then
  // forms each address where it is used, instead of keeping precomputed
  // addresses of the unrolled stages (and of the prologue's, which the last
  // round's next-tile loads repeat) in registers.
  auto issue = [&](int64_t w_off, int st, int slot) {
    int64_t oa = (int64_t)st * 512, ow = w_off + (int64_t)st * 512;
    asm volatile("" : "+s"(oa), "+s"(ow));
#pragma unroll
    for (int h = 0; h < 2; ++h)
      __builtin_amdgcn_global_load_lds(src_a[h] + oa,
                                       (lds_void_t*)(ta[slot] + (2 * wv + h) * 512), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(src_w0 + ow, (lds_void_t*)(tw[slot] + wv * 512), 16, 0,
                                     0);
    if constexpr (kExtra > 0)
      __builtin_amdgcn_global_load_lds(
          src_w1 + ow, (lds_void_t*)(wv < kExtra ? tw[slot] + (8 + wv) * 512 : spare), 16, 0,
          0);
  };

  f32x4_t acc[4][WB];
  auto read_frags = [&](const bf16_t* la, const bf16_t* lw, bf16x8_t* a, bf16x8_t* w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(la + (wm * 4 + i) * 512 + lane * 8));
#pragma unroll
    for (int j = 0; j < WB; ++j)
      w[j] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lw + (wn * WB + j) * 512 + lane * 8));
  };
  auto mfma_step = [&](const bf16x8_t* a, const bf16x8_t* w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], w[j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);       // MFMA
    __builtin_amdgcn_sched_group_barrier(0x020, kLoads, 0);  // VMEM read
    for (int g = 0; g < 4 + WB; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * WB - 8 - WB, 0);
  };

  // RMSNorm_2's per-tile sums of row m0 + tid % 256 (tiles past n_ss repeat
  // the last), loaded ahead of the ring so the first stage wait covers them.
  float ssv[kNMaxTiles];
  {
    const int m = min(m0 + (tid & (kNM - 1)), M - 1);
#pragma unroll
    for (int t = 0; t < kNMaxTiles; ++t) ssv[t] = ss_in[(int64_t)min(t, n_ss - 1) * M + m];
  }
#pragma unroll
  for (int st = 0; st < kAhead; ++st) issue(0, st, st);
  wait_vmcnt<(kAhead - 1) * kLoads>();
  __builtin_amdgcn_sched_barrier(0);
  if (tid < kNM) {
    float t2 = 0.f;
#pragma unroll
    for (int t = 0; t < kNMaxTiles; ++t) t2 += t < n_ss ? ssv[t] : 0.f;
    rn[tid] = 1.0f / sqrtf(t2 / (float)K + eps);
  }
  stage_barrier();  // stage 0 and the 1/rms are in LDS
  bf16x8_t fa[2][4], fw[2][WB];
  read_frags(ta[0], tw[0], fa[0], fw[0]);
  // One unrolled round: stages st0 .. st0 + kRound - 1 of the tile at w_off
  // (a tile is a whole number of rounds, kAhead < kRound). Only in a tile's
  // last round do the loads run into the next tile (at w_next; after the
  // last tile, that tile again: loaded, never multiplied), and that round
  // leaves the next tile's first fragments unread, so they are not held
  // through the epilogue.
  auto ring_round = [&](int st0, int64_t w_off, int64_t w_next, auto last) {
#pragma unroll
    for (int u = 0; u < kRound; ++u) {
      wait_vmcnt<(kAhead - 2) * kLoads>();
      stage_barrier();
      if (!decltype(last)::value || u + kAhead < kRound)
        issue(w_off, st0 + u + kAhead, (u + kAhead) % kBuf);
      else
        issue(w_next, u + kAhead - kRound, (u + kAhead) % kBuf);
      if (!decltype(last)::value || u + 1 < kRound)
        read_frags(ta[(u + 1) % kBuf], tw[(u + 1) % kBuf], fa[(u + 1) & 1], fw[(u + 1) & 1]);
      mfma_step(fa[u & 1], fw[u & 1]);
    }
  };
  bf16_t* const mine = stg[wv];
  for (int s = 0; s < T; ++s) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WB; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (s > 0) {
      // After an epilogue: every vector memory operation done (its stores
      // too, which the ring's partial wait counts do not allow for), then
      // the tile's first stage is published and read.
      wait_vmcnt<0>();
      stage_barrier();
      read_frags(ta[0], tw[0], fa[0], fw[0]);
    }
    const int64_t w_off = (int64_t)s * w_step;
    const int64_t w_next = s + 1 < T ? w_off + w_step : w_off;
    for (int st0 = 0; st0 + kRound < stages; st0 += kRound)
      ring_round(st0, w_off, w_off, std::false_type{});
    ring_round(stages - kRound, w_off, w_next, std::true_type{});
    // Epilogue: h = silu(gate) * up for outputs o0 + kWO wn + 16 q + c16
    // (gate in blocks q < WB / 2, up in WB / 2 + q), 16 rows at a time
    // through this wave's buffer, then 16-byte pieces of 8 outputs of a row
    // to H in tile order [M][F].
    const int o0 = (n_first + n_step * s) * (TN / 2) + kWO * wn;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float rs = rn[64 * wm + 16 * i + 4 * j4 + r];
#pragma unroll
        for (int q = 0; q < WB / 2; ++q) {
          const float g = acc[i][q][r] * rs, u = acc[i][WB / 2 + q][r] * rs;
          mine[(4 * j4 + r) * kWO + 16 * q + c16] = (bf16_t)f32_to_bf16(silu_mul(g, u));
        }
      }
      // Reads of the rows just written by this wave (LDS operations of a
      // wave are performed in order). tile_off(m, o0 + 8 pc, F) for
      // m = mr + row (mr a multiple of 16) splits into a wave-uniform block
      // offset and a lane part, so the address is a scalar base plus a
      // 32-bit offset.
      const int mr = m0 + 64 * wm + 16 * i;
      bf16_t* const hb = H + ((int64_t)(mr >> 4) * (F >> 5) + (o0 >> 5)) * 512;
#pragma unroll
      for (int c0 = 0; c0 < 16 * kWO / 8; c0 += 64) {
        const int c = c0 + lane;
        const int row = c / (kWO / 8), pc = c % (kWO / 8);
        const int kk = (o0 & 31) + 8 * pc;
        if (c < 16 * kWO / 8) {
          const u32x4_t v = *(const u32x4_t*)(mine + row * kWO + pc * 8);
          if (mr + row < M) *(u32x4_t*)(hb + ((kk >> 5) * 512 + ((kk & 31) >> 3) * 128 + row * 8)) = v;
        }
      }
    }
  }
  wait_vmcnt<0>();  // no direct load outlives the workgroup
}

template <int MODE>
hipError_t launch_narrow(int tn, const uint16_t* A, const uint16_t* W, int M, int N, int K,
                         const NarrowEpiArgs& ea, hipStream_t st) {
  if (tn == 0 || N % tn != 0 || K % kNK != 0) return hipErrorInvalidValue;
  const dim3 grid(((M + kNM - 1) / kNM) * (N / tn));
  if constexpr (MODE == kNarrowSwiglu) {
    if (tn != 192) return hipErrorInvalidValue;
    COCO_LAUNCH((gemm_narrow_kernel<192, MODE>), grid, dim3(kNThreads), 0, st,
                (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
  } else if constexpr (MODE == kNarrowSwigluPlain) {
    if (tn != 128) return hipErrorInvalidValue;
    COCO_LAUNCH((gemm_narrow_kernel<128, MODE>), grid, dim3(kNThreads), 0, st,
                (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
  } else if constexpr (MODE == kNarrowQkv) {
    if (tn == 224)
      COCO_LAUNCH((gemm_narrow_kernel<224, MODE>), grid, dim3(kNThreads), 0, st,
                  (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
    else if (tn == 192)
      COCO_LAUNCH((gemm_narrow_kernel<192, MODE>), grid, dim3(kNThreads), 0, st,
                  (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
    else if (tn == 160)
      COCO_LAUNCH((gemm_narrow_kernel<160, MODE>), grid, dim3(kNThreads), 0, st,
                  (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
    else
      return hipErrorInvalidValue;
  } else if (tn == 160) {
    COCO_LAUNCH((gemm_narrow_kernel<160, MODE>), grid, dim3(kNThreads), 0, st,
                (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
  } else if (tn == 128) {
    COCO_LAUNCH((gemm_narrow_kernel<128, MODE>), grid, dim3(kNThreads), 0, st,
                (const bf16_t*)A, (const bf16_t*)W, M, N, K, ea);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int narrow_tile_n(int N) {
  if (N > 0 && N % 128 == 0 && N / 128 <= kNMaxTiles) return 128;
  if (N > 0 && N % 160 == 0 && N / 160 <= kNMaxTiles) return 160;
  return 0;
}

hipError_t launch_gemm_narrow_resid_bf16(const uint16_t* A, const uint16_t* W, int M, int N,
                                         int K, const uint16_t* res_x, const int32_t* res_idx,
                                         const uint16_t* gamma, float* x1, uint16_t* h,
                                         float* ss_part, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!res_x || !gamma || !x1 || !h || !ss_part) return hipErrorInvalidValue;
  NarrowEpiArgs ea{};
  ea.res_x = res_x;
  ea.res_idx = res_idx;
  ea.gamma = gamma;
  ea.x1 = x1;
  ea.h = h;
  ea.ss_part = ss_part;
  return launch_narrow<kNarrowResid>(narrow_tile_n(N), A, W, M, N, K, ea, st);
}

hipError_t launch_gemm_narrow_scatter_bf16(const uint16_t* A, const uint16_t* W, int M, int N,
                                           int K, const float* x1, uint16_t* out,
                                           const int32_t* out_idx, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!x1 || !out) return hipErrorInvalidValue;
  NarrowEpiArgs ea{};
  ea.x1_in = x1;
  ea.out = out;
  ea.out_idx = out_idx;
  return launch_narrow<kNarrowScatter>(narrow_tile_n(N), A, W, M, N, K, ea, st);
}

bool narrow_swiglu_fits(int F, int K) { return F > 0 && (2 * F) % 192 == 0 && K % kNK == 0; }

hipError_t launch_gemm_narrow_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                          uint16_t* H, int M, int F, int K, const float* ss_in,
                                          int ss_tiles, float eps, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!narrow_swiglu_fits(F, K) || !H || !ss_in || ss_tiles < 1 || ss_tiles > kNMaxTiles)
    return hipErrorInvalidValue;
  // Persistent when the row tiles divide the 32 workgroups of an XCD and a
  // tile is a whole number of unrolled rounds.
  const int tiles_m = (M + kNM - 1) / kNM;
  if (32 % tiles_m == 0 && (K / kNK) % narrow_round(192) == 0) {
    COCO_LAUNCH((gemm_narrow_swiglu_persistent_kernel<192>), dim3(256), dim3(kNThreads), 0, st,
                (const bf16_t*)A, (const bf16_t*)W_gate_up, M, F, K, (bf16_t*)H, ss_in,
                ss_tiles, eps);
    return hipGetLastError();
  }
  NarrowEpiArgs ea{};
  ea.h = H;
  ea.ss_in = ss_in;
  ea.n_ss = ss_tiles;
  ea.eps = eps;
  return launch_narrow<kNarrowSwiglu>(192, A, W_gate_up, M, 2 * F, K, ea, st);
}

bool narrow_swiglu_plain_fits(int M, int F, int K) {
  if (M <= 0 || F <= 0 || (2 * F) % 128 != 0 || K % kNK != 0) return false;
  return (int64_t)((M + kNM - 1) / kNM) * (2 * F / 128) <= 256;  // one round of workgroups
}

hipError_t launch_gemm_narrow_swiglu_plain_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                                uint16_t* H, int M, int F, int K,
                                                hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!narrow_swiglu_plain_fits(M, F, K) || !H) return hipErrorInvalidValue;
  NarrowEpiArgs ea{};
  ea.h = H;
  return launch_narrow<kNarrowSwigluPlain>(128, A, W_gate_up, M, 2 * F, K, ea, st);
}

int narrow_qkv_tile_n(int Hq, int Hkv, int K) {
  const int N = (Hq + 2 * Hkv) * 128;
  if (K % kNK != 0) return 0;
  // Prefer a width whose tile count is a multiple of 32 (whole rounds of 256
  // CUs over a 2048-row chunk), else the widest that divides N.
  for (int tn : {224, 192, 160})
    if (N % tn == 0 && (N / tn) % 32 == 0) return tn;
  for (int tn : {224, 192, 160})
    if (N % tn == 0) return tn;
  return 0;
}

hipError_t launch_gemm_narrow_qkv_bf16(const uint16_t* A, const uint16_t* W_qkv, int M, int K,
                                       const NarrowEpiArgs& ea, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  const int tn = narrow_qkv_tile_n(ea.Hq, ea.Hkv, K);
  if (tn == 0 || !ea.row_info || !ea.rope || !ea.q_out || !ea.k_cache || !ea.v_cache)
    return hipErrorInvalidValue;
  return launch_narrow<kNarrowQkv>(tn, A, W_qkv, M, (ea.Hq + 2 * ea.Hkv) * 128, K, ea, st);
}

}  // namespace coco
