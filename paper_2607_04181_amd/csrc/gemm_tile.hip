// Large-tile GEMM for prefill-sized row counts (bf16 MFMA, fp32 out).
//
//   C[m][n] = sum_k A[m][k] * W[n][k]      A: [M][K], W: [N][K], both bf16
//
// W is in tile order (pack_tile_order), and so is A (tile_off: the prefill
// activations are written in it by their producers): each 16 rows x 32 k of
// either is one contiguous 1 KB block, which one 16-byte-per-lane load
// copies to LDS unchanged (lane l, chunk l), so each tile of a stage is 16
// such blocks. The bf16 activation outputs (SwiGLU and residual variants)
// are written in tile order for the next projection.
//
// Prefill is bound by MFMA throughput, so the kernel is built for reuse:
//   * a 512-thread workgroup computes a 256 x 256 tile; each of its eight
//     waves owns a 128 x 64 sub-tile as 4 x 2 v_mfma_f32_32x32x16_bf16
//     accumulators, two waves per SIMD so that one wave's MFMAs issue while
//     the other waits on LDS or the barrier;
//   * 32-deep K stages of the A and W tiles go straight from global memory
//     to LDS (global_load_lds, 16 bytes per lane, no register staging) into
//     a ring of four buffers, three stages in flight (a fifth buffer, the
//     whole 160 KB of LDS, measured no faster). Each wave fills 32 rows
//     of both tiles with four 1 KB loads per stage; the tile-order blocks
//     give each 16-lane group of a fragment read 256 contiguous bytes;
//   * one barrier per stage: the barrier at the top of stage st publishes
//     stage st + 1, so the first fragments of the next stage are read while
//     the second half of this stage's MFMAs runs, and the stage that the
//     next loads overwrite (st - 1) has been fully read by every wave;
//   * workgroups are remapped so that the tiles sharing a W column slab run
//     on the same XCD (blockIdx % 8) back to back and hit its L2;
//   * narrow outputs with a long K are split into K-slices (tile_splits, a
//     function of (N, K) only) so the grid covers the CUs;
//   * for the gate/up projection a variant pairs gate and up columns inside
//     each wave and writes silu(gate) * up directly in bf16;
//   * for the QKV projection (unsplit) a variant orders each head's columns so
//     that a lane holds both dims j and j + 64 of its rows, applies RoPE in
//     registers and writes queries and the cache tiles directly in bf16;
//   * for the O projection (unsplit) a variant adds the residual and writes
//     the RMSNorm_2 operand bf16(x1 * gamma) with per-tile row sums of x1^2,
//     which the gate/up variant turns into each row's 1/rms.
// Every output element is summed over k in ascending 16-steps within its
// slice, independent of M and of the tile it falls in, so request-aligned
// prefill splits give identical bits.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kTM = 256, kTN = 256, kTK = 32;
constexpr int kTBuf = 4;        // LDS ring depth (stages)
constexpr int kTAhead = kTBuf - 1;  // stages in flight
constexpr int kSliceQuant = 128;    // K-slice granularity of the plans
constexpr int kTThreads = 512;  // 8 waves, two per SIMD
constexpr int kXCDs = 8;

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;

// LDS element offset of chunk c (0..3) of tile row r in a tile of 16
// tile-order blocks.
__device__ __forceinline__ int wblk(int r, int c) { return (r >> 4) * 512 + (c * 16 + (r & 15)) * 8; }

// One LDS object per ring slot, so the compiler tracks each slot's pending
// direct loads on its own and never drains the ring before a fragment read.
__shared__ __attribute__((aligned(16))) bf16_t g_ta0[kTM * kTK], g_ta1[kTM * kTK],
    g_ta2[kTM * kTK], g_ta3[kTM * kTK];
__shared__ __attribute__((aligned(16))) bf16_t g_tw0[kTN * kTK], g_tw1[kTN * kTK],
    g_tw2[kTN * kTK], g_tw3[kTN * kTK];
// Per-row values of the tile for the epilogues: QKV: position (clamped to the
// RoPE table) and cache block; residual: source row of the residual; SwiGLU
// with RMSNorm_2 folded in: the row's 1/rms (bits of a float).
__shared__ int g_row_pos[kTM], g_row_blk[kTM];

enum { kTilePartial = 0, kTileSwiglu = 1, kTileQkv = 2, kTileResid = 3, kTileSwigluNorm = 4 };
constexpr int kMaxNormTiles = 32;  // d <= 32 * 256 for the folded RMSNorm_2

// kTilePartial: C is the fp32 partial of K-slice blockIdx.y.
// kTileSwiglu: W is the [2F][K] gate/up matrix; each 32-column half of a
// wave's 64 columns holds gate rows and the other the matching up rows, so
// each lane owns both factors of its outputs and the epilogue writes
// h = silu(gate) * up in bf16 to the [M][F] buffer `H` (N = 2F, one K-slice).
// kTileQkv: W is the [(Hq + 2 Hkv) * 128][K] QKV matrix, N a multiple of 256
// (two heads per tile), one K-slice; see the epilogue.
// kTileResid: one K-slice, N a multiple of 256; C = x1 = A W^T + residual
// (fp32), H = bf16(x1 * gamma) and ea.ss_part[n0 / 256][m] = sum over the
// tile's columns of x1^2.
// kTileSwigluNorm: kTileSwiglu whose gate and up of row m are first scaled by
// 1 / sqrt(sum_t ss_in[t][m] / ea.d + ea.eps), t < ea.n_ss, in tile order.
// k_slice is a multiple of kTK.
template <int MODE>
__global__ __launch_bounds__(kTThreads) void gemm_tile_kernel(const bf16_t* __restrict__ A,
                                                                 const bf16_t* __restrict__ W,
                                                                 float* __restrict__ C,
                                                                 bf16_t* __restrict__ H, int M,
                                                                 int N, int K, int k_slice,
                                                                 TileEpiArgs ea) {
  constexpr bool FUSE = MODE == kTileSwiglu || MODE == kTileSwigluNorm;
  bf16_t* const ta[kTBuf] = {g_ta0, g_ta1, g_ta2, g_ta3};
  bf16_t* const tw[kTBuf] = {g_tw0, g_tw1, g_tw2, g_tw3};

  const int tiles_m = (M + kTM - 1) / kTM;
  const int nb = gridDim.x;
  const int b = blockIdx.x;
  const int full = (nb / kXCDs) * kXCDs;
  const int lid = b < full ? (b % kXCDs) * (nb / kXCDs) + b / kXCDs : b;
  const int m0 = (lid % tiles_m) * kTM;
  const int n0 = (lid / tiles_m) * kTN;
  const int kb = blockIdx.y * k_slice;
  C += (int64_t)blockIdx.y * M * N;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv & 1, wn = wv >> 1;  // 128-row half, 64-column quarter
  const int l32 = lane & 31, hi = lane >> 5;

  // Fused tile of 128 outputs o0 .. o0+127: tile rows 64w + 32j + i hold gate
  // row o0 + 32w + i for j = 0 and up row F + o0 + 32w + i for j = 1.
  // QKV tile of heads n0/128 and n0/128 + 1: tile rows 64w + 32j + i hold
  // dim 32(w % 2) + 64j + i of head n0/128 + w/2, so wave column quarter w
  // gets dims jd and jd + 64 (jd = 32(w % 2) + i) of one head in its two
  // 32-column halves.
  const int F = N / 2, o0 = n0 / 2;
  auto w_row = [&](int r) {
    if (MODE == kTileQkv) return n0 + (r & 0x80) + ((r >> 6) & 1) * 32 + ((r >> 5) & 1) * 64 + (r & 31);
    if (!FUSE) return min(n0 + r, N - 1);
    const int w = r >> 6, j = (r >> 5) & 1, i = r & 31;
    return (j ? F : 0) + o0 + 32 * w + i;
  };

  // This lane's sources: wave wv fills rows 32 wv .. 32 wv + 31 of both tiles,
  // 16 rows (1 KB) per load, a stage of a 16-row group being one tile-order
  // block that lane l copies chunk by chunk. A: rows m0 + 16 g' ..; groups
  // past the last row read the last group (its rows past M are stale and
  // never stored). W: every 16-row group of tile rows maps to 16 consecutive
  // W rows from a multiple of 16 (w_row); groups past N read the last block
  // (never stored).
  const int stages = k_slice / kTK;
  const bf16_t* src_a[2];
  const bf16_t* src_w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ag = min((m0 + 32 * wv + 16 * h) >> 4, (M - 1) >> 4);
    src_a[h] = A + ((int64_t)ag * (K / kTK) + kb / kTK) * 512 + lane * 8;
    const int wg = w_row(32 * wv + 16 * h) >> 4;
    src_w[h] = W + ((int64_t)wg * (K / kTK) + kb / kTK) * 512 + lane * 8;
  }
  // Loads past the slice repeat its last stage (never multiplied).
  auto issue = [&](int st, int slot) {
    const int sc = min(st, stages - 1);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      __builtin_amdgcn_global_load_lds(src_a[h] + sc * 512,
                                       (lds_void_t*)(ta[slot] + (32 * wv + 16 * h) * kTK), 16,
                                       0, 0);
      __builtin_amdgcn_global_load_lds(src_w[h] + sc * 512,
                                       (lds_void_t*)(tw[slot] + (32 * wv + 16 * h) * kTK), 16,
                                       0, 0);
    }
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto read_frags = [&](const bf16_t* la, const bf16_t* lw, int kk, bf16x8_t* a, bf16x8_t* w) {
    const int c = kk * 2 + hi;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = __builtin_bit_cast(
          bf16x8_t, *(const u32x4_t*)(&la[wblk(wm * 128 + i * 32 + l32, c)]));
#pragma unroll
    for (int j = 0; j < 2; ++j)
      w[j] = __builtin_bit_cast(
          bf16x8_t, *(const u32x4_t*)(&lw[wblk(wn * 64 + j * 32 + l32, c)]));
  };
  auto mfma_step = [&](const bf16x8_t* a, const bf16x8_t* w) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], w[j], acc[i][j], 0, 0, 0);
    // Interleave the six fragment reads issued next to these MFMAs.
    for (int g = 0; g < 6; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
  };

  // Per-row inputs of the epilogues, loaded ahead of the ring so the stage
  // waits below also cover them: QKV row slot (position, cache block);
  // residual source row; the per-tile sums of squares of the row.
  u32x2_t rinfo = {0u, 0u};
  int rrow = 0;
  float ssv[kMaxNormTiles];
  constexpr bool fold_norm = MODE == kTileSwigluNorm;
  if (tid < kTM) {
    const int m = min(m0 + tid, M - 1);
    if constexpr (MODE == kTileQkv) rinfo = *(const u32x2_t*)(ea.row_info + 2 * m);
    if constexpr (MODE == kTileResid) rrow = ea.res_idx ? ea.res_idx[m] : m;
  }
  // Every thread loads the sums of row m0 + tid % 256, all kMaxNormTiles of
  // them (tiles past n_ss repeat the last one and are not added), with no
  // branch around a load: the wait for them then counts only the ring loads
  // issued after them.
  if constexpr (fold_norm) {
    const int m = min(m0 + (tid & (kTM - 1)), M - 1);
#pragma unroll
    for (int t = 0; t < kMaxNormTiles; ++t)
      ssv[t] = ea.ss_in[(int64_t)min(t, ea.n_ss - 1) * M + m];
  }

#pragma unroll
  for (int st = 0; st < kTAhead; ++st) issue(st, st);
  wait_vmcnt<4 * (kTAhead - 1)>();  // this wave's stage-0 loads are in LDS
  // The row's 1/rms (sums in tile order): its loads, older than the stage-0
  // loads, are in too. Nothing moves across this point, so the sums are
  // read after the wait above and need no wait of their own.
  float rnorm = 1.f;
  if constexpr (fold_norm) {
    __builtin_amdgcn_sched_barrier(0);
    float t2 = 0.f;
#pragma unroll
    for (int t = 0; t < kMaxNormTiles; ++t) t2 += t < ea.n_ss ? ssv[t] : 0.f;
    rnorm = 1.0f / sqrtf(t2 / (float)ea.d + ea.eps);
  }
  stage_barrier();                   // ... and every wave's
  bf16x8_t a0[4], w0[2], a1[4], w1[2];
  read_frags(ta[0], tw[0], 0, a0, w0);
  // One round of the ring: stages st0 .. st0 + kTBuf - 1. In the last,
  // partial round (MASKED) stages past the end load the last stage again and
  // multiply nothing.
  auto ring_round = [&](int st0, auto masked) {
#pragma unroll
    for (int u = 0; u < kTBuf; ++u) {
      const int st = st0 + u;
      const bool live = !decltype(masked)::value || st < stages;
      wait_vmcnt<4 * (kTAhead - 2)>();  // this wave's loads of stage st + 1 are in LDS
      stage_barrier();  // every wave's: stage st + 1 published, stage st - 1 read
      issue(st + kTAhead, (u + kTAhead) % kTBuf);
      read_frags(ta[u], tw[u], 1, a1, w1);
      if (live) mfma_step(a0, w0);
      read_frags(ta[(u + 1) % kTBuf], tw[(u + 1) % kTBuf], 0, a0, w0);
      if (live) mfma_step(a1, w1);
    }
  };
  const int full_end = stages - stages % kTBuf;
  for (int st0 = 0; st0 < full_end; st0 += kTBuf) ring_round(st0, std::false_type{});
  if (full_end < stages) ring_round(full_end, std::true_type{});
  wait_vmcnt<0>();  // no direct load outlives the workgroup

  if constexpr (MODE == kTileQkv) {
    // The tile rows' slots (position clamped to the RoPE table, cache block)
    // and, when a head of the tile is rotated, the RoPE table rows of their
    // positions, staged by direct loads into the now idle ring (row lr at
    // ring object lr / 32, 512 bytes per row), so the stores below wait on
    // no load.
    constexpr int kHd = 128, kTile = kBlockTokens * kHd;
    if (tid < kTM) {
      g_row_pos[tid] = (int)rinfo.x;
      g_row_blk[tid] = (int)rinfo.y;
    }
    __syncthreads();
    const int hh0 = n0 >> 7;
    auto ring = [](int k) -> bf16_t* {  // k wave-uniform
      switch (k) {
        case 0: return g_ta0;
        case 1: return g_ta1;
        case 2: return g_ta2;
        case 3: return g_ta3;
        case 4: return g_tw0;
        case 5: return g_tw1;
        case 6: return g_tw2;
        default: return g_tw3;
      }
    };
    if (hh0 < ea.Hq + ea.Hkv) {
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const int row = 32 * wv + 2 * c + hi;
        __builtin_amdgcn_global_load_lds(
            ea.rope + ((int64_t)g_row_pos[row] * (kHd / 2) + 2 * l32) * 2,
            (lds_void_t*)(ring(wv) + c * 512), 16, 0, 0);
      }
      wait_vmcnt<0>();
      __syncthreads();
    }
    // Rotate-half RoPE on query and key heads: this lane holds dims jd and
    // jd + 64 of head hh for its 64 rows. Queries go to q_out [M][Hq][128];
    // keys (rotated) and values to their cache slot (block, position % 16).
    const int hh = hh0 + (wn >> 1);
    const int jd = (wn & 1) * 32 + l32;
    const int kind = hh < ea.Hq ? 0 : (hh < ea.Hq + ea.Hkv ? 1 : 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int lr = wm * 128 + i * 32 + 8 * jj + 4 * hi + r;
          const int m = m0 + lr;
          if (m >= M) continue;
          float lo = acc[i][0][4 * jj + r], up = acc[i][1][4 * jj + r];
          const int pos = g_row_pos[lr];
          if (kind != 2) {
            const f32x2_t cs =
                ((const f32x2_t*)ring(wm * 4 + i))[(8 * jj + 4 * hi + r) * (kHd / 2) + jd];
            const float rlo = lo * cs.x - up * cs.y, rup = up * cs.x + lo * cs.y;
            lo = rlo;
            up = rup;
          }
          if (kind == 0) {
            bf16_t* dst = ea.q_out + ((int64_t)m * ea.Hq + hh) * kHd;
            dst[jd] = (bf16_t)f32_to_bf16(lo);
            dst[jd + 64] = (bf16_t)f32_to_bf16(up);
          } else {
            const int slot = pos % kBlockTokens;
            const int g = hh - ea.Hq - (kind == 2 ? ea.Hkv : 0);
            bf16_t* tile = (kind == 1 ? ea.k_cache : ea.v_cache) +
                           ((int64_t)g_row_blk[lr] * ea.Hkv + g) * kTile;
            if (kind == 1) {
              tile[k_tile_offset(slot, jd)] = (bf16_t)f32_to_bf16(lo);
              tile[k_tile_offset(slot, jd + 64)] = (bf16_t)f32_to_bf16(up);
            } else {
              tile[v_tile_offset(slot, jd)] = (bf16_t)f32_to_bf16(lo);
              tile[v_tile_offset(slot, jd + 64)] = (bf16_t)f32_to_bf16(up);
            }
          }
        }
    return;
  }
  if constexpr (MODE == kTileResid) {
    // x1 = acc + residual row (bf16 [*][N], row ea.res_idx[m] or m), staged by
    // direct loads into the idle ring (tile row lr at ring object lr / 32,
    // 512 bytes per row); H = bf16(x1 * gamma). Each lane's x1^2 over its two
    // columns goes back into the ring as [lr][128] with the 4-byte
    // slot k = 32 wn + l32 stored at k ^ (lr % 32) (conflict-free reads),
    // and thread t < 256 sums row t's 128 slots in slot order.
    if (tid < kTM) g_row_pos[tid] = rrow;
    __syncthreads();
    auto ring = [](int k) -> bf16_t* {  // k wave-uniform
      switch (k) {
        case 0: return g_ta0;
        case 1: return g_ta1;
        case 2: return g_ta2;
        case 3: return g_ta3;
        case 4: return g_tw0;
        case 5: return g_tw1;
        case 6: return g_tw2;
        default: return g_tw3;
      }
    };
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int row = 32 * wv + 2 * c + hi;
      __builtin_amdgcn_global_load_lds(ea.res_x + (int64_t)g_row_pos[row] * N + n0 + 8 * l32,
                                       (lds_void_t*)(ring(wv) + c * 512), 16, 0, 0);
    }
    float gam[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) gam[j] = bf16_to_f32(ea.gamma[n0 + wn * 64 + j * 32 + l32]);
    wait_vmcnt<0>();
    __syncthreads();
    float v[4][4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int lr = wm * 128 + i * 32 + 8 * jj + 4 * hi + r;
          const int m = m0 + lr;
          const bf16_t* xrow = ring(wm * 4 + i) + (8 * jj + 4 * hi + r) * 256;
          float sq = 0.f;
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int col = wn * 64 + j * 32 + l32;
            const float x1 = acc[i][j][4 * jj + r] + bf16_to_f32(xrow[col]);
            sq += x1 * x1;
            if (m < M) {
              C[(int64_t)m * N + n0 + col] = x1;
              H[tile_off(m, n0 + col, N)] = (bf16_t)f32_to_bf16(x1 * gam[j]);
            }
          }
          v[i][jj][r] = sq;
        }
    __syncthreads();  // every wave is done with the residual tile
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rr = 8 * jj + 4 * hi + r;  // row within ring object wm * 4 + i
          ((float*)ring(wm * 4 + i))[rr * 128 + ((wn * 32 + l32) ^ rr)] = v[i][jj][r];
        }
    __syncthreads();
    if (tid < kTM && m0 + tid < M) {
      const float* sr = (const float*)ring(tid >> 5) + (tid & 31) * 128;
      float t2 = 0.f;
      for (int k = 0; k < 128; ++k) t2 += sr[k ^ (tid & 31)];
      ea.ss_part[(int64_t)(n0 / kTN) * M + m0 + tid] = t2;
    }
    return;
  }
  if (FUSE) {
    if constexpr (fold_norm) {
      if (tid < kTM) g_row_pos[tid] = __float_as_int(rnorm);
      __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = o0 + 32 * wn + l32;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int lr = wm * 128 + i * 32 + 8 * jj + 4 * hi + r;
          const int m = m0 + lr;
          float g = acc[i][0][4 * jj + r], u = acc[i][1][4 * jj + r];
          if constexpr (fold_norm) {
            const float rs = __int_as_float(g_row_pos[lr]);
            g *= rs;
            u *= rs;
          }
          if (m < M) H[tile_off(m, o, F)] = (bf16_t)f32_to_bf16(silu_mul(g, u));
        }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + l32;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm * 128 + i * 32 + 8 * jj + 4 * hi + r;
          if (m < M && n < N) C[(int64_t)m * N + n] = acc[i][j][4 * jj + r];
        }
    }
}

}  // namespace

// K-slices from (N, K) alone: narrow outputs (few 256-column tiles) with a
// long K are split into ~8k-deep slices so the grid covers the CUs; the
// partials are summed in slice order by the consumer.
int tile_splits(int N, int K) {
  const int tiles_n = (N + kTN - 1) / kTN;
  if (tiles_n >= 48) return 1;
  int S = (K + 4096) / 8192;
  if (S < 1) S = 1;
  if (S > 4) S = 4;
  while (S > 1 && (K / kSliceQuant) % S != 0) --S;
  return S;  // 1..4: the split counts the epilogues are built for
}

hipError_t launch_gemm_tile_bf16(const uint16_t* A, const uint16_t* W, float* C, int M, int N,
                                 int K, int S, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (S < 1 || K % (kSliceQuant * S) != 0) return hipErrorInvalidValue;
  const int tiles = ((M + kTM - 1) / kTM) * ((N + kTN - 1) / kTN);
  COCO_LAUNCH(gemm_tile_kernel<kTilePartial>, dim3(tiles, S), dim3(kTThreads), 0, st, A,
                     W, C, nullptr, M, N, K, K / S, TileEpiArgs{});
  return hipGetLastError();
}

hipError_t launch_gemm_tile_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                        uint16_t* H, int M, int F, int K, const float* ss_in,
                                        int ss_tiles, float eps, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (F % (kTN / 2) != 0 || K % kSliceQuant != 0 || tile_splits(2 * F, K) != 1)
    return hipErrorInvalidValue;
  TileEpiArgs ea{};
  if (ss_in) {
    if (ss_tiles < 1 || ss_tiles > kMaxNormTiles) return hipErrorInvalidValue;
    ea.ss_in = ss_in;
    ea.n_ss = ss_tiles;
    ea.d = K;
    ea.eps = eps;
  }
  const int tiles = ((M + kTM - 1) / kTM) * (2 * F / kTN);
  if (ss_in)
    COCO_LAUNCH(gemm_tile_kernel<kTileSwigluNorm>, dim3(tiles, 1), dim3(kTThreads), 0, st, A,
                W_gate_up, nullptr, H, M, 2 * F, K, K, ea);
  else
    COCO_LAUNCH(gemm_tile_kernel<kTileSwiglu>, dim3(tiles, 1), dim3(kTThreads), 0, st, A,
                W_gate_up, nullptr, H, M, 2 * F, K, K, ea);
  return hipGetLastError();
}

bool tile_norm2_foldable(int d, int qdim, int F) {
  return d % kTN == 0 && d / kTN <= kMaxNormTiles && qdim % kSliceQuant == 0 &&
         tile_splits(d, qdim) == 1 && F % (kTN / 2) == 0 && tile_splits(2 * F, d) == 1;
}

hipError_t launch_gemm_tile_resid_bf16(const uint16_t* A, const uint16_t* W, int M, int N, int K,
                                       const uint16_t* res_x, const int32_t* res_idx,
                                       const uint16_t* gamma, float* x1, uint16_t* h,
                                       float* ss_part, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (N % kTN != 0 || N / kTN > kMaxNormTiles || K % kSliceQuant != 0 ||
      tile_splits(N, K) != 1 || !res_x || !gamma || !x1 || !h || !ss_part)
    return hipErrorInvalidValue;
  TileEpiArgs ea{};
  ea.res_x = res_x;
  ea.res_idx = res_idx;
  ea.gamma = gamma;
  ea.ss_part = ss_part;
  const int tiles = ((M + kTM - 1) / kTM) * (N / kTN);
  COCO_LAUNCH(gemm_tile_kernel<kTileResid>, dim3(tiles, 1), dim3(kTThreads), 0, st, A, W,
                     x1, h, M, N, K, K, ea);
  return hipGetLastError();
}

bool tile_qkv_fusable(int Hq, int Hkv, int K) {
  const int N = (Hq + 2 * Hkv) * 128;
  return N % kTN == 0 && K % kSliceQuant == 0 && tile_splits(N, K) == 1;
}

hipError_t launch_gemm_tile_qkv_bf16(const uint16_t* A, const uint16_t* W_qkv, int M, int K,
                                     const TileEpiArgs& ea, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!tile_qkv_fusable(ea.Hq, ea.Hkv, K) || !ea.row_info || !ea.rope) return hipErrorInvalidValue;
  const int N = (ea.Hq + 2 * ea.Hkv) * 128;
  const int tiles = ((M + kTM - 1) / kTM) * (N / kTN);
  COCO_LAUNCH(gemm_tile_kernel<kTileQkv>, dim3(tiles, 1), dim3(kTThreads), 0, st, A,
                     W_qkv, nullptr, nullptr, M, N, K, K, ea);
  return hipGetLastError();
}

}  // namespace coco
