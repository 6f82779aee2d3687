// Weight-streaming GEMM for decode-sized row counts (bf16 MFMA, fp32 out).
//
//   part[s][m][n] = sum over k in K-slice s of A[m][k] * W[n][k]
//
// A: [M][K] activations, bf16. W: the [N][K] weights (nn.Linear layout) in
// tile order (pack_tile_order below): every 16 rows x 32 k of W are one
// contiguous 1 KB block laid out as the B operand of a
// v_mfma_f32_16x16x32_bf16 step, lane by lane.
// Decode is bound by reading W once from HBM, so the kernel is built around
// that stream:
//   * a workgroup of WAVES waves owns 16*WAVES output columns and one K-slice;
//     each wave streams the 16 weight rows of its columns straight into VGPRs
//     (each 16-byte-per-lane load one contiguous 1 KB block; plain loads
//     measured faster here than non-temporal ones), keeping two stages of
//     128 k in flight;
//   * the activation tile [rows][128 k] of a stage is shared by the waves
//     through LDS (double-buffered); its 16-byte chunks are XOR-swizzled
//     with the row (chunk ^ row % 16), so both the row-wise stores and the
//     16-rows-per-instruction fragment reads hit distinct banks;
//   * each 16x16 output tile is accumulated with v_mfma_f32_16x16x32_bf16 in
//     ascending k.
// A pass covers up to 128 rows. For batches of more than 128 rows (8-wave
// and fused 7-wave plans) and of 65-128 rows (8-wave plans), a row-split
// variant takes over (gemm_skinny_rows_kernel below): there the weight tile
// of a stage goes to LDS and the row tiles are dealt to the waves, since every
// wave reading the whole activation tile from LDS costs more LDS time as the
// batch grows.
// The NORM variant (decode QKV projection) folds the row gather and the
// first RMSNorm into the activation staging: it reads the layer input rows
// x[row_idx[m]] directly, stages bf16(x * gamma), and writes each row's sum
// of x^2 over its K-slice; the 1/rms factor of a row is a scalar that the
// consumer applies to the summed partials.
// The plan (WAVES, split count S) is chosen from (N, K) alone (skinny_plan);
// every output element is
// summed in the same k order for any M, so a row's result does not depend on
// the other rows in the call (batch invariance). Partials of the S slices
// are added in slice order by the consumer epilogue.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kBK = 128;       // k per pipeline stage
constexpr int kCUs = 256;

// LDS element offset of 16-byte chunk c (0..15) of activation row r.
__device__ __forceinline__ int a_swz(int r, int c) { return r * kBK + ((c ^ (r & 15)) << 3); }

typedef __attribute__((address_space(3))) void lds_void_t;

// NORM row sums, by one wave: ss[blockIdx.y][r] = sum of x^2 over the K-slice
// for rows r = r_first, r_first + gridDim.x, ... below r_end (each row of a
// pass by one workgroup of the slice), per lane in chunk order, then a fixed
// butterfly: a row's sum never depends on the batch.
__device__ __forceinline__ void norm_row_sums(const bf16_t* __restrict__ A,
                                              const int32_t* __restrict__ row_idx, int M, int K,
                                              int k_begin, int k_slice, int r_first, int r_end,
                                              float* __restrict__ ss, int lane) {
  for (int r = r_first; r < r_end; r += gridDim.x) {
    const bf16_t* xr = A + (int64_t)((row_idx != nullptr) ? row_idx[r] : r) * K + k_begin;
    float t = 0.f;
    for (int c = lane; c < k_slice / 8; c += 64) {
      const u32x4_t u = *(const u32x4_t*)(xr + c * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(u[e] << 16), hi = __uint_as_float(u[e] & 0xFFFF0000u);
        t = fmaf(lo, lo, t);
        t = fmaf(hi, hi, t);
      }
    }
    t = wave_sum(t);
    if (lane == 0) ss[(int64_t)blockIdx.y * M + r] = t;
  }
}

// bf16(x * gamma) of eight packed elements, the product in fp32.
__device__ __forceinline__ u32x4_t scale_bf16x8(u32x4_t x, u32x4_t g) {
  u32x4_t y;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float lo = __uint_as_float(x[e] << 16), hi = __uint_as_float(x[e] & 0xFFFF0000u);
    const float glo = __uint_as_float(g[e] << 16), ghi = __uint_as_float(g[e] & 0xFFFF0000u);
    y[e] = pack_bf16x2(lo * glo, hi * ghi);
  }
  return y;
}

// FUSE: W is the [2F][K] gate/up matrix (N = 2F, one K-slice). Lanes
// c16 < 8 of a wave stream gate rows o0..o0+7 and lanes c16 >= 8 the
// matching up rows, so the epilogue pairs lanes c16 and c16+8 and writes
// h = silu(gate) * up in bf16 to H[M][F] instead of fp32 partials.
// NORM: A holds the layer input rows, row m of the call at A[row_idx[m]]
// (row_idx null: row m); the staged operand is bf16(A * gamma) and
// ss[blockIdx.y][m] receives the row's sum of squares over the K-slice
// (row m by the workgroup of the slice with blockIdx.x == m % gridDim.x).
template <int WAVES, int MT, int PF, bool FUSE, bool NORM>
__global__ __launch_bounds__(WAVES * 64) void gemm_skinny_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, float* __restrict__ part,
    bf16_t* __restrict__ H, int M, int N, int K, int k_slice,
    const int32_t* __restrict__ row_idx, const bf16_t* __restrict__ gamma,
    float* __restrict__ ss, bool h_tiled) {
  constexpr int NT = WAVES * 64;
  constexpr int kChunks = MT * 16 * (kBK / 8);  // 16-byte A chunks per stage
  constexpr int kPerT = (kChunks + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][MT * 16 * kBK];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, j4 = lane >> 4;
  const int o0 = (blockIdx.x * WAVES + wv) * 8;  // fused: this wave's 8 outputs
  const int n_col = FUSE ? (c16 < 8 ? o0 + c16 : N / 2 + o0 + c16 - 8)
                         : blockIdx.x * (16 * WAVES) + wv * 16 + c16;  // this lane's weight row
  const int k_begin = blockIdx.y * k_slice;
  const int stages = k_slice / kBK;
  float* out = FUSE ? nullptr : part + (int64_t)blockIdx.y * M * N;

  // This lane's chunk of the stage's step t (row n_col, k = k_begin + 128 st +
  // 32 t + 8 j4) in tile order: block (n_col / 16) * (K / 32) + k / 32, chunk
  // j4 * 16 + n_col % 16; a wave's load of one step is one 1 KB block.
  const bf16_t* wrow =
      W + ((int64_t)(n_col >> 4) * (K / 32) + k_begin / 32) * 512 + (j4 * 16 + (n_col & 15)) * 8;

  // The steady-state loop is branch-free so that the compiler can wait for
  // exactly the loads each step consumes: prefetches past the slice are
  // clamped to its last stage (an L2 hit, never used), and stages past the
  // slice in the final group get a zero activation tile (adding exact zeros
  // leaves every sum unchanged).
  const int groups = (stages + PF - 1) / PF;
  for (int m0 = 0; m0 < M; m0 += MT * 16) {
    f32x4_t acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Weight ring: PF stages x 4 k-steps of 8 bf16 per lane.
    u32x4_t wreg[PF][4];
    auto load_w = [&](int st, int u) {
      const bf16_t* src = wrow + min(st, stages - 1) * (kBK / 32) * 512;
#pragma unroll
      for (int t = 0; t < 4; ++t) wreg[u][t] = *(const u32x4_t*)(src + t * 512);
    };
#pragma unroll
    for (int u = 0; u < PF; ++u) load_w(u, u);

    // Activation ring: stage x lives in register slot x % 2 from the start of
    // stage x-2 until it is copied to LDS buffer x % 2 at the end of stage
    // x-1, so its L2 latency is hidden behind two stages of weight streaming.
    // A thread stages the same (row, 16-byte chunk column) of every stage:
    // rows (tid + v * NT) / 16 and chunk column tid % 16 (NT is a multiple of
    // 16), so under NORM it needs one gain chunk per stage and keeps one sum
    // of squares per row it stages.
    u32x4_t areg[2][kPerT];
    u32x4_t greg[2];
    int arow[kPerT];  // source row of each staged chunk (32-bit to spare registers)
#pragma unroll
    for (int v = 0; v < kPerT; ++v) {
      const int q = min(tid + v * NT, kChunks - 1);
      const int m = min(m0 + (q >> 4), M - 1);
      arow[v] = (NORM && row_idx) ? row_idx[m] : m;
    }
    const bf16_t* a_col = A + k_begin + (tid & 15) * 8;  // NT % 16 == 0: column tid % 16
    auto load_a = [&](int st, int slot) {
      const int sc = min(st, stages - 1);
#pragma unroll
      for (int v = 0; v < kPerT; ++v)
        areg[slot][v] = *(const u32x4_t*)(a_col + (int64_t)arow[v] * K + sc * kBK);
      if (NORM) greg[slot] = *(const u32x4_t*)(gamma + k_begin + sc * kBK + (tid & 15) * 8);
    };
    auto store_a = [&](int st, int slot, int buf) {
#pragma unroll
      for (int v = 0; v < kPerT; ++v) {
        const int q = tid + v * NT;
        const bool live = st < stages && m0 + (q >> 4) < M;
        u32x4_t val = live ? areg[slot][v] : u32x4_t{0u, 0u, 0u, 0u};
        if (NORM) val = scale_bf16x8(val, greg[slot]);  // x * gamma in fp32, rounded to bf16
        if (q < kChunks) *(u32x4_t*)(&lds[buf][a_swz(q >> 4, q & 15)]) = val;
      }
    };

    load_a(0, 0);
    load_a(1, 1);
    // Row sums of squares of this pass while the first weight stages are in flight.
    if (NORM && wv == 0)
      norm_row_sums(A, row_idx, M, K, k_begin, k_slice, m0 + blockIdx.x, min(M, m0 + MT * 16),
                    ss, lane);
    store_a(0, 0, 0);
    __syncthreads();

    static_assert(PF % 2 == 0, "ring slots are indexed by stage parity");
    for (int g = 0; g < groups; ++g) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        const int st = g * PF + u;
        const int buf = u & 1;  // == st & 1 since PF is even
        load_a(st + 2, u & 1);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bf16x8_t b = __builtin_bit_cast(bf16x8_t, wreg[u][t]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const bf16x8_t a = __builtin_bit_cast(
                bf16x8_t, *(const u32x4_t*)(&lds[buf][a_swz(mt * 16 + c16, t * 4 + j4)]));
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[mt], 0, 0, 0);
          }
        }
        load_w(st + PF, u);
        store_a(st + 1, (u + 1) & 1, buf ^ 1);
        __syncthreads();
      }
    }

    // D layout: lane holds rows 4*j4 + r of column c16 of each 16x16 tile.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + mt * 16 + j4 * 4 + r;
        if (FUSE) {
          // The up value of this lane's output sits 8 lanes up.
          const float u = __shfl_down(acc[mt][r], 8, 16);
          const float g = acc[mt][r];
          if (c16 < 8 && m < M)
            H[h_tiled ? tile_off(m, o0 + c16, N / 2) : (int64_t)m * (N / 2) + o0 + c16] =
                (bf16_t)f32_to_bf16(silu_mul(g, u));
        } else if (m < M) {
          // Non-temporal: the partials are read once, by the next kernel.
          __builtin_nontemporal_store(acc[mt][r], out + (int64_t)m * N + n_col);
        }
      }
    }
  }
}

// Row-split variant for passes of 256 or 128 rows (16 or 8 row tiles). Same
// outputs, bit for bit, as gemm_skinny_kernel: every 16x16 output tile is the same chain of
// v_mfma_f32_16x16x32_bf16 (activation fragment as the A operand, weight
// fragment as B) in ascending k.
//   * the workgroup's 16*WAVES weight rows of a 64-k stage go straight to LDS
//     (global_load_lds, 16 bytes per lane; wave w fills the 16 rows of column
//     tile w as two 1 KB loads, one per 32 k) into a ring of four slots, three
//     stages in flight. LDS holds each 16 rows x 32 k in tile order (chunk
//     (k / 8) * 16 + row), so a load reads one tile-order block of W (or, in
//     the SwiGLU variant, the halves of two blocks that hold the tile's eight
//     gate and eight up rows) and a fragment read gives each 16-lane group
//     256 contiguous bytes;
//   * row tile t of the pass (rows 16t .. 16t + 15) belongs to wave t % WAVES;
//     a wave loads its tiles' activation fragments from memory straight into
//     registers (A in tile order: one 1 KB block per load), AST stages deep (stage st + AST once stage st has been
//     multiplied), and multiplies them with all 16*WAVES weight rows (LDS
//     reads per stage: WAVES * 2 KB per wave);
//   * one barrier per stage: the wait before it covers this wave's direct
//     loads of the stage; after it, every wave's are in LDS and the slot the
//     stage's new loads overwrite was read by every wave in the stage before.
// The stage loop is unrolled by four (ring and activation slots then known at
// compile time); the stage counts of the 7- and 8-wave decode shapes are
// multiples of four, and other counts finish with up to three guarded stages.
constexpr int kRK = 64;        // k per stage
constexpr int kRSlots = 4;     // weight ring slots
constexpr int kRAhead = 3;     // weight stages in flight


// Weight ring of the row-split kernel, one LDS object per slot (sized for 8
// waves), so the compiler tracks each slot's pending direct loads on its own
// and an LDS read waits only for the loads into its slot.
constexpr int kRMaxRows = 16 * 8;
__shared__ __attribute__((aligned(16))) bf16_t g_rw0[kRMaxRows * kRK], g_rw1[kRMaxRows * kRK],
    g_rw2[kRMaxRows * kRK], g_rw3[kRMaxRows * kRK];

// ROWT: row tiles per pass (16 or 8). AST: activation stages in registers
// (2 or 4; stage st + AST is loaded after stage st's MFMAs).
template <int WAVES, bool FUSE, int ROWT, int AST>
__global__ __launch_bounds__(WAVES * 64) void gemm_skinny_rows_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, float* __restrict__ part,
    bf16_t* __restrict__ H, int M, int N, int K, int k_slice, bool h_tiled) {
  static_assert(kRSlots % AST == 0, "activation slots must follow the unrolled stages");
  constexpr int kRowTiles = ROWT;
  constexpr int kRAst = AST;
  constexpr int TPW = (kRowTiles + WAVES - 1) / WAVES;  // row tiles per wave
  constexpr int NR = 16 * WAVES;                         // weight rows per workgroup
  constexpr int kDLoads = 2;                             // direct loads per stage
  constexpr int kALoads = 2 * TPW;                       // activation loads per stage
  static_assert(NR <= kRMaxRows, "weight ring sized for 8 waves");
  bf16_t* const ring[kRSlots] = {g_rw0, g_rw1, g_rw2, g_rw3};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c16 = lane & 15, j4 = lane >> 4;
  const int k_begin = blockIdx.y * k_slice;
  const int stages = k_slice / kRK;
  float* out = FUSE ? nullptr : part + (int64_t)blockIdx.y * M * N;

  // Weight row of workgroup row rho = 16 j + c (column tile j, column c of
  // it): the rows wave j of gemm_skinny_kernel streams.
  auto w_row = [&](int rho) -> int {
    const int j = rho >> 4, c = rho & 15;
    if (FUSE) {
      const int o = (blockIdx.x * WAVES + j) * 8;
      return c < 8 ? o + c : N / 2 + o + c - 8;
    }
    return blockIdx.x * NR + rho;
  };
  // Direct load q of this wave: k 32q .. 32q + 31 of the stage for the 16
  // rows of column tile wv; lane l = 16 j4 + c16 lands at LDS chunk l of the
  // slot's block 2 wv + q and reads row w_row(16 wv + c16), k 32q + 8 j4 ..
  // + 7, which is chunk j4 * 16 + row % 16 of tile-order block
  // (row / 16) * (K / 32) + k / 32.
  // Addresses are a uniform base (advanced per stage) plus a fixed 32-bit byte
  // offset per lane, so no address register is rewritten inside the loop (a
  // rewrite of a register that a pending load shares would wait for it).
  const char* wbase = (const char*)(W + (int64_t)(k_begin / 32) * 512);
  uint32_t woff[kDLoads];
  {
    const int row = w_row(16 * wv + c16);
#pragma unroll
    for (int q = 0; q < kDLoads; ++q)
      woff[q] = (uint32_t)((row >> 4) * (K / 32) + q) * 1024u +
                (uint32_t)((j4 * 16 + (row & 15)) * 16);
  }
  // Stages past the slice repeat its last stage (never multiplied).
  auto issue_w = [&](int st, int slot) {
    const char* b = wbase + (size_t)min(st, stages - 1) * (kRK / 32) * 1024;
#pragma unroll
    for (int q = 0; q < kDLoads; ++q)
      __builtin_amdgcn_global_load_lds((const void*)(b + woff[q]),
                                       (lds_void_t*)(ring[slot] + (16 * wv + 8 * q) * kRK), 16,
                                       0, 0);
  };

  for (int m0 = 0; m0 < M; m0 += kRowTiles * 16) {
    // Activation fragments: lane (c16, j4) of row tile i holds, for k-step t,
    // elements 32t + 8j4 .. + 7 of the stage of row m0 + 16 tile + c16. A is
    // in tile order (tile_off), so that fragment is chunk j4 * 16 + c16 = lane
    // of a 1 KB block and each load reads one whole block. Row tiles past the
    // last row read the last tile (its rows past M are stale, never stored).
    const char* abase = (const char*)(A + (int64_t)(k_begin / 32) * 512);
    uint32_t aoff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int rt = min((m0 >> 4) + wv + i * WAVES, (M - 1) >> 4);
      aoff[i] = (uint32_t)rt * (uint32_t)(K / 32) * 1024u + (uint32_t)lane * 16u;
    }
    u32x4_t areg[kRAst][TPW][2];
    auto load_a = [&](int st, int slot) {
      const char* b = abase + (size_t)min(st, stages - 1) * ((kRK / 32) * 1024);
#pragma unroll
      for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int t = 0; t < 2; ++t) areg[slot][i][t] = *(const u32x4_t*)(b + aoff[i] + t * 1024);
    };

    f32x4_t acc[TPW][WAVES];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
      for (int j = 0; j < WAVES; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Issue order: weights of stage x + 3 at the top of stage x, activations
    // of x + AST at its end, so that after the weights of stage x come
    // exactly three activation groups and two weight groups, and after the
    // activations of stage x AST - 1 weight groups and as many activation
    // groups. The prologue issues the same sequence for stages -3 .. -1
    // (activations of stages below 0 do not exist: with AST = 2 stage 0's
    // weights are followed by one activation group fewer, hence its own wait).
#pragma unroll
    for (int j = 0; j < AST - 3; ++j) load_a(j, j);
#pragma unroll
    for (int x = 0; x < 3; ++x) {
      issue_w(x, x);
      if (x + AST - 3 >= 0) load_a(x + AST - 3, (x + AST - 3) % AST);
    }
    if constexpr (AST < 3) wait_vmcnt<AST * kALoads + 2 * kDLoads>();

    // Stage st: ring slot st % 4, activation slot st % 2. A wave whose last
    // row tile is past the pass multiplies that tile too (wave-uniform
    // branches around the MFMAs would break up the schedule); it is never
    // stored.
    auto stage = [&](int st, auto slot_c) {
      constexpr int u = decltype(slot_c)::value;
      constexpr int as = u % kRAst;
      wait_vmcnt<3 * kALoads + 2 * kDLoads>();
      stage_barrier();
      // This stage's activations before its MFMAs, stated here: the compiler
      // does not count direct and register loads in one queue and would wait
      // for all of them.
      wait_vmcnt<(AST - 1) * (kALoads + kDLoads)>();
      issue_w(st + kRAhead, (u + kRAhead) % kRSlots);
      const bf16_t* lw = ring[u];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int j = 0; j < WAVES; ++j) {
          const bf16x8_t b = __builtin_bit_cast(
              bf16x8_t, *(const u32x4_t*)(&lw[16 * j * kRK + ((t * 4 + j4) * 16 + c16) * 8]));
#pragma unroll
          for (int i = 0; i < TPW; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, areg[as][i][t]), b, acc[i][j], 0, 0, 0);
        }
      }
      // Weight fragments two reads ahead of their MFMAs, not all at once.
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read
      for (int x = 0; x < 2 * WAVES - 2; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, TPW, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * TPW, 0);
      // Refill this activation slot (read above) with stage st + AST; the
      // scheduler may not hoist these loads above the MFMAs (that would hold
      // one more activation stage in registers).
      __builtin_amdgcn_sched_barrier(0);
      load_a(st + kRAst, as);
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    using S3 = std::integral_constant<int, 3>;
    // Whole groups of four stages branch-free, then the rest.
    const int full = stages / kRSlots, rem = stages % kRSlots;
    for (int g = 0; g < full; ++g) {
      const int st = g * kRSlots;
      stage(st, S0{});
      stage(st + 1, S1{});
      stage(st + 2, S2{});
      stage(st + 3, S3{});
    }
    const int st = full * kRSlots;
    if (rem > 0) stage(st, S0{});
    if (rem > 1) stage(st + 1, S1{});
    if (rem > 2) stage(st + 2, S2{});
    wait_vmcnt<0>();  // no direct load outlives the pass
    __syncthreads();  // every wave is done with the ring

    // D layout: lane holds rows 4*j4 + r of column c16 of each 16x16 tile.
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int tile = wv + i * WAVES;
      if (tile >= kRowTiles) continue;  // wave-uniform
#pragma unroll
      for (int j = 0; j < WAVES; ++j) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + tile * 16 + j4 * 4 + r;
          if (FUSE) {
            const float u = __shfl_down(acc[i][j][r], 8, 16);
            const float g = acc[i][j][r];
            const int o = (blockIdx.x * WAVES + j) * 8;
            if (c16 < 8 && m < M)
              H[h_tiled ? tile_off(m, o + c16, N / 2) : (int64_t)m * (N / 2) + o + c16] =
                  (bf16_t)f32_to_bf16(silu_mul(g, u));
          } else if (m < M) {
            __builtin_nontemporal_store(acc[i][j][r],
                                        out + (int64_t)m * N + blockIdx.x * NR + 16 * j + c16);
          }
        }
      }
    }
  }
}

struct NormArgs {
  const int32_t* row_idx = nullptr;
  const uint16_t* gamma = nullptr;
  float* ss = nullptr;
};

template <int WAVES, int MT, bool FUSE, bool NORM>
hipError_t launch_plan(const uint16_t* A, const uint16_t* W, float* part, uint16_t* H, int M,
                       int N, int K, int S, NormArgs na, bool h_tiled, hipStream_t st) {
  // Two stages of weights in flight per wave (~56 KB per CU at 7 waves) cover
  // HBM latency for 64-row tiles; deeper rings measured slower there (more
  // requests queued behind each other) and cost registers. With 128-row tiles
  // and 8 waves, four stages measured faster (70B O and down shapes), and no
  // worse on the 32B gate/up shape (the NORM variant would spill with four).
  constexpr int PF = (MT == 8 && WAVES == 8 && !NORM) ? 4 : 2;
  COCO_LAUNCH((gemm_skinny_kernel<WAVES, MT, PF, FUSE, NORM>), dim3(N / (16 * WAVES), S),
                     dim3(WAVES * 64), 0, st, A, W, part, H, M, N, K, K / S, na.row_idx,
                     (const bf16_t*)na.gamma, na.ss, h_tiled);
  return hipGetLastError();
}

// Which kernel a plan of `waves` waves runs for M rows: the row-split kernel
// where it measured faster, above 128 rows for 7- and 8-wave plans (8B
// gate/up and down at 256 rows: 113 -> 89 us and 64 -> 46 us against two
// 128-row passes; with fewer waves or the folded norm it measured slower),
// and for 128-row passes of 8-wave plans. (No decode shape here has an
// unfused 7-wave plan; those keep the 128-row kernel.) Its per-lane byte
// offsets are 32-bit: both operands must be under 4 GB.
enum RowsKind { kNoRows = 0, kRows16, kRows8 };
RowsKind rows_kind(int waves, bool fuse, bool norm, int N, int K, int M) {
  if (M <= 64 || norm || !(waves == 8 || (waves == 7 && fuse))) return kNoRows;
  const bool fits = (int64_t)N * K * 2 < (int64_t(1) << 32) &&
                    (int64_t)((M + 15) / 16 * 16) * K * 2 < (int64_t(1) << 32);
  if (!fits) return kNoRows;
  if (M > 128) return kRows16;
  return waves == 8 ? kRows8 : kNoRows;
}

template <int WAVES, bool FUSE, bool NORM>
hipError_t launch_waves(const uint16_t* A, const uint16_t* W, float* part, uint16_t* H, int M,
                        int N, int K, int S, NormArgs na, bool h_tiled, hipStream_t st) {
  if (M <= 64)
    return launch_plan<WAVES, 4, FUSE, NORM>(A, W, part, H, M, N, K, S, na, h_tiled, st);
  if constexpr ((WAVES == 8 || (WAVES == 7 && FUSE)) && !NORM) {
    switch (rows_kind(WAVES, FUSE, NORM, N, K, M)) {
      case kRows16:
        COCO_LAUNCH((gemm_skinny_rows_kernel<WAVES, FUSE, 16, WAVES == 8 ? 4 : 2>),
                    dim3(N / (16 * WAVES), S), dim3(WAVES * 64), 0, st, A, W, part, H, M, N,
                    K, K / S, h_tiled);
        return hipGetLastError();
      case kRows8:
        COCO_LAUNCH((gemm_skinny_rows_kernel<8, FUSE, 8, 4>), dim3(N / 128, S), dim3(512), 0,
                    st, A, W, part, H, M, N, K, K / S, h_tiled);
        return hipGetLastError();
      default:
        break;
    }
  }
  return launch_plan<WAVES, 8, FUSE, NORM>(A, W, part, H, M, N, K, S, na, h_tiled, st);
}

template <bool FUSE, bool NORM>
hipError_t launch_any(const uint16_t* A, const uint16_t* W, float* part, uint16_t* H, int M,
                      int N, int K, SkinnyPlan plan, NormArgs na, bool h_tiled,
                      hipStream_t st) {
  switch (plan.waves) {
    case 4: return launch_waves<4, FUSE, NORM>(A, W, part, H, M, N, K, plan.S, na, h_tiled, st);
    case 5: return launch_waves<5, FUSE, NORM>(A, W, part, H, M, N, K, plan.S, na, h_tiled, st);
    case 6: return launch_waves<6, FUSE, NORM>(A, W, part, H, M, N, K, plan.S, na, h_tiled, st);
    case 7: return launch_waves<7, FUSE, NORM>(A, W, part, H, M, N, K, plan.S, na, h_tiled, st);
    default: return launch_waves<8, FUSE, NORM>(A, W, part, H, M, N, K, plan.S, na, h_tiled, st);
  }
}

}  // namespace

// Grid plan from (N, K) only (so a row's sums never depend on the batch).
// Measured on the decode shapes: the best plans fill the 256 CUs with exactly
// one round of workgroups; among those, K-slices of at least 1024 (eight
// stages) and then more waves per workgroup win. Without such a plan, the
// unsplit weight stream wins (split-K partials and short slices cost more),
// with the fullest last round of workgroups and then the most waves: on the
// 70B gate/up shape (N = 57344, K = 8192, 128 rows) 7 waves (two full rounds)
// took 206 us against 220 us for 8 waves (448 workgroups). The wave count
// does not change any output's k order.
SkinnyPlan skinny_plan(int N, int K) {
  auto valid = [&](int waves, int S) {
    if (N % (16 * waves)) return false;
    if (K % (S * kBK)) return false;
    if (S > 1 && K / S < 4 * kBK) return false;
    return true;
  };
  SkinnyPlan best{0, 0};
  int best_rank = -1;
  for (int waves = 4; waves <= 8; ++waves)
    for (int S = 1; S <= 16; S *= 2) {
      if (!valid(waves, S)) continue;
      const int wgs = (N / (16 * waves)) * S;
      if (wgs != kCUs) continue;
      const int rank = (K / S >= 8 * kBK ? 100 : 0) + waves * 2 + (S == 1 ? 1 : 0);
      if (rank > best_rank) {
        best_rank = rank;
        best = SkinnyPlan{waves, S};
      }
    }
  if (best.waves) return best;
  int64_t best_fill = -1;  // workgroups * 2^16 / (rounds * 256): last-round fill
  for (int waves = 8; waves >= 4; --waves) {
    if (!valid(waves, 1)) continue;
    const int64_t wgs = N / (16 * waves);
    const int64_t rounds = (wgs + kCUs - 1) / kCUs;
    const int64_t fill = (wgs << 16) / (rounds * kCUs);
    if (fill > best_fill) {
      best_fill = fill;
      best = SkinnyPlan{waves, 1};
    }
  }
  return best;  // {0, 0}: no plan (N not a multiple of 64 or K of 128)
}

hipError_t launch_gemm_skinny_bf16(const uint16_t* A, const uint16_t* W, float* part, int M,
                                   int N, int K, SkinnyPlan plan, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (plan.waves < 4 || plan.waves > 8 || N % (16 * plan.waves) != 0 ||
      K % (plan.S * kBK) != 0)
    return hipErrorInvalidValue;
  return launch_any<false, false>(A, W, part, nullptr, M, N, K, plan, NormArgs{}, false, st);
}

bool skinny_reads_tiled(int N, int K, int M, bool fuse) {
  const SkinnyPlan plan = skinny_plan(N, K);
  return plan.waves != 0 && rows_kind(plan.waves, fuse, false, N, K, M) != kNoRows;
}

hipError_t launch_gemm_skinny_norm_bf16(const uint16_t* X, const int32_t* row_idx,
                                        const uint16_t* gamma, const uint16_t* W, float* part,
                                        float* ss, int M, int N, int K, SkinnyPlan plan,
                                        hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (plan.waves < 4 || plan.waves > 8 || N % (16 * plan.waves) != 0 ||
      K % (plan.S * kBK) != 0)
    return hipErrorInvalidValue;
  NormArgs na;
  na.row_idx = row_idx;
  na.gamma = gamma;
  na.ss = ss;
  return launch_any<false, true>(X, W, part, nullptr, M, N, K, plan, na, false, st);
}

hipError_t launch_gemm_skinny_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                          uint16_t* H, int M, int F, int K, SkinnyPlan plan,
                                          bool h_tiled, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (plan.S != 1 || plan.waves < 4 || plan.waves > 8 || (2 * F) % (16 * plan.waves) != 0 ||
      K % kBK != 0)
    return hipErrorInvalidValue;
  return launch_any<true, false>(A, W_gate_up, nullptr, H, M, 2 * F, K, plan, NormArgs{},
                                 h_tiled, st);
}

// ----------------------------------------------------------------------------
// Tile order of a bf16 weight matrix [N][K] (N % 16 == 0, K % 32 == 0): the
// 1 KB block b = (n / 16) * (K / 32) + k / 32 holds rows 16 (n / 16) .. + 15
// and columns 32 (k / 32) .. + 31 as 64 chunks of 8 consecutive k, chunk
// ((k % 32) / 8) * 16 + n % 16 -- lane j4 * 16 + c16 of the B operand of a
// v_mfma_f32_16x16x32_bf16 step (row c16, k 8 j4 .. + 7). One thread per
// 16-byte chunk, read in row order.
// ----------------------------------------------------------------------------
namespace {
__global__ __launch_bounds__(256) void pack_tile_order_kernel(const u32x4_t* __restrict__ w,
                                                              int64_t n_chunks, int K,
                                                              u32x4_t* __restrict__ out) {
  const int64_t chunk = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (chunk >= n_chunks) return;
  const int64_t per_row = K / 8;
  const int64_t n = chunk / per_row, kc = chunk - n * per_row;
  out[((n >> 4) * (K / 32) + (kc >> 2)) * 64 + (kc & 3) * 16 + (n & 15)] = w[chunk];
}
}  // namespace

hipError_t launch_pack_tile_order(const uint16_t* W, int N, int K, uint16_t* out,
                                  hipStream_t st) {
  if (N <= 0 || K <= 0 || N % 16 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  const int64_t n_chunks = (int64_t)N * K / 8;
  COCO_LAUNCH(pack_tile_order_kernel, dim3((unsigned)((n_chunks + 255) / 256)), dim3(256), 0, st,
              (const u32x4_t*)W, n_chunks, K, (u32x4_t*)out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// fp32 GEMM for the tiny fp32 configuration: 16x16 LDS tiles, k ascending.
// ----------------------------------------------------------------------------
namespace {
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ W,
                                                       float* __restrict__ out, int M, int N,
                                                       int K) {
  __shared__ float as[16][17], ws[16][17];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m = blockIdx.y * 16 + ty, n = blockIdx.x * 16 + tx;
  float acc = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    const int am = blockIdx.y * 16 + ty, ak = k0 + tx;
    as[ty][tx] = (am < M && ak < K) ? A[(int64_t)am * K + ak] : 0.f;
    const int wn = blockIdx.x * 16 + ty;
    ws[ty][tx] = (wn < N && ak < K) ? W[(int64_t)wn * K + ak] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) acc = fmaf(as[ty][kk], ws[tx][kk], acc);
    __syncthreads();
  }
  if (m < M && n < N) out[(int64_t)m * N + n] = acc;
}
}  // namespace

hipError_t launch_gemm_f32(const float* A, const float* W, float* part, int M, int N, int K,
                           hipStream_t st) {
  if (M <= 0) return hipSuccess;
  COCO_LAUNCH(gemm_f32_kernel, dim3((N + 15) / 16, (M + 15) / 16), dim3(256), 0, st, A,
                     W, part, M, N, K);
  return hipGetLastError();
}

}  // namespace coco
