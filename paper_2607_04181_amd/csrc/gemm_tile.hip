// Large-tile GEMM for prefill-sized row counts (bf16 MFMA, fp32 out).
//
//   C[m][n] = sum_k A[m][k] * W[n][k]      A: [M][K], W: [N][K], both bf16
//
// Prefill is bound by MFMA throughput, so the kernel is built for reuse:
//   * a 512-thread workgroup computes a 256 x 256 tile; each of its eight
//     waves owns a 128 x 64 sub-tile as 4 x 2 v_mfma_f32_32x32x16_bf16
//     accumulators, two waves per SIMD so that one wave's MFMAs issue while
//     the other waits on LDS or the barrier (measured 20-25% faster than four
//     waves of 128 x 128 on the large shapes, with identical bits);
//   * 64-deep K stages of A and W tiles are staged through LDS (2 x 64 KB,
//     double-buffered) with 16-byte chunks XOR-swizzled by row pair, so the
//     rows a wave reads per MFMA operand fall in distinct banks; the next
//     stage's global loads are in flight while the current stage is
//     multiplied;
//   * workgroups are remapped so that the tiles sharing a W column slab run
//     on the same XCD (blockIdx % 8) back to back and hit its L2;
//   * narrow outputs with a long K are split into K-slices (tile_splits, a
//     function of (N, K) only) so the grid covers the CUs;
//   * for the gate/up projection a variant pairs gate and up columns inside
//     each wave and writes silu(gate) * up directly in bf16.
// Every output element is summed over k in ascending 16-steps within its
// slice, independent of M and of the tile it falls in, so request-aligned
// prefill splits give identical bits.
#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kTM = 256, kTN = 256, kTK = 64;
constexpr int kTThreads = 512;  // 8 waves, two per SIMD
constexpr int kXCDs = 8;

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// LDS element offset of 16-byte chunk c (0..7) of row r in a [256][64] tile.
// A 16-lane group of a 16-byte-per-lane LDS access covers 256 bytes (all 64
// banks) = two 128-byte rows; XOR-ing the chunk with (r / 2) % 8 gives the
// 16 consecutive rows a fragment read touches, and the two rows a store
// group writes, 16 distinct 4-bank slots.
__device__ __forceinline__ int swz(int r, int c) { return r * kTK + ((c ^ ((r >> 1) & 7)) << 3); }

// FUSE: W is the [2F][K] gate/up matrix; each 32-column half of a wave's
// 64 columns holds gate rows and the other the matching up rows, so each lane
// owns both factors of its outputs and the epilogue writes h = silu(gate) *
// up in bf16 to the [M][F] buffer `H` (N = 2F, one K-slice). Otherwise C is
// the fp32 partial.
template <bool FUSE>
__global__ __launch_bounds__(kTThreads) void gemm_tile_kernel(const bf16_t* __restrict__ A,
                                                                 const bf16_t* __restrict__ W,
                                                                 float* __restrict__ C,
                                                                 bf16_t* __restrict__ H, int M,
                                                                 int N, int K, int k_slice) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][2][kTM * kTK];  // [buf][A|W]

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
  const int lane = tid & 63, wv = tid >> 6;
  const int wm = wv & 1, wn = wv >> 1;  // 128-row half, 64-column quarter
  const int l32 = lane & 31, hi = lane >> 5;

  // Fused tile of 128 outputs o0 .. o0+127: tile rows 64w + 32j + i hold gate
  // row o0 + 32w + i for j = 0 and up row F + o0 + 32w + i for j = 1.
  const int F = N / 2, o0 = n0 / 2;
  auto w_row = [&](int r) {
    if (!FUSE) return min(n0 + r, N - 1);
    const int w = r >> 6, j = (r >> 5) & 1, i = r & 31;
    return (j ? F : 0) + o0 + 32 * w + i;
  };

  u32x4_t ra[4], rw[4];
  const int stages = k_slice / kTK;
  auto load = [&](int st) {
    const int k0 = kb + min(st, stages - 1) * kTK;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int q = tid + v * kTThreads;
      const int r = q >> 3, c = q & 7;
      const int m = min(m0 + r, M - 1), n = w_row(r);
      ra[v] = *(const u32x4_t*)(A + (int64_t)m * K + k0 + c * 8);
      rw[v] = *(const u32x4_t*)(W + (int64_t)n * K + k0 + c * 8);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int q = tid + v * kTThreads;
      const int r = q >> 3, c = q & 7;
      *(u32x4_t*)(&lds[buf][0][swz(r, c)]) = ra[v];
      *(u32x4_t*)(&lds[buf][1][swz(r, c)]) = rw[v];
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
          bf16x8_t, *(const u32x4_t*)(&la[swz(wm * 128 + i * 32 + l32, c)]));
#pragma unroll
    for (int j = 0; j < 2; ++j)
      w[j] = __builtin_bit_cast(
          bf16x8_t, *(const u32x4_t*)(&lw[swz(wn * 64 + j * 32 + l32, c)]));
  };

  load(0);
  store(0);
  __syncthreads();
  load(1);

  for (int st = 0; st < stages; ++st) {
    const int buf = st & 1;
    const bf16_t* la = lds[buf][0];
    const bf16_t* lw = lds[buf][1];
    bf16x8_t a[2][4], w[2][2];
    read_frags(la, lw, 0, a[0], w[0]);
#pragma unroll
    for (int kk = 0; kk < kTK / 16; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < kTK / 16) read_frags(la, lw, kk + 1, a[cur ^ 1], w[cur ^ 1]);
      if (kk == 1) store(buf ^ 1);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[cur][i], w[cur][j], acc[i][j], 0, 0, 0);
      if (kk == 1) load(st + 2);
      if (kk + 1 < kTK / 16) {
        for (int g = 0; g < 6; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      if (kk == 1) {
        for (int g = 0; g < 8; ++g) {
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
        }
      }
    }
    __syncthreads();
  }

  if (FUSE) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = o0 + 32 * wn + l32;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + wm * 128 + i * 32 + 8 * jj + 4 * hi + r;
          const float g = acc[i][0][4 * jj + r], u = acc[i][1][4 * jj + r];
          if (m < M) H[(int64_t)m * F + o] = (bf16_t)f32_to_bf16(g / (1.0f + expf(-g)) * u);
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
  while (S > 1 && (K / kTK) % S != 0) --S;
  return S;  // 1..4: the split counts the epilogues are built for
}

hipError_t launch_gemm_tile_bf16(const uint16_t* A, const uint16_t* W, float* C, int M, int N,
                                 int K, int S, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (S < 1 || K % (kTK * S) != 0) return hipErrorInvalidValue;
  const int tiles = ((M + kTM - 1) / kTM) * ((N + kTN - 1) / kTN);
  hipLaunchKernelGGL(gemm_tile_kernel<false>, dim3(tiles, S), dim3(kTThreads), 0, st, A, W, C,
                     nullptr, M, N, K, K / S);
  return hipGetLastError();
}

hipError_t launch_gemm_tile_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                        uint16_t* H, int M, int F, int K, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (F % (kTN / 2) != 0 || K % kTK != 0 || tile_splits(2 * F, K) != 1)
    return hipErrorInvalidValue;
  const int tiles = ((M + kTM - 1) / kTM) * (2 * F / kTN);
  hipLaunchKernelGGL(gemm_tile_kernel<true>, dim3(tiles, 1), dim3(kTThreads), 0, st, A,
                     W_gate_up, nullptr, H, M, 2 * F, K, K);
  return hipGetLastError();
}

}  // namespace coco
