// Weight-streaming GEMM for decode-sized row counts (bf16 MFMA, fp32 out).
//
//   part[s][m][n] = sum over k in K-slice s of A[m][k] * W[n][k]
//
// A: [M][K] activations, W: [N][K] weights (nn.Linear layout), both bf16.
// Decode is bound by reading W once from HBM, so the kernel is built around
// that stream:
//   * a workgroup owns 64 output columns and one K-slice; each of its four
//     waves streams the 16 weight rows of its columns straight into VGPRs
//     (16-byte loads, 64 contiguous bytes per row per instruction), keeping
//     PF stages of 128 k in flight;
//   * the activation tile [rows][128 k] of the stage is shared by the four
//     waves through LDS (double-buffered, rows padded by 16 bytes);
//   * each 16x16 output tile is accumulated with v_mfma_f32_16x16x32_bf16 in
//     ascending k.
// The K-slicing S (split-K) is a function of (N, K) only and every output
// element is summed in the same k order for any M, so a row's result does
// not depend on the other rows in the call (batch invariance). Partials of
// the S slices are added in slice order by the consumer epilogue.
#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kBN = 64;        // output columns per workgroup
constexpr int kBK = 128;       // k per pipeline stage
constexpr int kPad = 8;        // bf16 elements of LDS row padding
constexpr int kLdsRow = kBK + kPad;
constexpr int kThreads = 256;  // 4 waves
constexpr int kPF = 3;         // weight stages in flight per wave

template <int MT>
__global__ __launch_bounds__(kThreads) void gemm_skinny_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, float* __restrict__ part, int M,
    int N, int K, int k_slice) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][MT * 16][kLdsRow];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int c16 = lane & 15, j4 = lane >> 4;
  const int n_col = blockIdx.x * kBN + wv * 16 + c16;  // this lane's weight row
  const int k_begin = blockIdx.y * k_slice;
  const int stages = k_slice / kBK;
  float* out = part + (int64_t)blockIdx.y * M * N;

  const bf16_t* wrow = W + (int64_t)n_col * K + k_begin + j4 * 8;

  for (int m0 = 0; m0 < M; m0 += MT * 16) {
    f32x4_t acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Weight ring: kPF stages x 4 k-steps of 8 bf16 per lane.
    u32x4_t wreg[kPF][4];
#pragma unroll
    for (int u = 0; u < kPF; ++u)
      if (u < stages) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          wreg[u][t] = *(const u32x4_t*)(wrow + u * kBK + t * 32);
      }

    // Activation staging: MT 16-byte chunks per thread and stage.
    u32x4_t areg[MT];
    auto load_a = [&](int st) {
#pragma unroll
      for (int v = 0; v < MT; ++v) {
        const int q = tid + v * kThreads;
        const int row = q >> 4, ch = q & 15;
        const int m = m0 + row;
        if (m < M)
          areg[v] = *(const u32x4_t*)(A + (int64_t)m * K + k_begin + st * kBK + ch * 8);
        else
          areg[v] = u32x4_t{0u, 0u, 0u, 0u};
      }
    };
    auto store_a = [&](int buf) {
#pragma unroll
      for (int v = 0; v < MT; ++v) {
        const int q = tid + v * kThreads;
        const int row = q >> 4, ch = q & 15;
        *(u32x4_t*)(&lds[buf][row][ch * 8]) = areg[v];
      }
    };

    load_a(0);
    store_a(0);
    __syncthreads();

    for (int st0 = 0; st0 < stages; st0 += kPF) {
#pragma unroll
      for (int u = 0; u < kPF; ++u) {
        const int st = st0 + u;
        if (st < stages) {
          const int buf = st & 1;
          if (st + 1 < stages) load_a(st + 1);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const bf16x8_t b = __builtin_bit_cast(bf16x8_t, wreg[u][t]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              const bf16x8_t a =
                  __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(&lds[buf][mt * 16 + c16][t * 32 + j4 * 8]));
              acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[mt], 0, 0, 0);
            }
          }
          if (st + kPF < stages) {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              wreg[u][t] = *(const u32x4_t*)(wrow + (st + kPF) * kBK + t * 32);
          }
          if (st + 1 < stages) store_a(buf ^ 1);
          __syncthreads();
        }
      }
    }

    // D layout: lane holds rows 4*j4 + r of column c16 of each 16x16 tile.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + mt * 16 + j4 * 4 + r;
        if (m < M) out[(int64_t)m * N + n_col] = acc[mt][r];
      }
    }
  }
}

}  // namespace

int skinny_splits(int N, int K) {
  const int cols = N / kBN;
  int S = 1;
  while (cols * S < 384 && S < 16) S *= 2;
  while (S > 1 && K % (S * kBK) != 0) S >>= 1;
  return S;
}

hipError_t launch_gemm_skinny_bf16(const uint16_t* A, const uint16_t* W, float* part, int M,
                                   int N, int K, int S, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (N % kBN != 0 || K % (S * kBK) != 0) return hipErrorInvalidValue;
  const dim3 grid(N / kBN, S);
  if (M <= 64)
    hipLaunchKernelGGL(gemm_skinny_kernel<4>, grid, dim3(kThreads), 0, st, A, W, part, M, N, K,
                       K / S);
  else
    hipLaunchKernelGGL(gemm_skinny_kernel<8>, grid, dim3(kThreads), 0, st, A, W, part, M, N, K,
                       K / S);
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
  hipLaunchKernelGGL(gemm_f32_kernel, dim3((N + 15) / 16, (M + 15) / 16), dim3(256), 0, st, A,
                     W, part, M, N, K);
  return hipGetLastError();
}

}  // namespace coco
