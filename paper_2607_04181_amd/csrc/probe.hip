// Peak probes for benchmarks: what this GPU sustains on a plain HBM read
// stream and on a loop of bf16 MFMAs, so that measured kernels can be quoted
// against measured ceilings as well as against the published ones. Neither
// kernel is on the layer's path.
#include "../../include/coco.h"
#include "common.h"
#include "kernels.h"

namespace coco {
namespace {

constexpr int kProbeThreads = 256;

// Every thread reads 16-byte vectors with a grid-wide stride (consecutive
// lanes on consecutive vectors), U independent loads in flight per
// iteration (plain or non-temporal), and folds them into one word; each
// block writes one word so the loads cannot be dropped.
template <int U, bool NT>
__global__ __launch_bounds__(kProbeThreads) void probe_read_kernel(const u32x4_t* __restrict__ buf,
                                                                   int64_t n_vec,
                                                                   uint32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
  uint32_t acc = 0;
  int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
  for (; i + (U - 1) * stride < n_vec; i += U * stride) {
    u32x4_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = NT ? __builtin_nontemporal_load(buf + i + u * stride) : buf[i + u * stride];
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n_vec; i += stride) {
    const u32x4_t a = buf[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ uint32_t red[kProbeThreads / kWave];
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kProbeThreads / kWave; ++w) t ^= red[w];
    out[blockIdx.x] = t;
  }
}

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// C independent chains of v_mfma_f32_32x32x16_bf16 per wave (32*32*16*2
// flops each), operands held in registers; lane 0 of each wave writes one
// element of every chain so the chains cannot be dropped. RANDOM: eight
// operand sets per lane of random bf16 values (hashed from the lane and the
// set), instruction k of a round taking set (c + k) % 8 for A and
// (3c + k) % 8 for B; otherwise one set of small constants.
__device__ __forceinline__ uint32_t probe_hash(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

template <int kMfmaChains, bool RANDOM>
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_kernel(int64_t iters,
                                                                   float* __restrict__ out) {
  const int lane = threadIdx.x & (kWave - 1);
  constexpr int kSets = RANDOM ? 8 : 1;
  bf16x8_t a[kSets], b[kSets];
#pragma unroll
  for (int s = 0; s < kSets; ++s) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (RANDOM) {
        // Sign and 7 mantissa bits random, exponent that of [0.5, 2).
        const uint32_t h = probe_hash(((blockIdx.x * kProbeThreads + threadIdx.x) * 8 + s) * 8 + e);
        a[s][e] = __builtin_bit_cast(__bf16, (uint16_t)((h & 0x807Fu) | ((h & 0x100u) ? 0x3F80u : 0x3F00u)));
        b[s][e] = __builtin_bit_cast(__bf16, (uint16_t)(((h >> 16) & 0x807Fu) | ((h & 0x200u) ? 0x3F80u : 0x3F00u)));
      } else {
        a[s][e] = (__bf16)(0.001f * (float)(lane + e));
        b[s][e] = (__bf16)(0.002f * (float)(lane - e));
      }
    }
  }
  f32x16_t acc[kMfmaChains];
#pragma unroll
  for (int c = 0; c < kMfmaChains; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  for (int64_t it = 0; it < iters; it += 8) {
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int c = 0; c < kMfmaChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(c + k) % kSets], b[(3 * c + k) % kSets],
                                                         acc[c], 0, 0, 0);
  }
  if (lane == 0) {
    float t = 0.f;
#pragma unroll
    for (int c = 0; c < kMfmaChains; ++c) t += acc[c][0];
    out[(int64_t)blockIdx.x * (kProbeThreads / kWave) + threadIdx.x / kWave] = t;
  }
}

}  // namespace
}  // namespace coco

using namespace coco;

extern "C" {

int coco_probe_read(const void* buf, int64_t bytes, void* out, int32_t blocks, int32_t variant,
                    coco_stream_t stream) {
  if (!buf || !out || bytes < 16 || bytes % 16 || (uintptr_t)buf % 16 || blocks < 1)
    return COCO_EINVAL;
  const hipStream_t st = (hipStream_t)stream;
  const u32x4_t* b = (const u32x4_t*)buf;
  const int64_t n = bytes / 16;
  switch (variant) {
    case 0: COCO_LAUNCH((probe_read_kernel<4, false>), dim3(blocks), dim3(kProbeThreads), 0, st, b, n, (uint32_t*)out); break;
    case 1: COCO_LAUNCH((probe_read_kernel<8, false>), dim3(blocks), dim3(kProbeThreads), 0, st, b, n, (uint32_t*)out); break;
    case 2: COCO_LAUNCH((probe_read_kernel<8, true>), dim3(blocks), dim3(kProbeThreads), 0, st, b, n, (uint32_t*)out); break;
    default: return COCO_EINVAL;
  }
  return hipGetLastError() == hipSuccess ? COCO_OK : COCO_EHIP;
}

int coco_probe_mfma_bf16(int64_t iters, void* out, int32_t blocks, int32_t chains,
                         int32_t operands, double* flops, coco_stream_t stream) {
  if (!out || !flops || iters < 8 || iters % 8 || blocks < 1 || (chains != 4 && chains != 8) ||
      (operands != 0 && operands != 1))
    return COCO_EINVAL;
  *flops = 2.0 * 32 * 32 * 16 * chains * (double)iters * blocks * (kProbeThreads / kWave);
  const hipStream_t st = (hipStream_t)stream;
  const dim3 g(blocks), b(kProbeThreads);
  float* o = (float*)out;
  if (chains == 4 && operands == 0)
    COCO_LAUNCH((probe_mfma_kernel<4, false>), g, b, 0, st, iters, o);
  else if (chains == 4)
    COCO_LAUNCH((probe_mfma_kernel<4, true>), g, b, 0, st, iters, o);
  else if (operands == 0)
    COCO_LAUNCH((probe_mfma_kernel<8, false>), g, b, 0, st, iters, o);
  else
    COCO_LAUNCH((probe_mfma_kernel<8, true>), g, b, 0, st, iters, o);
  return hipGetLastError() == hipSuccess ? COCO_OK : COCO_EHIP;
}

}  // extern "C"
