// Row-wise kernels of the decoder layer: gather + RMSNorm, the epilogues that
// reduce split-K partials of the projections (RoPE + cache append, residual +
// RMSNorm, SwiGLU, residual + scatter) and the paged key/value append.
//
// Every kernel handles one call row per workgroup (or one element per thread)
// with a reduction order fixed by the block size alone, so a row's result
// never depends on which other rows share the call.
#include "common.h"
#include "kernels.h"

namespace coco {

constexpr int kRowThreads = 256;

// ----------------------------------------------------------------------------
// Segment-boundary gather of the sub-batch rows, fused with the first RMSNorm.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void gather_rmsnorm_kernel(
    const T* __restrict__ src, const int32_t* __restrict__ row_idx, int d,
    const T* __restrict__ gamma, float eps, T* __restrict__ x_out, T* __restrict__ h_out) {
  __shared__ float red[kRowThreads / kWave];
  const int i = blockIdx.x;
  const int64_t r = row_idx ? (int64_t)row_idx[i] : (int64_t)i;
  const T* x = src + r * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    const float v = Elem<T>::load(x + c);
    ss += v * v;
    if (x_out) x_out[(int64_t)i * d + c] = x[c];
  }
  ss = block_sum<kRowThreads>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += kRowThreads)
    Elem<T>::store(h_out + (int64_t)i * d + c,
                   Elem<T>::load(x + c) * inv * Elem<T>::load(gamma + c));
}

template <typename T>
hipError_t launch_gather_rmsnorm(const T* src, const int32_t* row_idx, int M, int d,
                                 const T* gamma, float eps, T* x_out, T* h_out,
                                 hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rmsnorm_kernel<T>, dim3(M), dim3(kRowThreads), 0, st, src,
                     row_idx, d, gamma, eps, x_out, h_out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// QKV epilogue: reduce the split-K partials, rotate query and key heads to the
// row's absolute position (rotate-half RoPE, angles in fp64), store queries,
// append the rotated key and the value to the sequence's cache slot.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void qkv_epilogue_kernel(
    const float* __restrict__ part, int S, int M, int Hq, int Hkv, int hd,
    const int32_t* __restrict__ positions, const int32_t* __restrict__ seq_starts, int n_seqs,
    const int32_t* __restrict__ block_table, int max_blocks, const double* __restrict__ inv_freq,
    T* __restrict__ q_out, T* __restrict__ k_cache, T* __restrict__ v_cache) {
  __shared__ float cs[2][128];
  const int i = blockIdx.x;
  const int half = hd >> 1;
  const int N = (Hq + 2 * Hkv) * hd;
  const int pos = positions[i];
  for (int j = threadIdx.x; j < half; j += kRowThreads) {
    double sn, cn;
    sincos((double)pos * inv_freq[j], &sn, &cn);
    cs[0][j] = (float)cn;
    cs[1][j] = (float)sn;
  }
  __syncthreads();
  const int seq = row_to_seq(seq_starts, n_seqs, i);
  const int64_t blk = block_table[(int64_t)seq * max_blocks + pos / kBlockTokens];
  const int slot = pos % kBlockTokens;
  const float* p = part + (int64_t)i * N;
  const int64_t pstride = (int64_t)M * N;
  auto val = [&](int n) {
    float a = 0.f;
    for (int s = 0; s < S; ++s) a += p[s * pstride + n];
    return a;
  };
  // Query and key heads: one thread per rotation pair (head, j).
  const int pairs = (Hq + Hkv) * half;
  for (int e = threadIdx.x; e < pairs; e += kRowThreads) {
    const int h = e / half, j = e - h * half;
    const float lo = val(h * hd + j), hi = val(h * hd + j + half);
    const float c = cs[0][j], sn = cs[1][j];
    const float rlo = lo * c - hi * sn, rhi = hi * c + lo * sn;
    if (h < Hq) {
      T* q = q_out + (int64_t)i * Hq * hd + h * hd;
      Elem<T>::store(q + j, rlo);
      Elem<T>::store(q + j + half, rhi);
    } else {
      T* k = k_cache + ((blk * Hkv + (h - Hq)) * kBlockTokens + slot) * hd;
      Elem<T>::store(k + j, rlo);
      Elem<T>::store(k + j + half, rhi);
    }
  }
  // Value heads: [blk][kvh][dim][slot].
  for (int e = threadIdx.x; e < Hkv * hd; e += kRowThreads) {
    const int h = e / hd, dim = e - h * hd;
    Elem<T>::store(v_cache + ((blk * Hkv + h) * hd + dim) * kBlockTokens + slot,
                   val((Hq + Hkv) * hd + e));
  }
}

template <typename T>
hipError_t launch_qkv_epilogue(const float* part, int S, int M, int Hq, int Hkv, int hd,
                               const int32_t* positions, const int32_t* seq_starts,
                               int n_seqs, const int32_t* block_table, int max_blocks,
                               const double* inv_freq, T* q_out, T* k_cache, T* v_cache,
                               hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(qkv_epilogue_kernel<T>, dim3(M), dim3(kRowThreads), 0, st, part, S, M,
                     Hq, Hkv, hd, positions, seq_starts, n_seqs, block_table, max_blocks,
                     inv_freq, q_out, k_cache, v_cache);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// O-projection epilogue: residual add (kept in fp32) fused with RMSNorm_2.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void residual_rmsnorm_kernel(
    const float* __restrict__ part, int S, int M, int d, const T* __restrict__ x,
    const T* __restrict__ gamma, float eps, float* __restrict__ x1, T* __restrict__ h2) {
  __shared__ float red[kRowThreads / kWave];
  const int i = blockIdx.x;
  const int64_t pstride = (int64_t)M * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    float a = Elem<T>::load(x + (int64_t)i * d + c);
    float acc = 0.f;
    for (int s = 0; s < S; ++s) acc += part[s * pstride + (int64_t)i * d + c];
    a += acc;
    x1[(int64_t)i * d + c] = a;
    ss += a * a;
  }
  ss = block_sum<kRowThreads>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += kRowThreads)
    Elem<T>::store(h2 + (int64_t)i * d + c,
                   x1[(int64_t)i * d + c] * inv * Elem<T>::load(gamma + c));
}

template <typename T>
hipError_t launch_residual_rmsnorm(const float* part, int S, int M, int d, const T* x,
                                   const T* gamma, float eps, float* x1, T* h2,
                                   hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(residual_rmsnorm_kernel<T>, dim3(M), dim3(kRowThreads), 0, st, part, S,
                     M, d, x, gamma, eps, x1, h2);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// SwiGLU: u = silu(gate) * up from the reduced gate/up partials.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void swiglu_kernel(const float* __restrict__ part,
                                                             int S, int M, int F,
                                                             T* __restrict__ u) {
  const int i = blockIdx.y;
  const int j = blockIdx.x * kRowThreads + threadIdx.x;
  if (j >= F) return;
  const int64_t pstride = (int64_t)M * 2 * F;
  const float* p = part + (int64_t)i * 2 * F;
  float g = 0.f, up = 0.f;
  for (int s = 0; s < S; ++s) {
    g += p[s * pstride + j];
    up += p[s * pstride + F + j];
  }
  Elem<T>::store(u + (int64_t)i * F + j, g / (1.0f + expf(-g)) * up);
}

template <typename T>
hipError_t launch_swiglu(const float* part, int S, int M, int F, T* u, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_kernel<T>, dim3((F + kRowThreads - 1) / kRowThreads, M),
                     dim3(kRowThreads), 0, st, part, S, M, F, u);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Down-projection epilogue: y = x1 + sum of partials, rounded to the hidden
// dtype, scattered to the row's place in the full-batch buffer.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void residual_scatter_kernel(
    const float* __restrict__ part, int S, int M, int d, const float* __restrict__ x1,
    T* __restrict__ out, const int32_t* __restrict__ row_idx) {
  const int i = blockIdx.x;
  const int64_t r = row_idx ? (int64_t)row_idx[i] : (int64_t)i;
  const int64_t pstride = (int64_t)M * d;
  for (int c = threadIdx.x; c < d; c += kRowThreads) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s) acc += part[s * pstride + (int64_t)i * d + c];
    Elem<T>::store(out + r * d + c, x1[(int64_t)i * d + c] + acc);
  }
}

template <typename T>
hipError_t launch_residual_scatter(const float* part, int S, int M, int d, const float* x1,
                                   T* out, const int32_t* row_idx, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(residual_scatter_kernel<T>, dim3(M), dim3(kRowThreads), 0, st, part, S,
                     M, d, x1, out, row_idx);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Paged key/value append (bit copy).
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kRowThreads) void kv_append_kernel(
    const T* __restrict__ k, const T* __restrict__ v, const int32_t* __restrict__ seq_idx,
    const int32_t* __restrict__ positions, int Hkv, int hd,
    const int32_t* __restrict__ block_table, int max_blocks, T* __restrict__ k_cache,
    T* __restrict__ v_cache) {
  const int t = blockIdx.x;
  const int pos = positions[t];
  const int64_t blk = block_table[(int64_t)seq_idx[t] * max_blocks + pos / kBlockTokens];
  const int slot = pos % kBlockTokens;
  const int64_t src = (int64_t)t * Hkv * hd;
  for (int e = threadIdx.x; e < Hkv * hd; e += kRowThreads) {
    const int h = e / hd, dim = e - h * hd;
    k_cache[((blk * Hkv + h) * kBlockTokens + slot) * hd + dim] = k[src + e];
    v_cache[((blk * Hkv + h) * hd + dim) * kBlockTokens + slot] = v[src + e];
  }
}

template <typename T>
hipError_t launch_kv_append(const T* k, const T* v, const int32_t* seq_idx,
                            const int32_t* positions, int n, int Hkv, int hd,
                            const int32_t* block_table, int max_blocks, T* k_cache,
                            T* v_cache, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(kv_append_kernel<T>, dim3(n), dim3(kRowThreads), 0, st, k, v, seq_idx,
                     positions, Hkv, hd, block_table, max_blocks, k_cache, v_cache);
  return hipGetLastError();
}

#define COCO_INSTANTIATE(T)                                                                   \
  template hipError_t launch_gather_rmsnorm<T>(const T*, const int32_t*, int, int, const T*, \
                                               float, T*, T*, hipStream_t);                  \
  template hipError_t launch_qkv_epilogue<T>(const float*, int, int, int, int, int,          \
                                             const int32_t*, const int32_t*, int,            \
                                             const int32_t*, int, const double*, T*, T*, T*, \
                                             hipStream_t);                                   \
  template hipError_t launch_residual_rmsnorm<T>(const float*, int, int, int, const T*,      \
                                                 const T*, float, float*, T*, hipStream_t);  \
  template hipError_t launch_swiglu<T>(const float*, int, int, int, T*, hipStream_t);        \
  template hipError_t launch_residual_scatter<T>(const float*, int, int, int, const float*,  \
                                                 T*, const int32_t*, hipStream_t);           \
  template hipError_t launch_kv_append<T>(const T*, const T*, const int32_t*, const int32_t*, \
                                          int, int, int, const int32_t*, int, T*, T*,        \
                                          hipStream_t);

COCO_INSTANTIATE(bf16_t)
COCO_INSTANTIATE(float)

}  // namespace coco
