// Row-wise kernels of the decoder layer: gather + RMSNorm, the epilogues that
// reduce split-K partials of the projections (RoPE + cache append, residual +
// RMSNorm, SwiGLU, residual + scatter) and the paged key/value append.
//
// These kernels move little data (a few MB per step) and are bound by memory
// latency, so they are written for memory-level parallelism: the split count
// S is a template parameter (all S partial loads of a column are issued back
// to back), fp32 partials are read as 16-byte vectors, and grids cover
// (row, column chunk) rather than one workgroup per row where no row-wide
// reduction is needed. Every reduction order is fixed by the block shape and
// S alone, so a row's result never depends on the other rows of the call.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int kRowThreads = 256;
constexpr int kNormThreads = 1024;

// Sum of S fp32 partials of 4 consecutive columns, in split order.
template <int S>
__device__ __forceinline__ f32x4_t sum_parts4(const float* __restrict__ p, int64_t stride) {
  f32x4_t v[S];
#pragma unroll
  for (int s = 0; s < S; ++s) v[s] = *(const f32x4_t*)(p + s * stride);
  f32x4_t a = v[0];
#pragma unroll
  for (int s = 1; s < S; ++s) a += v[s];
  return a;
}

template <int S>
__device__ __forceinline__ float sum_parts1(const float* __restrict__ p, int64_t stride) {
  float v[S];
#pragma unroll
  for (int s = 0; s < S; ++s) v[s] = p[s * stride];
  float a = v[0];
#pragma unroll
  for (int s = 1; s < S; ++s) a += v[s];
  return a;
}

__device__ __forceinline__ void unpack_bf16x8(u32x4_t u, float* f) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(u[i] << 16);
    f[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
  }
}

__device__ __forceinline__ u32x4_t pack_bf16x8(const float* f) {
  return u32x4_t{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                 pack_bf16x2(f[6], f[7])};
}

}  // namespace

// ----------------------------------------------------------------------------
// Segment-boundary gather of the sub-batch rows, fused with the first RMSNorm.
// ----------------------------------------------------------------------------
// Prefill row slots: row_info[i] = (position clamped to the RoPE table,
// cache block of the position), for the QKV projection's fused epilogue.
__device__ __forceinline__ void write_row_slot(const RowSlotArgs& rs, int i) {
  const int pos = rs.positions[i];
  int lo = 0, hi = rs.n_seqs - 1;  // the s with seq_starts[s] <= i < seq_starts[s + 1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (rs.seq_starts[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int blk = rs.block_table[(int64_t)lo * rs.max_blocks +
                                 min(max(pos, 0) / kBlockTokens, rs.max_blocks - 1)];
  rs.row_info[2 * i] = min(max(pos, 0), rs.rope_rows - 1);
  rs.row_info[2 * i + 1] = blk;
}

template <typename T>
__global__ __launch_bounds__(kRowThreads) void gather_rmsnorm_kernel(
    const T* __restrict__ src, const int32_t* __restrict__ row_idx, int d,
    const T* __restrict__ gamma, float eps, T* __restrict__ x_out, T* __restrict__ h_out,
    bool tiled, RowSlotArgs rs) {
  (void)tiled;  // bf16 only
  __shared__ float red[kRowThreads / kWave];
  const int i = blockIdx.x;
  if (rs.row_info != nullptr && threadIdx.x == 0) write_row_slot(rs, i);
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

// bf16 rows, d % 8 == 0: 16-byte vectors, row held in registers.
//   * Row of a workgroup: with `tiled`, consecutive rows run on one XCD
//     (blockIdx % 8 is the XCD), so the 16 rows that share each 1 KB
//     tile-order block fill it in that XCD's L2 and it leaves as whole lines;
//   * the row slot (prefill QKV epilogue) is found by the first wave with
//     scalar loads through the constant address space, which wait on their
//     own counter, so the chain of dependent loads overlaps the row's vector
//     loads instead of following them.
typedef __attribute__((address_space(4))) const int32_t* cint_ptr;

__device__ __forceinline__ void write_row_slot_uniform(const RowSlotArgs& rs, int i) {
  const cint_ptr positions = (cint_ptr)rs.positions;
  const cint_ptr seq_starts = (cint_ptr)rs.seq_starts;
  const cint_ptr block_table = (cint_ptr)rs.block_table;
  const int pos = positions[i];
  int lo = 0, hi = rs.n_seqs - 1;  // the s with seq_starts[s] <= i < seq_starts[s + 1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seq_starts[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int blk =
      block_table[(int64_t)lo * rs.max_blocks + min(max(pos, 0) / kBlockTokens, rs.max_blocks - 1)];
  if (threadIdx.x == 0) {
    rs.row_info[2 * i] = min(max(pos, 0), rs.rope_rows - 1);
    rs.row_info[2 * i + 1] = blk;
  }
}

// NV: 16-byte vectors per thread (the row's d / 8 vectors over the block),
// all loaded up front without a branch (past the row: its last vector again).
template <int NV>
__global__ __launch_bounds__(kRowThreads) void gather_rmsnorm_bf16_kernel(
    const bf16_t* __restrict__ src, const int32_t* __restrict__ row_idx, int d,
    const bf16_t* __restrict__ gamma, float eps, bf16_t* __restrict__ x_out,
    bf16_t* __restrict__ h_out, bool tiled, RowSlotArgs rs) {
  __shared__ float red[kRowThreads / kWave];
  constexpr int kXCDs = 8;
  const int nb = gridDim.x, b = blockIdx.x;
  const int full = (nb / kXCDs) * kXCDs;
  const int i = tiled && b < full ? (b % kXCDs) * (nb / kXCDs) + b / kXCDs : b;
  const int64_t r = row_idx ? (int64_t)row_idx[i] : (int64_t)i;
  const int nv = d / 8;
  const u32x4_t* x = (const u32x4_t*)(src + r * d);
  const u32x4_t* g = (const u32x4_t*)gamma;
  // The gains are loaded together with the row: one memory round trip.
  u32x4_t xv[NV], gv[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int v = min((int)threadIdx.x + u * kRowThreads, nv - 1);
    xv[u] = x[v];
    gv[u] = g[v];
  }
  if (rs.row_info != nullptr && threadIdx.x < kWave) write_row_slot_uniform(rs, i);
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int v = threadIdx.x + u * kRowThreads;
    if (v < nv) {
      float f[8];
      unpack_bf16x8(xv[u], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += f[e] * f[e];
      if (x_out) ((u32x4_t*)(x_out + (int64_t)i * d))[v] = xv[u];
    }
  }
  ss = block_sum<kRowThreads>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int v = threadIdx.x + u * kRowThreads;
    if (v < nv) {
      float f[8], gf[8];
      unpack_bf16x8(xv[u], f);
      unpack_bf16x8(gv[u], gf);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = f[e] * inv * gf[e];
      *(u32x4_t*)(h_out + (tiled ? tile_off(i, 8 * v, d) : (int64_t)i * d + 8 * v)) =
          pack_bf16x8(f);
    }
  }
}

template <typename T>
hipError_t launch_gather_rmsnorm(const T* src, const int32_t* row_idx, int M, int d,
                                 const T* gamma, float eps, T* x_out, T* h_out, bool tiled,
                                 const RowSlotArgs& rs, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (rs.row_info != nullptr && (rs.n_seqs < 1 || rs.max_blocks < 1 || rs.rope_rows < 1))
    return hipErrorInvalidValue;
  if (tiled && (!std::is_same<T, bf16_t>::value || d % 32 != 0)) return hipErrorInvalidValue;
  if constexpr (std::is_same<T, bf16_t>::value) {
    if (d % 8 != 0 || d > 8 * kRowThreads * 8) return hipErrorInvalidValue;
    const int nvt = (d / 8 + kRowThreads - 1) / kRowThreads;  // vectors per thread, 1..8
    switch (nvt) {
#define COCO_GN_CASE(n)                                                                       \
  case n:                                                                                     \
    COCO_LAUNCH(gather_rmsnorm_bf16_kernel<n>, dim3(M), dim3(kRowThreads), 0, st, src,         \
                row_idx, d, gamma, eps, x_out, h_out, tiled, rs);                             \
    break;
      COCO_GN_CASE(1) COCO_GN_CASE(2) COCO_GN_CASE(3) COCO_GN_CASE(4)
      COCO_GN_CASE(5) COCO_GN_CASE(6) COCO_GN_CASE(7) COCO_GN_CASE(8)
#undef COCO_GN_CASE
      default: return hipErrorInvalidValue;
    }
  } else {
    COCO_LAUNCH(gather_rmsnorm_kernel<T>, dim3(M), dim3(kRowThreads), 0, st, src, row_idx, d,
                gamma, eps, x_out, h_out, tiled, rs);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// RoPE table: rope[p][j] = (cos, sin)(p * inv_freq[j]), the angle and its
// cosine and sine evaluated in fp64 and rounded to fp32 exactly as the QKV
// epilogue below does, for every position p < n_pos the configuration
// admits. Built once at init for the prefill QKV projection's fused epilogue.
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void rope_table_kernel(const double* __restrict__ inv_freq,
                                                         int half, int n_pos,
                                                         float* __restrict__ rope) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)n_pos * half) return;
  const int p = (int)(e / half), j = (int)(e - (int64_t)p * half);
  double sn, cn;
  sincos((double)p * inv_freq[j], &sn, &cn);
  rope[2 * e] = (float)cn;
  rope[2 * e + 1] = (float)sn;
}

hipError_t launch_rope_table(const double* inv_freq, int half, int n_pos, float* rope,
                             hipStream_t st) {
  const int64_t n = (int64_t)n_pos * half;
  if (n <= 0) return hipErrorInvalidValue;
  COCO_LAUNCH(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     inv_freq, half, n_pos, rope);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// QKV epilogue: one wave per (row, head), kEpiHeads heads per workgroup.
// Reduce the split-K partials, rotate query and key heads to the row's
// absolute position (rotate-half RoPE; the angles' cos/sin in fp64, computed
// once per workgroup into LDS), store queries, append the rotated key and the
// value to the sequence's cache slot. The partial loads, which depend on
// nothing, are issued first; the cache slot lookup and the angles overlap
// them (a dependent load of the RoPE table measured slower here). In decode,
// one wave also writes the decode attention's work list.
// ----------------------------------------------------------------------------
constexpr int kEpiHeads = 8;

template <typename T, int S>
__global__ __launch_bounds__(kEpiHeads * kWave) void qkv_epilogue_kernel(
    const float* __restrict__ part, int M, int Hq, int Hkv, int hd,
    const int32_t* __restrict__ positions, const int32_t* __restrict__ seq_starts, int n_seqs,
    const int32_t* __restrict__ block_table, int max_blocks, const double* __restrict__ inv_freq,
    T* __restrict__ q_out, T* __restrict__ k_cache, T* __restrict__ v_cache,
    const int32_t* __restrict__ ctx_lens, int32_t* __restrict__ split_off, int max_splits,
    const float* __restrict__ ss, int d, float eps) {
  __shared__ float rot[2][128];  // cos, sin of the row's angles (hd / 2 <= 128)
  __shared__ int wl_rank[kDecodeSplit];  // work list: partial partitions per size, then ranks
  const int i = blockIdx.y, lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  const int nh = Hq + 2 * Hkv;
  const int h = blockIdx.x * kEpiHeads + wv;
  const bool live = h < nh;
  const int half = hd >> 1;
  const int N = nh * hd;
  const int64_t pstride = (int64_t)M * N;
  const float* p = part + (int64_t)i * N + (int64_t)(live ? h : 0) * hd;
  // Query/key heads: val[2t], val[2t+1] = dims j, j + hd/2 for j = lane + 64t;
  // value heads: val[t] = dim lane + 64t.
  float val[4] = {0.f, 0.f, 0.f, 0.f};
  if (live) {
    if (h < Hq + Hkv) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int j = lane + kWave * t;
        if (j < half) {
          val[2 * t] = sum_parts1<S>(p + j, pstride);
          val[2 * t + 1] = sum_parts1<S>(p + j + half, pstride);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int e = lane + kWave * t;
        if (e < hd) val[t] = sum_parts1<S>(p + e, pstride);
      }
    }
  }
  // RMSNorm_1 folded into the projection: this row's 1/rms from the
  // per-slice sums of squares, added in slice order.
  float rscale = 1.f;
  if (ss != nullptr) {
    const float t = sum_parts1<S>(ss + i, M);
    rscale = 1.0f / sqrtf(t / (float)d + eps);
  }
  const int pos = positions[i];
  int64_t blk = 0;
  int slot = 0;
  if (live && h >= Hq) {
    const int seq = row_to_seq(seq_starts, n_seqs, i);
    blk = block_table[(int64_t)seq * max_blocks + pos / kBlockTokens];
    slot = pos % kBlockTokens;
  }
  // The row's rotation angles in fp64, once for all the heads of the block.
  for (int j = threadIdx.x; j < half; j += kEpiHeads * kWave) {
    double sn, cn;
    sincos((double)pos * inv_freq[j], &sn, &cn);
    rot[0][j] = (float)cn;
    rot[1][j] = (float)sn;
  }
  __syncthreads();
  if (split_off != nullptr && blockIdx.x == 0 && i == 0 && wv == 0) {
    // Decode attention work list over the n = min(ctx_lens[s], positions[s]
    // + 1) keys row s attends, in 256-key partitions (at most max_splits; only
    // invalid lengths reach the cap). First every full partition: an
    // exclusive prefix sum of their counts in split_off[0 .. n_seqs]. Then
    // each sequence's last partition if it is partial, largest first: their
    // count in split_off[n_seqs + 1], the sequences in that order from
    // split_off[n_seqs + 2]. Dealt out in that order (snake-wise over the
    // workgroups), items of similar size meet at the end of the kernel.
    for (int r = lane; r < kDecodeSplit; r += kWave) wl_rank[r] = 0;
    int run = 0;
    if (lane == 0) split_off[0] = 0;
    for (int base = 0; base < n_seqs; base += kWave) {
      const int s = base + lane;
      const int n = s < n_seqs ? max(0, min(ctx_lens[s], positions[s] + 1)) : 0;
      const int nsp = (n + kDecodeSplit - 1) / kDecodeSplit;
      const int rem = (nsp <= max_splits) ? n % kDecodeSplit : 0;
      int v = min(nsp, max_splits) - (rem != 0);
      if (rem != 0) atomicAdd(&wl_rank[rem], 1);
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int t = __shfl_up(v, o, kWave);
        if (lane >= o) v += t;
      }
      if (s < n_seqs) split_off[s + 1] = run + v;
      run += __shfl(v, kWave - 1, kWave);
    }
    // Sizes largest first: wl_rank[r] becomes the number of partial
    // partitions longer than r keys (a suffix sum, four sizes per lane).
    static_assert(kDecodeSplit == 4 * kWave, "four partition sizes per lane");
    int c[4], tot = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[e] = wl_rank[kDecodeSplit - 1 - (lane * 4 + e)];
      tot += c[e];
    }
    int incl = tot;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int t = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += t;
    }
    int acc = incl - tot;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      wl_rank[kDecodeSplit - 1 - (lane * 4 + e)] = acc;
      acc += c[e];
    }
    if (lane == kWave - 1) split_off[n_seqs + 1] = incl;
    for (int base = 0; base < n_seqs; base += kWave) {
      const int s = base + lane;
      const int n = s < n_seqs ? max(0, min(ctx_lens[s], positions[s] + 1)) : 0;
      const int nsp = (n + kDecodeSplit - 1) / kDecodeSplit;
      const int rem = (nsp <= max_splits) ? n % kDecodeSplit : 0;
      if (rem != 0) split_off[n_seqs + 2 + atomicAdd(&wl_rank[rem], 1)] = s;
    }
  }
  if (!live) return;
#pragma unroll
  for (int t = 0; t < 4; ++t) val[t] *= rscale;
  if (h < Hq + Hkv) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int j = lane + kWave * t;
      if (j < half) {
        const float lo = val[2 * t], hi = val[2 * t + 1];
        const float c = rot[0][j], sn = rot[1][j];
        const float rlo = lo * c - hi * sn, rhi = hi * c + lo * sn;
        if (h < Hq) {
          T* dst = q_out + ((int64_t)i * Hq + h) * hd;
          Elem<T>::store(dst + j, rlo);
          Elem<T>::store(dst + j + half, rhi);
        } else {
          T* tile = k_cache + (blk * Hkv + (h - Hq)) * kBlockTokens * hd;
          Elem<T>::store(tile + k_tile_offset(slot, j), rlo);
          Elem<T>::store(tile + k_tile_offset(slot, j + half), rhi);
        }
      }
    }
  } else {
    T* tile = v_cache + (blk * Hkv + (h - Hq - Hkv)) * kBlockTokens * hd;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int e = lane + kWave * t;
      if (e < hd) Elem<T>::store(tile + v_tile_offset(slot, e), val[t]);
    }
  }
}

#define COCO_SWITCH_S(S, ...)                        \
  switch (S) {                                       \
    case 1: { constexpr int S_ = 1; __VA_ARGS__; } break;  \
    case 2: { constexpr int S_ = 2; __VA_ARGS__; } break;  \
    case 3: { constexpr int S_ = 3; __VA_ARGS__; } break;  \
    case 4: { constexpr int S_ = 4; __VA_ARGS__; } break;  \
    case 8: { constexpr int S_ = 8; __VA_ARGS__; } break;  \
    case 16: { constexpr int S_ = 16; __VA_ARGS__; } break; \
    default: return hipErrorInvalidValue;            \
  }

template <typename T>
hipError_t launch_qkv_epilogue(const float* part, int S, int M, int Hq, int Hkv, int hd,
                               const int32_t* positions, const int32_t* seq_starts,
                               int n_seqs, const int32_t* block_table, int max_blocks,
                               const double* inv_freq, T* q_out, T* k_cache, T* v_cache,
                               const int32_t* ctx_lens, int32_t* split_off, int max_splits,
                               const float* ss, int d, float eps, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (hd > 256 || hd % 2 != 0) return hipErrorInvalidValue;
  const dim3 grid((Hq + 2 * Hkv + kEpiHeads - 1) / kEpiHeads, M);
  COCO_SWITCH_S(S, COCO_LAUNCH((qkv_epilogue_kernel<T, S_>), grid,
                                      dim3(kEpiHeads * kWave), 0, st,
                                      part, M, Hq, Hkv, hd, positions, seq_starts, n_seqs,
                                      block_table, max_blocks, inv_freq, q_out, k_cache,
                                      v_cache, ctx_lens, split_off, max_splits, ss, d, eps));
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// O-projection epilogue: residual add (kept in fp32) fused with RMSNorm_2.
// One 1024-thread workgroup per row; every thread owns 4-column vectors.
// ----------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ f32x4_t load4(const T* p);
template <>
__device__ __forceinline__ f32x4_t load4<float>(const float* p) { return *(const f32x4_t*)p; }
template <>
__device__ __forceinline__ f32x4_t load4<bf16_t>(const bf16_t* p) {
  const u32x2_t u = *(const u32x2_t*)p;
  return f32x4_t{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                 __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u)};
}

template <typename T, int S>
__global__ __launch_bounds__(kNormThreads) void residual_rmsnorm_kernel(
    const float* __restrict__ part, int M, int d, const T* __restrict__ x,
    const int32_t* __restrict__ row_idx, const T* __restrict__ gamma, float eps,
    float* __restrict__ x1, T* __restrict__ h2, bool tiled) {
  __shared__ float red[kNormThreads / kWave];
  constexpr int kMaxVec = 4;  // d <= 16384
  const int i = blockIdx.x;
  const int64_t xr_row = row_idx ? (int64_t)row_idx[i] : (int64_t)i;
  const int64_t pstride = (int64_t)M * d;
  const int nv = d / 4;
  // Partials, residual and gains in one memory round trip.
  f32x4_t a[kMaxVec], xr[kMaxVec], g[kMaxVec];
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u) {
    const int v = threadIdx.x + u * kNormThreads;
    if (v < nv) {
      const int c = 4 * v;
      a[u] = sum_parts4<S>(part + (int64_t)i * d + c, pstride);
      xr[u] = load4<T>(x + xr_row * d + c);
      g[u] = load4<T>(gamma + c);
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u) {
    const int v = threadIdx.x + u * kNormThreads;
    if (v < nv) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[u][e] += xr[u][e];
        ss += a[u][e] * a[u][e];
      }
      *(f32x4_t*)(x1 + (int64_t)i * d + 4 * v) = a[u];
    }
  }
  ss = block_sum<kNormThreads>(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int u = 0; u < kMaxVec; ++u) {
    const int v = threadIdx.x + u * kNormThreads;
    if (v < nv) {
      const int c = 4 * v;
      // Four columns from a multiple of 4 stay contiguous in tile order.
      T* dst = h2 + (tiled ? tile_off(i, c, d) : (int64_t)i * d + c);
      store4(dst, a[u][0] * inv * g[u][0], a[u][1] * inv * g[u][1], a[u][2] * inv * g[u][2],
             a[u][3] * inv * g[u][3]);
    }
  }
}

template <typename T>
hipError_t launch_residual_rmsnorm(const float* part, int S, int M, int d, const T* x,
                                   const int32_t* row_idx, const T* gamma, float eps, float* x1,
                                   T* h2, bool tiled, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (d % 4 != 0 || d > 4 * 4 * kNormThreads) return hipErrorInvalidValue;
  if (tiled && (!std::is_same<T, bf16_t>::value || d % 32 != 0)) return hipErrorInvalidValue;
  COCO_SWITCH_S(S, COCO_LAUNCH((residual_rmsnorm_kernel<T, S_>), dim3(M),
                                      dim3(kNormThreads), 0, st, part, M, d, x, row_idx, gamma,
                                      eps, x1, h2, tiled));
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// SwiGLU: u = silu(gate) * up from the reduced gate/up partials; 4 columns
// per thread.
// ----------------------------------------------------------------------------
template <typename T, int S>
__global__ __launch_bounds__(kRowThreads) void swiglu_kernel(const float* __restrict__ part,
                                                             int M, int F, T* __restrict__ u,
                                                             bool tiled) {
  const int i = blockIdx.y;
  const int c = 4 * (blockIdx.x * kRowThreads + threadIdx.x);
  if (c >= F) return;
  const int64_t pstride = (int64_t)M * 2 * F;
  const float* p = part + (int64_t)i * 2 * F + c;
  const f32x4_t g = sum_parts4<S>(p, pstride);
  const f32x4_t up = sum_parts4<S>(p + F, pstride);
  T* dst = u + (tiled ? tile_off(i, c, F) : (int64_t)i * F + c);
  float r[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = silu_mul(g[e], up[e]);
  store4(dst, r[0], r[1], r[2], r[3]);
}

template <typename T>
hipError_t launch_swiglu(const float* part, int S, int M, int F, T* u, bool tiled,
                         hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (F % 4 != 0) return hipErrorInvalidValue;
  if (tiled && (!std::is_same<T, bf16_t>::value || F % 32 != 0)) return hipErrorInvalidValue;
  const dim3 grid((F / 4 + kRowThreads - 1) / kRowThreads, M);
  COCO_SWITCH_S(S, COCO_LAUNCH((swiglu_kernel<T, S_>), grid, dim3(kRowThreads), 0, st,
                                      part, M, F, u, tiled));
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Tile order back to row-major (inspection of the prefill activations): one
// thread per 8-column chunk, 16-byte copies.
// ----------------------------------------------------------------------------
namespace {
__global__ __launch_bounds__(kRowThreads) void untile_kernel(const uint16_t* __restrict__ src,
                                                             int K, int64_t n_chunks,
                                                             int64_t dst_elems,
                                                             uint16_t* __restrict__ dst) {
  const int64_t c = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  if (c >= n_chunks) return;
  const int64_t m = c / (K / 8);
  const int k = (int)(c - m * (K / 8)) * 8;
  if (m * K + k + 8 > dst_elems) return;
  *(u32x4_t*)(dst + m * K + k) = *(const u32x4_t*)(src + tile_off(m, k, K));
}
}  // namespace

hipError_t launch_untile(const uint16_t* src, int M, int K, uint16_t* dst, int64_t dst_elems,
                         hipStream_t st) {
  if (M <= 0 || dst_elems <= 0) return hipSuccess;
  if (K % 32 != 0) return hipErrorInvalidValue;
  const int64_t n_chunks = (int64_t)M * (K / 8);
  COCO_LAUNCH(untile_kernel, dim3((unsigned)((n_chunks + kRowThreads - 1) / kRowThreads)),
              dim3(kRowThreads), 0, st, src, K, n_chunks, dst_elems, dst);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Down-projection epilogue: y = x1 + sum of partials, rounded to the hidden
// dtype, scattered to the row's place in the full-batch buffer.
// ----------------------------------------------------------------------------
template <typename T, int S>
__global__ __launch_bounds__(kRowThreads) void residual_scatter_kernel(
    const float* __restrict__ part, int M, int d, const float* __restrict__ x1,
    T* __restrict__ out, const int32_t* __restrict__ row_idx) {
  const int i = blockIdx.y;
  const int c = 4 * (blockIdx.x * kRowThreads + threadIdx.x);
  if (c >= d) return;
  const int64_t r = row_idx ? (int64_t)row_idx[i] : (int64_t)i;
  const f32x4_t a = sum_parts4<S>(part + (int64_t)i * d + c, (int64_t)M * d);
  const f32x4_t x = *(const f32x4_t*)(x1 + (int64_t)i * d + c);
#pragma unroll
  for (int e = 0; e < 4; ++e) Elem<T>::store(out + r * d + c + e, x[e] + a[e]);
}

template <typename T>
hipError_t launch_residual_scatter(const float* part, int S, int M, int d, const float* x1,
                                   T* out, const int32_t* row_idx, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (d % 4 != 0) return hipErrorInvalidValue;
  const dim3 grid((d / 4 + kRowThreads - 1) / kRowThreads, M);
  COCO_SWITCH_S(S, COCO_LAUNCH((residual_scatter_kernel<T, S_>), grid, dim3(kRowThreads),
                                      0, st, part, M, d, x1, out, row_idx));
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Paged key/value append (bit copy into the tile layout).
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
    const int64_t tile = (blk * Hkv + h) * kBlockTokens * hd;
    k_cache[tile + k_tile_offset(slot, dim)] = k[src + e];
    v_cache[tile + v_tile_offset(slot, dim)] = v[src + e];
  }
}

template <typename T>
hipError_t launch_kv_append(const T* k, const T* v, const int32_t* seq_idx,
                            const int32_t* positions, int n, int Hkv, int hd,
                            const int32_t* block_table, int max_blocks, T* k_cache,
                            T* v_cache, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  COCO_LAUNCH(kv_append_kernel<T>, dim3(n), dim3(kRowThreads), 0, st, k, v, seq_idx,
                     positions, Hkv, hd, block_table, max_blocks, k_cache, v_cache);
  return hipGetLastError();
}

#define COCO_INSTANTIATE(T)                                                                   \
  template hipError_t launch_gather_rmsnorm<T>(const T*, const int32_t*, int, int, const T*, \
                                               float, T*, T*, bool, const RowSlotArgs&,      \
                                               hipStream_t);                                 \
  template hipError_t launch_qkv_epilogue<T>(const float*, int, int, int, int, int,          \
                                             const int32_t*, const int32_t*, int,            \
                                             const int32_t*, int, const double*, T*, T*, T*, \
                                             const int32_t*, int32_t*, int, const float*,    \
                                             int, float, hipStream_t);                       \
  template hipError_t launch_residual_rmsnorm<T>(const float*, int, int, int, const T*,      \
                                                 const int32_t*, const T*, float, float*, T*, \
                                                 bool, hipStream_t);                         \
  template hipError_t launch_swiglu<T>(const float*, int, int, int, T*, bool, hipStream_t);  \
  template hipError_t launch_residual_scatter<T>(const float*, int, int, int, const float*,  \
                                                 T*, const int32_t*, hipStream_t);           \
  template hipError_t launch_kv_append<T>(const T*, const T*, const int32_t*, const int32_t*, \
                                          int, int, int, const int32_t*, int, T*, T*,        \
                                          hipStream_t);

COCO_INSTANTIATE(bf16_t)
COCO_INSTANTIATE(float)

}  // namespace coco
