// Shared device helpers for the gfx950 kernels: bf16 conversion, vector
// types for MFMA operands, wave/block reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace coco {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kBlockTokens = 16;  // paged-cache block size

__device__ __forceinline__ float bf16_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Round to nearest even with the hardware converter (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16x2(f, 0.f) & 0xFFFFu; }

// SwiGLU's product silu(g) u = g u / (1 + e^-g), with the hardware 2^x
// (v_exp_f32) and reciprocal (v_rcp_f32), each within 1 ulp: the result is a
// few fp32 ulps from the exact value, far inside the bf16 rounding that
// follows, and costs eight VALU operations instead of the ~30 of a
// range-reduced expf and an IEEE division. Below g = -88, e^-g overflows and
// the product is a signed zero (the exact value is under 1e-36 |u|).
__device__ __forceinline__ float silu_mul(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(g * -1.4426950408889634f);
  return g * __builtin_amdgcn_rcpf(1.0f + e) * u;
}

// Element load/store for the two activation types.
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { *p = (bf16_t)f32_to_bf16(v); }
};
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};

// Four consecutive elements (p 8-byte aligned for bf16, 16-byte for fp32) in
// one store.
__device__ __forceinline__ void store4(bf16_t* p, float a, float b, float c, float d) {
  typedef uint32_t u2 __attribute__((ext_vector_type(2)));
  *(u2*)p = u2{pack_bf16x2(a, b), pack_bf16x2(c, d)};
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  *(f4*)p = f4{a, b, c, d};
}

// Waits until at most N vector-memory operations of this wave are in flight
// (vmcnt only; direct global-to-LDS loads count there). N counts the loads
// issued before this point in program order, so no memory operation may move
// across it: the fences and scheduling barriers pin it (the waitcnt builtin
// alone lets the compiler sink earlier loads below it, which would make the
// wait release too early). ALU and MFMA instructions may still cross.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  constexpr int kMayCross = 0x1 | 0x2 | 0x4 | 0x8 | 0x400;  // ALU, VALU, SALU, MFMA, transcendental
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_sched_barrier(kMayCross);
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
  __builtin_amdgcn_sched_barrier(kMayCross);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Workgroup barrier that keeps the compiler from moving memory operations
// across it and adds no waits of its own: the direct-to-LDS loads of later
// stages stay in flight through it (a __syncthreads() fence would drain them).
__device__ __forceinline__ void stage_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Reductions over the four lanes i, i^16, i^32, i^48 (one MFMA output
// column) with the cross-row swaps, no LDS round trip. Every lane of the
// column gets the same bits.
__device__ __forceinline__ float col_max4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float col_sum4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over a block of NT threads with a fixed reduction tree (the order does
// not depend on anything but NT). `red` holds NT/64 floats.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) t += red[i];
  __syncthreads();
  return t;
}

// Paged cache tiles. A (block, kv head) tile holds 16 tokens x hd dims
// (hd a multiple of 32) in MFMA operand order:
//  K: element (token t, dim h) at ((h/32)*64 + ((h%32)/8)*16 + t)*8 + h%8, so
//     1 KB piece s (dims 32s..32s+31) is the A operand of one 16x16x32 MFMA
//     step with lane i holding token i%16, dims 32s + 8(i/16) .. +8;
//  V: element (t, h) at (((h/32)*64 + (t/4)*16 + h%16)*2 + (h/16)%2)*4 + t%4,
//     so lane i of 1 KB piece p holds, for the two 16-dim tiles 2p and 2p+1,
//     dims 16n + i%16 at tokens 4(i/16) .. +4 (A operands of 16x16x16 MFMAs
//     computing V^T P^T).
__device__ __forceinline__ int k_tile_offset(int t, int h) {
  return (((h >> 5) * 64 + ((h >> 3) & 3) * 16 + t) << 3) + (h & 7);
}
__device__ __forceinline__ int v_tile_offset(int t, int h) {
  return ((((h >> 5) * 64 + (t >> 2) * 16 + (h & 15)) * 2 + ((h >> 4) & 1)) << 2) + (t & 3);
}

// Tile order of a bf16 matrix [M][K] (K % 32 == 0; rows padded to a multiple
// of 16): the 1 KB block (m / 16) * (K / 32) + k / 32 holds rows
// 16 (m / 16) .. + 15 and columns 32 (k / 32) .. + 31 as 64 chunks of 8
// consecutive columns, chunk ((k % 32) / 8) * 16 + m % 16 -- the layout of
// the weight copies, read by the prefill GEMM one block per load. Element
// offset of (m, k); 8 columns from a multiple of 8 are contiguous.
__device__ __forceinline__ int64_t tile_off(int64_t m, int k, int K) {
  return ((((m >> 4) * (K >> 5) + (k >> 5)) << 6) + ((k & 31) >> 3) * 16 + (m & 15)) * 8 +
         (k & 7);
}

// Sequence of a call row: identity for decode, else the s with
// seq_starts[s] <= row < seq_starts[s+1].
__device__ __forceinline__ int row_to_seq(const int32_t* seq_starts, int n_seqs, int row) {
  if (seq_starts == nullptr) return row;
  int lo = 0, hi = n_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seq_starts[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace coco
