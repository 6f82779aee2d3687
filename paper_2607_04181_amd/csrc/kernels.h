// Host-side launchers of the gfx950 kernels (internal to libcoco).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace coco {

// Per-kernel timing (benchmark mode): events that the next kernel launch of
// this thread passes to hipExtLaunchKernelGGL, which timestamps them at the
// kernel's own start and end, then clears. Null events: a plain launch.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

#define COCO_LAUNCH(kernel, grid, block, shmem, stream, ...)                                  \
  do {                                                                                        \
    ::coco::LaunchEvents& le_ = ::coco::launch_events();                                      \
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, le_.start, le_.stop, 0,         \
                          __VA_ARGS__);                                                       \
    le_ = ::coco::LaunchEvents{};                                                             \
  } while (0)

// ---------------------------------------------------------------- row kernels
// Prefill row slots (optional output of the gather kernel): row_info[2i] =
// positions[i] clamped to [0, rope_rows), row_info[2i + 1] = the cache block
// of that position in row i's sequence (rows of a sequence contiguous).
struct RowSlotArgs {
  const int32_t* positions = nullptr;
  const int32_t* seq_starts = nullptr;
  const int32_t* block_table = nullptr;
  int32_t* row_info = nullptr;  // null: not written
  int n_seqs = 0, max_blocks = 0, rope_rows = 0;
};

// x_out[i] = src[row_idx ? row_idx[i] : i];  h_out[i] = RMSNorm(x) * gamma.
// x_out may be null (span layers after the first read x in place).
// tiled (bf16 prefill): h_out in tile order (tile_off), the prefill GEMM's A
// operand layout; otherwise row-major.
template <typename T>
hipError_t launch_gather_rmsnorm(const T* src, const int32_t* row_idx, int M, int d,
                                 const T* gamma, float eps, T* x_out, T* h_out, bool tiled,
                                 const RowSlotArgs& rs, hipStream_t st);

// RoPE table rope[p][j] = (cos, sin)(p * inv_freq[j]) for p < n_pos and
// j < half, angle and both functions in fp64 (as the QKV epilogue computes
// them), stored as fp32 pairs.
hipError_t launch_rope_table(const double* inv_freq, int half, int n_pos, float* rope,
                             hipStream_t st);

// Sum of S split-K partials of the QKV projection, RoPE on query and key
// heads, queries to q_out [M][Hq*hd], keys/values into the paged cache.
// With ss non-null (decode, RMSNorm_1 folded into the projection), each row's
// sums are first scaled by 1 / sqrt(sum_s ss[s][row] / d + eps).
// With split_off non-null (decode), one workgroup also writes the decode
// attention's work list (layout at launch_attn_decode_bf16) from the keys
// each row attends, min(ctx_lens, positions + 1) (partition counts capped at
// max_splits).
template <typename T>
hipError_t launch_qkv_epilogue(const float* part, int S, int M, int Hq, int Hkv, int hd,
                               const int32_t* positions, const int32_t* seq_starts,
                               int n_seqs, const int32_t* block_table, int max_blocks,
                               const double* inv_freq, T* q_out, T* k_cache, T* v_cache,
                               const int32_t* ctx_lens, int32_t* split_off, int max_splits,
                               const float* ss, int d, float eps, hipStream_t st);

// x1 = x + sum_s part[s]  (fp32);  h2 = RMSNorm(x1) * gamma. Row i of x is
// x[row_idx ? row_idx[i] : i]. tiled: h2 in tile order.
template <typename T>
hipError_t launch_residual_rmsnorm(const float* part, int S, int M, int d, const T* x,
                                   const int32_t* row_idx, const T* gamma, float eps, float* x1,
                                   T* h2, bool tiled, hipStream_t st);

// u = silu(sum_s gate) * sum_s up, part rows [2F] = gate then up. tiled: u in
// tile order.
template <typename T>
hipError_t launch_swiglu(const float* part, int S, int M, int F, T* u, bool tiled,
                         hipStream_t st);

// dst[m][k] (row-major, at most dst_elems elements) = src (tile order, [M][K]).
hipError_t launch_untile(const uint16_t* src, int M, int K, uint16_t* dst, int64_t dst_elems,
                         hipStream_t st);

// y = x1 + sum_s part[s];  out[row_idx ? row_idx[i] : i] = y.
template <typename T>
hipError_t launch_residual_scatter(const float* part, int S, int M, int d, const float* x1,
                                   T* out, const int32_t* row_idx, hipStream_t st);

// Bit copy of [n][Hkv][hd] keys/values into the paged cache.
template <typename T>
hipError_t launch_kv_append(const T* k, const T* v, const int32_t* seq_idx,
                            const int32_t* positions, int n, int Hkv, int hd,
                            const int32_t* block_table, int max_blocks, T* k_cache,
                            T* v_cache, hipStream_t st);

// ---------------------------------------------------------------- GEMMs
// Every bf16 GEMM below reads its weights W [N][K] in tile order: the 1 KB
// block (n / 16) * (K / 32) + k / 32 holds rows 16 (n / 16) .. + 15 and k
// 32 (k / 32) .. + 31 as 64 chunks of 8 k, chunk ((k % 32) / 8) * 16 + n % 16.
// launch_pack_tile_order writes that layout from nn.Linear layout (N % 16 ==
// 0, K % 32 == 0).
hipError_t launch_pack_tile_order(const uint16_t* W, int N, int K, uint16_t* out,
                                  hipStream_t st);

// part[s][m][n] = sum_{k in slice s} A[m][k] * W[n][k]   (bf16 in, fp32 out)
// The plan (split count S, workgroup width) and the K-order of every output element depend only on
// (N, K), never on M: rows are independent and batch-invariant.
struct SkinnyPlan {
  int waves;  // 16-column wave groups per workgroup (4..8)
  int S;      // K-slices (split-K)
};
SkinnyPlan skinny_plan(int N, int K);
hipError_t launch_gemm_skinny_bf16(const uint16_t* A, const uint16_t* W, float* part, int M,
                                   int N, int K, SkinnyPlan plan, hipStream_t st);
// Same with the gather and RMSNorm_1 folded in: the operand of row m is
// bf16(X[row_idx ? row_idx[m] : m] * gamma), and ss[s][m] = sum of X^2 over
// K-slice s (the consumer scales row m's sums by its 1/rms).
hipError_t launch_gemm_skinny_norm_bf16(const uint16_t* X, const int32_t* row_idx,
                                        const uint16_t* gamma, const uint16_t* W, float* part,
                                        float* ss, int M, int N, int K, SkinnyPlan plan,
                                        hipStream_t st);
// Decode gate/up GEMM with the SwiGLU epilogue: H[M][F] = bf16(silu(A W_g^T) *
// (A W_u^T)), W_gate_up = [W_g; W_u] [2F][K]; plan = skinny_plan(2F, K) with S == 1.
// h_tiled: H in tile order (for a down projection that reads it so).
hipError_t launch_gemm_skinny_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                          uint16_t* H, int M, int F, int K, SkinnyPlan plan,
                                          bool h_tiled, hipStream_t st);
// Whether the decode GEMM of (N, K) at M rows (fuse: the SwiGLU variant) runs
// the row-split kernel, which reads its activations A in tile order
// (tile_off); the other decode kernels read A row-major.
bool skinny_reads_tiled(int N, int K, int M, bool fuse);

// part[s][m][n] = sum_{k in slice s} A[m][k] * W[n][k] with 256 x 256 MFMA
// tiles (prefill; K a multiple of 64 * S). S = tile_splits(N, K); the k
// order is fixed and M-independent. The tile GEMMs read A in tile order
// (tile_off; its buffer holds M rounded up to 16 rows) and write their bf16
// activation outputs (SwiGLU and residual variants) in tile order.
int tile_splits(int N, int K);
hipError_t launch_gemm_tile_bf16(const uint16_t* A, const uint16_t* W, float* C, int M, int N,
                                 int K, int S, hipStream_t st);
// Epilogue inputs of the tile GEMM variants below (unused fields zero).
struct TileEpiArgs {
  // QKV variant
  const int32_t* row_info = nullptr;  // [M][2] row slots from the gather kernel
  const float* rope = nullptr;        // [rope_rows][64] (cos, sin) pairs
  uint16_t* q_out = nullptr;
  uint16_t* k_cache = nullptr;
  uint16_t* v_cache = nullptr;
  int Hq = 0, Hkv = 0;
  // residual variant
  const uint16_t* res_x = nullptr;    // residual rows [*][N] (bf16)
  const int32_t* res_idx = nullptr;   // row m's residual row (null: m)
  const uint16_t* gamma = nullptr;    // RMSNorm_2 gains [N]
  float* ss_part = nullptr;           // [N / 256][M] per-tile row sums of x1^2
  // SwiGLU variant with RMSNorm_2 folded in
  const float* ss_in = nullptr;       // [n_ss][M] from the residual variant
  int n_ss = 0, d = 0;
  float eps = 0.f;
};

// Gate/up GEMM with the SwiGLU epilogue: H[M][F] = bf16(silu(A W_g^T) * (A W_u^T))
// where W_gate_up = [W_g; W_u] is [2F][K]; only for tile_splits(2F, K) == 1.
// With ss_in non-null (RMSNorm_2 folded in: A = bf16(x1 * gamma)), gate and
// up of row m are first scaled by 1 / sqrt(sum_t ss_in[t][m] / K + eps),
// t < ss_tiles (at most 32) in order.
hipError_t launch_gemm_tile_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                        uint16_t* H, int M, int F, int K, const float* ss_in,
                                        int ss_tiles, float eps, hipStream_t st);
// Prefill QKV projection with the QKV epilogue in the GEMM's own epilogue
// (head_dim 128): RoPE on query and key heads with the rotations of the RoPE
// table, queries to q_out [M][Hq*128] in bf16, keys and values into the
// paged cache tiles; no fp32 partials. Only when tile_qkv_fusable(Hq, Hkv, K).
bool tile_qkv_fusable(int Hq, int Hkv, int K);
hipError_t launch_gemm_tile_qkv_bf16(const uint16_t* A, const uint16_t* W_qkv, int M, int K,
                                     const TileEpiArgs& ea, hipStream_t st);
// Prefill O projection with the residual and the first half of RMSNorm_2 in
// its epilogue: x1[m] = A W^T + res_x[res_idx ? res_idx[m] : m] (fp32),
// h[m] = bf16(x1 * gamma), ss_part[t][m] = sum of x1^2 over columns
// 256t .. 256t + 255. With tile_norm2_foldable(d, qdim, F), the O projection
// (N = d, K = qdim) and the gate/up projection take this path.
bool tile_norm2_foldable(int d, int qdim, int F);
hipError_t launch_gemm_tile_resid_bf16(const uint16_t* A, const uint16_t* W, int M, int N, int K,
                                       const uint16_t* res_x, const int32_t* res_idx,
                                       const uint16_t* gamma, float* x1, uint16_t* h,
                                       float* ss_part, hipStream_t st);

// Narrow-output prefill GEMMs (N = the model width): 256 x TN tiles,
// TN = narrow_tile_n(N) (128 or 160, N / TN <= 32 column tiles; 0: no plan),
// unsplit along K (K a multiple of 128), A and W in tile order.
int narrow_tile_n(int N);
struct NarrowEpiArgs {
  // residual variant (O projection)
  const uint16_t* res_x = nullptr;   // residual rows [*][N] (bf16)
  const int32_t* res_idx = nullptr;  // row m's residual row (null: m)
  const uint16_t* gamma = nullptr;   // RMSNorm_2 gains [N]
  float* x1 = nullptr;               // [M][N] fp32
  uint16_t* h = nullptr;             // bf16(x1 * gamma), tile order
  float* ss_part = nullptr;          // [N / TN][M] per-tile row sums of x1^2
  // scatter variant (down projection)
  const float* x1_in = nullptr;      // [M][N] fp32 residual
  uint16_t* out = nullptr;           // output rows [*][N] (bf16)
  const int32_t* out_idx = nullptr;  // row m's output row (null: m)
  // SwiGLU variant (gate/up projection, RMSNorm_2 folded in); h above is
  // its output [M][N / 2] in tile order
  const float* ss_in = nullptr;      // [n_ss][M] from the residual variant
  int n_ss = 0;
  float eps = 0.f;
  // QKV variant (head_dim 128)
  const int32_t* row_info = nullptr;  // [M][2] row slots from the gather kernel
  const float* rope = nullptr;        // [rope_rows][64] (cos, sin) pairs
  uint16_t* q_out = nullptr;
  uint16_t* k_cache = nullptr;
  uint16_t* v_cache = nullptr;
  int Hq = 0, Hkv = 0;
};
// O projection with the residual and the first half of RMSNorm_2 in its
// epilogue: x1[m] = A W^T + res_x[res_idx ? res_idx[m] : m] (fp32),
// h[m] = bf16(x1 * gamma) in tile order, ss_part[t][m] = sum of x1^2 over
// columns TN t .. TN t + TN - 1, summed in a fixed order.
hipError_t launch_gemm_narrow_resid_bf16(const uint16_t* A, const uint16_t* W, int M, int N,
                                         int K, const uint16_t* res_x, const int32_t* res_idx,
                                         const uint16_t* gamma, float* x1, uint16_t* h,
                                         float* ss_part, hipStream_t st);
// Gate/up projection with RMSNorm_2's 1/rms and the SwiGLU in its epilogue,
// on 256 x 192 tiles (96 outputs each): H[m] = bf16(silu(g) * u) in tile
// order [M][F], where (g, u) = (A W_g^T, A W_u^T)[m] / sqrt(sum_t ss_in[t][m]
// / K + eps), t < ss_tiles (at most 32) in order, and W_gate_up = [W_g; W_u]
// is [2F][K]. Only when narrow_swiglu_fits(F, K): 2F a multiple of 192.
bool narrow_swiglu_fits(int F, int K);
hipError_t launch_gemm_narrow_swiglu_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                          uint16_t* H, int M, int F, int K, const float* ss_in,
                                          int ss_tiles, float eps, hipStream_t st);
// The same SwiGLU epilogue without the 1/rms (A already normalised), on
// 256 x 128 tiles, for decode batches whose gate/up GEMM takes one round of
// workgroups: narrow_swiglu_plain_fits(M, F, K). A is in tile order, H is
// written in tile order [M][F]. Every output is the v_mfma_f32_16x16x32_bf16
// chain over k in ascending 32-steps of the decode GEMMs, with the same
// epilogue arithmetic, so the bits equal theirs.
bool narrow_swiglu_plain_fits(int M, int F, int K);
hipError_t launch_gemm_narrow_swiglu_plain_bf16(const uint16_t* A, const uint16_t* W_gate_up,
                                                uint16_t* H, int M, int F, int K,
                                                hipStream_t st);
// Prefill QKV projection with RoPE and the cache append in its epilogue
// (head_dim 128), on 256 x TN tiles that each hold TN/2 whole rotation pairs
// (dims j and j + 64 of a head), TN = narrow_qkv_tile_n(Hq, Hkv, K) (224,
// 192 or 160; 0: no plan): queries to q_out [M][Hq*128] in bf16, keys
// (rotated) and values into the paged cache tiles.
int narrow_qkv_tile_n(int Hq, int Hkv, int K);
hipError_t launch_gemm_narrow_qkv_bf16(const uint16_t* A, const uint16_t* W_qkv, int M, int K,
                                       const NarrowEpiArgs& ea, hipStream_t st);
// Down projection with the residual and the scatter in its epilogue:
// out[out_idx ? out_idx[m] : m] = bf16(x1[m] + A W^T).
hipError_t launch_gemm_narrow_scatter_bf16(const uint16_t* A, const uint16_t* W, int M, int N,
                                           int K, const float* x1, uint16_t* out,
                                           const int32_t* out_idx, hipStream_t st);

// part[0][m][n] = sum_k A[m][k] * W[n][k], fp32 (tiny fp32 configurations).
hipError_t launch_gemm_f32(const float* A, const float* W, float* part, int M, int N, int K,
                           hipStream_t st);

// ---------------------------------------------------------------- attention
constexpr int kDecodeSplit = 256;  // tokens per split-KV partition
int decode_max_splits(int max_blocks_per_seq);
bool attn_combine_fits(int max_splits);

// split_off (at most 2 n_seqs + 2 entries, written by the QKV epilogue of the
// same call): [0 .. n_seqs] the exclusive prefix sum of each sequence's full
// 256-key partitions; [n_seqs + 1] the number of sequences whose last
// partition is partial; [n_seqs + 2 ..] those sequences, longest last
// partition first.
// Decode row s attends min(ctx_lens[s], positions[s] + 1) keys.
hipError_t launch_attn_decode_bf16(const uint16_t* q, const uint16_t* k_cache,
                                   const uint16_t* v_cache, const int32_t* block_table,
                                   int max_blocks, const int32_t* ctx_lens,
                                   const int32_t* positions, const int32_t* split_off,
                                   int n_seqs, int Hq, int Hkv, float* part_o, float* part_ml,
                                   int max_splits, int num_cus, hipStream_t st);
// tiled: o in tile order (for an O projection that reads it so).
hipError_t launch_attn_combine_bf16(const float* part_o, const float* part_ml,
                                    const int32_t* ctx_lens, const int32_t* positions,
                                    int n_seqs, int Hq, int max_splits, uint16_t* o, bool tiled,
                                    hipStream_t st);

// Causal attention of prefill rows over their sequences' caches; o [n_rows]
// [Hq * 128] is written in tile order (the O projection's A operand).
hipError_t launch_attn_prefill_bf16(const uint16_t* q, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const int32_t* block_table,
                                    int max_blocks, const int32_t* ctx_lens,
                                    const int32_t* positions, const int32_t* seq_starts,
                                    int n_seqs, int n_rows, int Hq, int Hkv, uint16_t* o,
                                    hipStream_t st);

// fp32 path: one wave per (row, query head), decode and prefill alike.
hipError_t launch_attn_f32(const float* q, const float* k_cache, const float* v_cache,
                           const int32_t* block_table, int max_blocks,
                           const int32_t* ctx_lens, const int32_t* positions,
                           const int32_t* seq_starts, int n_seqs, int n_rows, int Hq,
                           int Hkv, int hd, float* o, hipStream_t st);

}  // namespace coco
