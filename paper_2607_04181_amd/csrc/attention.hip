// Grouped-query attention over the paged key/value cache.
//
// Cache layout per layer (block = 16 tokens): [blocks][Hkv][tile], each tile
// of 16 tokens x hd in MFMA operand order (k_tile_offset / v_tile_offset).
//
// MFMA dataflow (bf16, hd = 128), shared by decode and prefill. A wave owns 16
// "query columns" per column tile and walks the key blocks of one key/value
// head:
//   S^T[16 tok][16 col] = K_blk[16][hd] . Q^T[hd][16]   4 x mfma 16x16x32
//   online softmax per column (column max/sum over the 4 lanes of a column)
//   O^T[hd][16 col]    += V^T_blk[hd][16] . P^T[16][16] 8 x mfma 16x16x16,
//                         or 8 x mfma 16x16x32 per pair of blocks
// With S^T the probabilities come out of the first MFMA already in the
// B-operand layout of the second, and O^T keeps a column's rescale factor in
// the lane that computed it: no cross-lane shuffles besides the column
// max/sum. Because tiles are stored in operand order, every K and V read is a
// contiguous 1 KB wave load.
//
// Decode: the columns are the G = Hq/Hkv query heads of one token (padded to
// 16). A workgroup handles (sequence, kv head, 256-token partition); its
// eight waves take interleaved blocks and merge in LDS in wave order;
// partitions are merged by a second kernel in partition order. Partitions
// depend only on the sequence's own length, so results are independent of
// the batch.
// Prefill: the columns are 16 query tokens of one head, masked causally by
// absolute position; key/value tiles are shared by the workgroup's waves
// through LDS.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace coco {

namespace {

constexpr int HD = 128;
constexpr float kLog2e = 1.4426950408889634f;

// One (block, kv head) tile: four contiguous 1 KB loads each for K and V,
// non-temporal (each tile is read once per step).
__device__ __forceinline__ void load_kv(const bf16_t* kb, const bf16_t* vb, int c16, int j4,
                                        u32x4_t kf[4], u32x2_t vf[8]) {
  const int lane = j4 * 16 + c16;
#pragma unroll
  for (int t = 0; t < 4; ++t)
    kf[t] = __builtin_nontemporal_load((const u32x4_t*)(kb + (t * 64 + lane) * 8));
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)(vb + (p * 64 + lane) * 8));
    vf[2 * p] = u32x2_t{v.x, v.y};
    vf[2 * p + 1] = u32x2_t{v.z, v.w};
  }
}

// ---------------------------------------------------------------- decode
// Persistent workgroups walk the work list of (partition, kv head) items that
// the QKV epilogue wrote (split_off): every full 256-key partition first, then
// each sequence's partial last partition, largest first. Workgroup b takes
// list positions k * grid + b for even k and k * grid + grid - 1 - b for odd
// k, so that every workgroup gets about the same number of keys (the items
// that differ in size come last, dealt out largest first and snake-wise).
// The order changes which workgroup computes an item, never what it computes
// or where its result goes. Eight waves take two
// blocks each of the 256-token partition; each wave scores both blocks
// first, takes one column max and then accumulates exp * V against it, and
// the eight wave results are merged in LDS in wave order. As soon as a
// wave's key/value registers are consumed it issues the loads of its next
// work item, so the LDS merge and the partial stores overlap the next
// item's HBM reads.
constexpr int kDecWaves = 8;
constexpr int kDecBPW = kDecodeSplit / kBlockTokens / kDecWaves;

struct DecItem {
  int s, g, sp, t1, b_first, b_last;
  int64_t pb[kDecBPW];  // physical blocks of this wave's share (clamped to b_last)
};

// Keys a decode row attends: positions 0 .. its own position, within the
// cached length (min(ctx_lens[s], positions[s] + 1), never negative).
__device__ __forceinline__ int decode_keys(const int32_t* ctx_lens, const int32_t* positions,
                                           int s) {
  return max(0, min(ctx_lens[s], positions[s] + 1));
}

// Item w of the work list: split_off[0 .. n_seqs] is the exclusive prefix sum
// of each sequence's full partitions, split_off[n_seqs + 1] the number of
// partial last partitions and split_off[n_seqs + 2 ..] their sequences,
// largest first.
__device__ __forceinline__ DecItem decode_item(int w, int Hkv, const int32_t* split_off,
                                               const int32_t* ctx_lens,
                                               const int32_t* positions, int n_seqs,
                                               int max_blocks) {
  DecItem it;
  const int item = w / Hkv;
  it.g = w - item * Hkv;
  const int n_full = split_off[n_seqs];
  if (item < n_full) {
    int lo = 0, hi = n_seqs - 1;  // the s with split_off[s] <= item < split_off[s + 1]
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (split_off[mid] <= item) lo = mid; else hi = mid - 1;
    }
    it.s = lo;
    it.sp = item - split_off[lo];
  } else {
    it.s = split_off[n_seqs + 2 + (item - n_full)];
    it.sp = split_off[it.s + 1] - split_off[it.s];
  }
  const int t0 = it.sp * kDecodeSplit;
  // Capped at the block table's width (only invalid lengths reach the cap).
  it.t1 = min(min(decode_keys(ctx_lens, positions, it.s), t0 + kDecodeSplit),
              max_blocks * kBlockTokens);
  it.b_first = t0 / kBlockTokens;
  it.b_last = (it.t1 - 1) / kBlockTokens;
  return it;
}

// The block-table entries of wave wv's blocks of item it: unconditional
// (blocks past the partition repeat its last block, an L2 hit that is then
// ignored), so that the waits before each MFMA can count exactly the loads
// still in flight behind the ones it needs.
__device__ __forceinline__ void decode_item_blocks(DecItem& it, const int32_t* block_table,
                                                   int max_blocks, int wv) {
  const int32_t* bt = block_table + (int64_t)it.s * max_blocks;
#pragma unroll
  for (int u = 0; u < kDecBPW; ++u) it.pb[u] = bt[min(it.b_first + wv + kDecWaves * u, it.b_last)];
}

__global__ __launch_bounds__(kDecWaves * 64, 4) void attn_decode_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k_cache,
    const bf16_t* __restrict__ v_cache, const int32_t* __restrict__ block_table, int max_blocks,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ positions,
    const int32_t* __restrict__ split_off, int n_seqs, int Hq, int Hkv,
    float* __restrict__ part_o, float* __restrict__ part_ml, int max_splits, float scale_log2) {
  __shared__ float sm_m[kDecWaves][16], sm_l[kDecWaves][16];
  __shared__ float sm_o[kDecWaves][16][HD + 4];

  const int total = (split_off[n_seqs] + split_off[n_seqs + 1]) * Hkv;
  const int G = Hq / Hkv;
  const int lane = threadIdx.x & 63;
  // Wave index as a uniform value: block-table reads then go through the
  // scalar cache and do not wait behind the key/value loads in flight.
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c16 = lane & 15, j4 = lane >> 4;
  const int64_t tile = (int64_t)kBlockTokens * HD;
  const int cq = c16 < G ? c16 : G - 1;  // padded columns read a real head

  u32x4_t kf[kDecBPW][4];
  u32x2_t vf[kDecBPW][8];
  u32x4_t qr[4];
  // Query first: the first MFMA needs it, and loads complete in issue order.
  auto issue = [&](const DecItem& it) {
    const bf16_t* qp = q + ((int64_t)it.s * Hq + it.g * G + cq) * HD + j4 * 8;
#pragma unroll
    for (int t = 0; t < 4; ++t) qr[t] = *(const u32x4_t*)(qp + t * 32);
#pragma unroll
    for (int u = 0; u < kDecBPW; ++u)
      load_kv(k_cache + (it.pb[u] * Hkv + it.g) * tile, v_cache + (it.pb[u] * Hkv + it.g) * tile,
              c16, j4, kf[u], vf[u]);
  };
  // The descriptor of the item after the current one, block-table entries
  // included, is looked up one item ahead: its chain of dependent scalar
  // loads runs while the current item's key/value loads are in flight, and
  // the next issue has its addresses at hand. Past the last item it repeats
  // the last one, which is never used.
  auto lookup = [&](int wi) {
    DecItem it = decode_item(min(wi, total - 1), Hkv, split_off, ctx_lens, positions, n_seqs,
                             max_blocks);
    decode_item_blocks(it, block_table, max_blocks, wv);
    return it;
  };

  // List position of this workgroup's k-th item (snake order).
  const int grid = gridDim.x;
  auto pos_of = [&](int k) { return k * grid + ((k & 1) ? grid - 1 - (int)blockIdx.x : (int)blockIdx.x); };
  int k = 0, w = pos_of(0);
  DecItem cur{}, nxt{};
  if (w < total) {
    cur = lookup(w);
    issue(cur);
    nxt = lookup(pos_of(1));
  }
  for (; w < total; w = pos_of(++k)) {
    // Columns c16 >= G repeat head G-1; their results are never stored.
    bf16x8_t qf[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) qf[t] = __builtin_bit_cast(bf16x8_t, qr[t]);
    // Pass 1: scores of all of the wave's blocks, one column max.
    float sc[kDecBPW][4];
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < kDecBPW; ++u) {
      const int b = cur.b_first + wv + kDecWaves * u;
      f32x4_t a = {0.f, 0.f, 0.f, 0.f};
      if (b <= cur.b_last) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf[u][t]),
                                                      qf[t], a, 0, 0, 0);
      }
      const int tok0 = b * kBlockTokens + j4 * 4;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc[u][r] = (b <= cur.b_last && tok0 + r < cur.t1) ? a[r] * scale_log2 : -INFINITY;
        m = fmaxf(m, sc[u][r]);
      }
    }
    m = col_max4(m);
    // Pass 2: probabilities against the fixed max, O^T += V^T P^T. A wave
    // with no block keeps m = -inf and contributes nothing.
    const float mref = m == -INFINITY ? 0.f : m;
    float l = 0.f;
    f32x4_t o[8];
#pragma unroll
    for (int n = 0; n < 8; ++n) o[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kDecBPW; ++u) {
      const int b = cur.b_first + wv + kDecWaves * u;
      if (b <= cur.b_last) {
        float p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) p[r] = exp2f(sc[u][r] - mref);
        l += (p[0] + p[1]) + (p[2] + p[3]);
        const s16x4_t pf = __builtin_bit_cast(
            s16x4_t, u32x2_t{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])});
#pragma unroll
        for (int n = 0; n < 8; ++n)
          o[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, vf[u][n]),
                                                           pf, o[n], 0, 0, 0);
      }
    }
    const float l_col = col_sum4(l);
    if (j4 == 0) {
      sm_m[wv][c16] = m;
      sm_l[wv][c16] = l_col;
    }
#pragma unroll
    for (int n = 0; n < 8; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm_o[wv][c16][n * 16 + j4 * 4 + r] = o[n][r];
    // The registers are free: start the next item's reads now, then look up
    // the one after it.
    const DecItem it = cur;
    cur = nxt;
    issue(cur);
    nxt = lookup(pos_of(k + 2));
    __syncthreads();

    for (int e = threadIdx.x; e < G * HD; e += kDecWaves * 64) {
      const int col = e / HD, dim = e - col * HD;
      float mx = sm_m[0][col];
#pragma unroll
      for (int v = 1; v < kDecWaves; ++v) mx = fmaxf(mx, sm_m[v][col]);
      float acc = 0.f, L = 0.f;
#pragma unroll
      for (int v = 0; v < kDecWaves; ++v) {
        const float f = exp2f(sm_m[v][col] - mx);
        acc += f * sm_o[v][col][dim];
        L += f * sm_l[v][col];
      }
      const int64_t idx = ((int64_t)it.s * Hq + it.g * G + col) * max_splits + it.sp;
      part_o[idx * HD + dim] = acc;
      if (dim == 0) {
        part_ml[idx * 2 + 0] = mx;
        part_ml[idx * 2 + 1] = L;
      }
    }
    __syncthreads();  // LDS is reused by the next work item
  }
}

// Merge the partitions of one (sequence, query head) in partition order.
// Partition weights exp2(m_sp - max) are computed once into LDS (dynamic,
// 2 * max_splits floats); each thread then owns one head dimension. Loads
// that do not depend on the sequence's length go out together with it (the
// first kPre partitions' values and the thread's own (max, sum) pair), so a
// sequence of up to kPre * 256 tokens needs one memory round trip.
constexpr int kPre = 8;

__global__ __launch_bounds__(HD) void attn_combine_kernel(const float* __restrict__ part_o,
                                                          const float* __restrict__ part_ml,
                                                          const int32_t* __restrict__ ctx_lens,
                                                          const int32_t* __restrict__ positions,
                                                          int Hq, int max_splits,
                                                          bf16_t* __restrict__ o, bool tiled) {
  extern __shared__ float sm[];  // [0, max_splits): weights; [max_splits, 2*max_splits): l
  __shared__ float red[HD / kWave];
  const int h = blockIdx.x, s = blockIdx.y, dim = threadIdx.x;
  const int64_t base = ((int64_t)s * Hq + h) * max_splits;
  const float* po = part_o + base * HD + dim;
  // Slots past the sequence's partition count hold stale values; they are
  // loaded (inside the workspace) but never used.
  float pre[kPre];
#pragma unroll
  for (int k = 0; k < kPre; ++k) pre[k] = k < max_splits ? po[k * HD] : 0.f;
  float m_own = -INFINITY, l_own = 0.f;
  if (dim < max_splits) {
    m_own = part_ml[(base + dim) * 2];
    l_own = part_ml[(base + dim) * 2 + 1];
  }
  const int nsp =
      min((decode_keys(ctx_lens, positions, s) + kDecodeSplit - 1) / kDecodeSplit, max_splits);
  float mx = -INFINITY;
  if (dim < nsp) {
    sm[dim] = m_own;
    sm[max_splits + dim] = l_own;
    mx = m_own;
  }
  for (int sp = dim + HD; sp < nsp; sp += HD) {
    const float m = part_ml[(base + sp) * 2];
    sm[sp] = m;
    sm[max_splits + sp] = part_ml[(base + sp) * 2 + 1];
    mx = fmaxf(mx, m);
  }
  mx = wave_max(mx);
  if ((dim & (kWave - 1)) == 0) red[dim / kWave] = mx;
  __syncthreads();
  mx = fmaxf(red[0], red[1]);
  for (int sp = dim; sp < nsp; sp += HD) sm[sp] = exp2f(sm[sp] - mx);
  __syncthreads();
  float acc = 0.f, L = 0.f;
#pragma unroll
  for (int k = 0; k < kPre; ++k)
    if (k < nsp) acc += sm[k] * pre[k];
  int sp = kPre;
  for (; sp + 4 <= nsp; sp += 4) {
    const float a0 = po[(sp + 0) * HD], a1 = po[(sp + 1) * HD];
    const float a2 = po[(sp + 2) * HD], a3 = po[(sp + 3) * HD];
    acc += sm[sp] * a0;
    acc += sm[sp + 1] * a1;
    acc += sm[sp + 2] * a2;
    acc += sm[sp + 3] * a3;
  }
  for (; sp < nsp; ++sp) acc += sm[sp] * po[sp * HD];
  for (sp = 0; sp < nsp; ++sp) L += sm[sp] * sm[max_splits + sp];
  o[tiled ? tile_off(s, h * HD + dim, Hq * HD) : ((int64_t)s * Hq + h) * HD + dim] =
      (bf16_t)f32_to_bf16(nsp > 0 ? acc / L : 0.f);
}

// ---------------------------------------------------------------- prefill
// Workgroup = (sequence, 128-row query tile, query head). Workgroups are
// remapped so that the query heads of one tile run back to back on one XCD
// (blockIdx % 8) and share its L2 for the key/value tiles of their group.
// Its sixteen waves form two key sets of eight; in each set a wave takes 16
// rows of the tile as one 16-column tile. The key/value tiles are staged
// through LDS eight blocks (128 keys) at a time by direct global->LDS loads
// (each wave fetches one block's K or V tile as four contiguous 1 KB
// pieces), double-buffered with one barrier per stage; key set 0 works on
// the stage's first four blocks and key set 1 on the last four. Per stage a
// wave scores its 64 keys (S^T = K Q^T), updates its online softmax once,
// and accumulates O^T += V^T P^T in 32-key MFMA steps: the V^T fragments of
// two blocks side by side against P^T packed to match (any fixed assignment
// of keys to MFMA k-slots gives the same sum). The row sums of P come from
// the same MFMA with an all-ones operand in place of V^T, and the running
// max moves only when a stage's max exceeds it by kPfLazy. At the end the
// two sets' softmax states of each row are merged in LDS, set 0 first.
// Splitting the keys halves the longest tile's chain of stages (the tiles
// of a long sequence's chunk see the most keys) against two workgroups of
// eight waves per CU that each walk all the keys: 114-117 -> 100-102 us on
// the 32B 2048-token chunked prefill (A/B, same box).
constexpr int kPfRows = 128;  // query rows per workgroup
constexpr int kPfLaunchWaves = 8;  // waves per key set, one 16-row column tile each (measured faster than 4 x 2)
constexpr int kPfKeySets = 2;      // key sets per workgroup
constexpr int kPfBlk = 4;     // key blocks per stage
// The running max of a row is kept while a stage's max stays within this
// many log2 units of it (P then stays below 2^8): rescaling the
// accumulators, a multiply per element, is needed only when the max jumps.
constexpr float kPfLazy = 8.f;
constexpr int kTileElems = kBlockTokens * HD;
constexpr int kXCDs = 8;

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) const volatile u32x2_t lds_u32x2_cv;

// 8-byte LDS read of p (a pointer into LDS). volatile keeps the two halves of
// a 16-byte chunk from being merged into one 16-byte read, which would need
// register moves to split.
__device__ __forceinline__ u32x2_t lds_read8(const bf16_t* p) { return *(lds_u32x2_cv*)p; }

// WAVES waves of COLS 16-column tiles each cover the workgroup's 128 rows;
// KS sets of WAVES waves split every stage's keys between them (set kh takes
// blocks kh * kPfBlk .. of a stage of KS * kPfBlk blocks) and merge their
// softmax states in LDS at the end.
template <int WAVES, int COLS, int KS>
__global__ __launch_bounds__(WAVES * KS * 64, KS > 1 ? 1 : 8 / WAVES) void attn_prefill_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k_cache,
    const bf16_t* __restrict__ v_cache, const int32_t* __restrict__ block_table, int max_blocks,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ positions,
    const int32_t* __restrict__ seq_starts, int n_seqs, int Hq, int Hkv, float scale_log2,
    bf16_t* __restrict__ o) {
  static_assert(KS == 1 || KS == 2, "one or two key sets");
  constexpr int kStBlk = kPfBlk * KS;  // key blocks per stage
  // Two K and two V slots of a stage's kStBlk tiles each, in one LDS array.
  constexpr int kSlot = kStBlk * kTileElems;
  __shared__ __attribute__((aligned(16))) bf16_t kv[4 * kSlot];
  auto k_slot = [&](int st) { return kv + (st & 1) * kSlot; };
  auto v_slot = [&](int st) { return kv + (2 + (st & 1)) * kSlot; };

  // Work unit = (tile, kv head) with its G query heads. Units go round-robin
  // over the XCDs (blockIdx % 8 is the XCD) and a unit's G workgroups run
  // back to back on its XCD, sharing the group's key/value tiles in that L2.
  // Tiles are taken last-first: later tiles of a sequence see more keys, so
  // the long workgroups start early.
  const int G = Hq / Hkv;
  const int n_tiles = gridDim.x / Hq;
  int unit, hg;
  if ((n_tiles * Hkv) % kXCDs == 0) {
    const int x = blockIdx.x % kXCDs, k = blockIdx.x / kXCDs;
    unit = x + kXCDs * (k / G);
    hg = k % G;
  } else {
    unit = blockIdx.x / G;
    hg = blockIdx.x % G;
  }
  int tile = n_tiles - 1 - unit / Hkv;
  const int g = unit % Hkv;
  const int h = g * G + hg;
  int s = 0;
  for (; s < n_seqs; ++s) {
    const int nt = (seq_starts[s + 1] - seq_starts[s] + kPfRows - 1) / kPfRows;
    if (tile < nt) break;
    tile -= nt;
  }
  if (s >= n_seqs) return;  // past the last tile: the whole workgroup leaves
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rg = wv % WAVES, kh = wv / WAVES;  // row group, key set
  const int c16 = lane & 15, j4 = lane >> 4;
  const int row_begin = seq_starts[s] + tile * kPfRows;
  const int row_end = min(seq_starts[s + 1], row_begin + kPfRows);
  // Rows are in position order: the tile's last row sees the most keys.
  const int kmax = min(ctx_lens[s] - 1, positions[row_end - 1]);
  const int n_blk = kmax / kBlockTokens + 1;
  const int stages = (n_blk + kStBlk - 1) / kStBlk;
  const int32_t* bt = block_table + (int64_t)s * max_blocks;

  // This wave's column tiles; padded columns repeat the tile's last row and
  // are never stored.
  const int w_row0 = row_begin + rg * 16 * COLS;
  const int w_kmax = w_row0 < row_end ? positions[min(row_end, w_row0 + 16 * COLS) - 1] : -1;
  // Stages whose keys all precede the wave's first row need no causal mask.
  const int w_kmin = w_row0 < row_end ? positions[w_row0] : -1;
  int pos[COLS];
  bf16x8_t qf[COLS][4];
#pragma unroll
  for (int c = 0; c < COLS; ++c) {
    const int row = min(w_row0 + 16 * c + c16, row_end - 1);
    pos[c] = positions[row];
    const bf16_t* qp = q + ((int64_t)row * Hq + h) * HD + j4 * 8;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      qf[c][t] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(qp + t * 32));
  }

  // The stage's blocks (clamped to the last block: a repeat that the causal
  // mask hides) x {K, V} tiles, four 1 KB pieces each; wave wv stages tiles
  // wv, wv + WAVES * KS, ... into LDS.
  auto issue = [&](int st) {
#pragma unroll
    for (int tt = wv; tt < 2 * kStBlk; tt += WAVES * KS) {
      const int kvsel = tt / kStBlk, bi = tt % kStBlk;
      const int blk = min(st * kStBlk + bi, n_blk - 1);
      const bf16_t* src = (kvsel ? v_cache : k_cache) +
                          ((int64_t)bt[blk] * Hkv + g) * kTileElems + lane * 8;
      bf16_t* dst = (kvsel ? v_slot(st) : k_slot(st)) + bi * kTileElems;
#pragma unroll
      for (int pc = 0; pc < 4; ++pc)
        __builtin_amdgcn_global_load_lds(src + pc * 512, (lds_void_t*)(dst + pc * 512), 16, 0,
                                         0);
    }
  };

  // l: the row sums of P, accumulated by an MFMA against an all-ones V^T
  // operand (every element of it holds the column's sum).
  float m[COLS];
  f32x4_t l[COLS];
  f32x4_t acc[COLS][8];
  const bf16x8_t ones =
      __builtin_bit_cast(bf16x8_t, u32x4_t{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u});
#pragma unroll
  for (int c = 0; c < COLS; ++c) {
    m[c] = -INFINITY;
    l[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int c = 0; c < COLS; ++c)
#pragma unroll
    for (int n = 0; n < 8; ++n) acc[c][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // V^T operands of a block pair: this lane's 16-byte chunk of piece pc of a
  // V tile holds 4 tokens of dim h, then the same 4 tokens of dim h + 16;
  // each 8-byte half is read from LDS straight into its place in the operand
  // (dims h: va, dims h + 16: vb; the pair's first block in the low half).
  bf16x8_t va[4], vb[4];
  auto read_v = [&](const bf16_t* vl, int pair) {
    const bf16_t* b0 = vl + 2 * pair * kTileElems;
#pragma unroll
    for (int pc = 0; pc < 4; ++pc) {
      const u32x2_t a0 = lds_read8(b0 + pc * 512);
      const u32x2_t a1 = lds_read8(b0 + kTileElems + pc * 512);
      const u32x2_t c0 = lds_read8(b0 + pc * 512 + 4);
      const u32x2_t c1 = lds_read8(b0 + kTileElems + pc * 512 + 4);
      va[pc] = __builtin_bit_cast(bf16x8_t, u32x4_t{a0.x, a0.y, a1.x, a1.y});
      vb[pc] = __builtin_bit_cast(bf16x8_t, u32x4_t{c0.x, c0.y, c1.x, c1.y});
    }
  };
  // P^T of the wave's 64 keys, packed as two 32-key operands.
  u32x4_t pk[COLS][2];
  // O^T += V^T P^T over the two block pairs; l += 1^T P^T. The first pair's
  // V^T operands are already in va / vb.
  auto pv = [&](const bf16_t* vl) {
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      if (pp == 1) read_v(vl, 1);
#pragma unroll
      for (int c = 0; c < COLS; ++c)
        l[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            ones, __builtin_bit_cast(bf16x8_t, pk[c][pp]), l[c], 0, 0, 0);
#pragma unroll
      for (int pc = 0; pc < 4; ++pc) {
#pragma unroll
        for (int c = 0; c < COLS; ++c) {
          const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, pk[c][pp]);
          acc[c][2 * pc] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[pc], pb, acc[c][2 * pc], 0, 0, 0);
          acc[c][2 * pc + 1] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb[pc], pb, acc[c][2 * pc + 1], 0, 0, 0);
        }
      }
    }
  };

  issue(0);
  __syncthreads();
  for (int st = 0; st < stages; ++st) {
    if (st + 1 < stages) issue(st + 1);
    // First key block of this wave's share of the stage.
    const int blk0 = st * kStBlk + kh * kPfBlk;
    const bool active = blk0 * kBlockTokens <= w_kmax;
    const bf16_t* vl = v_slot(st) + kh * kPfBlk * kTileElems + lane * 8;
    if (active) {
      const bf16_t* kl = k_slot(st) + kh * kPfBlk * kTileElems + lane * 8;
      // Scores of the stage's 4 blocks for both column tiles; the next
      // block's K fragments are read while the current block's MFMAs run.
      f32x4_t sc[COLS][kPfBlk];
      u32x4_t kfr[2][4];
#pragma unroll
      for (int pc = 0; pc < 4; ++pc) kfr[0][pc] = *(const u32x4_t*)(kl + pc * 512);
#pragma unroll
      for (int i = 0; i < kPfBlk; ++i) {
        if (i + 1 < kPfBlk) {
#pragma unroll
          for (int pc = 0; pc < 4; ++pc)
            kfr[(i + 1) & 1][pc] = *(const u32x4_t*)(kl + (i + 1) * kTileElems + pc * 512);
        }
#pragma unroll
        for (int c = 0; c < COLS; ++c) {
          f32x4_t a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int pc = 0; pc < 4; ++pc)
            a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, kfr[i & 1][pc]), qf[c][pc], a, 0, 0, 0);
          sc[c][i] = a;
        }
      }
      const bool unmasked = (blk0 + kPfBlk) * kBlockTokens - 1 <= w_kmin;
      read_v(vl, 0);
      // Online softmax, once per 64 keys (log2 domain: p = 2^(s*scale - m)).
      // Stages wholly before the wave's first row skip the causal mask.
#pragma unroll
      for (int c = 0; c < COLS; ++c) {
        float mx = -INFINITY;
        if (unmasked) {
#pragma unroll
          for (int i = 0; i < kPfBlk; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[c][i][r]);
        } else {
#pragma unroll
          for (int i = 0; i < kPfBlk; ++i) {
            const int tok0 = (blk0 + i) * kBlockTokens + j4 * 4;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              // Keys after the row's position score -inf: 2^-inf = 0 below.
              if (tok0 + r > pos[c]) sc[c][i][r] = -INFINITY;
              mx = fmaxf(mx, sc[c][i][r]);
            }
          }
        }
        mx = col_max4(mx) * scale_log2;
        // Stage 0 of key set 0 always holds key 0, so there mx is finite and
        // the first stage sets the max. Another key set can meet a column
        // whose keys are all masked (mx = -inf) and keeps m = -inf for it;
        // its exponents are then taken against 0 (2^-inf = 0, so p and alpha
        // are 0 and the still-zero state stays zero).
        const float m_new = mx > m[c] + kPfLazy ? mx : m[c];
        const float m_ref = (KS > 1 && m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m[c] - m_ref);
        uint32_t pw[kPfBlk][2];
#pragma unroll
        for (int i = 0; i < kPfBlk; ++i) {
          float pr[4];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            pr[r] = __builtin_amdgcn_exp2f(fmaf(sc[c][i][r], scale_log2, -m_ref));
          pw[i][0] = pack_bf16x2(pr[0], pr[1]);
          pw[i][1] = pack_bf16x2(pr[2], pr[3]);
        }
        m[c] = m_new;
        // alpha is exactly 1 for a column whose max was kept: rescale only
        // when some column's moved (multiplying by 1 would change nothing).
        if (__ballot(alpha != 1.f) != 0) {
#pragma unroll
          for (int n = 0; n < 8; ++n) acc[c][n] = acc[c][n] * alpha;
          l[c] = l[c] * alpha;
        }
#pragma unroll
        for (int pp = 0; pp < 2; ++pp)
          pk[c][pp] = u32x4_t{pw[2 * pp][0], pw[2 * pp][1], pw[2 * pp + 1][0], pw[2 * pp + 1][1]};
      }
      pv(vl);
    }
    __syncthreads();  // stage st+1 landed; buffer st is free for stage st+2
  }

  if constexpr (KS > 1) {
    // Key set 1 hands (m, l, O^T) of its columns to key set 0 through the
    // now free LDS ([row group][column tile][34 values][64 lanes] floats),
    // which adds them in: O = O_0 2^(m_0 - M) + O_1 2^(m_1 - M), likewise l,
    // with M = max(m_0, m_1). m_0 is finite (key 0), so a column that set 1
    // never saw (m_1 = -inf) takes weight 0 from it.
    constexpr int kVals = 8 * 4 + 2;
    static_assert(WAVES * COLS * kVals * 64 * 4 <= (int)sizeof(kv), "merge fits the K/V buffers");
    float* xs = reinterpret_cast<float*>(kv);
    if (kh == 1) {
#pragma unroll
      for (int c = 0; c < COLS; ++c) {
        float* d = xs + (rg * COLS + c) * kVals * 64 + lane;
#pragma unroll
        for (int n = 0; n < 8; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) d[(n * 4 + r) * 64] = acc[c][n][r];
        d[32 * 64] = m[c];
        d[33 * 64] = l[c][0];
      }
    }
    __syncthreads();
    if (kh == 1) return;
#pragma unroll
    for (int c = 0; c < COLS; ++c) {
      const float* d = xs + (rg * COLS + c) * kVals * 64 + lane;
      const float m1 = d[32 * 64], l1 = d[33 * 64];
      const float mm = fmaxf(m[c], m1);
      const float f0 = __builtin_amdgcn_exp2f(m[c] - mm), f1 = __builtin_amdgcn_exp2f(m1 - mm);
#pragma unroll
      for (int n = 0; n < 8; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[c][n][r] = acc[c][n][r] * f0 + d[(n * 4 + r) * 64] * f1;
      l[c][0] = l[c][0] * f0 + l1 * f1;
    }
  }

  // The output [rows][Hq * 128] is the O projection's A operand, written in
  // tile order (four columns from a multiple of 4 are contiguous there).
#pragma unroll
  for (int c = 0; c < COLS; ++c) {
    const int row = w_row0 + 16 * c + c16;
    const float inv = 1.0f / l[c][0];
    if (row < row_end) {
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        const uint32_t lo = pack_bf16x2(acc[c][n][0] * inv, acc[c][n][1] * inv);
        const uint32_t hi = pack_bf16x2(acc[c][n][2] * inv, acc[c][n][3] * inv);
        *(u32x2_t*)(o + tile_off(row, h * HD + n * 16 + j4 * 4, Hq * HD)) = u32x2_t{lo, hi};
      }
    }
  }
}

// ---------------------------------------------------------------- fp32 path
__global__ __launch_bounds__(64) void attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k_cache,
    const float* __restrict__ v_cache, const int32_t* __restrict__ block_table, int max_blocks,
    const int32_t* __restrict__ ctx_lens, const int32_t* __restrict__ positions,
    const int32_t* __restrict__ seq_starts, int n_seqs, int Hq, int Hkv, int hd,
    float* __restrict__ o) {
  const int i = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int s = row_to_seq(seq_starts, n_seqs, i);
  const int g = h / (Hq / Hkv);
  const int n = min(ctx_lens[s], positions[i] + 1);
  const float scale = 1.0f / sqrtf((float)hd);
  constexpr int kMaxPer = 4;  // hd <= 256
  float qv[kMaxPer], acc[kMaxPer];
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int e = lane + u * 64;
    qv[u] = e < hd ? q[((int64_t)i * Hq + h) * hd + e] : 0.f;
    acc[u] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int32_t* bt = block_table + (int64_t)s * max_blocks;
  for (int t = 0; t < n; ++t) {
    const int64_t blk = bt[t / kBlockTokens];
    const int slot = t % kBlockTokens;
    const float* kt = k_cache + (blk * Hkv + g) * kBlockTokens * hd;
    const float* vt = v_cache + (blk * Hkv + g) * kBlockTokens * hd;
    float d = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      const int e = lane + u * 64;
      if (e < hd) d = fmaf(qv[u], kt[k_tile_offset(slot, e)], d);
    }
    const float z = wave_sum(d) * scale;
    const float m_new = fmaxf(m, z);
    const float alpha = expf(m - m_new), p = expf(z - m_new);
    l = l * alpha + p;
    m = m_new;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      const int e = lane + u * 64;
      if (e < hd)
        acc[u] = acc[u] * alpha + p * vt[v_tile_offset(slot, e)];
    }
  }
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int e = lane + u * 64;
    if (e < hd) o[((int64_t)i * Hq + h) * hd + e] = n > 0 ? acc[u] / l : 0.f;
  }
}

}  // namespace

int decode_max_splits(int max_blocks_per_seq) {
  return (max_blocks_per_seq * kBlockTokens + kDecodeSplit - 1) / kDecodeSplit;
}

// The merge kernel keeps two floats per partition in dynamic LDS, within the
// 64 KB a launch gets without an opt-in (its static LDS is 8 bytes).
bool attn_combine_fits(int max_splits) {
  return max_splits >= 1 && (int64_t)max_splits * 2 * sizeof(float) <= 65536 - 64;
}

hipError_t launch_attn_decode_bf16(const uint16_t* q, const uint16_t* k_cache,
                                   const uint16_t* v_cache, const int32_t* block_table,
                                   int max_blocks, const int32_t* ctx_lens,
                                   const int32_t* positions, const int32_t* split_off,
                                   int n_seqs, int Hq, int Hkv, float* part_o, float* part_ml,
                                   int max_splits, int num_cus, hipStream_t st) {
  if (n_seqs <= 0) return hipSuccess;
  if (num_cus <= 0) return hipErrorInvalidValue;
  const float scale_log2 = kLog2e / sqrtf((float)HD);
  // Two resident workgroups per CU (at most 128 registers per lane and 68 KB
  // of LDS each): a persistent grid of two per CU, never more than the work.
  const int64_t work_bound = (int64_t)n_seqs * max_splits * Hkv;
  const int grid = (int)(work_bound < 2 * num_cus ? work_bound : 2 * num_cus);
  COCO_LAUNCH(attn_decode_kernel, dim3(grid), dim3(kDecWaves * 64), 0, st, q, k_cache,
                     v_cache, block_table, max_blocks, ctx_lens, positions, split_off, n_seqs,
                     Hq, Hkv, part_o, part_ml, max_splits, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_combine_bf16(const float* part_o, const float* part_ml,
                                    const int32_t* ctx_lens, const int32_t* positions,
                                    int n_seqs, int Hq, int max_splits, uint16_t* o, bool tiled,
                                    hipStream_t st) {
  if (n_seqs <= 0) return hipSuccess;
  COCO_LAUNCH(attn_combine_kernel, dim3(Hq, n_seqs), dim3(HD),
                     2 * max_splits * sizeof(float), st, part_o, part_ml, ctx_lens, positions,
                     Hq, max_splits, o, tiled);
  return hipGetLastError();
}

hipError_t launch_attn_prefill_bf16(const uint16_t* q, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const int32_t* block_table,
                                    int max_blocks, const int32_t* ctx_lens,
                                    const int32_t* positions, const int32_t* seq_starts,
                                    int n_seqs, int n_rows, int Hq, int Hkv, uint16_t* o,
                                    hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  const float scale_log2 = kLog2e / sqrtf((float)HD);
  // Upper bound on the per-sequence 128-row tiles; workgroups past the last
  // tile return at once.
  const int64_t tiles = (n_rows + kPfRows - 1) / kPfRows + n_seqs;
  if (tiles * Hq > 0x7fffffff) return hipErrorInvalidValue;
  COCO_LAUNCH((attn_prefill_kernel<kPfLaunchWaves, 8 / kPfLaunchWaves, kPfKeySets>),
                     dim3((unsigned)(tiles * Hq)), dim3(kPfLaunchWaves * kPfKeySets * 64), 0, st, q,
                     k_cache, v_cache, block_table, max_blocks, ctx_lens, positions, seq_starts,
                     n_seqs, Hq, Hkv, scale_log2, o);
  return hipGetLastError();
}

hipError_t launch_attn_f32(const float* q, const float* k_cache, const float* v_cache,
                           const int32_t* block_table, int max_blocks, const int32_t* ctx_lens,
                           const int32_t* positions, const int32_t* seq_starts, int n_seqs,
                           int n_rows, int Hq, int Hkv, int hd, float* o, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  COCO_LAUNCH(attn_f32_kernel, dim3(n_rows, Hq), dim3(64), 0, st, q, k_cache, v_cache,
                     block_table, max_blocks, ctx_lens, positions, seq_starts, n_seqs, Hq, Hkv,
                     hd, o);
  return hipGetLastError();
}

}  // namespace coco
