/*
 * coco.h -- C ABI of the layer-replica hot path on one MI355X (gfx950).
 *
 * A layer replica (Sec. 3.1 of the paper, replication mechanism) holds a full
 * copy of the weights of one or more consecutive decoder layers plus its own
 * partition of the paged key/value cache, and runs the unchanged layer on its
 * sub-batch: the rows of the in-flight batch it was given. The library does
 * exactly that step on one GPU:
 *
 *   gather rows -> RMSNorm -> QKV projection -> RoPE + KV append ->
 *   paged GQA attention -> O projection + residual -> RMSNorm ->
 *   SwiGLU MLP + residual -> scatter rows
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers. Every data pointer is a DEVICE pointer into memory the caller
 *   owns (weights, caches, hidden buffer, index arrays). The library borrows
 *   caches, RMSNorm gains and (fp32) weight matrices for the handle's
 *   lifetime and the rest for the call. dtype COCO_BF16: coco_layer_init
 *   copies the four weight matrices of every layer into library memory in
 *   tile order (below) and never reads the caller's matrices again; the
 *   caller may free or overwrite them once init has returned.
 *   The library owns that copy and its workspace, both allocated once in
 *   coco_layer_init and sized by the config (the paper's persistent memory
 *   pool with fixed addresses, Sec. 5.2, CUDA-graph compatibility): per-row
 *   activations and split-K partials for max_rows rows, the decode attention
 *   partials, and (bf16) a RoPE cos/sin table of max_blocks_per_seq * 16
 *   positions * head_dim * 4 bytes.
 * Streams. `stream` is a hipStream_t (NULL = the null stream). Work is
 *   enqueued on it; calls return without synchronising, never allocate, and
 *   keep every address fixed, so a call can be captured in a HIP graph --
 *   except with validation switched on, which copies index arrays to the host.
 * Element types. dtype COCO_BF16: weights, hidden, caches and k/v inputs are
 *   bfloat16 (uint16 bit patterns); accumulation and softmax are fp32.
 *   dtype COCO_F32: all of those are float32.
 * Errors. A negative return is an error; coco_last_error() gives a message
 *   (thread-local). Host-checkable faults return COCO_EINVAL before anything
 *   is enqueued; a failed launch returns COCO_EHIP. Device-side contents of
 *   index arrays are checked only in validation mode (coco_layer_set_validate).
 * Threads. A handle is not thread-safe; calls that overlap on one handle
 *   (including from different streams) race on its workspace.
 *
 * Layouts
 * -------
 * Weights of one layer, nn.Linear layout ([out][in], row-major):
 *   w_qkv     [(Hq + 2*Hkv) * hd][d]   query heads, then key heads, then value
 *                                      heads, hd rows each
 *   w_o       [d][Hq * hd]
 *   w_gate_up [2*F][d]                 F gate rows, then F up rows
 *   w_down    [d][F]
 *   gamma_attn, gamma_mlp [d]          RMSNorm gains
 * (bf16) The library's copy of a weight matrix [N][K] is in tile order: the
 *   1 KB block (n / 16) * (K / 32) + k / 32 holds rows 16 (n / 16) .. + 15 and
 *   k 32 (k / 32) .. + 31 as 64 chunks of 8 consecutive k, chunk
 *   ((k % 32) / 8) * 16 + n % 16 -- one MFMA operand fragment per 16 rows x
 *   32 k, read by one contiguous 1 KB load.
 * Paged cache of one layer, with block size B = 16 tokens:
 *   k_cache, v_cache [num_blocks][Hkv][B * hd]: one tile of B tokens x hd
 *   dimensions per (block, kv head), in MFMA operand order. Inside a tile,
 *   token slot t (0..15) and dimension h live at
 *     K: ((h/32)*64 + ((h%32)/8)*16 + t)*8 + h%8
 *     V: (((h/32)*64 + (t/4)*16 + h%16)*2 + (h/16)%2)*4 + t%4
 *   (hd must be a multiple of 32). Token t of sequence s lives in block
 *   block_table[s][t / 16], slot t % 16. Keys are stored after rotation
 *   (RoPE), values as projected.
 * Batch arrays (int32, device):
 *   row_idx[n_rows]        hidden row of each call row; distinct, < hidden_rows
 *   positions[n_rows]      absolute position of each call row's token
 *   seq_starts[n_seqs+1]   prefill: call rows of sequence s are
 *                          seq_starts[s] .. seq_starts[s+1]-1, in position
 *                          order. NULL = decode: call row i is sequence i
 *                          (then n_seqs == n_rows).
 *   block_table[n_seqs][max_blocks_per_seq]   physical block ids, -1 unused
 *   ctx_lens[n_seqs]       cached tokens of sequence s once this call's tokens
 *                          are appended (decode, normally positions[i] + 1)
 * Every token attends to the cached keys of its own sequence at positions
 * 0 .. its own position (causal), its own key included: a decode row i
 * attends min(ctx_lens[i], positions[i] + 1) keys, so cached tokens past its
 * position (positions[i] < ctx_lens[i] - 1) are not read.
 */
#ifndef COCO_H
#define COCO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct coco_layer* coco_layer_t;
typedef void* coco_stream_t; /* hipStream_t */

enum {
  COCO_OK = 0,
  COCO_EINVAL = -1, /* bad argument or unsupported configuration */
  COCO_ENOMEM = -2, /* workspace allocation failed (init only) */
  COCO_EHIP = -3,   /* a HIP runtime call or kernel launch failed */
  COCO_ESTATE = -4  /* handle unusable (e.g. destroyed, or a previous HIP fault) */
};

enum { COCO_BF16 = 0, COCO_F32 = 1 };

typedef struct {
  int32_t d_model;            /* d */
  int32_t n_q_heads;          /* Hq */
  int32_t n_kv_heads;         /* Hkv; Hq % Hkv == 0 */
  int32_t head_dim;           /* hd; 128 for COCO_BF16, multiple of 32 <= 256 for COCO_F32 */
  int32_t d_ffn;              /* F */
  int32_t n_layers;           /* layers held by this handle */
  int32_t dtype;              /* COCO_BF16 or COCO_F32 */
  int32_t block_size;         /* must be 16 */
  int32_t max_rows;           /* largest n_rows of any call (decode rows or prefill tokens) */
  int32_t max_seqs;           /* largest n_seqs of any call */
  int32_t max_blocks_per_seq; /* row stride of block_table (<= 2^24; bf16: <= 130944,
                                 the decode partition merge's limit) */
  float rope_theta;           /* RoPE base theta */
  float rms_eps;              /* RMSNorm epsilon */
} coco_layer_config;

typedef struct {
  const void* w_qkv;
  const void* w_o;
  const void* w_gate_up;
  const void* w_down;
  const void* gamma_attn;
  const void* gamma_mlp;
  void* k_cache;
  void* v_cache;
  int64_t num_blocks; /* blocks in this layer's k_cache and v_cache */
} coco_layer_weights;

/* Create a replica handle for n_layers consecutive layers (Sec. 3.1: the
 * replicated unit is a span of consecutive layers). `layers` points to
 * cfg->n_layers host structs of device pointers; they are copied. Allocates
 * the workspace on the current HIP device and, for bf16, the tile-order copy
 * of the weight matrices (the sum of their sizes over the handle's layers),
 * which it writes before returning (synchronising the device). Returns
 * COCO_EINVAL for an unsupported shape (bf16: head_dim != 128, Hq/Hkv > 16, d,
 * F or Hq*hd not multiples of 128), COCO_ENOMEM if the workspace or the
 * weight copy does not fit. */
int coco_layer_init(const coco_layer_config* cfg, const coco_layer_weights* layers,
                    coco_layer_t* out);

/* Release the workspace, the weight copy and the handle. First waits for the
 * handle's last call made outside graph capture to finish (an event recorded behind the
 * last kernel of every such call; calls on one handle are ordered, since they
 * share the workspace), not for other work on the device. A graph captured
 * from the handle's calls must not run after this. NULL is ignored. */
void coco_layer_destroy(coco_layer_t h);

/* Message of the last failed call on this thread ("" if none). */
const char* coco_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int coco_version(void);

/* Switch device-side argument validation on (1) or off (0). When on, every
 * forward/append copies its index arrays to the host, synchronising the
 * stream, and rejects duplicate or out-of-range row_idx, non-increasing
 * positions within a sequence, positions >= ctx_lens, ctx_lens beyond the
 * block table, and block ids outside [0, num_blocks) with COCO_EINVAL before
 * launching. Off by default. */
int coco_layer_set_validate(coco_layer_t h, int32_t on);

/* Write n_tok tokens of keys and values into layer `layer`'s paged cache
 * (Sec. 3.1: each replica appends key/value entries to its own partition).
 * k, v: [n_tok][Hkv][hd] in the handle's dtype, k already rotated.
 * seq_idx[n_tok]: sequence of each token (row of block_table, < n_seqs).
 * positions[n_tok]: position of each token. A bit copy: the stored values
 * equal the inputs bit for bit. Tokens must name distinct (sequence,
 * position) pairs. */
int coco_kv_append(coco_layer_t h, int32_t layer, const void* k, const void* v,
                   const int32_t* seq_idx, const int32_t* positions, int32_t n_tok,
                   const int32_t* block_table, int32_t n_seqs, coco_stream_t stream);

/* One decoder layer on the call rows of `hidden` ([hidden_rows][d], updated
 * in place): rows named in row_idx receive the layer output, every other row
 * is left untouched (Sec. 3.1: the replica processes its sub-batch and the
 * outputs are gathered back on the batch axis). The call's keys and values
 * are appended to the layer's cache before attention. n_rows == 0 is a no-op.
 * Results do not depend on which other rows share the call: any partition of
 * a decode batch, and any request-aligned partition of a prefill batch, gives
 * output rows and cache bytes identical bit for bit to the whole batch
 * (Sec. 5.2: outputs bit-wise consistent with the baseline). */
int coco_layer_forward(coco_layer_t h, int32_t layer, void* hidden, int64_t hidden_rows,
                       const int32_t* row_idx, int32_t n_rows, const int32_t* positions,
                       const int32_t* seq_starts, int32_t n_seqs,
                       const int32_t* block_table, const int32_t* ctx_lens,
                       coco_stream_t stream);

/* Layers first_layer .. first_layer+n_layers-1 as one replicated segment
 * (Sec. 3.1: consecutive layers are replicated as a unit, activations stay in
 * local memory and transfers happen only at the segment boundaries): one
 * gather, every layer on the resident rows, one scatter. Between layers the
 * rows are held in the handle's dtype, so the result equals n_layers
 * successive coco_layer_forward calls bit for bit. */
int coco_layer_span_forward(coco_layer_t h, int32_t first_layer, int32_t n_layers,
                            void* hidden, int64_t hidden_rows, const int32_t* row_idx,
                            int32_t n_rows, const int32_t* positions,
                            const int32_t* seq_starts, int32_t n_seqs,
                            const int32_t* block_table, const int32_t* ctx_lens,
                            coco_stream_t stream);

/* For callers that cannot allocate device memory at call time (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same call as coco_layer_forward, with the same results bit for bit, but
 * its per-call buffers (activations, split-K partials, decode attention
 * partials and work list) come from a static array of 64 MiB that every GPU
 * the library runs on holds from module load until the process ends, sized
 * for this call's rows instead of the handle's max_rows. The call itself
 * allocates nothing, host or device. Its address is looked up once per
 * device by coco_layer_init. Returns COCO_EINVAL, before anything is
 * enqueued, when the call's buffers exceed 64 MiB (a batch-64 decode of the
 * 8B-shaped layer with 8k-token block tables takes about 49 MB; a
 * 2048-token prefill of the 32B-shaped layer does not fit). All such calls
 * on one GPU share the
 * array, whatever their handle: calls that overlap on one GPU (other
 * streams, other threads, other handles) race on it. The array keeps the
 * last call's contents; no part of it needs to start at zero. Validation
 * mode is not run by this entry point, and coco_layer_workspace shows the
 * handle's own workspace, not this array. */
int coco_layer_forward_noalloc(coco_layer_t h, int32_t layer, void* hidden, int64_t hidden_rows,
                               const int32_t* row_idx, int32_t n_rows, const int32_t* positions,
                               const int32_t* seq_starts, int32_t n_seqs,
                               const int32_t* block_table, const int32_t* ctx_lens,
                               coco_stream_t stream);

/* Copy an intermediate buffer of the last call into `dst` (device memory of
 * at least dst_bytes bytes), for inspection by tests. which = COCO_WS_*;
 * row i holds call row i of the last layer run, row-major. Copies
 * min(dst_bytes, buffer size) bytes on `stream`. (A bf16 prefill call keeps
 * H, O, H2 and U, the A operands of its four projections, in the tile order
 * of the weight copies, 16 rows x 32 columns per 1 KB block; this copy puts
 * the call's rows back in row-major order.) */
enum {
  COCO_WS_X = 0,  /* layer input rows, [max_rows][d], dtype (written for the
                     second and later layers of a span; the first layer reads
                     its rows from the hidden buffer) */
  COCO_WS_H = 1,  /* RMSNorm_1 output, [max_rows][d], dtype (prefill and
                     fp32 calls; bf16 decode folds RMSNorm_1 into the QKV
                     projection and never writes it) */
  COCO_WS_Q = 2,  /* rotated queries, [max_rows][Hq*hd], dtype */
  COCO_WS_O = 3,  /* attention output, [max_rows][Hq*hd], dtype */
  COCO_WS_X1 = 4, /* residual after the O projection, [max_rows][d], fp32 */
  COCO_WS_H2 = 5, /* RMSNorm_2 output, [max_rows][d], dtype (bf16 prefill
                     with d a multiple of 256 folds the row's 1/rms into the
                     gate/up projection and holds x1 * gamma_2 here) */
  COCO_WS_U = 6   /* SwiGLU activation, [max_rows][F], dtype */
};
int coco_layer_workspace(coco_layer_t h, int32_t which, void* dst, int64_t dst_bytes,
                         coco_stream_t stream);

/* Per-kernel timing for benchmarks (calls of any handle are unaffected while
 * it is off). When on, every kernel launched by coco_layer_forward /
 * coco_layer_span_forward on this handle is launched with a pair of HIP events
 * (hipExtLaunchKernelGGL) that the runtime timestamps at the kernel's own
 * start and end, from a pool of events created here (so switching it on
 * allocates; timed calls themselves do not). Switch it off before capturing
 * calls into a HIP graph. */
enum {
  COCO_K_GATHER_NORM = 0,    /* gather + RMSNorm_1 (or RMSNorm_1 inside a span) */
  COCO_K_GEMM_QKV = 1,       /* QKV projection */
  COCO_K_QKV_EPILOGUE = 2,   /* split-K sum + RoPE + cache append */
  COCO_K_ATTENTION = 3,      /* paged attention (decode partitions or prefill) */
  COCO_K_ATTN_COMBINE = 4,   /* decode partition merge */
  COCO_K_GEMM_O = 5,         /* O projection */
  COCO_K_RESIDUAL_NORM = 6,  /* residual + RMSNorm_2 */
  COCO_K_GEMM_GATE_UP = 7,   /* gate/up projection */
  COCO_K_SWIGLU = 8,         /* SwiGLU */
  COCO_K_GEMM_DOWN = 9,      /* down projection */
  COCO_K_RESIDUAL_SCATTER = 10, /* residual + scatter */
  COCO_K_COUNT = 11
};
int coco_layer_set_timing(coco_layer_t h, int32_t on);

/* Sum of the event-measured durations (milliseconds) and the number of
 * launches of each kernel kind since timing was switched on or last read;
 * ms and launches hold n_kinds entries (<= COCO_K_COUNT). Synchronises with
 * the recorded events, then resets the sums. Returns COCO_ESTATE if more
 * launches were made than the pool holds (4096 per read). */
int coco_layer_read_timing(coco_layer_t h, double* ms, int64_t* launches, int32_t n_kinds);

/* Peak probes for benchmarks (not part of the layer): the rates this GPU
 * sustains, against which measured kernels are quoted next to the published
 * peaks. Both enqueue one kernel on `stream` and return COCO_EINVAL for bad
 * arguments or COCO_EHIP for a failed launch (without a coco_last_error
 * message); the caller times them with events on the same stream.
 *
 * coco_probe_read: reads `bytes` (a multiple of 16, 16-byte aligned) of device
 * memory at `buf` once, as 16-byte vector loads spread over `blocks`
 * 256-thread workgroups with a grid-wide stride; variant 0: four loads in
 * flight per thread, 1: eight, 2: eight non-temporal. Writes one 32-bit word
 * per workgroup to `out` (device, >= 4 * blocks bytes).
 *
 * coco_probe_mfma_bf16: `blocks` workgroups of four waves, each wave running
 * `iters` rounds (a multiple of 8) of `chains` (4 or 8) independent
 * v_mfma_f32_32x32x16_bf16 chains on register operands; writes one float per
 * wave to `out` (device, >= 16 * blocks bytes) and the dense flop count of
 * the launch to *flops (host). operands 0: the same small constants in every
 * instruction; 1: random bf16 values with random signs and magnitudes in
 * [0.5, 2), eight operand sets per lane taken in turn, so consecutive
 * instructions of a chain see different data (the rate under the power draw
 * of data like a GEMM's). */
int coco_probe_read(const void* buf, int64_t bytes, void* out, int32_t blocks, int32_t variant,
                    coco_stream_t stream);
int coco_probe_mfma_bf16(int64_t iters, void* out, int32_t blocks, int32_t chains,
                         int32_t operands, double* flops, coco_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* COCO_H */
