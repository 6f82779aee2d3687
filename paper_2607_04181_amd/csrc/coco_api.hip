// C ABI of the layer-replica hot path: handle, workspace, argument checks and
// the launch sequence of one decoder layer / one span of layers.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <type_traits>

#include <mutex>
#include <vector>

#include "../../include/coco.h"
#include "common.h"
#include "kernels.h"

using namespace coco;

namespace {

// Message of the last failure on this thread (a fixed buffer: reporting an
// error allocates nothing).
thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

#define HIPCHK(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return fail(COCO_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

}  // namespace

// Per-call buffers of the launch sequence, carved out of one region (the
// handle's workspace, or the static scratch array of the no-alloc entry
// point).
struct Work {
  void *x = nullptr, *h = nullptr, *q = nullptr, *o = nullptr, *h2 = nullptr, *u = nullptr;
  float *x1 = nullptr, *part = nullptr, *attn_o = nullptr, *attn_ml = nullptr;
  // Row sums of squares: per K-slice (decode QKV with RMSNorm_1 folded in) or
  // per 256-column tile (prefill O projection with RMSNorm_2 folded in).
  float* ss = nullptr;
  int32_t* split_off = nullptr;  // decode attention work list
  int32_t* row_info = nullptr;   // prefill row slots [rows][2] (position, cache block)
};

struct coco_layer {
  coco_layer_config cfg;
  std::vector<coco_layer_weights> layers;
  int device = 0;
  int num_cus = 0;  // compute units of `device` (persistent grid sizes)
  bool validate = false;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  // bf16: the library's tile-order copies of every layer's four weight
  // matrices (layers[l].w_* point into it after init).
  char* packed = nullptr;
  size_t packed_bytes = 0;
  Work w;  // the workspace's per-call buffers, sized for max_rows
  double* inv_freq = nullptr;
  float* rope = nullptr;  // RoPE table [rope_rows][head_dim / 2] (cos, sin)
  int rope_rows = 0;      // positions the configuration admits
  size_t act_rows_bytes[7] = {};
  int max_splits = 0;
  int dec_rows = 0;
  // Which of the last regular call's activations h, o, h2, u are in tile
  // order (act_layout), read back row-major by coco_layer_workspace, and
  // that call's rows.
  bool ws_tiled[7] = {};
  int last_rows = 0;
  // Per-kernel timing (benchmark mode).
  bool timing = false;
  std::vector<hipEvent_t> ev;  // pairs: start, stop
  std::vector<int> ev_kind;    // kind of each recorded pair
  bool ev_overflow = false;
  hipStream_t ev_stream = nullptr;
  // Recorded at the end of every call made outside graph capture.
  hipEvent_t done = nullptr;
};

namespace coco {
LaunchEvents& launch_events() {
  thread_local LaunchEvents le;
  return le;
}
}  // namespace coco

namespace {

constexpr int kTimingPairs = 4096;

// Times the one kernel launched in its scope when timing is on: the launch
// timestamps the event pair at the kernel's own start and end. A scope that
// launches nothing (empty work) records an empty interval.
struct KernelTimer {
  coco_layer* H;
  int kind;
  int pair = -1;
  KernelTimer(coco_layer* h, int k, hipStream_t st) : H(h), kind(k) {
    if (!H->timing) return;
    const int n = (int)H->ev_kind.size();
    if (n >= kTimingPairs) {
      H->ev_overflow = true;
      return;
    }
    pair = n;
    H->ev_kind.push_back(kind);
    H->ev_stream = st;
    coco::launch_events() = coco::LaunchEvents{H->ev[2 * pair], H->ev[2 * pair + 1]};
  }
  ~KernelTimer() {
    if (pair < 0) return;
    coco::LaunchEvents& le = coco::launch_events();
    if (le.start != nullptr) {
      (void)hipEventRecord(le.start, H->ev_stream);
      (void)hipEventRecord(le.stop, H->ev_stream);
      le = coco::LaunchEvents{};
    }
  }
};

}  // namespace

namespace {

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

int elem_bytes(int dtype) { return dtype == COCO_BF16 ? 2 : 4; }

// Largest split count either GEMM path uses for (N, K).
int gemm_splits(const coco_layer_config& c, int N, int K) {
  if (c.dtype != COCO_BF16) return 1;
  const int a = skinny_plan(N, K).S, b = tile_splits(N, K);
  return a > b ? a : b;
}

// Lays out the per-call buffers for `rows` call rows and `dec_seqs` decode
// sequences from `base`, each piece 256-byte aligned, and returns the bytes
// they take (base == nullptr: sizes only; `w` may then be null).
size_t carve_work(const coco_layer_config& c, int64_t rows, int64_t dec_seqs, int max_splits,
                  char* base, Work* w) {
  const int eb = elem_bytes(c.dtype);
  const int64_t R = rows, d = c.d_model, F = c.d_ffn;
  const int64_t qd = (int64_t)c.n_q_heads * c.head_dim;
  const int64_t nqkv = (int64_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  int64_t part_elems = 0;
  const int64_t shapes[4][2] = {{nqkv, d}, {d, qd}, {2 * F, d}, {d, F}};
  for (auto& sh : shapes) {
    const int64_t e = (int64_t)gemm_splits(c, (int)sh[0], (int)sh[1]) * R * sh[0];
    if (e > part_elems) part_elems = e;
  }
  const bool bf = c.dtype == COCO_BF16;
  // The prefill GEMMs' A operands (h, o, h2, u) are in tile order, read in
  // whole 16-row groups: room for the rows rounded up to 16.
  const int64_t R16 = (R + 15) / 16 * 16;
  const size_t sizes[13] = {
      align256(R * d * eb),      // x
      align256(R16 * d * eb),    // h
      align256(R * qd * eb),     // q
      align256(R16 * qd * eb),   // o
      align256(R16 * d * eb),    // h2
      align256(R16 * F * eb),    // u
      align256(R * d * 4),     // x1
      align256(part_elems * 4),  // part
      bf ? align256((size_t)dec_seqs * c.n_q_heads * max_splits * 128 * 4) : 0,  // attn_o
      bf ? align256((size_t)dec_seqs * c.n_q_heads * max_splits * 2 * 4) : 0,    // attn_ml
      align256((size_t)(2 * dec_seqs + 2) * 4),  // split_off (decode attention work list)
      // ss: per-slice row sums of squares (decode QKV, at most 16 K-slices)
      // or per-column-tile ones (prefill O projection, at most 32 tiles)
      align256((size_t)32 * R * 4),
      align256(R * 8)};  // row_info
  size_t off[13], total = 0;
  for (int i = 0; i < 13; ++i) {
    off[i] = total;
    total += sizes[i];
  }
  if (base && w) {
    w->x = base + off[0];
    w->h = base + off[1];
    w->q = base + off[2];
    w->o = base + off[3];
    w->h2 = base + off[4];
    w->u = base + off[5];
    w->x1 = (float*)(base + off[6]);
    w->part = (float*)(base + off[7]);
    w->attn_o = (float*)(base + off[8]);
    w->attn_ml = (float*)(base + off[9]);
    w->split_off = (int32_t*)(base + off[10]);
    w->ss = (float*)(base + off[11]);
    w->row_info = (int32_t*)(base + off[12]);
  }
  return total;
}

int check_config(const coco_layer_config* c) {
  if (!c) return fail(COCO_EINVAL, "config is NULL");
  if (c->d_model <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->d_ffn <= 0 || c->n_layers <= 0 || c->max_rows <= 0 || c->max_seqs <= 0 ||
      c->max_blocks_per_seq <= 0)
    return fail(COCO_EINVAL, "config sizes must be positive");
  if (c->block_size != kBlockTokens) return fail(COCO_EINVAL, "block_size must be 16");
  if (c->max_blocks_per_seq > (1 << 24))
    return fail(COCO_EINVAL, "max_blocks_per_seq must be <= 2^24 (positions fit in int32)");
  if (c->n_q_heads % c->n_kv_heads) return fail(COCO_EINVAL, "n_q_heads %% n_kv_heads != 0");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f))
    return fail(COCO_EINVAL, "rms_eps must be >= 0 and rope_theta > 0");
  if (c->dtype == COCO_BF16) {
    if (c->head_dim != 128) return fail(COCO_EINVAL, "bf16 path needs head_dim == 128");
    if (c->n_q_heads / c->n_kv_heads > 16)
      return fail(COCO_EINVAL, "bf16 path needs n_q_heads / n_kv_heads <= 16");
    if (c->d_model % 128 || c->d_ffn % 128)
      return fail(COCO_EINVAL, "bf16 path needs d_model and d_ffn multiples of 128");
    if (c->d_model > 16384) return fail(COCO_EINVAL, "bf16 path needs d_model <= 16384");
    // The decode partition merge keeps two floats per 256-token partition in LDS.
    if (!attn_combine_fits(decode_max_splits(c->max_blocks_per_seq)))
      return fail(COCO_EINVAL,
                  "max_blocks_per_seq = %d: its %d decode partitions exceed what the partition "
                  "merge holds in LDS (max_blocks_per_seq <= %d)",
                  c->max_blocks_per_seq, decode_max_splits(c->max_blocks_per_seq),
                  (65536 - 64) / 8 * (kDecodeSplit / kBlockTokens));
  } else if (c->dtype == COCO_F32) {
    if (c->head_dim % 32 || c->head_dim > 256)
      return fail(COCO_EINVAL, "fp32 path needs head_dim a multiple of 32, <= 256");
    if (c->d_model % 4 || c->d_ffn % 4 || c->d_model > 16384)
      return fail(COCO_EINVAL, "fp32 path needs d_model, d_ffn multiples of 4, d_model <= 16384");
  } else {
    return fail(COCO_EINVAL, "unknown dtype %d", c->dtype);
  }
  return COCO_OK;
}

}  // namespace

// ----------------------------------------------------------------------------
// Static scratch of the no-alloc entry point (coco_layer_forward_noalloc).
// Every GPU the library runs on holds its own copy of this array from module
// load until the process ends. In host code `scratch` names a host-side
// stand-in, not a device address: the device address of the current device's
// copy comes from hipGetSymbolAddress, taken once per device in
// coco_layer_init and kept in g_scratch; only that address is ever passed to
// kernels.
// ----------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices] = {};

// With `dev` current: look up and keep this device's scratch address.
int scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices)
    return fail(COCO_EINVAL, "device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] != nullptr) return COCO_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || p == nullptr) {
    (void)hipGetLastError();
    return fail(COCO_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                hipGetErrorString(e));
  }
  g_scratch[dev] = (char*)p;
  return COCO_OK;
}

char* scratch_ptr(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch[dev];
}

}  // namespace

namespace {

// bf16: copy every layer's weight matrices into one library-owned buffer in
// tile order (the layout the bf16 GEMM kernels read) and point the handle's
// layer structs at the copies. The caller's matrices are not read again.
int pack_weights(coco_layer* H) {
  const coco_layer_config& c = H->cfg;
  if (c.dtype != COCO_BF16) return COCO_OK;
  const int64_t d = c.d_model, F = c.d_ffn, qd = (int64_t)c.n_q_heads * c.head_dim;
  const int64_t nqkv = qd + 2LL * c.n_kv_heads * c.head_dim;
  struct Mat {
    int64_t N, K;
  };
  const Mat mats[4] = {{nqkv, d}, {d, qd}, {2 * F, d}, {d, F}};
  size_t per_layer = 0;
  for (const Mat& m : mats) per_layer += align256((size_t)(m.N * m.K * 2));
  H->packed_bytes = per_layer * c.n_layers;
  if (hipMalloc((void**)&H->packed, H->packed_bytes) != hipSuccess) {
    (void)hipGetLastError();
    H->packed = nullptr;
    return fail(COCO_ENOMEM, "tile-order weight copies of %zu bytes do not fit", H->packed_bytes);
  }
  char* p = H->packed;
  for (int l = 0; l < c.n_layers; ++l) {
    coco_layer_weights& w = H->layers[l];
    const void** src[4] = {&w.w_qkv, &w.w_o, &w.w_gate_up, &w.w_down};
    for (int i = 0; i < 4; ++i) {
      if (launch_pack_tile_order((const uint16_t*)*src[i], (int)mats[i].N, (int)mats[i].K,
                                 (uint16_t*)p, nullptr) != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(H->packed);
        H->packed = nullptr;
        return fail(COCO_EHIP, "weight packing failed (layer %d)", l);
      }
      *src[i] = p;
      p += align256((size_t)(mats[i].N * mats[i].K * 2));
    }
  }
  if (hipDeviceSynchronize() != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(H->packed);
    H->packed = nullptr;
    return fail(COCO_EHIP, "weight packing failed");
  }
  return COCO_OK;
}

}  // namespace

extern "C" {

const char* coco_last_error(void) { return g_err; }

int coco_version(void) { return 100; }

int coco_layer_init(const coco_layer_config* cfg, const coco_layer_weights* layers,
                    coco_layer_t* out) {
  if (!out) return fail(COCO_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!layers) return fail(COCO_EINVAL, "layers is NULL");
  const coco_layer_config& c = *cfg;
  for (int l = 0; l < c.n_layers; ++l) {
    const coco_layer_weights& w = layers[l];
    if (!w.w_qkv || !w.w_o || !w.w_gate_up || !w.w_down || !w.gamma_attn || !w.gamma_mlp ||
        !w.k_cache || !w.v_cache)
      return fail(COCO_EINVAL, "layer %d has a NULL weight or cache pointer", l);
    if (w.num_blocks <= 0) return fail(COCO_EINVAL, "layer %d: num_blocks must be > 0", l);
    // The kernels read weights, gains and cache tiles with 16-byte vector loads.
    const void* ptrs[8] = {w.w_qkv, w.w_o, w.w_gate_up, w.w_down, w.gamma_attn, w.gamma_mlp,
                           w.k_cache, w.v_cache};
    for (const void* ptr : ptrs)
      if ((uintptr_t)ptr % 16) return fail(COCO_EINVAL, "layer %d: a weight or cache pointer is not 16-byte aligned", l);
  }

  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return fail(COCO_EHIP, "cannot query the current device");
  if ((rc = scratch_setup(dev))) return rc;
  coco_layer* H = new coco_layer();
  H->cfg = c;
  H->layers.assign(layers, layers + c.n_layers);
  H->device = dev;
  H->num_cus = cus;

  const int eb = elem_bytes(c.dtype);
  const int64_t R = c.max_rows, d = c.d_model, F = c.d_ffn;
  const int64_t qd = (int64_t)c.n_q_heads * c.head_dim;
  H->max_splits = decode_max_splits(c.max_blocks_per_seq);
  H->dec_rows = c.max_rows < c.max_seqs ? c.max_rows : c.max_seqs;

  // Per-call buffers for max_rows rows, then the handle's constants: RoPE
  // inverse frequencies and (bf16) the RoPE table of the fused prefill QKV
  // epilogue.
  H->rope_rows = c.dtype == COCO_BF16 ? c.max_blocks_per_seq * kBlockTokens : 0;
  const size_t work_bytes = carve_work(c, R, H->dec_rows, H->max_splits, nullptr, nullptr);
  const size_t freq_bytes = align256((size_t)(c.head_dim / 2) * 8);
  const size_t rope_bytes = align256((size_t)H->rope_rows * (c.head_dim / 2) * 8);
  H->ws_bytes = work_bytes + freq_bytes + rope_bytes;
  if (hipMalloc((void**)&H->ws, H->ws_bytes) != hipSuccess) {
    (void)hipGetLastError();
    const size_t want = H->ws_bytes;
    delete H;
    return fail(COCO_ENOMEM, "workspace of %zu bytes does not fit", want);
  }
  carve_work(c, R, H->dec_rows, H->max_splits, H->ws, &H->w);
  H->inv_freq = (double*)(H->ws + work_bytes);
  H->rope = (float*)(H->ws + work_bytes + freq_bytes);
  H->act_rows_bytes[COCO_WS_X] = R * d * eb;
  H->act_rows_bytes[COCO_WS_H] = R * d * eb;
  H->act_rows_bytes[COCO_WS_Q] = R * qd * eb;
  H->act_rows_bytes[COCO_WS_O] = R * qd * eb;
  H->act_rows_bytes[COCO_WS_X1] = R * d * 4;
  H->act_rows_bytes[COCO_WS_H2] = R * d * eb;
  H->act_rows_bytes[COCO_WS_U] = R * F * eb;

  // RoPE inverse frequencies theta^(-2j/hd), in fp64.
  std::vector<double> inv(c.head_dim / 2);
  for (int j = 0; j < c.head_dim / 2; ++j)
    inv[j] = pow((double)c.rope_theta, -2.0 * j / (double)c.head_dim);
  if (hipMemcpy(H->inv_freq, inv.data(), inv.size() * 8, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset(H->ws, 0, work_bytes) != hipSuccess ||
      hipEventCreateWithFlags(&H->done, hipEventDisableTiming) != hipSuccess ||
      (H->rope_rows > 0 &&
       (launch_rope_table(H->inv_freq, c.head_dim / 2, H->rope_rows, H->rope, nullptr) !=
            hipSuccess ||
        hipDeviceSynchronize() != hipSuccess))) {
    (void)hipGetLastError();
    if (H->done) (void)hipEventDestroy(H->done);
    (void)hipFree(H->ws);
    delete H;
    return fail(COCO_EHIP, "workspace initialisation failed");
  }
  if ((rc = pack_weights(H))) {
    (void)hipEventDestroy(H->done);
    (void)hipFree(H->ws);
    delete H;
    return rc;
  }
  *out = H;
  return COCO_OK;
}

void coco_layer_destroy(coco_layer_t H) {
  if (!H) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(H->device);
  // The handle's last call outside graph capture recorded `done` after its
  // last kernel; calls on one handle are ordered (they share the workspace),
  // so this waits for all of its enqueued work and nothing else.
  if (H->done) {
    (void)hipEventSynchronize(H->done);
    (void)hipEventDestroy(H->done);
  }
  for (auto& e : H->ev) (void)hipEventDestroy(e);
  (void)hipFree(H->ws);
  if (H->packed) (void)hipFree(H->packed);
  (void)hipSetDevice(cur);
  delete H;
}

int coco_layer_set_validate(coco_layer_t H, int32_t on) {
  if (!H) return fail(COCO_EINVAL, "handle is NULL");
  H->validate = on != 0;
  return COCO_OK;
}

int coco_layer_set_timing(coco_layer_t H, int32_t on) {
  if (!H) return fail(COCO_EINVAL, "handle is NULL");
  HIPCHK(hipSetDevice(H->device));
  if (on && H->ev.empty()) {
    H->ev.resize(2 * kTimingPairs);
    for (auto& e : H->ev) HIPCHK(hipEventCreate(&e));
    H->ev_kind.reserve(kTimingPairs);  // timed calls then never allocate
  }
  H->timing = on != 0;
  H->ev_kind.clear();
  H->ev_overflow = false;
  return COCO_OK;
}

int coco_layer_read_timing(coco_layer_t H, double* ms, int64_t* launches, int32_t n_kinds) {
  if (!H || !ms || !launches) return fail(COCO_EINVAL, "NULL argument");
  if (n_kinds < 0 || n_kinds > COCO_K_COUNT) return fail(COCO_EINVAL, "bad n_kinds");
  for (int k = 0; k < n_kinds; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  const bool overflow = H->ev_overflow;
  HIPCHK(hipSetDevice(H->device));
  for (size_t p = 0; p < H->ev_kind.size(); ++p) {
    HIPCHK(hipEventSynchronize(H->ev[2 * p + 1]));
    float t = 0.f;
    HIPCHK(hipEventElapsedTime(&t, H->ev[2 * p], H->ev[2 * p + 1]));
    const int k = H->ev_kind[p];
    if (k < n_kinds) {
      ms[k] += t;
      launches[k] += 1;
    }
  }
  H->ev_kind.clear();
  H->ev_overflow = false;
  if (overflow) return fail(COCO_ESTATE, "more than %d timed launches between reads", kTimingPairs);
  return COCO_OK;
}

int coco_layer_workspace(coco_layer_t H, int32_t which, void* dst, int64_t dst_bytes,
                         coco_stream_t stream) {
  if (!H || !dst) return fail(COCO_EINVAL, "NULL argument");
  void* p[7] = {H->w.x, H->w.h, H->w.q, H->w.o, H->w.x1, H->w.h2, H->w.u};
  if (which < 0 || which > 6) return fail(COCO_EINVAL, "unknown workspace id %d", which);
  if (dst_bytes < 0) return fail(COCO_EINVAL, "dst_bytes < 0");
  const size_t n = (size_t)dst_bytes < H->act_rows_bytes[which] ? (size_t)dst_bytes
                                                                 : H->act_rows_bytes[which];
  HIPCHK(hipSetDevice(H->device));
  const coco_layer_config& c = H->cfg;
  const int cols[7] = {c.d_model, c.d_model, c.n_q_heads * c.head_dim,
                       c.n_q_heads * c.head_dim, c.d_model, c.d_model, c.d_ffn};
  if (H->ws_tiled[which]) {
    HIPCHK(launch_untile((const uint16_t*)p[which], H->last_rows, cols[which],
                         (uint16_t*)dst, (int64_t)(n / 2), (hipStream_t)stream));
    return COCO_OK;
  }
  HIPCHK(hipMemcpyAsync(dst, p[which], n, hipMemcpyDeviceToDevice, (hipStream_t)stream));
  return COCO_OK;
}

}  // extern "C"

// ----------------------------------------------------------------------------
// Validation of device-side index arrays (debug mode; synchronises).
// ----------------------------------------------------------------------------
namespace {

template <typename V>
int fetch(std::vector<V>& dst, const V* src, size_t n, hipStream_t st) {
  dst.resize(n);
  if (n == 0) return COCO_OK;
  HIPCHK(hipMemcpyAsync(dst.data(), src, n * sizeof(V), hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  return COCO_OK;
}

int validate_batch(coco_layer* H, int64_t hidden_rows, const int32_t* row_idx, int n_rows,
                   const int32_t* positions, const int32_t* seq_starts, int n_seqs,
                   const int32_t* block_table, const int32_t* ctx_lens, int first_layer,
                   int n_layers, hipStream_t st) {
  const coco_layer_config& c = H->cfg;
  std::vector<int32_t> ri, pos, ss, bt, cl;
  int rc;
  if ((rc = fetch(ri, row_idx, n_rows, st)) || (rc = fetch(pos, positions, n_rows, st)) ||
      (rc = fetch(cl, ctx_lens, n_seqs, st)) ||
      (rc = fetch(bt, block_table, (size_t)n_seqs * c.max_blocks_per_seq, st)))
    return rc;
  if (seq_starts) {
    if ((rc = fetch(ss, seq_starts, n_seqs + 1, st))) return rc;
  } else {
    ss.resize(n_seqs + 1);
    for (int s = 0; s <= n_seqs; ++s) ss[s] = s;
  }
  std::vector<char> seen(hidden_rows, 0);
  for (int i = 0; i < n_rows; ++i) {
    if (ri[i] < 0 || ri[i] >= hidden_rows)
      return fail(COCO_EINVAL, "row_idx[%d] = %d out of range [0, %lld)", i, ri[i],
                  (long long)hidden_rows);
    if (seen[ri[i]]) return fail(COCO_EINVAL, "row_idx[%d] = %d is a duplicate", i, ri[i]);
    seen[ri[i]] = 1;
  }
  if (ss[0] != 0 || ss[n_seqs] != n_rows)
    return fail(COCO_EINVAL, "seq_starts must run from 0 to n_rows");
  int64_t min_blocks = INT64_MAX;
  for (int l = first_layer; l < first_layer + n_layers; ++l)
    if (H->layers[l].num_blocks < min_blocks) min_blocks = H->layers[l].num_blocks;
  for (int s = 0; s < n_seqs; ++s) {
    if (ss[s + 1] < ss[s]) return fail(COCO_EINVAL, "seq_starts not monotone at %d", s);
    if (cl[s] < 1 || cl[s] > c.max_blocks_per_seq * kBlockTokens)
      return fail(COCO_EINVAL, "ctx_lens[%d] = %d out of range", s, cl[s]);
    for (int i = ss[s]; i < ss[s + 1]; ++i) {
      if (pos[i] < 0 || pos[i] >= cl[s])
        return fail(COCO_EINVAL, "positions[%d] = %d not in [0, ctx_lens[%d] = %d)", i, pos[i],
                    s, cl[s]);
      if (i > ss[s] && pos[i] <= pos[i - 1])
        return fail(COCO_EINVAL, "positions of sequence %d not increasing at row %d", s, i);
    }
    const int nb = (cl[s] + kBlockTokens - 1) / kBlockTokens;
    for (int b = 0; b < nb; ++b) {
      const int32_t v = bt[(size_t)s * c.max_blocks_per_seq + b];
      if (v < 0 || v >= min_blocks)
        return fail(COCO_EINVAL, "block_table[%d][%d] = %d out of range [0, %lld)", s, b, v,
                    (long long)min_blocks);
    }
  }
  return COCO_OK;
}

// ----------------------------------------------------------------------------
// Launch sequence.
// ----------------------------------------------------------------------------
// Decode uses the weight-streaming plan (split-K from (N, K) only); prefill
// uses the large-tile kernel with one split.
template <typename T>
int gemm(float* part, const T* A, const T* W, int M, int N, int K, bool prefill, int* S,
         hipStream_t st);

template <>
int gemm<bf16_t>(float* part, const bf16_t* A, const bf16_t* W, int M, int N, int K,
                 bool prefill, int* S, hipStream_t st) {
  if (prefill) {
    *S = tile_splits(N, K);
    HIPCHK(launch_gemm_tile_bf16(A, W, part, M, N, K, *S, st));
    return COCO_OK;
  }
  const SkinnyPlan plan = skinny_plan(N, K);
  if (plan.waves == 0) return fail(COCO_EINVAL, "no GEMM plan for N=%d K=%d", N, K);
  *S = plan.S;
  HIPCHK(launch_gemm_skinny_bf16(A, W, part, M, N, K, plan, st));
  return COCO_OK;
}

template <>
int gemm<float>(float* part, const float* A, const float* W, int M, int N, int K, bool prefill,
                int* S, hipStream_t st) {
  (void)prefill;
  *S = 1;
  HIPCHK(launch_gemm_f32(A, W, part, M, N, K, st));
  return COCO_OK;
}

// SwiGLU runs in the gate/up GEMM's epilogue whenever that GEMM is not split
// along K (bf16; decode and prefill kernels each have a fused variant).
template <typename T>
bool fused_swiglu(bool prefill, int F, int K) {
  if (!std::is_same<T, bf16_t>::value) return false;
  return prefill ? tile_splits(2 * F, K) == 1 : skinny_plan(2 * F, K).S == 1;
}

// Layout of the four projections' A operands in a call: tile order
// (tile_off) wherever the consuming GEMM reads it so -- every bf16 prefill
// GEMM, and the decode GEMMs that run the row-split kernel -- else row-major.
struct ActLayout {
  bool h = false, o = false, h2 = false, u = false;
};
ActLayout act_layout(const coco_layer_config& c, bool prefill, int M) {
  ActLayout a;
  if (c.dtype != COCO_BF16) return a;
  if (prefill) {
    a.h = a.o = a.h2 = a.u = true;
    return a;
  }
  const int d = c.d_model, F = c.d_ffn, qd = c.n_q_heads * c.head_dim;
  a.o = skinny_reads_tiled(d, qd, M, false);
  a.h2 = skinny_reads_tiled(2 * F, d, M, skinny_plan(2 * F, d).S == 1);
  a.u = skinny_reads_tiled(d, F, M, false);
  return a;
}

template <typename T>
int attention(coco_layer* H, const Work& W, const coco_layer_weights& w, int M,
              const int32_t* positions, const int32_t* seq_starts, int n_seqs, const int32_t* bt,
              const int32_t* ctx, bool o_tiled, hipStream_t st);

template <>
int attention<bf16_t>(coco_layer* H, const Work& W, const coco_layer_weights& w, int M,
                      const int32_t* positions, const int32_t* seq_starts, int n_seqs,
                      const int32_t* bt, const int32_t* ctx, bool o_tiled, hipStream_t st) {
  const coco_layer_config& c = H->cfg;
  if (!seq_starts) {
    {
      KernelTimer t(H, COCO_K_ATTENTION, st);
      HIPCHK(launch_attn_decode_bf16((const bf16_t*)W.q, (const bf16_t*)w.k_cache,
                                     (const bf16_t*)w.v_cache, bt, c.max_blocks_per_seq, ctx,
                                     positions, W.split_off, n_seqs, c.n_q_heads, c.n_kv_heads,
                                     W.attn_o, W.attn_ml, H->max_splits, H->num_cus, st));
    }
    KernelTimer t(H, COCO_K_ATTN_COMBINE, st);
    HIPCHK(launch_attn_combine_bf16(W.attn_o, W.attn_ml, ctx, positions, n_seqs, c.n_q_heads,
                                    H->max_splits, (bf16_t*)W.o, o_tiled, st));
  } else {
    KernelTimer t(H, COCO_K_ATTENTION, st);
    HIPCHK(launch_attn_prefill_bf16((const bf16_t*)W.q, (const bf16_t*)w.k_cache,
                                    (const bf16_t*)w.v_cache, bt, c.max_blocks_per_seq, ctx,
                                    positions, seq_starts, n_seqs, M, c.n_q_heads, c.n_kv_heads,
                                    (bf16_t*)W.o, st));
  }
  return COCO_OK;
}

template <>
int attention<float>(coco_layer* H, const Work& W, const coco_layer_weights& w, int M,
                     const int32_t* positions, const int32_t* seq_starts, int n_seqs,
                     const int32_t* bt, const int32_t* ctx, bool o_tiled, hipStream_t st) {
  (void)o_tiled;  // fp32: row-major throughout
  const coco_layer_config& c = H->cfg;
  KernelTimer t(H, COCO_K_ATTENTION, st);
  HIPCHK(launch_attn_f32((const float*)W.q, (const float*)w.k_cache, (const float*)w.v_cache,
                         bt, c.max_blocks_per_seq, ctx, positions, seq_starts, n_seqs, M,
                         c.n_q_heads, c.n_kv_heads, c.head_dim, (float*)W.o, st));
  return COCO_OK;
}

template <typename T>
int run_span(coco_layer* H, const Work& W, int first, int nl, T* hidden, const int32_t* row_idx,
             int M, const int32_t* positions, const int32_t* seq_starts, int n_seqs,
             const int32_t* bt, const int32_t* ctx, hipStream_t st) {
  const coco_layer_config& c = H->cfg;
  const int d = c.d_model, Hq = c.n_q_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.d_ffn;
  const int nqkv = (Hq + 2 * Hkv) * hd;
  T* x = (T*)W.x;
  T* h = (T*)W.h;
  T* q = (T*)W.q;
  T* o = (T*)W.o;
  T* h2 = (T*)W.h2;
  T* u = (T*)W.u;
  int S, rc;
  const bool pre = seq_starts != nullptr;
  const ActLayout lay = act_layout(c, pre, M);
#define TIMED(kind, stmt)                     \
  do {                                        \
    KernelTimer timer_(H, kind, st);          \
    stmt;                                     \
  } while (0)
  for (int l = first; l < first + nl; ++l) {
    const coco_layer_weights& w = H->layers[l];
    const bool first_l = l == first, last_l = l == first + nl - 1;
    // Decode (bf16) folds the gather and RMSNorm_1 into the QKV projection:
    // it stages bf16(x * gamma) straight from the input rows and the QKV
    // epilogue applies each row's 1/rms. Otherwise a gather + RMSNorm_1
    // kernel writes h first. The residual reads the input rows where they
    // are (hidden[row_idx] in the first layer of the call), so no copy of
    // them is made.
    const bool fold_norm = !pre && std::is_same<T, bf16_t>::value;
    // Prefill QKV projection with RoPE and the cache append in its epilogue:
    // the narrow-tile GEMM (whole rotation pairs per tile) when the head
    // count has a plan, else the 256 x 256 tile GEMM.
    const bool narrow_qkv =
        pre && std::is_same<T, bf16_t>::value && hd == 128 && narrow_qkv_tile_n(Hq, Hkv, d) != 0;
    const bool fuse_qkv =
        narrow_qkv || (pre && std::is_same<T, bf16_t>::value && tile_qkv_fusable(Hq, Hkv, d));
    // Prefill O and down projections on the narrow-tile GEMM (256 x d/32
    // tiles, unsplit), when d has such a plan and the SwiGLU runs in the
    // gate/up epilogue: the O epilogue then folds in the residual and
    // RMSNorm_2's first half, the down epilogue the residual and the scatter.
    const int ntn = pre && std::is_same<T, bf16_t>::value ? narrow_tile_n(d) : 0;
    const bool narrow_o = ntn != 0 && (Hq * hd) % 128 == 0 && fused_swiglu<T>(pre, F, d);
    const bool narrow_down = ntn != 0 && F % 128 == 0;
    const bool fold_norm2 =
        narrow_o ||
        (pre && std::is_same<T, bf16_t>::value && tile_norm2_foldable(d, Hq * hd, F));
    const int norm_tiles = narrow_o ? d / ntn : d / 256;
    const T* x_src = first_l ? hidden : x;                     // this layer's input rows
    const int32_t* x_idx = first_l ? row_idx : nullptr;
    // The fused prefill QKV epilogue reads each row's (position, cache block),
    // written once per call by the first layer's gather.
    RowSlotArgs rs;
    if (fuse_qkv && first_l) {
      rs.positions = positions;
      rs.seq_starts = seq_starts;
      rs.block_table = bt;
      rs.row_info = W.row_info;
      rs.n_seqs = n_seqs;
      rs.max_blocks = c.max_blocks_per_seq;
      rs.rope_rows = H->rope_rows;
    }
    if (!fold_norm)
      TIMED(COCO_K_GATHER_NORM,
            HIPCHK(launch_gather_rmsnorm<T>(first_l ? hidden : x, first_l ? row_idx : nullptr, M,
                                            d, (const T*)w.gamma_attn, c.rms_eps,
                                            nullptr, h, lay.h, rs, st)));
    // QKV projection, RoPE, local cache append.
    if (fold_norm) {
      const SkinnyPlan plan = skinny_plan(nqkv, d);
      if (plan.waves == 0) return fail(COCO_EINVAL, "no GEMM plan for N=%d K=%d", nqkv, d);
      S = plan.S;
      TIMED(COCO_K_GEMM_QKV,
            HIPCHK(launch_gemm_skinny_norm_bf16((const bf16_t*)x_src, x_idx,
                                                (const bf16_t*)w.gamma_attn,
                                                (const bf16_t*)w.w_qkv, W.part, W.ss, M, nqkv, d,
                                                plan, st)));
    } else if (narrow_qkv) {
      NarrowEpiArgs qa;
      qa.row_info = W.row_info;
      qa.rope = H->rope;
      qa.q_out = (uint16_t*)q;
      qa.k_cache = (uint16_t*)w.k_cache;
      qa.v_cache = (uint16_t*)w.v_cache;
      qa.Hq = Hq;
      qa.Hkv = Hkv;
      TIMED(COCO_K_GEMM_QKV,
            HIPCHK(launch_gemm_narrow_qkv_bf16((const uint16_t*)h, (const uint16_t*)w.w_qkv, M,
                                               d, qa, st)));
    } else if (fuse_qkv) {
      // Prefill (bf16, QKV projection not split along K): RoPE and the cache
      // append run in the GEMM's epilogue.
      TileEpiArgs qa;
      qa.row_info = W.row_info;
      qa.rope = H->rope;
      qa.q_out = (uint16_t*)q;
      qa.k_cache = (uint16_t*)w.k_cache;
      qa.v_cache = (uint16_t*)w.v_cache;
      qa.Hq = Hq;
      qa.Hkv = Hkv;
      TIMED(COCO_K_GEMM_QKV,
            HIPCHK(launch_gemm_tile_qkv_bf16((const uint16_t*)h, (const uint16_t*)w.w_qkv, M, d,
                                             qa, st)));
    } else {
      TIMED(COCO_K_GEMM_QKV, if ((rc = gemm<T>(W.part, h, (const T*)w.w_qkv, M, nqkv, d, pre, &S, st))) return rc);
    }
    if (!fuse_qkv)
      TIMED(COCO_K_QKV_EPILOGUE,
            HIPCHK(launch_qkv_epilogue<T>(W.part, S, M, Hq, Hkv, hd, positions, seq_starts,
                                          n_seqs, bt, c.max_blocks_per_seq, H->inv_freq, q,
                                          (T*)w.k_cache, (T*)w.v_cache, ctx,
                                          (seq_starts == nullptr && c.dtype == COCO_BF16)
                                              ? W.split_off
                                              : nullptr,
                                          H->max_splits, fold_norm ? W.ss : nullptr, d,
                                          c.rms_eps, st)));
    // Attention over the paged cache.
    if ((rc = attention<T>(H, W, w, M, positions, seq_starts, n_seqs, bt, ctx, lay.o, st)))
      return rc;
    // O projection + residual + RMSNorm_2. Prefill (bf16, unsplit O and
    // gate/up projections): the O projection's epilogue adds the residual and
    // writes bf16(x1 * gamma_2) with per-tile sums of x1^2; the gate/up
    // epilogue applies each row's 1/rms, so no separate norm kernel runs.
    if (narrow_o) {
      TIMED(COCO_K_GEMM_O,
            HIPCHK(launch_gemm_narrow_resid_bf16((const uint16_t*)o, (const uint16_t*)w.w_o, M,
                                                 d, Hq * hd, (const uint16_t*)x_src, x_idx,
                                                 (const uint16_t*)w.gamma_mlp, W.x1,
                                                 (uint16_t*)h2, W.ss, st)));
    } else if (fold_norm2) {
      TIMED(COCO_K_GEMM_O,
            HIPCHK(launch_gemm_tile_resid_bf16((const uint16_t*)o, (const uint16_t*)w.w_o, M, d,
                                               Hq * hd, (const uint16_t*)x_src, x_idx,
                                               (const uint16_t*)w.gamma_mlp, W.x1,
                                               (uint16_t*)h2, W.ss, st)));
    } else {
      TIMED(COCO_K_GEMM_O, if ((rc = gemm<T>(W.part, o, (const T*)w.w_o, M, d, Hq * hd, pre, &S, st))) return rc);
      TIMED(COCO_K_RESIDUAL_NORM,
            HIPCHK(launch_residual_rmsnorm<T>(W.part, S, M, d, x_src, x_idx,
                                              (const T*)w.gamma_mlp, c.rms_eps, W.x1, h2, lay.h2,
                                              st)));
    }
    // SwiGLU MLP (prefill: SwiGLU in the gate/up GEMM's epilogue when the
    // GEMM is not split along K).
    if (fused_swiglu<T>(pre, F, d)) {
      if (pre && fold_norm2 && narrow_swiglu_fits(F, d)) {
        TIMED(COCO_K_GEMM_GATE_UP,
              HIPCHK(launch_gemm_narrow_swiglu_bf16((const uint16_t*)h2,
                                                    (const uint16_t*)w.w_gate_up, (uint16_t*)u,
                                                    M, F, d, W.ss, norm_tiles, c.rms_eps, st)));
      } else if (pre) {
        TIMED(COCO_K_GEMM_GATE_UP,
              HIPCHK(launch_gemm_tile_swiglu_bf16((const bf16_t*)h2, (const bf16_t*)w.w_gate_up,
                                                  (bf16_t*)u, M, F, d,
                                                  fold_norm2 ? W.ss : nullptr, norm_tiles,
                                                  c.rms_eps, st)));
      } else if (c.dtype == COCO_BF16 && M > 128 && lay.h2 && lay.u &&
                 narrow_swiglu_plain_fits(M, F, d)) {
        // 129-256 rows with one round of 256 x 128 tiles (the 8B shape): the
        // prefill tile kernel, bit-identical to the decode GEMM, in ~half its
        // time (the row-split decode kernel streams 2.8 TB/s there).
        TIMED(COCO_K_GEMM_GATE_UP,
              HIPCHK(launch_gemm_narrow_swiglu_plain_bf16((const uint16_t*)h2,
                                                          (const uint16_t*)w.w_gate_up,
                                                          (uint16_t*)u, M, F, d, st)));
      } else {
        TIMED(COCO_K_GEMM_GATE_UP,
              HIPCHK(launch_gemm_skinny_swiglu_bf16((const bf16_t*)h2,
                                                    (const bf16_t*)w.w_gate_up, (bf16_t*)u, M, F,
                                                    d, skinny_plan(2 * F, d), lay.u, st)));
      }
    } else {
      TIMED(COCO_K_GEMM_GATE_UP,
            if ((rc = gemm<T>(W.part, h2, (const T*)w.w_gate_up, M, 2 * F, d, pre, &S, st))) return rc);
      TIMED(COCO_K_SWIGLU, HIPCHK(launch_swiglu<T>(W.part, S, M, F, u, lay.u, st)));
    }
    // Down projection and residual; the last layer of the segment scatters to
    // the full batch.
    if (narrow_down) {
      TIMED(COCO_K_GEMM_DOWN,
            HIPCHK(launch_gemm_narrow_scatter_bf16((const uint16_t*)u, (const uint16_t*)w.w_down,
                                                   M, d, F, W.x1,
                                                   (uint16_t*)(last_l ? hidden : x),
                                                   last_l ? row_idx : nullptr, st)));
    } else {
      TIMED(COCO_K_GEMM_DOWN, if ((rc = gemm<T>(W.part, u, (const T*)w.w_down, M, d, F, pre, &S, st))) return rc);
      TIMED(COCO_K_RESIDUAL_SCATTER,
            HIPCHK(launch_residual_scatter<T>(W.part, S, M, d, W.x1, last_l ? hidden : x,
                                              last_l ? row_idx : nullptr, st)));
    }
  }
#undef TIMED
  return COCO_OK;
}

int check_batch(coco_layer* H, int first, int nl, const void* hidden, int64_t hidden_rows,
                const int32_t* row_idx, int n_rows, const int32_t* positions,
                const int32_t* seq_starts, int n_seqs, const int32_t* bt, const int32_t* ctx) {
  const coco_layer_config& c = H->cfg;
  if (first < 0 || nl < 1 || first + nl > c.n_layers)
    return fail(COCO_EINVAL, "layers [%d, %d) outside [0, %d)", first, first + nl, c.n_layers);
  if (n_rows < 0 || n_rows > c.max_rows)
    return fail(COCO_EINVAL, "n_rows = %d outside [0, max_rows = %d]", n_rows, c.max_rows);
  if (n_rows == 0) return COCO_OK;
  if (!hidden || !row_idx || !positions || !bt || !ctx)
    return fail(COCO_EINVAL, "NULL batch pointer");
  if (hidden_rows < 1) return fail(COCO_EINVAL, "hidden_rows must be >= 1");
  if ((uintptr_t)hidden % 16) return fail(COCO_EINVAL, "hidden is not 16-byte aligned");
  if (n_seqs < 1 || n_seqs > c.max_seqs)
    return fail(COCO_EINVAL, "n_seqs = %d outside [1, max_seqs = %d]", n_seqs, c.max_seqs);
  if (!seq_starts) {
    if (n_seqs != n_rows)
      return fail(COCO_EINVAL, "decode (seq_starts NULL) needs n_seqs == n_rows");
    if (n_seqs > H->dec_rows)
      return fail(COCO_EINVAL, "decode batch larger than min(max_rows, max_seqs)");
  } else if (n_seqs > n_rows) {
    return fail(COCO_EINVAL, "more sequences than rows");
  }
  return COCO_OK;
}

// Records the handle's completion event behind the call's last kernel, unless
// the stream is being captured into a graph (the event would then only fire
// on replays).
int mark_done(coco_layer* H, hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  HIPCHK(hipStreamIsCapturing(st, &cs));
  if (cs == hipStreamCaptureStatusNone) HIPCHK(hipEventRecord(H->done, st));
  return COCO_OK;
}

// use_static: the per-call buffers come from this device's static scratch
// array, sized for the call (no allocation anywhere; validation mode, which
// copies index arrays to the host, is not run).
int forward_impl(coco_layer* H, int first, int nl, void* hidden, int64_t hidden_rows,
                 const int32_t* row_idx, int n_rows, const int32_t* positions,
                 const int32_t* seq_starts, int n_seqs, const int32_t* bt, const int32_t* ctx,
                 coco_stream_t stream, bool use_static = false) {
  if (!H) return fail(COCO_EINVAL, "handle is NULL");
  int rc = check_batch(H, first, nl, hidden, hidden_rows, row_idx, n_rows, positions,
                       seq_starts, n_seqs, bt, ctx);
  if (rc || n_rows == 0) return rc;
  hipStream_t st = (hipStream_t)stream;
  HIPCHK(hipSetDevice(H->device));
  Work W = H->w;
  if (use_static) {
    const int64_t dec_seqs = seq_starts ? 0 : n_seqs;
    const size_t need = carve_work(H->cfg, n_rows, dec_seqs, H->max_splits, nullptr, nullptr);
    if (need > kScratchBytes)
      return fail(COCO_EINVAL,
                  "call needs %zu bytes of scratch; the no-alloc entry point has %zu (%d rows)",
                  need, kScratchBytes, n_rows);
    char* base = scratch_ptr(H->device);
    if (!base) return fail(COCO_ESTATE, "static scratch of device %d not set up", H->device);
    carve_work(H->cfg, n_rows, dec_seqs, H->max_splits, base, &W);
  } else if (H->validate &&
             (rc = validate_batch(H, hidden_rows, row_idx, n_rows, positions, seq_starts, n_seqs,
                                  bt, ctx, first, nl, st))) {
    return rc;
  }
  if (!use_static) {
    const ActLayout a = act_layout(H->cfg, seq_starts != nullptr, n_rows);
    for (bool& t : H->ws_tiled) t = false;
    H->ws_tiled[COCO_WS_H] = a.h;
    H->ws_tiled[COCO_WS_O] = a.o;
    H->ws_tiled[COCO_WS_H2] = a.h2;
    H->ws_tiled[COCO_WS_U] = a.u;
    H->last_rows = n_rows;
  }
  if (H->cfg.dtype == COCO_BF16)
    rc = run_span<bf16_t>(H, W, first, nl, (bf16_t*)hidden, row_idx, n_rows, positions,
                          seq_starts, n_seqs, bt, ctx, st);
  else
    rc = run_span<float>(H, W, first, nl, (float*)hidden, row_idx, n_rows, positions,
                         seq_starts, n_seqs, bt, ctx, st);
  if (rc) return rc;
  return mark_done(H, st);
}

}  // namespace

extern "C" {

int coco_layer_forward(coco_layer_t H, int32_t layer, void* hidden, int64_t hidden_rows,
                       const int32_t* row_idx, int32_t n_rows, const int32_t* positions,
                       const int32_t* seq_starts, int32_t n_seqs, const int32_t* block_table,
                       const int32_t* ctx_lens, coco_stream_t stream) {
  return forward_impl(H, layer, 1, hidden, hidden_rows, row_idx, n_rows, positions, seq_starts,
                      n_seqs, block_table, ctx_lens, stream);
}

int coco_layer_forward_noalloc(coco_layer_t H, int32_t layer, void* hidden, int64_t hidden_rows,
                               const int32_t* row_idx, int32_t n_rows, const int32_t* positions,
                               const int32_t* seq_starts, int32_t n_seqs,
                               const int32_t* block_table, const int32_t* ctx_lens,
                               coco_stream_t stream) {
  return forward_impl(H, layer, 1, hidden, hidden_rows, row_idx, n_rows, positions, seq_starts,
                      n_seqs, block_table, ctx_lens, stream, true);
}

int coco_layer_span_forward(coco_layer_t H, int32_t first_layer, int32_t n_layers, void* hidden,
                            int64_t hidden_rows, const int32_t* row_idx, int32_t n_rows,
                            const int32_t* positions, const int32_t* seq_starts, int32_t n_seqs,
                            const int32_t* block_table, const int32_t* ctx_lens,
                            coco_stream_t stream) {
  return forward_impl(H, first_layer, n_layers, hidden, hidden_rows, row_idx, n_rows, positions,
                      seq_starts, n_seqs, block_table, ctx_lens, stream);
}

int coco_kv_append(coco_layer_t H, int32_t layer, const void* k, const void* v,
                   const int32_t* seq_idx, const int32_t* positions, int32_t n_tok,
                   const int32_t* block_table, int32_t n_seqs, coco_stream_t stream) {
  if (!H) return fail(COCO_EINVAL, "handle is NULL");
  const coco_layer_config& c = H->cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(COCO_EINVAL, "layer %d out of range", layer);
  if (n_tok < 0) return fail(COCO_EINVAL, "n_tok < 0");
  if (n_tok == 0) return COCO_OK;
  if (!k || !v || !seq_idx || !positions || !block_table)
    return fail(COCO_EINVAL, "NULL argument");
  if (n_seqs < 1) return fail(COCO_EINVAL, "n_seqs must be >= 1");
  hipStream_t st = (hipStream_t)stream;
  HIPCHK(hipSetDevice(H->device));
  if (H->validate) {
    std::vector<int32_t> si, pos, bt;
    int rc;
    if ((rc = fetch(si, seq_idx, n_tok, st)) || (rc = fetch(pos, positions, n_tok, st)) ||
        (rc = fetch(bt, block_table, (size_t)n_seqs * c.max_blocks_per_seq, st)))
      return rc;
    for (int t = 0; t < n_tok; ++t) {
      if (si[t] < 0 || si[t] >= n_seqs) return fail(COCO_EINVAL, "seq_idx[%d] out of range", t);
      if (pos[t] < 0 || pos[t] >= c.max_blocks_per_seq * kBlockTokens)
        return fail(COCO_EINVAL, "positions[%d] out of range", t);
      const int32_t b = bt[(size_t)si[t] * c.max_blocks_per_seq + pos[t] / kBlockTokens];
      if (b < 0 || b >= H->layers[layer].num_blocks)
        return fail(COCO_EINVAL, "token %d maps to block %d outside the pool", t, b);
    }
  }
  const coco_layer_weights& w = H->layers[layer];
  if (c.dtype == COCO_BF16)
    HIPCHK(launch_kv_append<bf16_t>((const bf16_t*)k, (const bf16_t*)v, seq_idx, positions, n_tok,
                                    c.n_kv_heads, c.head_dim, block_table, c.max_blocks_per_seq,
                                    (bf16_t*)w.k_cache, (bf16_t*)w.v_cache, st));
  else
    HIPCHK(launch_kv_append<float>((const float*)k, (const float*)v, seq_idx, positions, n_tok,
                                   c.n_kv_heads, c.head_dim, block_table, c.max_blocks_per_seq,
                                   (float*)w.k_cache, (float*)w.v_cache, st));
  return mark_done(H, st);
}

}  // extern "C"
