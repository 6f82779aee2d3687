"""ctypes binding of libcoco.so: argument marshalling only.

Every function has the name of the C entry point it calls (see
include/coco.h for semantics, layouts and errors). Tensors are torch tensors
on the GPU; only their device addresses are passed. Negative return codes
raise CocoError with the library's message. There is no fallback: if the
library is not built, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcoco.so")

COCO_OK, COCO_EINVAL, COCO_ENOMEM, COCO_EHIP, COCO_ESTATE = 0, -1, -2, -3, -4
COCO_BF16, COCO_F32 = 0, 1
COCO_WS_X, COCO_WS_H, COCO_WS_Q, COCO_WS_O, COCO_WS_X1, COCO_WS_H2, COCO_WS_U = range(7)

EXPORTS = ["coco_layer_init", "coco_layer_destroy", "coco_last_error", "coco_version",
           "coco_layer_set_validate", "coco_kv_append", "coco_layer_forward",
           "coco_layer_span_forward", "coco_layer_forward_noalloc", "coco_layer_workspace",
           "coco_layer_set_timing",
           "coco_layer_read_timing", "coco_probe_read", "coco_probe_mfma_bf16",
           # include/coco_scaling.h: host arithmetic of the speedup/cost model
           "coco_split_batch", "coco_comm_time", "coco_speedup", "coco_cost_mem",
           "coco_cost_comp", "coco_speedup_vec", "coco_scale_candidates"]
KERNEL_KINDS = ["gather_norm", "gemm_qkv", "qkv_epilogue", "attention", "attn_combine", "gemm_o",
                "residual_norm", "gemm_gate_up", "swiglu", "gemm_down", "residual_scatter"]


class CocoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"coco error {code}: {msg}")
        self.code = code


class coco_layer_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn", "n_layers", "dtype",
        "block_size", "max_rows", "max_seqs", "max_blocks_per_seq")] + [
        ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float)]


class coco_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "w_qkv", "w_o", "w_gate_up", "w_down", "gamma_attn", "gamma_mlp", "k_cache",
        "v_cache")] + [("num_blocks", ctypes.c_int64)]


class coco_scale_model(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("batch", ctypes.c_int64),
                ("tokens_per_row", ctypes.c_int64), ("d_hidden", ctypes.c_int64),
                ("elem_bytes", ctypes.c_double), ("t_comp", ctypes.c_double),
                ("bandwidth", ctypes.c_double)]


class coco_scale_candidate(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("parallel", ctypes.c_int32),
                ("speedup", ctypes.c_double), ("distance", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    sig = {
        "coco_layer_init": (ctypes.c_int, [ctypes.POINTER(coco_layer_config),
                                           ctypes.POINTER(coco_layer_weights),
                                           ctypes.POINTER(vp)]),
        "coco_layer_destroy": (None, [vp]),
        "coco_last_error": (ctypes.c_char_p, []),
        "coco_version": (ctypes.c_int, []),
        "coco_layer_set_validate": (ctypes.c_int, [vp, i32]),
        "coco_kv_append": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, i32, vp, i32, vp]),
        "coco_layer_forward": (ctypes.c_int, [vp, i32, vp, i64, vp, i32, vp, vp, i32, vp, vp,
                                              vp]),
        "coco_layer_span_forward": (ctypes.c_int, [vp, i32, i32, vp, i64, vp, i32, vp, vp, i32,
                                                   vp, vp, vp]),
        "coco_layer_forward_noalloc": (ctypes.c_int, [vp, i32, vp, i64, vp, i32, vp, vp, i32,
                                                      vp, vp, vp]),
        "coco_layer_workspace": (ctypes.c_int, [vp, i32, vp, i64, vp]),
        "coco_layer_set_timing": (ctypes.c_int, [vp, i32]),
        "coco_layer_read_timing": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_double),
                                                  ctypes.POINTER(i64), i32]),
        "coco_probe_read": (ctypes.c_int, [vp, i64, vp, i32, i32, vp]),
        "coco_probe_mfma_bf16": (ctypes.c_int, [i64, vp, i32, i32, i32,
                                                ctypes.POINTER(ctypes.c_double), vp]),
        "coco_split_batch": (ctypes.c_int, [i64, i32, ctypes.POINTER(i64)]),
        "coco_comm_time": (ctypes.c_double, [ctypes.POINTER(coco_scale_model), i32]),
        "coco_speedup": (ctypes.c_double, [ctypes.POINTER(coco_scale_model), i32, i32]),
        "coco_cost_mem": (ctypes.c_double, [ctypes.POINTER(coco_scale_model), i32, i32]),
        "coco_cost_comp": (ctypes.c_double, [ctypes.POINTER(coco_scale_model), i32, i32]),
        "coco_speedup_vec": (ctypes.c_double, [ctypes.POINTER(coco_scale_model),
                                               ctypes.POINTER(i32),
                                               ctypes.POINTER(ctypes.c_double),
                                               ctypes.POINTER(ctypes.c_double), i32]),
        "coco_scale_candidates": (ctypes.c_int, [ctypes.POINTER(coco_scale_model), i32, i32, i32,
                                                 i32, ctypes.c_double, i32,
                                                 ctypes.POINTER(coco_scale_candidate), i32,
                                                 ctypes.POINTER(i32), ctypes.POINTER(i32),
                                                 ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


def _check(rc: int) -> int:
    if rc < 0:
        raise CocoError(rc, _lib.coco_last_error().decode())
    return rc


def _ptr(t, dtype=None, what="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{what} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    return t.data_ptr() if t.numel() else None


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if isinstance(stream, torch.cuda.Stream) else stream


class Handle:
    """An initialised replica; keeps the borrowed tensors alive."""

    def __init__(self, raw, cfg, keep):
        self.raw = raw
        self.cfg = cfg
        self._keep = keep

    def __del__(self):
        if getattr(self, "raw", None):
            _lib.coco_layer_destroy(self.raw)
            self.raw = None


def coco_version() -> int:
    return _lib.coco_version()


def coco_last_error() -> str:
    return _lib.coco_last_error().decode()


def make_config(d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, n_layers, dtype, max_rows,
                max_seqs, max_blocks_per_seq, rope_theta, rms_eps, block_size=16):
    return coco_layer_config(d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, n_layers,
                             COCO_BF16 if dtype in ("bf16", COCO_BF16) else COCO_F32,
                             block_size, max_rows, max_seqs, max_blocks_per_seq,
                             float(rope_theta), float(rms_eps))


def coco_layer_init(cfg: coco_layer_config, layers) -> Handle:
    """layers: list of dicts with w_qkv, w_o, w_gate_up, w_down, gamma_attn,
    gamma_mlp, k_cache, v_cache (device tensors)."""
    arr = (coco_layer_weights * len(layers))()
    keep = []
    for i, w in enumerate(layers):
        for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "gamma_attn", "gamma_mlp", "k_cache",
                  "v_cache"):
            setattr(arr[i], k, _ptr(w[k], what=k))
            keep.append(w[k])
        arr[i].num_blocks = int(w["k_cache"].shape[0])
    raw = ctypes.c_void_p()
    _check(_lib.coco_layer_init(ctypes.byref(cfg), arr, ctypes.byref(raw)))
    return Handle(raw, cfg, keep)


def coco_layer_destroy(h: Handle) -> None:
    if h.raw:
        _lib.coco_layer_destroy(h.raw)
        h.raw = None


def coco_layer_set_validate(h: Handle, on: bool) -> None:
    _check(_lib.coco_layer_set_validate(h.raw, 1 if on else 0))


def _elem_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == COCO_BF16 else torch.float32


def _shape_check(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _check_batch(h: Handle, hidden, row_idx, positions, seq_starts, block_table, ctx_lens):
    """Shapes and dtypes against the handle's config, before any call: the
    library takes plain pointers and uses the config for every stride."""
    cfg = h.cfg
    for name, t in (("hidden", hidden), ("row_idx", row_idx), ("positions", positions),
                    ("block_table", block_table), ("ctx_lens", ctx_lens)):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch tensor")
    if hidden.dtype != _elem_dtype(cfg):
        raise TypeError(f"hidden must be {_elem_dtype(cfg)}, got {hidden.dtype}")
    _shape_check(hidden.dim() == 2 and hidden.shape[1] == cfg.d_model,
                 f"hidden must be [rows, {cfg.d_model}], got {tuple(hidden.shape)}")
    n = row_idx.numel()
    _shape_check(row_idx.dim() == 1, "row_idx must be 1-D")
    _shape_check(positions.numel() == n,
                 f"positions has {positions.numel()} entries for {n} rows")
    n_seqs = ctx_lens.numel()
    if seq_starts is None:
        _shape_check(n_seqs == n, f"decode: ctx_lens has {n_seqs} entries for {n} rows")
    else:
        _shape_check(isinstance(seq_starts, torch.Tensor) and seq_starts.numel() == n_seqs + 1,
                     f"seq_starts must have n_seqs + 1 = {n_seqs + 1} entries")
    _shape_check(block_table.dim() == 2 and block_table.shape[1] == cfg.max_blocks_per_seq,
                 f"block_table must be [n_seqs, {cfg.max_blocks_per_seq}], "
                 f"got {tuple(block_table.shape)}")
    _shape_check(block_table.shape[0] >= n_seqs,
                 f"block_table has {block_table.shape[0]} rows for {n_seqs} sequences")


def coco_kv_append(h: Handle, layer: int, k, v, seq_idx, positions, block_table, stream=None):
    i32 = torch.int32
    cfg = h.cfg
    n_tok = int(positions.numel())
    per_tok = cfg.n_kv_heads * cfg.head_dim
    for name, t in (("k", k), ("v", v)):
        if t.dtype != _elem_dtype(cfg):
            raise TypeError(f"{name} must be {_elem_dtype(cfg)}, got {t.dtype}")
        _shape_check(t.numel() == n_tok * per_tok,
                     f"{name} must hold [{n_tok}, {cfg.n_kv_heads}, {cfg.head_dim}] elements")
    _shape_check(seq_idx.numel() == n_tok, f"seq_idx has {seq_idx.numel()} entries for {n_tok} tokens")
    _shape_check(block_table.dim() == 2 and block_table.shape[1] == cfg.max_blocks_per_seq,
                 f"block_table must be [n_seqs, {cfg.max_blocks_per_seq}], "
                 f"got {tuple(block_table.shape)}")
    _check(_lib.coco_kv_append(h.raw, layer, _ptr(k, what="k"), _ptr(v, what="v"),
                               _ptr(seq_idx, i32, "seq_idx"), _ptr(positions, i32, "positions"),
                               int(positions.numel()), _ptr(block_table, i32, "block_table"),
                               int(block_table.shape[0]), _stream(stream)))


def coco_layer_forward(h: Handle, layer: int, hidden, row_idx, positions, seq_starts,
                       block_table, ctx_lens, stream=None):
    i32 = torch.int32
    _check_batch(h, hidden, row_idx, positions, seq_starts, block_table, ctx_lens)
    n_seqs = int(ctx_lens.numel())
    _check(_lib.coco_layer_forward(
        h.raw, layer, _ptr(hidden, what="hidden"), int(hidden.shape[0]),
        _ptr(row_idx, i32, "row_idx"), int(row_idx.numel()), _ptr(positions, i32, "positions"),
        _ptr(seq_starts, i32, "seq_starts"), n_seqs, _ptr(block_table, i32, "block_table"),
        _ptr(ctx_lens, i32, "ctx_lens"), _stream(stream)))


def coco_layer_forward_noalloc(h: Handle, layer: int, hidden, row_idx, positions, seq_starts,
                               block_table, ctx_lens, stream=None):
    i32 = torch.int32
    _check_batch(h, hidden, row_idx, positions, seq_starts, block_table, ctx_lens)
    n_seqs = int(ctx_lens.numel())
    _check(_lib.coco_layer_forward_noalloc(
        h.raw, layer, _ptr(hidden, what="hidden"), int(hidden.shape[0]),
        _ptr(row_idx, i32, "row_idx"), int(row_idx.numel()), _ptr(positions, i32, "positions"),
        _ptr(seq_starts, i32, "seq_starts"), n_seqs, _ptr(block_table, i32, "block_table"),
        _ptr(ctx_lens, i32, "ctx_lens"), _stream(stream)))


def coco_layer_span_forward(h: Handle, first_layer: int, n_layers: int, hidden, row_idx,
                            positions, seq_starts, block_table, ctx_lens, stream=None):
    i32 = torch.int32
    _check_batch(h, hidden, row_idx, positions, seq_starts, block_table, ctx_lens)
    n_seqs = int(ctx_lens.numel())
    _check(_lib.coco_layer_span_forward(
        h.raw, first_layer, n_layers, _ptr(hidden, what="hidden"), int(hidden.shape[0]),
        _ptr(row_idx, i32, "row_idx"), int(row_idx.numel()), _ptr(positions, i32, "positions"),
        _ptr(seq_starts, i32, "seq_starts"), n_seqs, _ptr(block_table, i32, "block_table"),
        _ptr(ctx_lens, i32, "ctx_lens"), _stream(stream)))


def coco_layer_workspace(h: Handle, which: int, dst, stream=None) -> None:
    _check(_lib.coco_layer_workspace(h.raw, which, _ptr(dst, what="dst"),
                                     dst.numel() * dst.element_size(), _stream(stream)))


def coco_layer_set_timing(h: Handle, on: bool) -> None:
    _check(_lib.coco_layer_set_timing(h.raw, 1 if on else 0))


def coco_layer_read_timing(h: Handle) -> dict:
    """{kind: (total_ms, launches)} since timing was switched on / last read."""
    n = len(KERNEL_KINDS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    _check(_lib.coco_layer_read_timing(h.raw, ms, cnt, n))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNEL_KINDS)}


def coco_probe_read(buf, out, blocks: int, variant: int = 0, stream=None) -> None:
    """One read pass over the whole of `buf` (device tensor); `out` holds at
    least `blocks` int32 words."""
    nbytes = buf.numel() * buf.element_size()
    _check(_lib.coco_probe_read(_ptr(buf, what="buf"), nbytes, _ptr(out, what="out"), blocks,
                                variant, _stream(stream)))


def coco_probe_mfma_bf16(iters: int, out, blocks: int, chains: int = 4, operands: int = 0,
                         stream=None) -> float:
    """Enqueues the MFMA loop; returns its dense flop count. `out` holds at
    least 4 * blocks floats; operands 0: constants, 1: random data."""
    flops = ctypes.c_double()
    _check(_lib.coco_probe_mfma_bf16(iters, _ptr(out, what="out"), blocks, chains, operands,
                                     ctypes.byref(flops), _stream(stream)))
    return flops.value


def raw_call(name: str, *args) -> int:
    """Call an entry point with raw ctypes arguments and return its code
    (used by error-path tests that pass deliberately bad arguments)."""
    return getattr(_lib, name)(*args)


# ----------------------------------------------------------------------------
# Speedup / cost model (include/coco_scaling.h): host arithmetic, no GPU.
# ----------------------------------------------------------------------------
def make_scale_model(n_layers: int, batch: int, tokens_per_row: int, d_hidden: int,
                     elem_bytes: float, t_comp: float, bandwidth: float) -> coco_scale_model:
    return coco_scale_model(n_layers, batch, tokens_per_row, d_hidden, elem_bytes, t_comp,
                            bandwidth)


def coco_split_batch(bs: int, v: int) -> list:
    out = (ctypes.c_int64 * max(v, 1))()
    _check(_lib.coco_split_batch(bs, v, out))
    return [int(x) for x in out[:v]]


def coco_comm_time(m: coco_scale_model, P: int) -> float:
    return _lib.coco_comm_time(ctypes.byref(m), P)


def coco_speedup(m: coco_scale_model, N: int, P: int) -> float:
    return _lib.coco_speedup(ctypes.byref(m), N, P)


def coco_cost_mem(m: coco_scale_model, N: int, P: int) -> float:
    return _lib.coco_cost_mem(ctypes.byref(m), N, P)


def coco_cost_comp(m: coco_scale_model, N: int, P: int) -> float:
    return _lib.coco_cost_comp(ctypes.byref(m), N, P)


def coco_speedup_vec(m: coco_scale_model, v, t_dev, bandwidths) -> float:
    n_dev = len(t_dev)
    if len(bandwidths) != n_dev:
        raise ValueError("one bandwidth per device")
    vv = (ctypes.c_int32 * len(v))(*[int(x) for x in v])
    tt = (ctypes.c_double * n_dev)(*[float(x) for x in t_dev])
    bb = (ctypes.c_double * n_dev)(*[float(x) for x in bandwidths])
    return _lib.coco_speedup_vec(ctypes.byref(m), vv, tt, bb, n_dev)


def coco_scale_candidates(m: coco_scale_model, first: int, p_max: int, n_cur: int, p_cur: int,
                          latency_over_slo: float, cold_devices: int):
    """Returns (alpha_req, [(N, P, S, distance), ...] ranked, chosen (N, P) or None)."""
    cap = 1 + (m.n_layers - first) * max(p_max - 1, 0)
    out = (coco_scale_candidate * cap)()
    n_out, chosen, alpha = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
    _check(_lib.coco_scale_candidates(ctypes.byref(m), first, p_max, n_cur, p_cur,
                                      latency_over_slo, cold_devices, out, cap,
                                      ctypes.byref(n_out), ctypes.byref(chosen),
                                      ctypes.byref(alpha)))
    ranked = [(c.n_layers, c.parallel, c.speedup, c.distance) for c in out[:n_out.value]]
    pick = None if chosen.value < 0 else ranked[chosen.value][:2]
    return alpha.value, ranked, pick
