"""The binding's shape and dtype checks, and the config checks of
coco_layer_init, on the CPU: each mismatch is refused before anything reaches
the library's kernels (no GPU needed)."""
import ctypes
import os

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_04181_amd", "libcoco.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libcoco.so not built")


def _handle(dtype="bf16", max_blocks=8):
    from paper_2607_04181_amd import _lib
    cfg = _lib.make_config(512, 8, 2, 128, 768, 1, dtype, 16, 16, max_blocks, 1e4, 1e-5)
    return _lib.Handle(None, cfg, [])


def _batch(n=4, d=512, max_blocks=8, dtype=torch.bfloat16):
    i32 = torch.int32
    return dict(hidden=torch.zeros(8, d, dtype=dtype), row_idx=torch.arange(n, dtype=i32),
                positions=torch.zeros(n, dtype=i32), seq_starts=None,
                block_table=torch.zeros(n, max_blocks, dtype=i32),
                ctx_lens=torch.ones(n, dtype=i32))


def _forward(h, b):
    import paper_2607_04181_amd as coco
    coco.coco_layer_forward(h, 0, b["hidden"], b["row_idx"], b["positions"], b["seq_starts"],
                            b["block_table"], b["ctx_lens"])


@pytest.mark.parametrize("field, value, exc, needle", [
    ("hidden", torch.zeros(8, 256, dtype=torch.bfloat16), ValueError, "hidden must be"),
    ("hidden", torch.zeros(8, 512, dtype=torch.float32), TypeError, "hidden must be"),
    ("positions", torch.zeros(3, dtype=torch.int32), ValueError, "positions has"),
    ("block_table", torch.zeros(4, 9, dtype=torch.int32), ValueError, "block_table must be"),
    ("block_table", torch.zeros(3, 8, dtype=torch.int32), ValueError, "block_table has"),
    ("ctx_lens", torch.ones(5, dtype=torch.int32), ValueError, "ctx_lens has"),
    ("seq_starts", torch.tensor([0, 4], dtype=torch.int32), ValueError, "seq_starts"),
])
def test_forward_refuses_mismatched_shapes_before_the_call(field, value, exc, needle):
    b = _batch()
    b[field] = value
    with pytest.raises(exc, match=needle):
        _forward(_handle(), b)


def test_forward_with_matching_shapes_reaches_the_device_check():
    with pytest.raises(ValueError, match="on the GPU"):
        _forward(_handle(), _batch())


def test_span_forward_checks_the_same_shapes():
    import paper_2607_04181_amd as coco
    b = _batch()
    b["block_table"] = torch.zeros(4, 7, dtype=torch.int32)
    with pytest.raises(ValueError, match="block_table must be"):
        coco.coco_layer_span_forward(_handle(), 0, 1, b["hidden"], b["row_idx"], b["positions"],
                                     None, b["block_table"], b["ctx_lens"])


def test_kv_append_refuses_mismatched_shapes():
    import paper_2607_04181_amd as coco
    h = _handle()
    i32 = torch.int32
    k = torch.zeros(3, 2, 128, dtype=torch.bfloat16)
    seq, pos, bt = torch.zeros(3, dtype=i32), torch.arange(3, dtype=i32), torch.zeros(1, 8, dtype=i32)
    with pytest.raises(ValueError, match="v must hold"):
        coco.coco_kv_append(h, 0, k, k[:2], seq, pos, bt)
    with pytest.raises(TypeError, match="k must be"):
        coco.coco_kv_append(h, 0, k.float(), k, seq, pos, bt)
    with pytest.raises(ValueError, match="seq_idx has"):
        coco.coco_kv_append(h, 0, k, k, seq[:2], pos, bt)
    with pytest.raises(ValueError, match="block_table must be"):
        coco.coco_kv_append(h, 0, k, k, seq, pos, torch.zeros(1, 4, dtype=i32))


def test_init_refuses_more_decode_partitions_than_the_merge_holds():
    # 2 floats per 256-token partition in 64 KB of LDS: at most 8184 partitions,
    # i.e. max_blocks_per_seq <= 130944; one block more is refused before any
    # HIP call.
    from paper_2607_04181_amd import _lib
    w = (_lib.coco_layer_weights * 1)()
    h = ctypes.c_void_p()
    cfg = _lib.make_config(512, 8, 2, 128, 768, 1, "bf16", 8, 8, 130944 + 16, 1e4, 1e-5)
    assert _lib.raw_call("coco_layer_init", ctypes.byref(cfg), w, ctypes.byref(h)) == _lib.COCO_EINVAL
    assert "partition" in _lib.coco_last_error()
    # At the limit the config passes (the call then stops at the NULL weights).
    cfg = _lib.make_config(512, 8, 2, 128, 768, 1, "bf16", 8, 8, 130944, 1e4, 1e-5)
    assert _lib.raw_call("coco_layer_init", ctypes.byref(cfg), w, ctypes.byref(h)) == _lib.COCO_EINVAL
    assert "NULL" in _lib.coco_last_error()
