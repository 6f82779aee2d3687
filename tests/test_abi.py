"""The C ABI library loads and exports every function include/*.h declares
(CPU only: no compute calls)."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]
LIB = os.path.join(ROOT, "paper_2607_04181_amd", "libcoco.so")


def declared_functions():
    src = "\n".join(open(h).read() for h in HEADERS)
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(coco_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("coco_layer_init", "coco_kv_append", "coco_layer_forward",
              "coco_layer_span_forward", "coco_layer_destroy", "coco_last_error"):
        assert n in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcoco.so not built")
def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if l.strip())
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, f"not exported: {missing}"


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcoco.so not built")
def test_binding_loads_and_reports_version():
    import paper_2607_04181_amd as coco
    from paper_2607_04181_amd import _lib
    assert coco.coco_version() >= 100
    assert set(_lib.EXPORTS) == set(declared_functions())
    assert coco.coco_last_error() == ""


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcoco.so not built")
def test_init_rejects_bad_config_without_a_gpu():
    # Config checks run before any HIP call.
    import ctypes
    from paper_2607_04181_amd import _lib
    cfg = _lib.make_config(512, 8, 3, 128, 768, 1, "bf16", 8, 8, 4, 1e4, 1e-5)
    h = ctypes.c_void_p()
    w = (_lib.coco_layer_weights * 1)()
    rc = _lib.raw_call("coco_layer_init", ctypes.byref(cfg), w, ctypes.byref(h))
    assert rc == _lib.COCO_EINVAL
    assert "n_kv_heads" in _lib.coco_last_error()
    assert _lib.raw_call("coco_layer_forward", None, 0, None, 0, None, 0, None, None, 0, None,
                         None, None) == _lib.COCO_EINVAL
    # Positions (max_blocks_per_seq * 16) must fit the int32 RoPE table index.
    cfg = _lib.make_config(512, 8, 2, 128, 768, 1, "bf16", 8, 8, (1 << 24) + 1, 1e4, 1e-5)
    rc = _lib.raw_call("coco_layer_init", ctypes.byref(cfg), w, ctypes.byref(h))
    assert rc == _lib.COCO_EINVAL
    assert "max_blocks_per_seq" in _lib.coco_last_error()
