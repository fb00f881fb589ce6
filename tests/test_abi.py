"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects bad arguments on the host before touching HIP."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2512_23236_amd import tbe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tbe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tbe_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for fn in ("tbe_forward", "tbe_backward", "tbe_backward_workspace_bytes", "tbe_plan_create",
               "tbe_plan_destroy", "tbe_abi_version"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(tbe.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert tbe.lib().tbe_abi_version() == tbe.ABI_VERSION


def _desc(rows=(100, 50), dims=(64, 128), dtype=tbe.F16, B=4, offs=None, elems=None, check=1, T=None,
          pooling=0, index_type=0, out_dtype=0):
    r = np.ascontiguousarray(rows, np.int64)
    d = np.ascontiguousarray(dims, np.int32)
    o = None if offs is None else np.ascontiguousarray(offs, np.int64)
    if elems is None:
        extra = 16 if dtype == tbe.U8_ROWWISE else 0
        elems = int((r * (d.astype(np.int64) + extra)).sum())
    desc = tbe._Desc(len(r) if T is None else T, dtype, B, r.ctypes.data, d.ctypes.data,
                     None if o is None else o.ctypes.data, elems, check, pooling, index_type, out_dtype)
    desc._keep = (r, d, o)
    return desc


def _create(desc):
    h = ctypes.c_void_p(123)
    rc = tbe.lib().tbe_plan_create(ctypes.byref(desc), ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("kwargs,code", [
    (dict(dtype=7), -3),
    (dict(T=0), -2),
    (dict(B=-1), -2),
    (dict(dims=(64, 12)), -4),                  # 12 fp16 = 24 bytes, not a multiple of 16
    (dict(dims=(4, 128), dtype=tbe.F16), -4),   # 4 fp16 = 8 bytes
    (dict(rows=(0, 50)), -2),
    (dict(elems=100), -2),                      # tables do not fit the buffer
    (dict(offs=(0, 4)), -4),                    # table 1 starts 8 bytes into a row boundary
    (dict(offs=(0, 6408)), -2),                 # table 1 runs past the end of the buffer
    (dict(check=2), -2),
    (dict(B=1 << 30), -2),                      # T*B beyond 32-bit bag ids
    (dict(pooling=2), -8),                      # unknown pooling mode
    (dict(index_type=2), -3),                   # unknown index type
    (dict(out_dtype=3), -3),                    # 8-bit row-wise is a table format only
    (dict(out_dtype=-1), -3),
    (dict(dtype=tbe.U8_ROWWISE, dims=(64, 24)), -4),          # 8-bit rows need D % 16 == 0
    (dict(dtype=tbe.U8_ROWWISE, offs=(0, 8008)), -4),         # 8-bit table offsets are 16-byte aligned
    (dict(dtype=tbe.U8_ROWWISE, offs=(0, 8000), elems=8000 + 50 * 144 - 1), -2),  # last row past the end
    (dict(rows=(2 ** 32 - 1, 50), dims=(16, 16), dtype=tbe.U8_ROWWISE), -2),  # row ids are 32-bit on the GPU
    (dict(rows=(2 ** 32, 50), dims=(8, 8)), -2),
])
def test_plan_create_rejects_bad_descriptors(kwargs, code):
    rc, h = _create(_desc(**kwargs))
    assert rc == code
    assert h.value is None  # *plan cleared, nothing allocated


def test_null_arguments_rejected_without_a_device():
    lib = tbe.lib()
    assert lib.tbe_plan_create(None, None) == -1
    h = ctypes.c_void_p()
    assert lib.tbe_plan_create(None, ctypes.byref(h)) == -1
    d = _desc()
    d.rows = None
    assert lib.tbe_plan_create(ctypes.byref(d), ctypes.byref(h)) == -1
    assert lib.tbe_forward(None, None, None, None, 0, None, None, None, None) == -1
    n = ctypes.c_size_t()
    assert lib.tbe_backward_workspace_bytes(None, 10, ctypes.byref(n)) == -1
    assert lib.tbe_backward(None, *([None] * 3), 0, None, None, 0, None, 0, *([None] * 6)) == -1
    assert lib.tbe_backward_timed(None, *([None] * 3), 0, None, None, 0, None, 0, *([None] * 7)) == -1
    assert lib.tbe_backward_index(None, None, None, 0, None, None, 0, *([None] * 7)) == -1
    assert lib.tbe_backward_reduce(None, None, 0, None, None, 0, None, 0, *([None] * 4)) == -1
    assert lib.tbe_plan_destroy(None) == 0
    assert lib.tbe_plan_info(None, None, None, None) == -1


def test_error_strings():
    lib = tbe.lib()
    for code in range(0, -9, -1):
        s = lib.tbe_error_string(code)
        assert s and s != b"unknown error code"
    assert lib.tbe_error_string(-99) == b"unknown error code"


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(tbe, "_lib", None)
    monkeypatch.setattr(tbe, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        tbe.lib()


def test_library_override_fails_loudly_when_missing(tmp_path):
    """TBE_LIBRARY names another build; a missing one raises, never falls back."""
    import subprocess
    import sys
    code = ("from paper_2512_23236_amd import tbe\n"
            "try:\n    tbe.lib()\nexcept ImportError as e:\n    print('raised', e)\n")
    env = dict(os.environ, TBE_LIBRARY=str(tmp_path / "other.so"))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert "raised" in r.stdout and "other.so" in r.stdout


def test_product_path_does_not_touch_the_oracle():
    """The package and its sources never import or link the CPU oracle."""
    pkg = os.path.join(ROOT, "paper_2512_23236_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), f
