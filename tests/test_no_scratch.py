"""No kernel of the built library uses scratch (private) memory.

A value the compiler cannot keep in registers (a by-value struct indexed at
run time, a spilled array) lands in per-lane scratch memory, which every wave
then writes and reads through the memory hierarchy; in the hot kernels that
costs as much as a share of their gathers.  The check reads the kernel
descriptors of the gfx950 code objects embedded in the built `libtbe.so`
(the `.hip_fatbin` section holds one offload bundle per source file) and
asserts that every kernel's private segment is empty.  Needs no GPU.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2512_23236_amd", "libtbe.so")
LLVM = "/opt/rocm/llvm/bin"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def _tools():
    need = [shutil.which("objcopy"), os.path.join(LLVM, "clang-offload-bundler"), os.path.join(LLVM, "llvm-readelf")]
    return all(t and os.path.exists(t) for t in need)


def _kernel_notes(d):
    """(kernel name, private segment bytes) for every kernel of every bundle."""
    fat = os.path.join(d, "fatbin")
    subprocess.run(["objcopy", f"--dump-section=.hip_fatbin={fat}", LIB, os.path.join(d, "discard.so")],
                   check=True, capture_output=True)
    blob = open(fat, "rb").read()
    starts = [m.start() for m in re.finditer(re.escape(MAGIC), blob)]
    out = []
    for k, s in enumerate(starts):
        e = starts[k + 1] if k + 1 < len(starts) else len(blob)
        part = os.path.join(d, f"b{k}")
        with open(part, "wb") as f:
            f.write(blob[s:e])
        co = os.path.join(d, f"b{k}.co")
        subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--type=o", f"--input={part}", "--unbundle",
                        f"--targets={TARGET}", f"--output={co}"], check=True, capture_output=True)
        notes = subprocess.run([os.path.join(LLVM, "llvm-readelf"), "--notes", co], check=True,
                               capture_output=True, text=True).stdout
        # each kernel's metadata map lists .name before .private_segment_fixed_size
        name = None
        for line in notes.splitlines():
            line = line.strip()
            if line.startswith(".name:"):
                name = line.split(":", 1)[1].strip()
            elif line.startswith(".private_segment_fixed_size:") and name is not None:
                out.append((name, int(line.split(":", 1)[1])))
                name = None
    return out


@pytest.mark.skipif(not os.path.exists(LIB), reason="libtbe.so is not built")
@pytest.mark.skipif(not _tools(), reason="needs objcopy and the ROCm LLVM tools")
def test_no_kernel_uses_scratch():
    with tempfile.TemporaryDirectory() as d:
        kernels = _kernel_notes(d)
    names = " ".join(n for n, _ in kernels)
    for k in ("forward_kernel", "keys_kernel", "radix_scatter_kernel", "reduce_kernel", "combine_kernel",
              "reduce_apply_kernel", "weight_grad_kernel", "map_ids_kernel"):
        assert k in names, f"{k} not found among the library's kernels"
    used = [(n, b) for n, b in kernels if b != 0]
    assert not used, f"kernels with a private segment: {used}"
