"""Resource use of the built device code: no kernel may spill to per-lane scratch.

Reads the AMDGPU code-object metadata of libgcn.so (built from this
repository's sources) with the ROCm LLVM tools; needs no GPU.  Scratch use in
a hot kernel is a silent slowdown (every spilled access becomes a global memory
round trip), e.g. a by-value argument struct that is both written and indexed
by a run-time value gets copied to scratch in its entirety.
"""
import os
import re
import shutil
import subprocess

import pytest

LLVM = "/opt/rocm/llvm/bin"
BUNDLER = os.path.join(LLVM, "clang-offload-bundler")
READELF = os.path.join(LLVM, "llvm-readelf")
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def kernel_metadata(lib, tmp):
    fat = os.path.join(tmp, "fatbin.bin")
    subprocess.run(["objcopy", "--dump-section", f".hip_fatbin={fat}", lib, os.path.join(tmp, "lib.copy")],
                   check=True, capture_output=True)
    data = open(fat, "rb").read()
    starts = [m.start() for m in re.finditer(re.escape(MAGIC), data)] + [len(data)]
    kernels = {}
    for i in range(len(starts) - 1):
        part = os.path.join(tmp, f"b{i}.bin")
        with open(part, "wb") as fh:
            fh.write(data[starts[i]:starts[i + 1]])
        dev = os.path.join(tmp, f"b{i}.o")
        subprocess.run([BUNDLER, "--unbundle", "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                        f"--input={part}", f"--output={dev}"], check=True, capture_output=True)
        if os.path.getsize(dev) == 0:
            continue
        notes = subprocess.run([READELF, "--notes", dev], check=True, capture_output=True, text=True).stdout
        name = None
        for line in notes.splitlines():
            m = re.match(r"\s*\.name:\s+(\S+)", line)
            if m:
                name = m.group(1)
                kernels.setdefault(name, {})
                continue
            m = re.match(r"\s*\.(private_segment_fixed_size|vgpr_spill_count|sgpr_spill_count):\s+(\d+)", line)
            if m and name:
                kernels[name][m.group(1)] = int(m.group(2))
    return {k: v for k, v in kernels.items() if "private_segment_fixed_size" in v}


@pytest.mark.skipif(not (os.path.exists(BUNDLER) and os.path.exists(READELF) and shutil.which("objcopy")),
                    reason="ROCm LLVM tools or objcopy missing")
def test_no_kernel_uses_scratch(tmp_path):
    import paper_2512_01678_amd.gcn as G
    meta = kernel_metadata(G.LIB_PATH, str(tmp_path))
    assert len(meta) >= 40, sorted(meta)
    assert any("k_aggregate" in k for k in meta) and any("k_gemm" in k for k in meta)
    # scalar-register spills land in vector-register lanes, not memory, and are allowed
    bad = {k: v for k, v in meta.items() if v.get("private_segment_fixed_size", 0) or v.get("vgpr_spill_count", 0)}
    assert not bad, bad
