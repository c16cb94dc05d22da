"""The built gfx950 code objects: no kernel keeps values in scratch memory.

A kernel whose accumulators or staged values spill to scratch still gives the
right results, so no parity test notices, but it runs several times slower
(a rolled loop over the GEMM epilogue's passes once moved the 256-wide tiles'
accumulators to scratch: the fused bias epilogue took 287 us instead of 31).
This reads the AMDGPU metadata of every kernel in the objects the build left
in ``paper_2608_27370_amd/_build``: no private segment, no dynamic stack, no
VGPR or SGPR spills.
"""

import glob
import os
import re
import subprocess
import tempfile

import pytest
import yaml

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_2608_27370_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def _kernels(obj):
    """Metadata of every kernel in the gfx950 code object embedded in obj."""
    with tempfile.TemporaryDirectory() as d:
        fat, co = os.path.join(d, "fatbin"), os.path.join(d, "co")
        subprocess.run([os.path.join(LLVM, "llvm-objcopy"), "--dump-section", ".hip_fatbin=" + fat, obj, os.devnull],
                       check=True, capture_output=True)
        subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle", "--type=o", "--targets=" + TARGET,
                        "--input=" + fat, "--output=" + co], check=True, capture_output=True)
        notes = subprocess.run([os.path.join(LLVM, "llvm-readelf"), "--notes", co], check=True,
                               capture_output=True, text=True).stdout
    doc = re.search(r"^(amdhsa\..*?)^\s*\.\.\.\s*$", notes, re.S | re.M)
    assert doc, "no AMDGPU metadata in %s" % obj
    return yaml.safe_load(doc.group(1))["amdhsa.kernels"]


def _objects():
    tools = all(os.access(os.path.join(LLVM, t), os.X_OK)
                for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readelf"))
    objs = [o for o in sorted(glob.glob(os.path.join(BUILD, "*.o"))) if not o.endswith("api.o")]
    if not tools or not objs:
        pytest.skip("needs the built objects (paper_2608_27370_amd/build.py) and the ROCm LLVM tools")
    return objs


def test_no_kernel_uses_scratch():
    seen = 0
    bad = []
    for obj in _objects():
        for k in _kernels(obj):
            seen += 1
            if (k.get(".private_segment_fixed_size", 0) or k.get(".uses_dynamic_stack", False)
                    or k.get(".vgpr_spill_count", 0) or k.get(".sgpr_spill_count", 0)):
                bad.append((os.path.basename(obj), k[".name"], k.get(".private_segment_fixed_size"),
                            k.get(".vgpr_spill_count"), k.get(".sgpr_spill_count")))
    assert seen > 100, "expected every GEMM and quantise instance, found %d kernels" % seen
    assert not bad, bad
