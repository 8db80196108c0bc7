"""Register and scratch use of the built gfx950 kernels, read from the code
object metadata of libtopoep.so (no GPU needed).

The one-launch plan runs its solver and its chunks in one kernel whose
workgroups wait for each other: a kernel that needs scratch memory pays for
its set-up at dispatch, which made a variant of that kernel with 720 bytes
of spilled registers per lane 3.4 times slower (11.8 -> 40.5 us per layer on
the DeepSeek-V3-like plan).  Every kernel therefore keeps its values in
registers; only the per-domain solver may keep a few (a 24-byte spill there
measured no different from none)."""
import os
import re
import shutil
import subprocess

import pytest

LLVM = "/opt/rocm/llvm/bin"
TOOLS = [os.path.join(LLVM, t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readelf")]
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def kernel_metadata(lib_path, tmp):
    """[(kernel name, private segment bytes, vgpr count)] over every code
    object bundled in the library's .hip_fatbin section."""
    fatbin = os.path.join(tmp, "fatbin")
    subprocess.run([TOOLS[0], "--dump-section=.hip_fatbin=" + fatbin, lib_path, os.path.join(tmp, "lib.copy")],
                   check=True, capture_output=True)
    data = open(fatbin, "rb").read()
    starts = [m.start() for m in re.finditer(re.escape(MAGIC), data)]
    assert starts, "no offload bundle in .hip_fatbin"
    out = []
    for i, s in enumerate(starts):
        piece = os.path.join(tmp, "bundle%d" % i)
        with open(piece, "wb") as f:
            f.write(data[s:starts[i + 1] if i + 1 < len(starts) else len(data)])
        co = piece + ".co"
        subprocess.run([TOOLS[1], "--unbundle", "--type=o", "--input=" + piece, "--targets=" + TARGET,
                        "--output=" + co], check=True, capture_output=True)
        notes = subprocess.run([TOOLS[2], "--notes", co], check=True, capture_output=True, text=True).stdout
        # one metadata map per kernel: its fields follow in source order
        for block in re.split(r"\n\s+- \.", notes):
            name = re.search(r"\.name:\s+(\S+)", block)
            priv = re.search(r"\.private_segment_fixed_size:\s+(\d+)", block)
            vgpr = re.search(r"\.vgpr_count:\s+(\d+)", block)
            if name and priv and vgpr and name.group(1).startswith("_Z"):
                out.append((name.group(1), int(priv.group(1)), int(vgpr.group(1))))
    return out


def _library_kernels(tmp_path_factory, path):
    if not all(os.path.exists(t) for t in TOOLS):
        pytest.skip("ROCm LLVM tools not installed")
    if not os.path.exists(path):
        pytest.skip("%s is not built" % os.path.basename(path))
    tmp = str(tmp_path_factory.mktemp("codeobj"))
    try:
        return kernel_metadata(path, tmp)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    from paper_2609_35481_amd import topoep
    return _library_kernels(tmp_path_factory, topoep.LIB_PATH)


@pytest.fixture(scope="module")
def stamp_kernels(tmp_path_factory):
    """The instrumented build used for phase timings: its kernels must keep
    the product's register budget, or the stamps would time a different
    kernel."""
    from paper_2609_35481_amd import build
    return _library_kernels(tmp_path_factory, build.STAMPS_LIB)


def test_every_kernel_is_in_the_library(kernels):
    names = " ".join(k[0] for k in kernels)
    for part in ("plan_fused_kernel", "solve_kernel", "solve_single_kernel", "hist_kernel", "reroute_kernel",
                 "empty_kernel"):
        assert part in names, part
    # the one-launch kernel: 4 id widths x 3 refinement forms (registers with
    # (instance, target) pairs, registers, LDS)
    assert sum("plan_fused_kernel" in k[0] for k in kernels) == 12
    # the dispatch layout and the replica gather sources add their own
    assert len(kernels) > 20


def test_no_kernel_spills_to_scratch(kernels):
    for name, priv, vgpr in kernels:
        if "12solve_kernel" in name:
            assert priv <= 64, (name, priv)
        else:
            assert priv == 0, (name, priv)
        assert vgpr <= 512, (name, vgpr)


def test_stamped_build_spills_nothing_either(stamp_kernels):
    for name, priv, vgpr in stamp_kernels:
        if "12solve_kernel" in name:
            assert priv <= 64, (name, priv)
        else:
            assert priv == 0, (name, priv)
