"""Register and scratch budget of every gfx950 kernel the build produced.

A kernel that spills vector registers to scratch memory pays an HBM round
trip per spilled value and needs a scratch allocation at every launch; a
change in one epilogue path can make the register allocator spill in the
whole kernel.  These checks read the kernel metadata the compiler wrote into
the code objects of this build (the objects under the package's _build
folder, made by __graft_entry__.build()) and run without a GPU.
"""
import glob
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_2607_12358_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def _tool(name):
    p = os.path.join(LLVM, name)
    return p if os.path.exists(p) else shutil.which(name)


def _kernels_of(obj, tmp):
    """Kernel metadata maps of the gfx950 code object embedded in obj."""
    objcopy, bundler, readelf = _tool("llvm-objcopy"), _tool("clang-offload-bundler"), \
        _tool("llvm-readelf")
    base = os.path.join(tmp, os.path.basename(obj))
    r = subprocess.run([objcopy, f"--dump-section=.hip_fatbin={base}.fat", obj, os.devnull],
                       capture_output=True, text=True)
    if r.returncode != 0:
        return None  # host-only object
    subprocess.run([bundler, "--unbundle", "--type=o", f"--input={base}.fat",
                    f"--targets={TARGET}", f"--output={base}.co"], check=True)
    notes = subprocess.run([readelf, "--notes", f"{base}.co"], check=True, capture_output=True,
                           text=True).stdout
    kernels, cur = [], None
    for line in notes.splitlines():
        if re.match(r"^  - \.", line):  # a new entry of amdhsa.kernels
            cur = {}
            kernels.append(cur)
            line = "    " + line[4:]
        m = re.match(r"^    \.(\w+):\s+(\S+)", line)
        if m and cur is not None:
            cur[m.group(1)] = m.group(2)
    return [k for k in kernels if "name" in k]


def _waits_of(obj, tmp):
    """Number of `s_waitcnt vmcnt(0)` per kernel in obj's gfx950 code (the
    code object extracted by _kernels_of, disassembled)."""
    co = os.path.join(tmp, os.path.basename(obj)) + ".co"
    dis = subprocess.run([_tool("llvm-objdump"), "-d", "--no-show-raw-insn", co], check=True,
                         capture_output=True, text=True).stdout
    out, name = {}, None
    for line in dis.splitlines():
        m = re.match(r"^[0-9a-f]+ <(\S+)>:", line)
        if m:
            name = m.group(1)
            out[name] = 0
        elif name and "s_waitcnt vmcnt(0)" in line:
            out[name] += 1
    return out


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    objs = sorted(glob.glob(os.path.join(BUILD, "*.o")))
    if not objs:
        pytest.skip("no build objects: run __graft_entry__.build() first")
    if not all(_tool(t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readelf")):
        pytest.skip("ROCm LLVM tools not found")
    tmp = str(tmp_path_factory.mktemp("co"))
    out = {}
    for o in objs:
        ks = _kernels_of(o, tmp)
        if ks:
            waits = _waits_of(o, tmp) if _tool("llvm-objdump") else {}
            for k in ks:
                k["vmcnt0"] = waits.get(k["name"])
            out[os.path.basename(o)] = ks
    return out


def test_every_source_with_kernels_was_found(kernels):
    assert {"attention.o", "elementwise.o", "gemm.o", "temb.o"} <= set(kernels)
    assert sum(len(v) for v in kernels.values()) > 40


def test_no_kernel_uses_scratch(kernels):
    """No vector-register spills and no private (scratch) segment: every
    value a kernel holds stays in registers or LDS."""
    bad = [(o, k["name"], k.get("private_segment_fixed_size"), k.get("vgpr_spill_count"))
           for o, ks in kernels.items() for k in ks
           if int(k.get("private_segment_fixed_size", 0)) != 0
           or int(k.get("vgpr_spill_count", 0)) != 0]
    assert not bad, bad


def test_matrix_kernels_fit_two_waves_per_simd(kernels):
    """The GEMM and attention kernels (8 waves per workgroup for the
    d = 128 attention and the GEMMs) need at most 256 registers per lane
    (VGPRs + AGPRs) so that two waves share each SIMD, and the GEMM's
    staging ring takes the whole 160 KB of LDS."""
    seen = 0
    for ks in kernels.values():
        for k in ks:
            if "gemm_bf16_kernel" in k["name"] or "attn_bf16_kernel" in k["name"]:
                seen += 1
                regs = int(k["vgpr_count"]) + int(k.get("agpr_count", 0))
                assert regs <= 256, (k["name"], regs)
                if "gemm_bf16_kernel" in k["name"]:
                    assert int(k["group_segment_fixed_size"]) == 160 * 1024, k["name"]
    assert seen >= 10


# Most full memory waits a hot kernel may contain.  A load under a bounds
# guard together with its use (or a load still in flight where guarded
# stores begin) turns into one wait per element, and such a kernel shows
# tens to hundreds of them; batched kernels wait a handful of times.
WAIT_BUDGET = {"gemm_bf16_kernel": 10, "attn_bf16_kernel": 8, "ln_modulate_kernel": 3,
               "temni_drift_kernel": 4, "cache_kernel": 4, "l1_partials_kernel": 3}


def test_hot_kernels_keep_memory_in_flight(kernels):
    checked = 0
    for ks in kernels.values():
        for k in ks:
            for key, budget in WAIT_BUDGET.items():
                if key in k["name"] and k.get("vmcnt0") is not None:
                    checked += 1
                    assert k["vmcnt0"] <= budget, (k["name"], k["vmcnt0"], budget)
    if checked == 0:
        pytest.skip("llvm-objdump not found")
    assert checked >= 30
