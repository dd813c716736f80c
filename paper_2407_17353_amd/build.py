"""Build of the HIP library libscalify.so for gfx950 (MI355X).

Every .hip source under csrc/ is compiled by hipcc in parallel and linked into
one shared library next to this file. Packed-fp32 instructions are disabled
for all device code.

The one-wave-per-SIMD GEMM kernels keep their accumulators in AGPRs that only
their inline asm names (AccTile in csrc/gemm_kernel.h); the compiler does not
know these registers hold values. The build therefore disassembles the GEMM
objects and fails if, in any kernel that uses those accumulators, any
instruction other than the accumulator asm's own forms (an MFMA whose
destination and C operand are the same a[n:n+3], a write of 0, a read into a
VGPR) names an AGPR -- the compiler spilling into AGPRs or using one as the
data of a load or an MFMA operand -- or the kernel uses scratch memory.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libscalify.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument", "-Wno-pass-failed",
]


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _llvm(tool: str) -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "llvm", "bin", tool)


_KERNEL = re.compile(r"^[0-9a-f]+ <(\S+)>:$")
_AGPR_MFMA = re.compile(r"v_mfma\S* a\[")
_ANY_AGPR = re.compile(r"\ba\d+\b|\ba\[\d+:\d+\]")
# The only instructions that may name an AGPR in a kernel whose accumulators
# the inline asm holds: the asm's MFMA on an accumulator tile (destination and
# C operand the same a[n:n+3]), its zeroing write and its read into a VGPR.
_ASM_MFMA = re.compile(r"^v_mfma\S*\s+(a\[\d+:\d+\]),\s*v\[\d+:\d+\],\s*v\[\d+:\d+\],\s*(a\[\d+:\d+\])")
_ASM_ZERO = re.compile(r"^v_accvgpr_write_b32\s+a\d+,\s*0\s*$")
_ASM_READ = re.compile(r"^v_accvgpr_read_b32\s+v\d+,\s*a\d+\s*$")


def _asm_agpr_form(insn: str) -> bool:
    """Whether an instruction that names an AGPR is one of the accumulator
    asm's own forms."""
    m = _ASM_MFMA.match(insn)
    if m:
        # the MFMA's remaining operands (block-scale words, modifiers) name no AGPR
        rest = insn[m.end():]
        return m.group(1) == m.group(2) and not _ANY_AGPR.search(rest)
    return bool(_ASM_ZERO.match(insn) or _ASM_READ.match(insn))


def check_accumulator_isolation(obj: str, tmp: str) -> int:
    """Disassemble the gfx950 code of one object and check every kernel that
    keeps accumulators in asm-named AGPRs. Returns the number of such
    kernels; raises RuntimeError on a violation."""
    base = os.path.join(tmp, os.path.basename(obj))
    subprocess.run([_llvm("llvm-objcopy"), f"--dump-section=.hip_fatbin={base}.fatbin", obj],
                   check=True, capture_output=True)
    subprocess.run([_llvm("clang-offload-bundler"), "--unbundle", "--type=o",
                    f"--input={base}.fatbin", f"--targets=hipv4-amdgcn-amd-amdhsa--{ARCH}",
                    f"--output={base}.co"], check=True, capture_output=True)
    dis = subprocess.run([_llvm("llvm-objdump"), "-d", f"--mcpu={ARCH}", f"{base}.co"],
                         check=True, capture_output=True, text=True).stdout
    kernels = {}
    name = None
    for line in dis.splitlines():
        m = _KERNEL.match(line)
        if m:
            name = m.group(1)
            kernels[name] = []
        elif name is not None:
            kernels[name].append(line)
    checked = 0
    for name, body in kernels.items():
        if not any(_AGPR_MFMA.search(l) for l in body):
            # Every other function (the 8-wave kernels, and the out-of-line
            # casts the 4-wave epilogues call while accumulators still sit in
            # AGPRs) must leave AGPRs alone.
            bad = [l.strip() for l in body if _ANY_AGPR.search(l.split("//")[0])]
            if bad:
                raise RuntimeError(f"{obj}: function {name} uses AGPRs: {bad[:4]}")
            continue
        checked += 1
        bad = []
        for line in body:
            insn = line.split("//")[0].strip()
            if "scratch_" in insn:
                bad.append(insn)
            elif _ANY_AGPR.search(insn) and not _asm_agpr_form(insn):
                bad.append(insn)
        if bad:
            raise RuntimeError(f"{obj}: kernel {name} has compiler-placed AGPR or scratch "
                               f"accesses next to the asm-held accumulators: {bad[:4]}")
    return checked


def build(verbose: bool = False) -> str:
    """Compile the library (always recompiles). Returns its path."""
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with tempfile.TemporaryDirectory(prefix="scalify_build_") as tmp:
        def compile_one(src: str) -> str:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [_hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
            if verbose and r.stderr.strip():
                print(r.stderr)
            if os.path.basename(src).startswith("gemm_"):
                check_accumulator_isolation(obj, tmp)
            return obj

        workers = min(len(sources), max(1, os.cpu_count() or 1), 8)
        with cf.ThreadPoolExecutor(workers) as ex:
            objs = list(ex.map(compile_one, sources))
        tmp_lib = LIB + ".tmp"
        cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp_lib, *objs]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr}")
        os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
