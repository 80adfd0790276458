"""Builds libfp8q.so (the HIP kernels and the C-ABI) for gfx950 with hipcc."""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libfp8q.so")
SOURCES = ["abi.hip", "quantize.hip", "gemm.hip", "clip.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    # packed fp32 instructions stay off (the host pass warns it does not
    # know the feature; that is harmless)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-I", INCLUDE, "-I", CSRC,
]
# Per-source additions.  GEMM: matrix-instruction results in ordinary VGPRs
# (the compiler otherwise puts the 128 x 128 and 64 x 64 tiles' partials in
# AGPRs, and every promotion FMA then waits for a v_accvgpr_read copy).
EXTRA = {"gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def check_no_scratch(src, remarks):
    """The tiled GEMM kernels read LDS with inline asm whose results are only
    valid after an explicit wait; a register spill could copy such a value
    early (and a spill in any GEMM kernel costs its memory path).  Refuse a
    build in which any GEMM kernel uses scratch memory."""
    name = None
    for line in remarks.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "ScratchSize [bytes/lane]:" in line and name and "gemm" in name:
            size = int(line.split("ScratchSize [bytes/lane]:")[1].split()[0])
            if size != 0:
                raise RuntimeError("%s: %s spills to scratch (%d bytes per lane)" % (src, name, size))


def build():
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        cmd = [HIPCC] + FLAGS + EXTRA.get(src, []) + ["-Rpass-analysis=kernel-resource-usage", "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed for %s:\n%s" % (src, r.stderr))
        check_no_scratch(src, r.stderr)
        return obj

    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s" % r.stderr)
    # every symbol must resolve (a missing kernel stub only shows at load)
    r = subprocess.run(["python3", "-c", "import ctypes, sys; ctypes.CDLL(sys.argv[1])", tmp],
                       capture_output=True, text=True)
    if r.returncode != 0:
        os.unlink(tmp)
        raise RuntimeError("built library does not load:\n%s" % r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
