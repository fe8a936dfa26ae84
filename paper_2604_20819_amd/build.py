"""Build libcqsa.so (HIP kernels for gfx950 + the C ABI) in-tree with hipcc.

Usage: python -m paper_2604_20819_amd.build   (or build() from Python)
"""
import concurrent.futures
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "libcqsa.so")
OBJ = os.path.join(PKG, "_build")

ARCH = "gfx950"
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep packed-fp32 VALU forms out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function",
]
SOURCES = [
    "plan.cpp", "capi_plan.cpp", "runtime.cpp", "fwd_driver.cpp", "bwd_driver.cpp", "guard.cpp",
    "attn_fwd.hip", "merge.hip", "attn_bwd.hip", "stage.hip",
]


def hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the HIP build needs ROCm")
    return exe


def _compile(src):
    path = os.path.join(CSRC, src)
    obj = os.path.join(OBJ, src + ".o")
    lang = ["-x", "hip"]
    cmd = [hipcc()] + COMMON + lang + ["-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj, r.stderr


def device_asm(src):
    """gfx950 assembly of one .hip source, compiled with the build's flags."""
    path = os.path.join(CSRC, src)
    cmd = [hipcc()] + COMMON + ["-x", "hip", "--cuda-device-only", "-S", path, "-o", "-"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    return r.stdout


def masked_spill_stores(asm):
    """Kernels of `asm` with a register spill stored right before an exec
    restore (s_or_b64 exec, exec, ...) in the same basic block: the store then
    runs under the closing branch's partial exec mask, so lanes (or whole
    waves) that skipped the branch lose the spilled value.  The compiler has
    emitted this for a kernel at its register limit; returns {kernel: count}."""
    out = {}
    for m in re.finditer(r"\n(_Z\S+):[^\n]*\n(.*?)\.Lfunc_end", asm, re.S):
        name, lines = m.group(1), m.group(2).split("\n")
        n = 0
        for k, line in enumerate(lines):
            if "scratch_store" not in line:
                continue
            for nxt in lines[k + 1:k + 8]:
                t = nxt.strip()
                if not t or t.startswith(";") or t.startswith("scratch_store"):
                    continue
                if re.match(r"s_or_b64 exec, exec,", t):
                    n += 1
                break
        if n:
            out[name] = n
    return out


def build(verbose=False):
    """Compile every source (always) and link libcqsa.so in the package dir."""
    os.makedirs(OBJ, exist_ok=True)
    srcs = [s for s in SOURCES if os.path.exists(os.path.join(CSRC, s))]
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(_compile, srcs))
    objs = [o for o, _ in results]
    if verbose:
        for (_, err), s in zip(results, srcs):
            if err.strip():
                print(f"--- {s}\n{err}", file=sys.stderr)
    tmp = OUT + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs + ["-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # A kernel whose host-side instantiation the compiler dropped links as an
    # undefined launch stub; refuse such a library instead of shipping it.
    nm = shutil.which("nm")
    if nm:
        syms = subprocess.run([nm, "-D", tmp], capture_output=True, text=True).stdout
        missing = [ln.split()[-1] for ln in syms.splitlines()
                   if " U " in ln and "__device_stub__" in ln]
        if missing:
            os.remove(tmp)
            raise RuntimeError("kernel launch stubs missing from the library: " + ", ".join(missing))
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
