"""Build ``libspingtp.so`` (HIP kernels + C ABI) in-tree for gfx950 with hipcc."""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libspingtp.so")
SOURCES = ["plan.cpp", "api.cpp", "forward.hip", "forward_big_parity.hip", "forward_big_padded.hip",
           "forward_big_parity_padded.hip", "forward_mfma.hip", "forward_pre.hip",
           "forward_pre_large.hip", "forward_pre_weighted.hip", "forward_direct.hip", "backward.hip", "backward_v1w.hip", "forward_uvw.hip"]
# per-source additions: the parity-basis large-degree kernels schedule for fewer registers
# (they spill less and run 22-35 % faster that way; the other kernels run slower with it)
_MINREG = ["-mllvm", "-amdgpu-sched-strategy=iterative-minreg"]
EXTRA_FLAGS = {"forward_big_parity.hip": _MINREG, "forward_big_parity_padded.hip": _MINREG}

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in generated code.
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found")
    return path


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source to an object (in parallel), then link the shared library."""
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs, objs = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmd = [hipcc()] + HIP_FLAGS + EXTRA_FLAGS.get(src, []) + ["-I", os.path.join(ROOT, "include"), "-c",
                                                                  os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd.insert(1, "-x")
            cmd.insert(2, "hip")
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        msg = "\n".join(f"--- {s} ---\n{t}" for s, t in failed)
        raise RuntimeError("hipcc failed:\n" + msg)
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


# host code checked by AddressSanitizer and UndefinedBehaviorSanitizer (device code is
# built as usual: -Xarch_host applies the flags to the host compilation only)
SANITIZED_SOURCES = ("plan.cpp", "api.cpp")
SANITIZE_FLAGS = ("-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
                  "-Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer "
                  "-Xarch_host -g").split()


def sanitizer_runtime() -> str:
    """The shared AddressSanitizer runtime of this toolchain (LD_PRELOAD for a Python host)."""
    out = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                         text=True).stdout.strip()
    if not out or not os.path.exists(out):
        import glob
        hits = glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        out = hits[0] if hits else ""
    if not out:
        raise RuntimeError("AddressSanitizer runtime not found")
    return out


def build_sanitized() -> str:
    """A copy of the library whose host table builders and entry points run under the
    sanitizers, at _build/sanitized/libspingtp.so (the kernels' objects are the regular ones)."""
    objdir = os.path.join(ROOT, "_build")
    sdir = os.path.join(objdir, "sanitized")
    os.makedirs(sdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        if src in SANITIZED_SOURCES:
            obj = os.path.join(sdir, os.path.splitext(src)[0] + ".o")
            cmd = [hipcc(), "-x", "hip"] + HIP_FLAGS + list(SANITIZE_FLAGS) + ["-I", os.path.join(ROOT, "include"), "-c",
                                                                        os.path.join(CSRC, src), "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError("hipcc failed:\n" + r.stdout + r.stderr)
        else:
            obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
            if not os.path.exists(obj):
                build()
        objs.append(obj)
    lib = os.path.join(sdir, "libspingtp.so")
    subprocess.run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", lib] + objs, check=True)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
