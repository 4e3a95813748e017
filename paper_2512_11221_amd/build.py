"""Build libasrkf.so (the HIP kernels + C ABI) for gfx950 with hipcc, in-tree."""
import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libasrkf.so")
SOURCES = ["attention.hip", "relevance.hip", "compact.hip", "entropy.hip", "xfer.hip", "runtime.hip"]
ARCH = "gfx950"
# no packed fp32 instructions anywhere in the device code
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# roctx ranges over the ABI calls (marker traces)
LINK = ["-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def compile_shared(sources, out, extra=(), cwd=None):
    fd, tmp = tempfile.mkstemp(suffix=".so", dir=os.path.dirname(out))
    os.close(fd)
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           *DEVICE_FLAGS, *extra, *sources, *LINK, "-o", tmp]
    try:
        subprocess.run(cmd, check=True, cwd=cwd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    except subprocess.CalledProcessError as e:
        os.unlink(tmp)
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + e.stdout.decode(errors="replace"))
    os.replace(tmp, out)
    return out


def build():
    return compile_shared([os.path.join(CSRC, s) for s in SOURCES], LIB)


def build_sanitized(kinds=("address", "undefined"), out=None):
    """The same library with the host code (the runtime and the launch code)
    built under clang sanitizers; the device code is compiled as usual.  An
    AddressSanitizer build needs the sanitizer runtime preloaded into the host
    process.  Returns the path of the library (default: libasrkf_<kinds>.so
    next to libasrkf.so); load it through ASRKF_LIBRARY."""
    extra = []
    for k in kinds:
        extra += ["-Xarch_host", f"-fsanitize={k}"]
    extra += ["-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-shared-libsan"]
    import glob
    rt_dirs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux"))
    if rt_dirs:                                   # find the sanitizer runtimes at load time
        extra += [f"-Wl,-rpath,{rt_dirs[-1]}"]
    out = out or os.path.join(HERE, "libasrkf_" + "_".join(kinds) + ".so")
    return compile_shared([os.path.join(CSRC, s) for s in SOURCES], out, extra=extra)


if __name__ == "__main__":
    import sys
    if len(sys.argv) > 1 and sys.argv[1] == "--sanitize":
        print(build_sanitized(tuple(sys.argv[2].split(",")) if len(sys.argv) > 2
                              else ("address", "undefined")))
    else:
        print(build())
