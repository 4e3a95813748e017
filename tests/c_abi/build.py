"""Build the plain C GPU caller of the ABI (tests/c_abi/abi_gpu_check) with
gcc against the in-tree libasrkf.so and the HIP runtime.  Called by
__graft_entry__.build(); the GPU test only runs the binary."""
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
EXE = os.path.join(HERE, "abi_gpu_check")


def build():
    gcc = shutil.which("gcc")
    if gcc is None:
        raise RuntimeError("gcc not found")
    lib_dir = os.path.join(ROOT, "paper_2512_11221_amd")
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-O2", "-D__HIP_PLATFORM_AMD__",
           os.path.join(HERE, "abi_gpu_check.c"), "-I", os.path.join(ROOT, "include"),
           "-I", "/opt/rocm/include", "-L", lib_dir, "-l:libasrkf.so", "-L", "/opt/rocm/lib",
           "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/../../paper_2512_11221_amd",
           "-Wl,-rpath,/opt/rocm/lib", "-Wl,-rpath-link,/opt/rocm/lib", "-o", EXE + ".tmp"]
    subprocess.run(cmd, check=True, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    os.replace(EXE + ".tmp", EXE)
    return EXE


if __name__ == "__main__":
    print(build())
