"""Build tests/c_driver/libgsq_c_driver.so: the plain C user of the GSQ library that
tests/test_gpu_c_driver.py loads.  gcc, C99, linked against libgsq.so and the HIP runtime (no
torch).  Called by __graft_entry__.build() after libgsq.so, and runnable on its own:
``python tests/c_driver/build_c_driver.py``."""
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "gsq_c_driver.c")
OUT = os.path.join(HERE, "libgsq_c_driver.so")
PKG = os.path.join(ROOT, "paper_2604_18556_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build():
    gcc = shutil.which("gcc")
    if not gcc:
        raise RuntimeError("gcc not found: the C driver of the GPU tests needs it")
    cmd = [gcc, "-std=c99", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC,
           "-o", OUT + ".tmp", "-L", PKG, "-lgsq", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-lm", "-Wl,-rpath,$ORIGIN/../../paper_2604_18556_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("building the C driver failed:\n" + r.stderr)
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    print(build())
