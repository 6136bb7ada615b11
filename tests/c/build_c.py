"""Build the C test programs of this folder with gcc (host code only; the
GPU work runs inside liblogo.so).  ``build()`` compiles layer_from_c.c into
layer_from_c.bin, linked against the in-tree liblogo.so (found through an
rpath relative to the binary) and the HIP runtime."""
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
LAYER_BIN = os.path.join(HERE, "layer_from_c.bin")


def build() -> str:
    gcc = shutil.which("gcc")
    if gcc is None:
        raise RuntimeError("gcc not found: needed for the C test programs")
    cmd = [gcc, "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           os.path.join(HERE, "layer_from_c.c"),
           "-L", os.path.join(ROOT, "paper_2608_29539_amd"), "-llogo",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2608_29539_amd",
           "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", LAYER_BIN]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("building layer_from_c failed:\n" + r.stderr)
    return LAYER_BIN


if __name__ == "__main__":
    print(build())
