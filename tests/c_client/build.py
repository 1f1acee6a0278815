"""Builds the C99 test client of the library (gcc; links the in-tree
libflashvla.so and the HIP runtime)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
LIBDIR = os.path.join(ROOT, "paper_2608_27384_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build_client(out_path: str) -> None:
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror=implicit-function-declaration",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           "-D__HIP_PLATFORM_AMD__", os.path.join(HERE, "decode_client.c"),
           "-L", LIBDIR, "-lflashvla", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{LIBDIR}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", out_path]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
