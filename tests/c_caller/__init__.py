"""Build helper of the plain C caller (realq_layer_c.c): gcc, the HIP runtime's C API and
librealq.so, nothing else."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
SRC = os.path.join(ROOT, "tests", "c_caller", "realq_layer_c.c")
LIBDIR = os.path.join(ROOT, "paper_2609_00049_amd")


def compile_c_caller(out_path):
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           f"-I{os.path.join(ROOT, 'include')}", SRC, "-o", str(out_path), "-L/opt/rocm/lib", "-lamdhip64",
           f"-L{LIBDIR}", "-lrealq", f"-Wl,-rpath,{LIBDIR}", "-Wl,-rpath,/opt/rocm/lib"]
    return subprocess.run(cmd, capture_output=True, text=True)
