"""Build the pure-C ABI demo (tests/c_abi/abi_demo.c) with gcc against
include/dqgan.h, libdqgan.so, the C oracle and the HIP runtime's C API."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "abi_demo")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(out=OUT):
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           os.path.join(HERE, "abi_demo.c"), "-o", out,
           "-L", os.path.join(ROOT, "paper_2010_13359_amd"), "-ldqgan",
           "-L", os.path.join(ROOT, "oracle"), "-ldqgan_oracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2010_13359_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib")]
    if out != OUT:  # a copy outside the tree finds the libraries by absolute path
        cmd[-1] = "-Wl,-rpath,%s:%s:%s" % (os.path.join(ROOT, "paper_2010_13359_amd"), os.path.join(ROOT, "oracle"),
                                           os.path.join(ROCM, "lib"))
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError("gcc failed:\n" + res.stdout)
    return out


if __name__ == "__main__":
    print(build())
