"""Build the plain-C client of the C ABI (test infrastructure) with gcc."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
EXE = os.path.join(HERE, "hg_c_roundtrip")
PKG = os.path.join(ROOT, "paper_2609_35800_amd")


def command(out: str):
    return ["gcc", "-std=c11", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
            f"-I{os.path.join(ROOT, 'include')}", f"-I{ROCM}/include",
            os.path.join(HERE, "roundtrip.c"), "-o", out,
            f"-L{PKG}", "-lheadguard", f"-Wl,-rpath,{PKG}",
            f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib"]


def build(out: str = EXE) -> str:
    tmp = out + ".tmp"
    subprocess.check_call(command(tmp))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
