"""Build the device arithmetic probes (test infrastructure) for gfx950."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
LIB = os.path.join(HERE, "libhg_probes.so")


def build() -> str:
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "hg_build", os.path.join(ROOT, "paper_2609_35800_amd", "build.py"))
    hg_build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(hg_build)  # not the package: its __init__ loads the library
    FLAGS = hg_build.FLAGS
    tmp = LIB + ".tmp"
    subprocess.check_call([os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), *FLAGS, "-shared", "-o", tmp,
                           os.path.join(HERE, "hg_probes.hip")])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
