"""Compile the plain C++ ABI client (tests/c_client/ris_client.cpp) against the
built libris.so into _build/libris_client.so.  Host code only; run by the build
step so that GPU tests only call it."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2607_21927_amd")
OUT = os.path.join(ROOT, "_build", "libris_client.so")


def build(verbose=False):
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), "-O2", "-std=c++17", "-shared", "-fPIC",
           "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "ris_client.cpp"),
           "-L", PKG, "-lris", "-Wl,-rpath,$ORIGIN/../paper_2607_21927_amd", "-o", OUT]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building the ABI client failed:\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
