"""Build libtrevs.so (the HIP library behind include/trevs.h) for gfx950.

Run as `python -m paper_2609_37581_amd.build` or call build().  Each HIP
source is compiled to an object in parallel, then linked into the package
directory; the result replaces any previous library atomically."""

import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtrevs.so")
ARCH = "gfx950"


def hipcc():
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return cand if os.path.exists(cand) else shutil.which("hipcc") or "hipcc"


def flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include")]


def _compile(src, obj, extra=()):
    cmd = [hipcc()] + flags() + list(extra) + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)}:\n{r.stderr}")
    return obj


def build(verbose=True, extra_flags=(), out=LIB):
    """Compile every HIP source and link `out` (default: the package library).
    extra_flags are passed to every hipcc compile (e.g. -D tile overrides)."""
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with tempfile.TemporaryDirectory(prefix="trevs_build_") as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            list(ex.map(lambda so: _compile(so[0], so[1], extra_flags), zip(srcs, objs)))
        dest = out
        lib_tmp = os.path.join(tmp, "libtrevs.so")
        cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", lib_tmp] + objs
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode:
            raise RuntimeError("link failed:\n" + r.stderr)
        shutil.move(lib_tmp, dest + ".tmp")
        os.replace(dest + ".tmp", dest)
    if verbose:
        print(f"built {dest}")
    return dest


if __name__ == "__main__":
    build()
    sys.exit(0)
