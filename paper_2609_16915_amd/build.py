"""Build librosetta.so (HIP kernels for gfx950 + the C ABI) in-tree.

    python -m paper_2609_16915_amd.build [-v]

Always recompiles.  The library lands next to this file, where the Python
binding loads it from.
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "librosetta.so")
SOURCES = ["kernels.hip", "keyswitch.hip", "lwe_ops.hip", "abi.cpp", "noalloc.hip",
           "host_helpers.cpp", "seglut.cpp", "lookup.cpp"]
ARCH = os.environ.get("ROSETTA_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
         # packed fp32 instructions are kept out of all device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-ffp-contract=off", "-Wall", "-Wno-unused-result",
         f"-I{INCLUDE}", f"-I{CSRC}"]


# Device-code scheduling of the transform kernels (kernels.hip): LLVM's
# iterative ILP scheduler interleaves the independent field products of the
# transform passes (the default occupancy-first strategy runs them back to
# back, and their carry chains then leave the VALU idle between dependent
# instructions); the register budget, and with it the waves per SIMD, stays
# the same.  keyswitch.hip keeps the default, which suits it better.
TRANSFORM_FLAGS = ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]


def source_digest() -> str:
    """First 16 hex digits of the SHA-256 over every source the library is
    built from (csrc/ and include/rosetta.h: each file's name, then its
    bytes, in name order).  The build bakes it into rosetta_version(), so a
    loaded library names the sources it was compiled from."""
    import hashlib
    files = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                   if f.endswith((".hip", ".cpp", ".hpp", ".h")))
    files.append(os.path.join(INCLUDE, "rosetta.h"))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode() + b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _flags(src: str, digest: str):
    return (FLAGS + [f'-DROSETTA_SOURCE_DIGEST="{digest}"'] +
            (TRANSFORM_FLAGS if src == "kernels.hip" else []))


def _filter(stderr: str) -> str:
    return "\n".join(l for l in (stderr or "").splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False) -> str:
    """Compile every source to an object (in parallel), then link."""
    import concurrent.futures
    import tempfile
    with tempfile.TemporaryDirectory(prefix="rosetta_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        digest = source_digest()
        cmds = [[hipcc(), *_flags(s, digest), "-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        with concurrent.futures.ThreadPoolExecutor(len(cmds)) as ex:
            results = list(ex.map(lambda c: subprocess.run(c, capture_output=True, text=True),
                                  cmds))
        for src, res in zip(SOURCES, results):
            if res.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src} ({res.returncode}):\n"
                                   f"{_filter(res.stderr)}")
            if verbose and _filter(res.stderr).strip():
                print(_filter(res.stderr), flush=True)
        tmp = LIB + ".tmp"
        link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
        res = subprocess.run(link, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed ({res.returncode}):\n{_filter(res.stderr)}")
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
