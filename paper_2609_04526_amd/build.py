"""Build libscaleqlora.so in-tree with hipcc for gfx950.

    python -m paper_2609_04526_amd.build

Compiles every .hip source under csrc/ (one hipcc process per source, in
parallel) and links them into one shared library next to this file.  Always
recompiles."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libscaleqlora.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-fvisibility=hidden",
    # codec, merge and re-quantisation steps are defined as separately rounded
    # fp32 operations: never contract a*b+c into a fused multiply-add
    "-ffp-contract=off",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src, obj, extra):
    cmd = [HIPCC, *FLAGS, *extra, "-c", "-o", obj, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    return cmd, res


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every .hip source to an object (in parallel), then link the
    shared library.  `defines` adds -D flags (probe builds only)."""
    import concurrent.futures
    import tempfile
    extra = [f"-D{d}" for d in defines]
    with tempfile.TemporaryDirectory(prefix="sq_build_") as tmpdir:
        srcs = sources()
        objs = [os.path.join(tmpdir, os.path.basename(src) + ".o") for src in srcs]
        with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            results = list(ex.map(lambda so: _compile(so[0], so[1], extra), zip(srcs, objs)))
        for cmd, res in results:
            err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
            if verbose:
                print(" ".join(cmd), flush=True)
            if res.returncode != 0:
                raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
        tmp = out + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed ({res.returncode}):\n{res.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
