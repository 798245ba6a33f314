"""Build step for libclq.so (HIP, gfx950).

Compiles every source under ``csrc/`` with hipcc into one shared library next
to this file.  Flags:
  --offload-arch=gfx950     the only target
  -O3 -ffp-contract=off     no implicit fma contraction: every fp32 add, sub
                            and mul rounds as written; fmas are explicit
  -Xclang -target-feature -Xclang -packed-fp32-ops
                            no packed fp32 vector ops
No fast-math flags: fp32 division and square root stay correctly rounded and
denormals are kept.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libclq.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include")]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _run(cmd):
    proc = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so: harmless
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    err = "\n".join(l for l in proc.stderr.splitlines() if noise not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"hipcc failed ({proc.returncode}):\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")


def build(extra_flags=(), out=LIB, objdir=None):
    """Compile libclq.so (one object per source, compiled in parallel, then
    linked); returns its path.  extra_flags go to every compile and to the
    link."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = objdir or os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(objdir, os.path.basename(f) + ".o") for f in srcs]
    compile_flags = [f for f in FLAGS if f != "-shared"]
    jobs = min(len(srcs), max(1, min(os.cpu_count() or 1, 8)))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(lambda so: _run([HIPCC, *compile_flags, *extra_flags, "-c", so[0], "-o", so[1]]),
                    zip(srcs, objs)))
    tmp = out + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *extra_flags, *objs, "-o", tmp])
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
