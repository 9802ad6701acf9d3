"""Build step for the HIP library: compiles csrc/*.hip for gfx950 into
_lib/libsbvr.so (in-tree, so the built library travels with the source).
``defines`` (NAME=VALUE) override launch-shape tuning macros for sweeps."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("api.hip", "pack.hip", "gemv_b1.hip", "gemv_b1s.hip", "gemm_sbs.hip",
                                                  "decompress.hip", "encode.hip", "prefill.hip")]
# The encoder's binary64 arithmetic is its definition: no fused multiply-add.
SOURCE_FLAGS = {
    "encode.hip": ["-ffp-contract=off"],
    # leading scalar kernel arguments preloaded into SGPRs (batch-1 kernels)
    "gemv_b1.hip": ["-mllvm", "-amdgpu-kernarg-preload-count=8"],
    "gemv_b1s.hip": ["-mllvm", "-amdgpu-kernarg-preload-count=10"],
}
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-result",
    # never emit packed-fp32 VALU instructions (v_pk_{add,mul,fma}_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def library_path() -> str:
    return os.path.join(HERE, "_lib", "libsbvr.so")


def probe_path() -> str:
    """The streaming-read measurement helper the benchmark loads (not part of
    the library)."""
    return os.path.join(HERE, "_lib", "libsbvr_probe.so")


def build_probe(verbose: bool = False) -> str:
    out = probe_path()
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *FLAGS, os.path.join(HERE, "csrc", "read_probe.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False, out: str | None = None, defines=(), jobs: int = 0) -> str:
    """Compile every source to an object (in parallel), then link libsbvr.so."""
    from concurrent.futures import ThreadPoolExecutor

    out = out or library_path()
    os.makedirs(os.path.dirname(out), exist_ok=True)
    objdir = os.path.join(os.path.dirname(out), "obj.%d" % os.getpid())
    os.makedirs(objdir, exist_ok=True)
    common = [*FLAGS, *("-D" + d for d in defines), "-I", os.path.join(ROOT, "include"),
              "-I", os.path.join(HERE, "csrc")]

    def run(cmd):
        if verbose:
            print(" ".join(cmd))
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)

    objs = [os.path.join(objdir, os.path.basename(src) + ".o") for src in SOURCES]
    compile_flags = [f for f in common if f != "-shared"]
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1, 8)
    try:
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            list(ex.map(run, [[HIPCC, *compile_flags, *SOURCE_FLAGS.get(os.path.basename(src), []), "-c", src,
                               "-o", obj] for src, obj in zip(SOURCES, objs)]))
        tmp = out + ".tmp%d" % os.getpid()
        run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
        os.replace(tmp, out)
    finally:
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
        if os.path.isdir(objdir):
            os.rmdir(objdir)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_probe(verbose=True))
