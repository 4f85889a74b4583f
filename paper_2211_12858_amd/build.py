"""Build libsketchboost.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2211_12858_amd.build
"""
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsketchboost.so")

HIPCC_FLAGS = [
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "--offload-arch=gfx950",
    # packed fp32 VALU forms are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no a*b+c contraction: the sketch is bit-reproducible against IEEE single ops
    "-ffp-contract=off",
    "-Wall",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose=False):
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    tmp = LIB + ".tmp"
    cmd = [hipcc()] + HIPCC_FLAGS + ["-o", tmp] + srcs
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature; that warning is harmless
    noise = [ln for ln in res.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln]
    if res.returncode != 0:
        sys.stderr.write("\n".join(noise) + "\n")
        raise RuntimeError("hipcc failed with exit code %d" % res.returncode)
    if noise and verbose:
        sys.stderr.write("\n".join(noise) + "\n")
    os.replace(tmp, LIB)
    return LIB


# Host-side sanitizer build: the library with AddressSanitizer and UBSan
# on its host code (the validation layer and the launch plumbing); the
# device code is built as usual.  Each -fsanitize applies to the host pass
# only (-Xarch_host).  The ABI tests run against it without a GPU: every
# call they make is refused on the host.
SANITIZE_FLAGS = [
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined",
    "-Xarch_host", "-fno-omit-frame-pointer",
]


def build_host_sanitized(out_path, jobs=8):
    """Build the sanitized library at out_path: one object per source, compiled in parallel, then linked."""
    import concurrent.futures

    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    flags = [f for f in HIPCC_FLAGS if f != "-shared"] + ["-g"] + SANITIZE_FLAGS
    objs = [out_path + "." + os.path.basename(src) + ".o" for src in srcs]

    def run(cmd):
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stderr[-4000:] + "\n")
            raise RuntimeError("hipcc (host sanitizer build) failed with exit code %d" % res.returncode)

    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as pool:
        list(pool.map(run, [[hipcc()] + flags + ["-c", "-o", o, src] for src, o in zip(srcs, objs)]))
    run([hipcc(), "-shared", "--offload-arch=gfx950"] + SANITIZE_FLAGS + ["-o", out_path] + objs)
    for o in objs:
        os.remove(o)
    return out_path


def sanitizer_runtime():
    """Path of the clang AddressSanitizer runtime that the sanitized build needs preloaded."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    res = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = res.stdout.strip()
    return path if res.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


if __name__ == "__main__":
    print(build(verbose=True))
