"""Build ``_lib/libhwkv.so`` (the C-ABI library) for gfx950 with hipcc, and
``_lib/libhwkv_probe.so``, the read-bandwidth probe the benchmark loads
beside the decode roofline (measurement tooling, not part of the ABI).

Every call recompiles all sources (in parallel), then links.  HIP code is
compiled with packed fp32 instructions disabled.
"""
import concurrent.futures as cf
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "hwkv")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libhwkv.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["hwkv_api.hip", "decode_kernels.hip", "decode_split_bf16.hip",
           "decode_split_f16.hip", "decode_split_fp8.hip", "write_kernels.hip",
           "prefill_attn_kernels.hip", "calib_kernels.hip"]
PROBE_SOURCE = os.path.join("probe", "read_probe.hip")
PROBE_LIB = os.path.join(LIBDIR, "libhwkv_probe.so")

CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-source hipcc flags beyond CFLAGS (none at present).
SOURCE_FLAGS = {}


def flags_for(src):
    """hipcc flags of one source (the common flags and its own)."""
    return [*CFLAGS, *SOURCE_FLAGS.get(src, [])]


def _compile(src, verbose):
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    os.makedirs(os.path.dirname(obj), exist_ok=True)
    cmd = [HIPCC, *flags_for(src), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Builds both libraries; returns the path of libhwkv.so."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    srcs = SOURCES + [PROBE_SOURCE]
    with cf.ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    _link(objs[:-1], LIB, verbose)
    _link(objs[-1:], PROBE_LIB, verbose)
    return LIB


# The CPU tests' sanitizer build: the same sources with AddressSanitizer and
# UndefinedBehaviorSanitizer on the host code only (device code is compiled
# as usual and never runs on the CPU), linked against clang's shared
# sanitizer runtime, which the loading process must preload.
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SAN_HOST_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_LINK_FLAGS = ["-fsanitize=address,undefined", "-shared-libsan"]


def sanitizer_runtime() -> str:
    """Path of the shared sanitizer runtime the sanitizer build needs."""
    r = subprocess.run([CLANGXX, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True, check=True)
    return r.stdout.strip()


def build_host_sanitized(out_dir: str, verbose: bool = False) -> str:
    """Builds libhwkv.so's sources into ``out_dir``/libhwkv_san.so with the
    host sanitizers on; returns its path."""
    os.makedirs(out_dir, exist_ok=True)

    def one(src):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        flags = [f for f in flags_for(src) if f != "-O3"]
        cmd = [HIPCC, *flags, "-O1", "-g", *SAN_HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(one, SOURCES))
    lib = os.path.join(out_dir, "libhwkv_san.so")
    cmd = [CLANGXX, "-shared", "-fPIC", *SAN_LINK_FLAGS, *objs, "-L/opt/rocm/lib",
           "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64", "-o", lib]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
