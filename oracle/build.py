"""Build the oracle's shared library (plain C, gcc, fp64, no fast-math).

Test infrastructure: the oracle is what the tests compare against, never part of the product
path.  ``build()`` compiles it every time it is called.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [
        "gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
        "-fPIC", "-shared", "-Wall", "-Wextra", "-D_POSIX_C_SOURCE=200809L",
        SRC, "-o", tmp, "-lm", "-lpthread",
    ]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_sanitized(out_dir: str, verbose: bool = False) -> str:
    """The same source with AddressSanitizer and UndefinedBehaviorSanitizer,
    built by clang against its shared sanitizer runtime (the one the
    library's sanitizer build uses, so both load into one process); returns
    the path of ``out_dir``/liboracle_san.so."""
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, "liboracle_san.so")
    cmd = [
        "/opt/rocm/llvm/bin/clang", "-std=c11", "-O1", "-g", "-ffp-contract=off",
        "-fno-fast-math", "-fPIC", "-shared", "-D_POSIX_C_SOURCE=200809L",
        "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
        "-fno-omit-frame-pointer", "-shared-libsan", SRC, "-o", lib, "-lm", "-lpthread",
    ]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
