"""CPU sanitizer tier: the oracle's pins and the host-side ABI tests, run
again against AddressSanitizer + UndefinedBehaviorSanitizer builds of
``oracle.c`` and of the library's host code (artifact parser, page-pool
bookkeeping, layout and workspace arithmetic, argument checks).

Both builds link clang's shared sanitizer runtime; the child pytest process
preloads it and loads the sanitizer builds in place of the usual ones
(``HWKV_LIBRARY``, ``HWKV_ORACLE_LIBRARY``).  Any sanitizer report aborts
the child (no recovery), so a clean exit with every test passed is the bar.
No GPU is touched: the library's host paths reject or finish before any
device work in these tests.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

SAN_DIR = os.path.join(ROOT, "_build", "san")


@pytest.fixture(scope="module")
def san_env():
    from oracle import build as ob
    from paper_2609_02029_amd import build as pb
    rt = pb.sanitizer_runtime()
    if not os.path.isabs(rt) or not os.path.exists(rt):
        pytest.skip("clang's shared sanitizer runtime is not installed")
    lib = pb.build_host_sanitized(SAN_DIR)
    olib = ob.build_sanitized(SAN_DIR)
    env = dict(os.environ)
    env.update(
        HWKV_LIBRARY=lib,
        HWKV_ORACLE_LIBRARY=olib,
        LD_PRELOAD=rt,
        # leaks of the Python interpreter and the HIP runtime are not ours
        ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
        UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
        HIP_VISIBLE_DEVICES="",
    )
    return env, lib, olib


def _run(env, args, timeout=600):
    r = subprocess.run([sys.executable, *args], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=timeout)
    out = r.stdout + r.stderr
    return r.returncode, out


def test_sanitizer_builds_are_the_ones_loaded(san_env):
    env, lib, olib = san_env
    code = (
        "import oracle; oracle._load()\n"
        "from paper_2609_02029_amd import hwkv\n"
        "maps = open('/proc/self/maps').read()\n"
        f"assert {lib!r} in maps and {olib!r} in maps, 'sanitizer builds not mapped'\n"
        "assert 'libclang_rt.asan' in maps\n"
        "print('ok')\n"
    )
    rc, out = _run(env, ["-c", code])
    assert rc == 0 and out.strip().endswith("ok"), out[-4000:]


def test_oracle_pins_and_host_abi_under_sanitizers(san_env):
    env, _, _ = san_env
    rc, out = _run(env, ["-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                         "tests/test_oracle_pins.py", "tests/test_host_abi.py"])
    assert "Sanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert rc == 0, out[-6000:]
    assert " passed" in out and "failed" not in out, out[-2000:]
