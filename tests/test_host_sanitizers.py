"""The C ABI's host code (argument validation and workspace sizing in
sa_api.hip) built for the CPU with AddressSanitizer and
UndefinedBehaviorSanitizer, linked against launcher stand-ins that only
count calls (tests/host_asan/).  The invalid-argument table of
test_host_api.py runs through it: every case must return the same code and
message, launch nothing, and trigger no sanitizer report; workspace sizes,
including extreme arguments, must match the regular library."""
import os
import shutil
import subprocess

import pytest

import paper_2608_15522_amd as sa
from test_host_api import INVALID, _attn, _mask, _mpool, _select, _xpool

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_asan")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
INT_MAX, INT_MIN = 2 ** 31 - 1, -2 ** 31

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    out = tmp_path_factory.mktemp("host_asan")
    # device code is compiled as usual (sa_api.hip holds a device array); only
    # the host side is instrumented
    common = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-I", os.path.join(ROOT, "include"), "-DSA_SRC_ID=\"host-asan\""]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all"]
    srcs = [os.path.join(ROOT, "paper_2608_15522_amd", "csrc", "sa_api.hip"),
            os.path.join(HERE, "stub_launchers.hip")]
    objs = []
    for src in srcs:
        obj = os.path.join(out, os.path.basename(src) + ".o")
        subprocess.run([*common, *san, "-c", src, "-o", obj], check=True, capture_output=True,
                       text=True)
        objs.append(obj)
    obj = os.path.join(out, "api_checks.o")
    subprocess.run([HIPCC, "-O1", "-g", "-std=c++17", "-I", os.path.join(ROOT, "include"),
                    *san, "-x", "c++", "-c", os.path.join(HERE, "api_checks.cpp"), "-o", obj],
                   check=True, capture_output=True, text=True)
    exe = os.path.join(out, "api_checks")
    subprocess.run([HIPCC, "--offload-arch=gfx950", *san, *objs, obj, "-o", exe], check=True,
                   capture_output=True, text=True)
    return exe


def _run(exe, lines):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                         env=env, timeout=120)
    return res


def _arg(v):
    if v is None:
        return "0"
    if isinstance(v, float):
        return repr(v)
    return str(int(v))


def test_invalid_arguments_under_sanitizers(checker):
    lines = []
    for call, kw, code, needle in INVALID:
        args = " ".join(_arg(v) for v in call.args(**kw))
        lines.append(f"call {call.name} {code} {needle.encode().hex()} {args}")
    res = _run(checker, lines)
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert f"cases {len(INVALID)} failed 0" in res.stdout, res.stdout


def test_valid_calls_reach_the_launchers_under_sanitizers(checker):
    """Accepted arguments pass validation and reach the (stand-in) launcher;
    the return code then reflects the launch check of a machine without a
    GPU, so only the message is not checked."""
    ok = [(_attn, {}), (_mask, {}), (_select, {}), (_xpool, {}), (_mpool, {}),
          (_xpool, dict(dtype=1)),
          (_attn, dict(B=2, H=24, L=75600, ws_bytes=1 << 20))]
    lines = [f"call {c.name} 0 - " + " ".join(_arg(v) for v in c.args(**kw)) for c, kw in ok]
    res = _run(checker, lines)
    # every case either succeeded or failed only in the launch check
    assert "BAD" not in res.stdout and res.returncode in (0, 1), res.stdout + res.stderr
    for ln in res.stdout.splitlines():
        if ln.startswith("FAIL"):
            assert "rc 4 (want 0)" in ln and "launched 1" in ln, ln


SIZES = [(c, B, H, L_v, L_a, d, blk)
         for c in range(7)
         for (B, H, L_v, L_a, d, blk) in [
             (1, 24, 32760, 512, 128, 128), (2, 24, 75600, 1024, 128, 128),
             (1, 1, INT_MAX, INT_MAX, 128, 128), (INT_MAX, INT_MAX, 1000, 64, 128, 128),
             (1, 1, INT_MIN, 64, 128, 128), (-1, 1, 1000, 64, 64, 64),
             (1, 65535, 2048 * 128, 1024, 128, 128), (65535, 1, 262144, 262144, 64, 64),
             (1, 1, 1, INT_MAX, 64, 64), (1, 1, 262144, INT_MIN, 64, 64)]]


def test_workspace_sizes_under_sanitizers(checker):
    res = _run(checker, ["ws " + " ".join(str(v) for v in s) for s in SIZES])
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    got = [int(ln.split()[1]) for ln in res.stdout.splitlines() if ln.startswith("ws ")]
    want = [sa.sa_workspace_size(*s) for s in SIZES]
    assert got == want
