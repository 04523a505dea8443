"""The host code of the library (planner, batch former, status strings) under
AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

A host-only build of those sources with the sanitizers (``g++
-fsanitize=address,undefined``, every report fatal) replaces the library in a
child pytest process that preloads the compiler's ASan runtime. The child runs
the planner and former tests of ``test_host_abi.py`` (those that call device
entry points are left out: the host-only build has none) and the serving-loop
lock-step tests of ``test_trace.py`` (but not the two that serve whole
2000-request traces, which run the same code for minutes); any report fails
the run. A last check
makes sure the sanitizer is live: a batch description whose block-table
offsets array is one entry short makes the planner read past its end, and the
child must die with an ASan report."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DEVICE_TESTS = ("exports_every", "park_and_attention", "kv_append_rejects", "plan_upload_rejects",
                "shape_is_refused", "noalloc", "row_path_option", "tile_path_option", "empty_batches")


def _asan_runtime():
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.fixture(scope="module")
def sanitized_env():
    runtime = _asan_runtime()
    if runtime is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    from paper_2512_04013_amd.build import build_host_sanitized
    lib = build_host_sanitized()
    env = dict(os.environ, AUG_HOST_ONLY_LIB=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return env


def _child(env, args, timeout=900):
    return subprocess.run([sys.executable, *args], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


@pytest.mark.slow
def test_planner_and_former_tests_pass_under_the_sanitizers(sanitized_env):
    r = _child(sanitized_env, ["-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                               "tests/test_host_abi.py", "tests/test_trace.py",
                               "-k", " and ".join(f"not {t}" for t in DEVICE_TESTS + ("whole_sweep_trace", "every_sweep_budget"))])
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
    assert " passed" in r.stdout


def test_the_sanitizer_catches_an_out_of_bounds_read(sanitized_env):
    code = (
        "import numpy as np, paper_2512_04013_amd as aug\n"
        "s = aug.make_shape(8, 8, 64, 'bf16', 'bf16', 'bf16', 0.125)\n"
        "L = aug.lib()\n"
        "n = 3\n"
        "q = np.arange(n + 1, dtype=np.int32)\n"
        "ctx = np.full(n, 5, np.int32)\n"
        "bt = np.arange(n, dtype=np.int32)     # one entry short: the planner reads bt[n]\n"
        "p32 = aug.C.POINTER(aug.C.c_int32)\n"
        "d = aug.aug_batch_desc(n, q.ctypes.data_as(p32), ctx.ctypes.data_as(p32), bt.ctypes.data_as(p32), None, 64)\n"
        "info = aug.aug_attn_plan_info()\n"
        "L.aug_attn_plan(aug.C.byref(s), aug.C.byref(d), 0, None, 0, aug.C.byref(info))\n"
        "print('no report')\n")
    r = _child(sanitized_env, ["-c", code], timeout=300)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr, (r.returncode, r.stdout[-500:], r.stderr[-2000:])
