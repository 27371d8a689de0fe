"""CPU hygiene: the oracle under AddressSanitizer + UndefinedBehaviorSanitizer,
and the library's behaviour on a host without a GPU.

* Every oracle entry point runs on small seeded graphs (degenerate sizes,
  duplicates, isolated rows, several heads) in a C driver built together with
  oracle/oracle.c under -fsanitize=address,undefined: an access outside an
  exactly sized buffer, a leak or undefined arithmetic fails the run. A copy
  of the oracle with one planted off-by-one write shows the build catches it.
* Without a device, an entry point whose arguments pass the host checks
  reports PYG_ERR_HIP (its first HIP call fails) instead of crashing."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_C = os.path.join(ROOT, "oracle", "oracle.c")
DRIVER_C = os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c")
SAN = ["gcc", "-g", "-O1", "-std=c11", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-ffp-contract=off", "-Wall"]


def _build(src, out):
    r = subprocess.run(SAN + [src, DRIVER_C, "-lm", "-o", out], capture_output=True, text=True)
    if r.returncode != 0 and "sanitize" in r.stderr and "cannot find" in r.stderr:
        pytest.skip("the sanitizer runtimes are not installed")
    assert r.returncode == 0, r.stderr
    return out


def _run(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)


def test_oracle_under_asan_ubsan(tmp_path):
    exe = _build(ORACLE_C, str(tmp_path / "oracle_asan"))
    r = _run(exe)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "every check passed" in r.stdout


def test_sanitizer_catches_a_planted_overflow(tmp_path):
    src = open(ORACLE_C).read()
    good = "for (int64_t i = 0; i < N; ++i) deg[i] = 0;"
    assert src.count(good) == 1
    bad = tmp_path / "oracle_overflow.c"
    bad.write_text(src.replace(good, "for (int64_t i = 0; i <= N; ++i) deg[i] = 0;"))
    r = _run(_build(str(bad), str(tmp_path / "oracle_overflow")))
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stderr


def test_no_device_reports_hip_error():
    import ctypes

    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("a GPU is present: this checks the host without one")
    import paper_1903_02428_amd as pyg
    from paper_1903_02428_amd.binding import _Csr
    if not os.path.exists(pyg.library_path()):
        from paper_1903_02428_amd import build
        build.build()
    lib = pyg.library()
    PYG_ERR_HIP = -4
    csr = _Csr(0x10000, 0x20000, 0x30000, None, 10, 20, 0)  # never dereferenced: the launch fails first
    assert lib.pyg_degree_csr(ctypes.byref(csr), ctypes.c_void_p(0x40000), None) == PYG_ERR_HIP
    # the allocation-free entry point: its device query fails
    assert lib.pyg_propagate_noalloc(ctypes.c_void_p(0x10000), 0, 10, 4, ctypes.c_void_p(0x50000), 20, None, None,
                                     0, 0, 1, ctypes.c_void_p(0x90000), None, None) == PYG_ERR_HIP
    assert pyg.strerror(PYG_ERR_HIP) == "HIP runtime or launch error"
