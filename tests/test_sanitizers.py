"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only):
the oracle's C code runs the whole pin suite (tests/oracle_pins.py), and the
C ABI's host side runs the host-only ABI tests, each in a child process in
which any out-of-bounds access, use after free or undefined operation
aborts."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from oracle import build  # noqa: E402


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = build.build(out=str(tmp_path / "liboracle_san.so"), sanitize=True)
    env = dict(os.environ, DEAMOE_ORACLE_LIB=lib, LD_PRELOAD=build.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    code = ("import sys, oracle; L = oracle.lib(); assert L._name == sys.argv[1], L._name; "
            "sys.path.insert(0, 'tests'); import oracle_pins as P; "
            "[c() for c in P.ALL_CHECKS]; print('pins', len(P.ALL_CHECKS))")
    r = subprocess.run([sys.executable, "-c", code, lib], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_pins
    assert f"pins {len(oracle_pins.ALL_CHECKS)}" in r.stdout, r.stdout


def test_abi_host_code_under_asan_ubsan(tmp_path):
    """The host side of the C ABI (api.hip: validation, workspace layout,
    the no-alloc size checks) built under ASan and UBSan runs the host-only
    ABI tests (tests/test_abi.py) in a child process."""
    from paper_2608_14385_amd import build as hb
    lib = hb.build_host_sanitized(str(tmp_path))
    env = dict(os.environ, LD_PRELOAD=hb.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    code = ("import sys, pytest; import paper_2608_14385_amd.deamoe as D; "
            "D.LIB_PATH = sys.argv[1]; "
            "rc = pytest.main(['-q', '-x', '-p', 'no:cacheprovider', 'tests/test_abi.py']); "
            "assert D.lib()._name == sys.argv[1]; sys.exit(rc)")
    r = subprocess.run([sys.executable, "-c", code, lib], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout, r.stdout
