"""The host library's validation, device-image construction and argument
checks, and the CPU oracle, under AddressSanitizer and UBSan: CPU-only builds
of both (g++ / gcc, no device code) run the ABI, template and oracle-pin test
files in a subprocess with the sanitizer runtimes preloaded; any report
aborts it."""
import os
import subprocess
import sys

import pytest

import oracle
from paper_2607_11262_amd import build

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def runtime(name):
    path = subprocess.check_output(["gcc", f"-print-file-name={name}"], text=True).strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"{name} not found")
    return path


@pytest.mark.slow
def test_host_library_and_oracle_under_asan_ubsan(tmp_path):
    host = build.build_host_sanitized(str(tmp_path / "libgts_host_san.so"))
    orc = oracle.build_sanitized(str(tmp_path / "libgts_oracle_san.so"))
    env = dict(os.environ)
    env.update(LD_PRELOAD=f"{runtime('libasan.so')}:{runtime('libubsan.so')}",
               ASAN_OPTIONS=f"detect_leaks=0:halt_on_error=1:log_path={tmp_path / 'asan'}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={tmp_path / 'ubsan'}",
               GTS_TEST_SANITIZED_HOST=host, GTS_TEST_SANITIZED_ORACLE=orc)
    files = [os.path.join(HERE, f) for f in ("test_abi.py", "test_templates.py", "test_oracle_pins.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", *files, "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    # a report goes to its log file (pytest's capture would swallow stderr)
    reports = "".join(open(tmp_path / f).read()[:4000] for f in sorted(os.listdir(tmp_path))
                      if f.startswith(("asan", "ubsan")))
    assert not reports, reports
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    mapped = [line for line in out.splitlines() if line.startswith("[sanitized] mapped:")]
    assert mapped and host in mapped[0] and orc in mapped[0], out[-2000:]
    assert os.path.join(ROOT, "paper_2607_11262_amd", "libgts.so") not in mapped[0]
