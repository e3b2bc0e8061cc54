import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the C ABI of libgts.so)")
    config.addinivalue_line("markers", "slow: large inputs; still part of the default suite")


def pytest_sessionstart(session):
    # CPU-only sanitizer runs (tests/test_sanitizers.py starts one in a
    # subprocess with the ASan / UBSan runtimes preloaded): route the library
    # and the oracle to their sanitized builds
    host = os.environ.get("GTS_TEST_SANITIZED_HOST")
    orc = os.environ.get("GTS_TEST_SANITIZED_ORACLE")
    if host:
        from paper_2607_11262_amd import api
        api.use_library(host)
    if orc:
        import oracle
        oracle.use_library(orc)


def pytest_sessionfinish(session, exitstatus):
    if os.environ.get("GTS_TEST_SANITIZED_HOST") or os.environ.get("GTS_TEST_SANITIZED_ORACLE"):
        with open("/proc/self/maps") as f:
            libs = sorted({line.split()[-1] for line in f if "libgts" in line})
        print(f"\n[sanitized] mapped: {' '.join(libs)}", flush=True)
