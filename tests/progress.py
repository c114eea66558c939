"""Progress lines of the GPU tests that reach the terminal while pytest
captures the tests' output (a long test that printed nothing would look hung
to whoever watches the run)."""
import sys

CAPMAN = None   # pytest's capture manager, set by conftest.pytest_configure


def say(*a):
    msg = " ".join(str(x) for x in a)
    if CAPMAN is not None:
        with CAPMAN.global_and_fixture_disabled():
            print(msg, flush=True)
    else:
        print(msg, flush=True)
    sys.stdout.flush()
