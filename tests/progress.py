"""Progress lines of long tests, written past pytest's output capture so
that a run without -s still shows a long test advancing."""
import sys
import time

CAPTURE = None  # pytest's capture manager, set by conftest.py


def say(msg: str, tag: str = "gpu-test") -> None:
    line = f"[{tag} {time.strftime('%H:%M:%S')}] {msg}"
    if CAPTURE is not None:
        with CAPTURE.global_and_fixture_disabled():
            print(line, file=sys.stderr, flush=True)
    else:
        print(line, file=sys.stderr, flush=True)
