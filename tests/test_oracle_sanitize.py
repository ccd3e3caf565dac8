"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (host code).

tests/oracle_sanitize_driver.c links oracle/oracle.c with
-fsanitize=address,undefined (no recovery: the first report aborts) and runs
every entry point over small seeded inputs with every option; it also checks
the codec round trip, the encoder's monotonicity, row-subset identity and the
cast-off S = 2^k identity (Prop. 2).  The test build of the oracle (with the
planted exp2 error compiled in) is run the same way.
"""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.parametrize("plant", [False, True])
def test_oracle_under_asan_and_ubsan(tmp_path, plant):
    exe = tmp_path / ("driver_plant" if plant else "driver")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-fast-math", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-pthread",
           *(["-DORACLE_TEST_PLANTS"] if plant else []),
           os.path.join(ROOT, "oracle", "oracle.c"),
           os.path.join(HERE, "oracle_sanitize_driver.c"), "-lm", "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    if plant:
        # the test build accepts a planted error: that check (once per input
        # shape) is expected to fail, and nothing else
        fails = [ln for ln in r.stderr.splitlines() if ln.startswith("FAIL")]
        assert fails and all("planted error accepted outside the test build" in ln
                             for ln in fails), r.stderr[-2000:]
        assert "Sanitizer" not in r.stderr, r.stderr[-4000:]
    else:
        assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
        assert "all checks passed" in r.stdout
