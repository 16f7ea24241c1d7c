"""The oracle and the input generator under AddressSanitizer and
UndefinedBehaviorSanitizer: both libraries are rebuilt instrumented (every
finding fatal) and the oracle's pin tests run against those builds in a
child process, with the sanitizer runtime preloaded (the interpreter itself
is not instrumented; leak checking is off, since the interpreter keeps
memory until it exits).  A copy of the oracle with a planted off-by-one
read must be stopped by a sanitizer report, so the tier is known to see."""
import glob
import os
import subprocess
import sys
import tempfile

from tests import helpers

PIN_TESTS = ["tests/test_oracle_pins.py", "tests/test_oracle_pipeline.py",
             "tests/test_oracle_sim.py", "tests/test_oracle_sage.py"]


def _run_pins(env, tests):
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu",
                           "-p", "no:cacheprovider", *tests], cwd=helpers.ROOT, env=env,
                          capture_output=True, text=True)


def test_oracle_pins_pass_under_asan_and_ubsan():
    sys.path.insert(0, helpers.ROOT)
    from oracle import build as oracle_build
    from synth import build as synth_build
    d = tempfile.mkdtemp(prefix="ggsan_")
    ggref = oracle_build.build(out=os.path.join(d, "libggref.so"), sanitize=True)
    synth = synth_build.build(out=os.path.join(d, "libsynth.so"), sanitize=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                          check=True).stdout.strip()
    logs = os.path.join(d, "report")
    env = dict(os.environ)
    env.update(GGREF_LIB=ggref, SYNTH_LIB=synth,
               LD_PRELOAD=":".join(x for x in (asan, os.environ.get("LD_PRELOAD")) if x),
               ASAN_OPTIONS=f"detect_leaks=0:abort_on_error=1:log_path={logs}",
               UBSAN_OPTIONS=f"print_stacktrace=1:halt_on_error=1:log_path={logs}")
    r = _run_pins(env, PIN_TESTS)
    reports = "".join(open(f).read() for f in glob.glob(logs + "*"))
    assert r.returncode == 0 and not reports, (r.stdout + r.stderr)[-2000:] + reports[:2000]
    assert " passed" in r.stdout

    # the planted mistake: staging reads one bucket entry past the end
    src = open(os.path.join(helpers.ROOT, "oracle", "ggref.cpp")).read()
    line = "for (int64_t s = 0; s < total; ++s) old_slot[(size_t)s] = before[bucket_ids[s]];"
    assert src.count(line) == 1
    bad = os.path.join(d, "ggref_bad.cpp")
    with open(bad, "w") as f:
        f.write(src.replace(line, line.replace("s < total", "s <= total")))
    lib = os.path.join(d, "libggref_bad.so")
    subprocess.run(["g++", *oracle_build.SANITIZE, "-std=c++17", "-shared", "-fPIC",
                    "-I" + os.path.join(helpers.ROOT, "oracle"), bad, "-o", lib], check=True)
    r = _run_pins(dict(env, GGREF_LIB=lib), ["tests/test_oracle_pipeline.py"])
    reports = "".join(open(f).read() for f in glob.glob(logs + "*"))
    assert r.returncode != 0 and "AddressSanitizer: heap-buffer-overflow" in reports
