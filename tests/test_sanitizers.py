"""CPU sanitizer runs (no GPU).

* The oracle (plain C) built with AddressSanitizer + UndefinedBehaviorSanitizer
  runs its pin tests: no out-of-bounds access, use after free or undefined
  arithmetic anywhere in the oracle.
* The HIP library's host code (argument validation, layouts, launch set-up)
  built with the same sanitizers through hipcc (-Xarch_host: device code is
  never instrumented) runs the ABI tests, which exercise every validation
  path without launching anything.
Both run in subprocesses with the sanitizer runtime preloaded (the Python
interpreter itself is not instrumented); a report fails the run."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_PINS = ["tests/test_oracle_retrieval.py", "tests/test_oracle_verify.py",
               "tests/test_oracle_select.py", "tests/test_oracle_project.py",
               "tests/test_oracle_ivf.py", "tests/test_oracle_trie.py"]
SAN_OPTS = "detect_leaks=0:verify_asan_link_order=0:halt_on_error=1:abort_on_error=0"


def _runtime(name):
    return subprocess.check_output(["gcc", f"-print-file-name={name}"], text=True).strip()


def _clang_asan():
    base = "/opt/rocm/llvm/lib/clang"
    for v in sorted(os.listdir(base), reverse=True):
        p = os.path.join(base, v, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    raise FileNotFoundError("clang AddressSanitizer runtime")


def _pytest(files, env_extra):
    env = dict(os.environ, ASAN_OPTIONS=SAN_OPTS, UBSAN_OPTIONS="print_stacktrace=1",
               OMP_NUM_THREADS="4", **env_extra)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *files], cwd=ROOT, env=env, capture_output=True,
                          text=True, timeout=900)


def _clean(r):
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    for marker in ("runtime error:", "ERROR: AddressSanitizer", "SUMMARY: "):
        assert marker not in out, out[-3000:]


def test_oracle_under_asan_and_ubsan(tmp_path):
    lib = str(tmp_path / "libsense_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "sense_oracle.c"),
                           "-o", lib, "-lm"])
    r = _pytest(ORACLE_PINS, {"SENSE_ORACLE_LIB": lib,
                              "LD_PRELOAD": f"{_runtime('libasan.so')} {_runtime('libubsan.so')}"})
    _clean(r)


def test_host_layer_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2606_00021_amd import build
    lib = build.build(out=str(tmp_path / "libsense_hostsan.so"), host_sanitize=True)
    r = _pytest(["tests/test_abi.py"], {"SENSE_LIB": lib, "LD_PRELOAD": _clang_asan()})
    _clean(r)
