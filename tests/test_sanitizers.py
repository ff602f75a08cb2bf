"""CPU sanitizer runs (AddressSanitizer + UndefinedBehaviorSanitizer).

Two builds, each loaded into a fresh Python process with its sanitizer
runtime preloaded:

* the oracle's C code, built with gcc, under the oracle pins and the
  capture tests;
* the host half of the HIP library (argument validation, the packed-layout
  arithmetic, the Gilbert-curve order), built with hipcc with the sanitizers
  on the host pass only (device code is compiled unoptimised and never runs
  here), under the ABI validation and query-order tests.

A sanitizer report aborts the child process (halt_on_error), which fails the
test with the report in the message. Leak checking is off: the interpreter
itself keeps allocations alive until exit.
"""
import os
import shutil
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
CSRC = ROOT / "paper_2607_12789_amd" / "csrc"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {
    "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
    "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
}


def _run_pytest_under(preload: str, extra_env: dict, tests: list, tmp: Path):
    env = dict(os.environ, **SAN_ENV, **extra_env)
    env["LD_PRELOAD"] = ":".join(x for x in (preload, os.environ.get("LD_PRELOAD", "")) if x)
    log = tmp / "child.log"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           *[str(ROOT / "tests" / t) for t in tests]]
    with open(log, "w") as f:
        rc = subprocess.run(cmd, cwd=ROOT, env=env, stdout=f, stderr=subprocess.STDOUT,
                            timeout=600).returncode
    text = log.read_text(errors="replace")
    assert rc == 0, f"sanitized run failed (rc {rc}):\n{text[-6000:]}"
    assert "runtime error" not in text and "AddressSanitizer" not in text, text[-6000:]


def test_oracle_under_asan_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    libasan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = tmp_path / "libavq_oracle_san.so"
    subprocess.run([gcc, "-O1", "-g", "-std=c99", "-fopenmp", "-fPIC", "-shared",
                    "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", str(ROOT / "oracle" / "avq_oracle.c"),
                    "-o", str(lib), "-lm"], check=True)
    _run_pytest_under(libasan, {"AVQ_ORACLE_LIB": str(lib), "OMP_NUM_THREADS": "2"},
                      ["test_oracle_pins.py", "test_capture.py"], tmp_path)


def _clang_asan_runtime() -> Path | None:
    res = subprocess.run([HIPCC, "--print-resource-dir"], capture_output=True, text=True)
    base = Path(res.stdout.strip()) if res.returncode == 0 else None
    if base is None:
        return None
    for cand in (base / "lib" / "linux" / "libclang_rt.asan-x86_64.so",
                 base / "lib" / "x86_64-unknown-linux-gnu" / "libclang_rt.asan.so"):
        if cand.exists():
            return cand
    return None


def test_host_abi_under_asan_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    rt = _clang_asan_runtime()
    if rt is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    sys.path.insert(0, str(ROOT))
    from paper_2607_12789_amd.build import SOURCES
    # sanitizers on the host pass only; each -fsanitize= follows -Xarch_host
    flags = ["--offload-arch=gfx950", "-std=c++17", "-fPIC", "-g", "-O1",
             "-fno-omit-frame-pointer", "-Xarch_device", "-O0",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Xarch_host", "-fsanitize=address,undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined"]
    procs, objs = [], []
    for src in SOURCES:
        obj = tmp_path / (Path(src).stem + ".o")
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", str(CSRC / src), "-o", str(obj)],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
        objs.append(str(obj))
    for p in procs:
        out, _ = p.communicate()
        assert p.returncode == 0, out.decode(errors="replace")[-4000:]
    lib = tmp_path / "libavq_san.so"
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
                    "-Xarch_host", "-fsanitize=address,undefined", *objs, "-o", str(lib)],
                   check=True)
    _run_pytest_under(str(rt), {"AVQ_LIB": str(lib)},
                      ["test_abi_host.py", "test_order.py"], tmp_path)
