"""CPU sanitizer builds (AddressSanitizer + UndefinedBehaviorSanitizer) of the host code:

- the oracle (plain C, gcc), run under its pins (tests/test_oracle_pins.py);
- libvx with its host side instrumented (hipcc, each -fsanitize= after -Xarch_host; the gfx950
  device code is built as usual but never runs here), run under the C-ABI tests
  (tests/test_abi.py): argument checks, workspace sizing, the thread-local error message.

Each suite runs in a child process with the sanitizer runtime preloaded; a report (any
out-of-bounds access, use after free, or undefined behaviour) writes a log and fails the run.
No GPU is used."""
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _gcc_runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _clang_asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _run_under(preload, tmp_dir, code, extra_env=None):
    log_dir = os.path.join(tmp_dir, "reports")
    os.makedirs(log_dir, exist_ok=True)
    env = dict(os.environ, LD_PRELOAD=preload, OMP_NUM_THREADS="2",
               ASAN_OPTIONS=f"detect_leaks=0:log_path={log_dir}/asan",
               UBSAN_OPTIONS=f"print_stacktrace=1:halt_on_error=1:log_path={log_dir}/ubsan", **(extra_env or {}))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    logs = sorted(glob.glob(os.path.join(log_dir, "*")))
    report = "".join(open(p, errors="replace").read()[:4000] for p in logs)
    assert r.returncode == 0 and not logs, (r.returncode, report or r.stdout[-3000:] + r.stderr[-3000:])


def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan, ubsan = _gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("gcc's sanitizer runtimes are not installed")
    lib = str(tmp_path / "libvxo_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                           "-o", lib, os.path.join(ROOT, "oracle", "vxo.c"), "-lm"])
    code = ("import sys, pytest; sys.exit(pytest.main(['tests/test_oracle_pins.py', '-x', '-q', "
            "'-p', 'no:cacheprovider']))")
    _run_under(f"{asan} {ubsan}", str(tmp_path), code, {"VXO_LIB": lib})


def test_abi_checks_under_asan_ubsan(tmp_path):
    from paper_2606_06453_amd import build as B
    runtime = _clang_asan_runtime()
    if runtime is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    srcs = sorted(glob.glob(os.path.join(B.CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(B.CSRC, "*.cpp")))

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        r = subprocess.run([B._hipcc(), *B.COMMON, *san, *lang, "-c", src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        return obj

    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, srcs))
    lib = str(tmp_path / "libvx_san.so")
    subprocess.check_call([B._hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-Xarch_host",
                           "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", "-o", lib,
                           *objs])
    code = ("import sys, pytest\n"
            "from paper_2606_06453_amd import vx\n"
            f"vx.LIB_PATH = {lib!r}\n"
            "sys.exit(pytest.main(['tests/test_abi.py', '-x', '-q', '-p', 'no:cacheprovider']))\n")
    _run_under(runtime, str(tmp_path), code)
