"""The CPU suite's native code under AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU): the fp64 oracle (gcc) and the host side of the C ABI (the library's
spire_abi.hip built with sanitized host code, linked with the normal device
objects) are rebuilt with -fsanitize=address,undefined, and the tests that
load them run again in a subprocess with the matching runtime preloaded.  The
two compilers' runtimes cannot share a process, so each library gets its own
run.  A run must pass and leave no sanitizer report; a copy of the oracle with
a planted out-of-bounds read shows that the runtime does catch one."""
import glob
import os
import subprocess
import sys

import pytest

from oracle import oracle as O
from paper_2504_06419_amd import build as hipbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG_ASAN = "libclang_rt.asan-x86_64.so"


def _gcc_asan():
    return subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                          check=True).stdout.strip()


def _clang_asan():
    llvm = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm")
    r = subprocess.run([os.path.join(llvm, "bin", "clang"), "-print-file-name=" + CLANG_ASAN],
                       capture_output=True, text=True)
    return r.stdout.strip() if r.returncode == 0 else ""


def _build_oracle(src_text, out):
    src = out + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", "-fopenmp", "-std=c99", "-shared", "-fPIC",
                           src, "-o", out, "-lm"])
    return out


def _run(tests, env_extra, preload, logdir):
    env = dict(os.environ)
    env.update(env_extra)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = f"detect_leaks=0:log_path={logdir}/asan"
    env["UBSAN_OPTIONS"] = f"print_stacktrace=1:halt_on_error=1:log_path={logdir}/ubsan"
    return subprocess.run([sys.executable, "-m", "pytest", *tests, "-q", "-x", "-p", "no:cacheprovider",
                           "-m", "not gpu"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)


def _reports(logdir):
    return sorted(glob.glob(os.path.join(logdir, "asan*")) + glob.glob(os.path.join(logdir, "ubsan*")))


def test_oracle_under_asan_and_ubsan(tmp_path):
    lib = _build_oracle(open(O.SRC).read(), str(tmp_path / "liboracle_san.so"))
    r = _run(["tests/test_oracle_pins.py", "tests/test_oracle_mutants.py"],
             {"SPIRE_TEST_ORACLE_LIB": lib}, _gcc_asan(), str(tmp_path))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert not _reports(str(tmp_path)), open(_reports(str(tmp_path))[0]).read()[:3000]


def test_sanitizer_catches_a_planted_out_of_bounds_read(tmp_path):
    src = open(O.SRC).read()
    anchor = "dot += q[d] * (load_elem(kv->k, kv->dtype, keys[t] + d) * ks);"
    assert anchor in src
    bad = src.replace(anchor, "dot += q[d] * (load_elem(kv->k, kv->dtype, keys[t] + d + (1 << 22)) * ks);")
    lib = _build_oracle(bad, str(tmp_path / "liboracle_oob.so"))
    r = _run(["tests/test_oracle_pins.py::test_verify_matches_torch_sdpa_float64"],
             {"SPIRE_TEST_ORACLE_LIB": lib}, _gcc_asan(), str(tmp_path))
    reports = _reports(str(tmp_path))
    assert r.returncode != 0 and reports
    assert "ERROR: AddressSanitizer" in open(reports[0]).read()


def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    rt = _clang_asan()
    if not rt or not os.path.exists(rt):
        pytest.skip("the ROCm clang AddressSanitizer runtime is not installed")
    objs = [os.path.join(hipbuild.BUILD, s.replace(".hip", ".o")) for s in hipbuild.SOURCES]
    if not all(os.path.exists(o) for o in objs):
        hipbuild.build()
    abi = str(tmp_path / "spire_abi_san.o")
    cmd = [hipbuild._hipcc(), "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={hipbuild.ARCH}",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer",
           "-c", os.path.join(hipbuild.CSRC, "spire_abi.hip"), "-o", abi]
    subprocess.run(cmd, check=True, capture_output=True)
    lib = str(tmp_path / "libspire_san.so")
    others = [o for o in objs if not o.endswith("spire_abi.o")]
    subprocess.run([hipbuild._hipcc(), f"--offload-arch={hipbuild.ARCH}", "-shared", "-fPIC", abi, *others,
                    "-o", lib], check=True, capture_output=True)
    r = _run(["tests/test_abi_cpu.py"], {"SPIRE_TEST_LIB": lib}, rt, str(tmp_path))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert not _reports(str(tmp_path)), open(_reports(str(tmp_path))[0]).read()[:3000]
