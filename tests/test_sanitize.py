"""Host builds with AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (oracle/qcnn_oracle.c) with gcc, driven by
  tests/sanitize/oracle_driver.c: every oracle function on small shapes with
  exact-size heap buffers, leak detection on.
* The library's host code (every csrc file compiled for the host only, the
  sanitizers on the host pass), driven by tests/sanitize/abi_driver.c: the
  argument validation of every entry point, the helpers, and the conv planners
  over many layer shapes.  Host-only objects refer to their device code
  objects by symbol; empty stand-ins are linked in, and no call of the driver
  reaches a kernel.
"""
import os
import re
import shutil
import subprocess
import concurrent.futures as cf

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1512_06473_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def run(cmd, env=None, timeout=300):
    return subprocess.run(cmd, capture_output=True, text=True, timeout=timeout, env=env)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_drv")
    r = run(["gcc"] + SAN + ["-std=c99", "-Wno-unknown-pragmas", "-o", exe,
             os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), os.path.join(ROOT, "oracle", "qcnn_oracle.c"),
             "-lm"])
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = run([exe], env=env)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM, "bin", "hipcc")), reason="no hipcc")
def test_abi_host_code_under_sanitizers(tmp_path):
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))

    def compile_host(src):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        cmd = [hipcc, "-x", "hip", "--offload-arch=gfx950", "--cuda-host-only", "-O1", "-g", "-fPIC", "-std=c++17"]
        cmd += HOST_SAN + ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        r = run(cmd)
        assert r.returncode == 0, (src, r.stderr[-2000:])
        return obj

    with cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_host, srcs))
    drv_o = str(tmp_path / "abi_driver.o")
    r = run([clang] + SAN + ["-I", os.path.join(ROOT, "include"), "-c",
                             os.path.join(ROOT, "tests", "sanitize", "abi_driver.c"), "-o", drv_o])
    assert r.returncode == 0, r.stderr
    # Empty stand-ins for the device code objects the host objects refer to.
    undef = set()
    for o in objs:
        out = run(["nm", "-u", o]).stdout
        undef.update(re.findall(r"\b(__hip_fatbin_\w+)", out))
    stub_c = tmp_path / "fatbin_stubs.c"
    stub_c.write_text("".join("__attribute__((aligned(4096))) const char %s[4096] = {0};\n" % s
                              for s in sorted(undef)))
    stub_o = str(tmp_path / "fatbin_stubs.o")
    r = run([clang, "-c", str(stub_c), "-o", stub_o])
    assert r.returncode == 0, r.stderr
    exe = str(tmp_path / "abi_drv")
    r = run([clang + "++"] + SAN + ["-o", exe, drv_o] + objs + [stub_o, "-L", os.path.join(ROCM, "lib"),
                                                                  "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    assert r.returncode == 0, r.stderr[-3000:]
    # The HIP runtime keeps allocations until exit: leak detection off here.
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = run([exe], env=env)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr[-3000:]
