"""Host code of the library under AddressSanitizer and UndefinedBehaviorSanitizer.

The library's sources are compiled host-only (no device code, relocatable
device-code mode so that the objects link without device images) with
-fsanitize=address,undefined and linked with tests/native/abi_host_check.cpp,
which drives the argument validation, the workspace layout of every size and
operation, the float64 transfer-function tables and the range checks; the
host-side plan and tile-layout checks of tests/native are built the same way.
Skipped where hipcc or the sanitizer runtimes are missing.
"""

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2306_11268_amd", "csrc")
SIZES = (64, 100, 128, 200, 256, 350, 400, 500, 512, 1000, 1024)
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return None


def _compile(cc, src, obj, extra=()):
    cmd = [cc, "--cuda-host-only", "-fgpu-rdc", "-O1", "-g", "-std=c++17", "-fPIC", *SAN, "-Xclang",
           "-target-feature", "-Xclang", "-packed-fp32-ops", *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return obj


def _link(cc, objs, exe):
    # host-only objects compiled for relocatable device code: the link step
    # supplies the (empty) device image their registration code refers to
    return [cc, "-fgpu-rdc", "--hip-link", "--offload-arch=gfx950", *SAN, *objs, "-o", str(exe)]


@pytest.fixture(scope="module")
def hipcc(tmp_path_factory):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not available")
    d = tmp_path_factory.mktemp("san_probe")
    src = d / "p.cpp"
    src.write_text("int main() { return 0; }\n")
    r = subprocess.run([cc, *SAN, str(src), "-o", str(d / "p")], capture_output=True, text=True)
    if r.returncode != 0 or subprocess.run([str(d / "p")], env=ENV).returncode != 0:
        pytest.skip("sanitizer runtimes not available")
    return cc


def test_the_build_instruments_host_code(hipcc, tmp_path):
    """Control: a use after free and a signed overflow built the same way are caught."""
    src = tmp_path / "bad.cpp"
    src.write_text("#include <climits>\n#include <cstdlib>\n"
                   "int main(int argc, char**) {\n"
                   "  int* p = static_cast<int*>(std::malloc(4 * sizeof(int)));\n"
                   "  if (argc > 1) { int x = INT_MAX; x += argc; std::free(p); return x; }\n"
                   "  p[0] = 1;\n  std::free(p);\n  return p[0];\n}\n")
    exe = tmp_path / "bad"
    obj = _compile(hipcc, str(src), str(tmp_path / "bad.o"))
    r = subprocess.run(_link(hipcc, [obj], exe), capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    heap = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV)
    assert heap.returncode != 0 and "AddressSanitizer" in heap.stderr
    ub = subprocess.run([str(exe), "x"], capture_output=True, text=True, env=ENV)
    assert ub.returncode != 0 and "runtime error" in ub.stderr


def test_c_abi_host_paths_under_sanitizers(hipcc, tmp_path):
    units = [(os.path.join(CSRC, "api.hip"), []), (os.path.join(CSRC, "kernels.hip"), [])]
    units += [(os.path.join(CSRC, "kern_size.hip"), [f"-DLR_FFT_N={n}"]) for n in SIZES]
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda iu: _compile(hipcc, iu[1][0], str(tmp_path / f"u{iu[0]}.o"), iu[1][1]),
                           enumerate(units)))
    drv = _compile(hipcc, os.path.join(HERE, "native", "abi_host_check.cpp"), str(tmp_path / "drv.o"))
    exe = tmp_path / "abi_host_check"
    r = subprocess.run(_link(hipcc, [drv, *objs], exe), capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600, env=ENV)
    assert out.returncode == 0, (out.stdout + out.stderr)[-6000:]
    assert "ALL OK" in out.stdout
    assert "runtime error" not in out.stderr


@pytest.mark.parametrize("src", ["fft_plans_host.cpp", "tile_layout_host.hip"])
def test_native_checks_under_sanitizers(hipcc, tmp_path, src):
    exe = tmp_path / "native"
    obj = _compile(hipcc, os.path.join(HERE, "native", src), str(tmp_path / "native.o"))
    r = subprocess.run(_link(hipcc, [obj], exe), capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600, env=ENV)
    assert out.returncode == 0, (out.stdout + out.stderr)[-6000:]
    assert "ALL OK" in out.stdout
    assert "runtime error" not in out.stderr
