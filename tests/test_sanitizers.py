"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer (gcc/g++, host code only):

  - the oracle (tests/sanitize/oracle_driver.c): every entry point on small seeded inputs;
  - the library's host C++ (cache, exact CPU residual, LoRE fit, speculative prefetch,
    split planner and the C ABI's validation; tests/sanitize/host_driver.cpp), with the GPU
    launchers replaced by stubs that report no device;
  - the LoRE fit's host linear algebra (Jacobi eigensolver, Cholesky; lore_math_driver.cpp);
  - a host model of the expert-FFN tile indexing (tile_driver.cpp): every tile of the
    grouped-FFN and decode-layer launches replays its operand loads and output stores,
    through the same index helpers as the kernels (csrc/tile_index.h), on host buffers of
    exactly the sizes a call passes.

Each driver runs in its own process; a sanitizer report, a leak or a failed check ends it
with a non-zero status.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2608_21240_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN_FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HOST_SOURCES = ["cache", "host_exact", "lore_fit", "spec_host", "spice_api", "split"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _have(tool):
    return shutil.which(tool) is not None


def _sanitizers_link(tmp):
    src = os.path.join(tmp, "probe.c")
    with open(src, "w") as f:
        f.write("int main(void) { return 0; }\n")
    r = subprocess.run(["gcc", *SAN_FLAGS, src, "-o", os.path.join(tmp, "probe")], capture_output=True)
    return r.returncode == 0


@pytest.fixture(scope="module")
def build_dir(tmp_path_factory):
    d = str(tmp_path_factory.mktemp("sanitize"))
    if not (_have("gcc") and _have("g++")) or not _sanitizers_link(d):
        pytest.skip("gcc/g++ with AddressSanitizer is not available")
    return d


def _hip_flags():
    return [f"-I{ROCM}/include", "-D__HIP_PLATFORM_AMD__"]


def _hip_libs():
    return [f"-L{ROCM}/lib", f"-Wl,-rpath,{ROCM}/lib", "-lamdhip64", "-lpthread"]


def _need_hip():
    if not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")) or not os.path.exists(
            os.path.join(ROCM, "lib", "libamdhip64.so")):
        pytest.skip("HIP headers / runtime not installed")


def _compile(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stderr[-4000:]}"


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), \
        f"{os.path.basename(exe)} exited {r.returncode}\nstdout: {r.stdout[-2000:]}\nstderr: {r.stderr[-6000:]}"
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-6000:]
    return r


@pytest.fixture(scope="module")
def host_objects(build_dir):
    """The library's host C++ compiled once with the sanitizers."""
    _need_hip()
    objs = []

    def one(name):
        obj = os.path.join(build_dir, f"{name}.o")
        _compile(["g++", "-std=c++17", "-fPIC", *SAN_FLAGS, f"-I{ROOT}/include", f"-I{CSRC}", *_hip_flags(), "-c",
                  os.path.join(CSRC, f"{name}.cpp"), "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(one, HOST_SOURCES))
    return objs


def test_oracle_under_sanitizers(build_dir):
    exe = os.path.join(build_dir, "oracle_driver")
    _compile(["gcc", "-std=c11", *SAN_FLAGS, "-ffp-contract=off", f"-I{ROOT}/oracle",
              os.path.join(SAN, "oracle_driver.c"), os.path.join(ROOT, "oracle", "spice_oracle.c"), "-lm", "-o", exe])
    _run(exe)


def test_host_library_under_sanitizers(build_dir, host_objects):
    exe = os.path.join(build_dir, "host_driver")
    _compile(["g++", "-std=c++17", *SAN_FLAGS, f"-I{ROOT}/include", f"-I{CSRC}", *_hip_flags(),
              os.path.join(SAN, "host_driver.cpp"), os.path.join(SAN, "device_stubs.cpp"), *host_objects,
              *_hip_libs(), "-o", exe])
    _run(exe)


def test_lore_fit_linear_algebra_under_sanitizers(build_dir, host_objects):
    exe = os.path.join(build_dir, "lore_math_driver")
    api = [o for o in host_objects if o.endswith("spice_api.o")]
    _compile(["g++", "-std=c++17", *SAN_FLAGS, f"-I{ROOT}/include", f"-I{CSRC}", *_hip_flags(),
              os.path.join(SAN, "lore_math_driver.cpp"), os.path.join(SAN, "device_stubs.cpp"), *api, *_hip_libs(),
              "-o", exe])
    _run(exe)


def test_tile_indexing_model_under_sanitizers(build_dir):
    _need_hip()
    exe = os.path.join(build_dir, "tile_driver")
    _compile(["g++", "-std=c++17", *SAN_FLAGS, f"-I{ROOT}/include", f"-I{CSRC}", *_hip_flags(),
              os.path.join(SAN, "tile_driver.cpp"), "-o", exe])
    r = _run(exe)
    assert int(r.stdout.split()[0]) > 10 ** 7  # accesses replayed
