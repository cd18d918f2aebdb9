"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The C-ABI library's sources are compiled for the host only (no device code
object exists in this build, so no kernel can run) and the fp64 oracle as
plain C++, both with -fsanitize=address,undefined. The host-ABI test modules
(shape bookkeeping, every validation path, the planner's workspace answers)
and the oracle's pin modules then run against these builds in a child
process with the sanitizer runtime preloaded; they must pass and no
sanitizer report may appear."""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_00125_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SOURCES = ["capi.cpp", "shape.cpp", "conv_host.cpp", "noalloc.hip", "gemm_f32.hip", "gemm_bf16.hip",
           "reduce.hip", "elementwise.hip", "conv.hip"]
# sanitizers on the host pass only (each -fsanitize= behind -Xarch_host)
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-fno-omit-frame-pointer"]
MODULES = ["tests/test_abi_host.py", "tests/test_abi_host_conv.py", "tests/test_abi_host_nn.py",
           "tests/test_zz_no_alloc.py", "tests/test_oracle.py", "tests/test_oracle_conv.py"]


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-2000:]}\n{r.stderr[-4000:]}"


@pytest.fixture(scope="module")
def sanitized_builds(tmp_path_factory):
    rt = _asan_runtime()
    if not (os.path.exists(HIPCC) and os.path.exists(CLANGXX) and rt):
        pytest.skip("hipcc, clang++ or the AddressSanitizer runtime is missing")
    out = tmp_path_factory.mktemp("sanitized")

    def compile_one(src):
        obj = str(out / (src + ".o"))
        _run([HIPCC, "-std=c++17", "-O1", "-g", "-fPIC", "-x", "hip", "--offload-host-only",
              "--offload-arch=gfx950", *SAN, "-I", os.path.join(ROOT, "include"), "-c",
              os.path.join(CSRC, src), "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    # Host-only objects refer to the device code object a full build embeds
    # (one __hip_fatbin_<id> symbol per HIP source). Here each is an empty
    # image: HIP reads code objects only at a first kernel launch, and no
    # test run against this build launches anything.
    nm = subprocess.run(["nm", *objs], capture_output=True, text=True, check=True).stdout
    ids = sorted({ln.split()[-1] for ln in nm.splitlines()
                  if ln.split()[:1] == ["U"] and ln.split()[-1].startswith("__hip_fatbin_")})
    stub_c = out / "empty_images.c"
    stub_c.write_text("".join(f"const unsigned char {s}[64] = {{0}};\n" for s in ids))
    stub_o = str(out / "empty_images.o")
    _run(["cc", "-c", "-fPIC", str(stub_c), "-o", stub_o])
    objs.append(stub_o)
    lib = str(out / "libminitensor_hip_sanitized.so")
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *SAN, "-shared-libasan", "-o", lib,
          *objs])
    orc = str(out / "liboracle_sanitized.so")
    _run([CLANGXX, "-std=c++17", "-O1", "-g", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
          "-fsanitize=address,undefined", "-shared-libasan", "-fno-omit-frame-pointer", "-o", orc,
          os.path.join(ROOT, "oracle", "oracle.cpp")])
    return {"lib": lib, "oracle": orc, "runtime": rt}


def test_host_abi_and_oracle_clean_under_address_and_ub_sanitizers(sanitized_builds):
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": sanitized_builds["runtime"],
        "MT_LIB_OVERRIDE": sanitized_builds["lib"],
        "MT_ORACLE_LIB_OVERRIDE": sanitized_builds["oracle"],
        # Python itself is not instrumented and keeps its objects until exit
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:alloc_dealloc_mismatch=0",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "OMP_NUM_THREADS": "4",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *MODULES],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    text = r.stdout + r.stderr
    assert "AddressSanitizer" not in text and "runtime error:" not in text, text[-6000:]
    assert r.returncode == 0, text[-6000:]
    assert " passed" in r.stdout
