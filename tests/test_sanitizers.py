"""AddressSanitizer + UndefinedBehaviorSanitizer builds, on the CPU:

- the oracle (oracle/mfpsn_oracle.c) driven over its edge cases by
  tests/sanitize/oracle_driver.c;
- the C-ABI host layer of libmfpsn.so (argument validation and launch
  planning in mfpsn_api.cpp and mfpsn_api_ext.cpp) driven by
  tests/sanitize/abi_driver.c, with the GPU launchers replaced by counting
  stubs (tests/sanitize/launch_stubs.cpp): rejected calls must launch nothing.

Built with gcc/g++ only (no GPU code), into a temporary directory."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2501_14490_amd", "csrc")
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None,
                                reason="needs gcc and g++")


def run(cmd, cwd):
    p = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert p.returncode == 0, f"{' '.join(cmd)}\n{p.stdout[-4000:]}\n{p.stderr[-4000:]}"
    return p.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    run(["gcc", "-std=c11", *SAN, "-ffp-contract=off", os.path.join(ROOT, "oracle", "mfpsn_oracle.c"),
         os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), "-lm", "-o", exe], tmp_path)
    assert "oracle driver: OK" in run([exe], tmp_path)


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"), reason="needs the HIP headers")
def test_abi_layer_under_sanitizers(tmp_path):
    inc = ["-I/opt/rocm/include", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    objs = []
    for src in (os.path.join(CSRC, "mfpsn_api.cpp"), os.path.join(CSRC, "mfpsn_api_ext.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        run(["g++", "-std=c++20", *SAN, "-D__HIP_PLATFORM_AMD__", *inc, "-c", src, "-o", obj], tmp_path)
        objs.append(obj)
    drv = str(tmp_path / "abi_driver.o")
    run(["gcc", "-std=c11", *SAN, f"-I{os.path.join(ROOT, 'include')}", "-c",
         os.path.join(ROOT, "tests", "sanitize", "abi_driver.c"), "-o", drv], tmp_path)
    exe = str(tmp_path / "abi_driver")
    run(["g++", "-fsanitize=address,undefined", *objs, drv, "-o", exe], tmp_path)
    assert "abi driver: OK" in run([exe], tmp_path)
