"""AddressSanitizer + UndefinedBehaviorSanitizer build of the host C/C++ code:
the synthetic-input generator (synth/gen.c), the oracle (oracle/oracle.c) and
the library's temporal-ROI selector (paper_2608_15437_amd/csrc/roi_policy.cpp),
linked into one executable with tests/host_sanitize_driver.c and run on small
workloads with edge cases.  Host code only: gcc and g++, nothing for the GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None, reason="no host compiler")
def test_host_code_under_asan_ubsan(tmp_path):
    inc = ["-I" + os.path.join(ROOT, d) for d in ("include", "oracle", "synth")]
    objs = []
    for src, cc, std in [("synth/gen.c", "gcc", "-std=c11"), ("oracle/oracle.c", "gcc", "-std=c11"),
                         ("tests/host_sanitize_driver.c", "gcc", "-std=c11"),
                         ("paper_2608_15437_amd/csrc/roi_policy.cpp", "g++", "-std=c++17")]:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        extra = ["-ffp-contract=off"] if src.startswith("oracle") else []
        subprocess.run([cc, std, *SAN, *extra, *inc, "-c", os.path.join(ROOT, src), "-o", obj], check=True,
                       capture_output=True, text=True)
        objs.append(obj)
    exe = str(tmp_path / "host_sanitize")
    subprocess.run(["g++", *SAN, *objs, "-o", exe, "-lm"], check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, f"sanitizer run failed ({r.returncode}):\n{r.stdout}\n{r.stderr[-4000:]}"
    lines = r.stdout.splitlines()
    assert lines and lines[-1].startswith("checksum "), r.stdout
    voxels = [int(l.split("voxels=")[1].split()[0]) for l in lines if l.startswith("batch ")]
    assert len(voxels) == 3 and min(voxels) > 0, r.stdout  # every batch did real work
