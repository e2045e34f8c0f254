"""The host runtime (paper_1712_06139_amd/csrc/runtime.cpp) built for its
host-only paths with the compiler's sanitizers and driven through the C ABI
without a GPU (tests/sanitize/host_paths.cpp): address and undefined-behaviour
checks over model and queue life cycles, trace replays with launch windows,
the serving calls, version transitions and queues replaced while serving;
thread checks over models created and destroyed on loader threads while the
main thread serves and swaps them in. The device runtime and the kernels are
replaced by stand-ins that stop the program if a host-only path reaches them
(tests/sanitize/hip_absent.cpp)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "paper_1712_06139_amd", "csrc", "runtime.cpp"),
       os.path.join(ROOT, "tests", "sanitize", "hip_absent.cpp"),
       os.path.join(ROOT, "tests", "sanitize", "host_paths.cpp")]
FLAGS = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-Wno-unused-result", "-D__HIP_PLATFORM_AMD__",
         "-I/opt/rocm/include", f"-I{os.path.join(ROOT, 'include')}"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                                reason="needs g++ and the HIP headers")


def _build_and_run(tmp_path, sanitize, args):
    exe = str(tmp_path / "host_paths")
    subprocess.run(["g++", *FLAGS, *sanitize, *SRC, "-o", exe, "-lpthread"], check=True, capture_output=True,
                   timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1",
               TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host paths ok" in r.stdout
    return r.stdout


def test_host_runtime_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"], [])
    print(out)


def test_host_runtime_loader_threads_under_thread_sanitizer(tmp_path):
    out = _build_and_run(tmp_path, ["-fsanitize=thread"], ["--threads"])
    print(out)
