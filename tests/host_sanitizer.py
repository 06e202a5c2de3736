"""Build of the library's host code (C ABI, block manager, planner, dispatch
rules) with AddressSanitizer and UndefinedBehaviorSanitizer, by g++ only:
no GPU code is built with a sanitizer. Kernel launches come from
tests/sanitizer_stubs.cpp and fail with hipErrorNoDevice. The binding loads
this library instead of libspork.so when SPORK_HOST_SANITIZER_LIB names it."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_03333_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
OUT = os.path.join(ROOT, "_build", "libspork_host_asan.so")
SOURCES = [os.path.join(CSRC, f) for f in ("block_manager.cpp", "plan.cpp", "capi.cpp", "dispatch_rules.cpp")]
SOURCES.append(os.path.join(ROOT, "tests", "sanitizer_stubs.cpp"))


def build():
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-shared", "-fPIC", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROCM, 'include')}", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           *SOURCES, "-o", OUT, f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("sanitizer build failed:\n" + r.stdout)
    return OUT


def runtime_preload():
    """The sanitizer runtimes to preload into an uninstrumented python."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        path = subprocess.run(["g++", f"-print-file-name={name}"], stdout=subprocess.PIPE, text=True).stdout.strip()
        libs.append(path)
    return ":".join(libs)
