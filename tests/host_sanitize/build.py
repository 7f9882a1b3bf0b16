"""Builds the host-only sanitizer executable: the library's sources compiled
for the host alone (no device code) with AddressSanitizer and
UndefinedBehaviorSanitizer, linked with the stub HIP runtime and the ABI
driver in this directory.  Run as ``python tests/host_sanitize/build.py OUT``."""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
from paper_2602_08376_amd.build import CSRC, INCLUDE, SOURCES  # noqa: E402

SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def tool(name):
    exe = shutil.which(name) or os.path.join("/opt/rocm/bin", name)
    if not os.path.exists(exe):
        raise RuntimeError(f"{name} not found")
    return exe


def build(out_dir):
    os.makedirs(out_dir, exist_ok=True)
    hipcc = tool("hipcc")
    clang = os.path.join("/opt/rocm/llvm/bin", "clang++")
    jobs = []
    for src in SOURCES:
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, "--cuda-host-only", "-O1", "-g", "-std=c++17", *SAN, "-I", INCLUDE, "-I", CSRC]
        if src.endswith(".cpp"):
            cmd += ["-x", "hip"]
        jobs.append((cmd + ["-c", os.path.join(CSRC, src), "-o", obj], obj))
    for src in ("hip_stub.cpp", "driver.cpp"):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        cmd = [clang, "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-fsanitize=address",
               "-fsanitize=undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
               "-I", "/opt/rocm/include", "-I", INCLUDE, "-c", os.path.join(HERE, src), "-o", obj]
        jobs.append((cmd, obj))

    def run(job):
        r = subprocess.run(job[0], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compile failed: {' '.join(job[0])}\n{r.stderr}")
        return job[1]

    with ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(run, jobs))
    # host-only objects still name the code-object blob their registration
    # wrapper would hand to the runtime; give each an empty one
    names = set()
    for obj in objs:
        r = subprocess.run(["nm", "-u", obj], capture_output=True, text=True, check=True)
        names.update(t.split()[-1] for t in r.stdout.splitlines()
                     if t.split() and t.split()[-1].startswith("__hip_fatbin_"))
    blobs = os.path.join(out_dir, "fatbin_stubs.c")
    with open(blobs, "w") as f:
        for n in sorted(names):
            f.write(f"const char {n}[64] = {{0}};\n")
    bobj = blobs[:-2] + ".o"
    r = subprocess.run([clang, "-x", "c", "-c", blobs, "-o", bobj], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {r.stderr}")
    objs.append(bobj)
    exe = os.path.join(out_dir, "abi_sanitized")
    r = subprocess.run([clang, "-fsanitize=address", "-fsanitize=undefined", *objs, "-o", exe],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    return exe


if __name__ == "__main__":
    print(build(sys.argv[1] if len(sys.argv) > 1 else os.path.join(ROOT, "_build", "host_sanitize")))
