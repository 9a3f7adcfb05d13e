"""Host AddressSanitizer run of the library (CPU only).

Builds libattn.so into _build/asan/ with the host half of every translation
unit instrumented by AddressSanitizer (the flag passed to the host compile
only; device code is built as usual), then runs the CPU test suite against
that build with the sanitizer runtime preloaded into the Python process.
Exit status 0 means the suite passed and the sanitizer reported nothing.

python tests/host_asan.py
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.join(ROOT, "paper_2609_10937_amd", "csrc"))
import build as B  # noqa: E402

OUT = os.path.join(ROOT, "_build", "asan")
HOST_ASAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def _compile(src):
    obj = os.path.join(OUT, src.replace(".", "_") + ".o")
    cmd = [B._hipcc(), *B.COMMON, "-g", *HOST_ASAN]
    if src.endswith(".hip"):
        cmd += ["-x", "hip", *B.DEVICE]
    cmd += ["-c", os.path.join(B.HERE, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise SystemExit(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    return obj


def build():
    os.makedirs(OUT, exist_ok=True)
    with cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, B.SOURCES))
    lib = os.path.join(OUT, "libattn.so")
    cmd = [B._hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *HOST_ASAN, "-o", lib, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise SystemExit(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    return lib


def runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise SystemExit("clang AddressSanitizer runtime not found")
    return hits[-1]


def instrumented(lib):
    """The build calls the sanitizer's checks (its undefined __asan_ symbols)."""
    r = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True, check=True)
    return "__asan_report_load" in r.stdout and "__asan_report_store" in r.stdout


def main():
    lib = build()
    if not instrumented(lib):
        print("host_asan: the build is not instrumented")
        return 24
    # ATTN_HOST_ASAN marks the inner run, whose own copy of the test that
    # drives this script skips instead of recursing.
    env = dict(os.environ, ATTN_LIB=lib, LD_PRELOAD=runtime(), ATTN_HOST_ASAN="1",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=23")
    cmd = [sys.executable, "-m", "pytest", "tests", "-q", "-x", "-m", "not gpu"]
    r = subprocess.run(cmd, env=env, capture_output=True, text=True, cwd=ROOT)
    out = r.stdout + r.stderr
    print(out[-3000:])
    if "AddressSanitizer" in out:
        print("host_asan: the sanitizer reported an error")
        return 23
    return r.returncode


if __name__ == "__main__":
    sys.exit(main())
