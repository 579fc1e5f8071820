"""CPU sanitizer builds.  The oracle (gcc) and the library's host code
(hipcc, host pass only: the device code is built as usual and never runs
here) are built with AddressSanitizer and UndefinedBehaviorSanitizer, and
tests/sanitize/driver.py exercises them in a subprocess with the sanitizer
runtime preloaded: the oracle on the tiny workload (features of all three
schemas, forest with leaf indices and fingerprints, linked walk, MLP, top-k,
regret, evaluation, static configuration, catalogue, linear scorer), the
library through every host-side rejection path of the C ABI and the host
forest packer on random forests of every packable depth.  A sanitizer finding
aborts the subprocess; the test checks its exit status and its last line."""
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "tests", "sanitize", "_build")
DRIVER = os.path.join(ROOT, "tests", "sanitize", "driver.py")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _stale(out: str, sources: list[str]) -> bool:
    return not os.path.exists(out) or os.path.getmtime(out) < max(os.path.getmtime(s) for s in sources)


def _run(kind: str, lib: str, preload: str) -> None:
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report_load" in syms and "__ubsan_handle" in syms, "library built without the sanitizers"
    env = dict(os.environ, LD_PRELOAD=preload, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, DRIVER, kind, lib], env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert f"{kind} ok" in r.stdout.strip().splitlines()[-1]


def test_oracle_under_asan_and_ubsan():
    src = os.path.join(ROOT, "oracle", "hwsel_oracle.c")
    lib = os.path.join(BUILD, "liboracle_san.so")
    os.makedirs(BUILD, exist_ok=True)
    if _stale(lib, [src]):
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC",
                        "-shared", *SAN, src, "-o", lib, "-lm"], check=True)
    preload = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    _run("oracle", lib, preload)


def test_library_host_code_under_asan_and_ubsan():
    sys.path.insert(0, os.path.join(ROOT, "paper_2609_35587_amd"))
    import build as B
    csrc = os.path.join(ROOT, "paper_2609_35587_amd", "csrc")
    sources = [os.path.join(csrc, s) for s in B.SOURCES]
    deps = sources + glob.glob(os.path.join(csrc, "*.hpp")) + [os.path.join(ROOT, "include", "hwsel.h")]
    lib = os.path.join(BUILD, "libhwsel_san.so")
    os.makedirs(BUILD, exist_ok=True)
    if _stale(lib, deps):
        # host pass only: every sanitizer flag goes to the host compiler
        host_san = [x for f in SAN for x in ("-Xarch_host", f)]
        flags = [f for f in B.COMMON if f != "-O3"] + ["-O1", "-g", *host_san]
        procs, objs = [], []
        for src in sources:
            obj = os.path.join(BUILD, os.path.basename(src).replace(".hip", ".san.o"))
            procs.append(subprocess.Popen([B.hipcc(), *flags, *B.PER_FILE.get(os.path.basename(src), []), "-c", src,
                                           "-o", obj], stderr=subprocess.DEVNULL))
            objs.append(obj)
        assert all(p.wait() == 0 for p in procs), "sanitizer build failed"
        subprocess.run([B.hipcc(), "-shared", "-fPIC", f"--offload-arch={B.ARCH}", *objs, "-o", lib], check=True)
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    assert rt, "clang's AddressSanitizer runtime is missing"
    _run("library", lib, rt[0])
