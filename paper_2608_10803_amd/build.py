"""Build libadaptcore.so (gfx950) in-tree with hipcc.

    python -m paper_2608_10803_amd.build [--if-stale] [--incremental]

Every source is compiled to an object under _build/ (in parallel) and linked
into paper_2608_10803_amd/libadaptcore.so. Device code is compiled with
packed-fp32 instructions disabled.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libadaptcore.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["kernels.hip", "kernels_dl.hip", "kernels_tall.hip", "planner.cpp", "adaptcore.cpp", "noalloc.hip"]
# compilation units: (source, object name, extra flags); the kernels are
# compiled once per input format (bf16, and fp16 in namespace ac::f16)
UNITS = [("kernels.hip", "kernels.hip.o", []), ("kernels.hip", "kernels_f16.hip.o", ["-DAC_INPUT_F16=1"]),
         ("kernels_dl.hip", "kernels_dl.hip.o", []), ("kernels_dl.hip", "kernels_dl_f16.hip.o", ["-DAC_INPUT_F16=1"]),
         ("kernels_tall.hip", "kernels_tall.hip.o", []),
         ("kernels_tall.hip", "kernels_tall_f16.hip.o", ["-DAC_INPUT_F16=1"]),
         ("planner.cpp", "planner.cpp.o", []), ("adaptcore.cpp", "adaptcore.cpp.o", []),
         ("noalloc.hip", "noalloc.hip.o", [])]
HEADERS = ["kernel_args.h", "variants.h", "planner.h", "registry.h", "noalloc.h", "device_common.h"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH, "-Wall", "-Wno-unused-function",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I" + os.path.join(ROOT, "include")]


def _inputs():
    files = [os.path.join(CSRC, s) for s in SOURCES + HEADERS]
    files.append(os.path.join(ROOT, "include", "adaptcore.h"))
    return files


def stale():
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in _inputs())


def _obj_stale(unit):
    src, name, _ = unit
    obj = os.path.join(BUILD, name)
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    deps = [os.path.join(CSRC, src)] + [os.path.join(CSRC, h) for h in HEADERS]
    deps.append(os.path.join(ROOT, "include", "adaptcore.h"))
    return any(os.path.getmtime(f) > t for f in deps)


def _compile(unit):
    src, name, extra = unit
    obj = os.path.join(BUILD, name)
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC] + COMMON + extra + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s" % (" ".join(cmd), err))
    return obj, err


def build(verbose=False, incremental=False):
    """Compiles every unit (incremental=True: only units whose object is older
    than its source or a header) and links the library."""
    os.makedirs(BUILD, exist_ok=True)
    todo = [u for u in UNITS if not incremental or _obj_stale(u)]
    with cf.ThreadPoolExecutor(max(1, len(todo))) as ex:
        results = list(ex.map(_compile, todo))
    for _, err in results:
        if verbose and err.strip():
            print(err, file=sys.stderr)
    objs = [os.path.join(BUILD, name) for _, name, _ in UNITS]
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    if "--if-stale" in sys.argv and not stale():
        print(LIB, "(up to date)")
    else:
        print(build(verbose=True, incremental="--incremental" in sys.argv))
