"""Build ``libpagedattn.so`` (the gfx950 kernels and their C ABI) in-tree with
hipcc.  Every HIP source is compiled for gfx950 only, with packed-fp32 VALU
instructions disabled (the compiler would otherwise form them from plain fp32
code); the host-only C++ sources (``*.cpp``) are compiled with g++; all are
linked into one shared library."""
import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libpagedattn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-I", os.path.join(ROOT, "include"), "-I", CSRC]

# Host-code sanitizer build (device code unchanged): every host pass gets
# AddressSanitizer and UndefinedBehaviorSanitizer, so the planning and
# validation of the C ABI can run under them in the CPU test suites
# (PAGEDATTN_LIB=<this path>, with clang's ASan runtime preloaded).
LIB_ASAN = os.path.join(OUT_DIR, "libpagedattn_asan.so")
SAN = ["-fsanitize=address", "-fsanitize=undefined"]
SAN_HIP = [f for s in SAN for f in ("-Xarch_host", s)] + [
    "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def _compile(src, obj, verbose, sanitize=False, defines=()):
    if src.endswith(".cpp"):
        if sanitize:  # clang's sanitizer runtime is the one loaded: compile with clang too
            cmd = [os.path.join(os.path.dirname(HIPCC), "amdclang++"), *HOST_FLAGS, *SAN,
                   "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-c", src, "-o", obj]
        else:
            cmd = ["g++", *HOST_FLAGS, "-c", src, "-o", obj]
    else:
        cmd = [HIPCC, *FLAGS, *(SAN_HIP if sanitize else []), *[f"-D{d}" for d in defines], "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"{cmd[0]} failed on {src}:\n{err}")
    if err.strip() and verbose:
        print(err)


def build(verbose: bool = False, sanitize: bool = False, defines=(), out: str | None = None) -> str:
    """Build the library.  defines: extra NAME=VALUE macros for the HIP
    sources (tuning switches such as PA_STREAM_MFMA=0, the VALU fold of the
    decode kernel); out: another output path for such a variant (load it with
    PAGEDATTN_LIB=<path>)."""
    os.makedirs(OUT_DIR, exist_ok=True)
    out = out or (LIB_ASAN if sanitize else LIB)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    tag = "_asan" if sanitize else ("_" + os.path.splitext(os.path.basename(out))[0] if out != LIB else "")
    objs = [os.path.join(OUT_DIR, os.path.splitext(os.path.basename(s))[0] + tag + ".o") for s in srcs]
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        list(ex.map(lambda so: _compile(so[0], so[1], verbose, sanitize, defines), zip(srcs, objs)))
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *(SAN_HIP if sanitize else []), "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    for o in objs:
        os.remove(o)
    return out


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--sanitize-host", action="store_true")
    ap.add_argument("--define", action="append", default=[], help="NAME=VALUE macro for the HIP sources")
    ap.add_argument("--out", default=None, help="output path of a variant build")
    a = ap.parse_args()
    print(build(verbose=True, sanitize=a.sanitize_host, defines=a.define,
                out=os.path.abspath(a.out) if a.out else None))
