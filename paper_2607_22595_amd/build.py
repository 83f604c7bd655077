"""Build libxmix.so (HIP for gfx950) in-tree.

Each source under csrc/ is compiled by hipcc into _build/, then linked into
paper_2607_22595_amd/libxmix.so.  The measured-ceiling kernels under
ceiling/ (a benchmark aid, no part of the hook step) become
libxmix_ceiling.so.  Packed-fp32 instruction selection is switched off for
device code."""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _compile(src: str, obj: str, extra) -> None:
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    # the host pass does not know the packed-fp32 feature; drop that warning
    noise = [ln for ln in r.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln]
    if noise:
        sys.stderr.write("\n".join(noise) + "\n")


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)


def build(extra=(), jobs: int = 8) -> str:
    out_dir = os.path.join(ROOT, "_build")
    os.makedirs(out_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))
    objs = [os.path.join(out_dir, os.path.basename(s) + ".o") for s in srcs]
    ceil_src = os.path.join(HERE, "ceiling", "ceiling.hip")
    ceil_obj = os.path.join(out_dir, "ceiling.hip.o")
    pairs = list(zip(srcs, objs)) + [(ceil_src, ceil_obj)]
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(lambda so: _compile(so[0], so[1], list(extra)), pairs))
    lib = os.path.join(HERE, "libxmix.so")
    _link(objs, lib)
    _link([ceil_obj], os.path.join(HERE, "libxmix_ceiling.so"))
    return lib


if __name__ == "__main__":
    print(build())
