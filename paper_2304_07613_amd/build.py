"""Build step for libnmg.so (hipcc, gfx950) -- run by ``__graft_entry__.build()``.

Every translation unit under csrc/ is compiled to an object in parallel, then
the objects are linked into one shared library; the link is checked for
undefined kernel launch stubs.  csrc/gen_gelu_table.py writes the binary16
GELU table into the build folder first.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
HEADER = os.path.join(ROOT, "include", "nmg.h")
LIB_PATH = os.path.join(HERE, "libnmg.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # no packed binary32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # binary32 subnormals take part in the group scores: never flush them
    "-fno-gpu-flush-denormals-to-zero", "-fno-fast-math",
]


def sources() -> list:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


GENERATORS = [os.path.join(CSRC, "gen_gelu_table.py")]


def inputs() -> list:
    """Every file the library is built from."""
    return sorted(sources() + glob.glob(os.path.join(CSRC, "*.hpp")) + [HEADER] + GENERATORS)


def _clean(text: str) -> str:
    return "\n".join(l for l in text.splitlines()
                     if "packed-fp32-ops" not in l and "not a recognized feature" not in l)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile csrc/*.hip into libnmg.so next to this file (always rebuilds)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    jobs = jobs or min(16, os.cpu_count() or 4)
    inc = ["-I", os.path.join(ROOT, "include")]
    with tempfile.TemporaryDirectory(prefix="nmg_build_") as tmpdir:
        # generated sources (the binary16 GELU table) go to the build folder
        gen = subprocess.run([sys.executable, GENERATORS[0], os.path.join(tmpdir, "gelu_f16_table.inc")],
                             capture_output=True, text=True)
        if gen.returncode != 0:
            raise RuntimeError(f"gen_gelu_table.py failed:\n{gen.stdout}{gen.stderr}")
        inc += ["-I", tmpdir]
        def compile_one(src):
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            res = subprocess.run([hipcc, *HIPCC_FLAGS, *inc, "-c", "-o", obj, src],
                                 capture_output=True, text=True)
            return src, obj, res
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            results = list(pool.map(compile_one, sources()))
        errors = [(s, r) for s, _, r in results if r.returncode != 0]
        if errors:
            s, r = errors[0]
            raise RuntimeError(f"hipcc failed on {os.path.basename(s)}:\n{_clean(r.stdout + r.stderr)}")
        if verbose:
            for s, _, r in results:
                out = _clean(r.stdout + r.stderr).strip()
                if out:
                    print(f"{os.path.basename(s)}:\n{out}")
        tmp = LIB_PATH + ".tmp"
        res = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp,
                              *[o for _, o, _ in results]], capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed:\n{_clean(res.stdout + res.stderr)}")
    # every kernel's host launch stub must be defined in the library
    nm = subprocess.run(["nm", "-D", "--undefined-only", tmp], capture_output=True, text=True)
    missing = [l.split()[-1] for l in nm.stdout.splitlines() if "__device_stub__" in l]
    if nm.returncode != 0 or missing:
        raise RuntimeError(f"libnmg.so has undefined kernel stubs: {missing[:3]} (nm rc {nm.returncode})")
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def is_stale() -> bool:
    if not os.path.exists(LIB_PATH):
        return True
    t = os.path.getmtime(LIB_PATH)
    return any(os.path.getmtime(p) > t for p in inputs())


if __name__ == "__main__":
    print(build(verbose=True))
