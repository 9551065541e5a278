"""Build libqkn.so (the HIP kernels and their C ABI) for gfx950, in-tree.

    python -m paper_2608_09160_amd.build [--asm]

The library is written to this package's directory so that it travels with
the source tree. `--asm` also writes the gfx950 assembly of each source next
to it (libqkn-<source>-gfx950.s) for inspection of register use and
instruction selection.
"""
from __future__ import annotations

import os
import re
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
# qkn_kern_*.hip instantiate the QK-Norm kernel tables (templates in
# qkn_kernels.h), split so that the units compile in parallel.
SOURCES = [os.path.join(PKG_DIR, "csrc", name)
           for name in ("qkn.hip", "qkn_kern_rows.hip", "qkn_kern_wait.hip", "qkn_kern_wait8.hip",
                        "qkn_kern_misc.hip", "qkn_proj.hip", "qkn_calib.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG_DIR, "libqkn.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 instructions are disabled for all device code: some of their forms
# have produced wrong results on this hardware; plain fp32 code is unaffected.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-I", INCLUDE, "-Wall",
          "-Wno-unused-variable"] + DEVICE_FLAGS


def _run(cmd):
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass does not know the device-only target feature; that warning is harmless
    out = "\n".join(l for l in proc.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"build failed ({proc.returncode}): {' '.join(cmd)}\n{out}")
    return out


# The compiler's per-kernel resource report (one remark per line, "Function
# Name: <symbol>" followed by "<field>: <value>" lines for that kernel).
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]
_REMARK = re.compile(r"remark:\s+(Function Name|ScratchSize \[bytes/lane\]|VGPRs Spill|SGPRs Spill|"
                     r"VGPRs|AGPRs|Occupancy \[waves/SIMD\]|LDS Size \[bytes/block\]): (\S+)")


def kernel_resources(compiler_output: str) -> dict:
    """{kernel symbol: {field: value}} from the resource remarks of one compile."""
    res, cur = {}, None
    for line in compiler_output.splitlines():
        m = _REMARK.search(line)
        if not m:
            continue
        key, val = m.groups()
        if key == "Function Name":
            cur = res.setdefault(val, {})
        elif cur is not None:
            cur[key] = val
    return res


def check_resources(res: dict) -> None:
    """Every kernel keeps its values in registers: no scratch memory and no
    vector-register spills (either would turn the register-resident rows into
    memory traffic). Scalar spills go to vector-register lanes, not memory."""
    bad = [f"{k}: scratch {v.get('ScratchSize [bytes/lane]')} B/lane, "
           f"VGPR spills {v.get('VGPRs Spill')}"
           for k, v in res.items()
           if v.get("ScratchSize [bytes/lane]", "0") != "0" or v.get("VGPRs Spill", "0") != "0"]
    if bad:
        raise RuntimeError("kernels using scratch memory:\n  " + "\n  ".join(bad))


def build(asm: bool = False, verbose: bool = False) -> str:
    """Compile libqkn.so (always recompiles): every source to an object in
    parallel, then one shared library. Fails if any kernel uses scratch
    memory; the per-kernel register, LDS and occupancy figures are written to
    _build/kernel_resources.txt. Returns the library path."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = os.path.join(PKG_DIR, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.splitext(os.path.basename(src))[0] + ".o")
            for src in SOURCES]
    jobs = max(1, min(len(SOURCES), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(jobs) as pool:
        outs = list(pool.map(lambda so: _run([HIPCC, *COMMON, *RESOURCE_REMARKS, "-fPIC", "-c",
                                              "-o", so[1], so[0]]),
                             zip(SOURCES, objs)))
    res = {}
    for o in outs:
        res.update(kernel_resources(o))
    with open(os.path.join(objdir, "kernel_resources.txt"), "w") as f:
        for k in sorted(res):
            f.write(k + "  " + "  ".join(f"{a}={b}" for a, b in sorted(res[k].items())) + "\n")
    check_resources(res)
    # the remarks (and the source excerpts and include chains they quote) are
    # in the resource file; the rest of the output is warnings
    outs = ["\n".join(l for l in o.splitlines() if "kernel-resource-usage" not in l
                       and not l.startswith("In file included from")
                       and not l.strip().startswith(("|", "^")) and not l.strip()[:1].isdigit())
            for o in outs]
    tmp = LIB + ".tmp"
    outs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]))
    os.replace(tmp, LIB)
    out = "\n".join(o for o in outs if o.strip())
    if verbose and out.strip():
        print(out)
    if asm:
        for src in SOURCES:
            stem = os.path.splitext(os.path.basename(src))[0]
            _run([HIPCC, *COMMON, "--cuda-device-only", "-S", "-o",
                  os.path.join(PKG_DIR, f"libqkn-{stem}-{ARCH}.s"), src])
    return LIB


if __name__ == "__main__":
    path = build(asm="--asm" in sys.argv, verbose=True)
    print(path)
