"""Build libasymspec.so (gfx950) in-tree with hipcc."""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "asymspec.hip")
INC = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libasymspec.so")
# per-kernel register and scratch use reported by the compiler for the last
# build (a kernel that spills to scratch loses most of its read rate)
RESOURCES = os.path.join(HERE, "libasymspec.resources.txt")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep the compiler from emitting packed-FP32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False, extra=()) -> str:
    tmp = OUT + ".tmp"
    cmd = [HIPCC, *FLAGS, "-Rpass-analysis=kernel-resource-usage", "-fno-caret-diagnostics", *extra, "-I", INC, SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = (r.stdout + r.stderr).splitlines()
    usage = [l for l in lines if "kernel-resource-usage" in l]
    msg = "\n".join(l for l in lines if "packed-fp32-ops" not in l and "unknown target feature" not in l
                    and "kernel-resource-usage" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{msg}")
    if verbose and msg.strip():
        print(msg)
    os.replace(tmp, OUT)
    with open(RESOURCES, "w") as f:
        f.write(resource_report(usage))
    return OUT


def resource_report(lines) -> str:
    """One line per kernel: name, VGPRs, scratch bytes per lane, occupancy."""
    rows, cur = [], {}
    for l in lines:
        txt = l.split("remark:", 1)[-1].split("[-Rpass", 1)[0].strip()
        key, _, val = txt.partition(":")
        key, val = key.strip(), val.strip()
        if key == "Function Name":
            if cur:
                rows.append(cur)
            cur = {"name": val}
        elif key in ("VGPRs", "ScratchSize [bytes/lane]", "Occupancy [waves/SIMD]"):
            cur[key.split()[0]] = val
    if cur:
        rows.append(cur)
    return "".join(f"{r['name']} vgprs={r.get('VGPRs', '?')} scratch={r.get('ScratchSize', '?')} "
                   f"occupancy={r.get('Occupancy', '?')}\n" for r in rows)


EXAMPLE_SRC = os.path.join(HERE, "examples", "fuse_verify_c.cpp")
EXAMPLE = os.path.join(HERE, "examples", "fuse_verify_c")


def build_example(verbose: bool = False) -> str:
    """The C-ABI example, a host program linked against libasymspec.so."""
    cmd = [HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17", "-I", INC, EXAMPLE_SRC,
           "-L", HERE, "-lasymspec", f"-Wl,-rpath,{HERE}", "-o", EXAMPLE]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"example build failed ({r.returncode}):\n{r.stdout}{r.stderr}")
    if verbose:
        print(f"built {EXAMPLE}")
    return EXAMPLE


PROBE_SRC = os.path.join(HERE, "csrc", "probe.hip")
PROBE = os.path.join(HERE, "libasymspec_probe.so")


def build_probe(verbose: bool = False) -> str:
    """libasymspec_probe.so: the read-ceiling probe (not the decision step)."""
    tmp = PROBE + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", INC, PROBE_SRC, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"probe build failed ({r.returncode}):\n{r.stdout}{r.stderr}")
    os.replace(tmp, PROBE)
    if verbose:
        print(f"built {PROBE}")
    return PROBE


if __name__ == "__main__":
    print(build(verbose=True))
    build_example(verbose=True)
    build_probe(verbose=True)
    sys.exit(0)
