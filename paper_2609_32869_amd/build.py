"""Build libwf.so (HIP kernels + C ABI) for gfx950 in-tree with hipcc."""
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwf.so")
OBJDIR = os.path.join(os.path.dirname(HERE), "_build")
SOURCES = ["k_gemv.hip", "k_attn.hip", "k_misc.hip", "k_mm.hip", "k_enc.hip", "wf_api.hip", "enc_api.hip"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         # packed fp32 arithmetic is kept out of every kernel
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-result",
         # per-kernel register / scratch report, checked below
         "-Rpass-analysis=kernel-resource-usage"]


def _filter(text):
    """Drop the packed-fp32 feature notes and the resource-usage remarks (each
    followed by its source excerpt)."""
    keep, in_remark = [], False
    for line in text.splitlines():
        if "packed-fp32-ops" in line:
            continue
        if "kernel-resource-usage" in line:
            in_remark = True
            continue
        if in_remark and re.match(r"^\s*(\d+\s*)?\|", line):
            continue
        in_remark = False
        keep.append(line)
    return "\n".join(keep)


def _scratch_kernels(text):
    """Kernels whose registers spill to scratch memory: a launch of such a kernel
    pays for per-dispatch scratch set-up, so none is allowed."""
    bad, name = [], None
    for line in text.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            bad.append(f"{name} ({m.group(1)} bytes/lane)")
    return bad


def build(verbose=False):
    """Compile every source to an object (in parallel), then link libwf.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJDIR, exist_ok=True)
    procs, objs = [], []
    for s in SOURCES:
        obj = os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o")
        objs.append(obj)
        cmd = [hipcc] + FLAGS + ["-c", os.path.join(CSRC, s), "-o", obj]
        procs.append((s, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    errors, notes = [], []
    for s, p in procs:
        raw = p.communicate()[0]
        out = _filter(raw)
        if p.returncode != 0:
            errors.append(f"{s}: hipcc failed ({p.returncode}):\n{out}")
            continue
        spills = _scratch_kernels(raw)
        if spills:
            errors.append(f"{s}: kernels spill registers to scratch: " + ", ".join(spills))
        if out.strip():
            notes.append(f"{s}:\n{out}")
    if errors:
        raise RuntimeError("\n".join(errors))
    if verbose and notes:
        print("\n".join(notes))
    tmp = LIB + ".tmp"
    r = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed ({r.returncode}):\n{_filter(r.stdout + r.stderr)}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
