"""Build liblamp.so (HIP for gfx950) in-tree.

`python -m paper_2609_39361_amd.build` (or build()) compiles the kernels and
the C ABI with hipcc into paper_2609_39361_amd/liblamp.so.  Flags:
  * -ffp-contract=off: every fused multiply-add is an explicit fma call, the
    stage-2 cost sums and the exponential code paths round every operation;
  * -Xclang -target-feature -Xclang -packed-fp32-ops: no packed fp32
    arithmetic is generated.

The logit loops issue DPP instructions from inline assembly, which the
compiler's hazard recognizer does not look into.  The build therefore keeps
the device assembly of the same compile (-save-temps) and rejects the library
if a DPP instruction reads a VGPR that a VALU instruction wrote less than two
wait states earlier, or follows a VALU write of EXEC by less than five (the
CDNA3/CDNA4 ISA's required wait states for DPP).
"""
import glob
import os
import re
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblamp.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["lamp_kernels.hip", "lamp_fwd.hip", "lamp_fwd16.hip", "lamp_fwd16_sr.hip", "lamp_decode.hip", "lamp_rates.hip",
           "lamp_noalloc.hip", "lamp_host.cpp"]

DPP_VGPR_WAITS = 2
DPP_EXEC_WAITS = 5
_HIST = max(DPP_VGPR_WAITS, DPP_EXEC_WAITS)


def _vgprs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return frozenset(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return frozenset([int(m.group(1))]) if m else frozenset()


def _operands(line):
    parts = line.split(None, 1)
    if len(parts) < 2:
        return []
    return [t.strip() for t in parts[1].split(",")]


def _slot(line):
    """(vgprs written by a VALU op, whether it is a VALU write of EXEC)."""
    op = line.split()[0]
    if not op.startswith("v_"):
        return (frozenset(), False)
    ops = _operands(line)
    if op.startswith("v_cmpx"):
        return (frozenset(), True)
    if not ops:
        return (frozenset(), False)
    first = ops[0].split()[0]
    if first == "exec" or first.startswith("exec"):
        return (frozenset(), True)
    if op.startswith(("v_cmp", "v_readlane", "v_readfirstlane")):
        return (frozenset(), False)
    return (_vgprs(first), False)


def _merge(a, b):
    if a is None:
        return b
    return tuple((x[0] | y[0], x[1] or y[1]) for x, y in zip(a, b))


def scan_dpp_hazards(asm):
    """Hazards in device assembly text: list of (dpp line, reason).

    The history of the last few wait states is tracked along the instruction
    stream; at a label it is merged over every branch that jumps there (to a
    fixed point, for loops) and the fall-through path."""
    lines = []
    for raw in asm.splitlines():
        s = raw.split(";")[0].strip()
        if not s or s.startswith("."):
            if re.match(r"^\.L\w+:$", s or ""):
                lines.append(("label", s[:-1]))
            continue
        if s.endswith(":"):
            lines.append(("label", s[:-1]))
            continue
        lines.append(("ins", s))

    empty = tuple((frozenset(), False) for _ in range(_HIST))
    at_label = {}
    for _ in range(8):
        changed = False
        hist = empty
        fall = True
        found = []
        for kind, s in lines:
            if kind == "label":
                h = at_label.get(s)
                hist = _merge(hist if fall else None, h) if h is not None else (hist if fall else empty)
                fall = True
                continue
            op = s.split()[0]
            if "_dpp" in op or "row_newbcast" in s or "row_bcast" in s or "quad_perm" in s \
                    or "row_shl" in s or "row_shr" in s or "row_ror" in s:
                ops = _operands(s)
                src0 = _vgprs(ops[1]) if len(ops) > 1 else frozenset()
                for dist in range(DPP_VGPR_WAITS):
                    if hist[dist][0] & src0:
                        found.append((s, "src VGPR written %d wait state(s) earlier" % (dist + 1)))
                for dist in range(DPP_EXEC_WAITS):
                    if hist[dist][1]:
                        found.append((s, "EXEC written by VALU %d wait state(s) earlier" % (dist + 1)))
            if op == "s_nop":
                n = int(s.split()[1], 0) + 1 if len(s.split()) > 1 else 1
                slots = [(frozenset(), False)] * n
            else:
                slots = [_slot(s)]
            for sl in slots:
                hist = (sl,) + hist[:-1]
            m = re.match(r"^s_(c?branch\w*)\s+(\.L\w+)", s)
            if m:
                tgt = m.group(2)
                new = _merge(at_label.get(tgt), hist)
                if new != at_label.get(tgt):
                    at_label[tgt] = new
                    changed = True
                if m.group(1) == "branch":
                    fall = False
            elif op in ("s_endpgm", "s_setpc_b64"):
                fall = False
        if not changed:
            return sorted(set(found))
    return sorted(set(found))


def _compile(src, work, flags, verbose):
    """One source to an object in its own directory (device assembly kept)."""
    sub = os.path.join(work, os.path.splitext(os.path.basename(src))[0])
    os.makedirs(sub, exist_ok=True)
    obj = os.path.join(sub, os.path.basename(src) + ".o")
    cmd = [HIPCC] + flags + ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, cwd=sub)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops' is not a recognized feature" not in l)
    return r.returncode, obj, out


PHASE_LIB = os.path.join(HERE, "liblamp_phase.so")


def build(verbose=False, extra=(), out=LIB):
    """Compile the library into `out` (default liblamp.so).  build_phase()
    makes the measurement variant with the phase timer."""
    from concurrent.futures import ThreadPoolExecutor
    tmp = out + ".tmp%d" % os.getpid()
    flags = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
             "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             "-Wno-unused-command-line-argument", "-save-temps"] + list(extra)
    jobs = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", "0")) or (os.cpu_count() or 1)))
    with tempfile.TemporaryDirectory(prefix="lamp_build_") as work:
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            res = list(ex.map(lambda s: _compile(os.path.join(CSRC, s), work, flags, verbose), SOURCES))
        failed = [out for rc, _, out in res if rc != 0]
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
        for _, _, msg in res:
            if verbose and msg.strip():
                print(msg)
        link = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC"] + [o for _, o, _ in res] + ["-o", tmp]
        if verbose:
            print(" ".join(link), flush=True)
        r = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, cwd=work)
        if r.returncode != 0:
            if os.path.exists(tmp):
                os.remove(tmp)
            raise RuntimeError("link failed:\n" + r.stdout)
        asm_files = sorted(glob.glob(os.path.join(work, "*", "*-hip-amdgcn-amd-amdhsa-" + ARCH + ".s")))
        names = {os.path.basename(f).split("-hip-")[0] for f in asm_files}
        if not {"lamp_fwd", "lamp_fwd16", "lamp_decode", "lamp_kernels"} <= names:
            os.remove(tmp)
            raise RuntimeError("device assembly of the kernel sources missing: %r" % asm_files)
        bad = []
        for f in asm_files:
            with open(f) as fh:
                bad += [(os.path.basename(f), s, why) for s, why in scan_dpp_hazards(fh.read())]
        if bad:
            os.remove(tmp)
            raise RuntimeError("DPP hazards in the generated code:\n" +
                               "\n".join("%s: %s  (%s)" % b for b in bad[:20]))
    os.replace(tmp, out)
    return out


def build_phase(verbose=False):
    """liblamp_phase.so: the library with the pipelined kernel's phase timer
    (-DLAMP_PHASE_TIMER), for measurement; load it with LAMP_LIBRARY."""
    return build(verbose, extra=("-DLAMP_PHASE_TIMER",), out=PHASE_LIB)


if __name__ == "__main__":
    if "--phase-timer" in sys.argv:
        build_phase(verbose=True)
    else:
        build(verbose=True)
    sys.exit(0)
