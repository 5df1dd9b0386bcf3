"""Static check of the kernels' gfx950 assembly for the inline-assembly
loads' register discipline.

The kernels issue LDS reads (and a few global loads) as inline assembly so
that the compiler's own waits do not tie them to loads of later tiles; the
compiler then believes their destination registers are written at issue.
Each such value is waited for explicitly (s_waitcnt lgkmcnt / vmcnt) and
passed through an empty volatile statement before use.  If the compiler
moved, copied or reused one of those registers before the wait (which it
may do under register pressure), the kernel would read or clobber data
still in flight.  This module compiles the launch translation units to
assembly and reports, within straight-line code, every instruction that
touches a register whose load may still be outstanding: memory operations
complete in issue order per counter, so after `s_waitcnt lgkmcnt(N)` only
the N youngest LDS/scalar-memory operations can be in flight (vmcnt
likewise for vector-memory ones).  Outstanding operations are dropped at
labels and branches (the kernels wait for their reads within a block).

    python -m paper_2609_04523_amd.asm_check      # compile and check all
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import subprocess
import sys
import tempfile

from paper_2609_04523_amd import build

LAUNCH_UNITS = [s for s in build.SOURCES if not s.endswith("mk_attn.hip")]


def _regs(text: str):
    out = set()
    for m in re.finditer(r"\b([va])\[(\d+):(\d+)\]", text):
        out.update((m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
    for m in re.finditer(r"\b([va])(\d+)\b", text):
        out.add((m.group(1), int(m.group(2))))
    return out


def _retire(pending, n):
    return pending[len(pending) - n:] if 0 < n < len(pending) else ([] if n == 0 else pending)


def hazards(asm: str):
    """[(function, line index, instruction, load line index)] for every
    instruction that touches a register of a load that may be in flight."""
    found = []
    for name, body in re.findall(r"^(_Z\w+):[^\n]*\n(.*?)^\.Lfunc_end", asm, re.M | re.S):
        lgkm, vm = [], []  # (destination registers, line) in issue order
        for k, raw in enumerate(body.split("\n")):
            line = raw.strip()
            if not line or line.startswith(";"):
                continue
            if line.endswith(":"):  # a label: control may enter from elsewhere
                lgkm, vm = [], []
                continue
            if line.startswith("."):
                continue
            op = line.split()[0]
            args = line[len(op):]
            if op == "s_waitcnt":
                m = re.search(r"lgkmcnt\((\d+)\)", line)
                if m:
                    lgkm = _retire(lgkm, int(m.group(1)))
                m = re.search(r"vmcnt\((\d+)\)", line)
                if m:
                    vm = _retire(vm, int(m.group(1)))
                continue
            if op.startswith(("s_cbranch", "s_branch", "s_setpc", "s_endpgm")):
                lgkm, vm = [], []
                continue
            touched = _regs(args)
            for dest, at in lgkm + vm:
                if touched & dest:
                    found.append((name, k, line, at))
            if op.startswith(("global_load", "buffer_load", "scratch_load")):
                # LDS-DMA forms name an address register, not a destination
                dest = set() if (" lds" in line or "_lds_" in op) else _regs(args.split(",")[0])
                vm.append((dest, k))
            elif op.startswith(("global_store", "buffer_store", "scratch_store", "global_atomic",
                                "buffer_atomic")):
                vm.append((set(), k))
            if op.startswith(("ds_read", "ds_load")):
                lgkm.append((_regs(args.split(",")[0]), k))
            elif op.startswith(("s_load", "s_buffer_load", "ds_")):
                lgkm.append((set(), k))
    return found


def compile_asm(src: str, out: str) -> None:
    cmd = [build.HIPCC, *[f for f in build.FLAGS if f != "-fPIC"], "--cuda-device-only", "-S",
           src, "-o", out]
    subprocess.run(cmd, check=True, stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)


def check_all(workers: int = 8):
    """{translation unit: hazards} for every launch translation unit."""
    with tempfile.TemporaryDirectory() as tmp:
        outs = {s: os.path.join(tmp, os.path.basename(s) + ".s") for s in LAUNCH_UNITS}
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(lambda s: compile_asm(s, outs[s]), LAUNCH_UNITS))
        return {os.path.basename(s): hazards(open(outs[s]).read()) for s in LAUNCH_UNITS}


if __name__ == "__main__":
    res = check_all()
    bad = 0
    for unit, hz in res.items():
        print(f"{unit}: {len(hz)} hazards")
        for name, k, line, at in hz[:5]:
            print(f"  {name[:70]} line {k}: {line[:80]} (load at line {at})")
        bad += len(hz)
    sys.exit(1 if bad else 0)
