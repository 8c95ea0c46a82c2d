"""Static check of the image-GEMM kernels' untracked filter loads.

The image GEMM loads its filter operand into registers with
buffer_load_dwordx4 issued as inline assembly, which the compiler does not
track as pending memory operations; correctness then rests on two properties
of the generated code, checked here on the gfx950 assembly of every
img_gemm_kernel instantiation, inside its main loop:

following each load's destination registers cyclically through the loop:
1. until the second s_barrier after the load (each stage waits for the loads
   of the stage before last, s_waitcnt vmcnt, right before its barrier) no
   instruction reads or writes them: the load may still be in flight;
2. from there to the last v_mfma that reads them, nothing writes them and
   only v_mfma instructions read them (no copies, no other use); after that
   the registers are free (the compiler may use them as temporaries).

build.build() runs this check after compiling the library.
"""
from __future__ import annotations

import re
import subprocess

REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")
FUNC = re.compile(r"^(_ZN6miconv15img_gemm_kernel\S+):", re.M)


def _regs(text: str) -> set:
    out = set()
    for m in REG.finditer(text):
        if m.group(3) is not None:
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _loop_lines(body: list) -> list:
    """Instruction lines of the function's loop blocks, in layout order."""
    header = None
    for line in body:
        m = re.search(r"; =>This Inner Loop Header: Depth=1", line)
        if m:
            header = line.split(":")[0].strip()
    if header is None:
        return []
    hdr = header.lstrip(".").replace("LBB", "BB")
    out, inside = [], False
    for line in body:
        t = line.strip()
        if re.match(r"^\.LBB\S+:", t):
            inside = t.split(":")[0] == header or f"Header={hdr}" in t
            continue
        if inside and t and not t.startswith((";", ".")):
            out.append(t.split(";")[0].strip())
    return out


def _dst_src(t: str):
    """(destination registers, source registers) of one instruction line."""
    op = t.split()[0]
    args = [a.strip() for a in t[len(op):].split(",")] if t[len(op):].strip() else []
    if not args:
        return set(), set()
    if op.startswith(("buffer_store", "global_store", "ds_write", "s_")):
        return set(), _regs(t[len(op):])
    return _regs(args[0]), set().union(*(_regs(a) for a in args[1:])) if len(args) > 1 else set()


def check_function(name: str, body: list) -> list:
    """Every untracked load's register set X, followed cyclically through the
    loop from its load: until the second s_barrier (whose wait completes the
    load) no instruction may read or write X; after that, until the last
    v_mfma that reads X, nothing may write X, and only v_mfma may read it."""
    errors = []
    loop = _loop_lines(body)
    n = len(loop)
    for p, t in enumerate(loop):
        # Register loads only: a direct-to-LDS load (suffix "lds") has no
        # destination register and is tracked by the compiler.
        if not t.startswith("buffer_load_dwordx4") or t.split()[-1] == "lds":
            continue
        X = _regs(t.split(",")[0])
        seq = [loop[(p + k) % n] for k in range(1, n)]
        last_read = max((k for k, u in enumerate(seq)
                         if u.startswith("v_mfma") and _dst_src(u)[1] & X), default=-1)
        if last_read < 0:
            errors.append(f"{name}: no v_mfma reads the load '{t}'")
            continue
        barriers = 0
        for k, u in enumerate(seq[:last_read + 1]):
            if u.startswith("s_barrier"):
                barriers += 1
                continue
            d, src = _dst_src(u)
            if barriers < 2 and (d | src) & X:
                errors.append(f"{name}: '{u}' touches {sorted(X)} while its load is in flight")
            elif d & X:
                errors.append(f"{name}: '{u}' overwrites {sorted(X)} before its last use")
            elif src & X and not u.startswith("v_mfma"):
                errors.append(f"{name}: '{u}' reads {sorted(X)} (only v_mfma may)")
    return errors


def check_assembly(text: str) -> list:
    errors, names = [], FUNC.findall(text)
    for name in names:
        i = text.index(name + ":")
        j = text.index(".Lfunc_end", i)
        errors += check_function(name, text[i:j].split("\n"))
    if not names:
        errors.append("no img_gemm_kernel found in the assembly")
    return errors


def compile_assembly(hipcc: str, flags: list, source: str) -> str:
    dev = [f for f in flags if f not in ("-shared", "-fPIC")]
    res = subprocess.run([hipcc] + dev + ["-S", "--cuda-device-only", source, "-o", "-"],
                         stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed ({res.returncode}):\n{res.stderr[-2000:]}")
    return res.stdout


def check(hipcc: str, flags: list, source: str) -> None:
    errors = check_assembly(compile_assembly(hipcc, flags, source))
    if errors:
        raise RuntimeError("untracked-load check failed:\n" + "\n".join(errors[:20]))
