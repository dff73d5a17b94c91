"""Post-build check of the library's gfx950 machine code: no MFMA may run under a
possibly-empty EXEC mask.

Matrix-core instructions do not honour EXEC: an MFMA reached with EXEC = 0
still reads its operands and writes its accumulator.  The compiler may lower
a branch on a per-lane value to an EXEC mask alone and drop the
s_cbranch_execz that skips a short block, so a guarded MFMA then runs
unguarded.  The kernels avoid such branches around MFMAs; this check scans
the disassembly of every built object (code built here, with the toolchain's
own llvm-objdump) and reports each MFMA that follows an EXEC-narrowing write
in program order with no execz skip or EXEC restore in between.
"""
from __future__ import annotations

import os
import re
import struct
import subprocess
import tempfile

LLVM_BIN = os.environ.get("OQ_LLVM_BIN", "/opt/rocm/llvm/bin")
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"

# Writes that may leave EXEC narrower than on entry (or empty).
_NARROW = re.compile(r"^(s_(and|andn2|xor|or|orn2|nand|nor|xnor|andn1|orn1)_saveexec_b64\b"
                     r"|s_(and|andn2|xor|mov|cselect|nand|nor|xnor|andn1|orn1)_b64 exec,"
                     r"|v_cmpx_)")
_RESTORE = re.compile(r"^(s_or_b64 exec, exec,|s_mov_b64 exec, -1\b)")
_SKIP = re.compile(r"^s_cbranch_execz\b")
_MFMA = re.compile(r"^v_(mfma|smfmac)_")
_FUNC = re.compile(r"^[0-9a-f]+ <([^>]+)>:")


def unguarded_mfma(disassembly: str) -> list[tuple[str, str]]:
    """(function, instruction) for every MFMA that may run with a narrowed EXEC and no skip."""
    hits = []
    fn, pending = None, False
    for line in disassembly.splitlines():
        m = _FUNC.match(line)
        if m:
            fn, pending = m.group(1), False
            continue
        ins = line.split("//")[0].strip()
        if not ins:
            continue
        if _SKIP.match(ins) or _RESTORE.match(ins):
            pending = False
        elif _NARROW.match(ins):
            pending = True
        elif pending and _MFMA.match(ins):
            hits.append((fn, ins))
    return hits


def device_code(obj: str) -> bytes:
    """The gfx950 code object embedded in a host object built by hipcc -c (empty if none)."""
    with tempfile.TemporaryDirectory() as d:
        sec = os.path.join(d, "fatbin")
        r = subprocess.run([os.path.join(LLVM_BIN, "llvm-objcopy"), f"--dump-section=.hip_fatbin={sec}", obj,
                            os.path.join(d, "stripped")], capture_output=True, text=True)
        if r.returncode != 0 or not os.path.exists(sec):
            return b""  # no device code in this object
        b = open(sec, "rb").read()
    if not b.startswith(_MAGIC):
        raise RuntimeError(f"{obj}: unexpected device code bundle")
    p = len(_MAGIC)
    (n,) = struct.unpack_from("<Q", b, p)
    p += 8
    for _ in range(n):
        off, size, tl = struct.unpack_from("<QQQ", b, p)
        p += 24
        triple = b[p:p + tl].decode()
        p += tl
        if triple == TARGET:
            return b[off:off + size]
    raise RuntimeError(f"{obj}: no {TARGET} code object")


def disassemble(code: bytes) -> str:
    with tempfile.NamedTemporaryFile(suffix=".co") as f:
        f.write(code)
        f.flush()
        r = subprocess.run([os.path.join(LLVM_BIN, "llvm-objdump"), "-d", "--mcpu=gfx950", f.name],
                           capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"llvm-objdump failed: {r.stderr}")
    return r.stdout


def tools_present() -> bool:
    return all(os.path.exists(os.path.join(LLVM_BIN, t)) for t in ("llvm-objcopy", "llvm-objdump"))


def check_objects(objs: list[str]) -> list[tuple[str, str, str]]:
    """(object, function, instruction) for every unguarded MFMA in the given objects (empty, with a
    warning on stderr, when the toolchain's llvm-objcopy / llvm-objdump are not there to run the check)."""
    if not tools_present():
        import sys
        print(f"isa_check: llvm-objcopy / llvm-objdump not found under {LLVM_BIN}; machine-code check skipped",
              file=sys.stderr)
        return []
    out = []
    for obj in objs:
        code = device_code(obj)
        if code:
            out += [(os.path.basename(obj), fn, ins) for fn, ins in unguarded_mfma(disassemble(code))]
    return out
