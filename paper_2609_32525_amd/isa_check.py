"""Build check of libflashslice.so's gfx950 machine code: wait states after wide stores.

A vector-memory store of more than 64 bits reads its data registers after it issues, and
the CDNA3/CDNA4 ISA requires wait states before a vector-ALU instruction may overwrite them
(two on gfx94x/gfx950). The compiler inserts them after global stores, but not after the
stores it emits for the raw buffer-resource builtins: compiled without the guard in bst128,
the one-kernel untied backward has a buffer_store_dwordx4 whose first data register the very
next VALU instruction rewrites, the pattern behind a corrupted first dword of some lanes'
dx stores seen in a full-size run. This module disassembles the code objects of the built
library (llvm-objdump, on code built here) and lists every wide store whose data registers a
VALU instruction writes within the required wait states, on every path (both sides of a
branch). build() refuses a library with any.
"""
from __future__ import annotations

import os
import re
import struct
import subprocess
import tempfile
from typing import Dict, List, Tuple

LLVM = os.environ.get("ROCM_LLVM_BIN", "/opt/rocm/llvm/bin")
WAIT_STATES = 2
_BUNDLE = b"__CLANG_OFFLOAD_BUNDLE__"
_STORE = re.compile(r"^(global|buffer|flat|scratch)_store_dwordx([34])\s+(.*)$")
_ADDR = re.compile(r"//\s*([0-9A-Fa-f]+):")
_TARGET = re.compile(r"<([^>+]+)(?:\+0x([0-9a-f]+))?>")


def code_objects(lib: str, outdir: str) -> List[str]:
    """Writes the gfx950 code objects bundled in lib's .hip_fatbin section to outdir."""
    rd = subprocess.run([os.path.join(LLVM, "llvm-readelf"), "-S", lib], capture_output=True,
                        text=True, check=True).stdout
    m = re.search(r"\.hip_fatbin\s+PROGBITS\s+[0-9a-f]+\s+([0-9a-f]+)\s+([0-9a-f]+)", rd)
    if m is None:
        raise RuntimeError(f"{lib}: no .hip_fatbin section")
    with open(lib, "rb") as fh:
        fh.seek(int(m.group(1), 16))
        sec = fh.read(int(m.group(2), 16))
    paths, pos = [], 0
    while True:
        p = sec.find(_BUNDLE, pos)
        if p < 0:
            break
        (n,) = struct.unpack_from("<Q", sec, p + 24)
        q = p + 32
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", sec, q)
            q += 24
            triple = sec[q:q + tlen].decode()
            q += tlen
            if "gfx950" in triple:
                path = os.path.join(outdir, f"co{len(paths)}.o")
                with open(path, "wb") as out:
                    out.write(sec[p + off:p + off + size])
                paths.append(path)
        pos = p + 1
    return paths


def _vregs(tok: str):
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def scan_object(path: str) -> Tuple[int, List[Tuple[str, str, str]]]:
    """(wide stores, violations) of one code object; a violation is (kernel, store, writer)."""
    txt = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--no-show-raw-insn", path],
                         capture_output=True, text=True, check=True).stdout
    insns: List[Tuple[int, str]] = []   # (address, instruction)
    labels: Dict[str, int] = {}         # symbol -> index of its first instruction
    kernel_of: List[str] = []
    kernel = ""
    for line in txt.splitlines():
        s = line.strip()
        if s.endswith(">:"):
            kernel = s[s.index("<") + 1:-2]
            labels[kernel] = len(insns)
            continue
        m = _ADDR.search(s)
        if not m or not s or s.startswith("//"):
            continue
        insns.append((int(m.group(1), 16), s.split("//")[0].strip()))
        kernel_of.append(kernel)
    index = {a: k for k, (a, _) in enumerate(insns)}

    def target(ins: str):
        m = _TARGET.search(ins)
        if not m or m.group(1) not in labels:
            return None
        base = insns[labels[m.group(1)]][0]
        return index.get(base + int(m.group(2) or "0", 16))

    bad = []
    stores = 0

    def walk(k: int, left: int, data, store: str, seen):
        while left > 0 and 0 <= k < len(insns):
            if (k, left) in seen:
                return
            seen.add((k, left))
            ins = insns[k][1]
            name = ins.split()[0]
            if name == "s_nop":
                left -= int(ins.split()[1], 0) + 1
                k += 1
                continue
            if name.startswith("v_"):
                parts = ins.split(None, 1)
                dst = parts[1].split(",")[0].strip() if len(parts) > 1 else ""
                if _vregs(dst) & data:
                    bad.append((kernel_of[k], store, ins))
            left -= 1
            if name in ("s_endpgm", "s_setpc_b64"):
                return
            if name.startswith("s_branch") or name.startswith("s_cbranch"):
                t = target(ins)
                if t is not None:
                    walk(t, left, data, store, seen)
                if name.startswith("s_branch"):
                    return
            k += 1

    for k, (_, ins) in enumerate(insns):
        m = _STORE.match(ins)
        if not m:
            continue
        stores += 1
        ops = [o.strip() for o in m.group(3).split(",")]
        # global / flat / scratch: vaddr (or off), vdata, ...; buffer: vdata, vaddr, ...
        data = _vregs(ops[0]) if m.group(1) == "buffer" else _vregs(ops[1])
        walk(k + 1, WAIT_STATES, data, ins, set())
    return stores, bad


def check_library(lib: str):
    """(wide stores, violations) over every gfx950 code object of the built library."""
    with tempfile.TemporaryDirectory() as d:
        total, bad = 0, []
        for co in code_objects(lib, d):
            n, b = scan_object(co)
            total += n
            bad += b
    return total, bad


if __name__ == "__main__":
    import sys
    here = os.path.dirname(os.path.abspath(__file__))
    n, bad = check_library(sys.argv[1] if len(sys.argv) > 1 else os.path.join(here, "libflashslice.so"))
    print(f"{n} wide stores, {len(bad)} without {WAIT_STATES} wait states before a VALU overwrite")
    for b in bad[:50]:
        print("  ", *b)
    sys.exit(1 if bad else 0)
