"""Machine code of a kernel in the built library, for tying a measurement to
the exact code it was taken on.

libdflow.so carries one clang offload bundle per HIP source in its
`.hip_fatbin` section; the gfx950 entry of a bundle is an AMDGPU code object
(ELF64).  `kernel_code_digest` hashes a kernel's instructions (its function
symbol) together with its kernel descriptor (`<name>.kd`: register counts, LDS,
kernel-argument size and launch settings) minus the descriptor's code-entry
offset, which only records where the linker placed the code.  The digest
changes when the code that runs changes, and not when other kernels of the
same source file do (unless the kernel's PC-relative references move, which
only makes the check stricter).
"""
from __future__ import annotations

import hashlib
import struct
from typing import Dict, Iterator, List, Tuple

BUNDLE_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
TARGET = b"hipv4-amdgcn-amd-amdhsa--gfx950"
KD_ENTRY_OFFSET = 16   # kernel_code_entry_byte_offset (int64) in the 64-byte kernel descriptor


def _sections(elf: bytes) -> List[Tuple[str, int, int, int, int, int, int]]:
    """(name, type, addr, offset, size, link, entsize) of every section of an ELF64 image."""
    if elf[:4] != b"\x7fELF" or elf[4] != 2:
        raise ValueError("not an ELF64 image")
    shoff, = struct.unpack_from("<Q", elf, 0x28)
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", elf, 0x3A)
    raw = []
    for i in range(shnum):
        name, typ, _flags, addr, off, size, link, _info, _align, entsize = struct.unpack_from(
            "<IIQQQQIIQQ", elf, shoff + i * shentsize)
        raw.append((name, typ, addr, off, size, link, entsize))
    stroff = raw[shstrndx][3]

    def cstr(o):
        return elf[o:elf.index(b"\0", o)].decode()

    return [(cstr(stroff + n), t, a, o, s, l, e) for (n, t, a, o, s, l, e) in raw]


def code_objects(lib_path: str) -> Iterator[bytes]:
    """The gfx950 code objects of every offload bundle in the library."""
    with open(lib_path, "rb") as f:
        so = f.read()
    fat = [s for s in _sections(so) if s[0] == ".hip_fatbin"]
    if not fat:
        raise ValueError(f"{lib_path}: no .hip_fatbin section")
    _, _, _, off, size, _, _ = fat[0]
    blob = so[off:off + size]
    pos = blob.find(BUNDLE_MAGIC)
    while pos >= 0:
        n, = struct.unpack_from("<Q", blob, pos + len(BUNDLE_MAGIC))
        p = pos + len(BUNDLE_MAGIC) + 8
        for _ in range(n):
            eoff, esize, tlen = struct.unpack_from("<QQQ", blob, p)
            triple = blob[p + 24:p + 24 + tlen]
            p += 24 + tlen
            if triple == TARGET and esize > 0:
                yield blob[pos + eoff:pos + eoff + esize]
        pos = blob.find(BUNDLE_MAGIC, p)


def symbols(co: bytes) -> Dict[str, bytes]:
    """name -> bytes of every sized symbol of a code object (.symtab, else .dynsym)."""
    secs = _sections(co)
    tabs = [s for s in secs if s[0] == ".symtab"] or [s for s in secs if s[0] == ".dynsym"]
    if not tabs:
        return {}
    _, _, _, off, size, link, entsize = tabs[0]
    stroff = secs[link][3]
    out = {}
    for i in range(size // entsize):
        name, _info, _other, shndx, value, sz = struct.unpack_from("<IBBHQQ", co, off + i * entsize)
        if sz == 0 or shndx == 0 or shndx >= len(secs):
            continue
        nm = co[stroff + name:co.index(b"\0", stroff + name)].decode()
        _, typ, addr, soff, _, _, _ = secs[shndx]
        if typ == 8:      # SHT_NOBITS: no bytes in the image
            continue
        out[nm] = co[soff + value - addr:soff + value - addr + sz]
    return out


def kernel_code_digest(lib_path: str, symbol: str) -> str:
    """sha256 over a kernel's instructions and its kernel descriptor."""
    for co in code_objects(lib_path):
        syms = symbols(co)
        if symbol in syms:
            h = hashlib.sha256()
            h.update(syms[symbol])
            kd = bytearray(syms.get(symbol + ".kd", b""))
            if len(kd) >= KD_ENTRY_OFFSET + 8:
                kd[KD_ENTRY_OFFSET:KD_ENTRY_OFFSET + 8] = bytes(8)
            h.update(bytes(kd))
            return h.hexdigest()
    raise KeyError(f"{symbol} not found in {lib_path}")


def kernel_symbols(lib_path: str, needle: str) -> List[str]:
    """Kernel entry symbols (those with a descriptor) whose name contains `needle`."""
    out = []
    for co in code_objects(lib_path):
        syms = symbols(co)
        out += sorted(n for n in syms if needle in n and n + ".kd" in syms)
    return out
