"""Fingerprint of one compiled kernel: a hash of its gfx950 machine code and
kernel descriptor, read from the code objects embedded in this package's own
library (libwsgemm.so, built here from source).

Counter records (HBM traffic per launch) are tagged with the fingerprint of
the kernel they were measured on, so they stay valid across source edits that
leave that kernel's code unchanged and lapse as soon as its code changes.

Layout read: the host ELF's ``.hip_fatbin`` section is a sequence of clang
offload bundles (magic ``__CLANG_OFFLOAD_BUNDLE__``, entry count, then
offset / size / target-id per entry); the ``amdgcn-amd-amdhsa--gfx950``
entries are ELF64 code objects whose symbol table locates each kernel's code
(``name``) and descriptor (``name.kd``).
"""
from __future__ import annotations

import hashlib
import os
import struct

_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def _sections(elf: bytes):
    """{name: (sh_addr, sh_offset, sh_size)} of an ELF64 little-endian image."""
    if elf[:4] != b"\x7fELF" or elf[4] != 2:
        raise ValueError("not an ELF64 image")
    shoff = struct.unpack_from("<Q", elf, 0x28)[0]
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", elf, 0x3A)
    raw = []
    for i in range(shnum):
        name, _typ, _flags, addr, off, size = struct.unpack_from("<IIQQQQ", elf, shoff + i * shentsize)
        raw.append((name, addr, off, size))
    stroff = raw[shstrndx][2]
    out = {}
    for name, addr, off, size in raw:
        end = elf.index(b"\0", stroff + name)
        out[elf[stroff + name:end].decode()] = (addr, off, size)
    return out


def _symbols(elf: bytes, secs):
    """{symbol name: (st_value, st_size)} from .symtab / .strtab."""
    _, symoff, symsize = secs[".symtab"]
    _, stroff, _ = secs[".strtab"]
    out = {}
    for i in range(symsize // 24):
        name, _info, _other, _shndx, value, size = struct.unpack_from("<IBBHQQ", elf, symoff + 24 * i)
        if name:
            end = elf.index(b"\0", stroff + name)
            out[elf[stroff + name:end].decode()] = (value, size)
    return out


def _code_objects(lib: bytes, target: str = "gfx950"):
    secs = _sections(lib)
    if ".hip_fatbin" not in secs:
        raise ValueError("no .hip_fatbin section")
    _, base, size = secs[".hip_fatbin"]
    blob = lib[base:base + size]
    pos = blob.find(_MAGIC)
    while pos >= 0:
        n = struct.unpack_from("<Q", blob, pos + len(_MAGIC))[0]
        p = pos + len(_MAGIC) + 8
        for _ in range(n):
            off, sz, tlen = struct.unpack_from("<QQQ", blob, p)
            triple = blob[p + 24:p + 24 + tlen].decode()
            p += 24 + tlen
            if triple.endswith(target) and sz:
                yield blob[pos + off:pos + off + sz]
        pos = blob.find(_MAGIC, pos + 1)


def _bytes_at(elf: bytes, secs, value: int, size: int) -> bytes:
    for addr, off, ssize in secs.values():
        if addr and addr <= value and value + size <= addr + ssize:
            return elf[off + (value - addr):off + (value - addr) + size]
    raise ValueError("symbol outside every section")


# Bytes 16-23 of an AMDHSA kernel descriptor hold the byte offset from the
# descriptor to the kernel's entry: it moves whenever another kernel of the
# code object changes size, so the fingerprint leaves it out.
_KD_ENTRY_OFFSET = slice(16, 24)


def kernel_fingerprint(symbol: str, lib_path: str | None = None) -> str:
    """16 hex digits of SHA-256 over the kernel's code and descriptor bytes
    (without the descriptor's entry offset, which depends on where the
    kernel sits in the code object); raises LookupError if the library holds
    no such kernel."""
    if lib_path is None:
        lib_path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwsgemm.so")
    with open(lib_path, "rb") as f:
        lib = f.read()
    for co in _code_objects(lib):
        secs = _sections(co)
        syms = _symbols(co, secs)
        if symbol in syms and symbol + ".kd" in syms:
            h = hashlib.sha256()
            for name in (symbol, symbol + ".kd"):
                value, size = syms[name]
                data = bytearray(_bytes_at(co, secs, value, size))
                if name.endswith(".kd"):
                    data[_KD_ENTRY_OFFSET] = bytes(8)
                h.update(name.encode() + bytes(data))
            return h.hexdigest()[:16]
    raise LookupError("kernel %s not found in %s" % (symbol, lib_path))


def gemm_symbol(tm, tn, tk, consumer_waves, producer_waves, split, bf16=True, trace=False, mode=0,
                general=False) -> str:
    """Mangled name of ws_gemm_kernel<TM, TN, TK, NC, NP, SPLIT, BF16, TRACE, MODE, GENERAL>."""
    return ("_ZN3wsg14ws_gemm_kernelILi%dELi%dELi%dELi%dELi%dELi%dELb%dELb%dELi%dELb%dEEEvNS_10KernelArgsE"
            % (tm, tn, tk, consumer_waves, producer_waves, split, int(bf16), int(trace), mode, int(general)))
