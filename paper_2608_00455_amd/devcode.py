"""Fingerprint of built device code: SHA-256 over the gfx950 machine code
of the kernels (by symbol name) in a library built by this package, read
from the library's offload bundles.  Two builds whose kernels assemble to
the same bytes get the same fingerprint whatever their sources' comments or
paths; any change of a matching kernel's code changes it.  Used to tie
recorded profiler counters to the code they were taken on.
"""
from __future__ import annotations

import hashlib
import re
import struct

_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def _code_objects(blob: bytes, arch: str):
    for m in re.finditer(re.escape(_MAGIC), blob):
        o = m.start()
        n = struct.unpack_from("<Q", blob, o + len(_MAGIC))[0]
        p = o + len(_MAGIC) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", blob, p)
            p += 24
            triple = blob[p:p + tlen].decode()
            p += tlen
            if triple.endswith(arch) and size:
                yield blob[o + off:o + off + size]


def _functions(elf: bytes):
    """(name, machine code) of every sized function symbol of an ELF64."""
    shoff = struct.unpack_from("<Q", elf, 0x28)[0]
    shentsize, shnum = struct.unpack_from("<HH", elf, 0x3A)
    sh = [struct.unpack_from("<IIQQQQIIQQ", elf, shoff + i * shentsize) for i in range(shnum)]
    for s in sh:
        if s[1] != 2:                                   # SHT_SYMTAB
            continue
        strtab_off = sh[s[6]][4]
        for k in range(s[5] // 24):
            name_off, info, _, shndx, value, size = struct.unpack_from("<IBBHQQ", elf,
                                                                       s[4] + k * 24)
            if info & 0xF != 2 or size == 0:            # STT_FUNC with a body
                continue
            a = strtab_off + name_off
            name = elf[a:elf.index(b"\0", a)].decode()
            sec = sh[shndx]
            start = sec[4] + value - sec[3]
            yield name, elf[start:start + size]


def kernel_sha256(lib_path: str, name_substring: str, arch: str = "gfx950") -> str:
    """SHA-256 over (name, code) of every function whose symbol name contains
    name_substring, in name order; '' when there is none."""
    blob = open(lib_path, "rb").read()
    found = {}
    for co in _code_objects(blob, arch):
        for name, code in _functions(co):
            if name_substring in name:
                found[name] = code
    if not found:
        return ""
    h = hashlib.sha256()
    for name in sorted(found):
        h.update(name.encode() + b"\0" + found[name])
    return h.hexdigest()
