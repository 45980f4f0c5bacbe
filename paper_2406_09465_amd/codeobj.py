"""Resource usage of a generated gfx950 code object (this library's own
builds): registers, LDS, and private (scratch) memory per lane, read from the
AMDGPU metadata note of the ELF (a msgpack map, note type 32, owner "AMDGPU").
A kernel that spills registers has a non-zero private segment; the tests use
this to keep the generated kernels spill-free."""

from __future__ import annotations

import struct

NT_AMDGPU_METADATA = 32


def _notes(elf: bytes):
    if elf[:4] != b"\x7fELF" or elf[4] != 2:
        raise ValueError("not a 64-bit ELF")
    shoff, = struct.unpack_from("<Q", elf, 0x28)
    shentsize, shnum = struct.unpack_from("<HH", elf, 0x3A)
    for i in range(shnum):
        base = shoff + i * shentsize
        sh_type, = struct.unpack_from("<I", elf, base + 4)
        if sh_type != 7:  # SHT_NOTE
            continue
        off, size = struct.unpack_from("<QQ", elf, base + 0x18)
        pos, end = off, off + size
        while pos + 12 <= end:
            namesz, descsz, ntype = struct.unpack_from("<III", elf, pos)
            pos += 12
            name = elf[pos:pos + namesz].rstrip(b"\0")
            pos += (namesz + 3) & ~3
            desc = elf[pos:pos + descsz]
            pos += (descsz + 3) & ~3
            yield name, ntype, desc


def kernel_resources(elf: bytes) -> dict:
    """{kernel symbol: {"vgpr", "agpr", "sgpr", "vgpr_spill", "sgpr_spill",
    "lds", "scratch"}} from a code object's metadata."""
    import msgpack
    out = {}
    for name, ntype, desc in _notes(elf):
        if name != b"AMDGPU" or ntype != NT_AMDGPU_METADATA:
            continue
        meta = msgpack.unpackb(desc, raw=False, strict_map_key=False)
        for k in meta.get("amdhsa.kernels", []):
            out[k.get(".name", "?")] = {
                "vgpr": k.get(".vgpr_count"), "agpr": k.get(".agpr_count"), "sgpr": k.get(".sgpr_count"),
                "vgpr_spill": k.get(".vgpr_spill_count", 0), "sgpr_spill": k.get(".sgpr_spill_count", 0),
                "lds": k.get(".group_segment_fixed_size"), "scratch": k.get(".private_segment_fixed_size", 0)}
    return out
