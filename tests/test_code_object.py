"""Resource checks on the gfx950 code object inside libtri.so (no GPU needed).

A kernel with a private (scratch) segment makes the runtime set up scratch for
its queue, and from then on every dispatch on that queue runs slower (the
grouped MoE GEMM of one-token decode by about a fifth); spills or a stack also
mean the kernel's registers did not fit.  So no kernel may have one.  The
metadata is read from the AMDGPU note of each code object in the library's
offload bundles.
"""
import os
import struct

import pytest

from paper_2606_29629_amd import _lib as T

msgpack = pytest.importorskip("msgpack")

BUNDLE_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
NT_AMDGPU_METADATA = 32
SHT_NOTE = 7


def _sections(elf: bytes):
    """(name, type, offset, size) of each section of a little-endian ELF64."""
    assert elf[:4] == b"\x7fELF" and elf[4] == 2 and elf[5] == 1, "ELF64 LE expected"
    shoff = struct.unpack_from("<Q", elf, 0x28)[0]
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", elf, 0x3A)
    hdrs = []
    for i in range(shnum):
        name, typ, _flags, _addr, off, size = struct.unpack_from("<IIQQQQ", elf,
                                                                 shoff + i * shentsize)
        hdrs.append((name, typ, off, size))
    stroff = hdrs[shstrndx][2]
    out = []
    for name, typ, off, size in hdrs:
        end = elf.index(b"\0", stroff + name)
        out.append((elf[stroff + name:end].decode(), typ, off, size))
    return out


def _code_objects(so_path: str):
    """The gfx950 code objects of every offload bundle in .hip_fatbin."""
    data = open(so_path, "rb").read()
    fat = [s for s in _sections(data) if s[0] == ".hip_fatbin"]
    assert fat, "no .hip_fatbin section"
    _, _, off, size = fat[0]
    blob = data[off:off + size]
    objs = []
    pos = blob.find(BUNDLE_MAGIC)
    while pos >= 0:
        n = struct.unpack_from("<Q", blob, pos + len(BUNDLE_MAGIC))[0]
        p = pos + len(BUNDLE_MAGIC) + 8
        for _ in range(n):
            e_off, e_size, t_len = struct.unpack_from("<QQQ", blob, p)
            triple = blob[p + 24:p + 24 + t_len].decode()
            p += 24 + t_len
            if "gfx950" in triple and e_size:
                objs.append(blob[pos + e_off:pos + e_off + e_size])
        pos = blob.find(BUNDLE_MAGIC, pos + 1)
    return objs


def _kernels(code_object: bytes):
    """amdhsa.kernels of the code object's AMDGPU metadata note."""
    for _name, typ, off, size in _sections(code_object):
        if typ != SHT_NOTE:
            continue
        p, end = off, off + size
        while p + 12 <= end:
            namesz, descsz, ntype = struct.unpack_from("<III", code_object, p)
            name = code_object[p + 12:p + 12 + namesz].rstrip(b"\0")
            d0 = p + 12 + ((namesz + 3) & ~3)
            if name == b"AMDGPU" and ntype == NT_AMDGPU_METADATA:
                meta = msgpack.unpackb(code_object[d0:d0 + descsz], raw=False)
                return meta["amdhsa.kernels"]
            p = d0 + ((descsz + 3) & ~3)
    raise AssertionError("no AMDGPU metadata note")


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(T.LIB_PATH):
        pytest.skip("libtri.so not built (run python -m paper_2606_29629_amd.build)")
    objs = _code_objects(T.LIB_PATH)
    assert objs, "no gfx950 code object in libtri.so"
    return [k for co in objs for k in _kernels(co)]


def test_code_objects_hold_the_kernels(kernels):
    names = {k[".name"] for k in kernels}
    for stem in ("gemm_kernel", "gemm_grouped_kernel", "attn_prefill_kernel",
                 "attn_decode_kernel", "prologue_kernel"):
        assert any(stem in n for n in names), stem


def test_no_kernel_uses_scratch_or_spills(kernels):
    bad = [(k[".name"], k[".private_segment_fixed_size"], k.get(".vgpr_spill_count", 0),
            k.get(".sgpr_spill_count", 0), k.get(".uses_dynamic_stack", False))
           for k in kernels
           if k[".private_segment_fixed_size"] or k.get(".vgpr_spill_count", 0)
           or k.get(".sgpr_spill_count", 0) or k.get(".uses_dynamic_stack", False)]
    assert not bad, bad
