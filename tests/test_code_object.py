"""Properties of the built gfx950 code object that no parity test sees.

The kernels are read from libmemsave.so: the HIP offload bundle in its
.hip_fatbin section holds one ELF code object per target, and every kernel
has a 64-byte AMDHSA kernel descriptor (symbol `<kernel>.kd`).  Two things
are checked on every kernel:

* no per-lane scratch (private segment size 0): a spill or a runtime index
  into a private array puts per-lane data in scratch memory;
* no dispatch-packet pointer: the compiler asks for it when a private array
  is promoted into LDS, and every wave then reads the workgroup size from the
  dispatch packet in host memory (it cost the GEMM epilogue 1-12 us a launch).
"""
import os
import struct

import pytest

import paper_2404_12406_amd._lib as L

MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
KD_PRIVATE_SEGMENT = 4          # uint32: private segment (scratch) bytes per lane
KD_CODE_PROPERTIES = 56         # uint16: enable_sgpr_* flags
SGPR_DISPATCH_PTR = 1 << 1


def _code_objects(path):
    """(target triple, ELF bytes) of every device entry of every offload
    bundle (one bundle per translation unit)."""
    data = open(path, "rb").read()
    out = []
    base = data.find(MAGIC)
    assert base >= 0, "no offload bundle in the library"
    while base >= 0:
        (n,) = struct.unpack_from("<Q", data, base + len(MAGIC))
        pos = base + len(MAGIC) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, pos)
            pos += 24
            triple = data[pos:pos + tlen].decode()
            pos += tlen
            if "amdgcn" in triple:
                out.append((triple, data[base + off:base + off + size]))
        base = data.find(MAGIC, base + 1)
    return out


def _kernel_descriptors(elf):
    """{kernel name: 64-byte descriptor} from an ELF64 code object."""
    assert elf[:4] == b"\x7fELF" and elf[4] == 2, "expected an uncompressed ELF64 code object"
    shoff, = struct.unpack_from("<Q", elf, 0x28)
    shentsize, shnum, _ = struct.unpack_from("<HHH", elf, 0x3A)
    secs = []
    for i in range(shnum):
        name, typ, _, addr, off, size, link, _, _, entsize = struct.unpack_from("<IIQQQQIIQQ", elf, shoff + i * shentsize)
        secs.append((typ, addr, off, size, link, entsize))
    kds = {}
    for typ, _, off, size, link, entsize in secs:
        if typ != 2:                                   # SHT_SYMTAB
            continue
        stroff = secs[link][2]
        for j in range(size // entsize):
            st_name, _, _, shndx, value, _ = struct.unpack_from("<IBBHQQ", elf, off + j * entsize)
            end = elf.index(b"\0", stroff + st_name)
            name = elf[stroff + st_name:end].decode()
            if not name.endswith(".kd") or shndx == 0:
                continue
            _, saddr, soff, _, _, _ = secs[shndx]
            pos = soff + (value - saddr)
            kds[name[:-3]] = elf[pos:pos + 64]
    return kds


@pytest.fixture(scope="module")
def descriptors():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libmemsave.so not built")
    objs = _code_objects(L.LIB_PATH)
    assert [t for t, _ in objs if t.endswith("gfx950")], [t for t, _ in objs]
    kds = {}
    for _, elf in objs:
        kds.update(_kernel_descriptors(elf))
    assert len(kds) > 20, "expected the GEMM, BN, reduction and fallback kernels"
    return kds


def test_every_expected_kernel_family_is_present(descriptors):
    names = " ".join(descriptors)
    for family in ("gemm_kernel", "gemm_pair_kernel", "halo_conv_kernel", "transpose_krsc_kernel",
                   "bn_fwd_flat_kernel", "rowcol_reduce_kernel", "finalize_kernel", "igemm_kernel"):
        assert family in names, family


def test_no_kernel_uses_scratch(descriptors):
    bad = {k: struct.unpack_from("<I", d, KD_PRIVATE_SEGMENT)[0] for k, d in descriptors.items()}
    bad = {k: v for k, v in bad.items() if v}
    assert not bad, f"kernels with per-lane scratch: {bad}"


def test_no_kernel_reads_the_dispatch_packet(descriptors):
    bad = [k for k, d in descriptors.items() if struct.unpack_from("<H", d, KD_CODE_PROPERTIES)[0] & SGPR_DISPATCH_PTR]
    assert not bad, f"kernels that enable the dispatch pointer: {bad}"
