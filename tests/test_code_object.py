"""Resource use of the built gfx950 kernels, read from the library's code
object without a GPU: every render kernel fits one workgroup's LDS, and the
top-N render kernels read neither the dispatch packet nor scratch memory.

A kernel that indexes a small per-lane array at a computed index gets that
array moved into a per-thread LDS block, whose address is built from the
workgroup size that each wave then loads from the dispatch packet in host
memory (measured: about 8,800 cycles per workgroup between the depth network
and the first sample).  The kernel descriptor's flag for the dispatch pointer
catches that, and its private segment size any register spill to scratch."""
import re
import struct

import pytest

from paper_2103_03231_amd import binding as b

LDS_PER_CU = 160 * 1024


def _sections(elf):
    shoff = struct.unpack_from("<Q", elf, 0x28)[0]
    shentsize, shnum, shstrndx = struct.unpack_from("<HHH", elf, 0x3A)
    raw = [struct.unpack_from("<IIQQQQIIQQ", elf, shoff + i * shentsize) for i in range(shnum)]
    names_off = raw[shstrndx][4]

    def name(s):
        o = names_off + s[0]
        return elf[o:elf.index(b"\0", o)].decode()

    return {name(s): s for s in raw}, raw


def _gfx950_code_objects(path):
    """The gfx950 code object of every offload bundle in the library's
    `.hip_fatbin` section (one bundle per translation unit)."""
    data = open(path, "rb").read()
    secs, _ = _sections(data)
    fat = secs[".hip_fatbin"]
    lo, hi = fat[4], fat[4] + fat[5]
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    out = []
    base = data.find(magic, lo, hi)
    while base >= 0:
        n = struct.unpack_from("<Q", data, base + len(magic))[0]
        p = base + len(magic) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, p)
            triple = data[p + 24:p + 24 + tlen].decode()
            p += 24 + tlen
            if triple.endswith("gfx950"):
                out.append(data[base + off:base + off + size])
        base = data.find(magic, p, hi)
    if not out and data.find(b"CCOB", lo, hi) >= 0:
        pytest.skip("the offload bundles are compressed; their descriptors are not read here")
    assert out, "no gfx950 code object in the library"
    return out


def _descriptors(co):
    """{kernel name: (LDS bytes, scratch bytes, dispatch pointer flag)} from
    the 64-byte AMDHSA kernel descriptors (symbols `<kernel>.kd`)."""
    secs, raw = _sections(co)
    symtab, strtab = secs[".symtab"], secs[".strtab"]
    out = {}
    for i in range(symtab[5] // 24):
        st_name, st_info, st_other, st_shndx, st_value, st_size = struct.unpack_from(
            "<IBBHQQ", co, symtab[4] + 24 * i)
        o = strtab[4] + st_name
        name = co[o:co.index(b"\0", o)].decode()
        if not name.endswith(".kd"):
            continue
        sec = raw[st_shndx]
        kd = co[sec[4] + (st_value - sec[3]):][:64]
        lds, scratch = struct.unpack_from("<II", kd, 0)
        props = struct.unpack_from("<H", kd, 56)[0]
        out[name[:-3]] = (lds, scratch, bool(props & 2))
    return out


@pytest.fixture(scope="module")
def kernels():
    b.lib()  # fails loudly when the library is not built
    out = {}
    for co in _gfx950_code_objects(b.LIB_PATH):
        out.update(_descriptors(co))
    return out


# render_kernel<PR, CB, NW, OCC, NCAP, PLACE, DIN>, mangled
RENDER = re.compile(r"render_kernelILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)EEEv")


def _render(kernels):
    out = []
    for name, d in kernels.items():
        m = RENDER.search(name)
        if m:
            out.append((tuple(int(x) for x in m.groups()), d))
    return out


def test_every_precision_and_placement_is_built(kernels):
    got = {(pr, place) for (pr, _, _, _, _, place, _), _ in _render(kernels)}
    assert got == {(pr, place) for pr in (0, 1, 2) for place in (0, 1, 2)}


def test_render_kernels_fit_the_lds(kernels):
    for params, (lds, _, _) in _render(kernels):
        assert 0 < lds <= LDS_PER_CU, (params, lds)


def test_topn_kernels_read_no_dispatch_packet_and_no_scratch(kernels):
    topn = [(p, d) for p, d in _render(kernels) if p[5] == 0]
    assert len(topn) == 3 * 3 * 2   # precisions x sample capacities x depth inputs
    for params, (lds, scratch, dispatch) in topn:
        assert not dispatch, ("reads the dispatch packet", params)
        assert scratch == 0, ("spills to scratch", params, scratch)
