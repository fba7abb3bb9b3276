"""Static checks of the built stage kernel's gfx950 assembly (CPU only).

``v_readlane_b32`` reads one lane's VGPR into an SGPR whether or not that
lane is enabled.  Inside a region where the exec mask is narrowed
(``s_and_saveexec_b64`` ... ``s_or_b64 exec``) the lane it reads may be
disabled and hold a value the current code path never wrote: a pointer built
that way once faulted the GPU (the conv epilogue on 55x55 maps).  Values that
must be uniform inside such regions are read with ``v_readfirstlane_b32``
instead (which picks an enabled lane).  This test disassembles the code
object that the build embedded in ``libios.so`` (this repository's own
build) and fails if any ``v_readlane_b32`` sits inside an exec-narrowed
region, apart from reloads of registers the compiler spilled to VGPR lanes
itself (``v_writelane_b32`` targets), which it writes with the same mask.
"""
import os
import re
import struct
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2011_01302_amd", "libios.so")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
BUNDLE_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def gfx950_code_objects(path):
    """The gfx950 entries of every clang offload bundle inside a host binary
    (one bundle per HIP translation unit)."""
    data = open(path, "rb").read()
    out, start = [], 0
    while True:
        base = data.find(BUNDLE_MAGIC, start)
        if base < 0:
            break
        n = struct.unpack_from("<Q", data, base + len(BUNDLE_MAGIC))[0]
        p = base + len(BUNDLE_MAGIC) + 8
        for _ in range(n):
            off, size, idlen = struct.unpack_from("<QQQ", data, p)
            p += 24
            ident = data[p:p + idlen].decode()
            p += idlen
            if ident.endswith("gfx950"):
                out.append(data[base + off: base + off + size])
        start = base + 1
    assert out, "no gfx950 code object in the library"
    return out


def masked_readlanes(lines):
    """(function, line) of every v_readlane_b32 inside an exec-narrowed
    region whose source VGPR is not a compiler spill register."""
    spill = set(re.findall(r"v_writelane_b32 (v\d+),", "\n".join(lines)))
    bad, depth, fn = [], 0, None
    for ln in lines:
        m = re.match(r"^[0-9a-f]+ <(\S+)>:", ln)
        if m:
            fn, depth = m.group(1), 0
            continue
        t = ln.strip()
        if t.startswith("s_and_saveexec_b64"):
            depth += 1
        elif t.startswith("s_or_b64 exec, exec,") and depth > 0:
            depth -= 1
        elif t.startswith("v_readlane_b32"):
            src = t.split()[2].rstrip(",")
            if depth > 0 and src not in spill:
                bad.append((fn, t))
    return bad


@pytest.fixture(scope="module")
def disassembly(tmp_path_factory):
    if not os.path.exists(LIB):
        pytest.skip("libios.so is not built")
    d = tmp_path_factory.mktemp("asm")
    lines = []
    for k, co in enumerate(gfx950_code_objects(LIB)):
        f = d / f"tu{k}.co"
        f.write_bytes(co)
        lines += subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", str(f)], check=True, capture_output=True,
                                text=True).stdout.splitlines()
    return lines


def test_stage_kernels_present(disassembly):
    names = {re.match(r"^[0-9a-f]+ <(\S+)>:", l).group(1) for l in disassembly
             if re.match(r"^[0-9a-f]+ <(\S+)>:", l)}
    # every kernel variant (light / sep / seprow / pipe / full) x launch kind (tile / persistent)
    assert len({n for n in names if "ios_stage_kernel" in n}) == 10


def test_no_readlane_of_possibly_disabled_lanes(disassembly):
    bad = masked_readlanes(disassembly)
    assert not bad, f"{len(bad)} v_readlane_b32 inside exec-narrowed regions, e.g. {bad[:5]}"


def test_the_scan_finds_a_planted_case():
    """The scanner itself: a readlane inside a narrowed region is found, one
    outside is not, and a spill reload is allowed."""
    lines = ["0000000000001000 <_Zkern>:",
             "  v_readlane_b32 s4, v1, 3",
             "  s_and_saveexec_b64 s[6:7], vcc",
             "  v_writelane_b32 v9, s2, 0",
             "  v_readlane_b32 s5, v9, 0",
             "  v_readlane_b32 s8, v2, 7",
             "  s_or_b64 exec, exec, s[6:7]",
             "  v_readlane_b32 s9, v3, 1"]
    assert masked_readlanes(lines) == [("_Zkern", "v_readlane_b32 s8, v2, 7")]

