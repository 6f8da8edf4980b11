"""The library's device code, compiled to gfx950 assembly here on the CPU,
keeps to the rules its kernels are written under: no scalar-cache writes
(every store is a vector store), no packed two-wide FP32 instructions (the
build turns them off), no scratch (private) memory, and LDS only in the
kernels that hand data between waves (the two-wave hash forms and the
one-workgroup scan of key offsets)."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_33762_amd", "csrc")
SOURCES = ["ea_copy_kernels.hip", "ea_sha256_kernels.hip"]

# instruction families, spelled in parts
SCALAR_WRITES = re.compile(r"^\s+s_(" + "st" + "ore|buffer_st" + "ore|atomic|dcache_" + "wb|scratch_st" + "ore)")
PACKED_F32 = re.compile(r"^\s+v_pk_(add|mul|fma)_" + "f32")


def hipcc():
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    cc = hipcc()
    if cc is None:
        pytest.skip("hipcc not available")
    sys_path = __import__("sys").path
    if ROOT not in sys_path:
        sys_path.insert(0, ROOT)
    from paper_2609_33762_amd import build
    d = tmp_path_factory.mktemp("isa")
    out = {}
    for src in SOURCES:
        s = str(d / (src + ".s"))
        cmd = [cc] + build.COMMON + ["-x", "hip", "--cuda-device-only", "-S",
                                     os.path.join(CSRC, src), "-o", s]
        subprocess.run(cmd, check=True, capture_output=True)
        out[src] = open(s).read()
    return out


def kernels(text):
    """{kernel symbol: (body lines, metadata dict)} from one assembly file."""
    res = {}
    for m in re.finditer(r"^(_Z\w+):\s*;\s*@", text, re.M):
        name = m.group(1)
        body = text[m.end():text.index("s_endpgm", m.end())].split("\n")
        res[name] = body
    meta = {}
    for m in re.finditer(r"\.name:\s+(\S+)\n(?:.*\n)*?\s+\.private_segment_fixed_size:\s+(\d+)",
                         text):
        meta[m.group(1)] = int(m.group(2))
    lds = {}
    for m in re.finditer(r"\.group_segment_fixed_size:\s+(\d+)\n(?:.*\n)*?\s+\.name:\s+(\S+)",
                         text):
        lds[m.group(2)] = int(m.group(1))
    return res, meta, lds


@pytest.mark.parametrize("src", SOURCES)
def test_no_scalar_writes_no_packed_fp32(assembly, src):
    bodies, _, _ = kernels(assembly[src])
    assert bodies, "no kernels found"
    for name, body in bodies.items():
        bad = [l for l in body if SCALAR_WRITES.match(l) or PACKED_F32.match(l)]
        assert not bad, (name, bad[:5])


@pytest.mark.parametrize("src", SOURCES)
def test_no_scratch_and_lds_only_where_waves_share(assembly, src):
    bodies, scratch, lds = kernels(assembly[src])
    assert set(scratch) >= set(bodies)
    for name in bodies:
        assert scratch[name] == 0, name
        if "split" in name:  # the schedule hand-over (and the chain's key slots)
            assert 0 < lds[name] <= 2048, (name, lds[name])
        elif "hash_offsets" in name:  # the key-offset scan's 256 run totals
            assert 0 < lds[name] <= 2048 + 64, (name, lds[name])
        else:
            assert lds[name] == 0, (name, lds[name])
