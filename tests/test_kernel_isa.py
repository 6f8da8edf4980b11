"""The library's device code, compiled to gfx950 assembly here on the CPU,
keeps to the rules its kernels are written under: no scalar-cache writes
(every store is a vector store), no packed two-wide FP32 instructions (the
build turns them off), no scratch (private) memory, and LDS only in the
kernels that hand data between waves (the two-wave hash forms and the
one-workgroup scan of key offsets), and every DPP instruction written as
inline asm keeps the wait states the hardware needs before it."""
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
            assert 0 < lds[name] <= 2560, (name, lds[name])
        elif "hash_offsets" in name or "fused_scan" in name:  # the key-offset scans
            assert 0 < lds[name] <= 2048 + 64, (name, lds[name])
        else:
            assert lds[name] == 0, (name, lds[name])


def test_argument_blocks_fit_what_the_runtime_takes(assembly):
    # The HBM gather/scatter of up to 2,048 pages passes its page ids in the
    # kernel arguments; the HIP runtime on MI355X was measured to take
    # argument blocks of 16,000 bytes and more, so every kernel's block
    # stays at or under 16,384 bytes, and only the argument-page kernels go
    # past 4 KiB.
    text = assembly["ea_copy_kernels.hip"]
    sizes = {}
    for m in re.finditer(r"^(\w+):\s*;\s*@", text, re.M):
        k = re.search(r"\.amdhsa_kernarg_size\s+(\d+)", text[m.end():])
        sizes[m.group(1)] = int(k.group(1))
    args = {n: v for n, v in sizes.items() if "copy_hbm_args" in n}
    assert len(args) == 6, sorted(args)  # two directions x three vector widths
    for n, v in sizes.items():
        assert v <= 16384, (n, v)
        assert v <= 4096 or n in args, (n, v)
    assert all(v >= 8192 for v in args.values()), args


# ---------------------------------------------------------------- DPP hazards
# A DPP instruction needs every VGPR it reads to have been written by a
# VALU instruction at least two wait states earlier, and an EXEC write at
# least five earlier (each instruction is one wait state, s_nop N is N + 1).
# The compiler inserts those waits for its own code, not inside inline asm,
# so the asm rounds of the hash chain are checked here.
VGPR = re.compile(r"\bv(\d+)\b|\bv\[(\d+):(\d+)\]")


def _vgprs(text):
    out = set()
    for m in VGPR.finditer(text):
        if m.group(1) is not None:
            out.add(int(m.group(1)))
        else:
            out.update(range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def _instructions(body):
    """(mnemonic, operand text, in_asm) per instruction, labels as ('LABEL', '', in_asm)."""
    res, in_asm = [], False
    for line in body:
        s = line.split(";")[0].strip() if "ASM" not in line else line.strip()
        if "ASMSTART" in s:
            in_asm = True
            continue
        if "ASMEND" in s:
            in_asm = False
            continue
        if not s or s.startswith("."):
            if s.startswith(".LBB"):
                res.append(("LABEL", "", in_asm))
            continue
        op, _, rest = s.partition(" ")
        res.append((op, rest, in_asm))
    return res


def _valu_dst(op, rest):
    if not op.startswith("v_") or op.startswith("v_cmp") or op.startswith("v_readlane") \
            or op.startswith("v_readfirstlane"):
        return set()
    first = rest.split(",")[0]
    return _vgprs(first)


def _writes_exec(op, rest):
    return ("saveexec" in op or op.startswith("v_cmpx")
            or (op.startswith("s_") and rest.split(",")[0].strip() == "exec"))


def _dpp_hazards(instrs):
    bad = []
    for k, (op, rest, in_asm) in enumerate(instrs):
        if not in_asm or ("_dpp" not in op and "quad_perm" not in rest and "row_" not in rest):
            continue
        reads = _vgprs(rest.partition(",")[2])
        waits = 0
        for j in range(k - 1, -1, -1):
            pop, prest, _ = instrs[j]
            if pop == "LABEL":
                bad.append((k, op, rest, "window crosses a label"))
                break
            if waits < 2 and reads & _valu_dst(pop, prest):
                bad.append((k, op, rest, f"reads a VGPR written {waits} wait states before"))
                break
            if waits < 5 and _writes_exec(pop, prest):
                bad.append((k, op, rest, f"EXEC written {waits} wait states before"))
                break
            waits += int(prest.split()[0]) + 1 if pop == "s_nop" else 1
            if waits >= 5:
                break
    return bad


def test_dpp_checker_catches_a_short_window():
    # a planted hazard: the DPP add reads v3 right after a VALU wrote it
    body = [";;#ASMSTART", "v_add_u32 v3, v1, v2",
            "v_add_u32_dpp v4, v3, v3 row_shl:12 row_mask:0xf bank_mask:0xf bound_ctrl:1",
            ";;#ASMEND"]
    assert _dpp_hazards(_instructions(body))
    ok = [";;#ASMSTART", "v_add_u32 v3, v1, v2", "v_add_u32 v5, v1, v2", "v_add_u32 v6, v1, v2",
          "v_add_u32_dpp v4, v3, v3 row_shl:12 row_mask:0xf bank_mask:0xf bound_ctrl:1",
          ";;#ASMEND"]
    assert not _dpp_hazards(_instructions(ok))


def test_asm_dpp_reads_keep_their_wait_states(assembly):
    bodies, _, _ = kernels(assembly["ea_sha256_kernels.hip"])
    checked = 0
    for name, body in bodies.items():
        instrs = _instructions(body)
        checked += sum(1 for op, rest, in_asm in instrs if in_asm and "_dpp" in op)
        bad = _dpp_hazards(instrs)
        assert not bad, (name, bad[:3])
    assert checked > 0, "no DPP instruction inside asm found"
