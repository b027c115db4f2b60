"""Every vector store wider than 8 bytes in the gfx950 code keeps the two
wait states that the hardware needs before a VALU instruction may overwrite
the store's data registers (CPU only: the kernels are compiled to assembly
here and the assembly is scanned).

The cache moves store through inline assembly (cache policy "nt sc1"), which
the compiler's hazard recognizer does not see; the statement therefore
carries its own wait states.  This test reads the code the compiler actually
produced for every kernel source, so a retuned kernel or another compiler
cannot place a register write too close to such a store unnoticed.  Every
path out of a store is followed (fall-through and branch targets) until two
wait states have passed.
"""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import pytest

from paper_2510_22876_amd import build

NEED = 2   # wait states between a store of more than 8 bytes and a VALU write of its data
STORE = re.compile(r"(global|flat|buffer)_store_dwordx(3|4)\s+(\S+?),\s*(\S+?)(,|\s|$)")


def _regs(tok: str) -> set:
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"v(\d+)", tok)
    return {int(m.group(1))} if m else set()


def _instructions(text: str):
    """(instructions, label -> index) of one assembly file; comments and
    directives dropped."""
    ins, labels = [], {}
    for line in text.splitlines():
        s = line.split(";", 1)[0].strip()
        if not s:
            continue
        if s.endswith(":"):
            labels[s[:-1]] = len(ins)
            continue
        if s.startswith("."):
            continue
        ins.append(s)
    return ins, labels


def _hazards(ins, labels):
    found, stores = [], 0
    for i, s in enumerate(ins):
        m = STORE.match(s)
        if not m:
            continue
        stores += 1
        data = _regs(m.group(3) if m.group(1) == "buffer" else m.group(4))
        assert data, s
        todo, seen = [(i + 1, 0)], set()
        while todo:
            j, ws = todo.pop()
            while ws < NEED and j < len(ins) and (j, ws) not in seen:
                seen.add((j, ws))
                t = ins[j]
                op = t.split()[0]
                mn = re.match(r"s_nop\s+(\d+)", t)
                if mn:
                    ws += int(mn.group(1)) + 1
                    j += 1
                    continue
                if op.startswith("v_") and len(t.split()) > 1 and _regs(t.split()[1].rstrip(",")) & data:
                    found.append((s, t, ws))
                    break
                if op == "s_endpgm":
                    break
                if op.startswith("s_branch") or op.startswith("s_cbranch") or op.startswith("s_setpc"):
                    tgt = t.split()[1] if len(t.split()) > 1 else ""
                    if tgt in labels:
                        todo.append((labels[tgt], ws + 1))
                    if op.startswith("s_branch") or op.startswith("s_setpc"):
                        break
                ws += 1
                j += 1
    return stores, found


def _assembly(src: Path, out: Path) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    cmd = [hipcc, *build.COMMON, "--cuda-device-only", "-S", str(src), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text()


SOURCES = sorted(build.CSRC.glob("*.hip"))


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    d = tmp_path_factory.mktemp("asm")
    with ThreadPoolExecutor(max_workers=4) as ex:
        texts = list(ex.map(lambda s: _assembly(s, d / (s.stem + ".s")), SOURCES))
    return dict(zip([s.name for s in SOURCES], texts))


def test_scanner_finds_a_planted_hazard():
    """The scan itself: a VALU write one wait state after a 16-byte store is
    reported, also behind a branch; two wait states are not."""
    bad = "global_store_dwordx4 v[10:11], v[2:5], off nt sc1\ns_nop 0\nv_mov_b64_e32 v[2:3], s[22:23]\ns_endpgm\n"
    assert len(_hazards(*_instructions(bad))[1]) == 1
    branch = ("buffer_store_dwordx4 v[6:9], v10, s[16:19], 0 offen nt sc1\ns_cbranch_vccnz .LBB0_2\n"
              "s_endpgm\n.LBB0_2:\nv_mov_b32_e32 v8, 0\ns_endpgm\n")
    assert len(_hazards(*_instructions(branch))[1]) == 1
    ok = "global_store_dwordx4 v[10:11], v[2:5], off nt sc1\ns_nop 1\nv_mov_b64_e32 v[2:3], s[22:23]\ns_endpgm\n"
    assert _hazards(*_instructions(ok))[1] == []
    other = ("global_store_dwordx4 v[10:11], v[2:5], off nt sc1\nv_mov_b32_e32 v6, 0\nv_mov_b32_e32 v7, 0\n"
             "v_add_u32_e32 v2, 1, v2\n")
    assert _hazards(*_instructions(other))[1] == []


@pytest.mark.parametrize("name", [s.name for s in SOURCES])
def test_no_store_data_hazard(assembly, name):
    stores, found = _hazards(*_instructions(assembly[name]))
    assert not found, f"{name}: VALU writes of store data within {NEED} wait states: {found[:5]}"


def test_cache_moves_use_the_policy_store(assembly):
    """The realignment, gather and compaction kernels store with "nt sc1"."""
    for name in ("specdec_kernels.hip", "exspec_kernels.hip", "rollback_kernels.hip"):
        assert re.search(r"global_store_dwordx4 [^\n]*nt sc1", assembly[name]), name
