"""The gfx950 assembly of the library's kernels, as hipcc builds them, has no VALU write of a
wide store's data registers directly behind the store.

A 16-byte buffer store reads its data registers after it issues; a VALU instruction right
behind it that writes one of them changed the stored data on the MI355X (the entries came
out as the moved value). The compiler models the hazard only for buffer stores without an
SGPR offset, and the row kernels' stores all have one, so the library's store helper puts two
wait states behind each store. This test compiles every source to assembly (CPU only) and
checks that no 12- or 16-byte store of any kernel is followed at once by such a write.
"""
import concurrent.futures as cf
import os
import re
import subprocess

import pytest

from paper_2605_12070_amd import build as B


def _vregs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _instructions(asm):
    """(function, instruction) pairs of the assembly, without labels, directives, comments."""
    fn = None
    for line in asm.splitlines():
        if re.match(r"^_Z\w+:", line):
            fn = line.split(":")[0]
            continue
        s = line.split(";")[0].strip()
        if not s or s.startswith(".") or s.endswith(":"):
            continue
        yield fn, s


def _store_data(instr):
    """Data registers of a 12- or 16-byte store, or None."""
    m = re.match(r"^(buffer|global|flat)_store_dwordx[34]\s+(.*)$", instr)
    if not m:
        return None
    ops = [o.strip() for o in m.group(2).split(",")]
    if m.group(1) == "buffer":
        return _vregs(ops[0])                     # vdata, vaddr, srsrc, soffset
    return _vregs(ops[1]) if len(ops) > 1 else None   # vaddr, vdata, ...


def hazards(asm):
    ins = list(_instructions(asm))
    found = []
    for i, (fn, s) in enumerate(ins[:-1]):
        data = _store_data(s)
        if not data:
            continue
        fn2, nxt = ins[i + 1]
        if fn2 != fn or not nxt.startswith("v_"):
            continue
        dst = nxt.split()[1].rstrip(",") if len(nxt.split()) > 1 else ""
        if _vregs(dst) & data:
            found.append((fn, s, nxt))
    return found


def test_scanner_finds_the_pattern():
    asm = "\n".join([
        "_Zk:", "\tbuffer_store_dwordx4 v[2:5], v78, s[96:99], s88 offen nt",
        "\tv_mov_b64_e32 v[2:3], s[0:1]",
        "\tbuffer_store_dwordx4 v[6:9], v78, s[96:99], s88 offen nt", "\ts_nop 1",
        "\tv_mov_b32_e32 v6, 0",
        "\tglobal_store_dwordx4 v1, v[10:13], s[4:5]", "\tv_add_u32_e32 v12, 1, v12"])
    got = hazards(asm)
    assert [g[2] for g in got] == ["v_mov_b64_e32 v[2:3], s[0:1]", "v_add_u32_e32 v12, 1, v12"]


def _asm_of(src, outdir):
    out = os.path.join(outdir, src + ".s")
    flags = [f for f in B.FLAGS if f != "-fPIC"]
    subprocess.run([B.hipcc(), *flags, "--cuda-device-only", "-S",
                    os.path.join(B.CSRC, src), "-o", out], check=True, capture_output=True)
    with open(out) as f:
        return src, f.read()


@pytest.mark.timeout(600)
def test_no_store_data_overwritten_behind_a_wide_store(tmp_path):
    with cf.ThreadPoolExecutor(len(B.SOURCES)) as ex:
        results = list(ex.map(lambda s: _asm_of(s, str(tmp_path)), B.SOURCES))
    bad = {src: hazards(asm) for src, asm in results}
    bad = {k: v for k, v in bad.items() if v}
    assert not bad, "\n".join(f"{k}: {v[:3]}" for k, v in bad.items())
