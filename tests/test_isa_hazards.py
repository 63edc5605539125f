"""CPU check of the generated gfx950 code: the inline-asm blocks that switch
EXEC (plane word as lane mask) also write SCC, so no carry or compare result
may be live across one.  A 64-bit address split as s_add_u32 / s_addc_u32
around such a block once produced wrong addresses; this scans every kernel of
the fused scan for an SCC reader whose nearest SCC writer lies before such a
block."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
READERS = ("s_cbranch_scc", "s_cselect", "s_addc", "s_subb", "s_cmov")
WRITER = re.compile(r"^s_(add|sub|and|or|xor|andn2|orn2|nand|nor|xnor|cmp|bitcmp|lshl|lshr|ashr|bfe|min|max|abs|"
                    r"not|addk|cmpk|absdiff|bitset)\w*")


def scc_hazards(asm: str):
    out = []
    for f in re.split(r"\n(?=_ZN6fathom[0-9A-Za-z_]+:)", asm):
        lines = [l.strip() for l in f.split("\n")]
        for i, t in enumerate(lines):
            if not t.startswith(READERS):
                continue
            crossed = False
            for j in range(i - 1, max(i - 400, 0), -1):
                u = lines[j]
                if u.startswith(("s_mov_b64 exec", "s_and_b64 exec", "s_andn2_b64 exec")):
                    crossed = True
                    continue
                if WRITER.match(u) or u.endswith(":"):
                    break
            if crossed:
                out.append((f.split(":")[0], t))
    return out


def test_scanner_detects_a_planted_hazard():
    planted = "_ZN6fathom1xE:\n\ts_add_u32 s4, s4, s6\n\ts_mov_b64 s[8:9], exec\n\ts_and_b64 exec, s[8:9], s[10:11]\n" \
              "\tv_or_b32 v1, 4, v1\n\ts_mov_b64 exec, s[8:9]\n\ts_addc_u32 s5, s5, 0\n"
    assert len(scc_hazards(planted)) == 1


@pytest.mark.skipif(not os.path.exists(HIPCC) or shutil.which("bash") is None, reason="hipcc not available")
def test_fused_kernels_keep_no_scc_live_across_exec_blocks(tmp_path):
    out = tmp_path / "fused.s"
    src = os.path.join(ROOT, "paper_2609_17652_amd", "csrc", "fused.hip")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off", "-Xclang",
                    "-target-feature", "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S", "-o", str(out), src],
                   check=True, capture_output=True)
    asm = out.read_text()
    assert "s_andn2_b64 exec" in asm  # the EXEC-masked gather is present
    assert scc_hazards(asm) == []
