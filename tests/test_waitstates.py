"""Wait-state check of the kernels' inline-assembly MFMA and DMA instructions
(no GPU): the compiler does not insert wait states inside inline assembly, so
each statement carries its own s_nop padding, and the generated code is
scanned for VALU writes of their operands and early reads of their results.

  * unit cases on hand-written assembly;
  * the device assembly of every library source has no violation;
  * a copy of the sources with the DMA padding removed, and one with the tail
    padding of the MFMA chains removed, are caught.
"""

import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2410_17243_amd import build as B
from paper_2410_17243_amd import waitstates as W


def _fn(body):
    return "_Zkernel:\n" + body + "\n\ts_endpgm\n"


def test_dma_after_valu_sgpr_write_is_caught():
    asm = _fn("\tv_readlane_b32 s16, v3, 0\n\t;;#ASMSTART\n\ts_nop 2\n\tbuffer_load_dwordx4 v4, s[16:19], 0 offen lds"
              "\n\t;;#ASMEND")
    v, n = W.scan(asm)
    assert n == 1 and len(v) == 1 and "v_readlane" in v[0].other


def test_dma_with_five_wait_states_passes():
    asm = _fn("\tv_readlane_b32 s16, v3, 0\n\ts_mov_b32 m0, s4\n\t;;#ASMSTART\n\ts_nop 4\n"
              "\tbuffer_load_dwordx4 v4, s[16:19], 0 offen lds\n\t;;#ASMEND")
    v, n = W.scan(asm)
    assert n == 1 and v == []


def test_dma_m0_written_right_before_is_caught():
    asm = _fn("\ts_mov_b32 m0, s4\n\t;;#ASMSTART\n\tbuffer_load_dwordx4 v4, s[16:19], 0 offen lds\n\t;;#ASMEND")
    v, _ = W.scan(asm)
    assert any("m0" in x.rule for x in v)


def test_mfma_source_restored_without_wait_is_caught():
    asm = _fn("\tv_accvgpr_read_b32 v20, a5\n\t;;#ASMSTART\n\tv_mfma_f32_32x32x16_bf16 v[0:15], v[20:23], "
              "v[24:27], v[0:15]\n\ts_nop 7\n\ts_nop 7\n\ts_nop 3\n\t;;#ASMEND")
    v, _ = W.scan(asm)
    assert len(v) == 1 and "v_accvgpr_read" in v[0].other


def test_mfma_result_read_early_is_caught():
    asm = _fn("\t;;#ASMSTART\n\ts_nop 1\n\tv_mfma_f32_32x32x16_bf16 v[0:15], v[20:23], v[24:27], v[0:15]\n"
              "\t;;#ASMEND\n\tv_mov_b32_e32 v40, v3")
    v, _ = W.scan(asm)
    assert len(v) == 1 and "result" in v[0].rule


def test_mfma_chain_link_followed_by_next_link_passes():
    link = "\t;;#ASMSTART\n\ts_nop 1\n\tv_mfma_f32_32x32x16_bf16 v[0:15], v[20:23], v[24:27], v[0:15]\n\t;;#ASMEND\n"
    last = ("\t;;#ASMSTART\n\ts_nop 1\n\tv_mfma_f32_32x32x16_bf16 v[0:15], v[28:31], v[24:27], v[0:15]\n"
            "\ts_nop 7\n\ts_nop 7\n\ts_nop 3\n\t;;#ASMEND\n")
    asm = _fn(link + "\tds_read_b128 v[28:31], v50\n" + last + "\tv_mov_b32_e32 v40, v3")
    v, n = W.scan(asm)
    assert n == 2 and v == []


def test_hazard_reached_through_a_branch_is_caught():
    asm = _fn("\tv_readfirstlane_b32 s16, v3\n\ts_branch .LBB0_2\n.LBB0_1:\n\ts_nop 7\n\ts_nop 7\n.LBB0_2:\n"
              "\t;;#ASMSTART\n\ts_nop 2\n\tbuffer_load_dwordx4 v4, s[16:19], 0 offen lds\n\t;;#ASMEND")
    v, _ = W.scan(asm)
    assert len(v) == 1


def _device_asm(csrc, names, work):
    def one(src):
        out = os.path.join(work, src + ".s")
        cmd = [B.hipcc(), *B.HIPCC_FLAGS, "--cuda-device-only", "-S", os.path.join(csrc, src), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return out

    with ThreadPoolExecutor(max_workers=len(names)) as ex:
        return list(ex.map(one, names))


@pytest.fixture(scope="module")
def work():
    d = tempfile.mkdtemp(prefix="infcl_waits_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_library_sources_have_no_violation(work):
    total = 0
    for path in _device_asm(B.CSRC, B.SOURCES, work):
        with open(path) as f:
            v, n = W.scan(f.read())
        assert v == [], [str(x) for x in v[:5]]
        total += n
    assert total > 1000  # every sweep kernel issues its MFMA chains and DMA from inline asm


@pytest.mark.parametrize("header,old,new", [
    ("common.hpp", '"s_nop 4\\n\\tbuffer_load_dwordx4', '"buffer_load_dwordx4'),
    ("sweep.hpp", '\\n\\ts_nop 7\\n\\ts_nop 7\\n\\ts_nop 3"', '"'),
])
def test_removed_padding_is_caught(work, header, old, new):
    mut = os.path.join(work, "mut_" + header.replace(".", "_"))
    shutil.copytree(B.CSRC, mut)
    path = os.path.join(mut, header)
    text = open(path).read()
    assert old in text
    open(path, "w").write(text.replace(old, new))
    (asm,) = _device_asm(mut, ["bwd_wide.hip"], mut)
    with open(asm) as f:
        v, _ = W.scan(f.read())
    assert len(v) > 0
