"""The kernels' inline-assembly loads keep their registers untouched until
waited for (paper_2609_04523_amd.asm_check), checked on the gfx950 assembly
that hipcc produces here (no GPU needed)."""
import os

import pytest

from paper_2609_04523_amd import asm_check, build

FN = "_ZN2mk4testEv:                         ; @x\n{}\n.Lfunc_end0:\n"


def test_checker_flags_registers_touched_in_flight():
    bad = FN.format("\n".join([
        "\tds_read_b128 v[4:7], v1",
        "\tds_read_b128 v[8:11], v2",
        "\ts_waitcnt lgkmcnt(1)",        # v[4:7] landed, v[8:11] may not have
        "\tv_mov_b32_e32 v20, v5",
        "\tv_accvgpr_write_b32 a3, v9",  # reads an in-flight register
    ]))
    hz = asm_check.hazards(bad)
    assert [h[2] for h in hz] == ["v_accvgpr_write_b32 a3, v9"]

    vm = FN.format("\n".join([
        "\tglobal_load_dwordx4 v[2:5], v[76:77], off",
        "\tbuffer_load_dwordx4 v72, s[0:3], 0 offen lds",  # LDS-DMA: v72 is an address
        "\tv_mul_hi_u32_u24_e32 v5, 0x38e38f, v76",         # clobbers a load target
        "\ts_waitcnt vmcnt(0)",
        "\tv_mov_b32_e32 v3, 0",
    ]))
    hz = asm_check.hazards(vm)
    assert [h[2] for h in hz] == ["v_mul_hi_u32_u24_e32 v5, 0x38e38f, v76"]


def test_checker_accepts_waited_reads():
    good = FN.format("\n".join([
        "\tds_read_b128 v[4:7], v1",
        "\tds_read_b128 v[8:11], v2",
        "\ts_waitcnt lgkmcnt(1)",
        "\tv_mov_b32_e32 v20, v5",
        "\ts_waitcnt lgkmcnt(0)",
        "\tv_mov_b32_e32 v21, v9",
        "\tbuffer_load_dwordx4 v72, s[0:3], 0 offen lds",
        "\tv_add_u32_e32 v72, 4, v72",
    ]))
    assert asm_check.hazards(good) == []


@pytest.mark.skipif(not os.path.exists(build.HIPCC), reason="hipcc not available")
def test_kernels_have_no_in_flight_register_hazards():
    res = asm_check.check_all()
    assert set(res) == {u.split("/")[-1] for u in asm_check.LAUNCH_UNITS}
    bad = {u: hz[:3] for u, hz in res.items() if hz}
    assert not bad, bad
