"""Host checks of the build script's kernel-resource rule (no GPU, no compiler run)."""
from paper_1904_03409_amd import build


def test_counted_wait_kernels():
    # the wide forward always counts its waits
    assert build.counted_waits("_Z10k_fwd_wideILi8ELi32EEv7RecArgs")
    # backward variants with direct dA staging: whole 1 KB segments, one workgroup per CU, <= 4 tiles
    assert build.counted_waits("_Z5k_bwdILi0ELi2ELi32ELi1ELb0EEv7RecArgs")       # fp32 H 512: 2 KB rows
    assert build.counted_waits("_Z5k_bwdILi1ELi4ELi16ELi1ELb0EEv7RecArgs")       # bf16 H 512: 1 KB rows
    assert not build.counted_waits("_Z5k_bwdILi0ELi2ELi32ELi1ELb1EEv7RecArgs")   # gate-split: no dA staging
    assert not build.counted_waits("_Z5k_bwdILi0ELi8ELi32ELi1ELb0EEv7RecArgs")   # eight tiles: built without it
    assert not build.counted_waits("_Z5k_bwdILi1ELi8ELi32ELi2ELb0EEv7RecArgs")   # two workgroups per CU
    assert not build.counted_waits("_Z5k_bwdILi0ELi1ELi8ELi1ELb0EEv7RecArgs")    # 512-byte rows
    assert not build.counted_waits("_Z5k_fwdILi0ELi1ELi1ELi32ELi1EEv7RecArgs")


def test_resource_report_parse():
    text = "\n".join([
        "a.hip:1:1: remark: Function Name: _Z5k_bwdILi0ELi2ELi32ELi1ELb0EEv7RecArgs [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark: Function Name: _Z5k_bwdILi0ELi8ELi32ELi1ELb0EEv7RecArgs [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark:     ScratchSize [bytes/lane]: 880 [-Rpass-analysis=kernel-resource-usage]",
    ])
    rep = build.resource_report(text)
    assert rep == {"_Z5k_bwdILi0ELi2ELi32ELi1ELb0EEv7RecArgs": 0, "_Z5k_bwdILi0ELi8ELi32ELi1ELb0EEv7RecArgs": 880}


def _asm(nop_taken: str) -> str:
    return "\n".join([
        "_Z5k_xxxv:",
        "\tv_mfma_f32_16x16x4_f32 a[0:3], v1, v2, a[0:3]",
        "\tv_mfma_f32_16x16x4_f32 a[4:7], v3, v4, a[4:7]",
        *nop_taken.splitlines(),
        "\ts_cbranch_vccnz .LBB0_5",
        "; %bb.4:",
        "\ts_memrealtime s[10:11]",
        "\ts_waitcnt lgkmcnt(0)",
        ".LBB0_5:",
        "\ts_nop 1",
        "\tv_accvgpr_read_b32 v0, a7",
        "\tv_accvgpr_read_b32 v2, a3",
        "\tv_add_f32_e32 v13, v2, v0",
        "\ts_endpgm",
    ])


def test_mfma_branch_hazard_scan():
    # the pattern that returned a stale accumulator: 1 (branch) + 2 (s_nop 1) wait states on the taken path
    hz = build.mfma_branch_hazards(_asm(""))
    assert len(hz) == 1 and "after 3 wait states (needs 10)" in hz[0] and hz[0].startswith("_Z5k_xxxv")
    # the explicit drain (12 wait states) before the branch clears it
    assert build.mfma_branch_hazards(_asm("\ts_nop 7\n\ts_nop 3")) == []
    # bf16 16x16x32 needs 8: 1 + 2 + 5 covers it
    bf = _asm("\ts_nop 4").replace("v_mfma_f32_16x16x4_f32 a[4:7], v3, v4", "v_mfma_f32_16x16x32_bf16 a[4:7], v[2:5], v[6:9]")
    assert build.mfma_branch_hazards(bf.replace("v_mfma_f32_16x16x4_f32 a[0:3]", "v_mfma_f32_16x16x32_bf16 a[0:3]")) == []
    # a read of registers the MFMA did not write is no hazard
    assert build.mfma_branch_hazards(_asm("").replace("a7", "a9").replace("a3", "a11")) == []
