"""Host checks of the build script's kernel-resource rule (no GPU, no compiler run)."""
from paper_1904_03409_amd import build


def test_counted_wait_kernels():
    # the wide forward always counts its waits
    assert build.counted_waits("_Z10k_fwd_wideILi8ELi32EEv7RecArgs")
    # backward variants with direct dA staging: whole 1 KB segments, one workgroup per CU, <= 4 tiles
    assert build.counted_waits("_Z5k_bwdILi0ELi2ELi32ELi1EEv7RecArgs")       # fp32 H 512: 2 KB rows
    assert build.counted_waits("_Z5k_bwdILi1ELi4ELi16ELi1EEv7RecArgs")       # bf16 H 512: 1 KB rows
    assert not build.counted_waits("_Z5k_bwdILi0ELi8ELi32ELi1EEv7RecArgs")   # eight tiles: built without it
    assert not build.counted_waits("_Z5k_bwdILi1ELi8ELi32ELi2EEv7RecArgs")   # two workgroups per CU
    assert not build.counted_waits("_Z5k_bwdILi0ELi1ELi8ELi1EEv7RecArgs")    # 512-byte rows
    assert not build.counted_waits("_Z5k_fwdILi0ELi1ELi1ELi32ELi1EEv7RecArgs")


def test_resource_report_parse():
    text = "\n".join([
        "a.hip:1:1: remark: Function Name: _Z5k_bwdILi0ELi2ELi32ELi1EEv7RecArgs [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark: Function Name: _Z5k_bwdILi0ELi8ELi32ELi1EEv7RecArgs [-Rpass-analysis=kernel-resource-usage]",
        "a.hip:9:1: remark:     ScratchSize [bytes/lane]: 880 [-Rpass-analysis=kernel-resource-usage]",
    ])
    rep = build.resource_report(text)
    assert rep == {"_Z5k_bwdILi0ELi2ELi32ELi1EEv7RecArgs": 0, "_Z5k_bwdILi0ELi8ELi32ELi1EEv7RecArgs": 880}
