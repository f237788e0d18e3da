"""The C-ABI library (no GPU needed): it loads, exports every function include/stacklstm.h
declares, and its host-only entry points (work-space size, status strings) answer."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stacklstm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)          # comments
    return sorted(set(re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b(stacklstm_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("stacklstm_workspace_bytes", "stacklstm_fwd", "stacklstm_fwd_static", "stacklstm_bwd",
              "stacklstm_sync_status", "stacklstm_status_string", "stacklstm_plan"):
        assert n in names, (n, names)


def test_library_exports_every_declared_function():
    from paper_1904_03409_amd import stacklstm
    assert os.path.exists(stacklstm.LIB_PATH), "libstacklstm.so is not built (run __graft_entry__.build())"
    lib = ctypes.CDLL(stacklstm.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(stacklstm.EXPORTS) == set(declared_functions())


def test_host_only_entry_points():
    from paper_1904_03409_amd import stacklstm as s
    s.load_library()
    d = s.make_dims(240, 256, 256, 512, s.SLSTM_FP32)
    n = s.stacklstm_workspace_bytes(d)
    # the forward's XW and gate stash alone are 2 * T*B*4H floats
    assert n >= 2 * 240 * 256 * 2048 * 4
    assert s.stacklstm_workspace_bytes(s.make_dims(8, 4, 3, 2000, s.SLSTM_FP32)) == 0    # H > 512 in fp32
    assert s.stacklstm_workspace_bytes(s.make_dims(8, 4, 3, 1024, s.SLSTM_BF16_GEMM)) > 0
    assert s.stacklstm_workspace_bytes(s.make_dims(8, 0, 3, 16, s.SLSTM_FP32)) == 0      # B < 1
    # the post-loop split-K partials are sized by the slices T*B rows allow (here one), not by
    # the 64-slice cap: a small problem at H = 1024 needs tens of MB, not a GB
    assert s.stacklstm_workspace_bytes(s.make_dims(8, 4, 3, 1024, s.SLSTM_BF16_GEMM)) < (64 << 20)
    for code in range(9):
        assert s._status_string(code) not in ("", "?", "unknown status")
    assert s._status_string(99) == "unknown status"
