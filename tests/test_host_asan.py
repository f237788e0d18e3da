"""Host code of the C-ABI library under AddressSanitizer (no GPU needed): api.hip is compiled
with the sanitizer on its host side only (device code is never instrumented), linked with the
other objects of the last build, and every entry point is called on its host-only paths
(argument checks, work-space sizes, status strings, plans that stop at the missing device) in
a child process with the sanitizer's runtime preloaded."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1904_03409_amd")
HIPCC = "/opt/rocm/bin/hipcc"

CALLS = r'''
import ctypes, sys
sys.path.insert(0, sys.argv[2])
from paper_1904_03409_amd import stacklstm as s
s.LIB_PATH = sys.argv[1]
lib = s.load_library()
out = []
if len(sys.argv) > 3:
    ctypes.CDLL(None).__asan_init   # the sanitizer runtime is loaded (AttributeError otherwise)
for dims in [(240, 256, 256, 512, 0), (8, 4, 3, 2000, 0), (8, 4, 3, 1024, 1), (8, 0, 3, 16, 0), (0, 4, 3, 16, 0),
             (1, 1, 1, 1, 0), (1 << 20, 1 << 12, 1 << 12, 512, 0), (-1, 4, 4, 4, 0), (4, 4, 4, 4, 7),
             (1024, 1024, 512, 1024, 1), (3, 17, 48, 200, 0)]:
    out.append(s.stacklstm_workspace_bytes(s.make_dims(*dims)))
for code in list(range(10)) + [-1, 99]:
    out.append(s._status_string(code))
nul = ctypes.c_void_p(0)
plan = s.slstm_plan()
for dims in [(8, 4, 3, 16, 0), (0, 4, 3, 16, 1), (8, 4, 3, 2000, 0)]:
    d = s.make_dims(*dims)
    out.append(lib.stacklstm_fwd(ctypes.byref(d), *([nul] * 14), ctypes.c_size_t(0), nul))
    out.append(lib.stacklstm_fwd_static(ctypes.byref(d), *([nul] * 13), nul))
    out.append(lib.stacklstm_bwd(ctypes.byref(d), *([nul] * 10), ctypes.c_size_t(0), *([nul] * 8), nul))
    out.append(lib.stacklstm_plan(ctypes.byref(d), ctypes.byref(plan)))
out.append(lib.stacklstm_fwd(None, *([nul] * 14), ctypes.c_size_t(0), nul))
out.append(lib.stacklstm_bwd(None, *([nul] * 10), ctypes.c_size_t(0), *([nul] * 8), nul))
out.append(lib.stacklstm_plan(None, ctypes.byref(plan)))
out.append(lib.stacklstm_sync_status(nul, ctypes.c_size_t(0), nul))
print(repr(out))
'''


def _asan_runtime():
    found = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return found[0] if found else None


def _run(lib, env=None, asan=False):
    args = [sys.executable, "-c", CALLS, lib, ROOT] + (["asan"] if asan else [])
    return subprocess.run(args, capture_output=True, text=True, timeout=300, env=env)


def test_host_entry_points_under_address_sanitizer(tmp_path):
    objs = sorted(glob.glob(os.path.join(PKG, "_build", "*.o")))
    rt = _asan_runtime()
    if not os.path.exists(HIPCC) or not rt or not objs:
        pytest.skip("hipcc, the sanitizer runtime or the library's objects (build first) are missing")
    api = os.path.join(str(tmp_path), "api_asan.o")
    lib = os.path.join(str(tmp_path), "libstacklstm_asan.so")
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC", "-Xclang", "-target-feature",
                           "-Xclang", "-packed-fp32-ops", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
                           "-fno-omit-frame-pointer", "-c", os.path.join(PKG, "csrc", "api.hip"), "-o", api],
                          stderr=subprocess.DEVNULL)
    others = [o for o in objs if os.path.basename(o) != "api.o"]
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
                           "-shared-libasan", "-o", lib, api, *others])
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = _run(lib, env, asan=True)
    assert r.returncode == 0 and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    # the same answers as the ordinary build
    plain = _run(os.path.join(PKG, "libstacklstm.so"))
    assert plain.returncode == 0, plain.stderr[-2000:]
    assert r.stdout.strip().splitlines()[-1] == plain.stdout.strip().splitlines()[-1]
