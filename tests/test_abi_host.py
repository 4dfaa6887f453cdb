"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects bad arguments on the host
before any HIP call (every case below fails validation, so nothing is
launched and no pointer is dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2608_02989_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "acceptmoe.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="HIP library not built")

V = ctypes.c_void_p
FAKE = V(0x100000)       # aligned non-null address, never dereferenced (validation fails first)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(acceptmoe_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 9
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.SIGNATURES)


def test_version_and_error_string():
    assert L.lib().acceptmoe_version() == 303
    assert isinstance(L.lib().acceptmoe_last_error(), bytes)


def test_workspace_sizes():
    lib = L.lib()
    assert lib.acceptmoe_select_workspace_size(32, 128, 8) >= 32 * 8 * 12
    assert lib.acceptmoe_select_workspace_size(-1, 128, 8) == 0
    # blocks of up to 256 tokens: activations (+ small lists); larger blocks also
    # hold one fp32 output row per (token, slot)
    a = lib.acceptmoe_moe_forward_workspace_size(32, 2048, 768, 128, 8, L.BF16)
    assert 32 * 8 * 768 * 2 <= a < 32 * 8 * 2048 * 4
    b = lib.acceptmoe_moe_forward_workspace_size(512, 2048, 768, 128, 8, L.BF16)
    assert b >= 512 * 8 * (768 * 2 + 2048 * 4)
    assert lib.acceptmoe_moe_forward_workspace_size(32, 2048, 768, 128, 8, 9) == 0
    assert lib.acceptmoe_packed_weights_bytes(L.BF16, 4, 32, 64) == 4 * 32 * 64 * 2
    assert lib.acceptmoe_packed_weights_bytes(L.F32, 4, 32, 64) == 4 * 32 * 64 * 4


def status_and_msg(rc):
    return rc, L.lib().acceptmoe_last_error().decode()


def test_pack_router_sizes_and_rejects():
    lib = L.lib()
    # three bf16 planes per weight, rows padded to 16 and columns to 32
    assert lib.acceptmoe_packed_router_bytes(128, 2048) == 128 * 2048 * 6
    assert lib.acceptmoe_packed_router_bytes(37, 256) == 48 * 256 * 6
    assert lib.acceptmoe_packed_router_bytes(16, 48) == 16 * 64 * 6
    assert lib.acceptmoe_packed_router_bytes(0, 256) == 0
    assert lib.acceptmoe_packed_router_bytes(16, 250) == 0
    f = lib.acceptmoe_pack_router_weights
    assert f(FAKE, 0, 256, FAKE, None) == L.ERR_UNSUPPORTED
    assert f(FAKE, 16, 250, FAKE, None) == L.ERR_UNSUPPORTED
    assert f(None, 16, 256, FAKE, None) == L.ERR_INVALID_ARG
    assert f(V(0x100004), 16, 256, FAKE, None) == L.ERR_INVALID_ARG       # misaligned
    rc, msg = status_and_msg(f(V(0x100000), 16, 256, V(0x100000 + 256), None))
    assert rc == L.ERR_INVALID_ARG and "overlap" in msg


def test_route_rejects():
    f = L.lib().acceptmoe_route
    assert status_and_msg(f(FAKE, L.BF16, FAKE, -1, 256, 16, FAKE, None))[0] == L.ERR_INVALID_ARG
    assert f(FAKE, L.BF16, FAKE, 8, 256, 0, FAKE, None) == L.ERR_UNSUPPORTED
    assert f(FAKE, L.BF16, FAKE, 65535 * 16 + 1, 256, 16, FAKE, None) == L.ERR_UNSUPPORTED   # token tiles
    assert f(FAKE, L.BF16, FAKE, 8, 256, 513, FAKE, None) == L.ERR_UNSUPPORTED
    assert f(FAKE, L.BF16, FAKE, 8, 250, 16, FAKE, None) == L.ERR_UNSUPPORTED
    assert f(FAKE, 7, FAKE, 8, 256, 16, FAKE, None) == L.ERR_INVALID_ARG
    rc, msg = status_and_msg(f(None, L.F32, FAKE, 8, 256, 16, FAKE, None))
    assert rc == L.ERR_INVALID_ARG and "null" in msg
    assert f(V(0x100004), L.F32, FAKE, 8, 256, 16, FAKE, None) == L.ERR_INVALID_ARG   # misaligned
    # T == 0 is a no-op
    assert f(None, L.F32, None, 0, 256, 16, None, None) == L.OK


def sel(**kw):
    a = dict(logits=FAKE, parent=FAKE, depth=FAKE, prob=FAKE, offs=None, B=1, T=8, E=16, k=2, beta=0.5,
             mode=0, budget=0, cap=-1, res=None, elig=FAKE, idx=FAKE, gate=FAKE, stats=FAKE,
             ws=None, wsb=0)
    a.update(kw)
    offs = a["offs"]
    offs_arr = None if offs is None else (ctypes.c_int32 * len(offs))(*offs)
    return L.lib().acceptmoe_select(a["logits"], a["parent"], a["depth"], a["prob"], offs_arr, a["B"],
                                    a["T"], a["E"], a["k"], a["beta"], a["mode"], a["budget"], a["cap"],
                                    a["res"], a["elig"], a["idx"], a["gate"], a["stats"], a["ws"],
                                    a["wsb"], None)


def test_select_rejects():
    assert sel(k=17) == L.ERR_UNSUPPORTED
    assert sel(k=0) == L.ERR_UNSUPPORTED
    assert sel(E=600, k=2) == L.ERR_UNSUPPORTED
    assert sel(E=64, k=33) == L.ERR_UNSUPPORTED
    assert sel(T=-3) == L.ERR_INVALID_ARG
    assert sel(B=0) == L.ERR_UNSUPPORTED
    assert sel(B=257, offs=list(range(258)), T=257) == L.ERR_UNSUPPORTED
    assert sel(beta=float("nan")) == L.ERR_INVALID_ARG
    assert sel(beta=-1.0) == L.ERR_INVALID_ARG
    assert sel(mode=5) == L.ERR_INVALID_ARG
    assert sel(B=2, offs=None) == L.ERR_INVALID_ARG
    assert sel(B=2, offs=[1, 4, 8]) == L.ERR_INVALID_ARG
    assert sel(B=2, offs=[0, 5, 4]) == L.ERR_INVALID_ARG
    assert sel(B=2, offs=[0, 4, 7]) == L.ERR_INVALID_ARG          # offs[B] != T
    assert sel(B=1, offs=[0, 1100], T=1100) == L.ERR_UNSUPPORTED  # tree too large
    assert sel(elig=None) == L.ERR_INVALID_ARG
    assert sel(depth=None) == L.ERR_INVALID_ARG
    rc, msg = status_and_msg(sel())                               # workspace missing
    assert rc == L.ERR_WORKSPACE and "workspace" in msg
    assert sel(ws=FAKE, wsb=16) == L.ERR_WORKSPACE
    assert sel(ws=V(0x100010), wsb=1 << 20) == L.ERR_WORKSPACE    # misaligned workspace
    assert sel(T=0, B=0) == L.OK


def sel_noalloc(**kw):
    a = dict(logits=FAKE, parent=FAKE, depth=FAKE, prob=FAKE, offs=None, B=1, T=8, E=16, k=2, beta=0.5,
             mode=0, budget=0, cap=-1, res=None, elig=FAKE, idx=FAKE, gate=FAKE, stats=FAKE)
    a.update(kw)
    offs = a["offs"]
    offs_arr = None if offs is None else (ctypes.c_int32 * len(offs))(*offs)
    return L.lib().acceptmoe_select_noalloc(a["logits"], a["parent"], a["depth"], a["prob"], offs_arr, a["B"],
                                            a["T"], a["E"], a["k"], a["beta"], a["mode"], a["budget"], a["cap"],
                                            a["res"], a["elig"], a["idx"], a["gate"], a["stats"], None)


# the allocation-free variant runs the same host checks, and refuses a call whose
# scratch need exceeds its static array, all before any HIP call
def test_select_noalloc_rejects():
    assert sel_noalloc(k=17) == L.ERR_UNSUPPORTED
    assert sel_noalloc(T=-3) == L.ERR_INVALID_ARG
    assert sel_noalloc(B=2, offs=[0, 4, 7]) == L.ERR_INVALID_ARG
    assert sel_noalloc(elig=None) == L.ERR_INVALID_ARG
    assert sel_noalloc(beta=float("inf")) == L.ERR_INVALID_ARG
    assert sel_noalloc(T=0, B=0) == L.OK
    # 256 trees of 1000 nodes at E = 512: far beyond the static scratch
    T, E, k = 256 * 1000, 512, 8
    need = L.lib().acceptmoe_select_workspace_size(T, E, k)
    assert need > L.SELECT_NOALLOC_MAX_WORKSPACE
    rc, msg = status_and_msg(sel_noalloc(T=T, E=E, k=k, B=256, offs=[1000 * b for b in range(257)]))
    assert rc == L.ERR_UNSUPPORTED and "scratch" in msg, msg
    # the largest single block that still fits at E = 128, k = 8 is refused one node later
    lo, hi = 1, 200_000
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if L.lib().acceptmoe_select_workspace_size(mid, 128, 8) <= L.SELECT_NOALLOC_MAX_WORKSPACE:
            lo = mid
        else:
            hi = mid - 1
    assert lo >= 7000
    T2 = lo + 1
    offs = [min(1000 * b, T2) for b in range((T2 + 999) // 1000)] + [T2]
    rc, msg = status_and_msg(sel_noalloc(T=T2, E=128, k=8, B=len(offs) - 1, offs=offs))
    assert rc == L.ERR_UNSUPPORTED and "scratch" in msg, msg


def test_pack_rejects():
    f = L.lib().acceptmoe_pack_expert_weights
    assert f(FAKE, L.BF16, 2, 24, 64, V(0x900000), None) == L.ERR_UNSUPPORTED     # N % 16
    assert f(FAKE, L.BF16, 2, 32, 48, V(0x900000), None) == L.ERR_UNSUPPORTED     # K % 32
    assert f(FAKE, L.F32, 2, 32, 40, V(0x900000), None) == L.ERR_UNSUPPORTED      # K % 16
    assert f(FAKE, 3, 2, 32, 64, V(0x900000), None) == L.ERR_INVALID_ARG
    assert f(None, L.BF16, 2, 32, 64, FAKE, None) == L.ERR_INVALID_ARG
    assert f(FAKE, L.BF16, 2, 32, 64, V(0x100000 + 4096), None) == L.ERR_INVALID_ARG  # overlap
    assert f(FAKE, L.BF16, 0, 32, 64, V(0x900000), None) == L.ERR_INVALID_ARG


def test_pack_gate_up_sizes_and_rejects():
    lib = L.lib()
    sz = lib.acceptmoe_packed_gate_up_bytes
    assert sz(L.BF16, 128, 768, 2048) == 2 * 128 * 768 * 2048 * 2        # I % 32 == 0: the two stacks
    assert sz(L.F32, 3, 80, 64) == 3 * 96 * 64 * 4 * 2                   # I/16 odd: padded to 96 rows
    assert sz(9, 3, 80, 64) == 0 and sz(L.F32, 0, 80, 64) == 0
    f = lib.acceptmoe_pack_gate_up_weights
    D = V(0x900000)
    assert f(FAKE, FAKE, L.BF16, 2, 24, 64, D, None) == L.ERR_UNSUPPORTED         # I % 16
    assert f(FAKE, FAKE, L.BF16, 2, 32, 48, D, None) == L.ERR_UNSUPPORTED         # H % 32
    assert f(FAKE, FAKE, L.F32, 2, 32, 40, D, None) == L.ERR_UNSUPPORTED          # H % 16
    assert f(FAKE, FAKE, 3, 2, 32, 64, D, None) == L.ERR_INVALID_ARG
    assert f(FAKE, None, L.BF16, 2, 32, 64, D, None) == L.ERR_INVALID_ARG
    assert f(FAKE, FAKE, L.BF16, 2, 32, 64, V(0x900008), None) == L.ERR_INVALID_ARG  # misaligned dst
    assert f(FAKE, V(0x900000 + 4096), L.BF16, 2, 32, 64, D, None) == L.ERR_INVALID_ARG  # up overlaps dst
    assert f(FAKE, FAKE, L.BF16, 0, 32, 64, D, None) == L.ERR_INVALID_ARG


def fwd(**kw):
    a = dict(h=FAKE, dt=L.BF16, wgu=FAKE, wd=FAKE, T=8, H=256, I=128, E=16, k=2, idx=FAKE,
             gate=FAKE, out=FAKE, ws=None, wsb=0)
    a.update(kw)
    return L.lib().acceptmoe_moe_forward(a["h"], a["dt"], a["wgu"], a["wd"], a["T"], a["H"], a["I"],
                                         a["E"], a["k"], a["idx"], a["gate"], a["out"], a["ws"], a["wsb"],
                                         None)


def test_forward_rejects():
    assert fwd(dt=5) == L.ERR_INVALID_ARG
    assert fwd(H=240) == L.ERR_UNSUPPORTED                 # bf16 needs H % 32
    assert fwd(I=80) == L.ERR_UNSUPPORTED
    assert fwd(dt=L.F32, H=248) == L.ERR_UNSUPPORTED       # fp32 needs H % 16
    assert fwd(E=0) == L.ERR_UNSUPPORTED
    assert fwd(k=40) == L.ERR_UNSUPPORTED
    assert fwd(T=-1) == L.ERR_INVALID_ARG
    assert fwd(out=None) == L.ERR_INVALID_ARG
    assert fwd(wgu=None) == L.ERR_INVALID_ARG
    assert fwd(h=V(0x100008)) == L.ERR_INVALID_ARG         # misaligned
    assert fwd() == L.ERR_WORKSPACE
    assert fwd(T=0, h=None, out=None) == L.OK
    # the combine grid holds T * ceil(H / 1024) workgroups in one dimension
    rc, msg = status_and_msg(fwd(T=1 << 24, H=512 * 1024, k=1))
    assert rc == L.ERR_UNSUPPORTED and "2^31" in msg, msg


def test_stream_read_rejects():
    f = L.lib().acceptmoe_stream_read
    assert f(FAKE, 1024, FAKE, 0, None) == L.ERR_INVALID_ARG           # grid < 1
    assert f(FAKE, 1024, FAKE, 65536, None) == L.ERR_INVALID_ARG       # grid > 65535
    assert f(FAKE, 1000, FAKE, 4, None) == L.ERR_INVALID_ARG           # bytes % 16
    assert f(None, 1024, FAKE, 4, None) == L.ERR_INVALID_ARG
    assert f(FAKE, 1024, None, 4, None) == L.ERR_INVALID_ARG
    assert f(V(0x100008), 1024, FAKE, 4, None) == L.ERR_INVALID_ARG    # misaligned
    assert f(None, 0, None, 4, None) == L.OK                           # empty: no launch


C_PROGRAM = r"""
#include <stdio.h>
#include "acceptmoe.h"
int main(void) {
  size_t ws = acceptmoe_select_workspace_size(64, 128, 8);
  int32_t rc = acceptmoe_route(NULL, ACCEPTMOE_BF16, NULL, 64, 4096, 128, NULL, NULL);
  printf("%d %zu %d\n", (int)acceptmoe_version(), ws, (int)rc);
  return ws > 0 && rc == ACCEPTMOE_ERR_INVALID_ARG ? 0 : 1;
}
"""


def test_header_is_c_and_links_from_c(tmp_path):
    """The boundary is plain C: a C99 program including the header links
    against the library and calls host-side entry points (no GPU work)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    src = tmp_path / "abi.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "abi"
    libdir = os.path.dirname(L.LIB_PATH)
    libname = os.path.basename(L.LIB_PATH)
    assert libname.startswith("lib") and libname.endswith(".so")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", os.path.join(ROOT, "include"),
           str(src), "-o", str(exe), "-L", libdir, "-l" + libname[3:-3], "-Wl,-rpath," + libdir]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    ver, ws, rc = out.stdout.split()
    assert int(ver) == L.lib().acceptmoe_version() and int(ws) > 0 and int(rc) == L.ERR_INVALID_ARG
