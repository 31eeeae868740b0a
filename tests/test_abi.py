"""C-ABI checks that need no GPU: every function the header declares is exported,
and host-side argument checks return their documented status without any
device work."""
import ctypes
import os
import re

import pytest

from paper_2401_06145_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spconv.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(spconv_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_header_symbols_exported():
    lib = B.lib()
    declared = _declared()
    assert len(declared) >= 15
    missing = [n for n in declared if not hasattr(lib, n)]
    assert missing == []
    assert set(declared) == set(B.EXPORTED)


def test_workspace_bytes_host_only():
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM) > 0
    assert B.spconv_map_workspace_bytes(1000, 0, 2, B.SPCONV_DOWN) > B.spconv_map_workspace_bytes(
        1000, 0, 2, B.SPCONV_SUBM)
    assert B.spconv_map_workspace_bytes(1000, 0, 0, B.SPCONV_SUBM) == 0      # K out of range
    assert B.spconv_map_workspace_bytes(1000, 0, 6, B.SPCONV_SUBM) == 0
    assert B.spconv_map_workspace_bytes(-1, 0, 3, B.SPCONV_SUBM) == 0
    assert B.spconv_map_workspace_bytes(10, 0, 3, 7) == 0                    # bad mode
    bad = B.Options.make(B=100)
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, bad) == 0
    # search workgroup size: 128, 256 or 512 threads, Cq / wg in {1, 2, 4, 8}
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(wg=100)) == 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(wg=512, Cq=256)) == 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(wg=128, Cq=2048)) == 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(wg=512, Cq=1024)) > 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(search=2)) == 0
    # offsets per count-pass workgroup: 0 (size rule) to 64
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(count_group=65)) == 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(count_group=-1)) == 0
    assert B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(count_group=64)) > 0
    # the hash-table search adds its table (2^11 slots of 12 bytes for 1000 inputs)
    hashed = B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM, B.Options.make(search=1))
    assert hashed >= B.spconv_map_workspace_bytes(1000, 0, 3, B.SPCONV_SUBM) + 2048 * 12


@pytest.mark.parametrize("K,stride,mode,status", [
    (0, 1, B.SPCONV_SUBM, B.SPCONV_EUNSUPPORTED),
    (3, 2, B.SPCONV_SUBM, B.SPCONV_EINVAL),
    (3, 0, B.SPCONV_DOWN, B.SPCONV_EINVAL),
    (3, 1, 9, B.SPCONV_EINVAL),
])
def test_build_map_argument_errors(K, stride, mode, status):
    L = B.lib()
    h = ctypes.c_void_p()
    st = L.spconv_build_map(None, 0, None, 0, K, stride, 1, mode, None, None, 0, None, ctypes.byref(h))
    assert st == status
    assert L.spconv_last_error()


def test_build_map_null_out_and_small_workspace():
    L = B.lib()
    assert L.spconv_build_map(None, 0, None, 0, 3, 1, 1, 0, None, None, 0, None, None) == B.SPCONV_EINVAL
    h = ctypes.c_void_p()
    # 10 inputs, no workspace -> ENOSPC before any device work
    st = L.spconv_build_map(ctypes.c_void_p(256), 10, None, 0, 3, 1, 1, 0, None, None, 0, None, ctypes.byref(h))
    assert st == B.SPCONV_ENOSPC


def test_forward_plan_null_map():
    L = B.lib()
    info = B.PlanInfo()
    assert L.spconv_forward_plan(None, 16, 16, 0, None, ctypes.byref(info)) == B.SPCONV_EINVAL
    assert L.spconv_forward_workspace_bytes(None, 16, 16, 0, None) == 0


def test_oracle_and_library_share_no_code():
    """The oracle is a separate library built from separate sources."""
    import oracle
    from oracle import build as ob
    csrc = os.path.join(ROOT, "paper_2401_06145_amd", "csrc")
    for f in os.listdir(csrc):
        txt = open(os.path.join(csrc, f)).read()
        assert "oracle" not in txt.lower()
    otxt = open(ob.SRC).read()
    assert "spconv.h" not in otxt and "common.h" not in otxt
    assert oracle.offsets(3).shape == (27, 3)
