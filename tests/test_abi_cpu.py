"""The C-ABI library on the CPU: it loads, exports every entry point the
header declares, and its host-only paths (status strings, workspace sizes,
argument validation, which return before any HIP call) behave as documented.
No compute call is made here."""
import ctypes
import os
import re

import pytest

import paper_2608_06912_amd as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lapsum.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="library not built")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lapsum_[a-z_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = _declared()
    for want in ("lapsum_forward", "lapsum_backward", "lapsum_forward_bracketed",
                 "lapsum_forward_workspace_size", "lapsum_backward_workspace_size",
                 "lapsum_forward_bracketed_workspace_size", "lapsum_status_string",
                 "lapsum_band_size", "lapsum_backward_band", "lapsum_backward_band_workspace_size"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(L.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name


def test_status_strings():
    assert L.lapsum_status_string(0) == "ok"
    assert "invalid" in L.lapsum_status_string(1)
    assert "workspace" in L.lapsum_status_string(2)
    assert "HIP" in L.lapsum_status_string(3)
    assert "gfx950" in L.lapsum_status_string(4)
    assert "unknown" in L.lapsum_status_string(99)


def test_workspace_sizes():
    # rows that fit on chip need no workspace
    assert L.lapsum_forward_workspace_size(256, 32768) == 0
    assert L.lapsum_forward_workspace_size(1, 16384) == 0
    # one row longer than 16384 goes through the device-wide sort
    assert L.lapsum_forward_workspace_size(1, 32768) > 0
    assert L.lapsum_forward_workspace_size(2, 32768) == 0
    assert L.lapsum_backward_workspace_size(256, 32768) == 0
    a = L.lapsum_forward_workspace_size(1, 10**6, False)
    b = L.lapsum_forward_workspace_size(1, 10**6, True)
    assert a >= 2 * 4 * 10**6 and b >= a + 2 * 4 * 10**6
    assert a % 256 == 0 and b % 256 == 0
    assert L.lapsum_backward_workspace_size(1, 10**7) > 0
    w1 = L.lapsum_forward_bracketed_workspace_size(1, 10**7, 46416, 1 << 16, False)
    w2 = L.lapsum_forward_bracketed_workspace_size(1, 10**7, 46416, 1 << 20, False)
    w3 = L.lapsum_forward_bracketed_workspace_size(1, 10**7, 46416, 1 << 20, True)
    assert 0 < w1 < w2 < w3
    # capacity beyond n is clamped
    assert (L.lapsum_forward_bracketed_workspace_size(1, 1000, 100, 10**6, False)
            == L.lapsum_forward_bracketed_workspace_size(1, 1000, 100, 1000, False))


def _fwd(lib, scores=1, batch=1, n=8, k=2.0, alpha=-1.0, p=1, b=1):
    v = ctypes.c_void_p
    return lib.lapsum_forward(v(scores), batch, n, k, alpha, v(p), v(b), v(0), v(0), 0, v(0))


@pytest.mark.parametrize("kw", [
    dict(scores=0), dict(p=0), dict(b=0), dict(batch=0), dict(n=0), dict(n=2**31),
    dict(k=0.0), dict(k=8.0), dict(k=-1.0), dict(k=float("nan")), dict(k=float("inf")),
    dict(alpha=0.0), dict(alpha=1.0), dict(alpha=float("-inf")), dict(alpha=float("nan")),
])
def test_forward_rejects_invalid_arguments(kw):
    assert _fwd(L.load(), **kw) == 1


def test_forward_rejects_missing_workspace():
    lib = L.load()
    v = ctypes.c_void_p
    # a long row needs a workspace: null, too small, misaligned
    assert lib.lapsum_forward(v(1), 1, 10**6, 5.0, -1.0, v(1), v(1), v(0), v(0), 0, v(0)) == 2
    need = L.lapsum_forward_workspace_size(1, 10**6)
    assert lib.lapsum_forward(v(1), 1, 10**6, 5.0, -1.0, v(1), v(1), v(0), v(256), need - 1, v(0)) == 2
    assert lib.lapsum_forward(v(1), 1, 10**6, 5.0, -1.0, v(1), v(1), v(0), v(128), need, v(0)) == 2


def test_backward_rejects_invalid_arguments():
    lib = L.load()
    v = ctypes.c_void_p
    z = (v(0), v(0))   # no budget / temperature gradients
    assert lib.lapsum_backward(v(0), v(1), v(0), 1, 8, -1.0, v(1), *z, v(0), 0, v(0)) == 1
    assert lib.lapsum_backward(v(1), v(1), v(0), 1, 8, 0.5, v(1), *z, v(0), 0, v(0)) == 1
    assert lib.lapsum_backward(v(1), v(1), v(0), 0, 8, -1.0, v(1), *z, v(0), 0, v(0)) == 1
    assert lib.lapsum_backward(v(1), v(1), v(0), 1, 10**6, -1.0, v(1), *z, v(0), 0, v(0)) == 2
    assert lib.lapsum_backward(v(1), v(1), v(0), 1, 10**6, -1.0, v(1), v(8), v(8), v(0), 0,
                               v(0)) == 2


@pytest.mark.parametrize("kw", [
    dict(K=1), dict(K=1001), dict(z=0.0), dict(z=float("nan")),
    dict(m_capacity=0), dict(flags=2), dict(k=1000.0),
])
def test_bracketed_rejects_invalid_arguments(kw):
    lib = L.load()
    v = ctypes.c_void_p
    a = dict(noise=1, K=100, z=5.16, m_capacity=64, flags=0, k=10.0)
    a.update(kw)
    st = lib.lapsum_forward_bracketed(v(1), 1, 1000, a["k"], -1.0, a["K"], a["z"], v(a["noise"]),
                                      7, v(0), a["m_capacity"], a["flags"], v(1), v(1), v(0), v(0),
                                      v(0), 0, v(0), 0, v(0))
    assert st == 1


def test_bracket_noise_rejects_invalid_arguments():
    lib = L.load()
    v = ctypes.c_void_p
    assert lib.lapsum_bracket_noise(3, 100, -1.0, v(0), v(0)) == 1      # no output
    assert lib.lapsum_bracket_noise(3, 0, -1.0, v(1), v(0)) == 1        # K < 1
    assert lib.lapsum_bracket_noise(3, 100, 0.0, v(1), v(0)) == 1       # alpha not < 0
    assert lib.lapsum_bracket_noise(3, 100, float("inf"), v(1), v(0)) == 1


def test_bracketed_rejects_a_short_or_misaligned_band():
    lib = L.load()
    v = ctypes.c_void_p
    need = L.lapsum_band_size(1, 1000)
    for ptr, size in ((256, need - 1), (128, need)):
        st = lib.lapsum_forward_bracketed(v(1), 1, 1000, 10.0, -1.0, 100, 5.16, v(1), 0, v(0), 64, 0,
                                          v(1),
                                          v(1), v(0), v(0), v(ptr), size, v(0), 0, v(0))
        assert st == 1


def test_band_sizes():
    # header + block records + four lists of at most 512 entries per block
    one = L.lapsum_band_size(1, 10**8)
    assert 8 * 10**8 * 0.08 < one < 8 * 10**8 * 0.09
    assert L.lapsum_band_size(3, 10**6) == 3 * L.lapsum_band_size(1, 10**6)
    assert L.lapsum_band_size(1, 1000) % 256 == 0
    assert L.lapsum_band_size(0, 1000) == 0
    # lists never hold more entries than the row has scores (small rows)
    assert L.lapsum_band_size(1, 4096) < 8 * 4096 + 4096
    assert L.lapsum_backward_band_workspace_size(1, 10**8) > 0


def test_backward_band_rejects_invalid_arguments():
    lib = L.load()
    v = ctypes.c_void_p
    need = L.lapsum_band_size(1, 1000)
    ws = L.lapsum_backward_band_workspace_size(1, 1000)
    args = lambda band, bb, alpha=-1.0, wsp=256, wsb=ws: lib.lapsum_backward_band(
        v(1), v(1), v(band), bb, 1, 1000, alpha, v(1), v(0), v(0), v(wsp), wsb, v(0))
    assert args(0, need) == 1            # no band
    assert args(256, need - 1) == 1      # band too small
    assert args(128, need) == 1          # misaligned
    assert args(256, need, alpha=1.0) == 1
    assert args(256, need, wsp=0) == 2   # workspace missing
    assert args(256, need, wsb=ws - 1) == 2


def test_topk_mask_rejects_invalid_arguments():
    lib = L.load()
    v = ctypes.c_void_p
    assert lib.lapsum_topk_mask(v(0), 1, 8, 2, v(1), v(0)) == 1     # no perm
    assert lib.lapsum_topk_mask(v(1), 1, 8, 2, v(0), v(0)) == 1     # no mask
    assert lib.lapsum_topk_mask(v(1), 0, 8, 2, v(1), v(0)) == 1     # batch < 1
    assert lib.lapsum_topk_mask(v(1), 1, 8, 9, v(1), v(0)) == 1     # k > n
    assert lib.lapsum_topk_mask(v(1), 1, 8, -1, v(1), v(0)) == 1    # k < 0


def test_comparators_reject_invalid_arguments():
    lib = L.load()
    v = ctypes.c_void_p
    assert lib.lapsum_bisect_forward(v(0), 1, 8, 2.0, -1.0, 60, v(1), v(1), v(0)) == 1
    assert lib.lapsum_bisect_forward(v(1), 1, 8, 8.0, -1.0, 60, v(1), v(1), v(0)) == 1   # k = n
    assert lib.lapsum_bisect_forward(v(1), 1, 8, 2.0, -1.0, 201, v(1), v(1), v(0)) == 1
    ws = L.lapsum_dftopk_workspace_size(1, 1000)
    assert ws > 0 and L.lapsum_dftopk_workspace_size(1, 1) == 0
    f = lambda k, alpha=-1.0, n=1000, wsp=256, wsb=ws: lib.lapsum_dftopk_forward(
        v(1), 1, n, k, alpha, v(1), v(1), v(1), v(wsp), wsb, v(0))
    assert f(0) == 1 and f(1000) == 1 and f(10, alpha=0.5) == 1 and f(1, n=1) == 1
    assert f(10, wsp=0) == 2 and f(10, wsb=ws - 1) == 2
    assert lib.lapsum_dftopk_backward(v(1), v(1), v(0), 1, 1000, -1.0, v(1), v(256), ws,
                                      v(0)) == 1


def test_bracketed_workspace_has_a_slice_per_row_in_flight():
    one = L.lapsum_forward_bracketed_workspace_size(1, 100000, 2000, 5000)
    assert one > 0
    assert L.lapsum_forward_bracketed_workspace_size(3, 100000, 2000, 5000) == 3 * one
    assert L.lapsum_forward_bracketed_workspace_size(9, 100000, 2000, 5000) == 4 * one
    # with the M indices the rows go one after another through one slice
    assert L.lapsum_forward_bracketed_workspace_size(9, 100000, 2000, 5000, True) == \
        L.lapsum_forward_bracketed_workspace_size(1, 100000, 2000, 5000, True)
