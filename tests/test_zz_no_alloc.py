"""The allocation-free full-sort forward (lapsum_forward_noalloc) against
lapsum_forward with a caller workspace: the same kernels, so the same p, b
and permutation bit for bit.  Two calls in a row share the library's device
scratch; the second, smaller one must not see the first one's contents."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


def _t(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _same(a, b):
    return np.array_equal(a.detach().cpu().numpy(), b.detach().cpu().numpy())


def test_noalloc_forward_equals_workspace_forward(lib):
    import torch
    cases = [
        (W.random_case(5, 1_000_000, dist="normal", ties=0.01), 1000.0, -0.05),   # the n1e6 shape
        (W.random_case(6, 300_007, dist="laplace_abs", ties=0.02), 37.5, -0.01),  # smaller, ragged
    ]
    for perm in (True, False):
        for r, k, alpha in cases:
            x = _t(r)
            print(f"noalloc n={r.shape[1]} perm={perm}", flush=True)
            got = lib.lapsum_forward_noalloc(x, k, alpha, perm=perm)
            want = lib.lapsum_forward(x, k, alpha, perm=perm)
            torch.cuda.synchronize()
            for g, w in zip(got, want):
                assert _same(g, w), (r.shape, perm)


def test_noalloc_on_chip_rows_and_preallocated_outputs(lib):
    import torch
    r = W.random_case(8, 32768, dist="normal", ties=0.01, batch=5)
    x = _t(r)
    p = torch.empty_like(x)
    b = torch.empty(5, dtype=torch.float64, device="cuda")
    pm = torch.empty(x.shape, dtype=torch.int32, device="cuda")
    out = lib.lapsum_forward_noalloc(x, 256.0, -0.1, perm=True, out=p, b_out=b, perm_out=pm)
    assert out[0] is p and out[1] is b and out[2] is pm
    want = lib.lapsum_forward(x, 256.0, -0.1, perm=True)
    for g, w in zip(out, want):
        assert _same(g, w)


def test_noalloc_rejects_rows_beyond_its_scratch(lib):
    import ctypes
    L = lib.load()
    v = ctypes.c_void_p
    n = 3_943_809           # one more score than fits with the permutation
    assert lib.lapsum_forward_workspace_size(1, n, True) > lib.NOALLOC_SCRATCH_BYTES
    assert lib.lapsum_forward_workspace_size(1, n - 1, True) <= lib.NOALLOC_SCRATCH_BYTES
    # rejected on the host before anything is launched (pointers never read)
    assert L.lapsum_forward_noalloc(v(256), 1, n, 10.0, -1.0, v(256), v(256), v(256), v(0)) == 2
    assert L.lapsum_forward_noalloc(v(0), 1, n, 10.0, -1.0, v(256), v(256), v(256), v(0)) == 1
    assert L.lapsum_forward_noalloc(v(256), 1, 100, 100.0, -1.0, v(256), v(256), v(0), v(0)) == 1
