"""Host-side logic of the autograd layer (CPU only): the straight-through
identity, the sample-size rules, the path switch, the cached bracket noise,
and that nothing falls back to the CPU."""
import numpy as np
import pytest
import torch

import paper_2608_06912_amd.autograd as A


def test_straight_through_forward_is_the_mask_and_gradient_is_the_surrogate():
    # Suppl. "Straight-Through Estimator": m^ = p + sg(m - p) equals m to
    # rounding and has the derivative of p
    rg = np.random.default_rng(3)
    x = torch.tensor(rg.standard_normal(257), dtype=torch.float32, requires_grad=True)
    p = torch.sigmoid(x)
    m = (x > 0.3).float()
    mh = A.straight_through(p, m)
    assert torch.max(torch.abs(mh.detach() - m)).item() <= 2.0 ** -23
    w = torch.tensor(rg.standard_normal(257), dtype=torch.float32)
    (mh * w).sum().backward()
    want = (w * p * (1 - p)).detach()
    assert torch.allclose(x.grad, want, rtol=1e-6, atol=1e-7)


def test_sample_size_rules():
    # ceil(n^(2/3)): the smallest K with K^3 >= n^2, checked by brute force
    for n in list(range(2, 2000)) + [10**6 - 1, 10**6, 10**6 + 1, 10**8, 2**30]:
        c = max(1, round(n ** (2 / 3)) - 3)
        while c ** 3 < n * n:
            c += 1
        assert A.sample_size(n) == min(max(c, 2), n), n
    assert A.sample_size(10**6) == 10**4 and A.sample_size(10**6 + 1) == 10**4 + 1
    assert A.sample_size(10**8, "sqrt") == 20000
    assert A.sample_size(5, "sqrt") == 5          # clamped to n
    with pytest.raises(ValueError):
        A.sample_size(100, "cube")


def test_path_switch():
    assert A.choose_path(1) == "full"
    assert A.choose_path(A.FULL_SORT_MAX_N) == "full"
    assert A.choose_path(A.FULL_SORT_MAX_N + 1) == "bracketed"


def test_no_cpu_fallback():
    x = torch.zeros(16, dtype=torch.float32)
    with pytest.raises(ValueError):
        A.soft_topk(x, 4.0, -1.0)
    with pytest.raises(ValueError):
        A.hard_topk_mask(x, 4)


def test_bracket_indices_are_uniform_and_cached():
    from scipy import stats
    idx = A.bracket_indices(50000, 1000, "cpu", seed=3)
    assert idx.dtype == torch.int32 and idx.shape == (50000,)
    assert int(idx.min()) >= 0 and int(idx.max()) < 1000
    assert A.bracket_indices(50000, 1000, "cpu", seed=3) is idx
    counts = np.bincount(idx.numpy(), minlength=1000)
    assert stats.chisquare(counts).pvalue > 1e-3
