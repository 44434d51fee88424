"""Differentiable soft top-k for training loops, and the straight-through
estimator of the supplement's "Straight-Through Estimator" section.

`soft_topk(scores, k, alpha)` returns p = LapSum_k(scores; alpha) (Eq. (1))
as an autograd node.  Its backward is the library's analytical
vector-Jacobian product (Eq. (5)); when k or alpha are tensors that require
grad (the exact-budget attack of §5 trains both), the same backward
reduction also returns dL/dk and dL/dalpha.  `soft_topk(..., ste=True)`
returns the hard top-k mask m in the forward and differentiates the soft p
in the backward, m^ = p + sg(m - p).

Everything here is orchestration over the C ABI: the threshold, p, the
gradients and the hard mask are computed by the library's kernels.  The
only tensor arithmetic done by torch is input preparation (the i.i.d.
sampler's indices, Suppl. C), reshaping, and summing the per-row dL/dk,
dL/dalpha of a batch that shares one k and one alpha; the bracket's kernel
noise is drawn by the library from the seed.
"""
from __future__ import annotations

import math

import torch

from . import (lapsum_backward, lapsum_backward_band, lapsum_bracket_noise, lapsum_forward,
               lapsum_forward_bracketed, lapsum_topk_mask, new_band)

__all__ = ["soft_topk", "hard_topk_mask", "straight_through", "choose_path", "sample_size",
           "bracket_noise", "bracket_indices", "LapSumFunction", "FULL_SORT_MAX_N"]

# Rows up to this length take the full sort; longer rows the sample bracket.
# §4 places the switch where the two paths cost the same.  On MI355X, one
# Gaussian row, forward + backward, sort against bracket: 0.065 / 0.072 ms
# at n = 2^17, 0.069 / 0.072 at 2^18, 0.076 / 0.074 at 4e5 and 0.088 / 0.072
# at 2^20 with k = n/20, alpha = -0.05; 0.069 / 0.069 at 2^18 and 0.075 /
# 0.071 at 4e5 with k = n/16, alpha = -1; with k = 1000, alpha = -0.05 the
# bracket is ahead from 2^17 on.  Batches of 8 rows of 2^18: 0.533 / 0.487.
FULL_SORT_MAX_N = 1 << 18


def choose_path(n: int) -> str:
    """"full" for n <= FULL_SORT_MAX_N, else "bracketed"."""
    return "full" if n <= FULL_SORT_MAX_N else "bracketed"


def sample_size(n: int, rule: str = "n23") -> int:
    """Bracket sample size K: ceil(n^(2/3)) (Suppl. C, balancing the sample
    sort against the middle-set sort) or, with rule="sqrt", ceil(2 sqrt(n))
    (the coarser choice the paper also allows).  Clamped to [2, n]."""
    if rule == "n23":
        # the smallest K with K^3 >= n^2, in integers (the float estimate
        # can miss by one either way)
        K = math.ceil(n ** (2.0 / 3.0))
        while K ** 3 < n * n:
            K += 1
        while K > 1 and (K - 1) ** 3 >= n * n:
            K -= 1
    elif rule == "sqrt":
        K = math.ceil(2.0 * math.sqrt(n))
    else:
        raise ValueError(f"unknown sample-size rule {rule!r}")
    return int(min(max(K, 2), n))


def bracket_noise(K: int, t: float, device, seed: int = 0):
    """The K draws of Laplace(0, t) kernel noise the bracketed forward uses
    for `seed` when given no table (Suppl. C caches its kernel noise; here
    the library's counter-based generator gives the same draws on every
    call, so nothing is cached)."""
    return lapsum_bracket_noise(seed, K, -float(t), device)


_index_cache: dict = {}


def bracket_indices(K: int, n: int, device, seed: int = 0):
    """K indices drawn uniformly from [0, n) with replacement (int32), for the
    i.i.d. sampler of the coverage theorem (Suppl. C); cached like the noise."""
    device = torch.device(device)
    key = (int(K), int(n), str(device), int(seed))
    hit = _index_cache.get(key)
    if hit is None:
        gen = torch.Generator(device="cpu").manual_seed(int(seed) + 0x5EED)
        hit = torch.randint(0, int(n), (int(K),), generator=gen, dtype=torch.int64)
        hit = hit.to(torch.int32).to(device)
        _index_cache[key] = hit
    return hit


def _as_rows(scores):
    if scores.dim() < 1:
        raise ValueError("scores must have at least one dimension")
    x = scores.detach()
    if x.dtype != torch.float32:
        x = x.float()
    n = x.shape[-1]
    return x.reshape(-1, n).contiguous(), n


class LapSumFunction(torch.autograd.Function):
    """p = LapSum_k(scores; alpha) over the last dimension.

    forward(scores, k, alpha, path, K, z, noise_seed, want_perm, sampler)
    returns p
    (and, with want_perm on the full path, the descending order as a
    non-differentiable int32 tensor).  k and alpha may be Python numbers or
    tensors; as tensors they receive dL/dk and dL/dalpha."""

    @staticmethod
    def forward(ctx, scores, k, alpha, path, K, z, noise_seed, want_perm, sampler="systematic"):
        kf = float(k)
        af = float(alpha)
        x, n = _as_rows(scores)
        if path == "full":
            out = lapsum_forward(x, kf, af, perm=want_perm)
            p, b = out[0], out[1]
            perm = out[2] if want_perm else None
            band = None
        elif path == "bracketed":
            if sampler == "systematic":
                idx = None
            elif sampler == "iid":
                idx = bracket_indices(K, n, x.device, noise_seed)
            else:
                raise ValueError(f"unknown sampler {sampler!r}")
            band = new_band(x.shape[0], n, x.device)
            p, b, _, _ = lapsum_forward_bracketed(x, kf, af, None, K=K, seed=noise_seed, z=z,
                                                  band=band, sample_idx=idx)
            perm = None
        else:
            raise ValueError(f"unknown path {path!r}")
        ctx.alpha = af
        ctx.shape = scores.shape
        ctx.k_like = k if isinstance(k, torch.Tensor) else None
        ctx.alpha_like = alpha if isinstance(alpha, torch.Tensor) else None
        ctx.save_for_backward(p, b, band)
        p_out = p.reshape(scores.shape)
        if perm is not None:
            perm = perm.reshape(scores.shape)
            ctx.mark_non_differentiable(perm)
            return p_out, perm
        return p_out

    @staticmethod
    def backward(ctx, grad_p, *unused):
        p, b, band = ctx.saved_tensors
        g = grad_p.reshape(p.shape)
        if g.dtype != torch.float32:
            g = g.float()
        g = g.contiguous()
        want = bool(ctx.needs_input_grad[1] or ctx.needs_input_grad[2])
        if band is None:
            res = lapsum_backward(g, p, b, ctx.alpha, params=want)
        else:
            res = lapsum_backward_band(g, p, band, ctx.alpha, params=want)
        grad_r, gk, ga = res if want else (res, None, None)
        grad_scores = grad_r.reshape(ctx.shape) if ctx.needs_input_grad[0] else None
        grad_k = grad_alpha = None
        if ctx.needs_input_grad[1]:
            like = ctx.k_like
            grad_k = gk.sum().to(device=like.device, dtype=like.dtype).reshape(like.shape)
        if ctx.needs_input_grad[2]:
            like = ctx.alpha_like
            grad_alpha = ga.sum().to(device=like.device, dtype=like.dtype).reshape(like.shape)
        return grad_scores, grad_k, grad_alpha, None, None, None, None, None, None


def straight_through(p, m):
    """m^ = p + sg(m - p): the forward value is m (to rounding), the gradient
    is that of p."""
    return p + (m - p).detach()


def hard_topk_mask(scores, k: int):
    """m_i = 1 when scores_i is among the k largest of its row (last
    dimension; equal scores ranked by index), else 0."""
    x, n = _as_rows(scores)
    if int(k) != k or not 0 <= int(k) <= n:
        raise ValueError("k must be an integer in [0, n]")
    # the descending order does not depend on the budget; n/2 is a valid one
    _, _, perm = lapsum_forward(x, n / 2.0, -1.0, perm=True)
    return lapsum_topk_mask(perm, int(k)).reshape(scores.shape)


def soft_topk(scores, k, alpha, *, path: str = "auto", sample: str = "n23", z: float = 5.16,
              noise_seed: int = 0, sampler: str = "systematic", ste: bool = False):
    """Differentiable exact-budget soft top-k over the last dimension.

    path: "full" (sort), "bracketed" (sample bracket, §4) or "auto"
    (choose_path by row length).  sample: the bracket's sample-size rule
    (sample_size); sampler: "systematic" (§4's strided view) or "iid"
    (uniform indices, the coverage theorem's model).  ste=True returns the hard mask with the soft p's
    gradient; k must then be an integer."""
    n = scores.shape[-1]
    if path == "auto":
        path = choose_path(n)
    K = sample_size(n, sample) if path == "bracketed" else 0
    if not ste:
        return LapSumFunction.apply(scores, k, alpha, path, K, z, noise_seed, False, sampler)
    kf = float(k)
    if int(kf) != kf:
        raise ValueError("ste=True needs an integer k")
    if path == "full":
        p, perm = LapSumFunction.apply(scores, k, alpha, path, K, z, noise_seed, True, sampler)
        m = lapsum_topk_mask(perm.reshape(-1, n).contiguous(), int(kf)).reshape(scores.shape)
    else:
        p = LapSumFunction.apply(scores, k, alpha, path, K, z, noise_seed, False, sampler)
        m = hard_topk_mask(scores.detach(), int(kf))
    return straight_through(p, m)
