"""Exact-budget LapSum soft top-k ("Fast LapSum") on AMD Instinct MI355X.

Thin Python binding over the C ABI of liblapsum.so (include/lapsum.h).  The
functions carry the C names and only marshal arguments: torch supplies
device memory and the current HIP stream, every step of the computation runs
in the library's HIP kernels.  There is no CPU fallback: if the library is
not built, or the tensors are not on a gfx950 device, the calls raise.

    p, b = lapsum_forward(scores, k, alpha)                 # full sort
    grad_r = lapsum_backward(grad_p, p, b, alpha)           # Eq. (5) VJP
    p, b, info, m_idx = lapsum_forward_bracketed(scores, k, alpha, noise)

`scores` is a float32 CUDA tensor of shape [n] or [batch, n]; k and alpha
are Python floats with 0 < k < n and alpha < 0.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "load", "LapsumError", "BracketInfo", "lapsum_status_string",
    "lapsum_forward_workspace_size", "lapsum_forward", "lapsum_forward_noalloc",
    "NOALLOC_SCRATCH_BYTES",
    "lapsum_backward_workspace_size", "lapsum_backward",
    "lapsum_forward_bracketed_workspace_size", "lapsum_forward_bracketed", "lapsum_bracket_noise",
    "LAPSUM_FLAG_FULL_SORT", "LIB_PATH", "lapsum_profile_start", "lapsum_profile_stop",
    "lapsum_band_size", "new_band", "lapsum_backward_band_workspace_size", "lapsum_backward_band",
    "lapsum_topk_mask", "lapsum_bisect_forward", "lapsum_dftopk_workspace_size",
    "lapsum_dftopk_forward", "lapsum_dftopk_backward",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblapsum.so")
LAPSUM_FLAG_FULL_SORT = 1
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024   # LAPSUM_NOALLOC_SCRATCH_BYTES

_lib = None


class LapsumError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lapsum_status_string(status)} (status {status})")


class BracketInfo(ctypes.Structure):
    """Mirror of lapsum_bracket_info."""
    _fields_ = [
        ("a_L", ctypes.c_float), ("a_R", ctypes.c_float),
        ("j", ctypes.c_int64), ("l", ctypes.c_int64),
        ("n_L", ctypes.c_int64), ("n_M", ctypes.c_int64), ("n_R", ctypes.c_int64),
        ("T_L", ctypes.c_double), ("T_R", ctypes.c_double),
        ("lap_aL", ctypes.c_double), ("lap_aR", ctypes.c_double),
        ("attempts", ctypes.c_int32), ("fell_back", ctypes.c_int32),
        ("m_overflow", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]

    _names = None

    def as_dict(self) -> dict:
        names = BracketInfo._names
        if names is None:
            names = BracketInfo._names = tuple(nm for nm, _ in self._fields_ if nm != "reserved")
        return {name: getattr(self, name) for name in names}


def load():
    """Load liblapsum.so (built in-tree) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_06912_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, f64, sz, u32, i32, u64 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_double,
                                       ctypes.c_size_t, ctypes.c_uint32, ctypes.c_int,
                                       ctypes.c_uint64)
    lib.lapsum_status_string.argtypes = [i32]
    lib.lapsum_status_string.restype = ctypes.c_char_p
    lib.lapsum_forward_workspace_size.argtypes = [i64, i64, i32]
    lib.lapsum_forward_workspace_size.restype = sz
    lib.lapsum_forward.argtypes = [vp, i64, i64, f64, f64, vp, vp, vp, vp, sz, vp]
    lib.lapsum_forward.restype = i32
    lib.lapsum_forward_noalloc.argtypes = [vp, i64, i64, f64, f64, vp, vp, vp, vp]
    lib.lapsum_forward_noalloc.restype = i32
    lib.lapsum_backward_workspace_size.argtypes = [i64, i64]
    lib.lapsum_backward_workspace_size.restype = sz
    lib.lapsum_backward.argtypes = [vp, vp, vp, i64, i64, f64, vp, vp, vp, vp, sz, vp]
    lib.lapsum_backward.restype = i32
    lib.lapsum_forward_bracketed_workspace_size.argtypes = [i64, i64, i64, i64, i32]
    lib.lapsum_forward_bracketed_workspace_size.restype = sz
    lib.lapsum_forward_bracketed.argtypes = [vp, i64, i64, f64, f64, i64, f64, vp, u64, vp, i64, u32,
                                             vp, vp, vp, vp, vp, sz, vp, sz, vp]
    lib.lapsum_forward_bracketed.restype = i32
    lib.lapsum_bracket_noise.argtypes = [u64, i64, f64, vp, vp]
    lib.lapsum_bracket_noise.restype = i32
    lib.lapsum_band_size.argtypes = [i64, i64]
    lib.lapsum_band_size.restype = sz
    lib.lapsum_backward_band_workspace_size.argtypes = [i64, i64]
    lib.lapsum_backward_band_workspace_size.restype = sz
    lib.lapsum_backward_band.argtypes = [vp, vp, vp, sz, i64, i64, f64, vp, vp, vp, vp, sz, vp]
    lib.lapsum_backward_band.restype = i32
    lib.lapsum_bisect_forward.argtypes = [vp, i64, i64, f64, f64, i32, vp, vp, vp]
    lib.lapsum_bisect_forward.restype = i32
    lib.lapsum_dftopk_workspace_size.argtypes = [i64, i64]
    lib.lapsum_dftopk_workspace_size.restype = sz
    lib.lapsum_dftopk_forward.argtypes = [vp, i64, i64, i64, f64, vp, vp, vp, vp, sz, vp]
    lib.lapsum_dftopk_forward.restype = i32
    lib.lapsum_dftopk_backward.argtypes = [vp, vp, vp, i64, i64, f64, vp, vp, sz, vp]
    lib.lapsum_dftopk_backward.restype = i32
    lib.lapsum_topk_mask.argtypes = [vp, i64, i64, i64, vp, vp]
    lib.lapsum_topk_mask.restype = i32
    lib.lapsum_profile_start.argtypes = []
    lib.lapsum_profile_start.restype = i32
    lib.lapsum_profile_stop.argtypes = []
    lib.lapsum_profile_stop.restype = i32
    lib.lapsum_profile_entry.argtypes = [i32, ctypes.c_char_p, sz, ctypes.POINTER(ctypes.c_int64),
                                         ctypes.POINTER(ctypes.c_double)]
    lib.lapsum_profile_entry.restype = i32
    _lib = lib
    return lib


def lapsum_status_string(status: int) -> str:
    return load().lapsum_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != 0:
        raise LapsumError(status, where)


_torch_mod = None


def _torch():
    global _torch_mod
    if _torch_mod is None:
        import torch
        _torch_mod = torch
    return _torch_mod


_get_device = None


def _current_device() -> int:
    """The current HIP device index.  torch's raw query skips the lazy-init
    check of torch.cuda.current_device(); every caller already holds a
    tensor on the device, so initialisation has happened."""
    global _get_device
    if _get_device is None:
        torch = _torch()
        _get_device = getattr(torch._C, "_cuda_getDevice", None) or torch.cuda.current_device
    return _get_device()


class _on_device:
    """Make `device` current for a call (a no-op when it already is, or when
    the device names no index, which means the current one)."""

    __slots__ = ("dev", "prev")

    def __init__(self, device):
        self.dev = device.index
        self.prev = None

    def __enter__(self):
        if self.dev is not None:
            cur = _current_device()
            if cur != self.dev:
                self.prev = cur
                _torch().cuda.set_device(self.dev)
        return self

    def __exit__(self, *exc):
        if self.prev is not None:
            _torch().cuda.set_device(self.prev)
        return False


def _rows(x, name):
    torch = _torch()
    # the common case in one test; the checks below say what is wrong
    if type(x) is torch.Tensor and x.is_cuda and x.dtype is torch.float32 and x.is_contiguous():
        shape = x.shape
        if len(shape) == 2:
            return shape[0], shape[1]
        if len(shape) == 1:
            return 1, shape[0]
    if not isinstance(x, torch.Tensor) or x.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if x.dtype != torch.float32:
        raise ValueError(f"{name} must be float32")
    if x.dim() not in (1, 2):
        raise ValueError(f"{name} must have shape [n] or [batch, n]")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    batch, n = (1, x.shape[0]) if x.dim() == 1 else (x.shape[0], x.shape[1])
    return int(batch), int(n)


_raw_stream = None


def _stream(device):
    """The caller's current HIP stream on `device` as a raw handle (an int,
    which ctypes passes as a pointer).  torch's raw-handle query (0.14 us a
    call on MI355X) skips building a Stream object (2.0 us), which shows on
    short rows; the public query is the fallback where the raw one is
    missing."""
    global _raw_stream
    torch = _torch()
    if _raw_stream is None:
        _raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", False)
    if _raw_stream:
        idx = device.index
        return _raw_stream(idx if idx is not None else _current_device())
    return torch.cuda.current_stream(device).cuda_stream


def _workspace(nbytes, device, workspace):
    torch = _torch()
    if nbytes == 0:
        return None, 0
    if workspace is not None and workspace.numel() * workspace.element_size() >= nbytes:
        ws = workspace
    else:
        ws = torch.empty(int(nbytes), dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise ValueError("workspace must be 256-byte aligned")
    return ws, ws.numel() * ws.element_size()


def _ptr(t):
    # an int (or None for NULL): ctypes converts both for a c_void_p argument
    # without building a c_void_p object per pointer
    return t.data_ptr() if t is not None else None


def lapsum_forward_workspace_size(batch: int, n: int, with_perm: bool = False) -> int:
    return int(load().lapsum_forward_workspace_size(batch, n, int(bool(with_perm))))


def lapsum_forward(scores, k: float, alpha: float, *, perm: bool = False, workspace=None):
    """Full-sort forward.  Returns (p, b) or (p, b, perm) with perm=True;
    p has the shape of scores, b is float64 of shape [batch]."""
    torch = _torch()
    lib = load()
    batch, n = _rows(scores, "scores")
    dev = scores.device
    p = torch.empty_like(scores)
    b = torch.empty(batch, dtype=torch.float64, device=dev)
    pm = torch.empty(scores.shape, dtype=torch.int32, device=dev) if perm else None
    ws, nbytes = _workspace(lib.lapsum_forward_workspace_size(batch, n, int(perm)), dev, workspace)
    with _on_device(dev):
        _check(lib.lapsum_forward(_ptr(scores), batch, n, float(k), float(alpha), _ptr(p), _ptr(b),
                                  _ptr(pm), _ptr(ws), nbytes, _stream(dev)), "lapsum_forward")
    return (p, b, pm) if perm else (p, b)


def lapsum_forward_noalloc(scores, k: float, alpha: float, *, perm: bool = False, out=None,
                           b_out=None, perm_out=None):
    """lapsum_forward with the library's own device scratch (no workspace,
    no allocation inside the call).  out / b_out / perm_out: optional
    preallocated outputs (float32 like scores, float64 [batch], int32 like
    scores), so that a caller under graph capture allocates nothing either.
    Returns (p, b) or (p, b, perm)."""
    torch = _torch()
    lib = load()
    batch, n = _rows(scores, "scores")
    dev = scores.device
    p = torch.empty_like(scores) if out is None else out
    b = torch.empty(batch, dtype=torch.float64, device=dev) if b_out is None else b_out
    if perm:
        pm = torch.empty(scores.shape, dtype=torch.int32, device=dev) if perm_out is None else perm_out
    else:
        pm = None
    for name, buf, dt, numel in (("out", p, torch.float32, batch * n), ("b_out", b, torch.float64, batch),
                                 ("perm_out", pm, torch.int32, batch * n)):
        if buf is not None and (buf.dtype != dt or buf.numel() != numel or not buf.is_contiguous()
                                or buf.device != dev):
            raise ValueError(f"{name} must be a contiguous {dt} tensor of {numel} elements on "
                             f"the scores' device")
    with _on_device(dev):
        _check(lib.lapsum_forward_noalloc(_ptr(scores), batch, n, float(k), float(alpha), _ptr(p),
                                          _ptr(b), _ptr(pm), _stream(dev)),
               "lapsum_forward_noalloc")
    return (p, b, pm) if perm else (p, b)


def lapsum_topk_mask(perm, k: int, *, out=None):
    """Hard top-k mask (1.0 for the k largest scores of each row, 0.0
    elsewhere) from a descending order `perm` (int32, lapsum_forward's
    perm)."""
    torch = _torch()
    lib = load()
    if not isinstance(perm, torch.Tensor) or perm.device.type != "cuda" or \
            perm.dtype != torch.int32 or perm.dim() not in (1, 2) or not perm.is_contiguous():
        raise ValueError("perm must be a contiguous int32 CUDA tensor of shape [n] or [batch, n]")
    batch, n = (1, perm.shape[0]) if perm.dim() == 1 else (perm.shape[0], perm.shape[1])
    if int(k) != k:
        raise ValueError("k must be an integer count")
    dev = perm.device
    mask = out if out is not None else torch.empty(perm.shape, dtype=torch.float32, device=dev)
    if mask.shape != perm.shape or mask.dtype != torch.float32 or not mask.is_contiguous():
        raise ValueError("out must be a contiguous float32 tensor shaped like perm")
    with _on_device(dev):
        _check(lib.lapsum_topk_mask(_ptr(perm), int(batch), int(n), int(k), _ptr(mask),
                                    _stream(dev)), "lapsum_topk_mask")
    return mask


def lapsum_bisect_forward(scores, k: float, alpha: float, steps: int = 60):
    """Comparator: the per-query bisection baseline (one thread per row,
    float32).  Returns (p, b)."""
    torch = _torch()
    lib = load()
    batch, n = _rows(scores, "scores")
    dev = scores.device
    p = torch.empty_like(scores)
    b = torch.empty(batch, dtype=torch.float64, device=dev)
    with _on_device(dev):
        _check(lib.lapsum_bisect_forward(_ptr(scores), batch, n, float(k), float(alpha), int(steps),
                                         _ptr(p), _ptr(b), _stream(dev)), "lapsum_bisect_forward")
    return p, b


def lapsum_dftopk_workspace_size(batch: int, n: int) -> int:
    return int(load().lapsum_dftopk_workspace_size(batch, n))


def lapsum_dftopk_forward(scores, k: int, alpha: float, *, workspace=None):
    """Comparator: DFTopK.  Returns (p, c, pair): c float64 [batch], pair
    int32 [batch, 2] (indices of the k-th and (k+1)-th largest scores)."""
    torch = _torch()
    lib = load()
    batch, n = _rows(scores, "scores")
    if int(k) != k:
        raise ValueError("k must be an integer")
    dev = scores.device
    p = torch.empty_like(scores)
    c = torch.empty(batch, dtype=torch.float64, device=dev)
    pair = torch.empty((batch, 2), dtype=torch.int32, device=dev)
    ws, nbytes = _workspace(lib.lapsum_dftopk_workspace_size(batch, n), dev, workspace)
    with _on_device(dev):
        _check(lib.lapsum_dftopk_forward(_ptr(scores), batch, n, int(k), float(alpha), _ptr(p),
                                         _ptr(c), _ptr(pair), _ptr(ws), nbytes, _stream(dev)),
               "lapsum_dftopk_forward")
    return p, c, pair


def lapsum_dftopk_backward(grad_p, p, pair, alpha: float, *, workspace=None, out=None):
    """Comparator: the DFTopK vector-Jacobian product."""
    torch = _torch()
    lib = load()
    batch, n = _rows(p, "p")
    if grad_p.shape != p.shape:
        raise ValueError("grad_p and p must have the same shape")
    _rows(grad_p, "grad_p")
    if pair.dtype != torch.int32 or tuple(pair.shape) != (batch, 2) or not pair.is_contiguous():
        raise ValueError("pair must be a contiguous int32 tensor [batch, 2]")
    dev = p.device
    grad = out if out is not None else torch.empty_like(p)
    ws, nbytes = _workspace(lib.lapsum_dftopk_workspace_size(batch, n), dev, workspace)
    with _on_device(dev):
        _check(lib.lapsum_dftopk_backward(_ptr(grad_p), _ptr(p), _ptr(pair), batch, n,
                                          float(alpha), _ptr(grad), _ptr(ws), nbytes,
                                          _stream(dev)), "lapsum_dftopk_backward")
    return grad


def lapsum_backward_workspace_size(batch: int, n: int) -> int:
    return int(load().lapsum_backward_workspace_size(batch, n))


def _param_grads(p, params: bool, params_out=None):
    """float64 outputs for dL/dk and dL/dalpha, one per row (shape
    p.shape[:-1]); params_out, if given, is a pair of such tensors to fill."""
    if not params:
        return None, None
    torch = _torch()
    shape = tuple(p.shape[:-1])
    if params_out is not None:
        for x in params_out:
            if x.dtype != torch.float64 or tuple(x.shape) != shape or x.device != p.device \
                    or not x.is_contiguous():
                raise ValueError(f"params_out: float64 tensors of shape {shape} on {p.device}")
        return params_out
    return (torch.empty(shape, dtype=torch.float64, device=p.device),
            torch.empty(shape, dtype=torch.float64, device=p.device))


def lapsum_backward(grad_p, p, b, alpha: float, *, params: bool = False, params_out=None,
                    workspace=None, out=None):
    """VJP of Eq. (5): grad_r = f * (g - <g, q>) with f from p.  With
    params=True returns (grad_r, grad_k, grad_alpha), the last two float64 of
    shape p.shape[:-1]: the gradients with respect to the budget and the
    temperature from the same reduction."""
    torch = _torch()
    lib = load()
    batch, n = _rows(p, "p")
    if grad_p.shape != p.shape:
        raise ValueError("grad_p and p must have the same shape")
    _rows(grad_p, "grad_p")
    dev = p.device
    grad = out if out is not None else torch.empty_like(p)
    gk, ga = _param_grads(p, params, params_out)
    ws, nbytes = _workspace(lib.lapsum_backward_workspace_size(batch, n), dev, workspace)
    with _on_device(dev):
        _check(lib.lapsum_backward(_ptr(grad_p), _ptr(p), _ptr(b), batch, n, float(alpha),
                                   _ptr(grad), _ptr(gk), _ptr(ga), _ptr(ws), nbytes, _stream(dev)),
               "lapsum_backward")
    return (grad, gk, ga) if params else grad


def lapsum_forward_bracketed_workspace_size(batch: int, n: int, K: int, m_capacity: int,
                                            with_m_idx: bool = False) -> int:
    return int(load().lapsum_forward_bracketed_workspace_size(batch, n, K, m_capacity,
                                                              int(bool(with_m_idx))))


def default_m_capacity(n: int, K: int) -> int:
    """A middle-set capacity comfortably above the expected band of a z = 5.16
    bracket (rank width ~ 2 z n / sqrt(K)) and its widenings."""
    return int(min(n, max(1 << 16, 64 * (n // max(1, int(K ** 0.5))))))


def lapsum_band_size(batch: int, n: int) -> int:
    return int(load().lapsum_band_size(batch, n))


def new_band(batch: int, n: int, device):
    """Device buffer for the band a bracketed forward saves for its backward."""
    torch = _torch()
    return torch.empty(max(1, lapsum_band_size(batch, n)), dtype=torch.uint8, device=device)


def _band_arg(band, batch, n):
    torch = _torch()
    if band is None:
        return ctypes.c_void_p(0), 0
    if not isinstance(band, torch.Tensor) or band.device.type != "cuda" or not band.is_contiguous():
        raise ValueError("band must be a contiguous CUDA tensor (see new_band)")
    return ctypes.c_void_p(band.data_ptr()), band.numel() * band.element_size()


def lapsum_bracket_noise(seed: int, K: int, alpha: float, device="cuda", *, out=None):
    """The default kernel noise of the bracket: K float32 Laplace(0, |alpha|)
    draws of the counter-based generator at `seed` (the table the bracketed
    forward uses when given noise=None)."""
    torch = _torch()
    if out is None:
        out = torch.empty(int(K), dtype=torch.float32, device=device)
    elif out.dtype != torch.float32 or out.numel() != int(K) or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 tensor of K elements")
    with _on_device(out.device):
        _check(load().lapsum_bracket_noise(int(seed) & ((1 << 64) - 1), int(K), float(alpha),
                                           _ptr(out), _stream(out.device)),
               "lapsum_bracket_noise")
    return out


def lapsum_forward_bracketed(scores, k: float, alpha: float, noise=None, *, K: int | None = None,
                             seed: int = 0, z: float = 5.16,
                             m_capacity: int | None = None, flags: int = 0,
                             m_idx: bool = False, band=None, workspace=None, out=None,
                             b_out=None, sample_idx=None):
    """Bracketed forward.  noise: float32 CUDA tensor [K] of Laplace(0, |alpha|)
    draws, or None for the library's default noise of `seed` (then K must be
    given).  sample_idx: None (systematic sample) or an int32 CUDA tensor [K]
    of indices in [0, n) for the i.i.d. sample.  band: None, or a buffer from new_band() that receives the band for
    lapsum_backward_band.  out / b_out: optional buffers for p (float32, the
    shape of scores) and b (float64, [batch]).  Returns (p, b, infos, m_idx or
    None) with infos a list of dicts."""
    torch = _torch()
    lib = load()
    batch, n = _rows(scores, "scores")
    if noise is not None:
        if noise.dim() != 1:
            raise ValueError("noise must be 1-D [K]")
        _rows(noise, "noise")
        if K is not None and int(K) != int(noise.shape[0]):
            raise ValueError("K differs from the noise table's length")
        K = int(noise.shape[0])
    elif K is None:
        raise ValueError("K is required when noise is None")
    K = int(K)
    if sample_idx is not None:
        if (not isinstance(sample_idx, torch.Tensor) or sample_idx.dtype != torch.int32
                or tuple(sample_idx.shape) != (K,) or sample_idx.device != scores.device
                or not sample_idx.is_contiguous()):
            raise ValueError("sample_idx must be a contiguous int32 tensor [K] on the scores' device")
    if m_capacity is None:
        m_capacity = default_m_capacity(n, K)
    dev = scores.device
    if out is not None:
        if (out.shape != scores.shape or out.dtype != torch.float32 or not out.is_contiguous()
                or out.device != dev):
            raise ValueError("out must be a contiguous float32 tensor shaped like scores")
        p = out
    else:
        p = torch.empty_like(scores)
    if b_out is not None:
        if (b_out.numel() != batch or b_out.dtype != torch.float64 or not b_out.is_contiguous()
                or b_out.device != dev):
            raise ValueError("b_out must be a contiguous float64 tensor of [batch] elements")
        b = b_out
    else:
        b = torch.empty(batch, dtype=torch.float64, device=dev)
    mi = torch.empty((batch, m_capacity), dtype=torch.int32, device=dev) if m_idx else None
    infos = (BracketInfo * batch)()
    ws, nbytes = _workspace(lib.lapsum_forward_bracketed_workspace_size(batch, n, K, m_capacity,
                                                                        int(m_idx)), dev, workspace)
    bp, bbytes = _band_arg(band, batch, n)
    with _on_device(dev):
        _check(lib.lapsum_forward_bracketed(_ptr(scores), batch, n, float(k), float(alpha), K,
                                            float(z), _ptr(noise), int(seed) & ((1 << 64) - 1),
                                            _ptr(sample_idx),
                                            int(m_capacity), int(flags),
                                            _ptr(p), _ptr(b), ctypes.cast(infos, ctypes.c_void_p),
                                            _ptr(mi), bp, bbytes, _ptr(ws), nbytes, _stream(dev)),
               "lapsum_forward_bracketed")
    return p, b, [infos[i].as_dict() for i in range(batch)], mi


def lapsum_backward_band_workspace_size(batch: int, n: int) -> int:
    return int(load().lapsum_backward_band_workspace_size(batch, n))


def lapsum_backward_band(grad_p, p, band, alpha: float, *, params: bool = False,
                         params_out=None, workspace=None, out=None):
    """Eq. (5) VJP from the band a bracketed forward saved (see new_band);
    params=True as in lapsum_backward."""
    torch = _torch()
    lib = load()
    batch, n = _rows(p, "p")
    if grad_p.shape != p.shape:
        raise ValueError("grad_p and p must have the same shape")
    _rows(grad_p, "grad_p")
    if band is None:
        raise ValueError("band is required")
    dev = p.device
    grad = out if out is not None else torch.empty_like(p)
    gk, ga = _param_grads(p, params, params_out)
    ws, nbytes = _workspace(lib.lapsum_backward_band_workspace_size(batch, n), dev, workspace)
    bp, bbytes = _band_arg(band, batch, n)
    with _on_device(dev):
        _check(lib.lapsum_backward_band(_ptr(grad_p), _ptr(p), bp, bbytes, batch, n, float(alpha),
                                        _ptr(grad), _ptr(gk), _ptr(ga), _ptr(ws), nbytes,
                                        _stream(dev)),
               "lapsum_backward_band")
    return (grad, gk, ga) if params else grad


def lapsum_profile_start() -> None:
    """Record HIP events around every kernel the library launches."""
    _check(load().lapsum_profile_start(), "lapsum_profile_start")


def lapsum_profile_stop() -> dict:
    """Stop recording; returns {kernel: (launches, total_ms)}."""
    lib = load()
    cnt = lib.lapsum_profile_stop()
    if cnt < 0:
        raise LapsumError(-cnt, "lapsum_profile_stop")
    out = {}
    buf = ctypes.create_string_buffer(128)
    for i in range(cnt):
        launches = ctypes.c_int64(0)
        ms = ctypes.c_double(0.0)
        _check(lib.lapsum_profile_entry(i, buf, 128, ctypes.byref(launches), ctypes.byref(ms)),
               "lapsum_profile_entry")
        out[buf.value.decode()] = (int(launches.value), float(ms.value))
    return out
