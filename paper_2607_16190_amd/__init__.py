"""Python binding of libfva.so: Top-p block-sparse video attention on MI355X.

Argument marshalling only: every step of the path runs in the gfx950 kernels
behind the C ABI declared in include/fva.h. PyTorch supplies device memory
and the current stream. Importing this module fails loudly when the library
has not been built; there is no fallback implementation.

    import paper_2607_16190_amd as fva
    mask, counts, kv_idx = fva.fva_route(q, k, 0.9, 4, fva.Tiling(21, 45, 80, 2, 8, 8))
    out = fva.fva_attn(q, k, v, tiling, mask, counts, kv_idx)

Hilbert-curve blocks: permute Q, K, V into curve order once, route and
attend with the one-dimensional tiling, and permute O back:

    perm = fva.fva_curve_order(21, 45, 80, device=q.device)
    qc, kc, vc = (fva.fva_permute_tokens(x, perm, fva.FVA_TO_CURVE) for x in (q, k, v))
    tc = fva.Tiling.curve(21 * 45 * 80, 128)
    oc = fva.fva_attn(qc, kc, vc, tc, *fva.fva_route(qc, kc, 0.9, 4, tc))
    out = fva.fva_permute_tokens(oc, perm, fva.FVA_FROM_CURVE)
"""

import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfva.so")

FVA_OK = 0
FVA_ERR_INVALID_ARG = -1
FVA_ERR_SHAPE = -2
FVA_ERR_UNSUPPORTED = -3
FVA_ERR_WORKSPACE = -4
FVA_ERR_HIP = -5
FVA_ERR_SCRATCH = -6

FVA_SCHED_PERSISTENT = 0
FVA_SCHED_NAIVE = 1
FVA_TRACE = 2
FVA_SCHED_UNPAIRED = 4

FVA_TO_CURVE = 0
FVA_FROM_CURVE = 1


def FVA_SPLIT_BLOCKS(s: int) -> int:
    """Flag bits forcing chunks of at most s kept blocks per split row (persistent scheduler)."""
    return (int(s) & 0xFFFF) << 8

EXPORTED = (
    "fva_num_blocks",
    "fva_route_workspace_size",
    "fva_route",
    "fva_route_sasa_workspace_size",
    "fva_route_sasa",
    "fva_attn_workspace_size",
    "fva_trace_words",
    "fva_attn",
    "fva_curve_workspace_size",
    "fva_curve_order",
    "fva_permute_tokens",
    "fva_v8_size",
    "fva_quantize_v_workspace_size",
    "fva_quantize_v",
    "fva_attn_fp8v",
    "fva_attn_noalloc",
    "fva_status_string",
)


class _Tiling(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("T", "H", "W", "bt", "bh", "bw")]


class _Desc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("tokens", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("stride_b", ctypes.c_int64),
        ("stride_h", ctypes.c_int64),
        ("stride_n", ctypes.c_int64),
    ]


@dataclass(frozen=True)
class Tiling:
    """T x H x W latent grid cut into bt x bh x bw blocks."""

    T: int
    H: int
    W: int
    bt: int
    bh: int
    bw: int

    def c(self) -> _Tiling:
        return _Tiling(self.T, self.H, self.W, self.bt, self.bh, self.bw)

    @property
    def tokens(self) -> int:
        return self.T * self.H * self.W

    @classmethod
    def curve(cls, tokens: int, block: int) -> "Tiling":
        """One-dimensional tiling of a curve-ordered sequence: runs of `block` tokens."""
        return cls(1, 1, int(tokens), 1, 1, int(block))


class FvaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {fva_status_string(status)} (status {status})")


def _load():
    # torch ships its own HIP runtime under the same soname; loading torch
    # first makes libfva.so bind to that runtime, so device pointers and
    # streams from torch are valid in the library's launches.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')"
        )
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    T = ctypes.POINTER(_Tiling)
    D = ctypes.POINTER(_Desc)
    sz = ctypes.POINTER(ctypes.c_size_t)
    sigs = {
        "fva_num_blocks": (ctypes.c_int32, [T]),
        "fva_route_workspace_size": (ctypes.c_int, [D, T, sz]),
        "fva_route": (
            ctypes.c_int,
            [P, P, D, ctypes.c_double, ctypes.c_int32, T, P, P, P, P, ctypes.c_size_t, P],
        ),
        "fva_route_sasa_workspace_size": (ctypes.c_int, [D, T, sz]),
        "fva_route_sasa": (
            ctypes.c_int,
            [P, P, D, ctypes.c_double, ctypes.c_int32, T, P, ctypes.c_int32, ctypes.c_double, ctypes.c_double, P, P,
             P, P, P, ctypes.c_size_t, P],
        ),
        "fva_attn_workspace_size": (ctypes.c_int, [D, T, ctypes.c_uint32, sz]),
        "fva_trace_words": (ctypes.c_int64, [D, T]),
        "fva_attn": (
            ctypes.c_int,
            [P, P, P, D, T, P, P, P, ctypes.c_float, ctypes.c_uint32, P, P, ctypes.c_size_t, P, P],
        ),
        "fva_curve_workspace_size": (ctypes.c_int, [ctypes.c_int32] * 3 + [sz]),
        "fva_curve_order": (ctypes.c_int, [ctypes.c_int32] * 3 + [P, P, ctypes.c_size_t, P]),
        "fva_permute_tokens": (ctypes.c_int, [P, P, D, P, ctypes.c_int32, P]),
        "fva_v8_size": (ctypes.c_int, [D, T, sz]),
        "fva_quantize_v_workspace_size": (ctypes.c_int, [D, T, sz]),
        "fva_quantize_v": (ctypes.c_int, [P, D, T, P, P, P, ctypes.c_size_t, P]),
        "fva_attn_fp8v": (
            ctypes.c_int,
            [P, P, P, P, D, T, P, P, P, ctypes.c_float, ctypes.c_uint32, P, P, ctypes.c_size_t, P, P],
        ),
        "fva_attn_noalloc": (
            ctypes.c_int,
            [P, P, P, D, T, P, P, ctypes.c_float, ctypes.c_uint32, P, P, P],
        ),
        "fva_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def fva_status_string(status: int) -> str:
    return lib.fva_status_string(int(status)).decode()


def fva_num_blocks(tiling: Tiling) -> int:
    return int(lib.fva_num_blocks(ctypes.byref(tiling.c())))


def _desc_of(x) -> _Desc:
    if x.dim() != 4:
        raise ValueError("expected a [batch, heads, tokens, head_dim] tensor")
    if x.stride(3) != 1:
        raise ValueError("head_dim must be contiguous")
    B, H, N, D = x.shape
    return _Desc(B, H, N, D, x.stride(0), x.stride(1), x.stride(2))


def _check(status: int, where: str):
    if status != FVA_OK:
        raise FvaError(status, where)


def fva_route_workspace_size(desc: _Desc, tiling: Tiling) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.fva_route_workspace_size(ctypes.byref(desc), ctypes.byref(tiling.c()), ctypes.byref(n)), "fva_route_workspace_size")
    return n.value


def fva_attn_workspace_size(desc: _Desc, tiling: Tiling, flags: int = 0) -> int:
    n = ctypes.c_size_t(0)
    _check(
        lib.fva_attn_workspace_size(ctypes.byref(desc), ctypes.byref(tiling.c()), int(flags), ctypes.byref(n)),
        "fva_attn_workspace_size",
    )
    return n.value


def fva_trace_words(desc: _Desc, tiling: Tiling) -> int:
    return int(lib.fva_trace_words(ctypes.byref(desc), ctypes.byref(tiling.c())))


def _stream_ptr(torch, stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _workspace(torch, nbytes: int, device, workspace):
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError("workspace too small")
        return workspace
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def fva_route(q, k, p: float, k_min: int, tiling: Tiling, *, kv_idx: bool = True, out=None, workspace=None, stream=None):
    """Top-p block routing (see include/fva.h). Returns (mask, counts, kv_idx or None)."""
    import torch

    if q.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or not q.is_cuda or not k.is_cuda:
        raise ValueError("q and k must be bf16 device tensors")
    if q.shape != k.shape or q.stride() != k.stride():
        raise ValueError("q and k must share shape and strides")
    desc = _desc_of(q)
    nb = fva_num_blocks(tiling)
    B, H = q.shape[0], q.shape[1]
    if out is None:
        mask = torch.empty((B, H, max(nb, 0), max(nb, 0)), dtype=torch.uint8, device=q.device)
        counts = torch.empty((B, H, max(nb, 0)), dtype=torch.int32, device=q.device)
        kv = torch.empty((B, H, max(nb, 0), max(nb, 0)), dtype=torch.int32, device=q.device) if kv_idx else None
    else:
        mask, counts, kv = out
    ws = _workspace(torch, fva_route_workspace_size(desc, tiling), q.device, workspace)
    st = lib.fva_route(
        _ptr(q), _ptr(k), ctypes.byref(desc), float(p), int(k_min), ctypes.byref(tiling.c()),
        _ptr(mask), _ptr(counts), _ptr(kv), _ptr(ws), ctypes.c_size_t(ws.numel() * ws.element_size()),
        _stream_ptr(torch, stream),
    )
    _check(st, "fva_route")
    return mask, counts, kv


def fva_route_sasa_workspace_size(desc: _Desc, tiling: Tiling) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.fva_route_sasa_workspace_size(ctypes.byref(desc), ctypes.byref(tiling.c()), ctypes.byref(n)),
           "fva_route_sasa_workspace_size")
    return n.value


def fva_route_sasa(q, k, p: float, k_min: int, tiling: Tiling, rank_of, n_ranks: int, n1: float = 0.8,
                   n2: float = 0.07, *, kv_idx: bool = True, out=None, rank_extra=None, workspace=None, stream=None):
    """Routing plus slack-aware augmentation over the ranks of rank_of (see include/fva.h).

    rank_of: int32 device tensor [batch * heads]. Returns (mask, counts, kv_idx or None, rank_extra).
    """
    import torch

    if q.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or not q.is_cuda or not k.is_cuda:
        raise ValueError("q and k must be bf16 device tensors")
    if q.shape != k.shape or q.stride() != k.stride():
        raise ValueError("q and k must share shape and strides")
    if (rank_of.dtype != torch.int32 or not rank_of.is_cuda or not rank_of.is_contiguous()
            or rank_of.numel() != q.shape[0] * q.shape[1]):
        raise ValueError("rank_of must be a contiguous int32 device tensor with one entry per (batch, head)")
    desc = _desc_of(q)
    nb = fva_num_blocks(tiling)
    B, H = q.shape[0], q.shape[1]
    if out is None:
        mask = torch.empty((B, H, max(nb, 0), max(nb, 0)), dtype=torch.uint8, device=q.device)
        counts = torch.empty((B, H, max(nb, 0)), dtype=torch.int32, device=q.device)
        kv = torch.empty((B, H, max(nb, 0), max(nb, 0)), dtype=torch.int32, device=q.device) if kv_idx else None
    else:
        mask, counts, kv = out
    if rank_extra is None:
        rank_extra = torch.empty(max(int(n_ranks), 1), dtype=torch.int32, device=q.device)
    ws = _workspace(torch, fva_route_sasa_workspace_size(desc, tiling), q.device, workspace)
    st = lib.fva_route_sasa(
        _ptr(q), _ptr(k), ctypes.byref(desc), float(p), int(k_min), ctypes.byref(tiling.c()), _ptr(rank_of),
        int(n_ranks), float(n1), float(n2), _ptr(mask), _ptr(counts), _ptr(kv), _ptr(rank_extra), _ptr(ws),
        ctypes.c_size_t(ws.numel() * ws.element_size()), _stream_ptr(torch, stream),
    )
    _check(st, "fva_route_sasa")
    return mask, counts, kv, rank_extra


def fva_attn(q, k, v, tiling: Tiling, mask, counts=None, kv_idx=None, *, scale: float = 0.0, flags: int = 0,
             out=None, workspace=None, trace=None, stream=None):
    """Block-sparse attention over the kept blocks (see include/fva.h). Returns O."""
    import torch

    for t in (q, k, v):
        if t.dtype != torch.bfloat16 or not t.is_cuda:
            raise ValueError("q, k, v must be bf16 device tensors")
    if not (q.shape == k.shape == v.shape) or not (q.stride() == k.stride() == v.stride()):
        raise ValueError("q, k, v must share shape and strides")
    desc = _desc_of(q)
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=torch.bfloat16, device=q.device)
    elif out.stride() != q.stride() or out.shape != q.shape or out.dtype != torch.bfloat16:
        raise ValueError("out must match q in shape, strides and dtype")
    ws = _workspace(torch, fva_attn_workspace_size(desc, tiling, flags), q.device, workspace)
    if (flags & FVA_TRACE) and trace is None:
        raise ValueError("FVA_TRACE needs a trace tensor of fva_trace_words int64")
    st = lib.fva_attn(
        _ptr(q), _ptr(k), _ptr(v), ctypes.byref(desc), ctypes.byref(tiling.c()), _ptr(mask), _ptr(counts),
        _ptr(kv_idx), ctypes.c_float(scale), int(flags), _ptr(out), _ptr(ws),
        ctypes.c_size_t(ws.numel() * ws.element_size()), _ptr(trace), _stream_ptr(torch, stream),
    )
    _check(st, "fva_attn")
    return out


def fva_attn_noalloc(q, k, v, tiling: Tiling, counts, kv_idx, out, *, scale: float = 0.0, flags: int = 0,
                     trace=None, stream=None):
    """fva_attn on the library's static scratch (see include/fva.h): no device
    allocation in the library or here; the caller passes every buffer,
    including `out`."""
    import torch

    for t in (q, k, v, out):
        if t.dtype != torch.bfloat16 or not t.is_cuda:
            raise ValueError("q, k, v, out must be bf16 device tensors")
    if not (q.shape == k.shape == v.shape == out.shape) or not (q.stride() == k.stride() == v.stride() == out.stride()):
        raise ValueError("q, k, v, out must share shape and strides")
    for t in (counts, kv_idx):
        if t is None or t.dtype != torch.int32 or not t.is_cuda:
            raise ValueError("counts and kv_idx must be int32 device tensors")
    if (flags & FVA_TRACE) and trace is None:
        raise ValueError("FVA_TRACE needs a trace tensor of fva_trace_words int64")
    desc = _desc_of(q)
    st = lib.fva_attn_noalloc(
        _ptr(q), _ptr(k), _ptr(v), ctypes.byref(desc), ctypes.byref(tiling.c()), _ptr(counts), _ptr(kv_idx),
        ctypes.c_float(scale), int(flags), _ptr(out), _ptr(trace), _stream_ptr(torch, stream),
    )
    _check(st, "fva_attn_noalloc")
    return out


def fva_curve_workspace_size(T: int, H: int, W: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.fva_curve_workspace_size(int(T), int(H), int(W), ctypes.byref(n)), "fva_curve_workspace_size")
    return n.value


def fva_curve_order(T: int, H: int, W: int, *, device=None, out=None, workspace=None, stream=None):
    """perm[r] = raster token id of the token of Hilbert-curve rank r (int32 device tensor)."""
    import torch

    dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
    N = int(T) * int(H) * int(W)
    perm = out if out is not None else torch.empty(N, dtype=torch.int32, device=dev)
    if perm.dtype != torch.int32 or perm.numel() != N or not perm.is_contiguous() or not perm.is_cuda:
        raise ValueError("perm must be a contiguous int32 device tensor of T*H*W entries")
    ws = _workspace(torch, fva_curve_workspace_size(T, H, W), perm.device, workspace)
    st = lib.fva_curve_order(int(T), int(H), int(W), _ptr(perm), _ptr(ws),
                             ctypes.c_size_t(ws.numel() * ws.element_size()), _stream_ptr(torch, stream))
    _check(st, "fva_curve_order")
    return perm


def fva_permute_tokens(x, perm, direction: int, *, out=None, stream=None):
    """Token rows of x into (FVA_TO_CURVE) or out of (FVA_FROM_CURVE) curve order."""
    import torch

    if x.dtype != torch.bfloat16 or not x.is_cuda:
        raise ValueError("x must be a bf16 device tensor")
    if perm.dtype != torch.int32 or not perm.is_cuda or not perm.is_contiguous() or perm.numel() != x.shape[2]:
        raise ValueError("perm must be a contiguous int32 device tensor with one entry per token")
    desc = _desc_of(x)
    if out is None:
        out = torch.empty_strided(x.shape, x.stride(), dtype=torch.bfloat16, device=x.device)
    elif out.stride() != x.stride() or out.shape != x.shape or out.dtype != torch.bfloat16:
        raise ValueError("out must match x in shape, strides and dtype")
    st = lib.fva_permute_tokens(_ptr(x), _ptr(out), ctypes.byref(desc), _ptr(perm), int(direction),
                                _stream_ptr(torch, stream))
    _check(st, "fva_permute_tokens")
    return out


def fva_v8_size(desc: _Desc, tiling: Tiling) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.fva_v8_size(ctypes.byref(desc), ctypes.byref(tiling.c()), ctypes.byref(n)), "fva_v8_size")
    return n.value


def fva_quantize_v_workspace_size(desc: _Desc, tiling: Tiling) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.fva_quantize_v_workspace_size(ctypes.byref(desc), ctypes.byref(tiling.c()), ctypes.byref(n)),
           "fva_quantize_v_workspace_size")
    return n.value


def fva_quantize_v(v, tiling: Tiling, *, out=None, workspace=None, stream=None):
    """E4M3 tiles and per-channel exponents of V (see include/fva.h). Returns (v8, v_exp)."""
    import torch

    if v.dtype != torch.bfloat16 or not v.is_cuda:
        raise ValueError("v must be a bf16 device tensor")
    desc = _desc_of(v)
    nb = fva_num_blocks(tiling)
    B, H = v.shape[0], v.shape[1]
    if out is None:
        v8 = torch.empty((B, H, max(nb, 0), 128, 128), dtype=torch.uint8, device=v.device)
        vexp = torch.empty((B, H, 128), dtype=torch.int32, device=v.device)
    else:
        v8, vexp = out
    if v8.numel() < fva_v8_size(desc, tiling) or not v8.is_contiguous() or vexp.numel() < B * H * 128:
        raise ValueError("v8 / v_exp too small or not contiguous")
    ws = _workspace(torch, fva_quantize_v_workspace_size(desc, tiling), v.device, workspace)
    st = lib.fva_quantize_v(_ptr(v), ctypes.byref(desc), ctypes.byref(tiling.c()), _ptr(v8), _ptr(vexp), _ptr(ws),
                            ctypes.c_size_t(ws.numel() * ws.element_size()), _stream_ptr(torch, stream))
    _check(st, "fva_quantize_v")
    return v8, vexp


def fva_attn_fp8v(q, k, v8, vexp, tiling: Tiling, mask, counts=None, kv_idx=None, *, scale: float = 0.0,
                  flags: int = 0, out=None, workspace=None, trace=None, stream=None):
    """Block-sparse attention with E4M3 V (see include/fva.h). Returns O (bf16, q's layout)."""
    import torch

    for t in (q, k):
        if t.dtype != torch.bfloat16 or not t.is_cuda:
            raise ValueError("q, k must be bf16 device tensors")
    if q.shape != k.shape or q.stride() != k.stride():
        raise ValueError("q and k must share shape and strides")
    if v8.dtype != torch.uint8 or vexp.dtype != torch.int32 or not v8.is_contiguous() or not vexp.is_contiguous():
        raise ValueError("v8 must be contiguous uint8 and v_exp contiguous int32 (from fva_quantize_v)")
    desc = _desc_of(q)
    if v8.numel() < fva_v8_size(desc, tiling) or vexp.numel() < q.shape[0] * q.shape[1] * 128:
        raise ValueError("v8 / v_exp do not match q and the tiling")
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=torch.bfloat16, device=q.device)
    elif out.stride() != q.stride() or out.shape != q.shape or out.dtype != torch.bfloat16:
        raise ValueError("out must match q in shape, strides and dtype")
    ws = _workspace(torch, fva_attn_workspace_size(desc, tiling, flags), q.device, workspace)
    if (flags & FVA_TRACE) and trace is None:
        raise ValueError("FVA_TRACE needs a trace tensor of fva_trace_words int64")
    st = lib.fva_attn_fp8v(
        _ptr(q), _ptr(k), _ptr(v8), _ptr(vexp), ctypes.byref(desc), ctypes.byref(tiling.c()), _ptr(mask),
        _ptr(counts), _ptr(kv_idx), ctypes.c_float(scale), int(flags), _ptr(out), _ptr(ws),
        ctypes.c_size_t(ws.numel() * ws.element_size()), _ptr(trace), _stream_ptr(torch, stream),
    )
    _check(st, "fva_attn_fp8v")
    return out

