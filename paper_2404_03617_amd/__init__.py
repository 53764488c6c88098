"""MI355X-native ConvFirst block fusion (Lavin, arXiv:2404.03617, Sec. 5.3).

Thin ctypes binding over ``libconvfirst.so`` (the gfx950 HIP kernels behind
the C ABI of ``include/convfirst.h``).  Every function here only marshals
arguments: torch supplies device memory and the current stream, the library
does all the arithmetic.  If the library is missing the import still works
but every call raises -- there is no fallback path.

Tensors are NHWC and contiguous: x [N, H, W, C] fp16/bf16 on the GPU.
Block parameters are a dict with dw_w [k,k,C], w1 [E*C,C], w2 [C,E*C] in the
I/O dtype and optional fp32 s0,b0 [C], s1,b1 [E*C], s2,b2 [C].
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "lib", "library_path", "block_forward", "block_autotune", "block_tuned_config", "stage_forward",
    "downsample_forward",
    "block_forward_unfused", "block_forward_split", "stack_forward", "capture_stack", "ConvFirstBlock",
    "CFError", "EXPORTED_SYMBOLS",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "_lib", "libconvfirst.so")

CF_OK, CF_ERR_INVALID, CF_ERR_UNSUPPORTED, CF_ERR_WORKSPACE, CF_ERR_HIP = range(5)
DTYPES = {torch.float16: 0, torch.bfloat16: 1}
ACTS = {"gelu": 0, "relu": 1, "none": 2}

EXPORTED_SYMBOLS = (
    "cf_block_forward", "cf_stage_forward", "cf_stage_workspace_bytes", "cf_downsample_forward",
    "cf_block_forward_unfused", "cf_unfused_workspace_bytes", "cf_block_forward_split",
    "cf_split_workspace_bytes", "cf_block_autotune", "cf_block_tuned_config", "cf_last_error",
    "cf_status_string", "cf_abi_version",
)


class CFError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class _BlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("dw_w", "dw_scale", "dw_bias", "w1", "s1", "b1", "w2", "s2", "b2")]


class _DownParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w", "scale", "bias")]


def library_path() -> str:
    return _LIB_PATH


_lib = None


def lib():
    """Load libconvfirst.so (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("libconvfirst.so is not built (%s); run "
                               "`python -m paper_2404_03617_amd.build`" % _LIB_PATH)
        L = ctypes.CDLL(_LIB_PATH)
        i, sz, vp = ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p
        bp, dp = ctypes.POINTER(_BlockParams), ctypes.POINTER(_DownParams)
        sig = {
            "cf_block_forward": (i, [vp, vp, bp, i, i, i, i, i, i, i, i, vp]),
            "cf_stage_forward": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_stage_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_downsample_forward": (i, [vp, vp, dp, i, i, i, i, i, i, vp]),
            "cf_block_forward_unfused": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, vp]),
            "cf_unfused_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_block_forward_split": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_split_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_block_autotune": (i, [vp, vp, bp, i, i, i, i, i, i, i, i, vp]),
            "cf_block_tuned_config": (i, [i, i, i, i, i, i, i, i]),
            "cf_last_error": (ctypes.c_char_p, []),
            "cf_status_string": (ctypes.c_char_p, [i]),
            "cf_abi_version": (i, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != CF_OK:
        L = lib()
        raise CFError(status, "%s: %s" % (L.cf_status_string(status).decode(),
                                          L.cf_last_error().decode()))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dims(x: torch.Tensor):
    if x.dim() != 4:
        raise ValueError("x must be [N, H, W, C]")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous NHWC")
    if x.dtype not in DTYPES:
        raise ValueError("x must be float16 or bfloat16")
    return tuple(int(v) for v in x.shape)


def _block_struct(p: dict, keep: list) -> _BlockParams:
    names = {"dw_w": "dw_w", "dw_scale": "s0", "dw_bias": "b0", "w1": "w1", "s1": "s1",
             "b1": "b1", "w2": "w2", "s2": "s2", "b2": "b2"}
    vals = {}
    for field, key in names.items():
        t = p.get(key)
        if t is not None:
            if not t.is_contiguous():
                raise ValueError("parameter %s must be contiguous" % key)
            keep.append(t)
        vals[field] = None if t is None else t.data_ptr()
    return _BlockParams(**vals)


def _block_shape(x, p):
    N, H, W, C = _dims(x)
    k = int(p["dw_w"].shape[0])
    EC = int(p["w1"].shape[0])
    if EC % C:
        raise ValueError("w1 rows must be a multiple of C")
    return N, H, W, C, EC // C, k


def block_forward(x: torch.Tensor, p: dict, act: str = "gelu", out: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """Fused ConvFirst block (one kernel launch): y = x + FFN(dwconv(x))."""
    N, H, W, C, E, k = _block_shape(x, p)
    y = torch.empty_like(x) if out is None else out
    keep = []
    bp = _block_struct(p, keep)
    _check(lib().cf_block_forward(_ptr(x), _ptr(y), ctypes.byref(bp), N, H, W, C, E, k,
                                  DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def block_autotune(x: torch.Tensor, p: dict, act: str = "gelu", out: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Time every kernel configuration that applies to this block shape, cache
    the fastest for later block_forward calls, return the block's output."""
    N, H, W, C, E, k = _block_shape(x, p)
    y = torch.empty_like(x) if out is None else out
    keep = []
    bp = _block_struct(p, keep)
    _check(lib().cf_block_autotune(_ptr(x), _ptr(y), ctypes.byref(bp), N, H, W, C, E, k,
                                   DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def block_tuned_config(x_shape, C: int, E: int, k: int, dtype=torch.float16, act: str = "gelu") -> int:
    """Cached configuration id for a block shape (0: default kernel and tiling)."""
    N, H, W = x_shape[0], x_shape[1], x_shape[2]
    return lib().cf_block_tuned_config(N, H, W, C, E, k, DTYPES[dtype], ACTS[act])


def stage_forward(x: torch.Tensor, blocks: list, act: str = "gelu", out=None, ws=None,
                  stream=None) -> torch.Tensor:
    """`len(blocks)` fused blocks of one shape, ping-ponging through ws."""
    N, H, W, C, E, k = _block_shape(x, blocks[0])
    y = torch.empty_like(x) if out is None else out
    L = lib()
    need = L.cf_stage_workspace_bytes(len(blocks), N, H, W, C, DTYPES[x.dtype])
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    keep = []
    arr = (_BlockParams * len(blocks))(*[_block_struct(b, keep) for b in blocks])
    _check(L.cf_stage_forward(_ptr(x), _ptr(y), _ptr(ws), 0 if ws is None else ws.numel(),
                              arr, len(blocks), N, H, W, C, E, k, DTYPES[x.dtype], ACTS[act],
                              _stream(stream)))
    return y


def downsample_forward(x: torch.Tensor, p: dict, out=None, stream=None) -> torch.Tensor:
    """2x2 stride-2 conv: p has wd [Cout,2,2,Cin] and optional fp32 sd, bd [Cout]."""
    N, H, W, Cin = _dims(x)
    Cout = int(p["wd"].shape[0])
    y = out if out is not None else torch.empty((N, H // 2, W // 2, Cout), dtype=x.dtype,
                                                device=x.device)
    dp = _DownParams(w=p["wd"].data_ptr(),
                     scale=None if p.get("sd") is None else p["sd"].data_ptr(),
                     bias=None if p.get("bd") is None else p["bd"].data_ptr())
    _check(lib().cf_downsample_forward(_ptr(x), _ptr(y), ctypes.byref(dp), N, H, W, Cin, Cout,
                                       DTYPES[x.dtype], _stream(stream)))
    return y


def block_forward_unfused(x: torch.Tensor, p: dict, act: str = "gelu", out=None, ws=None,
                          stream=None) -> torch.Tensor:
    """Layer-by-layer block: depth-wise, expand GEMM, project GEMM (3 launches)."""
    N, H, W, C, E, k = _block_shape(x, p)
    y = torch.empty_like(x) if out is None else out
    L = lib()
    need = L.cf_unfused_workspace_bytes(N, H, W, C, E, DTYPES[x.dtype])
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    keep = []
    bp = _block_struct(p, keep)
    _check(L.cf_block_forward_unfused(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(bp),
                                      N, H, W, C, E, k, DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def split_workspace_bytes(x_shape, C: int, E: int, groups: int = 0) -> int:
    N, H, W = x_shape[:3]
    return lib().cf_split_workspace_bytes(N, H, W, C, E, groups)


def block_forward_split(x: torch.Tensor, p: dict, act: str = "gelu", groups: int = 0, out=None,
                        ws=None, stream=None) -> torch.Tensor:
    """Fused block with hidden channels split over `groups` workgroups per tile."""
    N, H, W, C, E, k = _block_shape(x, p)
    y = torch.empty_like(x) if out is None else out
    L = lib()
    need = L.cf_split_workspace_bytes(N, H, W, C, E, groups)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    keep = []
    bp = _block_struct(p, keep)
    _check(L.cf_block_forward_split(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(bp),
                                    N, H, W, C, E, k, groups, DTYPES[x.dtype], ACTS[act],
                                    _stream(stream)))
    return y


def stack_forward(x: torch.Tensor, layers: list, act: str = "gelu", stream=None,
                  bufs: list | None = None) -> torch.Tensor:
    """Run [("block", p) | ("down", p), ...] in order.  Consecutive blocks of one
    shape go through stage_forward; `bufs` may hold preallocated outputs, one per
    stage/down-sampling step, to keep the sequence allocation-free."""
    y = x
    i = 0
    step = 0
    while i < len(layers):
        kind, p = layers[i]
        out = None if bufs is None else bufs[step]
        if kind == "down":
            y = downsample_forward(y, p, out=out, stream=stream)
            i += 1
        else:
            j = i
            while j < len(layers) and layers[j][0] == "block":
                j += 1
            y = stage_forward(y, [q for _, q in layers[i:j]], act=act, out=out, stream=stream)
            i = j
        step += 1
    return y


def capture_stack(x: torch.Tensor, layers: list, bufs: list, act: str = "gelu") -> "torch.cuda.CUDAGraph":
    """Record the launches of stack_forward(x, layers, bufs=bufs) -- one per
    fused stage and per down-sampling step -- into one HIP graph.  A replay
    reruns them on the contents x and bufs have at that time (write the next
    input into x in place); the result is bufs[-1].  The stage workspaces come
    from the graph's private memory pool during capture, so a replay allocates
    nothing.  x, bufs and the layer weights must outlive the graph."""
    stack_forward(x, layers, act=act, bufs=bufs)  # library loaded, device attributes cached
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        stack_forward(x, layers, act=act, bufs=bufs)
    return g


class ConvFirstBlock(torch.nn.Module):
    """nn.Module wrapper around the fused kernel (inference only).

    Holds the block's weights as buffers in the ABI layouts; ``forward`` takes
    and returns contiguous NHWC tensors."""

    def __init__(self, params: dict, act: str = "gelu"):
        super().__init__()
        self.act = act
        self._keys = [k for k, v in params.items() if v is not None]
        for k in self._keys:
            self.register_buffer(k, params[k])

    def params(self) -> dict:
        return {k: getattr(self, k) for k in self._keys}

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return block_forward(x, self.params(), act=self.act)
