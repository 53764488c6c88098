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

from .convert import (block_params_from_modules, down_params_from_modules, down_weight_from_conv2d,
                      dw_weight_from_conv2d, fold_batchnorm, grouped_block_params_from_modules,
                      grouped_weight_from_conv2d, pw_weight_from_conv2d, stem_params_from_modules)

__all__ = [
    "lib", "library_path", "block_forward", "block_autotune", "block_tuned_config", "stage_forward",
    "stage_forward_microbatch",
    "downsample_forward",
    "block_forward_unfused", "block_forward_split", "block_forward_split_noalloc", "gblock_forward",
    "convfirst_s2_forward",
    "mbconv_forward", "mbconv_workspace_bytes", "mbconv_s2_forward", "mbconv_s2_workspace_bytes", "stem_forward",
    "stem_gblock_forward", "stack_forward", "capture_stack", "ConvFirstBlock",
    "CFError", "EXPORTED_SYMBOLS", "dw_weight_from_conv2d", "grouped_weight_from_conv2d",
    "pw_weight_from_conv2d", "down_weight_from_conv2d", "fold_batchnorm", "block_params_from_modules",
    "grouped_block_params_from_modules", "down_params_from_modules", "stem_params_from_modules",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "_lib", "libconvfirst.so")

CF_OK, CF_ERR_INVALID, CF_ERR_UNSUPPORTED, CF_ERR_WORKSPACE, CF_ERR_HIP = range(5)
DTYPES = {torch.float16: 0, torch.bfloat16: 1}
ACTS = {"gelu": 0, "relu": 1, "none": 2}

EXPORTED_SYMBOLS = (
    "cf_block_forward", "cf_stage_forward", "cf_stage_workspace_bytes", "cf_stage_forward_microbatch",
    "cf_stage_microbatch_workspace_bytes", "cf_downsample_forward",
    "cf_block_forward_unfused", "cf_unfused_workspace_bytes", "cf_block_forward_split",
    "cf_split_workspace_bytes", "cf_block_forward_split_noalloc", "cf_gblock_forward", "cf_convfirst_s2_forward",
    "cf_mbconv_forward",
    "cf_mbconv_workspace_bytes", "cf_mbconv_s2_forward", "cf_mbconv_s2_workspace_bytes", "cf_stem_forward",
    "cf_stem_gblock_forward", "cf_block_autotune",
    "cf_block_tuned_config", "cf_last_error", "cf_status_string", "cf_abi_version",
)


class CFError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class _BlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("dw_w", "dw_scale", "dw_bias", "w1", "s1", "b1", "w2", "s2", "b2")]


class _GBlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("gw_w", "gw_scale", "gw_bias", "w1", "s1", "b1", "w2", "s2", "b2")]


class _StemParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w", "scale", "bias")]


class _MBConvParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w1", "s1", "b1", "gw_w", "s2", "b2", "wr", "br", "we", "be", "w2", "s3", "b3")]


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
        gp = ctypes.POINTER(_GBlockParams)
        mp = ctypes.POINTER(_MBConvParams)
        sp = ctypes.POINTER(_StemParams)
        sig = {
            "cf_block_forward": (i, [vp, vp, bp, i, i, i, i, i, i, i, i, vp]),
            "cf_stage_forward": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_stage_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_stage_forward_microbatch": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, i, i, vp]),
            "cf_stage_microbatch_workspace_bytes": (sz, [i, i, i, i, i, i, i]),
            "cf_downsample_forward": (i, [vp, vp, dp, i, i, i, i, i, i, vp]),
            "cf_block_forward_unfused": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, vp]),
            "cf_unfused_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_block_forward_split": (i, [vp, vp, vp, sz, bp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_split_workspace_bytes": (sz, [i, i, i, i, i, i]),
            "cf_block_forward_split_noalloc": (i, [vp, vp, bp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_gblock_forward": (i, [vp, vp, gp, i, i, i, i, i, i, i, i, vp]),
            "cf_convfirst_s2_forward": (i, [vp, vp, gp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_mbconv_forward": (i, [vp, vp, vp, sz, mp, i, i, i, i, i, i, i, i, i, vp]),
            "cf_mbconv_workspace_bytes": (sz, [i, i, i, i, i, i, i]),
            "cf_mbconv_s2_forward": (i, [vp, vp, vp, sz, mp, i, i, i, i, i, i, i, i, i, i, vp]),
            "cf_mbconv_s2_workspace_bytes": (sz, [i, i, i, i, i, i, i, i]),
            "cf_stem_forward": (i, [vp, vp, sp, i, i, i, i, i, vp]),
            "cf_stem_gblock_forward": (i, [vp, vp, sp, gp, i, i, i, i, i, i, i, i, vp]),
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
    if not isinstance(x, torch.Tensor):
        raise TypeError("x must be a torch.Tensor")
    if x.dim() != 4:
        raise ValueError("x must be [N, H, W, C]")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous NHWC")
    if x.dtype not in DTYPES:
        raise ValueError("x must be float16 or bfloat16")
    return tuple(int(v) for v in x.shape)


def _check_tensor(name: str, t, shape, dtype, device: torch.device):
    """Shape, dtype, layout and device of one argument, checked before any
    pointer reaches the library (the C ABI cannot check sizes or address
    spaces)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.device != device:
        raise ValueError("%s is on %s but x is on %s" % (name, t.device, device))


def _check_device(x: torch.Tensor):
    if x.device.type != "cuda":
        raise ValueError("x must be a GPU tensor (got device %s)" % x.device)


# parameter key -> (shape as a function of C, E*C, k; kind): kind "w" is in
# x's dtype, "v" is fp32
_BLOCK_SHAPES = {
    "dw_w": (lambda C, EC, k: (k, k, C), "w"),
    "s0": (lambda C, EC, k: (C,), "v"), "b0": (lambda C, EC, k: (C,), "v"),
    "w1": (lambda C, EC, k: (EC, C), "w"),
    "s1": (lambda C, EC, k: (EC,), "v"), "b1": (lambda C, EC, k: (EC,), "v"),
    "w2": (lambda C, EC, k: (C, EC), "w"),
    "s2": (lambda C, EC, k: (C,), "v"), "b2": (lambda C, EC, k: (C,), "v"),
}
_FIELDS = {"dw_w": "dw_w", "s0": "dw_scale", "b0": "dw_bias", "w1": "w1", "s1": "s1",
           "b1": "b1", "w2": "w2", "s2": "s2", "b2": "b2"}


def _block_shape(x, p):
    N, H, W, C = _dims(x)
    for key in ("dw_w", "w1", "w2"):
        if not isinstance(p.get(key), torch.Tensor):
            raise ValueError("block parameter %s is required" % key)
    if p["dw_w"].dim() != 3 or p["w1"].dim() != 2:
        raise ValueError("dw_w must be [k, k, C] and w1 [E*C, C]")
    k = int(p["dw_w"].shape[0])
    EC = int(p["w1"].shape[0])
    if EC % C or EC == 0:
        raise ValueError("w1 rows must be a positive multiple of C")
    return N, H, W, C, EC // C, k


def _block_struct(x: torch.Tensor, p: dict, keep: list) -> _BlockParams:
    """Validate every block parameter against x, then build the ABI struct."""
    N, H, W, C, E, k = _block_shape(x, p)
    unknown = set(p) - set(_BLOCK_SHAPES)
    if unknown:
        raise ValueError("unknown block parameters: %s" % sorted(unknown))
    vals = {}
    for key, (shape_of, kind) in _BLOCK_SHAPES.items():
        t = p.get(key)
        if t is not None:
            _check_tensor(key, t, shape_of(C, E * C, k), x.dtype if kind == "w" else torch.float32,
                          x.device)
            keep.append(t)
        vals[_FIELDS[key]] = None if t is None else t.data_ptr()
    return _BlockParams(**vals)


def _out(x: torch.Tensor, out, shape=None):
    shape = tuple(x.shape) if shape is None else tuple(shape)
    if out is None:
        return torch.empty(shape, dtype=x.dtype, device=x.device)
    _check_tensor("out", out, shape, x.dtype, x.device)
    return out


def _workspace(x: torch.Tensor, ws, need: int):
    """The caller's workspace (uint8, on x's device, at least `need` bytes) or a
    fresh one."""
    if ws is None:
        return torch.empty(need, dtype=torch.uint8, device=x.device) if need else None
    if not isinstance(ws, torch.Tensor) or ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous uint8 tensor")
    if ws.device != x.device:
        raise ValueError("ws is on %s but x is on %s" % (ws.device, x.device))
    if ws.numel() < need:
        raise ValueError("ws has %d bytes, needs %d" % (ws.numel(), need))
    return ws


def _prepare_block(x: torch.Tensor, p: dict, act: str, out):
    """Every check of a block call, in an order that needs no GPU: shapes and
    dtypes first, then devices.  Returns (y, struct, keep, dims)."""
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    keep = []
    bp = _block_struct(x, p, keep)
    _check_device(x)
    y = _out(x, out)
    return y, bp, keep, _block_shape(x, p)


def block_forward(x: torch.Tensor, p: dict, act: str = "gelu", out: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """Fused ConvFirst block (one kernel launch): y = x + FFN(dwconv(x))."""
    y, bp, keep, (N, H, W, C, E, k) = _prepare_block(x, p, act, out)
    _check(lib().cf_block_forward(_ptr(x), _ptr(y), ctypes.byref(bp), N, H, W, C, E, k,
                                  DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def block_autotune(x: torch.Tensor, p: dict, act: str = "gelu", out: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Time every kernel configuration that applies to this block shape, cache
    the fastest for later block_forward calls, return the block's output."""
    y, bp, keep, (N, H, W, C, E, k) = _prepare_block(x, p, act, out)
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
    if not blocks:
        raise ValueError("a stage needs at least one block")
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    keep = []
    structs = [_block_struct(x, b, keep) for b in blocks]
    dims = {_block_shape(x, b) for b in blocks}
    if len(dims) != 1:
        raise ValueError("every block of a stage must have the same shape")
    N, H, W, C, E, k = dims.pop()
    _check_device(x)
    y = _out(x, out)
    L = lib()
    need = L.cf_stage_workspace_bytes(len(blocks), N, H, W, C, DTYPES[x.dtype])
    ws = _workspace(x, ws, need)
    arr = (_BlockParams * len(blocks))(*structs)
    _check(L.cf_stage_forward(_ptr(x), _ptr(y), _ptr(ws), 0 if ws is None else ws.numel(),
                              arr, len(blocks), N, H, W, C, E, k, DTYPES[x.dtype], ACTS[act],
                              _stream(stream)))
    return y


def stage_forward_microbatch(x: torch.Tensor, blocks: list, act: str = "gelu", micro_batch: int = 0,
                             out=None, ws=None, stream=None) -> torch.Tensor:
    """The stage with the micro-batch schedule (Sec. 5.5.2): all blocks over
    `micro_batch` images at a time, so the intermediate activations of a
    micro-batch can stay in the caches between blocks (0: default size)."""
    if not blocks:
        raise ValueError("a stage needs at least one block")
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    keep = []
    structs = [_block_struct(x, b, keep) for b in blocks]
    dims = {_block_shape(x, b) for b in blocks}
    if len(dims) != 1:
        raise ValueError("every block of a stage must have the same shape")
    N, H, W, C, E, k = dims.pop()
    _check_device(x)
    y = _out(x, out)
    L = lib()
    need = L.cf_stage_microbatch_workspace_bytes(len(blocks), N, H, W, C, micro_batch, DTYPES[x.dtype])
    ws = _workspace(x, ws, need)
    arr = (_BlockParams * len(blocks))(*structs)
    _check(L.cf_stage_forward_microbatch(_ptr(x), _ptr(y), _ptr(ws), 0 if ws is None else ws.numel(), arr,
                                         len(blocks), N, H, W, C, E, k, micro_batch, DTYPES[x.dtype], ACTS[act],
                                         _stream(stream)))
    return y


def downsample_forward(x: torch.Tensor, p: dict, out=None, stream=None) -> torch.Tensor:
    """2x2 stride-2 conv: p has wd [Cout,2,2,Cin] and optional fp32 sd, bd [Cout]."""
    N, H, W, Cin = _dims(x)
    wd = p.get("wd")
    if not isinstance(wd, torch.Tensor) or wd.dim() != 4:
        raise ValueError("downsample parameter wd [Cout, 2, 2, Cin] is required")
    Cout = int(wd.shape[0])
    _check_tensor("wd", wd, (Cout, 2, 2, Cin), x.dtype, x.device)
    for key in ("sd", "bd"):
        if p.get(key) is not None:
            _check_tensor(key, p[key], (Cout,), torch.float32, x.device)
    _check_device(x)
    y = _out(x, out, (N, H // 2, W // 2, Cout))
    dp = _DownParams(w=wd.data_ptr(),
                     scale=None if p.get("sd") is None else p["sd"].data_ptr(),
                     bias=None if p.get("bd") is None else p["bd"].data_ptr())
    _check(lib().cf_downsample_forward(_ptr(x), _ptr(y), ctypes.byref(dp), N, H, W, Cin, Cout,
                                       DTYPES[x.dtype], _stream(stream)))
    return y


def block_forward_unfused(x: torch.Tensor, p: dict, act: str = "gelu", out=None, ws=None,
                          stream=None) -> torch.Tensor:
    """Layer-by-layer block: depth-wise, expand GEMM, project GEMM (3 launches)."""
    y, bp, keep, (N, H, W, C, E, k) = _prepare_block(x, p, act, out)
    L = lib()
    ws = _workspace(x, ws, L.cf_unfused_workspace_bytes(N, H, W, C, E, DTYPES[x.dtype]))
    _check(L.cf_block_forward_unfused(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(bp),
                                      N, H, W, C, E, k, DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def split_workspace_bytes(x_shape, C: int, E: int, groups: int = 0) -> int:
    N, H, W = x_shape[:3]
    return lib().cf_split_workspace_bytes(N, H, W, C, E, groups)


def block_forward_split(x: torch.Tensor, p: dict, act: str = "gelu", groups: int = 0, out=None,
                        ws=None, stream=None) -> torch.Tensor:
    """Fused block with hidden channels split over `groups` workgroups per tile."""
    y, bp, keep, (N, H, W, C, E, k) = _prepare_block(x, p, act, out)
    L = lib()
    ws = _workspace(x, ws, L.cf_split_workspace_bytes(N, H, W, C, E, groups))
    _check(L.cf_block_forward_split(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(bp),
                                    N, H, W, C, E, k, groups, DTYPES[x.dtype], ACTS[act],
                                    _stream(stream)))
    return y


GROUP_WIDTH = 8
_GBLOCK_SHAPES = dict(_BLOCK_SHAPES)
del _GBLOCK_SHAPES["dw_w"]
_GBLOCK_SHAPES["gw_w"] = (lambda C, EC, k: (k, k, C, GROUP_WIDTH), "w")
_GFIELDS = dict(_FIELDS, gw_w="gw_w", s0="gw_scale", b0="gw_bias")
del _GFIELDS["dw_w"]


def gblock_forward(x: torch.Tensor, p: dict, act: str = "relu", out=None, stream=None) -> torch.Tensor:
    """The paper's ConvFirst block (Sec. 5.3) fused: a k x k grouped conv of
    group width 8, then the FFN and the residual.  p holds gw_w [k,k,C,8],
    w1 [E*C,C], w2 [C,E*C] in x's dtype and optional fp32 s0,b0 [C],
    s1,b1 [E*C], s2,b2 [C].  ReLU is the paper's activation."""
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    N, H, W, C = _dims(x)
    for key in ("gw_w", "w1", "w2"):
        if not isinstance(p.get(key), torch.Tensor):
            raise ValueError("grouped-block parameter %s is required" % key)
    if p["gw_w"].dim() != 4 or p["w1"].dim() != 2:
        raise ValueError("gw_w must be [k, k, C, 8] and w1 [E*C, C]")
    k, EC = int(p["gw_w"].shape[0]), int(p["w1"].shape[0])
    if EC % C or EC == 0:
        raise ValueError("w1 rows must be a positive multiple of C")
    unknown = set(p) - set(_GBLOCK_SHAPES)
    if unknown:
        raise ValueError("unknown grouped-block parameters: %s" % sorted(unknown))
    vals, keep = {}, []
    for key, (shape_of, kind) in _GBLOCK_SHAPES.items():
        t = p.get(key)
        if t is not None:
            _check_tensor(key, t, shape_of(C, EC, k), x.dtype if kind == "w" else torch.float32, x.device)
            keep.append(t)
        vals[_GFIELDS[key]] = None if t is None else t.data_ptr()
    gp = _GBlockParams(**vals)
    _check_device(x)
    y = _out(x, out)
    _check(lib().cf_gblock_forward(_ptr(x), _ptr(y), ctypes.byref(gp), N, H, W, C, EC // C, k,
                                   DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


# stride-2 ConvFirst parameters: shape as a function of (C, R, K)
_CFS2_SHAPES = {
    "gw_w": (lambda C, R, K: (3, 3, C, GROUP_WIDTH), "w"),
    "w1": (lambda C, R, K: (R, 2 * C), "w"),
    "w2": (lambda C, R, K: (K, R), "w"),
    "s0": (lambda C, R, K: (C,), "v"), "b0": (lambda C, R, K: (C,), "v"),
    "s1": (lambda C, R, K: (R,), "v"), "b1": (lambda C, R, K: (R,), "v"),
    "s2": (lambda C, R, K: (K,), "v"), "b2": (lambda C, R, K: (K,), "v"),
}


def convfirst_s2_forward(x: torch.Tensor, p: dict, act: str = "relu", out=None, stream=None) -> torch.Tensor:
    """The stride-2 ConvFirst block (Fig. f:convfirst-block (c)) in one
    kernel, in the reading the speed-projection tables fix (App. A): grouped
    3x3 conv C -> C with s0, b0 at the input size, BlurPool (Triangle-3,
    reflect) of the conv output and of x, the two concatenated (2C channels,
    conv output first), expand to R with s1, b1 and the activation, project
    to K with s2, b2, no residual.  p holds gw_w [3,3,C,8], w1 [R,2C], w2
    [K,R] in x's dtype and optional fp32 s0,b0 [C], s1,b1 [R], s2,b2 [K].
    Returns [N, ceil(H/2), ceil(W/2), K]; out must not overlap x."""
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    N, H, W, C = _dims(x)
    for key in ("gw_w", "w1", "w2"):
        if not isinstance(p.get(key), torch.Tensor):
            raise ValueError("stride-2 ConvFirst parameter %s is required" % key)
    if p["gw_w"].dim() != 4 or p["w1"].dim() != 2 or p["w2"].dim() != 2:
        raise ValueError("gw_w must be [3, 3, C, 8], w1 [R, 2C] and w2 [K, R]")
    k, R, K = int(p["gw_w"].shape[0]), int(p["w1"].shape[0]), int(p["w2"].shape[0])
    unknown = set(p) - set(_CFS2_SHAPES)
    if unknown:
        raise ValueError("unknown stride-2 ConvFirst parameters: %s" % sorted(unknown))
    vals, keep = {}, []
    for key, (shape_of, kind) in _CFS2_SHAPES.items():
        t = p.get(key)
        if t is not None:
            shape = shape_of(C, R, K)
            if key == "gw_w":
                shape = (k, k, C, GROUP_WIDTH)
            _check_tensor(key, t, shape, x.dtype if kind == "w" else torch.float32, x.device)
            keep.append(t)
        vals[_GFIELDS[key]] = None if t is None else t.data_ptr()
    gp = _GBlockParams(**vals)
    _check_device(x)
    y = _out(x, out, (N, (H + 1) // 2, (W + 1) // 2, K))
    _check(lib().cf_convfirst_s2_forward(_ptr(x), _ptr(y), ctypes.byref(gp), N, H, W, C, R, K, k,
                                         DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


def _stem_struct(x: torch.Tensor, stem: dict, C: int):
    """The checked stem parameters (sw [C,3,3,3] in x's dtype, ss, sb fp32 [C])."""
    if not isinstance(stem.get("sw"), torch.Tensor):
        raise ValueError("stem parameter sw is required")
    unknown = set(stem) - {"sw", "ss", "sb"}
    if unknown:
        raise ValueError("unknown stem parameters: %s" % sorted(unknown))
    _check_tensor("sw", stem["sw"], (C, 3, 3, 3), x.dtype, x.device)
    for key in ("ss", "sb"):
        if stem.get(key) is not None:
            _check_tensor(key, stem[key], (C,), torch.float32, x.device)
    return _StemParams(w=stem["sw"].data_ptr(), scale=_ptr_val(stem.get("ss")), bias=_ptr_val(stem.get("sb")))


def _ptr_val(t):
    return None if t is None else t.data_ptr()


def _image_dims(x: torch.Tensor):
    N, H, W, C = _dims(x)
    if C != 3:
        raise ValueError("the stem's input must be an image [N, H, W, 3]")
    return N, H, W


def stem_forward(x: torch.Tensor, stem: dict, out=None, stream=None) -> torch.Tensor:
    """The network stem (App. A): 3x3 stride-2 conv of the image x [N,H,W,3]
    to C = 16 or 32 channels, folded norm, ReLU; stem holds sw [C,3,3,3] and
    optional fp32 ss, sb [C].  Returns [N, ceil(H/2), ceil(W/2), C]."""
    N, H, W = _image_dims(x)
    if not isinstance(stem.get("sw"), torch.Tensor) or stem["sw"].dim() != 4:
        raise ValueError("stem parameter sw [C, 3, 3, 3] is required")
    C = int(stem["sw"].shape[0])
    sp = _stem_struct(x, stem, C)
    _check_device(x)
    y = _out(x, out, (N, (H + 1) // 2, (W + 1) // 2, C))
    _check(lib().cf_stem_forward(_ptr(x), _ptr(y), ctypes.byref(sp), N, H, W, C, DTYPES[x.dtype], _stream(stream)))
    return y


def stem_gblock_forward(x: torch.Tensor, stem: dict, p: dict, act: str = "relu", out=None,
                        stream=None) -> torch.Tensor:
    """The stem fused into the first ConvFirst block (App. A): one kernel
    computing gblock_forward(stem_forward(x)); p as for gblock_forward with
    C = 16 or 32."""
    if act not in ACTS:
        raise ValueError("act must be one of %s" % sorted(ACTS))
    N, H, W = _image_dims(x)
    if not isinstance(stem.get("sw"), torch.Tensor) or stem["sw"].dim() != 4:
        raise ValueError("stem parameter sw [C, 3, 3, 3] is required")
    C = int(stem["sw"].shape[0])
    sp = _stem_struct(x, stem, C)
    for key in ("gw_w", "w1", "w2"):
        if not isinstance(p.get(key), torch.Tensor):
            raise ValueError("grouped-block parameter %s is required" % key)
    if p["gw_w"].dim() != 4 or p["w1"].dim() != 2:
        raise ValueError("gw_w must be [k, k, C, 8] and w1 [E*C, C]")
    k, EC = int(p["gw_w"].shape[0]), int(p["w1"].shape[0])
    if EC % C or EC == 0:
        raise ValueError("w1 rows must be a positive multiple of C")
    unknown = set(p) - set(_GBLOCK_SHAPES)
    if unknown:
        raise ValueError("unknown grouped-block parameters: %s" % sorted(unknown))
    vals = {}
    for key, (shape_of, kind) in _GBLOCK_SHAPES.items():
        t = p.get(key)
        if t is not None:
            _check_tensor(key, t, shape_of(C, EC, k), x.dtype if kind == "w" else torch.float32, x.device)
        vals[_GFIELDS[key]] = _ptr_val(t)
    gp = _GBlockParams(**vals)
    _check_device(x)
    y = _out(x, out, (N, (H + 1) // 2, (W + 1) // 2, C))
    _check(lib().cf_stem_gblock_forward(_ptr(x), _ptr(y), ctypes.byref(sp), ctypes.byref(gp), N, H, W, C, EC // C, k,
                                        DTYPES[x.dtype], ACTS[act], _stream(stream)))
    return y


# MBConv parameters: shape as a function of (C, E*C, R, K) with K the output
# channels (C for stride 1), and whether the tensor is a weight in x's dtype
# ("w") or an fp32 vector ("v").
_MBCONV_SHAPES = {
    "w1": (lambda C, EC, R, K: (EC, C), "w"),
    "gw_w": (lambda C, EC, R, K: (3, 3, EC, GROUP_WIDTH), "w"),
    "wr": (lambda C, EC, R, K: (R, EC), "w"),
    "we": (lambda C, EC, R, K: (EC, R), "w"),
    "w2": (lambda C, EC, R, K: (K, EC), "w"),
    "s1": (lambda C, EC, R, K: (EC,), "v"), "b1": (lambda C, EC, R, K: (EC,), "v"),
    "s2": (lambda C, EC, R, K: (EC,), "v"), "b2": (lambda C, EC, R, K: (EC,), "v"),
    "br": (lambda C, EC, R, K: (R,), "v"), "be": (lambda C, EC, R, K: (EC,), "v"),
    "s3": (lambda C, EC, R, K: (K,), "v"), "b3": (lambda C, EC, R, K: (K,), "v"),
}


def mbconv_workspace_bytes(N: int, H: int, W: int, C: int, E: int, R: int, dtype=torch.float16) -> int:
    """Recommended workspace of mbconv_forward on the current device (0 for a
    shape without a kernel)."""
    return int(lib().cf_mbconv_workspace_bytes(N, H, W, C, E, R, DTYPES[dtype]))


def mbconv_s2_workspace_bytes(N: int, H: int, W: int, C: int, E: int, R: int, K: int,
                              dtype=torch.float16) -> int:
    """Recommended workspace of mbconv_s2_forward on the current device (0 for
    a shape without a kernel)."""
    return int(lib().cf_mbconv_s2_workspace_bytes(N, H, W, C, E, R, K, DTYPES[dtype]))


LAUNCHES = {"cooperative": 0, "exclusive": 1}


def _mbconv_args(x: torch.Tensor, p: dict, launch: str, stride2: bool):
    """Checks an MBConv call's tensors; returns the sizes, the C struct of
    pointers and the tensors it points into (kept alive by the caller)."""
    if launch not in LAUNCHES:
        raise ValueError("launch must be one of %s" % sorted(LAUNCHES))
    N, H, W, C = _dims(x)
    for key in ("w1", "gw_w", "wr", "we", "w2"):
        if not isinstance(p.get(key), torch.Tensor):
            raise ValueError("MBConv parameter %s is required" % key)
    if p["w1"].dim() != 2 or p["wr"].dim() != 2 or p["w2"].dim() != 2:
        raise ValueError("w1 must be [E*C, C], wr [R, E*C] and w2 [K, E*C]")
    EC, R = int(p["w1"].shape[0]), int(p["wr"].shape[0])
    K = int(p["w2"].shape[0]) if stride2 else C
    if EC % C or EC == 0:
        raise ValueError("w1 rows must be a positive multiple of C")
    if p["gw_w"].dim() != 4 or p["gw_w"].shape[0] != p["gw_w"].shape[1]:
        raise ValueError("gw_w must be [k, k, E*C, 8]")
    k = int(p["gw_w"].shape[0])
    unknown = set(p) - set(_MBCONV_SHAPES)
    if unknown:
        raise ValueError("unknown MBConv parameters: %s" % sorted(unknown))
    vals, keep = {}, []
    for key, (shape_of, kind) in _MBCONV_SHAPES.items():
        t = p.get(key)
        if t is not None:
            shape = shape_of(C, EC, R, K)
            if key == "gw_w":
                shape = (k, k, EC, GROUP_WIDTH)
            _check_tensor(key, t, shape, x.dtype if kind == "w" else torch.float32, x.device)
            keep.append(t)
        vals[key] = None if t is None else t.data_ptr()
    _check_device(x)
    return (N, H, W, C, EC // C, R, K, k), _MBConvParams(**vals), keep


def mbconv_forward(x: torch.Tensor, p: dict, out=None, ws=None, launch: str = "cooperative",
                   stream=None) -> torch.Tensor:
    """The paper's MBConv block with Squeeze & Excitation (Sec. 5.4) fused
    into one cooperative kernel (Sec. 5.4.1).  p holds w1 [E*C,C], gw_w
    [3,3,E*C,8], wr [R,E*C], we [E*C,R], w2 [C,E*C] in x's dtype and optional
    fp32 s1,b1,s2,b2,be [E*C], br [R], s3,b3 [C].  out may be x itself
    (evaluation in place).  ws: a uint8 workspace, by default a zeroed one of
    mbconv_workspace_bytes(); a smaller one runs fewer images at a time.  A
    caller's ws must be zeroed before its first use (every call leaves it
    reusable); its first int32 becomes 1 if a barrier wait ever gave up.
    launch="exclusive" replaces the cooperative launch by an ordinary one,
    for callers that own the device (see the C header)."""
    (N, H, W, C, E, R, _, k), mp, keep = _mbconv_args(x, p, launch, False)
    y = _out(x, out)
    if ws is None:
        ws = torch.zeros(max(1, mbconv_workspace_bytes(N, H, W, C, E, R, x.dtype)), dtype=torch.uint8,
                         device=x.device)
    else:
        _workspace(x, ws, 0)
    _check(lib().cf_mbconv_forward(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(mp), N, H, W, C, E,
                                   R, k, DTYPES[x.dtype], LAUNCHES[launch], _stream(stream)))
    return y


def mbconv_s2_forward(x: torch.Tensor, p: dict, out=None, ws=None, launch: str = "cooperative",
                      stream=None) -> torch.Tensor:
    """The stride-2 MBConv block (Fig. f:mbconv with stride 2; Sec. 5.4): as
    mbconv_forward, then BlurPool with the Triangle-3 filter (reflect padding,
    stride 2) on the conv output, the squeeze over the down-sampled map, the
    project to K channels and no residual, in one launch.  p as for
    mbconv_forward except w2 [K,E*C] and s3,b3 [K]; the result is
    [N, ceil(H/2), ceil(W/2), K] and must not overlap x.  ws as for
    mbconv_forward, sized by mbconv_s2_workspace_bytes()."""
    (N, H, W, C, E, R, K, k), mp, keep = _mbconv_args(x, p, launch, True)
    y = _out(x, out, (N, (H + 1) // 2, (W + 1) // 2, K))
    if ws is None:
        ws = torch.zeros(max(1, mbconv_s2_workspace_bytes(N, H, W, C, E, R, K, x.dtype)), dtype=torch.uint8,
                         device=x.device)
    else:
        _workspace(x, ws, 0)
    _check(lib().cf_mbconv_s2_forward(_ptr(x), _ptr(y), _ptr(ws), ws.numel(), ctypes.byref(mp), N, H, W, C, E,
                                      R, K, k, DTYPES[x.dtype], LAUNCHES[launch], _stream(stream)))
    return y


def block_forward_split_noalloc(x: torch.Tensor, p: dict, act: str = "gelu", groups: int = 0, out=None,
                                stream=None) -> torch.Tensor:
    """block_forward_split without a workspace: the library keeps the fp32
    partials in a static device array (16 MiB per GPU), so with `out` given the
    call allocates nothing.  Calls that overlap on one GPU race (see the C
    header)."""
    y, bp, keep, (N, H, W, C, E, k) = _prepare_block(x, p, act, out)
    _check(lib().cf_block_forward_split_noalloc(_ptr(x), _ptr(y), ctypes.byref(bp), N, H, W, C, E, k, groups,
                                                DTYPES[x.dtype], ACTS[act], _stream(stream)))
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
        elif kind == "block":
            j = i
            while j < len(layers) and layers[j][0] == "block":
                j += 1
            y = stage_forward(y, [q for _, q in layers[i:j]], act=act, out=out, stream=stream)
            i = j
        else:
            raise ValueError("unknown layer kind %r" % (kind,))
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

    @classmethod
    def from_modules(cls, dw, bn0, pw1, bn1, pw2, bn2, act: str = "gelu", dtype=torch.float16):
        """Build from torch layers (depth-wise nn.Conv2d, 1x1 convs or Linears,
        inference-mode BatchNorm2d or None), folding each batch norm."""
        return cls(block_params_from_modules(dw, bn0, pw1, bn1, pw2, bn2, dtype), act=act)

    def params(self) -> dict:
        return {k: getattr(self, k) for k in self._keys}

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return block_forward(x, self.params(), act=self.act)
