"""Plain fp64 CPU oracle for the ConvFirst residual block.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this package; the product library never does.
It shares no code with the GPU library.  Arrays in, arrays out, all float64
numpy; callers widen their fp16/bf16 tensors exactly before calling.

Each function below states the passage of Lavin, "On the Efficiency of
Convolutional Neural Networks" (arXiv:2404.03617) that it implements; the
arithmetic itself lives in ``cfref.c`` next to this file.

Activation names: "gelu" (exact erf form), "relu", "none" (identity).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cfref.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ACTS = {"gelu": 0, "relu": 1, "none": 2}

_dp = ctypes.POINTER(ctypes.c_double)


def build(force: bool = True) -> str:
    """Compile cfref.c with gcc -O2 (no fast-math) into liboracle.so."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-D_POSIX_C_SOURCE=200809L", "-fPIC",
                               "-shared", "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        i64 = ctypes.c_int64
        ci = ctypes.c_int
        L.cfref_act.restype = ctypes.c_double
        L.cfref_act.argtypes = [ctypes.c_double, ci]
        L.cfref_depthwise.argtypes = [_dp, _dp, _dp, _dp, ci, ci, ci, ci, ci, _dp, ci]
        L.cfref_pointwise.argtypes = [_dp, _dp, _dp, _dp, i64, ci, ci, _dp, ci]
        blk = [_dp] * 10 + [ci] * 7 + [_dp, ci]
        L.cfref_block_forward.argtypes = blk
        L.cfref_block_forward_loopfused.argtypes = blk
        L.cfref_downsample.argtypes = [_dp, _dp, _dp, _dp, ci, ci, ci, ci, ci, _dp, ci]
        L.cfref_grouped_conv.argtypes = [_dp, _dp] + [ci] * 9 + [_dp]
        L.cfref_gconv.argtypes = [_dp, _dp, _dp, _dp, ci, ci, ci, ci, ci, ci, _dp, ci]
        L.cfref_gblock_forward.argtypes = [_dp] * 10 + [ci] * 8 + [_dp, ci]
        L.cfref_mbconv_forward.argtypes = [_dp] * 14 + [ci] * 8 + [_dp]
        L.cfref_mbconv_s2_forward.argtypes = [_dp] * 14 + [ci] * 9 + [_dp]
        L.cfref_blurpool_tri3.argtypes = [_dp, ci, ci, ci, ci, _dp]
        L.cfref_convfirst_s2_forward.argtypes = [_dp] * 10 + [ci] * 9 + [_dp]
        L.cfref_default_threads.restype = ci
        _lib = L
    return _lib


def _p(a):
    """Pointer to a C-contiguous float64 array, or NULL for None."""
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_dp)


def _f64(a):
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def default_threads() -> int:
    return lib().cfref_default_threads()


def act(u: float, name: str = "gelu") -> float:
    """phi of eq. e:ffn (Sec. 5.2), one scalar."""
    return lib().cfref_act(float(u), ACTS[name])


def depthwise(x, dw_w, s0=None, b0=None, nthreads: int = 0):
    """Depth-wise k x k conv with floor(k/2) zero padding (Sec. 4.1.1,
    eq. f:depth-wise-conv2d, K = C).  x [N,H,W,C], dw_w [k,k,C]."""
    x, dw_w, s0, b0 = _f64(x), _f64(dw_w), _f64(s0), _f64(b0)
    N, H, W, C = x.shape
    k = dw_w.shape[0]
    assert dw_w.shape == (k, k, C) and k % 2 == 1
    d = np.empty_like(x)
    lib().cfref_depthwise(_p(x), _p(dw_w), _p(s0), _p(b0), N, H, W, C, k, _p(d), nthreads)
    return d


def pointwise(x, a, s=None, b=None, nthreads: int = 0):
    """Point-wise conv as the matrix product of eq. f:pointwise-matrix-conv2d.
    x [..., Cin], a [Cout, Cin] -> [..., Cout]."""
    x, a, s, b = _f64(x), _f64(a), _f64(s), _f64(b)
    Cin = x.shape[-1]
    Cout = a.shape[0]
    assert a.shape == (Cout, Cin)
    P = int(np.prod(x.shape[:-1]))
    y = np.empty(x.shape[:-1] + (Cout,), dtype=np.float64)
    lib().cfref_pointwise(_p(x), _p(a), _p(s), _p(b), P, Cin, Cout, _p(y), nthreads)
    return y


def block_forward(x, p: dict, act: str = "gelu", loopfused: bool = False, nthreads: int = 0,
                  return_threads: bool = False):
    """The ConvFirst block (Sec. 5.3 / 5.3.1) with depth-wise conv, folded norms
    and the residual shortcut.  ``loopfused`` selects the eq. e:ffn-eff
    evaluation order instead of the layer-by-layer one (eq. e:ffn).

    p holds dw_w [k,k,C], w1 [E*C,C], w2 [C,E*C] and optional s0,b0 [C],
    s1,b1 [E*C], s2,b2 [C]."""
    x = _f64(x)
    N, H, W, C = x.shape
    dw_w, w1, w2 = _f64(p["dw_w"]), _f64(p["w1"]), _f64(p["w2"])
    k = dw_w.shape[0]
    EC = w1.shape[0]
    assert dw_w.shape == (k, k, C) and w1.shape == (EC, C) and w2.shape == (C, EC)
    assert EC % C == 0
    E = EC // C
    vec = [_f64(p.get(n)) for n in ("s0", "b0", "s1", "b1", "s2", "b2")]
    y = np.empty_like(x)
    fn = lib().cfref_block_forward_loopfused if loopfused else lib().cfref_block_forward
    used = fn(_p(x), _p(dw_w), _p(vec[0]), _p(vec[1]), _p(w1), _p(vec[2]), _p(vec[3]),
              _p(w2), _p(vec[4]), _p(vec[5]), N, H, W, C, E, k, ACTS[act], _p(y), nthreads)
    return (y, used) if return_threads else y


def downsample(x, wd, sd=None, bd=None, nthreads: int = 0):
    """2x2 stride-2 conv (eq. f:conv2d with R = S = 2, stride 2, no padding).
    x [N,H,W,Cin], wd [Cout,2,2,Cin] -> [N,H/2,W/2,Cout]."""
    x, wd, sd, bd = _f64(x), _f64(wd), _f64(sd), _f64(bd)
    N, H, W, Cin = x.shape
    Cout = wd.shape[0]
    assert wd.shape == (Cout, 2, 2, Cin) and H % 2 == 0 and W % 2 == 0
    y = np.empty((N, H // 2, W // 2, Cout), dtype=np.float64)
    rc = lib().cfref_downsample(_p(x), _p(wd), _p(sd), _p(bd), N, H, W, Cin, Cout, _p(y), nthreads)
    assert rc >= 0
    return y


def grouped_conv(x, a, groups: int, stride: int = 1, pad: int = 0):
    """Grouped convolution exactly as eq. f:grouped-conv2d (Sec. 4.1.1) writes
    it: weights a [K, R, S, T] in the paper's index order, T = C / groups,
    group of output channel k = floor(k C / (K T)).  x [N,H,W,C] -> [N,Ho,Wo,K].
    Serial, for small cross-checks."""
    x, a = _f64(x), _f64(a)
    N, H, W, C = x.shape
    K, R, S, T = a.shape
    assert R == S and C % groups == 0 and T == C // groups
    Ho = (H + 2 * pad - R) // stride + 1
    Wo = (W + 2 * pad - R) // stride + 1
    y = np.empty((N, Ho, Wo, K), dtype=np.float64)
    rc = lib().cfref_grouped_conv(_p(x), _p(a), N, H, W, C, K, R, T, stride, pad, _p(y))
    assert rc == 0
    return y


def gconv(x, a, s0=None, b0=None, nthreads: int = 0):
    """The block's grouped layer: k x k, C -> C channels, group width gw,
    floor(k/2) zero padding (Sec. 5.3 with eq. f:grouped-conv2d).
    x [N,H,W,C], a [k,k,C,gw] (the library's tap layout)."""
    x, a, s0, b0 = _f64(x), _f64(a), _f64(s0), _f64(b0)
    N, H, W, C = x.shape
    k, _, C2, gw = a.shape
    assert a.shape == (k, k, C, gw) and C2 == C and C % gw == 0 and k % 2 == 1
    d = np.empty_like(x)
    rc = lib().cfref_gconv(_p(x), _p(a), _p(s0), _p(b0), N, H, W, C, k, gw, _p(d), nthreads)
    assert rc > 0
    return d


def gblock_forward(x, p: dict, act: str = "relu", nthreads: int = 0):
    """The ConvFirst block as the paper defines it (Sec. 5.3): grouped k x k
    conv (group width gw), FFN, residual; norms folded to scale and bias.
    p holds gw_w [k,k,C,gw], w1 [E*C,C], w2 [C,E*C] and optional s0,b0 [C],
    s1,b1 [E*C], s2,b2 [C].  The paper's block uses ReLU (Sec. 5.3)."""
    x = _f64(x)
    N, H, W, C = x.shape
    a, w1, w2 = _f64(p["gw_w"]), _f64(p["w1"]), _f64(p["w2"])
    k, _, _, gw = a.shape
    EC = w1.shape[0]
    assert a.shape == (k, k, C, gw) and w1.shape == (EC, C) and w2.shape == (C, EC) and EC % C == 0
    vec = [_f64(p.get(n)) for n in ("s0", "b0", "s1", "b1", "s2", "b2")]
    y = np.empty_like(x)
    rc = lib().cfref_gblock_forward(_p(x), _p(a), _p(vec[0]), _p(vec[1]), _p(w1), _p(vec[2]),
                                    _p(vec[3]), _p(w2), _p(vec[4]), _p(vec[5]), N, H, W, C, EC // C,
                                    k, gw, ACTS[act], _p(y), nthreads)
    assert rc > 0
    return y


def stem_forward(x, w, scale=None, bias=None):
    """The network's stem (App. A: a 3 x 3 convolution with stride 2 from the
    image's 3 channels to the first stage's C channels; caption of Fig.
    f:convfirstnet: ReLU), its batch norm folded to scale and bias: the
    grouped convolution of eq. f:grouped-conv2d with one group, stride 2 and
    one pixel of zero padding, then s * conv + b and ReLU.
    x [N,H,W,3], w [C,3,3,3] in the paper's [K][R][S][T] order -> [N,ceil(H/2),ceil(W/2),C]."""
    w = _f64(w)
    K, R, S, T = w.shape
    assert R == S == 3 and T == _f64(x).shape[3]
    u = grouped_conv(x, w, groups=1, stride=2, pad=1)
    if scale is not None:
        u = u * _f64(scale)
    if bias is not None:
        u = u + _f64(bias)
    return np.maximum(u, 0.0)


def stem_gblock_forward(x, stem: dict, p: dict, act: str = "relu"):
    """The stem followed by the first ConvFirst block (App. A: the stem
    would be fused with the kernel of the first block): gblock_forward of
    stem_forward.  stem holds sw [C,3,3,3] and optional ss, sb [C]."""
    return gblock_forward(stem_forward(x, stem["sw"], stem.get("ss"), stem.get("sb")), p, act=act)


def mbconv_forward(x, p: dict):
    """The paper's MBConv block with Squeeze & Excitation (Sec. 5.4, 5.4.1):
    expand + SiLU, grouped k x k conv (group width gw) + SiLU, SE (average,
    squeeze to R with ReLU, excite with sigmoid, gate), project, residual;
    norms folded to scale and bias.  p holds w1 [E*C,C], gw_w [k,k,E*C,gw],
    wr [R,E*C], we [E*C,R], w2 [C,E*C] and optional fp vectors s1,b1,s2,b2
    [E*C], br [R], be [E*C], s3,b3 [C]."""
    x = _f64(x)
    N, H, W, C = x.shape
    w1, a, wr, we, w2 = (_f64(p[k]) for k in ("w1", "gw_w", "wr", "we", "w2"))
    EC = w1.shape[0]
    k, _, _, gw = a.shape
    R = wr.shape[0]
    assert w1.shape == (EC, C) and a.shape == (k, k, EC, gw) and wr.shape == (R, EC)
    assert we.shape == (EC, R) and w2.shape == (C, EC) and EC % C == 0
    vec = [_f64(p.get(n)) for n in ("s1", "b1", "s2", "b2", "br", "be", "s3", "b3")]
    y = np.empty_like(x)
    rc = lib().cfref_mbconv_forward(_p(x), _p(w1), _p(vec[0]), _p(vec[1]), _p(a), _p(vec[2]), _p(vec[3]),
                                    _p(wr), _p(vec[4]), _p(we), _p(vec[5]), _p(w2), _p(vec[6]), _p(vec[7]),
                                    N, H, W, C, EC // C, R, k, gw, _p(y))
    assert rc == 0
    return y


def blurpool_tri3(x):
    """BlurPool with the Triangle-3 filter (Sec. 5.4: the down-sampling layer
    of the stride-2 MBConv block): per channel, taps [1, 2, 1]/4 in each
    direction, one pixel of reflect padding, stride 2.  x [N,H,W,Ch] with
    H, W >= 2 -> [N, ceil(H/2), ceil(W/2), Ch]."""
    x = _f64(x)
    N, H, W, Ch = x.shape
    y = np.empty((N, (H + 1) // 2, (W + 1) // 2, Ch))
    assert lib().cfref_blurpool_tri3(_p(x), N, H, W, Ch, _p(y)) == 0
    return y


def mbconv_s2_forward(x, p: dict):
    """The stride-2 MBConv block (Fig. f:mbconv, stride 2; Sec. 5.4): as
    mbconv_forward up to the grouped conv's SiLU, then blurpool_tri3, the
    squeeze over the down-sampled map, the gates, and the project to K
    channels without a residual (the output has another shape).  p as for
    mbconv_forward with w2 [K,E*C] and s3, b3 [K].  x [N,H,W,C] -> [N,
    ceil(H/2), ceil(W/2), K]."""
    x = _f64(x)
    N, H, W, C = x.shape
    w1, a, wr, we, w2 = (_f64(p[k]) for k in ("w1", "gw_w", "wr", "we", "w2"))
    EC = w1.shape[0]
    k, _, _, gw = a.shape
    R, K = wr.shape[0], w2.shape[0]
    assert w1.shape == (EC, C) and a.shape == (k, k, EC, gw) and wr.shape == (R, EC)
    assert we.shape == (EC, R) and w2.shape == (K, EC) and EC % C == 0
    vec = [_f64(p.get(n)) for n in ("s1", "b1", "s2", "b2", "br", "be", "s3", "b3")]
    y = np.empty((N, (H + 1) // 2, (W + 1) // 2, K))
    rc = lib().cfref_mbconv_s2_forward(_p(x), _p(w1), _p(vec[0]), _p(vec[1]), _p(a), _p(vec[2]), _p(vec[3]),
                                       _p(wr), _p(vec[4]), _p(we), _p(vec[5]), _p(w2), _p(vec[6]), _p(vec[7]),
                                       N, H, W, C, EC // C, R, K, k, gw, _p(y))
    assert rc == 0
    return y


def convfirst_s2_forward(x, p: dict, act: str = "relu"):
    """The stride-2 ConvFirst block (Fig. f:convfirst-block (c)) in the
    reading the speed-projection counts support (App. A): grouped conv C -> C
    with its folded norm at the input size, blurpool_tri3 of the conv output
    and of the block input, the two concatenated (2C channels, conv output
    first), expand to R with activation, project to K, no residual.  p holds
    gw_w [k,k,C,gw], w1 [R,2C], w2 [K,R] and optional s0,b0 [C], s1,b1 [R],
    s2,b2 [K].  x [N,H,W,C] with H, W >= 2 -> [N, ceil(H/2), ceil(W/2), K]."""
    x = _f64(x)
    N, H, W, C = x.shape
    a, w1, w2 = _f64(p["gw_w"]), _f64(p["w1"]), _f64(p["w2"])
    k, _, _, gw = a.shape
    R, K = w1.shape[0], w2.shape[0]
    assert a.shape == (k, k, C, gw) and w1.shape == (R, 2 * C) and w2.shape == (K, R)
    vec = [_f64(p.get(n)) for n in ("s0", "b0", "s1", "b1", "s2", "b2")]
    y = np.empty((N, (H + 1) // 2, (W + 1) // 2, K))
    rc = lib().cfref_convfirst_s2_forward(_p(x), _p(a), _p(vec[0]), _p(vec[1]), _p(w1), _p(vec[2]), _p(vec[3]),
                                          _p(w2), _p(vec[4]), _p(vec[5]), N, H, W, C, R, K, k, gw, ACTS[act],
                                          _p(y))
    assert rc == 0
    return y


def stack_forward(x, layers: list, act: str = "gelu", nthreads: int = 0):
    """A sequence of blocks and down-sampling layers applied in order.
    layers: list of ("block", params) or ("down", params with wd, sd, bd)."""
    y = _f64(x)
    for kind, p in layers:
        if kind == "block":
            y = block_forward(y, p, act=act, nthreads=nthreads)
        elif kind == "down":
            y = downsample(y, p["wd"], p.get("sd"), p.get("bd"), nthreads=nthreads)
        else:
            raise ValueError(kind)
    return y
