"""Generator of the packed-fp16 GELU coefficients of cf_device.h.

The fused kernel evaluates GELU on fp16 pairs in the scaled variable
w = u / 4 (the hidden activations are kept at a quarter of their value so
that fp16 never overflows):

    GELU(u) / 4 = w * Phi(4 w),   Phi(4 w) ~= clamp01(0.5 + w * Q(w * w)),

with Q a polynomial of degree 4 (five fused multiply-adds per pair).

Step 1 fits Q by iteratively reweighted least squares towards the minimax
error of u * (P - Phi) over |u| <= A.  Step 2 refines the coefficients by a
Nelder-Mead search on the error of the exact fp16 evaluation (every rounding
of the device sequence emulated) over every finite fp16 w with |4 w| < 10.
Prints the coefficients and the error figures quoted in cf_device.h.

    python gelu_fit.py
"""
import numpy as np
from scipy.optimize import minimize
from scipy.special import erf

A = 3.5       # fit range in u
DEG = 4       # degree of Q in w*w


def phi(u):
    return 0.5 * (1.0 + erf(u / np.sqrt(2.0)))


def f16(x):
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def irls(a=A, deg=DEG, iters=80):
    u = np.cos(np.linspace(0.0, np.pi, 6000)) * a
    u = u[u > 0]
    w = u / 4.0
    basis = np.stack([w * (w * w) ** j for j in range(deg + 1)], 1)
    tgt = phi(u) - 0.5
    wt = np.ones_like(u)
    for _ in range(iters):
        sw = np.sqrt(wt) * np.maximum(u, 0.3)
        c, *_ = np.linalg.lstsq(basis * sw[:, None], tgt * sw, rcond=None)
        e = np.abs(basis @ c - tgt) * np.maximum(u, 0.3)
        wt = wt * (e / e.max()) ** 0.5 + 1e-12
    return c


def device_eval(w, c):
    """The kernel's fp16 sequence: s = w*w; q by Horner with fma; p = fma(w, q, 0.5);
    clamp to [0, 1]; return w * p (= GELU(4 w) / 4).  Each fma rounds once."""
    c = [float(f16(x)) for x in c]
    s = f16(w * w)
    q = f16(s * c[4] + c[3])
    q = f16(s * q + c[2])
    q = f16(s * q + c[1])
    q = f16(s * q + c[0])
    p = np.clip(f16(w * q + 0.5), 0.0, 1.0)
    return f16(w * p)


def all_f16():
    h = np.arange(65536, dtype=np.uint16).view(np.float16)
    return h[np.isfinite(h)].astype(np.float64)


def errors(c):
    w = all_f16()
    u = 4.0 * w
    with np.errstate(all="ignore"):
        g = 4.0 * device_eval(w, c)
        err = np.abs(g - u * phi(u))
    inner = np.abs(u) < 10
    return err[inner].max(), (err[~inner] / np.abs(u[~inner])).max(), int(np.isnan(g).sum())


def main():
    c0 = irls()
    w = all_f16()
    w = w[np.abs(4.0 * w) < 10]
    ref = 4.0 * w * phi(4.0 * w)

    def obj(c):
        with np.errstate(all="ignore"):
            return np.abs(4.0 * device_eval(w, c) - ref).max()

    r = minimize(obj, c0, method="Nelder-Mead", options=dict(maxiter=4000, xatol=1e-7, fatol=1e-8))
    c = r.x
    assert c[-1] > 0, "leading coefficient must be positive for the clamp to saturate correctly"
    e_in, e_out, nans = errors(c)
    print("coefficients c0..c4:", ", ".join("%.8f" % x for x in c))
    print("max |error| for |u| < 10: %.2e;  max |error| / |u| beyond: %.2e;  NaNs: %d" % (e_in, e_out, nans))


if __name__ == "__main__":
    main()
