"""Host-side checks of the kernels' own arithmetic choices (CPU only).

The fp16 fused kernels evaluate GELU with a packed-fp16 polynomial in the
scaled variable w = u / 4 (cf_device.h).  The header promises
|GELU_device(u) - u * Phi(u)| < 3.4e-3 for |u| < 10 and exact saturation
beyond.  This test replays the device sequence -- every fp16 rounding of
s = w*w, four Horner fmas, p = fma(w, q, 0.5), clamp to [0, 1], w * p --
over every finite fp16 w, with the coefficients parsed from the kernel
header (so it checks what the kernels compile), against Phi computed with
math.erf in double precision.
"""
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEVICE_H = os.path.join(ROOT, "paper_2404_03617_amd", "csrc", "cf_device.h")
HEADER = os.path.join(ROOT, "include", "convfirst.h")

BOUND = 3.4e-3  # the figure quoted by include/convfirst.h and cf_device.h


def kernel_coefficients():
    src = open(DEVICE_H).read()
    c = [float(re.search(r"GELU_Q%d\s*=\s*([-+0-9.eE]+)f" % i, src).group(1)) for i in range(5)]
    return c


def f16(v):
    return np.asarray(v, dtype=np.float64).astype(np.float16).astype(np.float64)


def device_gelu_quarter(w, c):
    """GELU(4 w) / 4 as the kernels evaluate it: each packed fp16 operation
    rounds once to fp16 (fp16 x fp16 products are exact in fp64, so rounding
    the fp64 fma result once reproduces the hardware fma)."""
    c = [float(f16(v)) for v in c]
    s = f16(w * w)
    q = f16(s * c[4] + c[3])
    q = f16(s * q + c[2])
    q = f16(s * q + c[1])
    q = f16(s * q + c[0])
    p = np.minimum(np.maximum(f16(w * q + 0.5), 0.0), 1.0)
    return f16(w * p)


def all_finite_f16():
    h = np.arange(65536, dtype=np.uint16).view(np.float16)
    return h[np.isfinite(h)].astype(np.float64)


def exact_gelu(u):
    phi = np.frompyfunc(lambda v: 0.5 * (1.0 + math.erf(v / math.sqrt(2.0))), 1, 1)
    return u * phi(u).astype(np.float64)


def gelu_errors(c):
    w = all_finite_f16()
    u = 4.0 * w
    with np.errstate(over="ignore", invalid="ignore"):
        got = 4.0 * device_gelu_quarter(w, c)
    err = np.abs(got - exact_gelu(u))
    inner = np.abs(u) < 10.0
    return got, err, inner, u


def test_header_quotes_the_bound_this_test_checks():
    assert "3.4e-3" in open(HEADER).read()
    assert "3.4e-3" in open(DEVICE_H).read()


def test_fp16_gelu_error_bound_over_every_finite_input():
    got, err, inner, u = gelu_errors(kernel_coefficients())
    assert np.isfinite(got).all(), "the device sequence produced inf or NaN"
    assert err[inner].max() < BOUND, "max |error| for |u| < 10 is %.3e" % err[inner].max()
    # beyond |u| = 10 the clamp saturates: GELU(u) = u above, 0 below, to
    # within the fp16 rounding of u itself (u is exact: w is fp16)
    assert (err[~inner] / np.abs(u[~inner])).max() < 1e-15


def test_fp16_gelu_is_monotone_where_the_exact_function_is():
    """GELU is increasing for u > -0.75; the device curve must not dip by more
    than the error bound there (a wrong-signed coefficient would)."""
    w = np.sort(all_finite_f16())
    u = 4.0 * w
    keep = (u > -0.5) & (u < 10.0)
    with np.errstate(over="ignore", invalid="ignore"):
        g = 4.0 * device_gelu_quarter(w[keep], kernel_coefficients())
    drops = np.maximum.accumulate(g) - g
    assert drops.max() < 2 * BOUND


@pytest.mark.parametrize("i,delta", [(0, 0.01), (2, -0.05), (4, 0.02)])
def test_the_bound_detects_a_perturbed_coefficient(i, delta):
    """A small change to any one coefficient breaks the bound: the test is
    tight enough to notice a mistyped constant."""
    c = kernel_coefficients()
    c[i] += delta
    _, err, inner, _ = gelu_errors(c)
    assert err[inner].max() > BOUND


# ---------------------------------------------------------------- operation count
def _table_rows():
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "convfirst_kernel_table.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                c, e, h, w, ms, tf, pct = line.split()
                rows.append((int(c), int(e), int(h), int(w), float(ms), float(tf), float(pct)))
    return rows


@pytest.mark.parametrize("row", _table_rows(), ids=lambda r: "C%d_a%d_%dx%d" % r[:4])
def test_grouped_block_operation_count_reproduces_the_papers_table(row):
    """roofline.gblock_flops (2 * 128 * H * W * (72 C + 2 alpha C^2)) divided by
    the paper's measured times gives its TFLOPS column, and TFLOPS / 76.7 its
    percent-of-peak column (the printed values are rounded, the times to two
    digits, and the percentages were evidently taken from unrounded figures:
    51.3 / 76.7 = 66.88 is printed as 67.0, hence the tolerances)."""
    from paper_2404_03617_amd import roofline as rl
    C, E, H, W, ms, tflops, pct = row
    got = rl.gblock_flops(128, H, W, C, E) / (ms * 1e-3) / 1e12
    assert got == pytest.approx(tflops, rel=0.02)
    assert tflops / 76.7 * 100 == pytest.approx(pct, abs=0.2)


def _mbconv_rows():
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "mbconv_projection_rows.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                v = line.split()
                rows.append(tuple(int(a) for a in v[:6]) + tuple(float(a) for a in v[6:10]) + (int(v[10]),
                                                                                            float(v[11])))
    return rows


@pytest.mark.parametrize("row", _mbconv_rows(), ids=lambda r: "s%d_%dx%d_C%d_K%d" % (r[0], r[1], r[2], r[3], r[5]))
def test_mbconv_operation_counts_reproduce_the_projection_tables(row):
    """Each printed column of the paper's MBConv rows (two decimals, in
    millions per image) from the operation count of the stride-1 or stride-2
    block: the total, and each layer isolated by zeroing the other layers'
    widths (zero pixels leave the squeeze/excitation, group width 0 removes
    the grouped conv, K = 0 the project of the stride-2 block; the stride-1
    expand and project count alike)."""
    from paper_2404_03617_amd import roofline as rl
    s, H, W, C, EC, K, conv, exp, prj, se, depth, total = row
    E, R = EC // C, C // 4
    assert E * C == EC

    def f(H=H, W=W, gw=8, K=K):
        if s == 1:
            return rl.mbconv_flops(1, H, W, C, E, R, gw=gw) / 1e6
        return rl.mbconv_s2_flops(1, H, W, C, E, R, K, gw=gw) / 1e6

    if s == 1:
        assert K == C
    full = f()
    assert full == pytest.approx(total / depth, abs=0.015)
    assert full == pytest.approx(conv + exp + prj + se, abs=0.015)
    assert f(H=0, W=0) == pytest.approx(se, abs=0.005)
    assert full - f(gw=0) == pytest.approx(conv, abs=0.005)
    if s == 1:
        assert (f(gw=0) - f(H=0, W=0)) / 2 == pytest.approx(prj, abs=0.005)
        assert exp == prj
    else:
        assert full - f(K=0) == pytest.approx(prj, abs=0.005)
        assert f(gw=0, K=0) - f(H=0, W=0, K=0) == pytest.approx(exp, abs=0.005)


# ---- the slice kernel's fp32 GELU: erf by Abramowitz & Stegun 7.1.26
SLICE_HIP = os.path.join(ROOT, "paper_2404_03617_amd", "csrc", "cf_slice.hip")
AS_BOUND = 1.5e-7  # the published bound of 7.1.26 on |erf error|


def slice_gelu_constants():
    """(p, a5, a4, a3, a2, a1) as the kernel writes them, in Horner order."""
    src = open(SLICE_HIP).read()
    body = src[src.index("float gelu_as(float u)"):]
    body = body[:body.index("\n}\n")]
    nums = [float(v) for v in re.findall(r"(-?\d+\.\d+)f", body)]
    # in source order: 1/sqrt(2), p, 1.0, a5, a4, a3, a2, a1, -log2(e), 1.0, 0.5
    assert len(nums) == 11 and nums[2] == 1.0 and nums[9] == 1.0 and nums[10] == 0.5, nums
    return [nums[0], nums[1], nums[3], nums[4], nums[5], nums[6], nums[7], -nums[8]]


def f32(v):
    return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)


def slice_gelu(u, nums):
    """The kernel's sequence in float32 (each operation rounded once; the
    reciprocal and exponential as correctly rounded float32 results)."""
    r2, p, a5, a4, a3, a2, a1, l2e = [float(f32(v)) for v in nums[:8]]
    u = f32(u)
    x = f32(np.abs(u) * r2)
    t = f32(1.0 / f32(p * x + 1.0))
    q = f32(a5 * t + a4)
    q = f32(q * t + a3)
    q = f32(q * t + a2)
    q = f32(q * t + a1)
    q = f32(q * t)
    e = f32(np.exp2(f32(f32(x * x) * -l2e)))
    erf_x = f32(-q * e + 1.0)
    hu = f32(0.5 * u)
    return f32(hu * np.copysign(erf_x, u) + hu)


def test_slice_gelu_constants_are_the_published_ones():
    nums = slice_gelu_constants()
    assert nums[:7] == [0.70710678118654752, 0.3275911, 1.061405429, -1.453152027, 1.421413741, -0.284496736,
                        0.254829592]
    assert abs(nums[7] - 1.4426950408889634) < 1e-15


def _slice_gelu_max_error(nums):
    u = np.concatenate([np.linspace(-12.0, 12.0, 480001), np.array([-1e4, -50.0, 50.0, 1e4, 1e-30, -1e-30, 0.0])])
    got = slice_gelu(u, nums)
    ref = exact_gelu(u)
    return np.max(np.abs(got - ref) / np.maximum(1.0, np.abs(u)))


def test_slice_gelu_meets_the_erf_bound():
    """|GELU_kernel(u) - u Phi(u)| <= (0.5 * 1.5e-7 + float32 rounding) * max(1, |u|)."""
    err = _slice_gelu_max_error(slice_gelu_constants())
    assert err < 3e-7, err


def test_slice_gelu_bound_catches_a_wrong_coefficient():
    nums = slice_gelu_constants()
    bad = list(nums)
    bad[2] *= 1.001  # a5
    assert _slice_gelu_max_error(bad) > 3e-7
    bad = list(nums)
    bad[1] = 0.33  # p
    assert _slice_gelu_max_error(bad) > 3e-7
