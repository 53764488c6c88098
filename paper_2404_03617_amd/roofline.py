"""Work and traffic counts for the roofline / waterline report.

Counting rule of the paper (Sec. 5.1): only the multiply-accumulates of
convolutions and matrix products count, two operations each; bias adds,
activations and the residual add are free.  Bytes are the compulsory DRAM
transfers of Sec. 4.1.2: every input and output element once, every weight
once.

Formulas
  block (depth-wise k x k, group width gw = 1; the paper's grouped conv has
  gw = 8):   ops/pixel = 2 * (k*k*gw*C + 2*E*C*C)
  2x2/s2 down-sampling:  ops/output pixel = 2 * 4 * Cin * Cout
  roofline:  t_min = n / min(R, B * n / b)
  waterline: T_min = sum_i t_min,i ;  C_max = sum_i n_i / (T_min * R)   (eq.
             e:total-attainable-latency, e:max-comp-eff)
  computational efficiency C = R_actual / R_peak = (n / R_peak) / t  (eq. e:comp-eff)
"""
from __future__ import annotations

# MI355X published peaks
PEAK_FP16_FLOPS = 2.5166e15   # dense fp16/bf16 MFMA, FLOP/s
PEAK_HBM_BPS = 8.0e12         # HBM3E, bytes/s


def block_ops_per_pixel(C: int, E: int, k: int, gw: int = 1) -> int:
    return 2 * (k * k * gw * C + 2 * E * C * C)


def block_layer_ops_per_image(H: int, W: int, C: int, E: int, k: int, gw: int = 1):
    """(conv, expand, project) operation counts for one image, as the paper's
    per-layer tables list them."""
    conv = 2 * H * W * C * gw * k * k
    exp = 2 * H * W * C * E * C
    return conv, exp, exp


def block_flops(N, H, W, C, E, k, gw=1) -> int:
    return N * H * W * block_ops_per_pixel(C, E, k, gw)


def gblock_flops(N, H, W, C, E, k=3, gw=8) -> int:
    """The paper's count for its own block (Sec. 5.5.3): 2 * P * (k*k*gw*C + 2*E*C*C),
    i.e. 2 * 128 * H * W * (72 C + 2 alpha C^2) at batch 128, k = 3, gw = 8."""
    return block_flops(N, H, W, C, E, k, gw)


def gblock_bytes_fused(N, H, W, C, E, k=3, gw=8, eb=2) -> int:
    return 2 * N * H * W * C * eb + eb * (k * k * gw * C + 2 * E * C * C) + 4 * (4 * C + 2 * E * C)


def stem_flops(N, Hin, Win, C) -> int:
    """The stem: 2 * 27 * C per output pixel (App. A's Conv column: 14.16 M
    per image at 256 x 256 -> 128 x 128, C = 16)."""
    return N * ((Hin + 1) // 2) * ((Win + 1) // 2) * 2 * 27 * C


def stem_gblock_bytes_fused(N, Hin, Win, C, E, k=3, gw=8, eb=2) -> int:
    """Image read once, block output written once, weights once."""
    Hs, Ws = (Hin + 1) // 2, (Win + 1) // 2
    return (N * Hin * Win * 3 + N * Hs * Ws * C) * eb + eb * (27 * C + k * k * gw * C + 2 * E * C * C) + \
        4 * (2 * C + 4 * C + 2 * E * C)


def mbconv_flops(N, H, W, C, E, R, k=3, gw=8) -> int:
    """MBConv + SE (Sec. 5.4): expand 2 P E C^2, grouped conv 2 P E C k^2 gw,
    squeeze and excitation 4 E C R per image, project 2 P E C^2 -- the
    columns Exp, Conv, Sqz Exc and Prj of the paper's projection tables."""
    P = H * W
    EC = E * C
    return N * (2 * P * EC * C + 2 * P * EC * k * k * gw + 4 * EC * R + 2 * P * C * EC)


def mbconv_bytes_fused(N, H, W, C, E, R, k=3, gw=8, eb=2) -> int:
    """x read once, y written once, the five weight tensors and the fp32
    vectors once."""
    EC = E * C
    weights = eb * (2 * EC * C + k * k * gw * EC + 2 * R * EC)
    vectors = 4 * (5 * EC + R + 2 * C)
    return 2 * N * H * W * C * eb + weights + vectors


def mbconv_s2_flops(N, H, W, C, E, R, K, k=3, gw=8) -> int:
    """Stride-2 MBConv + SE (Fig. f:mbconv, stride 2): expand and grouped conv
    at the input size, squeeze and excitation, project from E*C to K channels
    at ceil(H/2) x ceil(W/2) -- the same four columns of the projection
    tables, which leave out the BlurPool (9 multiply-adds per down-sampled
    hidden value, not a matrix product)."""
    P, Po = H * W, ((H + 1) // 2) * ((W + 1) // 2)
    EC = E * C
    return N * (2 * P * EC * C + 2 * P * EC * k * k * gw + 4 * EC * R + 2 * Po * K * EC)


def mbconv_s2_bytes_fused(N, H, W, C, E, R, K, k=3, gw=8, eb=2) -> int:
    """x read once, the down-sampled y written once, the five weight tensors
    and the fp32 vectors once."""
    EC = E * C
    weights = eb * (EC * C + k * k * gw * EC + 2 * R * EC + K * EC)
    vectors = 4 * (5 * EC + R + 2 * K)
    return N * H * W * C * eb + N * ((H + 1) // 2) * ((W + 1) // 2) * K * eb + weights + vectors


def convfirst_s2_flops(N, H, W, C, R, K, k=3, gw=8) -> int:
    """Stride-2 ConvFirst block (Fig. f:convfirst-block (c)): grouped conv
    2 H W C k^2 gw at the input size, expand 2 Ho Wo (2C) R and project
    2 Ho Wo R K at the output size -- the Conv, Exp and Prj columns of the
    projection tables (the BlurPool is not counted)."""
    Po = ((H + 1) // 2) * ((W + 1) // 2)
    return N * (2 * H * W * C * k * k * gw + 2 * Po * 2 * C * R + 2 * Po * R * K)


def convfirst_s2_bytes_fused(N, H, W, C, R, K, k=3, gw=8, eb=2) -> int:
    """x read once, the down-sampled y written once, the weights and fp32
    vectors once."""
    Po = ((H + 1) // 2) * ((W + 1) // 2)
    weights = eb * (k * k * C * gw + 2 * C * R + R * K)
    vectors = 4 * (2 * C + 2 * R + 2 * K)
    return N * H * W * C * eb + N * Po * K * eb + weights + vectors


def block_weight_bytes(C, E, k, eb=2, vec_bytes=4) -> int:
    """dw taps, W1, W2 in the I/O dtype plus six fp32 scale/bias vectors."""
    return eb * (k * k * C + 2 * E * C * C) + vec_bytes * (2 * C + 2 * E * C + 2 * C)


def block_bytes_fused(N, H, W, C, E, k, eb=2) -> int:
    """x read once, y written once, weights once."""
    return 2 * N * H * W * C * eb + block_weight_bytes(C, E, k, eb)


def block_bytes_unfused(N, H, W, C, E, k, eb=2):
    """Per-kernel compulsory bytes of the layer-by-layer schedule:
    depth-wise (x -> d), expand (d -> h), project (h, x -> y)."""
    P = N * H * W
    dw = 2 * P * C * eb + eb * k * k * C + 8 * C
    g1 = P * C * eb + P * E * C * eb + eb * E * C * C + 8 * E * C
    g2 = P * E * C * eb + 2 * P * C * eb + eb * E * C * C + 8 * C
    return dw, g1, g2


def block_unfused_ops(N, H, W, C, E, k, gw=1):
    P = N * H * W
    return 2 * P * k * k * gw * C, 2 * P * E * C * C, 2 * P * E * C * C


def down_flops(N, H, W, Cin, Cout) -> int:
    return 2 * N * (H // 2) * (W // 2) * 4 * Cin * Cout


def down_bytes(N, H, W, Cin, Cout, eb=2) -> int:
    return eb * (N * H * W * Cin + N * (H // 2) * (W // 2) * Cout + 4 * Cin * Cout) + 8 * Cout


def t_min(n, b, R=PEAK_FP16_FLOPS, B=PEAK_HBM_BPS) -> float:
    """Roofline minimum latency of one kernel."""
    return n / min(R, B * n / b)


def waterline(kernels, R=PEAK_FP16_FLOPS, B=PEAK_HBM_BPS):
    """kernels: [(n_i, b_i)].  Returns (T_min, C_max)."""
    T = sum(t_min(n, b, R, B) for n, b in kernels)
    N = sum(n for n, _ in kernels)
    return T, N / (T * R)


def amdahl_roofline(f_B: float, f_R: float) -> float:
    """Largest speed-up from making one memory-bound kernel compute bound
    (eq. e:amdahl-roofline): 1 / (1 - f_B + f_R)."""
    return 1.0 / (1.0 - f_B + f_R)


def stack_kernels(N, H, W, depths, widths, E, k, eb=2):
    """[(kind, n, b)] for every launch of a stage stack with 2x2/s2
    down-sampling between stages (fused blocks)."""
    out = []
    h, w = H, W
    for s, (d, c) in enumerate(zip(depths, widths)):
        if s > 0:
            out.append(("down", down_flops(N, h, w, widths[s - 1], c), down_bytes(N, h, w, widths[s - 1], c, eb)))
            h, w = h // 2, w // 2
        for _ in range(d):
            out.append(("block", block_flops(N, h, w, c, E, k), block_bytes_fused(N, h, w, c, E, k, eb)))
    return out


def comp_eff(flops: float, seconds: float, R=PEAK_FP16_FLOPS) -> float:
    return flops / (R * seconds)
