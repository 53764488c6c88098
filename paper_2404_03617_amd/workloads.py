"""The five workloads the library is measured and checked on.

Shapes follow the benchmark definitions: fp16/bf16 NHWC activations, E = 4,
depth-wise k x k, GELU(erf), weights ~ N(0, 1/fan_in), biases ~ N(0, 0.01),
scales 1, all seeded (``seed`` below feeds ``synth``).
"""
from __future__ import annotations

WORKLOADS = {
    # small latency case, oracle-sized
    "block_n1_14x14_c64_e4_k3_f16": dict(kind="block", N=1, H=14, W=14, C=64, E=4, k=3,
                                         dtype="f16", seed=1),
    # the batch-128 single-block case the throughput metric is quoted on
    "block_n128_56x56_c64_e4_k3_f16": dict(kind="block", N=128, H=56, W=56, C=64, E=4, k=3,
                                           dtype="f16", seed=2),
    "block_n128_14x14_c256_e4_k7_f16": dict(kind="block", N=128, H=14, W=14, C=256, E=4, k=7,
                                            dtype="f16", seed=3),
    # four stages, depths 2/2/6/2, widths 64/128/256/512 at 56/28/14/7, 2x2/s2 down-sampling
    "stack_n128_56x56_d2262_c64to512_e4_k3_f16": dict(kind="stack", N=128, H=56, W=56,
                                                      depths=(2, 2, 6, 2),
                                                      widths=(64, 128, 256, 512), E=4, k=3,
                                                      dtype="f16", seed=4),
    "block_n1_7x7_c512_e4_k3_bf16": dict(kind="block", N=1, H=7, W=7, C=512, E=4, k=3,
                                         dtype="bf16", seed=5),
}

BENCH_WORKLOAD = "block_n128_56x56_c64_e4_k3_f16"

# The paper's own block (3 x 3 grouped conv of group width 8, ReLU) at the
# eight shapes of its kernel benchmark table (Sec. 5.5.3, Table
# t:conv-first-speed): channels, expansion, height = width, batch 128, fp16.
# paper_pct is the block-fusion kernel's fraction of peak that table reports
# on an A5000 (context only: other hardware).
GBLOCK_WORKLOADS = {
    "gblock_n128_%dx%d_c%d_e%d_k3_f16" % (hw, hw, c, e): dict(kind="gblock", N=128, H=hw, W=hw, C=c, E=e, k=3,
                                                            dtype="f16", act="relu", seed=20 + i,
                                                            paper_pct=pct, paper_ms=ms)
    for i, (c, e, hw, pct, ms) in enumerate([
        (16, 3, 128, 35.1, 0.42), (32, 3, 128, 46.6, 0.99), (32, 6, 64, 66.9, 0.30), (48, 6, 64, 71.6, 0.59),
        (64, 6, 64, 76.2, 0.96), (48, 6, 32, 67.0, 0.16), (64, 6, 32, 74.0, 0.25), (96, 6, 32, 68.7, 0.58)])
}

# The MBConv + Squeeze & Excitation kernel benchmark (Sec. 5.4.1, Table
# t:mbconv-speed): channels 128..256, expansion 4, SE ratio 0.25 of the input
# channels (R = C/4), height = width 16 or 8, batch 128, fp16.  paper_pct is
# the block-fusion kernel's fraction of an A5000's peak in that table (context
# only: other hardware).
MBCONV_WORKLOADS = {
    "mbconv_n128_%dx%d_c%d_e4_r%d_f16" % (hw, hw, c, c // 4): dict(kind="mbconv", N=128, H=hw, W=hw, C=c, E=4,
                                                                 R=c // 4, k=3, dtype="f16", seed=40 + i,
                                                                 paper_pct=pct, paper_ms=ms)
    for i, (c, hw, pct, ms) in enumerate([
        (128, 16, 46.2, 2.48), (144, 16, 44.4, 3.19), (160, 16, 41.9, 4.09), (192, 16, 44.4, 5.39),
        (256, 16, 51.0, 8.01), (128, 8, 45.0, 0.64), (144, 8, 32.5, 1.09), (160, 8, 31.3, 1.37),
        (192, 8, 43.1, 1.39), (256, 8, 51.4, 1.99)])
}

# The stride-2 MBConv + SE blocks of the speed-projection tables at 16 x 16
# (App. A: the four model sizes' C = K = 128, 160, 192, 256, E = 4, down to
# 8 x 8), batch 128, fp16, squeeze R = C/4 as for the stride-1 rows.  The
# paper builds no kernel for them: paper_proj_ms is its projection (80% of
# the stride-1 kernel's efficiency), not a measurement.
MBCONV_S2_WORKLOADS = {
    "mbconv_s2_n128_16x16_c%d_k%d_e4_r%d_f16" % (c, c, c // 4): dict(kind="mbconv_s2", N=128, H=16, W=16, C=c,
                                                                    E=4, R=c // 4, K=c, k=3, dtype="f16",
                                                                    seed=70 + i, paper_proj_ms=ms)
    for i, (c, ms) in enumerate([(128, 0.282), (160, 0.595), (192, 0.819), (256, 0.835)])
}

# The stride-2 ConvFirst blocks of the speed-projection tables (App. A: the
# distinct stride-2 ConvFirst rows over the four model sizes), batch 128,
# fp16, ReLU: input H = W, C channels, hidden R, output K.  The paper builds
# no kernel for them: paper_proj_ms is its projection, not a measurement.
CONVFIRST_S2_WORKLOADS = {
    "convfirst_s2_n128_%dx%d_c%d_r%d_k%d_f16" % (hw, hw, c, r, k): dict(kind="convfirst_s2", N=128, H=hw, W=hw, C=c,
                                                                      R=r, K=k, dtype="f16", act="relu",
                                                                      seed=80 + i, paper_proj_ms=ms)
    for i, (hw, c, r, k, ms) in enumerate([
        (128, 16, 96, 32, 0.275), (64, 32, 192, 48, 0.196), (128, 24, 144, 48, 0.495), (64, 48, 288, 64, 0.336),
        (64, 48, 288, 72, 0.380), (128, 32, 192, 64, 0.758), (64, 64, 384, 96, 0.650)])
}

# The network stem (a 3x3 stride-2 conv from the 256 x 256 image's 3 channels,
# ReLU) fused into the first ConvFirst block at 128 x 128 (App. A, the first two
# rows of the speed-projection tables: the Pico stem 3 -> 16 before ConvFirst
# C = 16, alpha = 3; the 3 -> 32 stem before ConvFirst C = 32, alpha = 3), batch
# 128, fp16, ReLU.  The image is seed-drawn N(0, 1).
STEM_WORKLOADS = {
    "stem_gblock_n128_256x256_c%d_e3_f16" % c: dict(kind="stem_gblock", N=128, Hin=256, Win=256, C=c, E=3, k=3,
                                                    dtype="f16", act="relu", seed=60 + i)
    for i, c in enumerate([16, 32])
}
