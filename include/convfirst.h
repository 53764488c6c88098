/*
 * convfirst.h -- C ABI of the MI355X (gfx950) ConvFirst block-fusion library.
 *
 * The library evaluates the ConvFirst residual block of A. Lavin, "On the
 * Efficiency of Convolutional Neural Networks" (arXiv:2404.03617), Sec. 5.3,
 * with the block-fusion schedule of Sec. 5.3.1: one kernel loads an input
 * tile, runs the k x k depth-wise convolution, initialises the output
 * accumulators with the input tile (residual shortcut), then loops over
 * chunks of hidden channels -- expand, activation, project -- in the
 * loop-fused order of eq. e:ffn-eff, and stores the output tile once.  The
 * hidden layer (E*C channels per pixel) never reaches device memory.
 *
 * Block definition (every batch norm folded into a per-channel scale and bias
 * after its linear layer, Sec. 5.3.1 last paragraph):
 *   D = s0 * dwconv_k(X) + b0                 depth-wise, zero padding k/2, Sec. 4.1.1
 *   U = s1 * (D W1^T) + b1                    expand to E*C channels, eq. e:ffn
 *   Z = s2 * (phi(U) W2^T) + b2               project back to C
 *   Y = X + Z                                 residual shortcut
 *
 * Conventions shared by every entry point
 *   - Pointers named x, y, w*, s*, b*, ws are DEVICE pointers; the
 *     cf_*_params structs themselves live in host memory and are read during
 *     the call only.
 *   - Activations are NHWC, channels fastest: x[N][H][W][C].  All tensors of a
 *     call share one I/O dtype (cf_dtype); scales and biases are fp32.
 *   - A NULL scale means all ones; a NULL bias means all zeros.
 *   - The caller owns every buffer.  The library allocates no device memory;
 *     buffers must stay valid until the work queued on `stream` completes.
 *   - Every *_forward call is asynchronous on `stream` (a hipStream_t passed
 *     as void*; NULL is the null stream).  Nothing is synchronised.
 *   - Arguments are validated on the host before anything is queued; on any
 *     non-CF_OK status nothing was launched and outputs are untouched, except
 *     CF_ERR_HIP, which reports a launch failure after validation passed.
 *     cf_last_error() returns a thread-local message for the last failure.
 *   - x, y and ws must not overlap each other (fused halos make in-place
 *     evaluation unsafe) and must be 16-byte aligned.
 *   - Results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef CONVFIRST_H
#define CONVFIRST_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CF_ABI_VERSION 1

typedef enum {
    CF_OK = 0,
    CF_ERR_INVALID = 1,     /* null pointer, bad size, overlap, misalignment, bad enum */
    CF_ERR_UNSUPPORTED = 2, /* valid request the library has no kernel for (e.g. C % 32 != 0) */
    CF_ERR_WORKSPACE = 3,   /* workspace smaller than the matching *_workspace_bytes() */
    CF_ERR_HIP = 4          /* the HIP runtime reported an error at launch */
} cf_status;

typedef enum { CF_F16 = 0, CF_BF16 = 1 } cf_dtype;

/* Activation phi after the expand layer (eq. e:ffn).  GELU is the exact
 * Gaussian-CDF form u * Phi(u).  The fused fp16 kernels evaluate it with a
 * packed-fp16 polynomial whose absolute error is below 3.4e-3 for |u| < 10
 * and zero beyond (it saturates to 0 and u); the fused bf16 kernels and the
 * layer-by-layer kernels use fp32 erf, the kernel for N*H*W <= 64 the fp32
 * erf of Abramowitz & Stegun 7.1.26 (|error| <= 1.5e-7).
 * CF_ACT_NONE makes the block affine (used by tests). */
typedef enum { CF_ACT_GELU_ERF = 0, CF_ACT_RELU = 1, CF_ACT_NONE = 2 } cf_act;

/* Weights of one block (all device pointers).
 *   dw_w  [k][k][C]     depth-wise taps (tap-major, channels fastest)
 *   w1    [E*C][C]      expand, row r = hidden channel r (torch Linear layout)
 *   w2    [C][E*C]      project, row c = output channel c
 *   dw_scale/dw_bias [C], s1/b1 [E*C], s2/b2 [C]  fp32, each may be NULL */
typedef struct {
    const void *dw_w;
    const float *dw_scale, *dw_bias;
    const void *w1;
    const float *s1, *b1;
    const void *w2;
    const float *s2, *b2;
} cf_block_params;

/* 2x2 stride-2 down-sampling conv: w [Cout][2][2][Cin]; scale/bias [Cout] fp32. */
typedef struct {
    const void *w;
    const float *scale, *bias;
} cf_down_params;

/* One ConvFirst block, fused (Sec. 5.3.1, eq. e:ffn-eff): y = block(x).
 * x, y: [N][H][W][C].  Supported: C in {64, 128, 256, 512}, E >= 1,
 * k in {1, 3, 5, 7}; any N, H, W >= 1.  Other C return CF_ERR_UNSUPPORTED.
 * With N*H*W <= 64 and C >= 128 the block runs on one workgroup per 32
 * output channels (each recomputing the expand, no workspace; Sec. 4.1.2:
 * the weights are the bytes), unless the autotuner cached another
 * configuration for the shape. */
cf_status cf_block_forward(const void *x, void *y, const cf_block_params *p,
                           int N, int H, int W, int C, int E, int k,
                           cf_dtype dt, cf_act act, void *stream);

/* `depth` consecutive blocks of the same shape (a network stage, the unit the
 * paper benchmarks, Sec. 5.5.3).  Intermediate activations ping-pong between
 * y and ws; blocks[depth] are host-side structs of device pointers.
 * cf_stage_workspace_bytes() returns the recommended ws size.  The minimum is
 * N*H*W*C*2 bytes (rounded up to 256) for depth > 1 and 0 for depth == 1;
 * for C = 512 fp16 the recommended size adds 16*N*H*W*C bytes.  With that
 * room, at N*H*W >= 4096 pixels and E <= 6, each block runs layer by layer
 * (Sec. 5.2): a depth-wise kernel, the expand and project as hipBLASLt
 * GEMMs with the hidden tensor in ws (s1, b1 and the activation in the
 * expand's epilogue, with the library's GELU, when s1 and b1 are given;
 * else an elementwise kernel after it), and s2, b2 and the residual in the
 * project's epilogue (else an elementwise kernel after it, the project's
 * output rounded to fp16 first); within the block tolerance of the fused
 * kernels, deterministic.
 * Otherwise, with the room, each block splits its hidden layer over several
 * workgroups (results identical up to fp32 summation order, deterministic).
 * The library GEMMs are given no workspace of their own. */
cf_status cf_stage_forward(const void *x, void *y, void *ws, size_t ws_bytes,
                           const cf_block_params *blocks, int depth,
                           int N, int H, int W, int C, int E, int k,
                           cf_dtype dt, cf_act act, void *stream);
size_t cf_stage_workspace_bytes(int depth, int N, int H, int W, int C, cf_dtype dt);

/* The stage with the micro-batch schedule of Sec. 5.5.2: the `depth` blocks
 * run over micro-batches of `micro_batch` images -- all blocks over images
 * 0..m-1, then all blocks over the next m images, and so on -- so the
 * intermediate activations of one micro-batch (2 * m*H*W*C*2 bytes in the
 * ping-pong buffers) can stay in on-chip caches between the blocks instead
 * of making a round trip to DRAM per block.  Consecutive launches give a
 * pixel range the same workgroup index, hence the same L2 (XCD), so a
 * micro-batch whose activations fit the L2s is read back from them; one that
 * fits the 256 MiB Infinity Cache is read back from it.  Only the stage's
 * input and output need DRAM.  Results equal cf_stage_forward's up to the
 * fp32 summation order of the hidden split it may use at C = 512 (none
 * here).  micro_batch <= 0 picks a default: the largest micro-batch whose
 * input and output activations fit 128 MiB (the whole batch whenever the
 * stage's activations already fit the Infinity Cache); a micro_batch >= N
 * runs the whole batch per block.  ws needs cf_stage_microbatch_workspace_bytes() bytes: two
 * micro-batch buffers for depth > 2, one for depth == 2, none for depth 1. */
cf_status cf_stage_forward_microbatch(const void *x, void *y, void *ws, size_t ws_bytes,
                                      const cf_block_params *blocks, int depth,
                                      int N, int H, int W, int C, int E, int k, int micro_batch,
                                      cf_dtype dt, cf_act act, void *stream);
size_t cf_stage_microbatch_workspace_bytes(int depth, int N, int H, int W, int C, int micro_batch,
                                           cf_dtype dt);

/* 2x2 stride-2 conv between stages: y[n][i][j][o] = scale[o] * sum_{a,b,c}
 * w[o][a][b][c] * x[n][2i+a][2j+b][c] + bias[o]  (eq. f:conv2d with R = S = 2,
 * stride 2, no padding; no activation, no residual).  H and W must be even;
 * y is [N][H/2][W/2][Cout].  Cin must be a multiple of 32, Cout of 64, and
 * N*(H/2)*(W/2) below 2^31 (CF_ERR_UNSUPPORTED otherwise). */
cf_status cf_downsample_forward(const void *x, void *y, const cf_down_params *p,
                                int N, int H, int W, int Cin, int Cout,
                                cf_dtype dt, void *stream);

/* The same block executed layer by layer (Fig. f:convfirst-tensor-machine (a)):
 * three kernels -- depth-wise, expand GEMM + activation, project GEMM +
 * residual -- with the depth-wise output (P*C) and the hidden layer (P*E*C)
 * round-tripping through ws.  The comparison path for the fused kernel. */
cf_status cf_block_forward_unfused(const void *x, void *y, void *ws, size_t ws_bytes,
                                   const cf_block_params *p,
                                   int N, int H, int W, int C, int E, int k,
                                   cf_dtype dt, cf_act act, void *stream);
size_t cf_unfused_workspace_bytes(int N, int H, int W, int C, int E, cf_dtype dt);

/* The fused block with its hidden channels split over `groups` workgroups per
 * pixel tile, for small N*H*W where one tile per CU would idle the chip
 * (the channel partition with partial sums of Sec. 5.3.1, Fig.
 * f:convfirst-tensor-machine (c), applied to the hidden dimension).  Each
 * group writes an fp32 partial of the projected output to ws; a second kernel
 * adds the groups in a fixed order, plus b2 and the residual, so the result is
 * deterministic.  groups must divide E*C/32; groups <= 0 picks a default.
 * ws needs cf_split_workspace_bytes() bytes. */
cf_status cf_block_forward_split(const void *x, void *y, void *ws, size_t ws_bytes,
                                 const cf_block_params *p,
                                 int N, int H, int W, int C, int E, int k, int groups,
                                 cf_dtype dt, cf_act act, void *stream);
size_t cf_split_workspace_bytes(int N, int H, int W, int C, int E, int groups);

/* The ConvFirst block as the paper defines it (Sec. 5.3): the first layer is
 * a k x k grouped convolution of group width CF_GROUP_WIDTH = 8 with C input
 * and C output channels (eq. f:grouped-conv2d with K = C, T = 8: output
 * channel c reads input channels floor(c/8)*8 .. +7), followed by the same
 * FFN and residual as cf_block_forward, all in one fused kernel (Sec. 5.3.1):
 *   D[n,h,w,c] = s0[c] * sum_{i,j<k} sum_{t<8} gw_w[i][j][c][t]
 *                 * X[n, h+i-k/2, w+j-k/2, floor(c/8)*8 + t] + b0[c]
 * The paper's block uses ReLU (Sec. 5.3, benchmarked in Table
 * t:conv-first-speed at C = 16..96, E = 3 or 6); GELU and identity are
 * available too.
 *   gw_w  [k][k][C][8]  grouped taps: torch's grouped nn.Conv2d weight
 *                       [C][8][k][k] permuted to (2, 3, 0, 1)
 *   w1, w2, and the fp32 vectors as in cf_block_params.
 * Supported: k = 3; C a multiple of 16 from 16 to 112; any E >= 1 (E*C need
 * not be a multiple of 32); any N, H, W >= 1.  C not a multiple of 8 returns
 * CF_ERR_INVALID, other unsupported shapes CF_ERR_UNSUPPORTED.  fp16 or bf16
 * I/O, fp32 accumulation; the conv output and the hidden values are rounded
 * to the I/O dtype before the next product. */
#define CF_GROUP_WIDTH 8
typedef struct {
    const void *gw_w;
    const float *gw_scale, *gw_bias;
    const void *w1;
    const float *s1, *b1;
    const void *w2;
    const float *s2, *b2;
} cf_gblock_params;

cf_status cf_gblock_forward(const void *x, void *y, const cf_gblock_params *p,
                            int N, int H, int W, int C, int E, int k,
                            cf_dtype dt, cf_act act, void *stream);

/* The stride-2 ConvFirst block (Fig. f:convfirst-block (c): the variant that
 * down-samples with BlurPool, Triangle-3), in one kernel.  The figure is not
 * in the paper's text; the layer order and sizes are the reading its
 * speed-projection tables fix (App. A: the conv at the input size over C
 * channels, the expand at the output size over 2C, the project to K):
 *   D  = s0 * gconv3x3(X) + b0                     grouped conv, C -> C (as
 *                                                  cf_gblock_forward's D)
 *   Z  = [bp(D), bp(X)]                            2C channels, D's first;
 *   bp(V)[i,j,c] = sum_{a,b<3} t[a] t[b] V[rf(2i+a-1), rf(2j+b-1), c],
 *        t = (1, 2, 1) / 4, one pixel of reflect padding (rf(-1) = 1,
 *        rf(H) = H - 2)
 *   Y  = s2 * (w2 act(s1 * (w1 Z) + b1)) + b2      no residual
 * Tensors (row-major, I/O dtype unless noted):
 *   x [N][H][W][C];  y [N][ceil(H/2)][ceil(W/2)][K]
 *   p->gw_w [3][3][C][8] (with gw_scale, gw_bias fp32 [C]);  p->w1 [R][2C];
 *   p->w2 [K][R];  s1, b1 fp32 [R];  s2, b2 fp32 [K]  (NULL scale 1, bias 0).
 * The paper's block uses ReLU; GELU and identity are available too.
 * Supported: k = 3; C = 16, 24, 32, 48 or 64; R a multiple of 16 up to 1024;
 * K a multiple of 8 up to 128; H, W >= 2.  C not a multiple of 8, H or W below 2, or y
 * overlapping x return CF_ERR_INVALID, other shapes CF_ERR_UNSUPPORTED.  fp16
 * or bf16 I/O; the conv accumulates pair products in fp32; D, the blurred
 * maps and the hidden values are rounded to the I/O dtype before the next
 * product.  Deterministic. */
cf_status cf_convfirst_s2_forward(const void *x, void *y, const cf_gblock_params *p,
                                  int N, int H, int W, int C, int R, int K, int k,
                                  cf_dtype dt, cf_act act, void *stream);

/* The network's stem (App. A: a 3 x 3 convolution with stride 2 from the
 * image's 3 channels to the first stage's channels; caption of Fig.
 * f:convfirstnet: ReLU), its batch norm folded to a scale and a bias:
 *   S[n,i,j,c] = ReLU(scale[c] * sum_{r,s<3} sum_{t<3} w[c][r][s][t]
 *                 * X[n, 2i+r-1, 2j+s-1, t] + bias[c])     (zero outside X)
 *   x [N][Hin][Win][3]; y [N][ceil(Hin/2)][ceil(Win/2)][C]
 *   w [C][3][3][3]: torch's conv weight [C][3][3][3] permuted (0, 2, 3, 1),
 *   the paper's [K][R][S][T] order; scale, bias fp32 [C] (NULL: 1, 0).
 * C = 16, 24 or 32, the paper's three stem widths (another multiple of 8
 * returns CF_ERR_UNSUPPORTED, C not a multiple of 8 CF_ERR_INVALID).  fp16 or
 * bf16, fp32 accumulation, output rounded once to the I/O dtype.  x and y
 * must not overlap; pointers 16-byte aligned. */
typedef struct {
    const void *w;
    const float *scale, *bias;
} cf_stem_params;

cf_status cf_stem_forward(const void *x, void *y, const cf_stem_params *p, int N, int Hin, int Win, int C,
                          cf_dtype dt, void *stream);

/* The stem fused into the first ConvFirst block, as App. A proposes:
 * y = cf_gblock_forward(stem(x)) in one kernel.  Each block's halo of stem
 * output is computed from the image on the matrix unit and kept in LDS, so
 * the stem output never reaches memory; it is rounded to the I/O dtype as a
 * stored one would be.  x [N][Hin][Win][3]; y [N][ceil(Hin/2)][ceil(Win/2)][C];
 * blk as for cf_gblock_forward with this C, k = 3 and act (the paper's first
 * block uses ReLU); C = 16 or 32 (the grouped block has no C = 24 kernel:
 * its channel tiles are 16 wide; C = 24 returns CF_ERR_UNSUPPORTED). */
cf_status cf_stem_gblock_forward(const void *x, void *y, const cf_stem_params *stem, const cf_gblock_params *blk,
                                 int N, int Hin, int Win, int C, int E, int k, cf_dtype dt, cf_act act,
                                 void *stream);

/* The MBConv block with Squeeze & Excitation of Sec. 5.4 (Fig. f:mbconv:
 * the paper's variant with a grouped 3 x 3 conv of group width 8 in place of
 * the depth-wise one), fused into one kernel as Sec. 5.4.1 describes (Fig.
 * f:mbconv-block-fusion-tensor-machine).  With EC = E*C hidden channels:
 *   U[n,h,w,:] = SiLU(s1 * (w1 X[n,h,w,:]) + b1)                     expand
 *   V[n,h,w,c] = SiLU(s2[c] * sum_{i,j<3} sum_{t<8} gw_w[i][j][c][t]
 *                 * U[n, h+i-1, w+j-1, floor(c/8)*8 + t] + b2[c])     grouped conv
 *   z[n] = ReLU(wr mean_{h,w} V[n,h,w,:] + br)                        squeeze
 *   g[n] = sigmoid(we z[n] + be)                                       excitation
 *   Y[n,h,w,:] = X[n,h,w,:] + s3 * (w2 (V[n,h,w,:] * g[n])) + b3       project, residual
 * Tensors (row-major, I/O dtype unless noted):
 *   x, y  [N][H][W][C]
 *   w1    [EC][C]        expand (torch 1x1 conv weight [EC][C][1][1])
 *   gw_w  [3][3][EC][8]  grouped taps: torch's weight [EC][8][3][3] permuted (2, 3, 0, 1)
 *   wr    [R][EC]        squeeze;  we [EC][R] excitation;  w2 [C][EC] project
 *   s1, b1, s2, b2, be  fp32 [EC];  br fp32 [R];  s3, b3 fp32 [C]
 *   (NULL scale means 1, NULL bias 0; folded batch norms go into the s/b pairs)
 * Each work item (an image and 64 of its hidden channels) computes its
 * expand and conv layers alone; the squeeze sums over every hidden channel
 * and the projection reads all of them, so the work items of an image
 * exchange their conv outputs and squeeze shares through ws and meet once in
 * global memory.  The kernel is therefore launched cooperatively, with each
 * image's work items resident together.  The target is the late stages of a
 * network: supported are k = 3, 1 <= H, W <= 16, C a multiple of 16, E*C a
 * multiple of 64 and at most 4096, 1 <= R <= 256, and a shared-memory layout
 * (the group's W1 rows, the gates of all E*C channels, the staged hidden
 * layer) within the 160 KB of a CU: C up to 768 at E = 2, 512 at E = 4, 256
 * at E = 8 (CF_ERR_UNSUPPORTED otherwise; C not a multiple of 8 is
 * CF_ERR_INVALID).  y may equal x
 * (evaluation in place); any other overlap among x, y and ws is
 * CF_ERR_INVALID.  ws: cf_mbconv_workspace_bytes() bytes (queried on the
 * current device) let every image the device can hold be in flight; a
 * smaller ws runs fewer images at once, and one too small for a single image
 * returns CF_ERR_WORKSPACE.  ws must be zero-filled before its first use:
 * its first 256 + 2048 * 128 bytes hold the barrier lines of the images in
 * flight, and every call leaves them zero again, whatever the shapes of the
 * calls that share the workspace, so a call is a single launch.  If a
 * barrier wait ever gives up (that call's output is then invalid; the
 * cooperative launch rules this out), the first int of ws is set to 1 and the
 * library never clears it.  Calls that share a workspace must not overlap in
 * time.
 * launch: CF_LAUNCH_COOPERATIVE (hipLaunchCooperativeKernel: the runtime
 * makes every workgroup resident at once, and refuses a grid that cannot be)
 * or CF_LAUNCH_EXCLUSIVE, an ordinary launch of the same grid (sized to what
 * fits on the device) for callers that own the device for the call -- no
 * kernel of theirs or anyone else's runs beside it.  It saves the cooperative
 * launch's fixed cost (about 17 us per call measured on MI355X); if other
 * work does keep a workgroup from starting, a wait gives up after about a
 * second and the flag above is set (the kernel still ends).  fp16 or bf16 I/O, fp32
 * accumulation; U, V and the gated project weights are rounded to the I/O
 * dtype before their products.  Deterministic: every sum has a fixed order. */
typedef struct {
    const void *w1;
    const float *s1, *b1;
    const void *gw_w;
    const float *s2, *b2;
    const void *wr;
    const float *br;
    const void *we;
    const float *be;
    const void *w2;
    const float *s3, *b3;
} cf_mbconv_params;

typedef enum { CF_LAUNCH_COOPERATIVE = 0, CF_LAUNCH_EXCLUSIVE = 1 } cf_launch;

cf_status cf_mbconv_forward(const void *x, void *y, void *ws, size_t ws_bytes, const cf_mbconv_params *p,
                            int N, int H, int W, int C, int E, int R, int k, cf_dtype dt, cf_launch launch,
                            void *stream);
/* 0 for shapes the kernel does not support. */
size_t cf_mbconv_workspace_bytes(int N, int H, int W, int C, int E, int R, cf_dtype dt);

/* The stride-2 MBConv block (Fig. f:mbconv with stride 2; Sec. 5.4), the
 * first block of a stage that halves the image and changes the channel
 * count.  Same expand, grouped conv and SiLU as cf_mbconv_forward; then
 *   V'[n,i,j,c] = sum_{a,b<3} t[a] t[b] V[n, rf(2i+a-1, H), rf(2j+b-1, W), c]
 *                 with t = (1, 2, 1) / 4 and rf reflecting one pixel past the
 *                 border (rf(-1) = 1, rf(H) = H - 2)          BlurPool, Triangle-3
 *   z[n] = ReLU(wr mean_{i,j} V'[n,i,j,:] + br);  g[n] = sigmoid(we z[n] + be)
 *   Y[n,i,j,:] = s3 * (w2 (V'[n,i,j,:] * g[n])) + b3           project, no residual
 * The paper names the BlurPool filter and places the down-sampling in the
 * stride-2 block but leaves the padding and the squeeze's input unstated;
 * reflect padding and the squeeze over the down-sampled map are the readings
 * taken here.  Tensors as for cf_mbconv_forward except
 *   x [N][H][W][C];  y [N][ceil(H/2)][ceil(W/2)][K];  w2 [K][EC];
 *   s3, b3 fp32 [K].
 * Supported: as cf_mbconv_forward, plus 2 <= H, W (reflect padding needs a
 * second row and column) and K a positive multiple of 16 with the LDS layout
 * (now also holding the work item's full-resolution V, H*W*144 bytes)
 * within 160 KB; K <= 0 or H, W < 2 is CF_ERR_INVALID, K not a multiple of
 * 16 CF_ERR_UNSUPPORTED.  y must not overlap x (no in-place form: the shapes
 * differ); ws as for cf_mbconv_forward, sized by
 * cf_mbconv_s2_workspace_bytes (the exchanged map is V', a quarter of V).
 * Each work item blurs its own 64 channels from its LDS copy of V before the
 * exchange, so the block is still one launch with one barrier per image.
 * V and V' are rounded to the I/O dtype (V' sums 9 rounded V values in fp32);
 * the squeeze sums the unrounded fp32 V'.  Deterministic. */
cf_status cf_mbconv_s2_forward(const void *x, void *y, void *ws, size_t ws_bytes, const cf_mbconv_params *p,
                               int N, int H, int W, int C, int E, int R, int K, int k, cf_dtype dt,
                               cf_launch launch, void *stream);
/* 0 for shapes the kernel does not support. */
size_t cf_mbconv_s2_workspace_bytes(int N, int H, int W, int C, int E, int R, int K, cf_dtype dt);

/* Allocation-free variant of cf_block_forward_split, for callers that cannot
 * allocate device memory: code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments and result as
 * cf_block_forward_split with the same `groups` (bit for bit), minus the
 * workspace: the fp32 partials go to a static device array of
 * CF_SPLIT_SCRATCH_BYTES bytes that the library holds on every GPU it runs on
 * until the process ends.  It calls no allocating routine.  A call whose
 * partials (cf_split_workspace_bytes) exceed the array returns
 * CF_ERR_WORKSPACE and launches nothing.  Every call on one GPU shares that
 * GPU's array, so calls that overlap in time on one GPU (other streams, other
 * threads) race and must be serialised by the caller; the array needs no
 * clearing (each call overwrites the part it reads). */
#define CF_SPLIT_SCRATCH_BYTES ((size_t)16 << 20)
cf_status cf_block_forward_split_noalloc(const void *x, void *y, const cf_block_params *p,
                                         int N, int H, int W, int C, int E, int k, int groups,
                                         cf_dtype dt, cf_act act, void *stream);

/* Autotune (Sec. 5.5: the kernel class enumerates the valid kernel
 * configurations for the block's parameters, runs each, keeps the fastest).
 * Same arguments and validation as cf_block_forward.  Synchronous: runs every
 * configuration that applies to the shape on `stream` (a few launches each,
 * timed with events), stores the fastest in a per-process cache keyed by
 * (device, N, H, W, C, E, k, dtype, act), and leaves y holding the block's
 * output computed with it.  Later cf_block_forward calls with that key use the
 * cached configuration.  The cache is guarded by a mutex; results of every
 * configuration agree within the parity tolerance (they differ only in tiling
 * and in which kernel implements the block). */
cf_status cf_block_autotune(const void *x, void *y, const cf_block_params *p,
                            int N, int H, int W, int C, int E, int k,
                            cf_dtype dt, cf_act act, void *stream);
/* The cached configuration id for a key (0 = default kernel and tiling), or -1
 * for invalid arguments. */
int cf_block_tuned_config(int N, int H, int W, int C, int E, int k, cf_dtype dt, cf_act act);

/* Thread-local message describing the most recent non-CF_OK status. */
const char *cf_last_error(void);
const char *cf_status_string(cf_status s);
int cf_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CONVFIRST_H */
