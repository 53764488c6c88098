// cf_api.hip -- the C ABI of include/convfirst.h: argument validation on the
// host (no HIP call before every check has passed), dispatch to the launchers
// of cf_fused.hip / cf_unfused.hip, and error reporting.
#include "convfirst.h"
#include "cf_kernels.h"

#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>

// The fp32 partials of cf_block_forward_split_noalloc live in this static
// device array; each GPU the library runs on holds its own copy until the
// process ends.  In host code the name is not a device address: launches and
// copies use the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[CF_SPLIT_SCRATCH_BYTES];

namespace {

constexpr size_t SCRATCH_BYTES = CF_SPLIT_SCRATCH_BYTES;

thread_local char g_err[512] = "";

cf_status fail(cf_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

cf_status hip_fail(hipError_t e, const char *what) {
    return fail(CF_ERR_HIP, "%s: HIP error %d (%s)", what, (int)e, hipGetErrorString(e));
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x0 = (uintptr_t)a, x1 = x0 + na, y0 = (uintptr_t)b, y1 = y0 + nb;
    return x0 < y1 && y0 < x1;
}

size_t elem_bytes(cf_dtype dt) { return 2; }

// Checks shared by every block entry point.  `what` names the entry point.
cf_status check_block(const char *what, const void *x, const void *y, const cf_block_params *p, int N, int H, int W,
                      int C, int E, int k, cf_dtype dt, cf_act act) {
    if (!x || !y)
        return fail(CF_ERR_INVALID, "%s: x and y must be non-NULL", what);
    if (!p)
        return fail(CF_ERR_INVALID, "%s: params must be non-NULL", what);
    if (!p->dw_w || !p->w1 || !p->w2)
        return fail(CF_ERR_INVALID, "%s: dw_w, w1 and w2 must be non-NULL", what);
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0 || k <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive (N=%d H=%d W=%d C=%d E=%d k=%d)", what, N, H, W, C,
                    E, k);
    if (k % 2 == 0 || k > 7)
        return fail(CF_ERR_INVALID, "%s: k must be 1, 3, 5 or 7 (got %d)", what, k);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    if ((int)act != CF_ACT_GELU_ERF && (int)act != CF_ACT_RELU && (int)act != CF_ACT_NONE)
        return fail(CF_ERR_INVALID, "%s: unknown activation %d", what, (int)act);
    const double elems = (double)N * H * W * C;
    const double hidden = (double)E * C;
    if (elems > 4.0e12 || hidden > 65536.0 || (double)H * W > 2.0e9)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {x, y, p->dw_w, p->w1, p->w2, p->dw_scale, p->dw_bias, p->s1, p->b1, p->s2, p->b2};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (overlap(x, bytes, y, bytes))
        return fail(CF_ERR_INVALID, "%s: x and y overlap (in-place evaluation is not supported)", what);
    if (C != 64 && C != 128 && C != 256 && C != 512)
        return fail(CF_ERR_UNSUPPORTED, "%s: C=%d has no kernel (supported: 64, 128, 256, 512)", what, C);
    if ((double)N * H * W > 2147483647.0 - 4096.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: N*H*W must stay below 2^31 pixels", what);
    return CF_OK;
}

cf::BlockW to_w(const cf_block_params *p) {
    cf::BlockW w;
    w.dw_w = p->dw_w;
    w.s0 = p->dw_scale;
    w.b0 = p->dw_bias;
    w.w1 = p->w1;
    w.s1 = p->s1;
    w.b1 = p->b1;
    w.w2 = p->w2;
    w.s2 = p->s2;
    w.b2 = p->b2;
    return w;
}

cf::Shape to_shape(int N, int H, int W, int C, int E, int k, cf_dtype dt, cf_act act) {
    cf::Shape s;
    s.N = N;
    s.H = H;
    s.W = W;
    s.C = C;
    s.E = E;
    s.k = k;
    s.bf16 = dt == CF_BF16;
    s.act = (int)act;
    return s;
}

// slice_ok: the caller runs one hidden group, so the slice kernel may serve
// a shape no tile kernel fits
cf_status check_fit(const char *what, const cf::Shape &s, bool slice_ok = true) {
    if (cf::tile_fits(s) || (slice_ok && cf::slice_applies(s)))
        return CF_OK;
    const size_t lds = cf::fused_lds_bytes(s);
    return fail(CF_ERR_UNSUPPORTED, "%s: tile for W=%d C=%d k=%d needs %zu bytes of LDS (limit 163840)", what, s.W,
                s.C, s.k, lds);
}

size_t round256(size_t v) { return (v + 255) & ~(size_t)255; }

// ---- autotune cache: (device, shape, dtype, activation) -> kernel configuration
struct TuneKey {
    int dev, N, H, W, C, E, k, bf16, act;
    bool operator<(const TuneKey &o) const {
        const int a[9] = {dev, N, H, W, C, E, k, bf16, act};
        const int b[9] = {o.dev, o.N, o.H, o.W, o.C, o.E, o.k, o.bf16, o.act};
        for (int i = 0; i < 9; i++)
            if (a[i] != b[i])
                return a[i] < b[i];
        return false;
    }
};
std::mutex g_tune_mu;
std::map<TuneKey, int> g_tune;

TuneKey tune_key(const cf::Shape &s) {
    int dev = 0;
    (void)hipGetDevice(&dev);
    return TuneKey{dev, s.N, s.H, s.W, s.C, s.E, s.k, s.bf16, s.act};
}

int tuned_config(const cf::Shape &s) {
    std::lock_guard<std::mutex> lk(g_tune_mu);
    const auto it = g_tune.find(tune_key(s));
    return it == g_tune.end() ? cf::CFG_DEFAULT : it->second;
}

int default_groups(int N, int H, int W, int C, int E) {
    // enough (tile, group) pairs to give every CU one, with groups | E*C/32
    const int chunks = E * C / 32;
    const int64_t P = (int64_t)N * H * W;
    const int M = C == 64 ? 256 : C == 512 ? 64 : 128;
    const int64_t tiles = (P + M - 1) / M;
    int best = 1;
    for (int g = 1; g <= chunks; g++) {
        if (chunks % g)
            continue;
        if (tiles * g <= 256)
            best = g;
    }
    return best;
}

// Checks shared by the two split entry points; on success *need holds the
// bytes of fp32 partials the call writes (groups * N*H*W * C * 4).
cf_status check_split(const char *what, const void *x, const void *y, const cf_block_params *p, int N, int H, int W,
                      int C, int E, int k, int &groups, cf_dtype dt, cf_act act, size_t *need) {
    cf_status st = check_block(what, x, y, p, N, H, W, C, E, k, dt, act);
    if (st != CF_OK)
        return st;
    if (groups <= 0)
        groups = default_groups(N, H, W, C, E);
    const int chunks = E * C / 32;
    if (groups > chunks || chunks % groups)
        return fail(CF_ERR_INVALID, "%s: groups=%d must divide E*C/32=%d", what, groups, chunks);
    *need = (size_t)groups * N * H * W * C * sizeof(float);
    const cf::Shape s = to_shape(N, H, W, C, E, k, dt, act);
    const size_t small_lds = cf::small_split_lds_bytes(s);
    if (!(small_lds > 0 && small_lds <= 160 * 1024) && (st = check_fit(what, s, groups <= 1)) != CF_OK)
        return st;
    return CF_OK;
}

// ---- the allocation-free split variant's scratch (the array is defined at
// file scope above the namespace): its device address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

hipError_t scratch_on_current_device(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= MAX_DEVICES)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!ptr || ((uintptr_t)ptr & 255u))
            return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

// Checks of the stem's own arguments (image x [N][Hin][Win][3], output
// [N][ceil(Hin/2)][ceil(Win/2)][C] at y).
cf_status check_stem(const char *what, const void *x, const void *y, const cf_stem_params *p, int N, int Hin,
                     int Win, int C, cf_dtype dt) {
    if (!x || !y)
        return fail(CF_ERR_INVALID, "%s: x and y must be non-NULL", what);
    if (!p || !p->w)
        return fail(CF_ERR_INVALID, "%s: stem params and w must be non-NULL", what);
    if (N <= 0 || Hin <= 0 || Win <= 0 || C <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive (N=%d Hin=%d Win=%d C=%d)", what, N, Hin, Win, C);
    if (C % CF_GROUP_WIDTH)
        return fail(CF_ERR_INVALID, "%s: C=%d is not a multiple of %d", what, C, CF_GROUP_WIDTH);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    const void *ptrs[] = {x, y, p->w, p->scale, p->bias};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const double hs = (Hin + 1) / 2, ws = (Win + 1) / 2;
    if ((double)N * Hin * Win * 3 > 4.0e12 || (double)N * hs * ws * C > 4.0e12)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const size_t xb = (size_t)N * Hin * Win * 3 * elem_bytes(dt);
    const size_t yb = (size_t)N * (size_t)hs * (size_t)ws * C * elem_bytes(dt);
    if (overlap(x, xb, y, yb))
        return fail(CF_ERR_INVALID, "%s: x and y overlap", what);
    if ((double)N * hs * ws > 2147483647.0 - 4096.0 || (double)Hin * Win * 3 > 2147483647.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: image too large for 32-bit pixel offsets", what);
    return CF_OK;
}

cf::StemW to_stem(const void *x, const cf_stem_params *p, int Hin, int Win) {
    cf::StemW s;
    s.x = x;
    s.w = p->w;
    s.s = p->scale;
    s.b = p->bias;
    s.Hin = Hin;
    s.Win = Win;
    return s;
}

// MBConv + SE, stride 1 (K = 0: C output channels, residual) or stride 2
// (K output channels on a ceil(H/2) x ceil(W/2) map, no residual).
size_t mbconv_ws(int N, int H, int W, int C, int E, int R, int K, cf_dtype dt) {
    if (N <= 0 || E <= 0 || (double)E * C > 65536.0 || !cf::mbconv_supported(H, W, C, E, R, K) ||
        ((int)dt != CF_F16 && (int)dt != CF_BF16))
        return 0;
    int slots = 0;
    if (cf::mbconv_resident_slots(H, W, C, E, R, K, dt == CF_BF16, &slots) != hipSuccess || slots < 1)
        slots = 1;
    return cf::mbconv_workspace_bytes(N, H, W, C, E, R, K, slots < N ? slots : N);
}

cf_status mbconv_call(const char *what, const void *x, void *y, void *ws, size_t ws_bytes, const cf_mbconv_params *p,
                      int N, int H, int W, int C, int E, int R, int K, int k, cf_dtype dt, cf_launch launch,
                      void *stream) {
    if (!x || !y)
        return fail(CF_ERR_INVALID, "%s: x and y must be non-NULL", what);
    if (!p || !p->w1 || !p->gw_w || !p->wr || !p->we || !p->w2)
        return fail(CF_ERR_INVALID, "%s: params, w1, gw_w, wr, we and w2 must be non-NULL", what);
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0 || R <= 0 || k <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive (N=%d H=%d W=%d C=%d E=%d R=%d k=%d)", what, N, H,
                    W, C, E, R, k);
    if (k % 2 == 0)
        return fail(CF_ERR_INVALID, "%s: k must be odd (got %d)", what, k);
    if (C % CF_GROUP_WIDTH)
        return fail(CF_ERR_INVALID, "%s: C=%d is not a multiple of the group width %d", what, C, CF_GROUP_WIDTH);
    if (K > 0 && (H < 2 || W < 2))
        return fail(CF_ERR_INVALID, "%s: BlurPool's reflect padding needs H, W >= 2 (H=%d W=%d)", what, H, W);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    if ((int)launch != CF_LAUNCH_COOPERATIVE && (int)launch != CF_LAUNCH_EXCLUSIVE)
        return fail(CF_ERR_INVALID, "%s: unknown launch mode %d", what, (int)launch);
    if ((double)N * H * W * C > 4.0e12 || (double)E * C > 65536.0 || (double)K > 65536.0)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {x, y, ws, p->w1, p->gw_w, p->wr, p->we, p->w2, p->s1, p->b1,
                          p->s2, p->b2, p->br, p->be, p->s3, p->b3};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const size_t xbytes = (size_t)N * H * W * C * elem_bytes(dt);
    const size_t ybytes = K > 0 ? (size_t)N * ((H + 1) / 2) * ((W + 1) / 2) * K * elem_bytes(dt) : xbytes;
    if (K > 0 ? overlap(x, xbytes, y, ybytes) : (x != y && overlap(x, xbytes, y, ybytes)))
        return fail(CF_ERR_INVALID, K > 0 ? "%s: x and y overlap" : "%s: x and y overlap without being equal", what);
    if (k != 3)
        return fail(CF_ERR_UNSUPPORTED, "%s: k=%d has no kernel (supported: 3)", what, k);
    if (!cf::mbconv_supported(H, W, C, E, R, K))
        return fail(CF_ERR_UNSUPPORTED,
                    "%s: no kernel for H=%d W=%d C=%d E=%d R=%d K=%d (supported: H, W <= 16, C %% 16 == 0, "
                    "E*C %% 64 == 0, E*C <= 4096, R <= 256, K %% 16 == 0)",
                    what, H, W, C, E, R, K);
    const size_t need = cf::mbconv_workspace_bytes(N, H, W, C, E, R, K, 1);
    if (!ws || ws_bytes < need)
        return fail(CF_ERR_WORKSPACE, "%s: ws has %zu bytes, needs at least %zu", what, ws ? ws_bytes : (size_t)0,
                    need);
    if (overlap(ws, ws_bytes, x, xbytes) || overlap(ws, ws_bytes, y, ybytes))
        return fail(CF_ERR_INVALID, "%s: ws overlaps x or y", what);
    cf::MBConvW w;
    w.w1 = p->w1;
    w.s1 = p->s1;
    w.b1 = p->b1;
    w.gw = p->gw_w;
    w.s2 = p->s2;
    w.b2 = p->b2;
    w.wr = p->wr;
    w.br = p->br;
    w.we = p->we;
    w.be = p->be;
    w.w2 = p->w2;
    w.s3 = p->s3;
    w.b3 = p->b3;
    hipError_t e = cf::launch_mbconv(x, y, w, N, H, W, C, E, R, K, dt == CF_BF16, ws, ws_bytes,
                                     launch == CF_LAUNCH_COOPERATIVE, (hipStream_t)stream);
    if (e == hipErrorInvalidConfiguration)
        return fail(CF_ERR_UNSUPPORTED, "%s: the %d work items of one image do not fit on the device at once", what,
                    E * C / 64);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

}  // namespace

extern "C" {

int cf_abi_version(void) { return CF_ABI_VERSION; }

const char *cf_last_error(void) { return g_err; }

const char *cf_status_string(cf_status s) {
    switch (s) {
    case CF_OK: return "CF_OK";
    case CF_ERR_INVALID: return "CF_ERR_INVALID";
    case CF_ERR_UNSUPPORTED: return "CF_ERR_UNSUPPORTED";
    case CF_ERR_WORKSPACE: return "CF_ERR_WORKSPACE";
    case CF_ERR_HIP: return "CF_ERR_HIP";
    }
    return "unknown cf_status";
}

cf_status cf_block_forward(const void *x, void *y, const cf_block_params *p, int N, int H, int W, int C, int E, int k,
                           cf_dtype dt, cf_act act, void *stream) {
    cf_status st = check_block("cf_block_forward", x, y, p, N, H, W, C, E, k, dt, act);
    if (st != CF_OK)
        return st;
    cf::Shape s = to_shape(N, H, W, C, E, k, dt, act);
    if ((st = check_fit("cf_block_forward", s)) != CF_OK)
        return st;
    s.cfg = tuned_config(s);
    hipError_t e = cf::launch_fused_block(x, y, to_w(p), s, 1, nullptr, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, "cf_block_forward");
    g_err[0] = 0;
    return CF_OK;
}

// Minimum stage workspace: the ping-pong buffer (depth > 1).
size_t stage_ws_min(int depth, int N, int H, int W, int C, cf_dtype dt) {
    if (depth <= 1 || N <= 0 || H <= 0 || W <= 0 || C <= 0)
        return 0;
    return round256((size_t)N * H * W * C * elem_bytes(dt));
}

// Hidden-layer groups a C = 512 fp16 stage uses when the workspace allows it:
// enough (tile, group) pairs to fill the chip, at most STAGE_GROUPS.
constexpr int STAGE_GROUPS = 4;
int stage_groups(int N, int H, int W, int C, int E, cf_dtype dt) {
    if (C != 512 || dt != CF_F16)
        return 1;
    const int64_t tiles = ((int64_t)N * H * W + 127) / 128;
    const int chunks = E * C / 32;
    const int cus = cf::device_cu_count();
    int g = 1;
    while (g * 2 <= STAGE_GROUPS && chunks % (g * 2) == 0 && tiles * g * 2 <= cus + cus / 4)
        g *= 2;
    return g;
}

size_t cf_stage_workspace_bytes(int depth, int N, int H, int W, int C, cf_dtype dt) {
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0)
        return 0;
    size_t b = stage_ws_min(depth, N, H, W, C, dt);
    if (C == 512 && dt == CF_F16)
        b += (size_t)STAGE_GROUPS * N * H * W * C * sizeof(float);
    return b;
}

cf_status cf_stage_forward(const void *x, void *y, void *ws, size_t ws_bytes, const cf_block_params *blocks,
                           int depth, int N, int H, int W, int C, int E, int k, cf_dtype dt, cf_act act,
                           void *stream) {
    if (depth <= 0 || !blocks)
        return fail(CF_ERR_INVALID, "cf_stage_forward: depth must be positive and blocks non-NULL");
    for (int i = 0; i < depth; i++) {
        cf_status st = check_block("cf_stage_forward", x, y, &blocks[i], N, H, W, C, E, k, dt, act);
        if (st != CF_OK)
            return st;
    }
    const size_t need = stage_ws_min(depth, N, H, W, C, dt);
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (need) {
        if (!ws)
            return fail(CF_ERR_INVALID, "cf_stage_forward: ws must be non-NULL for depth > 1");
        if (!aligned16(ws))
            return fail(CF_ERR_INVALID, "cf_stage_forward: ws must be 16-byte aligned");
        if (ws_bytes < need)
            return fail(CF_ERR_WORKSPACE, "cf_stage_forward: ws has %zu bytes, needs %zu", ws_bytes, need);
        if (overlap(ws, need, x, bytes) || overlap(ws, need, y, bytes))
            return fail(CF_ERR_INVALID, "cf_stage_forward: ws overlaps x or y");
    }
    const cf::Shape s = to_shape(N, H, W, C, E, k, dt, act);
    cf_status st = check_fit("cf_stage_forward", s);
    if (st != CF_OK)
        return st;
    // wide blocks over many pixels: depth-wise conv, two library GEMMs and
    // two elementwise passes, the hidden tensor in the workspace after the
    // ping-pong buffer, when the workspace holds it
    const size_t lbytes = cf::libgemm_applies(s) ? cf::libgemm_scratch_bytes(s) : 0;
    if (lbytes && ws && aligned16(ws) && ws_bytes >= need + lbytes && !overlap((char *)ws + need, lbytes, x, bytes) &&
        !overlap((char *)ws + need, lbytes, y, bytes) && cf::libgemm_ready(s, (hipStream_t)stream)) {
        void *scratch = (char *)ws + need;
        const void *in = x;
        for (int i = 0; i < depth; i++) {
            void *out = ((depth - 1 - i) % 2 == 0) ? y : ws;
            hipError_t e = cf::launch_block_libgemm(in, out, to_w(&blocks[i]), s, scratch, (hipStream_t)stream);
            if (e != hipSuccess)
                return hip_fail(e, "cf_stage_forward");
            in = out;
        }
        g_err[0] = 0;
        return CF_OK;
    }
    // hidden-layer split with fp32 partials after the ping-pong buffer, when
    // the workspace holds them
    int groups = 1;
    float *partial = nullptr;
    // (a handful of pixels: the slice kernel, which needs no partials)
    const int g = cf::slice_applies(s) ? 1 : stage_groups(N, H, W, C, E, dt);
    const size_t pbytes = (size_t)g * N * H * W * C * sizeof(float);
    if (g > 1 && ws && aligned16(ws) && ws_bytes >= need + pbytes &&
        !overlap((char *)ws + need, pbytes, x, bytes) && !overlap((char *)ws + need, pbytes, y, bytes)) {
        groups = g;
        partial = (float *)((char *)ws + need);
    }
    // block i writes y when (depth-1-i) is even, else ws, so the last one lands in y
    const void *in = x;
    for (int i = 0; i < depth; i++) {
        void *out = ((depth - 1 - i) % 2 == 0) ? y : ws;
        hipError_t e = cf::launch_fused_block(in, out, to_w(&blocks[i]), s, groups, partial, (hipStream_t)stream);
        if (e != hipSuccess)
            return hip_fail(e, "cf_stage_forward");
        in = out;
    }
    g_err[0] = 0;
    return CF_OK;
}

// Micro-batch size of the stage schedule: the given one clamped to [1, N], or
// the largest whose activations (one micro-batch's input and output) fit
// 128 MiB, half of the 256 MiB Infinity Cache.  Micro-batches small enough
// for the L2 caches (4 MiB per XCD) leave most of the 256 CUs idle at these
// image sizes, so the memory-side cache is the level the schedule targets.
static int microbatch_size(int N, int H, int W, int C, int micro_batch, cf_dtype dt) {
    if (micro_batch > 0)
        return micro_batch < N ? micro_batch : N;
    const double per_image = 2.0 * H * W * C * elem_bytes(dt);
    int m = (int)((128.0 * 1024 * 1024) / per_image);
    if (m < 1)
        m = 1;
    return m < N ? m : N;
}

size_t cf_stage_microbatch_workspace_bytes(int depth, int N, int H, int W, int C, int micro_batch, cf_dtype dt) {
    if (depth <= 1 || N <= 0 || H <= 0 || W <= 0 || C <= 0)
        return 0;
    const int m = microbatch_size(N, H, W, C, micro_batch, dt);
    const size_t one = round256((size_t)m * H * W * C * elem_bytes(dt));
    return depth == 2 ? one : 2 * one;
}

cf_status cf_stage_forward_microbatch(const void *x, void *y, void *ws, size_t ws_bytes,
                                      const cf_block_params *blocks, int depth, int N, int H, int W, int C, int E,
                                      int k, int micro_batch, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_stage_forward_microbatch";
    if (depth <= 0 || !blocks)
        return fail(CF_ERR_INVALID, "%s: depth must be positive and blocks non-NULL", what);
    for (int i = 0; i < depth; i++) {
        cf_status st = check_block(what, x, y, &blocks[i], N, H, W, C, E, k, dt, act);
        if (st != CF_OK)
            return st;
    }
    const int m = microbatch_size(N, H, W, C, micro_batch, dt);
    const size_t need = cf_stage_microbatch_workspace_bytes(depth, N, H, W, C, micro_batch, dt);
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (need) {
        if (!ws)
            return fail(CF_ERR_INVALID, "%s: ws must be non-NULL for depth > 1", what);
        if (!aligned16(ws))
            return fail(CF_ERR_INVALID, "%s: ws must be 16-byte aligned", what);
        if (ws_bytes < need)
            return fail(CF_ERR_WORKSPACE, "%s: ws has %zu bytes, needs %zu", what, ws_bytes, need);
        if (overlap(ws, need, x, bytes) || overlap(ws, need, y, bytes))
            return fail(CF_ERR_INVALID, "%s: ws overlaps x or y", what);
    }
    // every micro-batch shape the loop launches must have a kernel
    cf_status st = check_fit(what, to_shape(m, H, W, C, E, k, dt, act));
    if (st != CF_OK)
        return st;
    if (N % m && (st = check_fit(what, to_shape(N % m, H, W, C, E, k, dt, act))) != CF_OK)
        return st;
    const size_t img = (size_t)H * W * C * elem_bytes(dt);
    const size_t one = round256((size_t)m * img);
    char *buf[2] = {(char *)ws, (char *)ws + one};
    // the schedule reproduces the plain stage bit for bit: a micro-batch small
    // enough for the slice kernel (whose expand sums in another order) runs
    // the tile kernels of the whole batch when that batch is not itself a
    // slice shape
    const bool full_slice = cf::slice_applies(to_shape(N, H, W, C, E, k, dt, act));
    for (int n0 = 0; n0 < N; n0 += m) {
        const int mb = N - n0 < m ? N - n0 : m;
        cf::Shape s = to_shape(mb, H, W, C, E, k, dt, act);
        s.cfg = tuned_config(s);
        if (s.cfg == cf::CFG_DEFAULT && !full_slice && cf::slice_applies(s) && cf::tile_fits(s))
            s.cfg = cf::CFG_TILE;
        const void *in = (const char *)x + (size_t)n0 * img;
        for (int i = 0; i < depth; i++) {
            void *out = (i == depth - 1) ? (void *)((char *)y + (size_t)n0 * img) : (void *)buf[i & 1];
            hipError_t e = cf::launch_fused_block(in, out, to_w(&blocks[i]), s, 1, nullptr, (hipStream_t)stream);
            if (e != hipSuccess)
                return hip_fail(e, what);
            in = out;
        }
    }
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_downsample_forward(const void *x, void *y, const cf_down_params *p, int N, int H, int W, int Cin,
                                int Cout, cf_dtype dt, void *stream) {
    const char *what = "cf_downsample_forward";
    if (!x || !y || !p || !p->w)
        return fail(CF_ERR_INVALID, "%s: x, y, params and w must be non-NULL", what);
    if (N <= 0 || H <= 0 || W <= 0 || Cin <= 0 || Cout <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive", what);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    if ((double)N * H * W * (Cin > Cout ? Cin : Cout) > 4.0e12)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {x, y, p->w, p->scale, p->bias};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const size_t xb = (size_t)N * H * W * Cin * 2, yb = (size_t)N * (H / 2) * (W / 2) * Cout * 2;
    if (overlap(x, xb, y, yb))
        return fail(CF_ERR_INVALID, "%s: x and y overlap", what);
    if (H % 2 || W % 2)
        return fail(CF_ERR_UNSUPPORTED, "%s: H and W must be even (got %d x %d)", what, H, W);
    if (Cin % 32 || Cout % 64)
        return fail(CF_ERR_UNSUPPORTED, "%s: needs Cin %% 32 == 0 and Cout %% 64 == 0 (got %d, %d)", what, Cin,
                    Cout);
    if ((int64_t)N * (H / 2) * (W / 2) >= ((int64_t)1 << 31))
        return fail(CF_ERR_UNSUPPORTED, "%s: N*(H/2)*(W/2) must be below 2^31", what);
    hipError_t e = cf::launch_downsample(x, y, p->w, p->scale, p->bias, N, H, W, Cin, Cout, dt == CF_BF16,
                                         (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

size_t cf_unfused_workspace_bytes(int N, int H, int W, int C, int E, cf_dtype dt) {
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0)
        return 0;
    const size_t P = (size_t)N * H * W;
    return round256(P * C * elem_bytes(dt)) + P * (size_t)E * C * elem_bytes(dt);
}

cf_status cf_block_forward_unfused(const void *x, void *y, void *ws, size_t ws_bytes, const cf_block_params *p, int N,
                                   int H, int W, int C, int E, int k, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_block_forward_unfused";
    cf_status st = check_block(what, x, y, p, N, H, W, C, E, k, dt, act);
    if (st != CF_OK)
        return st;
    const size_t need = cf_unfused_workspace_bytes(N, H, W, C, E, dt);
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (!ws)
        return fail(CF_ERR_INVALID, "%s: ws must be non-NULL", what);
    if (!aligned16(ws))
        return fail(CF_ERR_INVALID, "%s: ws must be 16-byte aligned", what);
    if (ws_bytes < need)
        return fail(CF_ERR_WORKSPACE, "%s: ws has %zu bytes, needs %zu", what, ws_bytes, need);
    if (overlap(ws, need, x, bytes) || overlap(ws, need, y, bytes))
        return fail(CF_ERR_INVALID, "%s: ws overlaps x or y", what);
    void *d = ws;
    void *h = (char *)ws + round256((size_t)N * H * W * C * elem_bytes(dt));
    hipError_t e = cf::launch_unfused_block(x, y, d, h, to_w(p), to_shape(N, H, W, C, E, k, dt, act),
                                            (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

size_t cf_split_workspace_bytes(int N, int H, int W, int C, int E, int groups) {
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0)
        return 0;
    if (groups <= 0)
        groups = default_groups(N, H, W, C, E);
    return (size_t)groups * N * H * W * C * sizeof(float);
}

cf_status cf_block_forward_split(const void *x, void *y, void *ws, size_t ws_bytes, const cf_block_params *p, int N,
                                 int H, int W, int C, int E, int k, int groups, cf_dtype dt, cf_act act,
                                 void *stream) {
    const char *what = "cf_block_forward_split";
    size_t need = 0;
    cf_status st = check_split(what, x, y, p, N, H, W, C, E, k, groups, dt, act, &need);
    if (st != CF_OK)
        return st;
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (!ws)
        return fail(CF_ERR_INVALID, "%s: ws must be non-NULL", what);
    if (!aligned16(ws))
        return fail(CF_ERR_INVALID, "%s: ws must be 16-byte aligned", what);
    if (ws_bytes < need)
        return fail(CF_ERR_WORKSPACE, "%s: ws has %zu bytes, needs %zu", what, ws_bytes, need);
    if (overlap(ws, need, x, bytes) || overlap(ws, need, y, bytes))
        return fail(CF_ERR_INVALID, "%s: ws overlaps x or y", what);
    hipError_t e = cf::launch_fused_block(x, y, to_w(p), to_shape(N, H, W, C, E, k, dt, act), groups, (float *)ws,
                                          (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_block_forward_split_noalloc(const void *x, void *y, const cf_block_params *p, int N, int H, int W, int C,
                                         int E, int k, int groups, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_block_forward_split_noalloc";
    size_t need = 0;
    cf_status st = check_split(what, x, y, p, N, H, W, C, E, k, groups, dt, act, &need);
    if (st != CF_OK)
        return st;
    if (need > SCRATCH_BYTES)
        return fail(CF_ERR_WORKSPACE,
                    "%s: the fp32 partials of %d groups need %zu bytes; the static scratch holds %zu "
                    "(use fewer groups or cf_block_forward_split with a workspace)",
                    what, groups, need, SCRATCH_BYTES);
    void *ws = nullptr;
    hipError_t e = scratch_on_current_device(&ws);
    if (e != hipSuccess)
        return hip_fail(e, what);
    e = cf::launch_fused_block(x, y, to_w(p), to_shape(N, H, W, C, E, k, dt, act), groups, (float *)ws,
                               (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_gblock_forward(const void *x, void *y, const cf_gblock_params *p, int N, int H, int W, int C, int E,
                            int k, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_gblock_forward";
    if (!x || !y)
        return fail(CF_ERR_INVALID, "%s: x and y must be non-NULL", what);
    if (!p || !p->gw_w || !p->w1 || !p->w2)
        return fail(CF_ERR_INVALID, "%s: params, gw_w, w1 and w2 must be non-NULL", what);
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0 || k <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive (N=%d H=%d W=%d C=%d E=%d k=%d)", what, N, H, W, C,
                    E, k);
    if (k % 2 == 0 || k > 7)
        return fail(CF_ERR_INVALID, "%s: k must be 1, 3, 5 or 7 (got %d)", what, k);
    if (C % CF_GROUP_WIDTH)
        return fail(CF_ERR_INVALID, "%s: C=%d is not a multiple of the group width %d", what, C, CF_GROUP_WIDTH);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    if ((int)act != CF_ACT_GELU_ERF && (int)act != CF_ACT_RELU && (int)act != CF_ACT_NONE)
        return fail(CF_ERR_INVALID, "%s: unknown activation %d", what, (int)act);
    if ((double)N * H * W * C > 4.0e12 || (double)E * C > 65536.0)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {x, y, p->gw_w, p->w1, p->w2, p->gw_scale, p->gw_bias, p->s1, p->b1, p->s2, p->b2};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const size_t bytes = (size_t)N * H * W * C * elem_bytes(dt);
    if (overlap(x, bytes, y, bytes))
        return fail(CF_ERR_INVALID, "%s: x and y overlap (in-place evaluation is not supported)", what);
    if (k != 3)
        return fail(CF_ERR_UNSUPPORTED, "%s: k=%d has no kernel (supported: 3)", what, k);
    if (!cf::gblock_supported_c(C))
        return fail(CF_ERR_UNSUPPORTED, "%s: C=%d has no kernel (supported: multiples of 16 up to 112)", what, C);
    if ((double)N * H * W > 2147483647.0 - 4096.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: N*H*W must stay below 2^31 pixels", what);
    if ((double)W * C * 6.0 > 2147483647.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: W*C=%.0f is too wide (6 rows must stay below 2^31 elements)", what,
                    (double)W * C);
    cf::GBlockW w;
    w.gw = p->gw_w;
    w.s0 = p->gw_scale;
    w.b0 = p->gw_bias;
    w.w1 = p->w1;
    w.s1 = p->s1;
    w.b1 = p->b1;
    w.w2 = p->w2;
    w.s2 = p->s2;
    w.b2 = p->b2;
    hipError_t e = cf::launch_gblock(x, y, w, to_shape(N, H, W, C, E, k, dt, act), (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_convfirst_s2_forward(const void *x, void *y, const cf_gblock_params *p, int N, int H, int W, int C,
                                  int R, int K, int k, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_convfirst_s2_forward";
    if (!x || !y)
        return fail(CF_ERR_INVALID, "%s: x and y must be non-NULL", what);
    if (!p || !p->gw_w || !p->w1 || !p->w2)
        return fail(CF_ERR_INVALID, "%s: params, gw_w, w1 and w2 must be non-NULL", what);
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || R <= 0 || K <= 0 || k <= 0)
        return fail(CF_ERR_INVALID, "%s: sizes must be positive (N=%d H=%d W=%d C=%d R=%d K=%d k=%d)", what, N, H,
                    W, C, R, K, k);
    if (k % 2 == 0)
        return fail(CF_ERR_INVALID, "%s: k must be odd (got %d)", what, k);
    if (H < 2 || W < 2)
        return fail(CF_ERR_INVALID, "%s: BlurPool's reflect padding needs H, W >= 2 (H=%d W=%d)", what, H, W);
    if (C % CF_GROUP_WIDTH)
        return fail(CF_ERR_INVALID, "%s: C=%d is not a multiple of the group width %d", what, C, CF_GROUP_WIDTH);
    if ((int)dt != CF_F16 && (int)dt != CF_BF16)
        return fail(CF_ERR_INVALID, "%s: unknown dtype %d", what, (int)dt);
    if ((int)act != CF_ACT_GELU_ERF && (int)act != CF_ACT_RELU && (int)act != CF_ACT_NONE)
        return fail(CF_ERR_INVALID, "%s: unknown activation %d", what, (int)act);
    if ((double)N * H * W * C > 4.0e12 || (double)R * C > 1.0e7 || (double)K * R > 1.0e7)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {x, y, p->gw_w, p->w1, p->w2, p->gw_scale, p->gw_bias, p->s1, p->b1, p->s2, p->b2};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    const size_t xbytes = (size_t)N * H * W * C * elem_bytes(dt);
    const size_t ybytes = (size_t)N * ((H + 1) / 2) * ((W + 1) / 2) * K * elem_bytes(dt);
    if (overlap(x, xbytes, y, ybytes))
        return fail(CF_ERR_INVALID, "%s: x and y overlap", what);
    if (k != 3)
        return fail(CF_ERR_UNSUPPORTED, "%s: k=%d has no kernel (supported: 3)", what, k);
    if (!cf::convfirst_s2_supported(H, W, C, R, K))
        return fail(CF_ERR_UNSUPPORTED,
                    "%s: no kernel for C=%d R=%d K=%d (supported: C = 16, 24, 32, 48, 64; R a multiple of 16 "
                    "up to 1024; K a multiple of 8 up to 128)",
                    what, C, R, K);
    if ((double)N * H * W > 2147483647.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: N*H*W must stay below 2^31 pixels", what);
    cf::BlockW w;
    w.dw_w = p->gw_w;
    w.s0 = p->gw_scale;
    w.b0 = p->gw_bias;
    w.w1 = p->w1;
    w.s1 = p->s1;
    w.b1 = p->b1;
    w.w2 = p->w2;
    w.s2 = p->s2;
    w.b2 = p->b2;
    hipError_t e = cf::launch_convfirst_s2(x, y, w, N, H, W, C, R, K, dt == CF_BF16, (int)act, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_stem_forward(const void *x, void *y, const cf_stem_params *p, int N, int Hin, int Win, int C,
                          cf_dtype dt, void *stream) {
    const char *what = "cf_stem_forward";
    cf_status st = check_stem(what, x, y, p, N, Hin, Win, C, dt);
    if (st != CF_OK)
        return st;
    if (C != 16 && C != 24 && C != 32)
        return fail(CF_ERR_UNSUPPORTED, "%s: C=%d has no kernel (supported: 16, 24, 32)", what, C);
    hipError_t e = cf::launch_stem(to_stem(x, p, Hin, Win), y, N, C, dt == CF_BF16, (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

cf_status cf_stem_gblock_forward(const void *x, void *y, const cf_stem_params *stem, const cf_gblock_params *p,
                                 int N, int Hin, int Win, int C, int E, int k, cf_dtype dt, cf_act act,
                                 void *stream) {
    const char *what = "cf_stem_gblock_forward";
    cf_status st = check_stem(what, x, y, stem, N, Hin, Win, C, dt);
    if (st != CF_OK)
        return st;
    if (!p || !p->gw_w || !p->w1 || !p->w2)
        return fail(CF_ERR_INVALID, "%s: block params, gw_w, w1 and w2 must be non-NULL", what);
    if (E <= 0 || k <= 0 || k % 2 == 0 || k > 7)
        return fail(CF_ERR_INVALID, "%s: E must be positive and k odd up to 7 (E=%d k=%d)", what, E, k);
    if ((int)act != CF_ACT_GELU_ERF && (int)act != CF_ACT_RELU && (int)act != CF_ACT_NONE)
        return fail(CF_ERR_INVALID, "%s: unknown activation %d", what, (int)act);
    if ((double)E * C > 65536.0)
        return fail(CF_ERR_INVALID, "%s: tensor too large", what);
    const void *ptrs[] = {p->gw_w, p->w1, p->w2, p->gw_scale, p->gw_bias, p->s1, p->b1, p->s2, p->b2};
    for (const void *q : ptrs)
        if (q && !aligned16(q))
            return fail(CF_ERR_INVALID, "%s: every tensor pointer must be 16-byte aligned", what);
    if (k != 3)
        return fail(CF_ERR_UNSUPPORTED, "%s: k=%d has no kernel (supported: 3)", what, k);
    if (C != 16 && C != 32)
        return fail(CF_ERR_UNSUPPORTED, "%s: C=%d has no kernel (supported: 16, 32)", what, C);
    const int Hs = (Hin + 1) / 2, Ws = (Win + 1) / 2;
    if ((double)Ws * C * 6.0 > 2147483647.0)
        return fail(CF_ERR_UNSUPPORTED, "%s: image too wide", what);
    cf::GBlockW w;
    w.gw = p->gw_w;
    w.s0 = p->gw_scale;
    w.b0 = p->gw_bias;
    w.w1 = p->w1;
    w.s1 = p->s1;
    w.b1 = p->b1;
    w.w2 = p->w2;
    w.s2 = p->s2;
    w.b2 = p->b2;
    hipError_t e = cf::launch_stem_gblock(to_stem(x, stem, Hin, Win), y, w, to_shape(N, Hs, Ws, C, E, k, dt, act),
                                          (hipStream_t)stream);
    if (e != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

size_t cf_mbconv_workspace_bytes(int N, int H, int W, int C, int E, int R, cf_dtype dt) {
    return mbconv_ws(N, H, W, C, E, R, 0, dt);
}

size_t cf_mbconv_s2_workspace_bytes(int N, int H, int W, int C, int E, int R, int K, cf_dtype dt) {
    return K > 0 ? mbconv_ws(N, H, W, C, E, R, K, dt) : 0;
}

cf_status cf_mbconv_forward(const void *x, void *y, void *ws, size_t ws_bytes, const cf_mbconv_params *p, int N,
                            int H, int W, int C, int E, int R, int k, cf_dtype dt, cf_launch launch, void *stream) {
    return mbconv_call("cf_mbconv_forward", x, y, ws, ws_bytes, p, N, H, W, C, E, R, 0, k, dt, launch, stream);
}

cf_status cf_mbconv_s2_forward(const void *x, void *y, void *ws, size_t ws_bytes, const cf_mbconv_params *p, int N,
                               int H, int W, int C, int E, int R, int K, int k, cf_dtype dt, cf_launch launch,
                               void *stream) {
    if (K <= 0)
        return fail(CF_ERR_INVALID, "cf_mbconv_s2_forward: K must be positive (got %d)", K);
    return mbconv_call("cf_mbconv_s2_forward", x, y, ws, ws_bytes, p, N, H, W, C, E, R, K, k, dt, launch, stream);
}

cf_status cf_block_autotune(const void *x, void *y, const cf_block_params *p, int N, int H, int W, int C, int E,
                            int k, cf_dtype dt, cf_act act, void *stream) {
    const char *what = "cf_block_autotune";
    cf_status st = check_block(what, x, y, p, N, H, W, C, E, k, dt, act);
    if (st != CF_OK)
        return st;
    cf::Shape s = to_shape(N, H, W, C, E, k, dt, act);
    if ((st = check_fit(what, s)) != CF_OK)
        return st;
    hipStream_t strm = (hipStream_t)stream;
    hipEvent_t e0, e1;
    hipError_t e;
    if ((e = hipEventCreate(&e0)) != hipSuccess)
        return hip_fail(e, what);
    if ((e = hipEventCreate(&e1)) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return hip_fail(e, what);
    }
    int best = cf::CFG_DEFAULT;
    float best_ms = 0.0f;
    for (int cfg = 0; cfg < cf::CFG_COUNT; cfg++) {
        s.cfg = cfg;
        if (!cf::cfg_applies(s, cfg))
            continue;
        // one untimed launch, then three timed ones
        if ((e = cf::launch_fused_block(x, y, to_w(p), s, 1, nullptr, strm)) != hipSuccess)
            break;
        (void)hipEventRecord(e0, strm);
        for (int r = 0; r < 3 && e == hipSuccess; r++)
            e = cf::launch_fused_block(x, y, to_w(p), s, 1, nullptr, strm);
        (void)hipEventRecord(e1, strm);
        if (e != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess)
            break;
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, e0, e1);
        if (cfg == cf::CFG_DEFAULT || ms < best_ms) {
            best = cfg;
            best_ms = ms;
        }
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (e != hipSuccess)
        return hip_fail(e, what);
    {
        std::lock_guard<std::mutex> lk(g_tune_mu);
        g_tune[tune_key(s)] = best;
    }
    // leave y holding the output of the chosen configuration
    s.cfg = best;
    if ((e = cf::launch_fused_block(x, y, to_w(p), s, 1, nullptr, strm)) != hipSuccess ||
        (e = hipStreamSynchronize(strm)) != hipSuccess)
        return hip_fail(e, what);
    g_err[0] = 0;
    return CF_OK;
}

int cf_block_tuned_config(int N, int H, int W, int C, int E, int k, cf_dtype dt, cf_act act) {
    if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || E <= 0 || k <= 0 || (dt != CF_F16 && dt != CF_BF16) ||
        (act != CF_ACT_GELU_ERF && act != CF_ACT_RELU && act != CF_ACT_NONE))
        return -1;
    return tuned_config(to_shape(N, H, W, C, E, k, dt, act));
}

}  // extern "C"
