// C ABI of the MoE decode library: argument validation, workspace carve-up and the
// launch sequence of one decode step.  Declared in include/moe_decode.h.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>

#include "../../include/moe_decode.h"
#include "moe_internal.h"

namespace moe {

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

size_t carve_workspace(int H, int E, int I, int kmax, int Tmax, int wfmt, void *base, Workspace *ws)
{
    const size_t P = (size_t)Tmax * kmax;  // (token, choice) pairs = slots
    const MetaIdx mi{E, max_mfma_chunks(E, Tmax, kmax)};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return (char *)base + o;
    };
    Workspace w = {};
    w.logits = (float *)take(sizeof(float) * (size_t)Tmax * E);
    w.ids = (int32_t *)take(sizeof(int32_t) * P);
    w.wts = (float *)take(sizeof(float) * P);
    w.meta = (int32_t *)take(sizeof(int32_t) * (size_t)mi.words());
    w.slot_of = (int32_t *)take(sizeof(int32_t) * P);
    w.tok_of = (int32_t *)take(sizeof(int32_t) * P);
    w.h = (float *)take(sizeof(float) * P * I);
    w.o = (float *)take(sizeof(float) * P * H);
    w.sync = (int32_t *)take(sizeof(int32_t) * ((size_t)Tmax + 2) * kCounterStride);
    if (wfmt == MOE_WFMT_NVFP4_E2M1_B16) {
        w.hb = (__bf16 *)take(2 * P * I);
        w.x16 = (_Float16 *)take((size_t)2 * Tmax * H);
        w.xk = (int32_t *)take(sizeof(int32_t) * (size_t)Tmax);
    } else {
        w.xs_hi = (uint8_t *)take((size_t)Tmax * H);
        w.xs_lo = (uint8_t *)take((size_t)Tmax * H);
        w.xe_hi = (uint8_t *)take((size_t)Tmax * H / 32);
        w.xe_lo = (uint8_t *)take((size_t)Tmax * H / 32);
        w.hs_hi = (uint8_t *)take(P * I);
        w.hs_lo = (uint8_t *)take(P * I);
        w.he_hi = (uint8_t *)take(P * I / 32);
        w.he_lo = (uint8_t *)take(P * I / 32);
    }
    w.ks_max = screen_ks_max(H, E, Tmax);
    if (w.ks_max) {
        w.part = take((size_t)16 * w.ks_max * Tmax * E);
        w.xmax = (float *)take(sizeof(float) * (size_t)w.ks_max * Tmax);
        w.wmax = (float *)take(sizeof(float) * (size_t)w.ks_max * E);
    }
    w.bytes = off;
    if (ws) *ws = w;
    return off;
}

}  // namespace moe

using namespace moe;

struct moe_decode_s {
    moe_decode_config cfg;
    Layer L;
    Workspace ws;
    int mstar;  // MFMA threshold in tokens per expert (<= 0: GEMV only)
    int screen_min;  // screened routing from this many tokens per step (INT32_MAX: never)
    int synced;  // routing counters zeroed (by the first call on this handle)
    hipStream_t last_stream;
    int last_T;
    char err[256];
    // profiler
    int prof_cap, prof_n;
    hipEvent_t *prof_ev;  // [prof_cap][MOE_N_STAGES + 1]
};

static thread_local char g_init_err[256];

// Experts with at least this many tokens in a step run on MFMA tiles by default.
// Measured on MI355X at the 235B-shaped layer: the MFMA path (two-term FP8 split
// activations) streams an expert faster than the GEMV path already at one token,
// so by default every expert runs on MFMA tiles.
static const int kDefaultMfmaMinTokens = 1;

#define FAIL(buf, code, ...)            \
    do {                                \
        snprintf(buf, 256, __VA_ARGS__); \
        return code;                    \
    } while (0)

static moe_status check_config(const moe_decode_config *c, char *err)
{
    if (!c) FAIL(err, MOE_ERR_INVALID, "config is NULL");
    for (int i = 0; i < 5; ++i)
        if (c->reserved[i] != 0) FAIL(err, MOE_ERR_INVALID, "config.reserved[%d] must be zero", i);
    if (c->wfmt != MOE_WFMT_FP8_E4M3_B128 && c->wfmt != MOE_WFMT_MXFP4_E2M1_B32 && c->wfmt != MOE_WFMT_NVFP4_E2M1_B16)
        FAIL(err, MOE_ERR_INVALID, "unknown weight format %d", c->wfmt);
    const int q = c->wfmt == MOE_WFMT_FP8_E4M3_B128 ? 128 : 256;
    if (c->hidden <= 0 || c->hidden % q) FAIL(err, MOE_ERR_INVALID, "hidden=%d must be a positive multiple of %d", c->hidden, q);
    if (c->inter <= 0 || c->inter % q) FAIL(err, MOE_ERR_INVALID, "inter=%d must be a positive multiple of %d", c->inter, q);
    if (c->n_experts < 1 || c->n_experts > 1024) FAIL(err, MOE_ERR_INVALID, "n_experts=%d outside 1..1024", c->n_experts);
    const int kcap = c->n_experts < 64 ? c->n_experts : 64;
    if (c->max_topk < 1 || c->max_topk > kcap) FAIL(err, MOE_ERR_INVALID, "max_topk=%d outside 1..%d", c->max_topk, kcap);
    if (c->max_tokens < 1 || c->max_tokens > 1024) FAIL(err, MOE_ERR_INVALID, "max_tokens=%d outside 1..1024", c->max_tokens);
    if ((long)c->n_experts * ((c->max_tokens + 31) / 32) > 8192)
        FAIL(err, MOE_ERR_INVALID, "n_experts * ceil(max_tokens/32) = %ld exceeds 8192",
             (long)c->n_experts * ((c->max_tokens + 31) / 32));
    if (c->act_dtype != MOE_DTYPE_F32 && c->act_dtype != MOE_DTYPE_BF16)
        FAIL(err, MOE_ERR_INVALID, "unknown act_dtype %d", c->act_dtype);
    if (c->router_dtype != MOE_DTYPE_F32 && c->router_dtype != MOE_DTYPE_BF16)
        FAIL(err, MOE_ERR_INVALID, "unknown router_dtype %d", c->router_dtype);
    if (c->weight_layout != MOE_WLAYOUT_ROW_MAJOR && c->weight_layout != MOE_WLAYOUT_TILED16)
        FAIL(err, MOE_ERR_INVALID, "unknown weight_layout %d", c->weight_layout);
    if (c->weight_layout == MOE_WLAYOUT_TILED16 && c->mfma_min_tokens != 0 && c->mfma_min_tokens != 1)
        FAIL(err, MOE_ERR_UNSUPPORTED, "packed 16-row tiles need MFMA tiles for every expert (mfma_min_tokens 0 or 1)");
    if (c->wfmt == MOE_WFMT_NVFP4_E2M1_B16 && c->act_dtype != MOE_DTYPE_BF16)
        FAIL(err, MOE_ERR_UNSUPPORTED, "NVFP4 weights need bf16 activations (the bf16 matrix cores take x as it is)");
    {
        // The GEMV path stages 4 activation rows of max(H, I) elements in LDS.  The
        // bound also keeps the MFMA path's 32-bit buffer offsets (T*H and T*k*I
        // bytes of split activations) below 2^31.
        const long stage = 4L * (c->hidden > c->inter ? c->hidden : c->inter) * (c->act_dtype == MOE_DTYPE_BF16 ? 2 : 4);
        if (stage > 65536)
            FAIL(err, MOE_ERR_UNSUPPORTED, "activation staging of %ld bytes exceeds 64 KiB of LDS", stage);
    }
    return MOE_OK;
}

extern "C" {

size_t moe_decode_workspace_bytes(const moe_decode_config *cfg)
{
    char err[256];
    if (check_config(cfg, err) != MOE_OK) return 0;
    return carve_workspace(cfg->hidden, cfg->n_experts, cfg->inter, cfg->max_topk, cfg->max_tokens, cfg->wfmt, nullptr,
                           nullptr);
}

size_t moe_decode_expert_weight_bytes(const moe_decode_config *cfg)
{
    char err[256];
    if (check_config(cfg, err) != MOE_OK) return 0;
    const size_t H = cfg->hidden, I = cfg->inter;
    return cfg->wfmt == MOE_WFMT_FP8_E4M3_B128 ? 3 * H * I : 3 * H * I / 2;
}

size_t moe_decode_expert_scale_bytes(const moe_decode_config *cfg)
{
    char err[256];
    if (check_config(cfg, err) != MOE_OK) return 0;
    const size_t H = cfg->hidden, I = cfg->inter;
    if (cfg->wfmt == MOE_WFMT_FP8_E4M3_B128) return 4 * 3 * (H / 128) * (I / 128);
    if (cfg->wfmt == MOE_WFMT_MXFP4_E2M1_B32) return 3 * H * I / 32;
    return 16 + 3 * H * I / 16;
}

}  // extern "C"

// Fill a handle for a validated configuration whose workspace starts at `workspace`.
static void fill_handle(moe_decode_s *h, const moe_decode_config *cfg, void *workspace)
{
    h->cfg = *cfg;
    h->L.H = cfg->hidden;
    h->L.E = cfg->n_experts;
    h->L.I = cfg->inter;
    h->L.wfmt = cfg->wfmt;
    h->L.act_bf16 = cfg->act_dtype == MOE_DTYPE_BF16;
    h->L.router_bf16 = cfg->router_dtype == MOE_DTYPE_BF16;
    h->L.wlayout = cfg->weight_layout;
    h->L.expert_w_bytes = moe_decode_expert_weight_bytes(cfg);
    h->L.expert_s_bytes = moe_decode_expert_scale_bytes(cfg);
    carve_workspace(cfg->hidden, cfg->n_experts, cfg->inter, cfg->max_topk, cfg->max_tokens, cfg->wfmt, workspace,
                    &h->ws);
    h->mstar = cfg->mfma_min_tokens == 0 ? kDefaultMfmaMinTokens : (cfg->mfma_min_tokens < 0 ? 0 : cfg->mfma_min_tokens);
    {
        // screened routing: bf16 x and router, H a multiple of 256 (ks_max > 0), E <= 1024
        const long work = (long)cfg->n_experts * cfg->hidden;
        const int dflt = (int)((kScreenMinMacs + work - 1) / work);
        const bool able = h->ws.ks_max > 0 && h->L.act_bf16 && h->L.router_bf16;
        h->screen_min = !able || cfg->screen_min_tokens < 0 ? INT32_MAX
                        : cfg->screen_min_tokens == 0    ? dflt
                                                         : cfg->screen_min_tokens;
    }
    h->synced = 0;
    h->last_stream = nullptr;
    h->last_T = -1;
    h->err[0] = 0;
    h->prof_cap = h->prof_n = 0;
    h->prof_ev = nullptr;
}

extern "C" {

moe_status moe_decode_init(const moe_decode_config *cfg, void *workspace, size_t workspace_bytes, moe_decode_t *out)
{
    g_init_err[0] = 0;
    if (!out) FAIL(g_init_err, MOE_ERR_INVALID, "out is NULL");
    *out = nullptr;
    moe_status s = check_config(cfg, g_init_err);
    if (s != MOE_OK) return s;
    const size_t need = moe_decode_workspace_bytes(cfg);
    if (!workspace) FAIL(g_init_err, MOE_ERR_WORKSPACE, "workspace is NULL");
    if ((uintptr_t)workspace % 256) FAIL(g_init_err, MOE_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (workspace_bytes < need)
        FAIL(g_init_err, MOE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    moe_decode_s *h = new (std::nothrow) moe_decode_s();
    if (!h) FAIL(g_init_err, MOE_ERR_INVALID, "out of host memory");
    fill_handle(h, cfg, workspace);
    *out = h;
    return MOE_OK;
}

static bool overlap(const void *p, const void *q, size_t bytes)
{
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + bytes && b < a + bytes;
}

moe_status moe_decode_pack_weights(const moe_decode_config *cfg, void *stream, const void *src, void *dst,
                                   const void *src_scales, void *dst_scales, int32_t n_experts)
{
    g_init_err[0] = 0;
    moe_status s = check_config(cfg, g_init_err);
    if (s != MOE_OK) return s;
    if (n_experts < 1 || n_experts > cfg->n_experts)
        FAIL(g_init_err, MOE_ERR_INVALID, "n_experts=%d outside 1..%d", n_experts, cfg->n_experts);
    if (!src || !dst) FAIL(g_init_err, MOE_ERR_INVALID, "src or dst is NULL");
    if ((uintptr_t)src % 16 || (uintptr_t)dst % 16) FAIL(g_init_err, MOE_ERR_INVALID, "src and dst must be 16-byte aligned");
    const size_t bytes = (size_t)n_experts * moe_decode_expert_weight_bytes(cfg);
    if (overlap(src, dst, bytes)) FAIL(g_init_err, MOE_ERR_INVALID, "src and dst overlap");
    const bool nv = cfg->wfmt != MOE_WFMT_FP8_E4M3_B128;  // E2M1 weights: their scales are packed too
    if (nv) {
        if (!src_scales || !dst_scales) FAIL(g_init_err, MOE_ERR_INVALID, "MXFP4 and NVFP4 scales need src_scales and dst_scales");
        if ((uintptr_t)src_scales % 4 || (uintptr_t)dst_scales % 4)
            FAIL(g_init_err, MOE_ERR_INVALID, "src_scales and dst_scales must be 4-byte aligned");
        if (overlap(src_scales, dst_scales, (size_t)n_experts * moe_decode_expert_scale_bytes(cfg)))
            FAIL(g_init_err, MOE_ERR_INVALID, "src_scales and dst_scales overlap");
    } else if (src_scales || dst_scales) {
        FAIL(g_init_err, MOE_ERR_INVALID, "FP8 scales keep their layout: pass NULL scale pointers");
    }
    Layer L = {};
    L.H = cfg->hidden;
    L.E = cfg->n_experts;
    L.I = cfg->inter;
    L.wfmt = cfg->wfmt;
    L.expert_w_bytes = moe_decode_expert_weight_bytes(cfg);
    L.expert_s_bytes = moe_decode_expert_scale_bytes(cfg);
    if (launch_pack_weights(L, src, dst, n_experts, (hipStream_t)stream) != hipSuccess)
        FAIL(g_init_err, MOE_ERR_HIP, "pack kernel launch failed");
    if (nv && launch_pack_scales(L, src_scales, dst_scales, n_experts, (hipStream_t)stream) != hipSuccess)
        FAIL(g_init_err, MOE_ERR_HIP, "scale pack kernel launch failed");
    return MOE_OK;
}

static moe_status check_ptr(moe_decode_t h, const void *p, const char *name, int align, bool nullable)
{
    if (!p) {
        if (nullable) return MOE_OK;
        FAIL(h->err, MOE_ERR_INVALID, "%s is NULL", name);
    }
    if ((uintptr_t)p % align) FAIL(h->err, MOE_ERR_INVALID, "%s is not %d-byte aligned", name, align);
    return MOE_OK;
}

#define CHECK(expr)                     \
    do {                                \
        moe_status _s = (expr);         \
        if (_s != MOE_OK) return _s;    \
    } while (0)

#define HIPCHECK(h, expr)                                                                  \
    do {                                                                                   \
        hipError_t _e = (expr);                                                            \
        if (_e != hipSuccess) FAIL((h)->err, MOE_ERR_HIP, "%s: %s", #expr, hipGetErrorString(_e)); \
    } while (0)

static moe_status check_common(moe_decode_t h, const void *x, int32_t T, const void *router_w, const float *bias,
                               int32_t topk, const int32_t *ids, const float *wts)
{
    if (!h) return MOE_ERR_INVALID;
    h->err[0] = 0;
    if (T < 0 || T > h->cfg.max_tokens)
        FAIL(h->err, MOE_ERR_INVALID, "n_tokens=%d outside 0..%d", T, h->cfg.max_tokens);
    if (topk < 1 || topk > h->cfg.max_topk)
        FAIL(h->err, MOE_ERR_INVALID, "topk=%d outside 1..%d", topk, h->cfg.max_topk);
    CHECK(check_ptr(h, x, "x", 16, false));
    CHECK(check_ptr(h, router_w, "router_w", 16, false));
    CHECK(check_ptr(h, bias, "router_bias", 4, true));
    CHECK(check_ptr(h, ids, "topk_ids", 4, true));
    CHECK(check_ptr(h, wts, "topk_weights", 4, true));
    return MOE_OK;
}

static void prof_mark(moe_decode_t h, int stage_boundary, hipStream_t st)
{
    if (h->prof_n < h->prof_cap) hipEventRecord(h->prof_ev[h->prof_n * (MOE_N_STAGES + 1) + stage_boundary], st);
}

static moe_status ensure_synced(moe_decode_t h, hipStream_t st)
{
    if (!h->synced) {
        HIPCHECK(h, launch_zero(h->ws.sync, (h->cfg.max_tokens + 2) * kCounterStride, st));
        h->synced = 1;
    }
    return MOE_OK;
}

static RouteParams route_params(moe_decode_t h, const void *x, int T, int k, const void *router_w, const float *bias,
                                int32_t *ids_user, float *wts_user, bool split, bool group)
{
    const Workspace &w = h->ws;
    RouteParams P;
    P.x = x;
    P.T = T;
    P.k = k;
    P.router_w = router_w;
    P.bias = bias;
    P.logits = w.logits;
    P.ids = w.ids;
    P.ids_user = ids_user;
    P.wts = w.wts;
    P.wts_user = wts_user;
    P.meta = w.meta;
    P.slot_of = w.slot_of;
    P.tok_of = w.tok_of;
    P.cnt_tok = w.sync;
    P.cnt_all = w.sync + (size_t)h->cfg.max_tokens * kCounterStride;
    P.fb_acc = w.sync + ((size_t)h->cfg.max_tokens + 1) * kCounterStride;
    P.xs_hi = split && w.xs_hi ? w.xs_hi : nullptr;
    P.x16 = split && w.x16 ? w.x16 : nullptr;
    P.xk = w.xk;
    P.xs_lo = w.xs_lo;
    P.xe_hi = w.xe_hi;
    P.xe_lo = w.xe_lo;
    P.part = w.part;
    P.xmax = w.xmax;
    P.wmax = w.wmax;
    P.ks_max = w.ks_max;
    P.Tmax = h->cfg.max_tokens;
    P.mstar = h->mstar;
    P.screen = T >= h->screen_min ? 1 : 0;
    P.do_group = group ? 1 : 0;
    P.max_chunks = max_mfma_chunks(h->L.E, h->cfg.max_tokens, h->cfg.max_topk);
    return P;
}

moe_status moe_decode_route(moe_decode_t h, void *stream, const void *x, int32_t n_tokens, const void *router_w,
                            const float *router_bias, int32_t topk, float *logits, int32_t *topk_ids,
                            float *topk_weights)
{
    CHECK(check_common(h, x, n_tokens, router_w, router_bias, topk, topk_ids, topk_weights));
    CHECK(check_ptr(h, logits, "logits", 4, true));
    if (n_tokens == 0) return MOE_OK;
    hipStream_t st = (hipStream_t)stream;
    CHECK(ensure_synced(h, st));
    const RouteParams P = route_params(h, x, n_tokens, topk, router_w, router_bias, topk_ids, topk_weights, false, false);
    HIPCHECK(h, launch_route(h->L, P, st));
    if (logits)
        HIPCHECK(h, hipMemcpyAsync(logits, h->ws.logits, sizeof(float) * (size_t)n_tokens * h->L.E,
                                   hipMemcpyDeviceToDevice, st));
    return MOE_OK;
}

moe_status moe_decode_forward(moe_decode_t h, void *stream, const void *x, int32_t n_tokens, const void *router_w,
                              const float *router_bias, const void *expert_w, const void *scales, int32_t topk,
                              void *y, int32_t *topk_ids, float *topk_weights)
{
    CHECK(check_common(h, x, n_tokens, router_w, router_bias, topk, topk_ids, topk_weights));
    CHECK(check_ptr(h, expert_w, "expert_w", 16, false));
    CHECK(check_ptr(h, scales, "scales", 4, false));
    CHECK(check_ptr(h, y, "y", 16, false));
    if (y == x) FAIL(h->err, MOE_ERR_INVALID, "y must not alias x");
    hipStream_t st = (hipStream_t)stream;
    h->last_stream = st;
    h->last_T = n_tokens;
    if (n_tokens == 0) return MOE_OK;
    const Workspace &w = h->ws;
    const Layer &L = h->L;
    const int T = n_tokens, k = topk;
    const bool prof = h->prof_n < h->prof_cap;
    // Expert paths this step can use: MFMA tiles for experts with >= mstar tokens
    // (impossible when T < mstar), the GEMV path for the others (none when mstar <= 1).
    const bool mfma = h->mstar > 0 && T >= h->mstar;
    const bool gemv = h->mstar != 1;
    CHECK(ensure_synced(h, st));
    if (prof) prof_mark(h, 0, st);
    // The MFMA kernels read x as the routing kernel rewrites it: FP8 and MXFP4 ones its
    // 2-term FP8 split, NVFP4 ones an f16 copy scaled per token by a power of two.
    const bool nv = L.wfmt == MOE_WFMT_NVFP4_E2M1_B16;
    const RouteParams P = route_params(h, x, T, k, router_w, router_bias, topk_ids, topk_weights, mfma, true);
    HIPCHECK(h, launch_route(L, P, st));
    if (prof) prof_mark(h, 1, st);
    if (gemv) HIPCHECK(h, launch_w13(L, expert_w, scales, x, T, k, w.meta, w.tok_of, w.h, st));
    if (mfma && nv) HIPCHECK(h, launch_w13_nvfp4(L, expert_w, scales, T, k, w.meta, w.tok_of, w, st));
    if (mfma && !nv) HIPCHECK(h, launch_w13_mfma(L, expert_w, scales, T, k, w.meta, w.tok_of, w, st));
    if (prof) prof_mark(h, 2, st);
    if (gemv) HIPCHECK(h, launch_w2(L, expert_w, scales, T, k, w.meta, w.h, w.o, st));
    if (mfma && nv) HIPCHECK(h, launch_w2_nvfp4(L, expert_w, scales, T, k, w.meta, w, st));
    if (mfma && !nv) HIPCHECK(h, launch_w2_mfma(L, expert_w, scales, T, k, w.meta, w, st));
    if (prof) prof_mark(h, 3, st);
    HIPCHECK(h, launch_combine(L, T, k, w.slot_of, w.wts, w.o, y, st));
    if (prof) {
        prof_mark(h, 4, st);
        h->prof_n++;
    }
    return MOE_OK;
}

}  // extern "C"

// ---- forward without allocation: the workspace is a static device array.
//
// Layout of `scratch`: the routing counters first, sized for the largest token count
// any configuration accepts (1024), then the workspace of the call's configuration,
// carved as for a handle.  The counters are zero when the code object is loaded
// (static storage), are cleared once more when a device is set up, and every forward
// call leaves them at zero again (each counter is reset by the workgroup that
// consumes it), so nothing has to be cleared per call.
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr size_t kScratchCounterBytes =
    ((size_t)(1024 + 2) * kCounterStride * sizeof(int32_t) + 255) & ~(size_t)255;
constexpr int kScratchMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static void *g_scratch_dev[kScratchMaxDevices];  // device address of `scratch` on each device

// Device address of this device's copy of `scratch` (set up on the first call on the
// device, with that device current).  Host code never uses the array's own name: on
// the host it is a stand-in, not a device address.
static moe_status scratch_base(hipStream_t st, void **out, char *err)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) FAIL(err, MOE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (st) {
        hipDevice_t sdev = -1;
        e = hipStreamGetDevice(st, &sdev);
        if (e != hipSuccess) FAIL(err, MOE_ERR_HIP, "hipStreamGetDevice: %s", hipGetErrorString(e));
        if (sdev != dev) FAIL(err, MOE_ERR_INVALID, "the stream belongs to device %d but device %d is current", (int)sdev, dev);
    }
    if (dev < 0 || dev >= kScratchMaxDevices) FAIL(err, MOE_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kScratchMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            FAIL(err, MOE_ERR_HIP, "hipGetSymbolAddress(scratch): %s", e != hipSuccess ? hipGetErrorString(e) : "NULL");
        e = launch_zero((int32_t *)p, (int)(kScratchCounterBytes / sizeof(int32_t)), st);
        if (e != hipSuccess) FAIL(err, MOE_ERR_HIP, "clearing the scratch counters: %s", hipGetErrorString(e));
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return MOE_OK;
}

extern "C" {

moe_status moe_decode_forward_noalloc(const moe_decode_config *cfg, void *stream, const void *x, int32_t n_tokens,
                                      const void *router_w, const float *router_bias, const void *expert_w,
                                      const void *scales, int32_t topk, void *y, int32_t *topk_ids,
                                      float *topk_weights)
{
    g_init_err[0] = 0;
    moe_status s = check_config(cfg, g_init_err);
    if (s != MOE_OK) return s;
    const size_t need = moe_decode_workspace_bytes(cfg);
    if (need > kScratchBytes - kScratchCounterBytes)
        FAIL(g_init_err, MOE_ERR_WORKSPACE, "the configuration needs %zu bytes of workspace; the static scratch holds %zu",
             need, kScratchBytes - kScratchCounterBytes);
    void *base = nullptr;
    s = scratch_base((hipStream_t)stream, &base, g_init_err);
    if (s != MOE_OK) return s;
    moe_decode_s h{};  // on the stack: no allocation of any kind
    fill_handle(&h, cfg, (char *)base + kScratchCounterBytes);
    h.ws.sync = (int32_t *)base;
    h.synced = 1;
    s = moe_decode_forward(&h, stream, x, n_tokens, router_w, router_bias, expert_w, scales, topk, y, topk_ids,
                           topk_weights);
    if (s != MOE_OK) memcpy(g_init_err, h.err, sizeof g_init_err);
    return s;
}

moe_status moe_decode_get_stats(moe_decode_t h, moe_decode_stats *out, int32_t *counts_host)
{
    if (!h) return MOE_ERR_INVALID;
    if (!out) FAIL(h->err, MOE_ERR_INVALID, "out is NULL");
    memset(out, 0, sizeof *out);
    if (h->last_T < 0) FAIL(h->err, MOE_ERR_INVALID, "no forward call on this handle yet");
    out->n_tokens = h->last_T;
    if (h->last_T == 0) {
        if (counts_host) memset(counts_host, 0, sizeof(int32_t) * h->L.E);
        return MOE_OK;
    }
    HIPCHECK(h, hipStreamSynchronize(h->last_stream));
    const MetaIdx mi{h->L.E, max_mfma_chunks(h->L.E, h->cfg.max_tokens, h->cfg.max_topk)};
    int32_t head[8];
    HIPCHECK(h, hipMemcpy(head, h->ws.meta, sizeof head, hipMemcpyDeviceToHost));
    out->n_active = head[mi.n_active()];
    out->n_active_mfma = head[mi.n_mfma()];
    out->n_fallback = head[mi.n_fallback()];
    out->n_exact_logits = head[mi.n_exact()];
    out->route_screened = head[mi.screened()];
    out->active_weight_bytes = (int64_t)out->n_active * (int64_t)(h->L.expert_w_bytes + h->L.expert_s_bytes);
    if (counts_host)
        HIPCHECK(h, hipMemcpy(counts_host, h->ws.meta + mi.counts(), sizeof(int32_t) * h->L.E, hipMemcpyDeviceToHost));
    return MOE_OK;
}

static void prof_release(moe_decode_t h)
{
    if (h->prof_ev) {
        for (int i = 0; i < h->prof_cap * (MOE_N_STAGES + 1); ++i)
            if (h->prof_ev[i]) hipEventDestroy(h->prof_ev[i]);
        free(h->prof_ev);
    }
    h->prof_ev = nullptr;
    h->prof_cap = h->prof_n = 0;
}

moe_status moe_decode_profile_enable(moe_decode_t h, int32_t max_calls)
{
    if (!h) return MOE_ERR_INVALID;
    prof_release(h);
    if (max_calls <= 0) return MOE_OK;
    const int n = max_calls * (MOE_N_STAGES + 1);
    h->prof_ev = (hipEvent_t *)calloc((size_t)n, sizeof(hipEvent_t));
    if (!h->prof_ev) FAIL(h->err, MOE_ERR_INVALID, "out of host memory");
    h->prof_cap = max_calls;
    for (int i = 0; i < n; ++i) {
        hipError_t e = hipEventCreate(&h->prof_ev[i]);
        if (e != hipSuccess) {
            prof_release(h);
            FAIL(h->err, MOE_ERR_HIP, "hipEventCreate: %s", hipGetErrorString(e));
        }
    }
    return MOE_OK;
}

moe_status moe_decode_profile_read(moe_decode_t h, float *stage_ms, int32_t *n_calls)
{
    if (!h) return MOE_ERR_INVALID;
    if (!n_calls) FAIL(h->err, MOE_ERR_INVALID, "n_calls is NULL");
    *n_calls = h->prof_n;
    for (int c = 0; c < h->prof_n; ++c) {
        hipEvent_t *ev = h->prof_ev + c * (MOE_N_STAGES + 1);
        HIPCHECK(h, hipEventSynchronize(ev[MOE_N_STAGES]));
        for (int s = 0; s < MOE_N_STAGES; ++s) {
            float ms = 0.f;
            HIPCHECK(h, hipEventElapsedTime(&ms, ev[s], ev[s + 1]));
            if (stage_ms) stage_ms[c * MOE_N_STAGES + s] = ms;
        }
    }
    h->prof_n = 0;
    return MOE_OK;
}

void moe_decode_free(moe_decode_t h)
{
    if (!h) return;
    prof_release(h);
    delete h;
}

const char *moe_decode_status_string(moe_status s)
{
    switch (s) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported configuration";
    case MOE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case MOE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char *moe_decode_last_error(moe_decode_t h) { return h ? h->err : g_init_err; }

}  // extern "C"
