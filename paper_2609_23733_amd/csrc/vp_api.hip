// C ABI of libvggtprime.so (declared in include/vggt_prime.h): argument
// validation, workspace layout and launch sequencing on the caller's stream.
// Validation runs entirely on the host before anything is enqueued.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/vggt_prime.h"
#include "vp_internal.hpp"

namespace {

thread_local char g_err[512] = "";

constexpr int64_t kMaxTokens = (int64_t)1 << 28;   // 268M tokens: int32-safe grids
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Layout {
    int64_t N;
    int64_t n1, chunk1, n2, chunk2, nkt, n3, chunk3;
    size_t off_part1, off_part2, off_vt, off_kh, off_kmax, off_vpart, off_vsc, off_qflag,
        off_fpart, off_lpart, off_lsum, total;
};

// Chunking of the router reductions and the workspace carve-up; a pure
// function of the shape, shared by vp_workspace_bytes and the launches.
bool make_layout(const vp_shape* s, Layout* L) {
    if (!s) return false;
    if (s->S < 1 || s->P < 1 || s->S > kMaxTokens || s->P > kMaxTokens) return false;
    if (s->S * s->P > kMaxTokens) return false;
    if (s->H < 1 || s->H > VP_MAX_HEADS || s->d != VP_HEAD_DIM) return false;
    if (s->dtype != VP_F32 && s->dtype != VP_BF16) return false;
    const int64_t N = s->S * s->P;
    L->N = N;
    int64_t c1 = cdiv(N, 64);
    c1 = c1 < 256 ? 256 : cdiv(c1, 128) * 128;
    L->chunk1 = c1;
    L->n1 = cdiv(N, c1);
    int64_t c2 = cdiv(N, 512);
    L->chunk2 = c2 < 64 ? 64 : c2;
    L->n2 = cdiv(N, L->chunk2);
    L->nkt = cdiv(N, 64);
    // linear-attention chunks: at most 128 per head, whole 64-token tiles
    int64_t c3 = cdiv(cdiv(N, 128), 64) * 64;
    L->chunk3 = c3 < 256 ? 256 : c3;
    L->n3 = cdiv(N, L->chunk3);
    size_t off = kAlign;   // first 256 bytes reserved
    L->off_part1 = off;
    off = align_up(off + (size_t)L->n1 * s->H * (2 + VP_HEAD_DIM) * sizeof(float));
    L->off_part2 = off;
    off = align_up(off + (size_t)L->n2 * s->H * (2 + 2 * VP_HEAD_DIM) * sizeof(float));
    L->off_vt = off;
    if (s->dtype == VP_BF16) off = align_up(off + (size_t)s->H * L->nkt * 64 * 64 * 2);
    L->off_kh = off;
    if (s->dtype == VP_BF16) off = align_up(off + (size_t)s->H * L->nkt * 64 * 64 * 2);
    L->off_kmax = off;
    if (s->dtype == VP_BF16) off = align_up(off + (size_t)s->H * L->nkt * sizeof(float));
    L->off_vpart = off;
    if (s->dtype == VP_BF16)
        off = align_up(off + (size_t)s->H * vp::flash_vmax_parts(N) * sizeof(float));
    L->off_vsc = off;
    if (s->dtype == VP_BF16) off = align_up(off + (size_t)s->H * 2 * sizeof(float));
    L->off_qflag = off;
    if (s->dtype == VP_BF16)
        off = align_up(off + (size_t)s->H * cdiv(N, vp::flash_q_tile(VP_BF16)) * sizeof(int32_t));
    L->off_fpart = off;
    off = align_up(off + (s->dtype == VP_BF16 ? vp::flash_part_bytes(N, (int)s->H)
                                              : vp::flash_f32_part_bytes(N, (int)s->H)));
    L->off_lpart = off;
    off = align_up(off + (size_t)L->n3 * s->H * vp::kLinSums * sizeof(float));
    L->off_lsum = off;
    off = align_up(off + (size_t)s->H * vp::kLinSums * sizeof(float));
    L->total = off;
    return true;
}

vp_status shape_status(const vp_shape* s) {
    if (!s) return VP_ERR_INVALID_ARG;
    if (s->S < 1 || s->P < 1 || s->H < 1) return VP_ERR_INVALID_ARG;
    if (s->dtype != VP_F32 && s->dtype != VP_BF16) return VP_ERR_INVALID_ARG;
    if (s->S > kMaxTokens || s->P > kMaxTokens || s->S * s->P > kMaxTokens)
        return VP_ERR_UNSUPPORTED;
    if (s->H > VP_MAX_HEADS || s->d != VP_HEAD_DIM) return VP_ERR_UNSUPPORTED;
    return VP_OK;
}

vp_status check_ws(const vp_shape* s, void* ws, size_t ws_bytes, Layout* L) {
    if (!make_layout(s, L)) return VP_ERR_INVALID_ARG;
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    if (ws_bytes < L->total) return VP_ERR_WORKSPACE;
    return VP_OK;
}

vp_status hip_status(const char* where) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        snprintf(g_err, sizeof(g_err), "%s: %s", where, hipGetErrorString(e));
        return VP_ERR_HIP;
    }
    return VP_OK;
}

}  // namespace

extern "C" {

const char* vp_status_string(vp_status s) {
    switch (s) {
        case VP_OK: return "ok";
        case VP_ERR_INVALID_ARG: return "invalid argument";
        case VP_ERR_UNSUPPORTED: return "unsupported shape";
        case VP_ERR_WORKSPACE: return "workspace too small";
        case VP_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* vp_last_error(void) { return g_err; }

size_t vp_workspace_bytes(const vp_shape* shape) {
    Layout L;
    return make_layout(shape, &L) ? L.total : 0;
}

}  // extern "C"

namespace {

// Host-side checks of vp_router_score's arguments other than the workspace.
vp_status check_router(const vp_shape* shape, const void* Q, const void* K, const void* V,
                       const vp_router_weights* rw, const vp_router_state* out) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (!Q || !K || !V || !rw || !out) return VP_ERR_INVALID_ARG;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V)) return VP_ERR_INVALID_ARG;
    if (rw->pool != VP_POOL_GATED && rw->pool != VP_POOL_MEAN) return VP_ERR_INVALID_ARG;
    if (rw->pool == VP_POOL_GATED &&
        (!rw->W || !rw->U || !rw->w || !aligned16(rw->W) || !aligned16(rw->U) ||
         !aligned16(rw->w)))
        return VP_ERR_INVALID_ARG;
    if (rw->L != VP_HIDDEN) return VP_ERR_UNSUPPORTED;
    if (!isfinite(rw->scale) || rw->scale < 0.f) return VP_ERR_INVALID_ARG;
    if (!out->q_pool || !out->stats || !out->score || !out->ctx || !out->vmean)
        return VP_ERR_INVALID_ARG;
    if (!aligned16(out->q_pool) || !aligned16(out->ctx) || !aligned16(out->vmean))
        return VP_ERR_INVALID_ARG;
    return VP_OK;
}

// Enqueues the router with its partial sums at ws + L.off_part1 / L.off_part2.
vp_status launch_router_at(const vp_shape* shape, const Layout& L, const void* Q, const void* K,
                           const void* V, const vp_router_weights* rw, vp_router_state* out,
                           void* ws, void* stream, const char* where) {
    (void)hipGetLastError();
    vp::RouterArgs a;
    a.dtype = shape->dtype == VP_BF16 ? 1 : 0;
    a.Q = Q; a.K = K; a.V = V;
    a.W = rw->W; a.U = rw->U; a.w = rw->w;
    a.N = L.N;
    a.H = shape->H;
    a.n1 = L.n1; a.chunk1 = L.chunk1;
    a.part1 = (float*)((char*)ws + L.off_part1);
    a.n2 = L.n2; a.chunk2 = L.chunk2;
    a.part2 = (float*)((char*)ws + L.off_part2);
    a.scale = rw->scale > 0.f ? rw->scale : 1.f / sqrtf((float)shape->d);
    a.mean_pool = rw->pool == VP_POOL_MEAN ? 1 : 0;
    a.q_pool = out->q_pool; a.stats = out->stats; a.score = out->score;
    a.ctx = out->ctx; a.vmean = out->vmean;
    vp::launch_router(a, (hipStream_t)stream);
    return hip_status(where);
}

// Bytes of the workspace that the router uses (its partial sums, from offset 0).
size_t router_scratch_bytes(const vp_shape* shape, const Layout& L) {
    return align_up(L.off_part2 + (size_t)L.n2 * shape->H * (2 + 2 * VP_HEAD_DIM) * sizeof(float));
}

// Scratch of vp_router_score_noalloc: the router's partial sums (at most 64
// pooling chunks and 512 routing chunks of 16 heads, 4.32 MiB, for every
// shape the library accepts).  Each device holds its own copy for the life
// of the process; host code uses it only through the address that
// hipGetSymbolAddress returns on that device.
constexpr size_t kNoAllocScratchBytes = (size_t)9 << 19;   // 4.5 MiB
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first
// call made with that device current.
vp_status scratch_address(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        snprintf(g_err, sizeof(g_err), "vp_router_score_noalloc: hipGetDevice: %s",
                 hipGetErrorString(e));
        return VP_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        snprintf(g_err, sizeof(g_err), "vp_router_score_noalloc: device %d beyond %d", dev,
                 kMaxDevices);
        return VP_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            snprintf(g_err, sizeof(g_err), "vp_router_score_noalloc: hipGetSymbolAddress: %s",
                     hipGetErrorString(e));
            return VP_ERR_HIP;
        }
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return VP_OK;
}

}  // namespace

extern "C" {

vp_status vp_router_score(const vp_shape* shape, const void* Q, const void* K, const void* V,
                          const vp_router_weights* rw, vp_router_state* out, void* ws,
                          size_t ws_bytes, void* stream) {
    vp_status st = check_router(shape, Q, K, V, rw, out);
    if (st != VP_OK) return st;
    Layout L;
    if ((st = check_ws(shape, ws, ws_bytes, &L)) != VP_OK) return st;
    return launch_router_at(shape, L, Q, K, V, rw, out, ws, stream, "vp_router_score");
}

vp_status vp_router_score_noalloc(const vp_shape* shape, const void* Q, const void* K,
                                  const void* V, const vp_router_weights* rw,
                                  vp_router_state* out, void* stream) {
    vp_status st = check_router(shape, Q, K, V, rw, out);
    if (st != VP_OK) return st;
    Layout L;
    if (!make_layout(shape, &L)) return VP_ERR_INVALID_ARG;
    const size_t need = router_scratch_bytes(shape, L);
    if (need > kNoAllocScratchBytes) {
        snprintf(g_err, sizeof(g_err),
                 "vp_router_score_noalloc: %zu bytes of scratch needed, %zu available", need,
                 kNoAllocScratchBytes);
        return VP_ERR_WORKSPACE;
    }
    void* ws = nullptr;
    if ((st = scratch_address(&ws)) != VP_OK) return st;
    return launch_router_at(shape, L, Q, K, V, rw, out, ws, stream, "vp_router_score_noalloc");
}

vp_status vp_router_logits(const float* u, const void* W_r, const float* b_r, int32_t H,
                           int32_t Din, int32_t M, vp_dtype w_dtype, float* logits,
                           void* stream) {
    if (!u || !W_r || !b_r || !logits) return VP_ERR_INVALID_ARG;
    if (H < 1 || Din < 1 || Din > 65536 || M < 1) return VP_ERR_INVALID_ARG;
    if (H > VP_MAX_HEADS || M != VP_NUM_MODES) return VP_ERR_UNSUPPORTED;
    if (w_dtype != VP_F32 && w_dtype != VP_BF16) return VP_ERR_INVALID_ARG;
    if (((uintptr_t)u & 3u) || ((uintptr_t)b_r & 3u) || ((uintptr_t)logits & 3u) ||
        ((uintptr_t)W_r & (w_dtype == VP_BF16 ? 1u : 3u)))
        return VP_ERR_INVALID_ARG;
    (void)hipGetLastError();
    vp::launch_router_logits(u, W_r, b_r, H * VP_NUM_MODES, Din, w_dtype == VP_BF16 ? 1 : 0,
                             logits, (hipStream_t)stream);
    return hip_status("vp_router_logits");
}

vp_status vp_assign_heads(const float* scores, int32_t H, int32_t M, vp_assign_rule rule,
                          float tau_low, float tau_high, uint8_t* modes, int32_t* buckets,
                          void* stream) {
    if (!scores || !modes || !buckets) return VP_ERR_INVALID_ARG;
    if (H < 1 || M < 1) return VP_ERR_INVALID_ARG;
    if (H > VP_MAX_HEADS) return VP_ERR_UNSUPPORTED;
    if (rule != VP_ASSIGN_THRESHOLD && rule != VP_ASSIGN_ARGMAX &&
        rule != VP_ASSIGN_THRESHOLD_BINARY && rule != VP_ASSIGN_ARGMAX_BINARY)
        return VP_ERR_INVALID_ARG;
    const bool by_logits = rule == VP_ASSIGN_ARGMAX || rule == VP_ASSIGN_ARGMAX_BINARY;
    if (M != (by_logits ? VP_NUM_MODES : 1)) return VP_ERR_UNSUPPORTED;
    if ((rule == VP_ASSIGN_THRESHOLD || rule == VP_ASSIGN_THRESHOLD_BINARY) &&
        (!isfinite(tau_low) || !isfinite(tau_high) || tau_low < 0.f || tau_low > tau_high))
        return VP_ERR_INVALID_ARG;
    if (((uintptr_t)scores & 3u) || ((uintptr_t)buckets & 3u)) return VP_ERR_INVALID_ARG;
    (void)hipGetLastError();
    vp::launch_assign(scores, H, (int)rule, tau_low, tau_high, modes, buckets,
                      (hipStream_t)stream);
    return hip_status("vp_assign_heads");
}

namespace {

vp_status check_attn_common(const vp_shape* shape, const void* V, const void* Y,
                            vp_dtype y_dtype) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (!V || !Y || !aligned16(V) || !aligned16(Y)) return VP_ERR_INVALID_ARG;
    if (y_dtype != VP_F32 && y_dtype != VP_BF16) return VP_ERR_INVALID_ARG;
    return VP_OK;
}

vp_status check_linear(const vp_shape* shape, const void* V, const uint8_t* modes,
                       const vp_router_state* state, const vp_surrogate_weights* surr,
                       const void* Y, vp_dtype y_dtype) {
    vp_status st = check_attn_common(shape, V, Y, y_dtype);
    if (st != VP_OK) return st;
    if (!modes || !state || !surr) return VP_ERR_INVALID_ARG;
    if (!state->ctx || !state->vmean || ((uintptr_t)state->ctx & 3u) ||
        ((uintptr_t)state->vmean & 3u))
        return VP_ERR_INVALID_ARG;
    if ((int)surr->variant < VP_SURR_EQ7 || (int)surr->variant > VP_SURR_LINEAR_ATTN)
        return VP_ERR_INVALID_ARG;
    if (surr->variant == VP_SURR_NO_RESIDUAL || surr->variant == VP_SURR_LINEAR_ATTN)
        return VP_OK;   // no MLP weight is read
    if (!surr->g_w1 || !surr->g_w2 || !surr->d_w1 || !surr->d_w2 || !surr->g_b1 ||
        !surr->g_b2 || !surr->d_b1 || !surr->d_b2)
        return VP_ERR_INVALID_ARG;
    if (!aligned16(surr->g_w1) || !aligned16(surr->g_w2) || !aligned16(surr->d_w1) ||
        !aligned16(surr->d_w2))
        return VP_ERR_INVALID_ARG;
    if (((uintptr_t)surr->g_b1 & 3u) || ((uintptr_t)surr->g_b2 & 3u) ||
        ((uintptr_t)surr->d_b1 & 3u) || ((uintptr_t)surr->d_b2 & 3u))
        return VP_ERR_INVALID_ARG;
    if (surr->L != VP_HIDDEN) return VP_ERR_UNSUPPORTED;
    if (surr->act != VP_ACT_GELU_ERF && surr->act != VP_ACT_RELU) return VP_ERR_INVALID_ARG;
    return VP_OK;
}

vp::AttnArgs attn_args(const vp_shape* shape, const Layout& L, const void* Q, const void* K,
                       const void* V, const uint8_t* modes, const int32_t* buckets, void* Y,
                       vp_dtype y_dtype, void* ws) {
    vp::AttnArgs a;
    memset(&a, 0, sizeof(a));
    a.dtype = shape->dtype == VP_BF16 ? 1 : 0;
    a.ydt = y_dtype == VP_BF16 ? 1 : 0;
    a.Q = Q; a.K = K; a.V = V;
    a.modes = modes;
    a.buckets = buckets;
    a.N = L.N;
    a.H = shape->H;
    a.vt = ws ? (char*)ws + L.off_vt : nullptr;
    a.kh = ws ? (char*)ws + L.off_kh : nullptr;
    a.kmax = ws ? (float*)((char*)ws + L.off_kmax) : nullptr;
    a.vpart = ws ? (float*)((char*)ws + L.off_vpart) : nullptr;
    a.vsc = ws ? (float*)((char*)ws + L.off_vsc) : nullptr;
    a.qflag = ws ? (int32_t*)((char*)ws + L.off_qflag) : nullptr;
    a.part = ws ? (float*)((char*)ws + L.off_fpart) : nullptr;
    a.n3 = L.n3;
    a.chunk3 = L.chunk3;
    a.lpart = ws ? (float*)((char*)ws + L.off_lpart) : nullptr;
    a.lsum = ws ? (float*)((char*)ws + L.off_lsum) : nullptr;
    a.Y = Y;
    return a;
}

void set_linear(vp::AttnArgs& a, const vp_router_state* state, const vp_surrogate_weights* surr) {
    a.ctx = state->ctx;
    a.vmean = state->vmean;
    a.g_w1 = surr->g_w1; a.g_w2 = surr->g_w2; a.d_w1 = surr->d_w1; a.d_w2 = surr->d_w2;
    a.g_b1 = surr->g_b1; a.g_b2 = surr->g_b2; a.d_b1 = surr->d_b1; a.d_b2 = surr->d_b2;
    a.act = (int)surr->act;
    a.variant = (int)surr->variant;
}

}  // namespace

vp_status vp_gather_full_heads(const vp_shape* shape, const void* K, const void* V,
                               const int32_t* buckets, void* ws, size_t ws_bytes, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (!K || !V || !aligned16(K) || !aligned16(V) || !buckets || ((uintptr_t)buckets & 3u))
        return VP_ERR_INVALID_ARG;
    Layout L;
    if ((st = check_ws(shape, ws, ws_bytes, &L)) != VP_OK) return st;
    if (shape->dtype != VP_BF16) return VP_OK;
    (void)hipGetLastError();
    vp::AttnArgs a = attn_args(shape, L, nullptr, K, V, nullptr, buckets, nullptr, VP_F32, ws);
    vp::launch_gather(a, (hipStream_t)stream);
    return hip_status("vp_gather_full_heads");
}

vp_status vp_full_head_attention(const vp_shape* shape, const void* Q, const void* K,
                                 const void* V, const int32_t* buckets, void* Y,
                                 vp_dtype y_dtype, void* ws, size_t ws_bytes, void* stream) {
    vp_status st = check_attn_common(shape, V, Y, y_dtype);
    if (st != VP_OK) return st;
    if (!Q || !K || !aligned16(Q) || !aligned16(K)) return VP_ERR_INVALID_ARG;
    if (!buckets || ((uintptr_t)buckets & 3u)) return VP_ERR_INVALID_ARG;
    Layout L;
    if ((st = check_ws(shape, ws, ws_bytes, &L)) != VP_OK) return st;
    (void)hipGetLastError();
    vp::AttnArgs a = attn_args(shape, L, Q, K, V, nullptr, buckets, Y, y_dtype, ws);
    vp::launch_flash(a, (hipStream_t)stream);
    return hip_status("vp_full_head_attention");
}

vp_status vp_linear_heads(const vp_shape* shape, const void* Q, const void* K, const void* V,
                          const uint8_t* modes, const vp_router_state* state,
                          const vp_surrogate_weights* surr, void* Y, vp_dtype y_dtype, void* ws,
                          size_t ws_bytes, void* stream) {
    vp_status st = check_linear(shape, V, modes, state, surr, Y, y_dtype);
    if (st != VP_OK) return st;
    Layout L;
    if (surr->variant == VP_SURR_LINEAR_ATTN) {
        if (!Q || !K || !aligned16(Q) || !aligned16(K)) return VP_ERR_INVALID_ARG;
        if ((st = check_ws(shape, ws, ws_bytes, &L)) != VP_OK) return st;
    } else {
        make_layout(shape, &L);
        ws = nullptr;   // not read
    }
    (void)hipGetLastError();
    vp::AttnArgs a = attn_args(shape, L, Q, K, V, modes, nullptr, Y, y_dtype, ws);
    set_linear(a, state, surr);
    vp::launch_linear_heads(a, (hipStream_t)stream);
    return hip_status("vp_linear_heads");
}

vp_status vp_routed_global_attention(const vp_shape* shape, const void* Q, const void* K,
                                     const void* V, const uint8_t* modes,
                                     const int32_t* buckets, const vp_router_state* state,
                                     const vp_surrogate_weights* surr, void* Y, vp_dtype y_dtype,
                                     void* ws, size_t ws_bytes, void* stream) {
    vp_status st = check_linear(shape, V, modes, state, surr, Y, y_dtype);
    if (st != VP_OK) return st;
    if (!Q || !K || !aligned16(Q) || !aligned16(K)) return VP_ERR_INVALID_ARG;
    if (!buckets || ((uintptr_t)buckets & 3u)) return VP_ERR_INVALID_ARG;
    Layout L;
    if ((st = check_ws(shape, ws, ws_bytes, &L)) != VP_OK) return st;
    (void)hipGetLastError();
    vp::AttnArgs a = attn_args(shape, L, Q, K, V, modes, buckets, Y, y_dtype, ws);
    set_linear(a, state, surr);
    hipStream_t s = (hipStream_t)stream;
    if (a.dtype == 1) vp::launch_gather(a, s);
    vp::launch_flash(a, s);
    vp::launch_linear_heads(a, s);
    return hip_status("vp_routed_global_attention");
}

// ------------------------------------------------ dense block around the layer

namespace {

constexpr int64_t kBlockD = 1024;

bool block_shape_ok(const vp_shape* s) {
    return s && s->S >= 1 && s->P >= 1 && s->S <= kMaxTokens && s->P <= kMaxTokens &&
           s->S * s->P <= kMaxTokens && s->H == VP_MAX_HEADS && s->d == VP_HEAD_DIM &&
           s->dtype == VP_BF16;
}

size_t block_ws(int64_t N) { return align_up((size_t)N * kBlockD * 2 * (1 + 1 + 4)); }

bool aligned4(const void* p) { return ((uintptr_t)p & 3u) == 0; }

vp_status check_block(const vp_shape* shape, const vp_block_weights* w, void* ws,
                      size_t ws_bytes, vp::BlockArgs* a) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (!block_shape_ok(shape)) return VP_ERR_UNSUPPORTED;
    if (!w) return VP_ERR_INVALID_ARG;
    const void* mats[] = {w->w_qkv, w->w_o, w->w_fc1, w->w_fc2};
    for (const void* m : mats)
        if (!m || !aligned16(m)) return VP_ERR_INVALID_ARG;
    const float* vecs[] = {w->ln1_w, w->ln1_b, w->b_qkv, w->b_o, w->ls1, w->ln2_w,
                           w->ln2_b, w->b_fc1, w->b_fc2, w->ls2};
    for (const float* v : vecs)
        if (!v || !aligned4(v)) return VP_ERR_INVALID_ARG;
    if (!isfinite(w->ln_eps) || w->ln_eps < 0.f || !isfinite(w->rope_base) ||
        w->rope_base < 0.f || (w->rope_base > 0.f && w->rope_base <= 1.f))
        return VP_ERR_INVALID_ARG;
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    const int64_t N = shape->S * shape->P;
    if (ws_bytes < block_ws(N)) return VP_ERR_WORKSPACE;
    memset(a, 0, sizeof(*a));
    a->T = N;
    a->ln1_w = w->ln1_w; a->ln1_b = w->ln1_b; a->ln2_w = w->ln2_w; a->ln2_b = w->ln2_b;
    a->ls1 = w->ls1; a->ls2 = w->ls2;
    a->w_qkv = (const __bf16*)w->w_qkv; a->w_o = (const __bf16*)w->w_o;
    a->w_fc1 = (const __bf16*)w->w_fc1; a->w_fc2 = (const __bf16*)w->w_fc2;
    a->b_qkv = w->b_qkv; a->b_o = w->b_o; a->b_fc1 = w->b_fc1; a->b_fc2 = w->b_fc2;
    a->eps = w->ln_eps > 0.f ? w->ln_eps : 1e-6f;
    a->rope_base = w->rope_base > 0.f ? w->rope_base : 100.f;
    char* p = (char*)ws;
    a->ln = (__bf16*)p;
    a->xa = (__bf16*)(p + (size_t)N * kBlockD * 2);
    a->hid = (__bf16*)(p + (size_t)N * kBlockD * 4);
    return VP_OK;
}

}  // namespace

size_t vp_block_workspace_bytes(const vp_shape* shape) {
    if (shape_status(shape) != VP_OK || !block_shape_ok(shape)) return 0;
    return block_ws(shape->S * shape->P);
}

vp_status vp_block_qkv(const vp_shape* shape, const void* X, const int32_t* pos,
                       const vp_block_weights* w, void* Q, void* K, void* V, void* ws,
                       size_t ws_bytes, void* stream) {
    vp::BlockArgs a;
    vp_status st = check_block(shape, w, ws, ws_bytes, &a);
    if (st != VP_OK) return st;
    if (!X || !Q || !K || !V || !pos || !aligned16(X) || !aligned16(Q) || !aligned16(K) ||
        !aligned16(V) || ((uintptr_t)pos & 7u))
        return VP_ERR_INVALID_ARG;
    a.X = (const __bf16*)X;
    a.pos = pos;
    a.Q = (__bf16*)Q; a.K = (__bf16*)K; a.V = (__bf16*)V;
    (void)hipGetLastError();
    vp::launch_block_qkv(a, (hipStream_t)stream);
    return hip_status("vp_block_qkv");
}

vp_status vp_block_out(const vp_shape* shape, const void* X, const void* Y,
                       const vp_block_weights* w, void* X_out, void* ws, size_t ws_bytes,
                       void* stream) {
    vp::BlockArgs a;
    vp_status st = check_block(shape, w, ws, ws_bytes, &a);
    if (st != VP_OK) return st;
    if (!X || !Y || !X_out || !aligned16(X) || !aligned16(Y) || !aligned16(X_out))
        return VP_ERR_INVALID_ARG;
    a.X = (const __bf16*)X;
    a.Y = (const __bf16*)Y;
    a.Xout = (__bf16*)X_out;
    (void)hipGetLastError();
    vp::launch_block_out(a, (hipStream_t)stream);
    return hip_status("vp_block_out");
}

// ------------------------------------------- distillation targets and losses

namespace {

struct TeacherLayout {
    Layout attn;
    size_t off_off, off_y, off_buckets, total;
};

bool teacher_layout(const vp_shape* s, TeacherLayout* T) {
    if (!make_layout(s, &T->attn) || s->dtype != VP_BF16) return false;
    const size_t N = (size_t)T->attn.N, H = (size_t)s->H;
    size_t off = T->attn.total;
    T->off_off = off;
    off = align_up(off + H * N * sizeof(float));
    T->off_y = off;
    off = align_up(off + N * H * VP_HEAD_DIM * sizeof(float));
    T->off_buckets = off;
    off = align_up(off + VP_BUCKETS_LEN * sizeof(int32_t));
    T->total = off;
    return true;
}

}  // namespace

size_t vp_teacher_workspace_bytes(const vp_shape* shape) {
    TeacherLayout T;
    if (shape_status(shape) != VP_OK || !teacher_layout(shape, &T)) return 0;
    return T.total;
}

size_t vp_loss_workspace_bytes(const vp_shape* shape) {
    if (shape_status(shape) != VP_OK) return 0;
    return align_up(vp::distill_part_bytes(shape->H));
}

vp_status vp_teacher_targets(const vp_shape* shape, const void* Q, const void* K, const void* V,
                             float* colmax, float* smax, void* delta, vp_dtype y_dtype, void* ws,
                             size_t ws_bytes, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (shape->dtype != VP_BF16) return VP_ERR_UNSUPPORTED;
    if (!Q || !K || !V || !colmax || !smax || !delta || !aligned16(Q) || !aligned16(K) ||
        !aligned16(V) || !aligned16(delta) || ((uintptr_t)colmax & 3u) || ((uintptr_t)smax & 3u))
        return VP_ERR_INVALID_ARG;
    if (y_dtype != VP_F32 && y_dtype != VP_BF16) return VP_ERR_INVALID_ARG;
    TeacherLayout T;
    teacher_layout(shape, &T);
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    if (ws_bytes < T.total) return VP_ERR_WORKSPACE;
    char* w = (char*)ws;
    vp::TeacherArgs a;
    int32_t* buckets = (int32_t*)(w + T.off_buckets);
    a.attn = attn_args(shape, T.attn, Q, K, V, nullptr, buckets, w + T.off_y, VP_F32, ws);
    a.attn.off = (float*)(w + T.off_off);
    a.colmax = colmax;
    a.smax = smax;
    a.delta = delta;
    a.delta_dt = y_dtype == VP_BF16 ? 1 : 0;
    (void)hipGetLastError();
    vp::launch_teacher_targets(a, (hipStream_t)stream);
    return hip_status("vp_teacher_targets");
}

vp_status vp_router_loss(const vp_shape* shape, const void* K, const vp_router_state* state,
                         float scale, const float* colmax, const float* smax, float lambda,
                         float* loss, void* ws, size_t ws_bytes, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (shape->dtype != VP_BF16) return VP_ERR_UNSUPPORTED;
    if (!K || !aligned16(K) || !state || !state->q_pool || !state->stats || !colmax || !smax ||
        !loss || ((uintptr_t)state->q_pool & 3u) || ((uintptr_t)state->stats & 3u) ||
        ((uintptr_t)colmax & 3u) || ((uintptr_t)smax & 3u) || ((uintptr_t)loss & 3u))
        return VP_ERR_INVALID_ARG;
    if (!isfinite(scale) || scale < 0.f || !isfinite(lambda)) return VP_ERR_INVALID_ARG;
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    if (ws_bytes < vp_loss_workspace_bytes(shape)) return VP_ERR_WORKSPACE;
    vp::LossArgs a;
    memset(&a, 0, sizeof(a));
    a.dtype = 1;
    a.A = K;
    a.q_pool = state->q_pool;
    a.stats = state->stats;
    a.colmax = colmax;
    a.smax = smax;
    a.scale = scale > 0.f ? scale : 1.f / sqrtf((float)shape->d);
    a.lambda = lambda;
    a.N = shape->S * shape->P;
    a.H = shape->H;
    a.part = (float*)ws;
    a.loss = loss;
    (void)hipGetLastError();
    vp::launch_router_loss(a, (hipStream_t)stream);
    return hip_status("vp_router_loss");
}

vp_status vp_latent_loss(const vp_shape* shape, const void* D_hat, const void* D_t,
                         vp_dtype dtype, float lambda, float* loss, void* ws, size_t ws_bytes,
                         void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (dtype != VP_F32 && dtype != VP_BF16) return VP_ERR_INVALID_ARG;
    if (!D_hat || !D_t || !loss || !aligned16(D_hat) || !aligned16(D_t) ||
        ((uintptr_t)loss & 3u))
        return VP_ERR_INVALID_ARG;
    if (!isfinite(lambda)) return VP_ERR_INVALID_ARG;
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    if (ws_bytes < vp_loss_workspace_bytes(shape)) return VP_ERR_WORKSPACE;
    vp::LossArgs a;
    memset(&a, 0, sizeof(a));
    a.dtype = dtype == VP_BF16 ? 1 : 0;
    a.A = D_hat;
    a.B = D_t;
    a.lambda = lambda;
    a.N = shape->S * shape->P;
    a.H = shape->H;
    a.part = (float*)ws;
    a.loss = loss;
    (void)hipGetLastError();
    vp::launch_latent_loss(a, (hipStream_t)stream);
    return hip_status("vp_latent_loss");
}

}  // extern "C"

// ------------------------------------------------------------ token merging

namespace {

int64_t tome_sources(int64_t S, int64_t np, int64_t g) {
    return (S - 1) * (np - (np + g - 1) / g);
}

bool tome_geom(const vp_shape* s, int64_t M, int32_t nsp, vp::TomeGeom* G) {
    if (shape_status(s) != VP_OK) return false;
    const int64_t S = s->S, P = s->P, N = S * P;
    if (nsp < 0 || nsp >= P || M < 0) return false;
    const int64_t np = P - nsp;
    if (M > tome_sources(S, np, np)) return false;
    // smallest g in [1, np] with at least M sources (the count grows with g)
    int64_t lo = 1, hi = np;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (tome_sources(S, np, mid) >= M) hi = mid;
        else lo = mid + 1;
    }
    G->N = N;
    G->P = P;
    G->nsp = nsp;
    G->np = np;
    G->g = lo;
    G->ndp = (np + lo - 1) / lo;
    G->nsv = np - G->ndp;
    G->nA = (S - 1) * G->nsv;
    G->nD = N - G->nA;
    return true;
}

}  // namespace

vp_status vp_tome_split(const vp_shape* shape, int64_t M, int32_t nspecial, int64_t* g,
                        int64_t* nrows) {
    vp::TomeGeom G;
    if (!tome_geom(shape, M, nspecial, &G)) return VP_ERR_INVALID_ARG;
    if (g) *g = G.g;
    if (nrows) *nrows = G.N - M;
    return VP_OK;
}

size_t vp_tome_workspace_bytes(const vp_shape* shape) {
    if (shape_status(shape) != VP_OK) return 0;
    return align_up(vp::tome_workspace_bytes(shape->S * shape->P));
}

vp_status vp_tome_plan(const vp_shape* shape, const void* K, int64_t M, int32_t nspecial,
                       int32_t* row, int32_t* row_start, int32_t* members, int32_t* best,
                       float* score, void* ws, size_t ws_bytes, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (shape->dtype != VP_BF16) return VP_ERR_UNSUPPORTED;
    vp::TomeGeom G;
    if (!tome_geom(shape, M, nspecial, &G)) return VP_ERR_INVALID_ARG;
    if (!K || !aligned16(K) || !row || !row_start || !members || !aligned4(row) ||
        !aligned4(row_start) || !aligned4(members) || (best && !aligned4(best)) ||
        (score && !aligned4(score)))
        return VP_ERR_INVALID_ARG;
    if (!ws || ((uintptr_t)ws & (kAlign - 1))) return VP_ERR_INVALID_ARG;
    if (ws_bytes < vp::tome_workspace_bytes(G.N)) return VP_ERR_WORKSPACE;
    vp::TomeArgs a;
    a.G = G;
    a.M = M;
    a.K = (const __bf16*)K;
    a.H = shape->H;
    a.row = row;
    a.row_start = row_start;
    a.members = members;
    a.best = best;
    a.score = score;
    a.ws = ws;
    (void)hipGetLastError();
    vp::launch_tome_plan(a, (hipStream_t)stream);
    return hip_status("vp_tome_plan");
}

vp_status vp_tome_merge(const vp_shape* shape, const void* X, int64_t nrows,
                        const int32_t* row_start, const int32_t* members, void* Xm,
                        void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    const int64_t N = shape->S * shape->P;
    if (!X || !Xm || !aligned16(X) || !aligned16(Xm) || !row_start || !members ||
        !aligned4(row_start) || !aligned4(members) || nrows < 1 || nrows > N)
        return VP_ERR_INVALID_ARG;
    (void)hipGetLastError();
    vp::launch_tome_merge(shape->dtype == VP_BF16 ? 1 : 0, X, N, shape->H * VP_HEAD_DIM, nrows,
                          row_start, members, Xm, (hipStream_t)stream);
    return hip_status("vp_tome_merge");
}

vp_status vp_tome_merge_qkv(const vp_shape* shape, const void* Q, const void* K, const void* V,
                            int64_t nrows, const int32_t* row_start, const int32_t* members,
                            void* Qm, void* Km, void* Vm, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    if (shape->dtype != VP_BF16) return VP_ERR_UNSUPPORTED;
    const int64_t N = shape->S * shape->P;
    if (!Q || !K || !V || !Qm || !Km || !Vm || !aligned16(Q) || !aligned16(K) || !aligned16(V) ||
        !aligned16(Qm) || !aligned16(Km) || !aligned16(Vm) || !row_start || !members ||
        !aligned4(row_start) || !aligned4(members) || nrows < 1 || nrows > N)
        return VP_ERR_INVALID_ARG;
    (void)hipGetLastError();
    vp::launch_tome_merge_qkv(Q, K, V, N, shape->H * VP_HEAD_DIM, nrows, row_start, members, Qm,
                              Km, Vm, (hipStream_t)stream);
    return hip_status("vp_tome_merge_qkv");
}

vp_status vp_tome_unmerge(const vp_shape* shape, const void* Ym, int64_t nrows,
                          const int32_t* row, void* Y, void* stream) {
    vp_status st = shape_status(shape);
    if (st != VP_OK) return st;
    const int64_t N = shape->S * shape->P;
    if (!Ym || !Y || !aligned16(Ym) || !aligned16(Y) || !row || !aligned4(row) || nrows < 1 ||
        nrows > N)
        return VP_ERR_INVALID_ARG;
    (void)hipGetLastError();
    vp::launch_tome_unmerge(shape->dtype == VP_BF16 ? 1 : 0, Ym, nrows, row, N,
                            shape->H * VP_HEAD_DIM, Y, (hipStream_t)stream);
    return hip_status("vp_tome_unmerge");
}

