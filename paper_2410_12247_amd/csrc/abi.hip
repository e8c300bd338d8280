// C-ABI entry points (argument checks, workspace layout, error reporting)
// for the single-step calls; moe_ffn_forward lives in forward.hip.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <vector>

#include "common.h"

namespace moe {

namespace {
thread_local char g_last_error[512] = "";

size_t align_up(size_t v) { return (v + 255) & ~size_t(255); }
}  // namespace

moe_status fail(moe_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

moe_status hip_check(hipError_t e, const char *what) {
    if (e == hipSuccess) return MOE_OK;
    return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

moe_status check_dims(const moe_dims *d) {
    if (!d) return fail(MOE_ERR_INVALID, "dims is NULL");
    if (d->tokens < 0) return fail(MOE_ERR_INVALID, "tokens < 0");
    if (d->experts > kMaxExperts)
        return fail(MOE_ERR_UNSUPPORTED, "experts %d > %d", d->experts, kMaxExperts);
    if (d->top_k > kMaxTopK) return fail(MOE_ERR_UNSUPPORTED, "top_k %d > %d", d->top_k, kMaxTopK);
    if (d->experts < 1) return fail(MOE_ERR_INVALID, "experts < 1");
    if (d->top_k < 1 || d->top_k > d->experts)
        return fail(MOE_ERR_INVALID, "top_k %d outside [1, experts]", d->top_k);
    if (d->hidden <= 0 || d->hidden % kDimAlign)
        return fail(MOE_ERR_INVALID, "hidden %d not a positive multiple of %d", d->hidden,
                    kDimAlign);
    if (d->inter <= 0 || d->inter % kDimAlign)
        return fail(MOE_ERR_INVALID, "inter %d not a positive multiple of %d", d->inter,
                    kDimAlign);
    if (d->hidden > (1 << 20) || d->inter > (1 << 20) || d->shared_inter > (1 << 20))
        return fail(MOE_ERR_INVALID, "hidden/inter above 2^20");
    if (d->local_begin < 0 || d->local_count < 1 ||
        d->local_begin + d->local_count > d->experts)
        return fail(MOE_ERR_INVALID, "local experts [%d, %d) outside [0, %d)", d->local_begin,
                    d->local_begin + d->local_count, d->experts);
    if (d->renormalize != 0 && d->renormalize != 1)
        return fail(MOE_ERR_INVALID, "renormalize must be 0 or 1");
    if (d->shared_inter < 0 || d->shared_inter % kDimAlign)
        return fail(MOE_ERR_INVALID, "shared_inter %d not a multiple of %d", d->shared_inter,
                    kDimAlign);
    if (d->tokens * (int64_t)d->top_k >= (int64_t(1) << 31))
        return fail(MOE_ERR_INVALID, "tokens * top_k >= 2^31");
    return MOE_OK;
}

bool gather_foldable(const moe_dims &d) {
    return (uint64_t)d.tokens * (uint64_t)d.hidden * 2u < (uint64_t(1) << 32);
}

WsLayout ws_layout(const moe_dims *d, const moe_opts *opt, bool shared_apart) {
    WsLayout L{};
    const bool forward = opt != nullptr;
    const int nbuckets = forward ? forward_buckets(d, opt) : d->local_count;
    const int64_t T = d->tokens, k = d->top_k, EL = d->local_count;
    const int64_t nslots = T * k;
    const int64_t NB = nbuckets;
    L.nbuckets = nbuckets;
    L.nchunks = (nslots + kPermChunk - 1) / kPermChunk;
    L.rcap = T * (k < EL ? k : EL);
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o = align_up(o + bytes);
        if (L.nguards < kMaxWsGuards) L.guard[L.nguards++] = o;
        o += kWsGuardBytes;
        return at;
    };
    L.chunk_counts = take(sizeof(int32_t) * L.nchunks * NB);
    L.chunk_base = take(sizeof(int32_t) * L.nchunks * NB);
    L.slot_rank = take(sizeof(int32_t) * nslots);
    if (forward) {
        L.ids = take(sizeof(int32_t) * nslots);
        L.weights = take(sizeof(float) * nslots);
        L.logits = d->experts > 16 && T <= kRouteLogitsMaxTokens
                       ? take(sizeof(float) * T * d->experts)
                       : 0;
        L.counts = take(sizeof(int32_t) * NB);
        L.counts_el = take(sizeof(int32_t) * EL);
        L.offsets = take(sizeof(int32_t) * (NB + 1));
        L.sorted_slot = take(sizeof(int32_t) * L.rcap);
        L.slot_row = take(sizeof(int32_t) * nslots);
        // gathered token rows: only read when the input is too large for the
        // gate/up GEMM's folded gather (32-bit byte offsets into x)
        const bool xperm = !gather_foldable(*d);
        L.x_perm = take(xperm ? sizeof(bf16_t) * L.rcap * d->hidden : 0);
        L.act = take(sizeof(bf16_t) * L.rcap * d->inter);
        L.y_perm = take(sizeof(float) * L.rcap * d->hidden);
        L.shared_act = take(sizeof(bf16_t) * T * d->shared_inter);
        // K-split partials, unless every GEMM is one pass over K
        L.split_part = take((opt->flags & MOE_FLAG_EXACT_ORDER) ? 0 : gemm_split_bytes());
        L.split_meta = take(sizeof(int32_t) * kSplitMetaInts);
        if (shared_apart && d->shared_inter > 0 && (opt->flags & MOE_FLAG_EXACT_ORDER) == 0 &&
            (opt->flags & MOE_FLAG_SERIAL) == 0) {
            L.split_part_sh = take(gemm_split_bytes());
            L.split_meta_sh = take(sizeof(int32_t) * kSplitMetaInts);
        }
    }
    L.total = o;
    return L;
}

int device_cu_count() {
    static std::mutex mu;
    static std::vector<int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    std::lock_guard<std::mutex> lock(mu);
    if ((int)cache.size() <= dev) cache.resize(dev + 1, 0);
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}

}  // namespace moe

using namespace moe;

extern "C" {

const char *moe_status_string(moe_status s) {
    switch (s) {
        case MOE_OK: return "ok";
        case MOE_ERR_INVALID: return "invalid argument";
        case MOE_ERR_UNSUPPORTED: return "unsupported size";
        case MOE_ERR_WORKSPACE: return "workspace too small";
        case MOE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char *moe_last_error(void) { return g_last_error; }

size_t moe_workspace_bytes(const moe_dims *dims, const moe_opts *opts) {
    if (check_dims(dims) != MOE_OK) return 0;
    if (opts && forward_buckets(dims, opts) <= 0) return 0;
    return ws_layout(dims, opts).total;
}

int32_t moe_workspace_guards(const moe_dims *dims, const moe_opts *opts, int64_t *offsets,
                             int32_t capacity) {
    if (check_dims(dims) != MOE_OK) return -1;
    if (opts && forward_buckets(dims, opts) <= 0) return -1;
    if (capacity < 0 || (capacity > 0 && !offsets)) {
        fail(MOE_ERR_INVALID, "moe_workspace_guards: offsets NULL or capacity < 0");
        return -1;
    }
    const WsLayout L = ws_layout(dims, opts);
    for (int i = 0; i < L.nguards && i < capacity; ++i) offsets[i] = (int64_t)L.guard[i];
    return L.nguards;
}

moe_status moe_route(const moe_dims *dims, const moe_bf16 *x, const float *w_router,
                     const float *bias, int32_t *topk_ids, float *topk_w, void *stream) {
    MOE_TRY(check_dims(dims));
    if (dims->tokens == 0) return MOE_OK;
    if (!x || !w_router || !topk_ids || !topk_w)
        return fail(MOE_ERR_INVALID, "moe_route: NULL tensor");
    MOE_HIP(launch_route(*dims, x, w_router, bias, topk_ids, topk_w, nullptr,
                         (hipStream_t)stream));
    return MOE_OK;
}

moe_status moe_permute(const moe_dims *dims, const int32_t *topk_ids, const moe_bf16 *x,
                       int32_t *counts, int32_t *offsets, int32_t *sorted_slot,
                       int32_t *slot_row, moe_bf16 *x_perm, void *ws, size_t ws_bytes,
                       void *stream) {
    MOE_TRY(check_dims(dims));
    if (dims->tokens == 0) return MOE_OK;
    if (!topk_ids || !counts || !offsets || !sorted_slot || !slot_row)
        return fail(MOE_ERR_INVALID, "moe_permute: NULL index tensor");
    if (x_perm && !x) return fail(MOE_ERR_INVALID, "moe_permute: x_perm given without x");
    const WsLayout L = ws_layout(dims, nullptr);
    if (!ws || ws_bytes < L.total)
        return fail(MOE_ERR_WORKSPACE, "moe_permute: workspace %zu < %zu bytes", ws_bytes,
                    L.total);
    hipStream_t s = (hipStream_t)stream;
    MOE_HIP(launch_permute(*dims, topk_ids, ws, L, 0, counts, offsets, nullptr, sorted_slot,
                           slot_row, s));
    if (x_perm)
        MOE_HIP(launch_gather(*dims, 0, dims->local_count, offsets, sorted_slot, x, x_perm,
                              L.rcap, s));
    return MOE_OK;
}

moe_status moe_gather(const moe_dims *dims, int32_t e_first, int32_t e_count,
                      const int32_t *offsets, const int32_t *sorted_slot, const moe_bf16 *x,
                      moe_bf16 *x_perm, void *stream) {
    MOE_TRY(check_dims(dims));
    if (e_first < 0 || e_count < 0 || e_first + e_count > dims->local_count)
        return fail(MOE_ERR_INVALID, "moe_gather: expert range outside [0, local_count)");
    if (dims->tokens == 0 || e_count == 0) return MOE_OK;
    if (!offsets || !sorted_slot || !x || !x_perm)
        return fail(MOE_ERR_INVALID, "moe_gather: NULL tensor");
    const int64_t rcap = dims->tokens * std::min<int64_t>(dims->top_k, dims->local_count);
    MOE_HIP(launch_gather(*dims, e_first, e_count, offsets, sorted_slot, x, x_perm, rcap,
                          (hipStream_t)stream));
    return MOE_OK;
}

moe_status moe_ffn_group(const moe_dims *dims, int32_t e_first, int32_t e_count,
                         const int32_t *offsets, const moe_bf16 *x_perm,
                         const moe_bf16 *w_gate, const moe_bf16 *w_up,
                         const moe_bf16 *w_down, moe_bf16 *act, float *y_perm,
                         int32_t cu_budget, void *stream) {
    MOE_TRY(check_dims(dims));
    if (e_first < 0 || e_count < 0 || e_first + e_count > dims->local_count)
        return fail(MOE_ERR_INVALID, "moe_ffn_group: expert range outside [0, local_count)");
    if (cu_budget < 0) return fail(MOE_ERR_INVALID, "moe_ffn_group: cu_budget < 0");
    if (dims->tokens == 0 || e_count == 0) return MOE_OK;
    if (!offsets || !x_perm || !w_gate || !w_up || !w_down || !act || !y_perm)
        return fail(MOE_ERR_INVALID, "moe_ffn_group: NULL tensor");
    int grid = cu_budget > 0 ? cu_budget : device_cu_count();
    grid = std::max(8, (grid / 8) * 8);
    hipStream_t s = (hipStream_t)stream;
    // no workspace here: every tile covers the whole K range in one pass;
    // no expert has more rows than there are tokens
    const int bm = group_launch_rows(dims->tokens, nullptr, e_count, dims->tokens,
                                     (double)dims->top_k / dims->experts, dims->hidden,
                                     dims->inter, grid, false);
    MOE_HIP(launch_group_gateup(*dims, e_first, e_count, offsets, x_perm, nullptr, w_gate, w_up,
                                act, grid, nullptr, nullptr, bm, s));
    // decode-sized experts with enough tiles: the skinny down tile
    const int64_t active = std::min<int64_t>(e_count, dims->tokens * dims->top_k);
    const int sk = skinny_down_rows(dims->tokens, active, dims->hidden);
    if (sk > 0)
        MOE_HIP(launch_skinny_down(*dims, e_first, e_count, offsets, act, w_down, y_perm, sk,
                                   active, s));
    else
        MOE_HIP(launch_group_down(*dims, e_first, e_count, offsets, act, w_down, y_perm, grid,
                                  nullptr, nullptr, bm, s));
    return MOE_OK;
}

moe_status moe_ffn_dense(int64_t rows, int32_t hidden, int32_t inter, const moe_bf16 *x,
                         const moe_bf16 *w_gate, const moe_bf16 *w_up,
                         const moe_bf16 *w_down, moe_bf16 *act, float *y, void *stream) {
    if (rows < 0) return fail(MOE_ERR_INVALID, "moe_ffn_dense: rows < 0");
    if (hidden <= 0 || hidden % kDimAlign || inter <= 0 || inter % kDimAlign ||
        hidden > (1 << 20) || inter > (1 << 20))
        return fail(MOE_ERR_INVALID, "moe_ffn_dense: hidden %d / inter %d not multiples of %d",
                    hidden, inter, kDimAlign);
    if (rows == 0) return MOE_OK;
    if (!x || !w_gate || !w_up || !w_down || !act || !y)
        return fail(MOE_ERR_INVALID, "moe_ffn_dense: NULL tensor");
    hipStream_t s = (hipStream_t)stream;
    // the tile height whose tile count fills the chip best for these rows
    const int bm = dense_tile_rows(rows, hidden, inter, device_cu_count(), false);
    MOE_HIP(launch_dense_gateup(rows, hidden, inter, x, w_gate, w_up, act, bm, s));
    MOE_HIP(launch_dense_down(rows, hidden, inter, act, w_down, y, bm, s));
    return MOE_OK;
}

moe_status moe_combine(const moe_dims *dims, int32_t e_first, int32_t e_count,
                       const float *y_perm, const int32_t *topk_ids, const int32_t *slot_row,
                       const float *topk_w, float *y, int32_t accumulate, void *stream) {
    MOE_TRY(check_dims(dims));
    if (e_first < 0 || e_count < 0 || e_first + e_count > dims->local_count)
        return fail(MOE_ERR_INVALID, "moe_combine: expert range outside [0, local_count)");
    if (accumulate != 0 && accumulate != 1)
        return fail(MOE_ERR_INVALID, "moe_combine: accumulate must be 0 or 1");
    if (dims->tokens == 0) return MOE_OK;
    if (!topk_ids || !slot_row || !topk_w || !y || (!y_perm && e_count > 0))
        return fail(MOE_ERR_INVALID, "moe_combine: NULL tensor");
    MOE_HIP(launch_combine(*dims, e_first, e_count, 0, dims->tokens, y_perm, topk_ids, slot_row,
                           topk_w, y, accumulate, (hipStream_t)stream));
    return MOE_OK;
}

}  // extern "C"
