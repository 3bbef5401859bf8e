// js_api.hip -- the C ABI of the Jensen--Shannon functional distance
// (Sec. 4.4, JS distance; Appendix D.2): argument checks and launches of the
// kernels in js.hip.  No engine is involved; the calls run on the caller's
// current device.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "../../include/fgd.h"
#include "api.hpp"
#include "js.hpp"

namespace {

using fgd::api_fail;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

fgd_status check_sizes(int32_t dtype, int32_t num_workers, int64_t num_tokens) {
    if (dtype != FGD_F32 && dtype != FGD_BF16) return api_fail(FGD_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (num_workers < 1 || num_workers > FGD_MAX_JS_WORKERS)
        return api_fail(FGD_ERR_INVALID_ARG, "num_workers %d is outside [1, %d]", num_workers, FGD_MAX_JS_WORKERS);
    if (num_tokens < 1 || num_tokens > INT32_MAX)
        return api_fail(FGD_ERR_INVALID_ARG, "num_tokens must be in [1, 2^31)");
    return FGD_OK;
}

bool ranges_overlap(const void *a, int64_t na, const void *b, int64_t nb) {
    if (!a || !b || na <= 0 || nb <= 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + static_cast<uint64_t>(nb) && b0 < a0 + static_cast<uint64_t>(na);
}

// The checks fgd_js_distance and fgd_stream_js_pattern share: the logits and
// the workspace.
fgd_status check_rows(const void *logits_avg, const void *logits_workers, int32_t dtype, int32_t num_workers,
                      int64_t num_tokens, int64_t vocab, int64_t ldk, const void *workspace,
                      int64_t workspace_bytes) {
    if (fgd_status st = check_sizes(dtype, num_workers, num_tokens)) return st;
    const int es = dtype == FGD_BF16 ? 2 : 4;
    if (!logits_avg || !logits_workers || !workspace) return api_fail(FGD_ERR_INVALID_ARG, "NULL array");
    if (!aligned16(logits_avg) || !aligned16(logits_workers) || !aligned16(workspace))
        return api_fail(FGD_ERR_INVALID_ARG, "logit arrays and the workspace must be 16-byte aligned");
    if (vocab < 1 || ldk < vocab) return api_fail(FGD_ERR_INVALID_ARG, "need 1 <= vocab <= ldk");
    if ((ldk * es) % 16 != 0 || ldk * es > INT32_MAX)
        return api_fail(FGD_ERR_INVALID_ARG, "rows must be a multiple of 16 bytes and below 2 GB");
    const int64_t need = fgd::js_workspace_bytes(dtype == FGD_BF16, num_workers, num_tokens);
    if (workspace_bytes < need)
        return api_fail(FGD_ERR_INVALID_ARG, "workspace of %lld bytes is below the %lld this call needs",
                        static_cast<long long>(workspace_bytes), static_cast<long long>(need));
    const int64_t M = num_workers, U = num_tokens;
    if (ranges_overlap(workspace, need, logits_avg, U * ldk * es) ||
        ranges_overlap(workspace, need, logits_workers, M * U * ldk * es))
        return api_fail(FGD_ERR_INVALID_ARG, "the workspace must not overlap the logits");
    return FGD_OK;
}

}  // namespace

extern "C" {

fgd_status fgd_js_workspace_size(int32_t dtype, int32_t num_workers, int64_t num_tokens, int64_t *bytes) {
    fgd::api_clear();
    if (!bytes) return api_fail(FGD_ERR_INVALID_ARG, "NULL bytes");
    if (fgd_status st = check_sizes(dtype, num_workers, num_tokens)) return st;
    *bytes = fgd::js_workspace_bytes(dtype == FGD_BF16, num_workers, num_tokens);
    return FGD_OK;
}

fgd_status fgd_js_distance(const void *logits_avg, const void *logits_workers, int32_t dtype, int32_t num_workers,
                           int64_t num_tokens, int64_t vocab, int64_t ldk, int32_t top_k, double *d_out,
                           double *mean_out, int32_t *topk_out, void *workspace, int64_t workspace_bytes,
                           void *stream) {
    fgd::api_clear();
    if (fgd_status st = check_rows(logits_avg, logits_workers, dtype, num_workers, num_tokens, vocab, ldk, workspace,
                                   workspace_bytes))
        return st;
    if (!d_out) return api_fail(FGD_ERR_INVALID_ARG, "NULL array");
    if ((reinterpret_cast<uintptr_t>(d_out) & 7u) || (mean_out && (reinterpret_cast<uintptr_t>(mean_out) & 7u)) ||
        (topk_out && (reinterpret_cast<uintptr_t>(topk_out) & 3u)))
        return api_fail(FGD_ERR_INVALID_ARG, "outputs must be aligned to their element size");
    if (top_k < 1 || top_k > FGD_MAX_JS_TOPK || top_k > vocab)
        return api_fail(FGD_ERR_INVALID_ARG, "top_k %d is outside [1, min(vocab, %d)]", top_k, FGD_MAX_JS_TOPK);
    const int64_t M = num_workers, U = num_tokens;
    const int64_t need = fgd::js_workspace_bytes(dtype == FGD_BF16, num_workers, num_tokens);
    if (ranges_overlap(workspace, need, d_out, M * U * 8) ||
        (mean_out && ranges_overlap(workspace, need, mean_out, M * 8)) ||
        (topk_out && ranges_overlap(workspace, need, topk_out, U * top_k * 4)))
        return api_fail(FGD_ERR_INVALID_ARG, "the workspace must not overlap the outputs");
    int num_cus = 0;
    if (fgd_status st = fgd::api_device_cus(num_cus)) return st;
    if (!fgd::js_launch(logits_avg, logits_workers, dtype == FGD_BF16, num_workers, num_tokens, vocab, ldk, top_k,
                        d_out, mean_out, topk_out, workspace, num_cus, static_cast<hipStream_t>(stream)))
        return api_fail(FGD_ERR_HIP, "JS distance launch failed");
    return FGD_OK;
}

fgd_status fgd_stream_js_pattern(const void *logits_avg, const void *logits_workers, int32_t dtype,
                                 int32_t num_workers, int64_t num_tokens, int64_t vocab, int64_t ldk, void *workspace,
                                 int64_t workspace_bytes, void *stream) {
    fgd::api_clear();
    if (fgd_status st = check_rows(logits_avg, logits_workers, dtype, num_workers, num_tokens, vocab, ldk, workspace,
                                   workspace_bytes))
        return st;
    int num_cus = 0;
    if (fgd_status st = fgd::api_device_cus(num_cus)) return st;
    if (!fgd::js_pattern_launch(logits_avg, logits_workers, dtype == FGD_BF16, num_workers, num_tokens, vocab, ldk,
                                workspace, num_cus, static_cast<hipStream_t>(stream)))
        return api_fail(FGD_ERR_HIP, "JS pattern launch failed");
    return FGD_OK;
}

}  // extern "C"
