// host_abi.cpp -- the host-only part of the C ABI of libsaem_moe.so: version,
// status strings, the shape rules every call checks first (moe_check_dims) and
// the stage-boundary residency plan (Section IV-C.2).  Plain C++, built with the
// system compiler; no device code and no HIP runtime calls.
#include <stdint.h>

#include <algorithm>

#include "saem_moe.h"

namespace {

constexpr long long kMaxRows = 1ll << 24;  // T*k + S*T rows handled by one call

}  // namespace

extern "C" {

int moe_abi_version(void) { return MOE_ABI_VERSION; }

const char* moe_status_str(moe_status s) {
    switch (s) {
        case MOE_OK: return "ok";
        case MOE_ERR_INVALID_ARG: return "invalid argument";
        case MOE_ERR_UNSUPPORTED: return "unsupported shape or option";
        case MOE_ERR_WORKSPACE: return "workspace missing or too small";
        case MOE_ERR_HIP: return "HIP launch or runtime error";
        case MOE_ERR_SCRATCH_LIMIT:
            return "layer needs more workspace than the fixed scratch array of the no-allocation entry point";
    }
    return "unknown status";
}

moe_status moe_check_dims(const moe_dims* d) {
    if (!d) return MOE_ERR_INVALID_ARG;
    if (d->tokens < 0 || d->hidden <= 0 || d->experts <= 0 || d->ffn <= 0 || d->top_k <= 0 || d->shared < 0 ||
        d->slots < 0)
        return MOE_ERR_INVALID_ARG;
    if (d->dtype != MOE_F32 && d->dtype != MOE_BF16) return MOE_ERR_INVALID_ARG;
    if (d->top_k > d->experts || d->slots > d->experts) return MOE_ERR_INVALID_ARG;
    if (d->shared > 0 && d->shared_ffn <= 0) return MOE_ERR_INVALID_ARG;
    if (d->experts > 256 || d->top_k > 8 || d->shared > 8) return MOE_ERR_UNSUPPORTED;
    if (d->hidden % 64 != 0 || d->ffn % 64 != 0) return MOE_ERR_UNSUPPORTED;
    if (d->shared > 0 && d->shared_ffn % 64 != 0) return MOE_ERR_UNSUPPORTED;
    const long long rows = (long long)d->tokens * d->top_k + (long long)d->shared * d->tokens;
    if (rows > kMaxRows) return MOE_ERR_UNSUPPORTED;
    if ((long long)d->hidden > (1 << 20) || (long long)d->ffn > (1 << 20) || (long long)d->shared_ffn > (1 << 20))
        return MOE_ERR_UNSUPPORTED;
    return MOE_OK;
}

moe_status moe_stage_plan(int32_t experts, int32_t slots, const int64_t* log, const int32_t* prev_slot,
                          int32_t* new_slot) {
    if (experts <= 0 || experts > 256 || slots < 0 || slots > experts || !log || !prev_slot || !new_slot)
        return MOE_ERR_INVALID_ARG;
    int order[256];
    for (int e = 0; e < experts; ++e) order[e] = e;
    std::stable_sort(order, order + experts, [&](int a, int b) { return log[a] > log[b]; });
    bool keep[256] = {false};
    for (int i = 0; i < slots; ++i) keep[order[i]] = true;
    bool used[256] = {false};
    for (int e = 0; e < experts; ++e) {
        new_slot[e] = -1;
        const int ps = prev_slot[e];
        if (keep[e] && ps >= 0 && ps < slots && !used[ps]) {
            new_slot[e] = ps;
            used[ps] = true;
        }
    }
    int next_free = 0;
    for (int i = 0; i < slots; ++i) {
        const int e = order[i];
        if (new_slot[e] >= 0) continue;
        while (next_free < slots && used[next_free]) ++next_free;
        new_slot[e] = next_free;
        used[next_free] = true;
    }
    return MOE_OK;
}

}  // extern "C"
