// Exercises the library's host-only C++ (shape rules, stage plan, the cue
// machine, the host FFN of the offloaded experts, the copy-or-host plan) under AddressSanitizer and
// UndefinedBehaviorSanitizer.  Built and run by tests/test_host_asan.py with g++;
// exits non-zero on a wrong result, the sanitizers abort on a memory error.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <random>
#include <vector>

#include "saem_moe.h"

static int fail(const char* what) {
    fprintf(stderr, "driver: %s\n", what);
    return 1;
}

// longest cue that ends the window (brute force), lowest id among identical cues
static int naive_match(const std::vector<std::vector<int32_t>>& cues, const std::vector<int32_t>& win) {
    int best = -1;
    size_t best_len = 0;
    for (size_t c = 0; c < cues.size(); ++c) {
        const auto& q = cues[c];
        if (q.size() > win.size() || q.size() <= best_len) continue;
        if (std::equal(q.begin(), q.end(), win.end() - q.size())) {
            best = (int)c;
            best_len = q.size();
        }
    }
    return best;
}

static int cue_machine(std::mt19937& rng) {
    for (int round = 0; round < 50; ++round) {
        const int V = 2 + (int)(rng() % 5), n = (int)(rng() % 10);
        std::vector<std::vector<int32_t>> cues(n);
        std::vector<int32_t> off(1, 0), tok;
        for (auto& q : cues) {
            q.resize(1 + rng() % 6);
            for (auto& t : q) t = (int32_t)(rng() % V);
            tok.insert(tok.end(), q.begin(), q.end());
            off.push_back((int32_t)tok.size());
        }
        const int64_t words = moe_cue_fsm_words((int64_t)tok.size());
        std::vector<int32_t> fsm((size_t)words);
        if (moe_cue_build(n, off.data(), tok.data(), fsm.data(), words) != MOE_OK) return fail("build");
        if (n > 0 && moe_cue_build(n, off.data(), tok.data(), fsm.data(), words - 1) != MOE_ERR_WORKSPACE)
            return fail("short buffer accepted");
        const int B = 1 + (int)(rng() % 7);
        std::vector<int32_t> state(B, 0), matched(B), t(B);
        std::vector<std::vector<int32_t>> win(B);
        for (int step = 0; step < 400; ++step) {
            for (int b = 0; b < B; ++b) {
                t[b] = (rng() % 50 == 0) ? -1 : (int32_t)(rng() % V);
                if (t[b] < 0) win[b].clear();
                else win[b].push_back(t[b]);
            }
            if (moe_cue_step(fsm.data(), B, t.data(), state.data(), matched.data()) != MOE_OK) return fail("step");
            for (int b = 0; b < B; ++b)
                if (matched[b] != (t[b] < 0 ? -1 : naive_match(cues, win[b]))) return fail("cue match differs");
        }
        state[0] = 1 << 30;
        if (moe_cue_step(fsm.data(), B, t.data(), state.data(), matched.data()) != MOE_ERR_INVALID_ARG)
            return fail("state out of range accepted");
    }
    return 0;
}

static uint16_t bf16_of(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static int host_ffn(std::mt19937& rng) {
    std::normal_distribution<float> nd(0.f, 1.f);
    for (int dt = 0; dt < 2; ++dt) {
        // 5 tokens, top-2, 4 experts, none resident: segments 0:[0,3) 1:[3,3) 2:[3,8) 3:[8,10)
        const int T = 5, k = 2, E = 4, H = 64, F = 64, P = T * k;
        moe_dims d = {T, H, E, F, k, 0, 0, 0, dt == 0 ? MOE_F32 : MOE_BF16};
        const int32_t counts[E] = {3, 0, 5, 2}, seg[E] = {0, 3, 3, 8};
        const size_t es = dt == 0 ? 4 : 2;
        std::vector<std::vector<uint8_t>> w13(E), w2(E);
        std::vector<const void*> p13(E, nullptr), p2(E, nullptr);
        auto fill = [&](std::vector<uint8_t>& v, size_t n, float scale) {
            v.resize(n * es);
            for (size_t i = 0; i < n; ++i) {
                const float f = nd(rng) * scale;
                if (dt == 0) memcpy(&v[i * 4], &f, 4);
                else {
                    const uint16_t b = bf16_of(f);
                    memcpy(&v[i * 2], &b, 2);
                }
            }
        };
        for (int e = 0; e < E; ++e) {
            if (!counts[e]) continue;
            fill(w13[e], (size_t)2 * F * H, 0.02f);
            fill(w2[e], (size_t)H * F, 0.02f);
            p13[e] = w13[e].data();
            p2[e] = w2[e].data();
        }
        std::vector<uint8_t> rows;
        fill(rows, (size_t)P * H, 1.f);
        std::vector<float> y((size_t)P * H, -1.f);
        for (int threads : {1, 3, 0})
            for (uint32_t flags : {0u, (uint32_t)MOE_HOST_NO_BF16_DOT})  // bf16 dot products where the CPU has them, and widened
                if (moe_host_ffn(&d, counts, seg, 0, p13.data(), p2.data(), rows.data(), y.data(), threads, flags) !=
                    MOE_OK)
                    return fail("host ffn");
        for (float v : y)
            if (v == -1.f || v != v) return fail("host ffn left a row unwritten");
        const int32_t bad_seg[E] = {0, 3, 4, 8};  // segments do not tile [0, P)
        if (moe_host_ffn(&d, counts, bad_seg, 0, p13.data(), p2.data(), rows.data(), y.data(), 2, 0) !=
            MOE_ERR_INVALID_ARG)
            return fail("bad segments accepted");
    }
    return 0;
}

static int offload_plan(std::mt19937& rng) {
    moe_offload_rates r = {17.3e6, 6.0 * 2048 * 1408, 55, 90, 500, 5900};
    for (int round = 0; round < 200; ++round) {
        const int E = 1 + (int)(rng() % 256), slots = (int)(rng() % (E + 1));
        std::vector<int32_t> counts(E), slot(E, -1), choice(E);
        for (auto& c : counts) c = (int32_t)(rng() % 40);
        for (int s = 0; s < slots; ++s) slot[rng() % E] = s;
        if (moe_offload_plan(E, counts.data(), slot.data(), slots, &r, (int)(rng() % 8), choice.data()) != MOE_OK)
            return fail("offload plan");
        for (int e = 0; e < E; ++e)
            if (choice[e] < -1 || choice[e] > 1) return fail("offload plan choice out of range");
    }
    return 0;
}

static int host_abi(std::mt19937& rng) {
    moe_dims ok = {32, 4096, 8, 14336, 2, 0, 0, 4, MOE_BF16};
    if (moe_check_dims(&ok) != MOE_OK) return fail("valid dims rejected");
    moe_dims bad = ok;
    bad.top_k = 9;
    if (moe_check_dims(&bad) == MOE_OK) return fail("k > E accepted");
    bad = ok;
    bad.hidden = 100;
    if (moe_check_dims(&bad) != MOE_ERR_UNSUPPORTED) return fail("H % 64 accepted");
    if (moe_check_dims(nullptr) != MOE_ERR_INVALID_ARG) return fail("NULL dims accepted");
    for (int s = -1; s <= 5; ++s)
        if (!moe_status_str((moe_status)s)) return fail("status string");
    for (int round = 0; round < 200; ++round) {
        const int E = 1 + (int)(rng() % 256), slots = (int)(rng() % (E + 1));
        std::vector<int64_t> log(E);
        std::vector<int32_t> prev(E, -1), next(E);
        for (auto& v : log) v = (int64_t)(rng() % 6);
        for (int s = 0; s < slots; ++s) prev[rng() % E] = s;
        if (moe_stage_plan(E, slots, log.data(), prev.data(), next.data()) != MOE_OK) return fail("stage plan");
        std::vector<int> seen(slots + 1, 0);
        for (int e = 0; e < E; ++e) {
            if (next[e] < -1 || next[e] >= slots) return fail("stage plan slot out of range");
            if (next[e] >= 0 && seen[next[e]]++) return fail("stage plan slot used twice");
        }
    }
    return 0;
}

int main() {
    std::mt19937 rng(12345);
    if (int rc = host_abi(rng)) return rc;
    if (int rc = cue_machine(rng)) return rc;
    if (int rc = host_ffn(rng)) return rc;
    if (int rc = offload_plan(rng)) return rc;
    printf("host code ok\n");
    return 0;
}
