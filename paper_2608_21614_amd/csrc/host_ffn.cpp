// host_ffn.cpp -- in-situ CPU execution of the offloaded experts (SAEM Section
// IV-D: experts that are not GPU-resident run where their weights are, on the
// host, over the packed offloaded rows; Section IV-D.2: in parallel with the
// GPU's resident experts, by threads kept on one NUMA node, merged afterwards
// through moe_combine's y_off).
//
// Host code only (built with the system C++ compiler).  Per offloaded expert e
// with c_e packed rows X_e (rows [seg_start[e] - n_res, + c_e) of off_rows):
//   A_e = silu(X_e W1_e) * (X_e W3_e)      [c_e, F]   fp32
//   Y_e = A_e W2_e                          [c_e, H]   fp32 -> y_off rows
// A work item is 64 output features of one expert; it walks K in 512-wide
// slices so that the slice of (up to) 8 token rows stays in L1 while the
// item's 64 weight rows stream past it: every weight element is read from
// memory once per block of 8 rows (from L2 for later blocks), so the work is
// bound by host memory bandwidth on the expert weights, as the device FFN is
// by HBM.  Dot products: AVX2 FMAs on fp32 (bf16 widened); for bf16 layers on a
// CPU with the AVX-512 bf16 dot-product instruction, phase 1 (bf16 token rows
// times bf16 weights) uses it instead: 32 products per instruction, each exact
// in fp32, added in pairs into fp32 accumulators.
#include <errno.h>
#include <immintrin.h>
#include <pthread.h>
#include <sched.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <thread>
#include <vector>

#include "saem_moe.h"

namespace {

constexpr int kRowBlock = 8;   // token rows per weight-row pass (fp32 accumulators)
constexpr int kChunk = 64;     // output features per work item

inline float bf16_bits_to_f32(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

constexpr int kKBlock = 512;   // K elements per pass: kRowBlock fp32 token rows (16 KB) stay in L1

// sums[f * kRowBlock + r] += sum_{k < klen} W[f][k] * x[r * ldx + k]  for f < nf, r < R,
// where W[f] = w + f * ldw (elements of the weight dtype); klen % 8 == 0.
template <int R, bool kBf16>
void block_dot_generic(const void* w, size_t ldw, const float* x, size_t ldx, int klen, int nf, float* sums) {
    for (int f = 0; f < nf; ++f) {
        for (int r = 0; r < R; ++r) {
            float acc = 0.f;
            for (int k = 0; k < klen; ++k) {
                const float wk = kBf16 ? bf16_bits_to_f32(static_cast<const uint16_t*>(w)[f * ldw + k])
                                       : static_cast<const float*>(w)[f * ldw + k];
                acc += wk * x[(size_t)r * ldx + k];
            }
            sums[f * kRowBlock + r] += acc;
        }
    }
}

template <int R, bool kBf16>
__attribute__((target("avx2,fma"))) void block_dot_avx2(const void* w, size_t ldw, const float* x, size_t ldx,
                                                       int klen, int nf, float* sums) {
    for (int f = 0; f < nf; ++f) {
        __m256 acc[R];
        for (int r = 0; r < R; ++r) acc[r] = _mm256_setzero_ps();
        for (int k = 0; k < klen; k += 8) {
            __m256 wv;
            if (kBf16) {
                const __m128i h = _mm_loadu_si128(
                    reinterpret_cast<const __m128i*>(static_cast<const uint16_t*>(w) + f * ldw + k));
                wv = _mm256_castsi256_ps(_mm256_slli_epi32(_mm256_cvtepu16_epi32(h), 16));
            } else {
                wv = _mm256_loadu_ps(static_cast<const float*>(w) + f * ldw + k);
            }
            for (int r = 0; r < R; ++r) acc[r] = _mm256_fmadd_ps(wv, _mm256_loadu_ps(x + (size_t)r * ldx + k), acc[r]);
        }
        for (int r = 0; r < R; ++r) {
            const __m128 lo = _mm256_castps256_ps128(acc[r]), hi = _mm256_extractf128_ps(acc[r], 1);
            __m128 s = _mm_add_ps(lo, hi);
            s = _mm_add_ps(s, _mm_movehl_ps(s, s));
            s = _mm_add_ss(s, _mm_shuffle_ps(s, s, 0x55));
            sums[f * kRowBlock + r] += _mm_cvtss_f32(s);
        }
    }
}

// The same over bf16 token rows x (elements), bf16 weights, with vdpbf16ps: every
// product of two bf16 values is exact in fp32; pairs of products are added into the
// fp32 accumulators.  The instruction treats inputs below the fp32 normal range as
// zero and flushes such results to zero.  klen % 32 == 0.
template <int R>
__attribute__((target("avx512f,avx512bw,avx512bf16"))) void block_dot_bf16dp(const void* w, size_t ldw,
                                                                           const uint16_t* x, size_t ldx,
                                                                           int klen, int nf, float* sums) {
    for (int f = 0; f < nf; ++f) {
        const uint16_t* wr = static_cast<const uint16_t*>(w) + f * ldw;
        __m512 acc[R];
        for (int r = 0; r < R; ++r) acc[r] = _mm512_setzero_ps();
        for (int k = 0; k < klen; k += 32) {
            const __m512bh wv = (__m512bh)_mm512_loadu_si512(wr + k);
            for (int r = 0; r < R; ++r)
                acc[r] = _mm512_dpbf16_ps(acc[r], wv, (__m512bh)_mm512_loadu_si512(x + (size_t)r * ldx + k));
        }
        for (int r = 0; r < R; ++r) sums[f * kRowBlock + r] += _mm512_reduce_add_ps(acc[r]);
    }
}

using BlockDotBf16 = void (*)(const void*, size_t, const uint16_t*, size_t, int, int, float*);

BlockDotBf16 pick_rows_bf16dp(int R) {
#define SAEM_ROWS(n) \
    case n: return block_dot_bf16dp<n>;
    switch (R) {
        SAEM_ROWS(1) SAEM_ROWS(2) SAEM_ROWS(3) SAEM_ROWS(4) SAEM_ROWS(5) SAEM_ROWS(6) SAEM_ROWS(7)
        default: return block_dot_bf16dp<8>;
    }
#undef SAEM_ROWS
}

// rows_times_weights for bf16 token rows and bf16 weights on the dot-product instruction.
void rows_times_weights_bf16dp(const void* w, size_t ldw, int K, int nf, const uint16_t* x, size_t ldx, int R,
                               float* out) {
    const BlockDotBf16 fn = pick_rows_bf16dp(R);
    for (int i = 0; i < nf * kRowBlock; ++i) out[i] = 0.f;
    for (int k0 = 0; k0 < K; k0 += kKBlock) {
        const int klen = std::min(kKBlock, K - k0);
        fn(static_cast<const uint16_t*>(w) + k0, ldw, x + k0, ldx, klen, nf, out);
    }
}

using BlockDot = void (*)(const void*, size_t, const float*, size_t, int, int, float*);

template <bool kBf16>
BlockDot pick_rows(int R, bool avx2) {
#define SAEM_ROWS(n) \
    case n: return avx2 ? block_dot_avx2<n, kBf16> : block_dot_generic<n, kBf16>;
    switch (R) {
        SAEM_ROWS(1) SAEM_ROWS(2) SAEM_ROWS(3) SAEM_ROWS(4) SAEM_ROWS(5) SAEM_ROWS(6) SAEM_ROWS(7)
        default: return avx2 ? block_dot_avx2<8, kBf16> : block_dot_generic<8, kBf16>;
    }
#undef SAEM_ROWS
}

// out[f * kRowBlock + r] = W[f] . x[r] over the full K, f < nf (<= kChunk), all `rows`
// token rows (kRowBlock at a time, out has room for kChunk * kRowBlock per block of rows
// -- called once per row block).  K is walked in kKBlock slices so the token slice is
// reused from L1 by all nf weight rows.
void rows_times_weights(bool bf16, const void* w, size_t ldw, int K, int nf, const float* x, size_t ldx, int R,
                        float* out) {
    static const bool avx2 = __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma");
    const BlockDot fn = bf16 ? pick_rows<true>(R, avx2) : pick_rows<false>(R, avx2);
    const size_t elt = bf16 ? 2 : 4;
    for (int i = 0; i < nf * kRowBlock; ++i) out[i] = 0.f;
    for (int k0 = 0; k0 < K; k0 += kKBlock) {
        const int klen = std::min(kKBlock, K - k0);
        fn(static_cast<const char*>(w) + (size_t)k0 * elt, ldw, x + k0, ldx, klen, nf, out);
    }
}

// CPUs of the calling thread's affinity mask that sit on the NUMA node of the
// first of them (all of them if the node map cannot be read).
std::vector<int> local_cpus() {
    cpu_set_t set;
    CPU_ZERO(&set);
    std::vector<int> allowed;
    if (sched_getaffinity(0, sizeof(set), &set) == 0)
        for (int c = 0; c < CPU_SETSIZE; ++c)
            if (CPU_ISSET(c, &set)) allowed.push_back(c);
    if (allowed.empty()) return allowed;
    for (int node = 0; node < 64; ++node) {
        char path[96];
        snprintf(path, sizeof(path), "/sys/devices/system/node/node%d/cpulist", node);
        FILE* f = fopen(path, "r");
        if (!f) {
            if (node == 0) return allowed;
            continue;
        }
        std::vector<int> cpus;
        int a, b;
        char sep;
        while (fscanf(f, "%d", &a) == 1) {
            b = a;
            if (fscanf(f, "%c", &sep) == 1 && sep == '-') {
                if (fscanf(f, "%d", &b) != 1) break;
                if (fscanf(f, "%c", &sep) != 1) sep = '\n';
            }
            for (int c = a; c <= b; ++c) cpus.push_back(c);
            if (sep != ',') break;
        }
        fclose(f);
        if (std::find(cpus.begin(), cpus.end(), allowed[0]) != cpus.end()) {
            std::vector<int> local;
            for (int c : allowed)
                if (std::find(cpus.begin(), cpus.end(), c) != cpus.end()) local.push_back(c);
            return local.empty() ? allowed : local;
        }
    }
    return allowed;
}

// Runs fn(item) for item in [0, n_items) on `nthreads` threads, items taken in
// order from an atomic counter.  Unpinned, the caller is one of the threads.
// Pinned (cpus given), all `nthreads` are new threads, worker i on cpus[i % n],
// and the caller only waits: its own affinity is never changed.
template <typename Fn>
void parallel_items(int n_items, int nthreads, const std::vector<int>& cpus, Fn fn) {
    std::atomic<int> next{0};
    auto work = [&]() {
        for (int i = next.fetch_add(1); i < n_items; i = next.fetch_add(1)) fn(i);
    };
    std::vector<std::thread> pool;
    if (cpus.empty()) {
        pool.reserve(nthreads > 1 ? nthreads - 1 : 0);
        for (int t = 1; t < nthreads; ++t) pool.emplace_back(work);
        work();
    } else {
        pool.reserve(nthreads);
        for (int t = 0; t < nthreads; ++t)
            pool.emplace_back([&, t]() {
                cpu_set_t one;
                CPU_ZERO(&one);
                CPU_SET(cpus[t % cpus.size()], &one);
                pthread_setaffinity_np(pthread_self(), sizeof(one), &one);
                work();
            });
    }
    for (auto& th : pool) th.join();
}

struct Job {
    int e;       // expert
    int row0;    // first row in off_rows / y_off
    int rows;
};

}  // namespace

extern "C" {

moe_status moe_host_ffn(const moe_dims* dims, const int32_t* counts, const int32_t* seg_start, int32_t n_res,
                        const void* const* w13, const void* const* w2, const void* off_rows, float* y_off,
                        int32_t threads, uint32_t flags) {
    if (moe_status st = moe_check_dims(dims); st != MOE_OK) return st;
    if (!counts || !seg_start || !w13 || !w2 || (flags & ~(MOE_HOST_PIN | MOE_HOST_NO_BF16_DOT)))
        return MOE_ERR_INVALID_ARG;
    const int T = dims->tokens, H = dims->hidden, E = dims->experts, F = dims->ffn, k = dims->top_k;
    const int P = T * k;
    if (n_res < 0 || n_res > P) return MOE_ERR_INVALID_ARG;
    const int n_off = P - n_res;
    if (n_off > 0 && (!off_rows || !y_off)) return MOE_ERR_INVALID_ARG;
    // offloaded experts: segments inside [n_res, P), non-overlapping, covering it
    std::vector<Job> jobs;
    long long covered = 0;
    for (int e = 0; e < E; ++e) {
        const int c = counts[e], s = seg_start[e];
        if (c < 0) return MOE_ERR_INVALID_ARG;
        if (c == 0 || s < n_res) continue;  // idle, or a resident segment (rows before n_res)
        if (s + (long long)c > P) return MOE_ERR_INVALID_ARG;
        if (!w13[e] || !w2[e]) return MOE_ERR_INVALID_ARG;
        jobs.push_back({e, s - n_res, c});
        covered += c;
    }
    if (covered != n_off) return MOE_ERR_INVALID_ARG;
    std::sort(jobs.begin(), jobs.end(), [](const Job& a, const Job& b) { return a.row0 < b.row0; });
    for (size_t i = 1; i < jobs.size(); ++i)
        if (jobs[i].row0 < jobs[i - 1].row0 + jobs[i - 1].rows) return MOE_ERR_INVALID_ARG;
    if (n_off == 0) return MOE_OK;

    const bool bf16 = dims->dtype == MOE_BF16;
    const size_t elt = bf16 ? 2 : 4;
    int nthreads = threads > 0 ? threads : (int)std::max(1u, std::thread::hardware_concurrency());
    std::vector<int> cpus;
    if (flags & MOE_HOST_PIN) cpus = local_cpus();
    if (!cpus.empty() && threads <= 0) nthreads = (int)cpus.size();

    // phase 1 on the bf16 dot-product instruction where the CPU has it (bf16 rows as they
    // are), else on fp32 rows
    static const bool cpu_bf16dp = __builtin_cpu_supports("avx512bf16");
    const bool bf16dp = bf16 && cpu_bf16dp && !(flags & MOE_HOST_NO_BF16_DOT);
    const uint16_t* xb = static_cast<const uint16_t*>(off_rows);
    std::vector<float> xf(bf16dp ? 0 : (size_t)n_off * H), act((size_t)n_off * F);
    if (!bf16dp)
        for (size_t i = 0; i < (size_t)n_off * H; ++i)
            xf[i] = bf16 ? bf16_bits_to_f32(xb[i]) : static_cast<const float*>(off_rows)[i];

    // work items: (job, block of kChunk output features); inside an item every
    // weight row is applied to all of the expert's rows, kRowBlock at a time,
    // while it sits in the core's L1
    struct Item {
        int job, f0;
    };
    std::vector<Item> items;
    auto make_items = [&](int width) {
        items.clear();
        for (int j = 0; j < (int)jobs.size(); ++j)
            for (int f0 = 0; f0 < width; f0 += kChunk) items.push_back({j, f0});
    };

    // phase 1: act[row, f] = silu(x . W1[f]) * (x . W3[f])
    make_items(F);
    parallel_items((int)items.size(), nthreads, cpus, [&](int i) {
        const Item it = items[i];
        const Job& jb = jobs[it.job];
        const char* w = static_cast<const char*>(w13[jb.e]);
        const int nf = std::min(kChunk, F - it.f0);
        float g[kChunk * kRowBlock], u[kChunk * kRowBlock];
        for (int r0 = 0; r0 < jb.rows; r0 += kRowBlock) {
            const int R = std::min(kRowBlock, jb.rows - r0);
            if (bf16dp) {
                const uint16_t* x = xb + (size_t)(jb.row0 + r0) * H;
                rows_times_weights_bf16dp(w + (size_t)it.f0 * H * elt, H, H, nf, x, H, R, g);
                rows_times_weights_bf16dp(w + (size_t)(F + it.f0) * H * elt, H, H, nf, x, H, R, u);
            } else {
                const float* x = xf.data() + (size_t)(jb.row0 + r0) * H;
                rows_times_weights(bf16, w + (size_t)it.f0 * H * elt, H, H, nf, x, H, R, g);
                rows_times_weights(bf16, w + (size_t)(F + it.f0) * H * elt, H, H, nf, x, H, R, u);
            }
            for (int f = 0; f < nf; ++f)
                for (int r = 0; r < R; ++r) {
                    const float gv = g[f * kRowBlock + r], uv = u[f * kRowBlock + r];
                    act[(size_t)(jb.row0 + r0 + r) * F + it.f0 + f] = gv / (1.0f + std::exp(-gv)) * uv;
                }
        }
    });
    // phase 2: y_off[row, h] = act[row] . W2[h]
    make_items(H);
    parallel_items((int)items.size(), nthreads, cpus, [&](int i) {
        const Item it = items[i];
        const Job& jb = jobs[it.job];
        const char* w = static_cast<const char*>(w2[jb.e]);
        const int nf = std::min(kChunk, H - it.f0);
        float y[kChunk * kRowBlock];
        for (int r0 = 0; r0 < jb.rows; r0 += kRowBlock) {
            const int R = std::min(kRowBlock, jb.rows - r0);
            rows_times_weights(bf16, w + (size_t)it.f0 * F * elt, F, F, nf, act.data() + (size_t)(jb.row0 + r0) * F, F,
                               R, y);
            for (int f = 0; f < nf; ++f)
                for (int r = 0; r < R; ++r) y_off[(size_t)(jb.row0 + r0 + r) * H + it.f0 + f] = y[f * kRowBlock + r];
        }
    });
    return MOE_OK;
}

moe_status moe_offload_plan(int32_t experts, const int32_t* counts, const int32_t* expert_slot, int32_t slots,
                            const moe_offload_rates* rates, int32_t max_copies, int32_t* choice) {
    if (experts <= 0 || experts > 256 || !counts || !expert_slot || !rates || !choice || slots < 0 ||
        max_copies < 0)
        return MOE_ERR_INVALID_ARG;
    const moe_offload_rates& r = *rates;
    if (!(r.expert_bytes > 0) || !(r.flops_per_pair > 0) || !(r.link_GBps > 0) || !(r.host_GBps > 0) ||
        !(r.host_GFLOPs > 0) || !(r.gpu_GBps > 0))
        return MOE_ERR_INVALID_ARG;
    struct Cand {
        int e;
        double t_host, t_gpu;
    };
    std::vector<Cand> cand;
    double host_total = 0.0;
    for (int e = 0; e < experts; ++e) {
        const bool resident = expert_slot[e] >= 0 && expert_slot[e] < slots;
        choice[e] = -1;
        if (resident || counts[e] <= 0) continue;
        choice[e] = 0;
        // host: stream the expert's weights from host memory, or its FLOPs, whichever is slower
        const double t_host =
            std::max(r.expert_bytes / (r.host_GBps * 1e9), counts[e] * r.flops_per_pair / (r.host_GFLOPs * 1e9));
        // GPU: copy the weights over the host link, then stream them from HBM once
        const double t_gpu = r.expert_bytes / (r.link_GBps * 1e9) + r.expert_bytes / (r.gpu_GBps * 1e9);
        host_total += t_host;
        if (t_gpu < t_host) cand.push_back({e, t_host, t_gpu});
    }
    // largest saving first; the host runs its experts one after another on all its
    // threads and the copies queue on the link, so stop once another copy would not
    // shorten the longer of the two queues
    std::stable_sort(cand.begin(), cand.end(),
                     [](const Cand& a, const Cand& b) { return a.t_host - a.t_gpu > b.t_host - b.t_gpu; });
    double link_total = 0.0;
    for (size_t i = 0; i < cand.size() && (int)i < max_copies; ++i) {
        const Cand& c = cand[i];
        if (std::max(host_total - c.t_host, link_total + c.t_gpu) >= std::max(host_total, link_total)) break;
        host_total -= c.t_host;
        link_total += c.t_gpu;
        choice[c.e] = 1;
    }
    return MOE_OK;
}

}  // extern "C"
