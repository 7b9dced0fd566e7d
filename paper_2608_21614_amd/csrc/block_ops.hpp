// block_ops.hpp -- workgroup-level building blocks of the routing front end:
// router scores on MFMA, the wave-argmax top-k gate, and the chunked counting
// sort that repacks the (token, expert) pairs.
#pragma once

#include <limits.h>
#include <math.h>

#include "common.hpp"

namespace saem {

constexpr int kFrontThreads = 1024;            // 16 waves
constexpr int kFrontWaves = kFrontThreads / kWave;
constexpr int kLgPitch = 257;                   // LDS row pitch of a score tile (E <= 256)
constexpr int kScoreChunk = 64;                 // experts (4 MFMA row tiles) per reduction pass

// Integer key with the order of the float scores: equal keys iff equal scores
// (-0 is folded into +0), larger key iff larger score.
__device__ __forceinline__ int score_key(float f) {
    int b = __float_as_int(f);
    if (b == (int)0x80000000) b = 0;
    return b >= 0 ? b : (b ^ 0x7fffffff);
}

// Maximum over the wave: DPP within each row of 16 lanes (each step folds into
// one v_max_i32 with a DPP operand), then the four row maxima on the scalar unit.
__device__ __forceinline__ int wave_max_i32(int v) {
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));   // quad_perm 1,0,3,2
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));   // quad_perm 2,3,0,1
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x124, 0xF, 0xF, true));  // row_ror 4
    v = max(v, __builtin_amdgcn_mov_dpp(v, 0x128, 0xF, 0xF, true));  // row_ror 8
    const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return max(max(r0, r1), max(r2, r3));
}

__device__ __forceinline__ int wave_min_i32(int v) {
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x124, 0xF, 0xF, true));
    v = min(v, __builtin_amdgcn_mov_dpp(v, 0x128, 0xF, 0xF, true));
    const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return min(min(r0, r1), min(r2, r3));
}

// LDS the top-k needs: selected (score, expert) of up to 64 rows x 8.
constexpr int kTopkLdsWords = 2 * 64 * 8;

// Top-k gate of `rows` tokens whose scores sit in LDS (s_lg, pitch kLgPitch),
// by the whole workgroup.  Experts are totally ordered by (score desc, expert
// id asc); the rank of expert e in row t is the number of experts before it in
// that order, and e is the j-th choice of t iff its rank is j < k.  One wave
// per token picks the choices in rank order, k rounds of a wave argmax over
// integer keys with the scores' order: one expert per lane for E <= 64, up to
// four per lane (E <= 256) with the lowest id among the lanes' equal offers.  The gate of choice j is exp(s_j - s_0) /
// sum_j' exp(s_j' - s_0), summed in j order; a score equal to the top one
// contributes exactly 1 (so all-equal rows, -inf included, get 1/k).
// Writes out_idx/out_w rows [t0, t0 + rows) and, if given, lds_idx[t*k + j].
// Ends with a barrier.  (NaN scores: undefined selection, never an index
// outside [-1, E).)
__device__ inline void topk_block(const float* s_lg, int rows, int E, int k, int t0, int32_t* out_idx,
                                       float* out_w, int32_t* lds_idx, float* s_selv, int* s_sele) {
    for (int i = threadIdx.x; i < rows * 8; i += blockDim.x) s_sele[i] = -1;
    __syncthreads();
    if (E <= kWave) {
        // one wave per row, lane e holds score e; round j takes the largest
        // score among the experts not yet chosen (wave max) and, among equal
        // scores, the lowest expert id (lowest set bit of a ballot)
        const int lane = lane_id(), nw = blockDim.x / kWave;
        for (int t = threadIdx.x / kWave; t < rows; t += nw) {
            const float v = (lane < E) ? s_lg[t * kLgPitch + lane] : 0.f;
            const int key = score_key(v);
            bool open = lane < E;
            for (int j = 0; j < k; ++j) {
                const int m = wave_max_i32(open ? key : INT_MIN);
                const unsigned long long cand = __ballot(open && key == m);  // never empty: k <= E
                const int e = cand ? __ffsll((long long)cand) - 1 : -1;
                if (lane == e) open = false;
                if (lane == 0 && e >= 0) {
                    s_selv[t * 8 + j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), e));
                    s_sele[t * 8 + j] = e;
                }
            }
        }
    } else {
        // E <= 256: lane l holds experts l, l + 64, l + 128, l + 192.  Each round a
        // lane offers its best open expert (largest key, then lowest id), the wave
        // takes the largest key, and among the lanes offering it the lowest id.
        const int lane = lane_id(), nw = blockDim.x / kWave;
        for (int t = threadIdx.x / kWave; t < rows; t += nw) {
            int key[4];
            bool open[4];
#pragma unroll
            for (int sl = 0; sl < 4; ++sl) {
                const int e = lane + kWave * sl;
                open[sl] = e < E;
                key[sl] = score_key(open[sl] ? s_lg[t * kLgPitch + e] : 0.f);
            }
            for (int j = 0; j < k; ++j) {
                int kb = INT_MIN, eb = INT_MAX;
#pragma unroll
                for (int sl = 0; sl < 4; ++sl)
                    if (open[sl] && (eb == INT_MAX || key[sl] > kb)) {
                        kb = key[sl];
                        eb = lane + kWave * sl;
                    }
                const int m = wave_max_i32(eb != INT_MAX ? kb : INT_MIN);
                const int e = wave_min_i32((eb != INT_MAX && kb == m) ? eb : INT_MAX);  // never INT_MAX: k <= E
#pragma unroll
                for (int sl = 0; sl < 4; ++sl)
                    if (lane + kWave * sl == e) open[sl] = false;
                if (lane == 0 && e != INT_MAX) {
                    s_selv[t * 8 + j] = s_lg[t * kLgPitch + e];
                    s_sele[t * 8 + j] = e;
                }
            }
        }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < rows * k; idx += blockDim.x) {
        const int t = idx / k, j = idx % k;
        const float top = s_selv[t * 8];
        float sum = 0.f, mine = 0.f;
        for (int jj = 0; jj < k; ++jj) {
            const float sv = s_selv[t * 8 + jj];
            const float term = (sv == top) ? 1.0f : expf(sv - top);
            sum += term;
            if (jj == j) mine = term;
        }
        const int e = s_sele[t * 8 + j];
        out_idx[(size_t)(t0 + t) * k + j] = e;
        out_w[(size_t)(t0 + t) * k + j] = mine / sum;
        if (lds_idx) lds_idx[t * k + j] = e;
    }
    __syncthreads();
}

// Router scores of tokens [t0, t0 + 16*TT) for all E experts on MFMA (bf16
// inputs: 16x16x32; fp32 inputs: 16x16x4, two per 8-element fragment).
// The 16 waves of the workgroup are TT token tiles x KP K parts (TT * KP = 16);
// K part p takes the 32-wide K steps p, p + KP, p + 2 KP, ...  Partial tiles go
// through `red` ([KP][16 TT][64] fp32) and are added in K-part order, so the
// fp32 scores do not depend on timing.  Result: s_lg[row][e] = score + bias[e]
// for row = t - t0 (rows of tokens >= T are left as garbage).
template <typename Elt, int TT, int KP>
__device__ void router_scores_mfma(int T, int H, int E, const Elt* __restrict__ x, const Elt* __restrict__ wr,
                                   const float* __restrict__ bias, int t0, float* s_lg, float* red) {
    static_assert(TT * KP == kFrontWaves, "16 waves");
    constexpr int U = sizeof(Elt) == 2 ? 4 : 2;  // K steps per load batch (registers: 1024-thread workgroups)
    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;
    const int tt = wave % TT, kp = wave / TT;
    const int tok = t0 + 16 * tt + r;
    const Elt* xp = (tok < T) ? x + (size_t)tok * H + kq : nullptr;
    const int nsteps = H / 32;
    const int n_my = (nsteps > kp) ? (nsteps - kp + KP - 1) / KP : 0;
    for (int c0 = 0; c0 < E; c0 += kScoreChunk) {
        f32x4 acc[4];
        const Elt* wp[4];
        bool live[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int e = c0 + 16 * m + r;
            live[m] = c0 + 16 * m < E;
            wp[m] = (e < E) ? wr + (size_t)e * H + kq : nullptr;
        }
        for (int i = 0; i < n_my; i += U) {
            Frag8<Elt> A[U][4], B[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int s = kp + KP * (i + u);
                const bool ok = i + u < n_my;
                B[u] = (ok && xp) ? load_frag(xp + s * 32) : zero_frag<Elt>();
#pragma unroll
                for (int m = 0; m < 4; ++m) A[u][m] = (ok && wp[m]) ? load_frag(wp[m] + s * 32) : zero_frag<Elt>();
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    if (live[m]) acc[m] = mma_frag(A[u][m], B[u], acc[m]);
        }
        // lane holds experts 16m + 4(lane/16) + i of token row 16 tt + r
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                red[(kp * 16 * TT + 16 * tt + r) * kScoreChunk + 16 * m + 4 * (lane >> 4) + i] = acc[m][i];
        __syncthreads();
        for (int idx = threadIdx.x; idx < 16 * TT * kScoreChunk; idx += kFrontThreads) {
            const int row = idx / kScoreChunk, el = idx % kScoreChunk, e = c0 + el;
            if (e >= E) continue;
            float v = red[row * kScoreChunk + el];
            for (int p = 1; p < KP; ++p) v += red[(p * 16 * TT + row) * kScoreChunk + el];
            s_lg[row * kLgPitch + e] = v + (bias ? bias[e] : 0.f);
        }
        __syncthreads();
    }
}

// LDS ints the repack needs with NT threads.
template <int NT>
constexpr int repack_lds_ints() {
    return 4 * 256 + (NT / 64) * 256 + 4;
}

// Expert-aligned repacking of the T*k pairs in chunks of NT pairs (chunk c =
// pairs [c NT, (c + 1) NT)); a workgroup of NT threads scatters the chunks
// [c_begin, c_end) in order:
//   1. it counts all pairs per expert, and separately the pairs before c_begin,
//      with LDS atomics (order-free; the ids are a few tens of KB and stay in L2);
//   2. one wave scans the counts in group order -- resident experts by id, then
//      offloaded experts by id -- into segment starts and n_res; the first
//      chunk's pairs of expert e start after the earlier chunks' pairs of e;
//   3. one pair per thread per chunk: inside a wave the lanes holding the same
//      expert are found with 8 ballots over the bits of the expert id, a lane's
//      rank is the popcount of the matching lanes below it, and each wave adds
//      the counts of the waves before it (LDS); after the chunk every expert's
//      start moves past the chunk's pairs.  Pairs keep their index order inside
//      an expert: a stable counting sort with no global atomics, and the same
//      result for any split of the chunks over workgroups.
// The workgroup with c_begin == 0 also writes counts, seg_start and n_res.
// ids outside [0, E) are dropped (inv_perm = -1); the packed rows they leave
// over at the end, [sum(counts), T*k), get perm = -1.
template <int NT>
__device__ inline void repack_chunks(int T, int E, int k, int slots, int c_begin, int c_end,
                                     const int32_t* __restrict__ idx, const int32_t* __restrict__ expert_slot,
                                     int32_t* __restrict__ counts, int32_t* __restrict__ seg_start,
                                     int32_t* __restrict__ perm, int32_t* __restrict__ inv_perm,
                                     int32_t* __restrict__ n_res, int* lds) {
    int* s_cnt = lds;
    int* s_pre = lds + 256;
    int* s_base = lds + 512;
    int* s_res = lds + 768;
    constexpr int NW = NT / 64;
    int* s_wcnt = lds + 1024;               // [NW][256]
    int* s_nres = lds + 1024 + NW * 256;
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int P = T * k;
    const int c0 = c_begin * NT;

    for (int e = tid; e < 256; e += NT) {
        s_cnt[e] = 0;
        s_pre[e] = 0;
        s_res[e] = (e < E) ? (is_resident(expert_slot[e], slots) ? 1 : 0) : 0;
    }
    __syncthreads();
    for (int q = tid; q < P; q += NT) {
        const int e = idx[q];
        if (e >= 0 && e < E) {
            atomicAdd(&s_cnt[e], 1);
            if (q < c0) atomicAdd(&s_pre[e], 1);
        }
    }
    __syncthreads();
    if (wave == 0) {
        int rs = 0, os = 0;  // lane owns experts 4 lane .. 4 lane + 3
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            if (e < E) {
                if (s_res[e]) rs += s_cnt[e];
                else os += s_cnt[e];
            }
        }
        int rinc = rs, oinc = os;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int a = __shfl_up(rinc, off, 64);
            const int b = __shfl_up(oinc, off, 64);
            if (lane >= off) {
                rinc += a;
                oinc += b;
            }
        }
        const int rtot = __shfl(rinc, 63, 64);
        const int otot = __shfl(oinc, 63, 64);
        int rp = rinc - rs, op = rtot + (oinc - os);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            if (e < E) {
                if (s_res[e]) {
                    s_base[e] = rp;
                    rp += s_cnt[e];
                } else {
                    s_base[e] = op;
                    op += s_cnt[e];
                }
            }
        }
        if (lane == 0) {
            s_nres[0] = rtot;
            s_nres[1] = rtot + otot;  // valid pairs: the packed rows that get a pair
        }
    }
    __syncthreads();
    if (c_begin == 0) {
        for (int e = tid; e < E; e += NT) {
            counts[e] = s_cnt[e];
            seg_start[e] = s_base[e];
        }
        if (tid == 0) *n_res = s_nres[0];
        // rows past the valid pairs (there are some only when ids outside [0, E) were
        // dropped) get no pair: mark them, so no reader takes a stale entry for one
        for (int p = s_nres[1] + tid; p < P; p += NT) perm[p] = -1;
    }
    for (int e = tid; e < E; e += NT) s_base[e] += s_pre[e];

    const unsigned long long lt_mask = (1ull << lane) - 1ull;
    for (int c = c_begin; c < c_end; ++c) {
        for (int i = tid; i < NW * 256; i += NT) s_wcnt[i] = 0;
        __syncthreads();
        const int q = c * NT + tid;
        const int e = (q < P) ? idx[q] : -1;
        const bool valid = (e >= 0 && e < E);
        unsigned long long m = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = valid && ((e >> b) & 1);
            const unsigned long long bb = __ballot(bit);
            m &= bit ? bb : ~bb;
        }
        const int rank = __popcll(m & lt_mask);
        if (valid && rank == 0) s_wcnt[wave * 256 + e] = __popcll(m);
        __syncthreads();
        if (valid) {
            int p = s_base[e] + rank;
            for (int w = 0; w < wave; ++w) p += s_wcnt[w * 256 + e];
            perm[p] = q;
            inv_perm[q] = p;
        } else if (q < P) {
            inv_perm[q] = -1;
        }
        __syncthreads();
        for (int ee = tid; ee < E; ee += NT) {
            int sum = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) sum += s_wcnt[w * 256 + ee];
            s_base[ee] += sum;
        }
        __syncthreads();
    }
}

}  // namespace saem
