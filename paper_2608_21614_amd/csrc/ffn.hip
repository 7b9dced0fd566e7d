// ffn.hip -- grouped SwiGLU expert FFN over the resident and shared experts
// (SAEM Section IV-D.2: resident experts on the matrix cores; Section IV-E.1:
// one batched execution per expert over its contiguous, repacked rows).
//
// Row space: packed rows [0, T*k) (resident experts first, see repack.hip),
// then the rows of shared expert s at T*k + s*T + t.
//   phase 1: act[p, f] = silu(x[tok(p)] . W1[:,f]) * (x[tok(p)] . W3[:,f])
//   phase 2: y[c][p, h] = sum over K chunk c of act[p, :] . W2[:,h]
//
// Three kernel families:
//  * stream  (bf16, T <= 64, decode): the weights are streamed from HBM exactly
//    once.  A workgroup owns 32 features (phase 1: 32 gate + 32 up weight
//    rows) or 64 outputs (phase 2: 64 rows of W2) of one expert; the weights are
//    the MFMA M side and the expert's tokens the N side, in tiles of 16.  Its
//    four waves split K and their partial tiles are summed through LDS in wave
//    order.  Phase 2 additionally splits K across workgroups into `ks` chunks
//    whose partial sums the combine adds in fixed order.  SwiGLU is applied in
//    the phase-1 epilogue, so gate and up projections are never stored.
//  * tiled   (bf16, T > 64, prefill): MFMA tiles of 64 weight rows x 64 tokens,
//    K staged through LDS in double-buffered 64-wide slabs; the phase-1 tile
//    interleaves 16 gate and 16 up rows per wave so SwiGLU runs in registers.
//  * f32     (fp32 layers): plain fp32 FMA, one output per thread.
// All of them read counts and offsets from device memory: the grid is sized for
// the worst case on the host and surplus workgroups exit at once.
#include "common.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

struct Args {
    int T, H, E, F, k, S, Fs, slots;
    const void* x;
    const int32_t* perm;
    const int32_t* counts;
    const int32_t* seg_start;
    const int32_t* expert_slot;
    const void* w13;
    const void* w2;
    const void* ws13;
    const void* ws2;
    void* act;
    int Fa;
    float* y;
    int ks;
    long long y_ks_stride;
    int max_routed;   // routed groups the grid reserves (>= active resident experts)
    int ipg_r;        // items (workgroups) per routed group
    int ipg_s;        // items per shared group
};

// One group of rows: a resident routed expert or a shared expert.
struct Group {
    int rowbase;   // first row in the row space
    int count;     // rows
    int routed;    // 1: rows are packed pairs (token = perm[p] / k); 0: row n is token n
    int Fg;        // expert width
    const uint8_t* w13;
    const uint8_t* w2;
};

// Active resident routed experts (ascending id) into s_list; returns their number.
// Must be called by all threads of a 256-thread workgroup.
__device__ int list_active(const Args& a, int* s_list, int* s_wsum) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int e = tid;
    bool act = false;
    if (e < a.E) {
        const int sl = a.expert_slot[e];
        act = is_resident(sl, a.slots) && a.counts[e] > 0;
    }
    const unsigned long long b = __ballot(act);
    if (lane == 0) s_wsum[wave] = __popcll(b);
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += s_wsum[w];
    if (act) s_list[base + __popcll(b & ((1ull << lane) - 1ull))] = e;
    const int n = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
    return n;
}

__device__ Group routed_group(const Args& a, int e, size_t elt) {
    Group g;
    const int P = a.T * a.k;
    int rb = a.seg_start[e];
    int c = a.counts[e];
    rb = rb < 0 ? 0 : (rb > P ? P : rb);
    c = c < 0 ? 0 : (c > P - rb ? P - rb : c);
    g.rowbase = rb;
    g.count = c;
    g.routed = 1;
    g.Fg = a.F;
    const size_t slot = (size_t)a.expert_slot[e];
    g.w13 = static_cast<const uint8_t*>(a.w13) + slot * 2 * a.F * a.H * elt;
    g.w2 = static_cast<const uint8_t*>(a.w2) + slot * a.H * a.F * elt;
    return g;
}

__device__ Group shared_group(const Args& a, int s, size_t elt) {
    Group g;
    g.rowbase = a.T * a.k + s * a.T;
    g.count = a.T;
    g.routed = 0;
    g.Fg = a.Fs;
    g.w13 = static_cast<const uint8_t*>(a.ws13) + (size_t)s * 2 * a.Fs * a.H * elt;
    g.w2 = static_cast<const uint8_t*>(a.ws2) + (size_t)s * a.H * a.Fs * elt;
    return g;
}

// Token of row n of a group, or -1 when out of range.
__device__ __forceinline__ int group_token(const Args& a, const Group& g, int n) {
    if (n >= g.count) return -1;
    int t;
    if (g.routed) {
        const int q = a.perm[g.rowbase + n];
        t = (q >= 0) ? q / a.k : -1;
    } else {
        t = n;
    }
    return (t >= 0 && t < a.T) ? t : -1;
}

// ---------------------------------------------------------------------------
// stream kernel (decode)
// ---------------------------------------------------------------------------

template <int NT, bool kDown>
__global__ void __launch_bounds__(256) k_ffn_stream(Args a) {
    constexpr int MT = 4;                    // 16-row weight tiles per workgroup
    constexpr int U = (NT <= 2) ? 4 : 2;     // K steps per load batch
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    __shared__ f32x4 s_red[4][MT][NT][kWave];

    const int nact = list_active(a, s_list, s_wsum);
    const int item = blockIdx.x;
    Group g;
    int sub;
    if (item < a.max_routed * a.ipg_r) {
        const int gi = item / a.ipg_r;
        if (gi >= nact) return;
        g = routed_group(a, s_list[gi], 2);
        sub = item % a.ipg_r;
    } else {
        const int i2 = item - a.max_routed * a.ipg_r;
        const int s = i2 / a.ipg_s;
        if (s >= a.S) return;
        g = shared_group(a, s, 2);
        sub = i2 % a.ipg_s;
    }
    if (g.count == 0) return;

    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;

    // weight rows of this workgroup and the K range of this wave
    const uint16_t* wp[MT];
    int row0, kc = 0, s0, s1;
    if (!kDown) {
        const int f0 = sub * 32;
        row0 = f0;
        const uint16_t* w = reinterpret_cast<const uint16_t*>(g.w13);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const int feat = f0 + 16 * (m & 1) + r;
            const int row = (m < 2) ? feat : g.Fg + feat;
            wp[m] = w + (size_t)row * a.H + kq;
        }
        const int nsteps = a.H / 32;
        s0 = wave * nsteps / 4;
        s1 = (wave + 1) * nsteps / 4;
    } else {
        const int h0 = (sub / a.ks) * 64;
        kc = sub % a.ks;
        row0 = h0;
        const uint16_t* w = reinterpret_cast<const uint16_t*>(g.w2);
#pragma unroll
        for (int m = 0; m < MT; ++m) wp[m] = w + (size_t)(h0 + 16 * m + r) * g.Fg + kq;
        const int nsteps = g.Fg / 32;
        const int c0 = kc * nsteps / a.ks, c1 = (kc + 1) * nsteps / a.ks;
        s0 = c0 + wave * (c1 - c0) / 4;
        s1 = c0 + (wave + 1) * (c1 - c0) / 4;
    }

    // token operand rows (N side)
    const int ntile = min(NT, (g.count + 15) / 16);
    const uint16_t* bp[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        bp[j] = nullptr;
        const int n = 16 * j + r;
        if (!kDown) {
            const int t = group_token(a, g, n);
            if (t >= 0) bp[j] = static_cast<const uint16_t*>(a.x) + (size_t)t * a.H + kq;
        } else if (n < g.count) {
            bp[j] = static_cast<const uint16_t*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + kq;
        }
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    int s = s0;
    for (; s + U <= s1; s += U) {
        bf16x8 A[U][MT], B[U][NT];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int m = 0; m < MT; ++m) A[u][m] = load_bf16x8_stream(wp[m] + (s + u) * 32);
#pragma unroll
            for (int j = 0; j < NT; ++j) B[u][j] = (j < ntile && bp[j]) ? load_bf16x8(bp[j] + (s + u) * 32) : zero_bf16x8();
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < NT; ++j)
                if (j < ntile)
#pragma unroll
                    for (int m = 0; m < MT; ++m) acc[m][j] = mfma16x16x32(A[u][m], B[u][j], acc[m][j]);
    }
    for (; s < s1; ++s) {
        bf16x8 A[MT], B[NT];
#pragma unroll
        for (int m = 0; m < MT; ++m) A[m] = load_bf16x8_stream(wp[m] + s * 32);
#pragma unroll
        for (int j = 0; j < NT; ++j) B[j] = (j < ntile && bp[j]) ? load_bf16x8(bp[j] + s * 32) : zero_bf16x8();
#pragma unroll
        for (int j = 0; j < NT; ++j)
            if (j < ntile)
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[m][j] = mfma16x16x32(A[m], B[j], acc[m][j]);
    }

#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) s_red[wave][m][j][lane] = acc[m][j];
    __syncthreads();

    if (!kDown) {
        // pair gate tile m with up tile m + 2; lane l holds features 4*(l/16)..+3 of token l%16
        for (int task = threadIdx.x; task < 2 * NT * kWave; task += 256) {
            const int m = task / (NT * kWave);
            const int j = (task / kWave) % NT;
            const int l = task % kWave;
            const int n = 16 * j + (l & 15);
            if (j >= ntile || n >= g.count) continue;
            f32x4 gv = s_red[0][m][j][l], uv = s_red[0][m + 2][j][l];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                gv += s_red[w][m][j][l];
                uv += s_red[w][m + 2][j][l];
            }
            const int f = row0 + 16 * m + 4 * (l >> 4);
            u32x2 packed;
            packed.x = pack_bf16x2(silu(gv.x) * uv.x, silu(gv.y) * uv.y);
            packed.y = pack_bf16x2(silu(gv.z) * uv.z, silu(gv.w) * uv.w);
            uint16_t* dst = static_cast<uint16_t*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + f;
            *reinterpret_cast<u32x2*>(dst) = packed;
        }
    } else {
        for (int task = threadIdx.x; task < MT * NT * kWave; task += 256) {
            const int m = task / (NT * kWave);
            const int j = (task / kWave) % NT;
            const int l = task % kWave;
            const int n = 16 * j + (l & 15);
            if (j >= ntile || n >= g.count) continue;
            f32x4 v = s_red[0][m][j][l];
#pragma unroll
            for (int w = 1; w < 4; ++w) v += s_red[w][m][j][l];
            const int h = row0 + 16 * m + 4 * (l >> 4);
            float* dst = a.y + (long long)kc * a.y_ks_stride + (size_t)(g.rowbase + n) * a.H + h;
            *reinterpret_cast<f32x4*>(dst) = v;
        }
    }
}

// ---------------------------------------------------------------------------
// tiled kernel (prefill)
// ---------------------------------------------------------------------------

constexpr int kTm = 64;      // weight rows per tile
constexpr int kTn = 64;      // tokens per tile
constexpr int kTk = 64;      // K slab
constexpr int kPitch = kTk + 8;  // LDS row pitch (bf16 elements)

// Active routed experts and the prefix of their 64-token tile counts.
__device__ int list_tiles(const Args& a, int* s_list, int* s_wsum, int* s_tpre, int nact) {
    // s_tpre[g] = sum_{g' < g} ceil(count(g') / 64); s_tpre[nact] = total
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int v[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int gi = 4 * lane + i;
            v[i] = 0;
            if (gi < nact) {
                const int e = s_list[gi];
                int c = a.counts[e];
                c = c < 0 ? 0 : c;
                v[i] = (c + kTn - 1) / kTn;
            }
            sum += v[i];
        }
        int inc = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(inc, off, 64);
            if (lane >= off) inc += o;
        }
        int run = inc - sum;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int gi = 4 * lane + i;
            if (gi <= nact) s_tpre[gi] = run;
            run += v[i];
        }
        if (lane == 63) s_wsum[0] = inc;
    }
    __syncthreads();
    return s_wsum[0];
}

template <bool kDown>
__global__ void __launch_bounds__(256) k_ffn_tiled(Args a, int max_rtiles, int ntn_r, int ntn_s) {
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    __shared__ int s_tpre[260];
    __shared__ __attribute__((aligned(16))) uint16_t sW[2][kTm][kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t sX[2][kTn][kPitch];

    const int nact = list_active(a, s_list, s_wsum);
    const int total_rt = list_tiles(a, s_list, s_wsum, s_tpre, nact);
    const int item = blockIdx.x;
    Group g;
    int mt_local, wn;
    if (item < max_rtiles * ntn_r) {
        const int mt = item / ntn_r;
        wn = item % ntn_r;
        if (mt >= total_rt) return;
        int lo = 0, hi = nact - 1;  // last gi with s_tpre[gi] <= mt
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_tpre[mid] <= mt) lo = mid;
            else hi = mid - 1;
        }
        g = routed_group(a, s_list[lo], 2);
        mt_local = mt - s_tpre[lo];
    } else {
        const int i2 = item - max_rtiles * ntn_r;
        const int tps = (a.T + kTn - 1) / kTn;
        const int mt = i2 / ntn_s;
        wn = i2 % ntn_s;
        const int s = mt / tps;
        if (s >= a.S) return;
        g = shared_group(a, s, 2);
        mt_local = mt % tps;
    }
    const int n0 = mt_local * kTn;
    if (n0 >= g.count) return;

    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int K = kDown ? g.Fg : a.H;
    const uint16_t* wbase = reinterpret_cast<const uint16_t*>(kDown ? g.w2 : g.w13);
    const int ldw = kDown ? g.Fg : a.H;
    const int wrow0 = wn * (kDown ? 64 : 32);  // first output feature (phase 1) or output row (phase 2)

    // global -> LDS copy assignment: 512 chunks of 16 B per tile, 2 per thread
    const uint16_t* gW[2];
    const uint16_t* gX[2];
    int cr[2], cc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int c = tid + 256 * i;
        cr[i] = c >> 3;
        cc[i] = (c & 7) * 8;
        int row;
        if (!kDown) {
            const int half = cr[i] >> 5, sub = cr[i] & 31;
            const int feat = wrow0 + 16 * half + (sub & 15);
            row = (sub < 16) ? feat : g.Fg + feat;
        } else {
            row = wrow0 + cr[i];
        }
        gW[i] = wbase + (size_t)row * ldw + cc[i];
        const int n = n0 + cr[i];
        gX[i] = nullptr;
        if (!kDown) {
            const int t = group_token(a, g, n);
            if (t >= 0) gX[i] = static_cast<const uint16_t*>(a.x) + (size_t)t * a.H + cc[i];
        } else if (n < g.count) {
            gX[i] = static_cast<const uint16_t*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + cc[i];
        }
    }

    const int wr = wave >> 1, wc = wave & 1;
    const int r = lane & 15, kq = (lane >> 4) * 8;
    f32x4 acc[2][2];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = K / kTk;
    u32x4 rw[2], rx[2];
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            rw[i] = *reinterpret_cast<const u32x4*>(gW[i] + kt * kTk);
            rx[i] = gX[i] ? *reinterpret_cast<const u32x4*>(gX[i] + kt * kTk) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *reinterpret_cast<u32x4*>(&sW[buf][cr[i]][cc[i]]) = rw[i];
            *reinterpret_cast<u32x4*>(&sX[buf][cr[i]][cc[i]]) = rx[i];
        }
    };

    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < kTk / 32; ++ks) {
            bf16x8 A[2], B[2];
#pragma unroll
            for (int m = 0; m < 2; ++m)
                A[m] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&sW[buf][32 * wr + 16 * m + r][ks * 32 + kq]));
#pragma unroll
            for (int j = 0; j < 2; ++j)
                B[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&sX[buf][32 * wc + 16 * j + r][ks * 32 + kq]));
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[m][j] = mfma16x16x32(A[m], B[j], acc[m][j]);
        }
        if (kt + 1 < nk) lstore(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int n = n0 + 32 * wc + 16 * j + r;
        if (n >= g.count) continue;
        if (!kDown) {
            // acc[0] = gate, acc[1] = up for features wrow0 + 16*wr + 4*(lane/16) + i
            const f32x4 gv = acc[0][j], uv = acc[1][j];
            const int f = wrow0 + 16 * wr + 4 * (lane >> 4);
            u32x2 packed;
            packed.x = pack_bf16x2(silu(gv.x) * uv.x, silu(gv.y) * uv.y);
            packed.y = pack_bf16x2(silu(gv.z) * uv.z, silu(gv.w) * uv.w);
            *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + f) = packed;
        } else {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int h = wrow0 + 32 * wr + 16 * m + 4 * (lane >> 4);
                *reinterpret_cast<f32x4*>(a.y + (size_t)(g.rowbase + n) * a.H + h) = acc[m][j];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 kernels
// ---------------------------------------------------------------------------

__device__ bool resolve_group_f32(const Args& a, int gidx, int* s_list, int* s_wsum, Group* g) {
    const int nact = list_active(a, s_list, s_wsum);
    if (gidx < a.max_routed) {
        if (gidx >= nact) return false;
        *g = routed_group(a, s_list[gidx], 4);
    } else {
        const int s = gidx - a.max_routed;
        if (s >= a.S) return false;
        *g = shared_group(a, s, 4);
    }
    return g->count > 0;
}

__global__ void __launch_bounds__(256) k_ffn1_f32(Args a) {
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    Group g;
    if (!resolve_group_f32(a, blockIdx.x, s_list, s_wsum, &g)) return;
    const int f = blockIdx.y * 64 + (threadIdx.x & 63);
    if (f >= g.Fg) return;
    const float* x = static_cast<const float*>(a.x);
    const float* wg = reinterpret_cast<const float*>(g.w13) + (size_t)f * a.H;
    const float* wu = reinterpret_cast<const float*>(g.w13) + (size_t)(g.Fg + f) * a.H;
    float* act = static_cast<float*>(a.act);
    for (int n = threadIdx.x >> 6; n < g.count; n += 4) {
        const int t = group_token(a, g, n);
        if (t < 0) continue;
        const float* xr = x + (size_t)t * a.H;
        float gs = 0.f, us = 0.f;
        for (int h = 0; h < a.H; ++h) {
            gs = fmaf(xr[h], wg[h], gs);
            us = fmaf(xr[h], wu[h], us);
        }
        act[(size_t)(g.rowbase + n) * a.Fa + f] = silu(gs) * us;
    }
}

__global__ void __launch_bounds__(256) k_ffn2_f32(Args a) {
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    Group g;
    if (!resolve_group_f32(a, blockIdx.x, s_list, s_wsum, &g)) return;
    const int h = blockIdx.y * 64 + (threadIdx.x & 63);
    if (h >= a.H) return;
    const float* w = reinterpret_cast<const float*>(g.w2) + (size_t)h * g.Fg;
    const float* act = static_cast<const float*>(a.act);
    for (int n = threadIdx.x >> 6; n < g.count; n += 4) {
        const float* ar = act + (size_t)(g.rowbase + n) * a.Fa;
        float s = 0.f;
        for (int f = 0; f < g.Fg; ++f) s = fmaf(ar[f], w[f], s);
        a.y[(size_t)(g.rowbase + n) * a.H + h] = s;
    }
}

// y_out[p] = sum_c y[c][p] for resident packed rows p < n_res and all shared rows.
__global__ void __launch_bounds__(256) k_reduce_splits(int T, int H, int E, int k, int S, int slots,
                                                       const int32_t* __restrict__ counts,
                                                       const int32_t* __restrict__ expert_slot,
                                                       const float* __restrict__ y, int ks, long long stride,
                                                       float* __restrict__ y_out) {
    __shared__ int s_nres;
    if (threadIdx.x == 0) {
        int n = 0;
        for (int e = 0; e < E; ++e)
            if (is_resident(expert_slot[e], slots)) n += counts[e] > 0 ? counts[e] : 0;
        s_nres = n;
    }
    __syncthreads();
    const int P = T * k, rows = P + S * T;
    const int row = blockIdx.x;
    if (row >= rows || (row < P && row >= s_nres)) return;
    for (int h = threadIdx.x * 4; h < H; h += 1024) {
        f32x4 v = *reinterpret_cast<const f32x4*>(y + (size_t)row * H + h);
        for (int c = 1; c < ks; ++c) v += *reinterpret_cast<const f32x4*>(y + c * stride + (size_t)row * H + h);
        *reinterpret_cast<f32x4*>(y_out + (size_t)row * H + h) = v;
    }
}

int max_routed_groups(const Shape& s) {
    int m = s.E < s.slots ? s.E : s.slots;
    const int pairs = s.T * s.k;
    return m < pairs ? m : pairs;
}

bool use_stream(const Shape& s) { return s.bf16 && s.T <= 64; }

}  // namespace

int ffn_down_splits(const Shape& s) {
    if (!use_stream(s)) return 1;
    // phase-2 work items: (groups) x (H / 64 row tiles) x ks; aim for >= ~2048
    // workgroups while every wave keeps >= 2 K steps of 32.
    const int groups = max_routed_groups(s) + s.S;
    if (groups == 0) return 1;
    int steps = s.F / 32;
    if (s.S > 0 && s.Fs / 32 < steps) steps = s.Fs / 32;
    int ks = 1;
    while (ks < 16 && (long long)groups * (s.H / 64) * ks < 2048 && steps / (ks * 2) >= 8) ks *= 2;
    return ks;
}

hipError_t launch_grouped_ffn(const Shape& s, const FfnArgs& fa, hipStream_t st) {
    if (s.T == 0) return hipSuccess;
    Args a;
    a.T = s.T; a.H = s.H; a.E = s.E; a.F = s.F; a.k = s.k; a.S = s.S; a.Fs = s.Fs; a.slots = s.slots;
    a.x = fa.x; a.perm = fa.perm; a.counts = fa.counts; a.seg_start = fa.seg_start; a.expert_slot = fa.expert_slot;
    a.w13 = fa.w13; a.w2 = fa.w2; a.ws13 = fa.ws13; a.ws2 = fa.ws2;
    a.act = fa.act; a.Fa = fa.Fa; a.y = fa.y; a.ks = fa.ks; a.y_ks_stride = fa.y_ks_stride;
    a.max_routed = max_routed_groups(s);
    if (!s.bf16) {
        a.ipg_r = a.ipg_s = 1;
        const int groups = a.max_routed + s.S;
        if (groups == 0) return hipSuccess;
        const int fmax = s.S > 0 && s.Fs > s.F ? s.Fs : s.F;
        hipLaunchKernelGGL(k_ffn1_f32, dim3(groups, fmax / 64), dim3(256), 0, st, a);
        hipLaunchKernelGGL(k_ffn2_f32, dim3(groups, s.H / 64), dim3(256), 0, st, a);
        return hipGetLastError();
    }
    if (use_stream(s)) {
        const int nt = (s.T + 15) / 16;
        // phase 1: 32 features per workgroup
        a.ipg_r = s.F / 32;
        a.ipg_s = s.S > 0 ? s.Fs / 32 : 1;
        int grid = a.max_routed * a.ipg_r + s.S * a.ipg_s;
        if (grid > 0) {
            switch (nt) {
                case 1: hipLaunchKernelGGL((k_ffn_stream<1, false>), dim3(grid), dim3(256), 0, st, a); break;
                case 2: hipLaunchKernelGGL((k_ffn_stream<2, false>), dim3(grid), dim3(256), 0, st, a); break;
                case 3: hipLaunchKernelGGL((k_ffn_stream<3, false>), dim3(grid), dim3(256), 0, st, a); break;
                default: hipLaunchKernelGGL((k_ffn_stream<4, false>), dim3(grid), dim3(256), 0, st, a); break;
            }
        }
        // phase 2: 64 output rows x one K chunk per workgroup
        a.ipg_r = (s.H / 64) * a.ks;
        a.ipg_s = (s.H / 64) * a.ks;
        grid = a.max_routed * a.ipg_r + s.S * a.ipg_s;
        if (grid > 0) {
            switch (nt) {
                case 1: hipLaunchKernelGGL((k_ffn_stream<1, true>), dim3(grid), dim3(256), 0, st, a); break;
                case 2: hipLaunchKernelGGL((k_ffn_stream<2, true>), dim3(grid), dim3(256), 0, st, a); break;
                case 3: hipLaunchKernelGGL((k_ffn_stream<3, true>), dim3(grid), dim3(256), 0, st, a); break;
                default: hipLaunchKernelGGL((k_ffn_stream<4, true>), dim3(grid), dim3(256), 0, st, a); break;
            }
        }
        return hipGetLastError();
    }
    // tiled: worst-case number of 64-token tiles over the routed groups
    const int P = s.T * s.k;
    const int max_rtiles = (a.max_routed == 0) ? 0 : (P + kTn - 1) / kTn + a.max_routed;
    const int tps = (s.T + kTn - 1) / kTn;
    a.ipg_r = a.ipg_s = 0;
    {
        const int ntn_r = s.F / 32, ntn_s = s.S > 0 ? s.Fs / 32 : 0;
        const long long grid = (long long)max_rtiles * ntn_r + (long long)s.S * tps * ntn_s;
        if (grid > 0) hipLaunchKernelGGL((k_ffn_tiled<false>), dim3((unsigned)grid), dim3(256), 0, st, a, max_rtiles, ntn_r, ntn_s > 0 ? ntn_s : 1);
    }
    {
        const int ntn = s.H / 64;
        const long long grid = (long long)max_rtiles * ntn + (long long)s.S * tps * ntn;
        if (grid > 0) hipLaunchKernelGGL((k_ffn_tiled<true>), dim3((unsigned)grid), dim3(256), 0, st, a, max_rtiles, ntn, ntn);
    }
    return hipGetLastError();
}

hipError_t launch_reduce_splits(const Shape& s, const int32_t* counts, const int32_t* expert_slot, const float* y,
                                int ks, long long y_ks_stride, float* y_out, hipStream_t st) {
    const int rows = s.T * s.k + s.S * s.T;
    if (rows == 0) return hipSuccess;
    hipLaunchKernelGGL(k_reduce_splits, dim3(rows), dim3(256), 0, st, s.T, s.H, s.E, s.k, s.S, s.slots, counts,
                       expert_slot, y, ks, y_ks_stride, y_out);
    return hipGetLastError();
}

}  // namespace saem
