// ffn.hip -- grouped SwiGLU expert FFN over the resident and shared experts
// (SAEM Section IV-D.2: resident experts on the matrix cores; Section IV-E.1:
// one batched execution per expert over its contiguous, repacked rows).
//
// Row space: packed rows [0, T*k) (resident experts first, see repack.hip),
// then the rows of shared expert s at T*k + s*T + t.
//   phase 1: act[p, f] = silu(x[tok(p)] . W1[:,f]) * (x[tok(p)] . W3[:,f])
//   phase 2: y[c][p, h] = sum over K chunk c of act[p, :] . W2[:,h]
//
// Expert weights are in the MFMA tile layout (pack.hip): a 16-row x 32-column
// block is 1 KB of contiguous memory whose 64 16-byte pieces are the 64 lanes'
// MFMA A operands.
//
// Three kernel families:
//  * stream  (T <= 64, decode; bf16 MFMA 16x16x32, fp32 MFMA 16x16x4): the
//    weights are streamed from HBM exactly once.  A workgroup owns 32 features (phase 1: 32 gate + 32 up weight
//    rows) or 64 outputs (phase 2: 64 rows of W2) of one expert; the weights are
//    the MFMA M side and the expert's tokens the N side, in tiles of 16.  Its
//    four waves split K interleaved -- wave w takes the 32-wide K steps w, w+4,
//    w+8, ... -- so at any moment the workgroup reads 4 KB of contiguous memory
//    per weight tile; each wave double-buffers its loads in registers (the next
//    two K steps are in flight while the MFMAs of the current two run).  The
//    waves' partial tiles are summed through LDS in wave order.  Phase 2 also
//    splits K across workgroups into `ks` chunks whose partial sums the combine
//    adds in fixed order.  SwiGLU is applied in the phase-1 epilogue, so the gate
//    and up projections are never stored.
//  * tiled   (bf16, T > 64, prefill): workgroup tiles of 128 weight rows x 128
//    tokens (64 x 64 per wave); K runs in 64-wide slabs through one LDS buffer
//    while the next slab is loaded into registers, so three workgroups fit on a
//    CU; each phase-1 wave holds the gate and up rows of the same features so
//    SwiGLU runs in registers.
//  * f32     (fp32, T > 64): plain fp32 FMA, one output per thread.
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
    // offloaded-row pack done by the workgroups past the FFN items (phase 1 only)
    const float* topk_w;
    const int32_t* n_res;
    void* off_rows;
    float* off_w;
};

// off_rows[p - n_res] = x[perm[p] / k] and off_w[p - n_res] = topk_w[perm[p]] for the
// offloaded rows p = n_res + wg, n_res + wg + nwg, ...
__device__ void pack_offloaded(const Args& a, int wg, int nwg, int elt) {
    const int P = a.T * a.k;
    const int nres = *a.n_res;
    const int chunks = a.H * elt / 16;  // 16-byte chunks of a row
    for (int p = nres + wg; p < P; p += nwg) {
        const int q = a.perm[p];
        if (q < 0 || q >= P) continue;
        const int t = q / a.k;
        if (a.off_rows) {
            const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(a.x) + (size_t)t * a.H * elt);
            u32x4* dst = reinterpret_cast<u32x4*>(static_cast<uint8_t*>(a.off_rows) + (size_t)(p - nres) * a.H * elt);
            for (int c = threadIdx.x; c < chunks; c += blockDim.x) dst[c] = src[c];
        }
        if (a.off_w && threadIdx.x == 0) a.off_w[p - nres] = a.topk_w[q];
    }
}

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
// With s_info, entry i also gets expert s_list[i]'s (segment start, count, slot),
// read in the same round trip as the counts.
// Must be called by all threads of a 256-thread workgroup.
__device__ int list_active(const Args& a, int* s_list, int* s_wsum, int4* s_info = nullptr) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int e = tid;
    bool act = false;
    int sl = -1, cnt = 0, seg = 0;
    if (e < a.E) {
        sl = a.expert_slot[e];
        cnt = a.counts[e];
        if (s_info) seg = a.seg_start[e];
        act = is_resident(sl, a.slots) && cnt > 0;
    }
    const unsigned long long b = __ballot(act);
    if (lane == 0) s_wsum[wave] = __popcll(b);
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += s_wsum[w];
    if (act) {
        const int pos = base + __popcll(b & ((1ull << lane) - 1ull));
        s_list[pos] = e;
        if (s_info) s_info[pos] = make_int4(seg, cnt, sl, 0);
    }
    const int n = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
    return n;
}

// Routed group from its expert's segment start, count and slot.
__device__ Group routed_group_of(const Args& a, int rb, int c, int slot_, size_t elt) {
    Group g;
    const int P = a.T * a.k;
    rb = rb < 0 ? 0 : (rb > P ? P : rb);
    c = c < 0 ? 0 : (c > P - rb ? P - rb : c);
    g.rowbase = rb;
    g.count = c;
    g.routed = 1;
    g.Fg = a.F;
    const size_t slot = (size_t)slot_;
    g.w13 = static_cast<const uint8_t*>(a.w13) + slot * 2 * a.F * a.H * elt;
    g.w2 = static_cast<const uint8_t*>(a.w2) + slot * a.H * a.F * elt;
    return g;
}

__device__ Group routed_group(const Args& a, int e, size_t elt) {
    return routed_group_of(a, a.seg_start[e], a.counts[e], a.expert_slot[e], elt);
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

// 16-row weight tiles per stream workgroup: two with a single token tile (twice
// the workgroups, for the small grids of the smallest batches), else four.
constexpr int stream_mt(int nt) { return nt == 1 ? 2 : 4; }

// kStreamW: the weights are loaded non-temporally (they do not stay in the
// caches for a later use), which raises the streaming rate when the call's
// weights are far larger than the caches; small weight sets that stay in the
// MALL between calls are read with plain loads.
template <typename Elt, int NT, bool kDown, bool kStreamW>
__global__ void __launch_bounds__(256) k_ffn_stream(Args a) {
    using F8 = Frag8<Elt>;
    constexpr int MT = stream_mt(NT);              // 16-row weight tiles per workgroup
    constexpr int MH = MT / 2;                     // phase 1: gate tiles (then as many up tiles)
    constexpr int U = sizeof(Elt) == 2 ? 2 : 1;    // K steps per load batch (two batches in flight)
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    __shared__ int4 s_info[256];
    __shared__ f32x4 s_red[4][MT][NT][kWave];

    const int item = blockIdx.x;
    const int n_items = a.max_routed * a.ipg_r + a.S * a.ipg_s;
    if (!kDown && item >= n_items) {  // trailing workgroups pack the offloaded rows
        pack_offloaded(a, item - n_items, gridDim.x - n_items, sizeof(Elt));
        return;
    }
    const int nact = list_active(a, s_list, s_wsum, s_info);
    // shared groups first: their items can be longer (Fs > F in phase 2), so they
    // start in the first wave of workgroups instead of forming a tail
    Group g;
    int sub;
    if (item < a.S * a.ipg_s) {
        g = shared_group(a, item / a.ipg_s, sizeof(Elt));
        sub = item % a.ipg_s;
    } else {
        const int i2 = item - a.S * a.ipg_s;
        const int gi = i2 / a.ipg_r;
        if (gi >= nact) return;
        const int4 info = s_info[gi];
        g = routed_group_of(a, info.x, info.y, info.z, sizeof(Elt));
        sub = i2 % a.ipg_r;
    }
    if (g.count == 0) return;

    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;

    // weight tiles of this workgroup (16-row tiles in the tile layout) and the K chunk
    const Elt* wp[MT];
    int row0, kc = 0, c0, c1;
    if (!kDown) {
        const int f0 = sub * 16 * MH;
        row0 = f0;
        const int nst = a.H / 32;
        const Elt* w = reinterpret_cast<const Elt*>(g.w13);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const int rt = (m < MH ? 0 : g.Fg / 16) + f0 / 16 + m % MH;  // gate tiles, then up tiles
            wp[m] = w + (size_t)rt * nst * 512 + lane * 8;
        }
        c0 = 0;
        c1 = nst;
    } else {
        const int h0 = (sub / a.ks) * 16 * MT;
        kc = sub % a.ks;
        row0 = h0;
        const int nst = g.Fg / 32;
        const Elt* w = reinterpret_cast<const Elt*>(g.w2);
#pragma unroll
        for (int m = 0; m < MT; ++m) wp[m] = w + (size_t)(h0 / 16 + m) * nst * 512 + lane * 8;
        c0 = kc * nst / a.ks;
        c1 = (kc + 1) * nst / a.ks;
    }
    // this wave's K steps: c0 + wave + 4 i
    const int n_my = (c1 - c0 > wave) ? (c1 - c0 - wave + 3) / 4 : 0;
    const int sbase = c0 + wave;

    const int nb = n_my / U;
    // batch b holds this wave's steps i = U*b .. U*b+U-1
    auto load_w = [&](F8 (&A)[U][MT], int b) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = sbase + 4 * (U * b + u);
#pragma unroll
            for (int m = 0; m < MT; ++m)
                A[u][m] = kStreamW ? load_frag_stream(wp[m] + (size_t)s * 512) : load_frag(wp[m] + (size_t)s * 512);
        }
    };
    // the first batch's weights go out before the token rows are looked up
    F8 A0[U][MT], B0[U][NT], A1[U][MT], B1[U][NT];
    if (nb > 0) load_w(A0, 0);

    // token operand rows (N side)
    const int ntile = min(NT, (g.count + 15) / 16);
    const Elt* bp[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        bp[j] = nullptr;
        const int n = 16 * j + r;
        if (!kDown) {
            const int t = group_token(a, g, n);
            if (t >= 0) bp[j] = static_cast<const Elt*>(a.x) + (size_t)t * a.H + kq;
        } else if (n < g.count) {
            bp[j] = static_cast<const Elt*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + kq;
        }
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto load_x = [&](F8 (&B)[U][NT], int b) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = sbase + 4 * (U * b + u);
#pragma unroll
            for (int j = 0; j < NT; ++j) B[u][j] = (j < ntile && bp[j]) ? load_frag(bp[j] + s * 32) : zero_frag<Elt>();
        }
    };
    auto load = [&](F8 (&A)[U][MT], F8 (&B)[U][NT], int b) {
        load_w(A, b);
        load_x(B, b);
    };
    auto mma = [&](const F8 (&A)[U][MT], const F8 (&B)[U][NT]) {
        // tiles past the group's last token see zero operands: no branch, fewer live registers
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[m][j] = mma_frag(A[u][m], B[u][j], acc[m][j]);
    };
    {
        if (nb > 0) load_x(B0, 0);
        for (int b = 0; b < nb; b += 2) {
            if (b + 1 < nb) load(A1, B1, b + 1);
            mma(A0, B0);
            if (b + 2 < nb) load(A0, B0, b + 2);
            if (b + 1 < nb) mma(A1, B1);
        }
    }
    for (int i = nb * U; i < n_my; ++i) {
        const int s = sbase + 4 * i;
        F8 A[MT], B[NT];
#pragma unroll
        for (int m = 0; m < MT; ++m)
            A[m] = kStreamW ? load_frag_stream(wp[m] + (size_t)s * 512) : load_frag(wp[m] + (size_t)s * 512);
#pragma unroll
        for (int j = 0; j < NT; ++j) B[j] = (j < ntile && bp[j]) ? load_frag(bp[j] + s * 32) : zero_frag<Elt>();
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m][j] = mma_frag(A[m], B[j], acc[m][j]);
    }

#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) s_red[wave][m][j][lane] = acc[m][j];
    __syncthreads();

    if (!kDown) {
        // pair gate tile m with up tile m + MH; lane l holds features 4*(l/16)..+3 of token l%16
        for (int task = threadIdx.x; task < MH * NT * kWave; task += 256) {
            const int m = task / (NT * kWave);
            const int j = (task / kWave) % NT;
            const int l = task % kWave;
            const int n = 16 * j + (l & 15);
            if (j >= ntile || n >= g.count) continue;
            f32x4 gv = s_red[0][m][j][l], uv = s_red[0][m + MH][j][l];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                gv += s_red[w][m][j][l];
                uv += s_red[w][m + MH][j][l];
            }
            const int f = row0 + 16 * m + 4 * (l >> 4);
            const f32x4 av = {silu(gv.x) * uv.x, silu(gv.y) * uv.y, silu(gv.z) * uv.z, silu(gv.w) * uv.w};
            Elt* dst = static_cast<Elt*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + f;
            if constexpr (sizeof(Elt) == 2) {
                u32x2 packed;
                packed.x = pack_bf16x2(av.x, av.y);
                packed.y = pack_bf16x2(av.z, av.w);
                *reinterpret_cast<u32x2*>(dst) = packed;
            } else {
                *reinterpret_cast<f32x4*>(dst) = av;
            }
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

constexpr int kTn = 128;         // tokens per tile
constexpr int kTk = 64;          // K slab
constexpr int kXPitch = kTk + 8;  // LDS row pitch of the token tile (bf16 elements)

// Active routed experts and the prefix of their kTn-token tile counts.
__device__ int list_tiles(const Args& a, int* s_list, int* s_wsum, int* s_tpre, int nact) {
    // s_tpre[g] = sum_{g' < g} ceil(count(g') / kTn); s_tpre[nact] = total
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
        // the end entry: written above for nact < 256 (its run is then the total); with all
        // 256 experts active it lies past the lanes' entries, so lane 63 writes it
        if (lane == 63) {
            s_wsum[0] = inc;
            s_tpre[nact] = inc;
        }
    }
    __syncthreads();
    return s_wsum[0];
}

// Workgroup tile: 128 weight rows x 128 tokens; phase 1 takes 64 features (their
// 64 gate rows and 64 up rows), phase 2 128 rows of W2.  Four waves in 2 x 2,
// each 64 rows x 64 tokens (16 MFMA 16x16x32 tiles, 64 fp32 accumulators per
// lane); phase-1 waves hold the gate and up rows of the same 32 features so
// SwiGLU runs in registers.  K runs in 64-wide slabs through one LDS buffer:
// the weight slab is 16 blocks of 1 KB copied as they sit in the tile layout,
// the token slab 128 gathered rows.  Consecutive tiles (same weight tile, next
// token tile of the group) are placed on the same XCD so they share its L2.
template <bool kDown>
__global__ void __launch_bounds__(256, 3) k_ffn_tiled(Args a, int max_rtiles, int ntn_r, int ntn_s, int grid8) {
    __shared__ int s_list[256];
    __shared__ int s_wsum[4];
    __shared__ int s_tpre[260];
    __shared__ __attribute__((aligned(16))) uint16_t sW[16][512];
    __shared__ __attribute__((aligned(16))) uint16_t sX[kTn][kXPitch];

    const int pid = blockIdx.x;
    if (!kDown && pid >= grid8) {  // workgroups past the items pack the offloaded rows (phase 1 only)
        pack_offloaded(a, pid - grid8, gridDim.x - grid8, 2);
        return;
    }
    const int nact = list_active(a, s_list, s_wsum);
    const int total_rt = list_tiles(a, s_list, s_wsum, s_tpre, nact);
    // XCD-aware order: workgroups are dealt to the 8 XCDs round-robin, so logical
    // items pid/8, pid/8 + 1, ... of one XCD are consecutive in this numbering.
    const int item = (pid % 8) * (grid8 / 8) + pid / 8;
    Group g;
    int mt_local, wn;
    // inside a group, items run weight tile by weight tile and, for each, over
    // all of the group's token tiles: the token tiles of one weight panel are
    // consecutive on one XCD, so the panel is read from HBM about once
    if (item < max_rtiles * ntn_r) {
        const int gt = item / ntn_r;  // group gi owns items [ntn_r s_tpre[gi], ntn_r s_tpre[gi + 1])
        if (gt >= total_rt) return;
        int lo = 0, hi = nact - 1;  // last gi with s_tpre[gi] <= gt
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_tpre[mid] <= gt) lo = mid;
            else hi = mid - 1;
        }
        g = routed_group(a, s_list[lo], 2);
        const int tg = s_tpre[lo + 1] - s_tpre[lo];
        const int local = item - ntn_r * s_tpre[lo];
        wn = local / tg;
        mt_local = local % tg;
    } else {
        const int i2 = item - max_rtiles * ntn_r;
        const int tps = (a.T + kTn - 1) / kTn;
        const int s = i2 / (tps * ntn_s);
        if (s >= a.S) return;
        g = shared_group(a, s, 2);
        const int local = i2 % (tps * ntn_s);
        wn = local / tps;
        mt_local = local % tps;
    }
    const int n0 = mt_local * kTn;
    if (n0 >= g.count) return;

    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int K = kDown ? g.Fg : a.H;
    const int nst = K / 32;
    const uint16_t* wbase = reinterpret_cast<const uint16_t*>(kDown ? g.w2 : g.w13);
    const int wrow0 = wn * (kDown ? 128 : 64);  // first output row (phase 2) or feature (phase 1)
    const int rows_total = kDown ? a.H : 2 * g.Fg;

    // the 8 row tiles of the weight slab: phase 1 gate f0/16 + 0..3, then up; phase 2 h0/16 + 0..7
    int rt_of[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        rt_of[i] = kDown ? wrow0 / 16 + i : (i < 4 ? 0 : g.Fg / 16) + wrow0 / 16 + (i & 3);

    // global -> LDS copy assignment, 4 chunks of 16 B per thread per operand
    const uint16_t* gW[4];
    const uint16_t* gX[4];
    int wb[4], wl[4], cr[4], cc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int c = tid + 256 * i;
        wb[i] = c >> 6;
        wl[i] = c & 63;
        const int rtl = wb[i] >> 1, ks = wb[i] & 1;
        gW[i] = (16 * rt_of[rtl] < rows_total) ? wbase + ((size_t)rt_of[rtl] * nst + ks) * 512 + wl[i] * 8 : nullptr;
        cr[i] = c >> 3;
        cc[i] = (c & 7) * 8;
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
    int rtl_of[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) rtl_of[m] = kDown ? 4 * wr + m : (m < 2 ? 2 * wr + m : 4 + 2 * wr + (m - 2));
    f32x4 acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // one LDS buffer (so three workgroups fit on a CU); slab kt + 1 is loaded
    // into registers while slab kt is multiplied out of LDS
    const int nk = K / kTk;
    u32x4 rw[4], rx[4];
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            rw[i] = gW[i] ? *reinterpret_cast<const u32x4*>(gW[i] + (size_t)kt * 2 * 512) : u32x4{0u, 0u, 0u, 0u};
            rx[i] = gX[i] ? *reinterpret_cast<const u32x4*>(gX[i] + kt * kTk) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    gload(0);
    for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *reinterpret_cast<u32x4*>(&sW[wb[i]][wl[i] * 8]) = rw[i];
            *reinterpret_cast<u32x4*>(&sX[cr[i]][cc[i]]) = rx[i];
        }
        __syncthreads();
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < kTk / 32; ++ks) {
            bf16x8 A[4], B[4];
#pragma unroll
            for (int m = 0; m < 4; ++m)
                A[m] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&sW[rtl_of[m] * 2 + ks][lane * 8]));
#pragma unroll
            for (int j = 0; j < 4; ++j)
                B[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&sX[64 * wc + 16 * j + r][ks * 32 + kq]));
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[m][j] = mfma16x16x32(A[m], B[j], acc[m][j]);
        }
        __syncthreads();
    }

#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = n0 + 64 * wc + 16 * j + r;
        if (n >= g.count) continue;
        if (!kDown) {
            // acc[m] = gate, acc[m + 2] = up, features wrow0 + 16 (2 wr + m) + 4 (lane/16) + i
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const f32x4 gv = acc[m][j], uv = acc[m + 2][j];
                const int f = wrow0 + 16 * (2 * wr + m) + 4 * (lane >> 4);
                if (f >= g.Fg) continue;
                u32x2 packed;
                packed.x = pack_bf16x2(silu(gv.x) * uv.x, silu(gv.y) * uv.y);
                packed.y = pack_bf16x2(silu(gv.z) * uv.z, silu(gv.w) * uv.w);
                *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + f) = packed;
            }
        } else {
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int h = wrow0 + 16 * (4 * wr + m) + 4 * (lane >> 4);
                if (h < a.H) *reinterpret_cast<f32x4*>(a.y + (size_t)(g.rowbase + n) * a.H + h) = acc[m][j];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 kernels
// ---------------------------------------------------------------------------

// Element (row, k) of a [R, K] matrix stored in the tile layout.
__device__ __forceinline__ size_t tile_off(int row, int k, int K) {
    return ((size_t)(row >> 4) * (K >> 5) + (k >> 5)) * 512 + ((k & 31) >> 3) * 128 + (row & 15) * 8 + (k & 7);
}

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
    const float* w13 = reinterpret_cast<const float*>(g.w13);
    float* act = static_cast<float*>(a.act);
    for (int n = threadIdx.x >> 6; n < g.count; n += 4) {
        const int t = group_token(a, g, n);
        if (t < 0) continue;
        const float* xr = x + (size_t)t * a.H;
        float gs = 0.f, us = 0.f;
        for (int h = 0; h < a.H; ++h) {
            gs = fmaf(xr[h], w13[tile_off(f, h, a.H)], gs);
            us = fmaf(xr[h], w13[tile_off(g.Fg + f, h, a.H)], us);
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
    const float* w2 = reinterpret_cast<const float*>(g.w2);
    const float* act = static_cast<const float*>(a.act);
    for (int n = threadIdx.x >> 6; n < g.count; n += 4) {
        const float* ar = act + (size_t)(g.rowbase + n) * a.Fa;
        float s = 0.f;
        for (int f = 0; f < g.Fg; ++f) s = fmaf(ar[f], w2[tile_off(h, f, g.Fg)], s);
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
        constexpr int kMax = 16;  // same order as the combine: chunk 0, then 1, ...
        f32x4 p[kMax];
#pragma unroll
        for (int c = 0; c < kMax; ++c)
            if (c < ks) p[c] = *reinterpret_cast<const f32x4*>(y + c * stride + (size_t)row * H + h);
        f32x4 v = p[0];
#pragma unroll
        for (int c = 1; c < kMax; ++c)
            if (c < ks) v += p[c];
        *reinterpret_cast<f32x4*>(y_out + (size_t)row * H + h) = v;
    }
}

int max_routed_groups(const Shape& s) {
    int m = s.E < s.slots ? s.E : s.slots;
    const int pairs = s.T * s.k;
    return m < pairs ? m : pairs;
}

bool use_stream(const Shape& s) { return s.T <= 64; }

template <typename Elt, bool kDown, bool kStreamW>
void launch_stream_w(int nt, int grid, const Args& a, hipStream_t st) {
    switch (nt) {
        case 1: hipLaunchKernelGGL((k_ffn_stream<Elt, 1, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        case 2: hipLaunchKernelGGL((k_ffn_stream<Elt, 2, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        case 3: hipLaunchKernelGGL((k_ffn_stream<Elt, 3, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        default: hipLaunchKernelGGL((k_ffn_stream<Elt, 4, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
    }
}

template <typename Elt, bool kDown>
void launch_stream(int nt, bool stream_w, int grid, const Args& a, hipStream_t st) {
    if (stream_w) launch_stream_w<Elt, kDown, true>(nt, grid, a, st);
    else launch_stream_w<Elt, kDown, false>(nt, grid, a, st);
}

// Non-temporal weight loads when the weights one call can touch (every slot and
// shared expert) exceed a quarter of the 256 MB MALL: then they cannot stay in
// the caches from one call to the next anyway.
bool stream_weights(const Shape& s) {
    const long long b = s.bf16 ? 2 : 4;
    const long long bytes = 3ll * s.H * ((long long)s.slots * s.F + (long long)s.S * s.Fs) * b;
    return bytes > (64ll << 20);
}

}  // namespace

bool ffn_packs_offloaded(const Shape& s) { return use_stream(s) || s.bf16; }

int ffn_down_splits(const Shape& s) {
    if (!use_stream(s)) return 1;
    // Phase-2 work items: (groups) x (H / rows) x ks, each streaming `rows` rows
    // (16 per weight tile) of one K chunk.  Smallest ks (a power of two <= 16) such that
    //  * there are >= 512 workgroups (two per CU), and
    //  * the longest workgroup streams at most 1/400 of the phase's weights: one
    //    workgroup streams at about 1/200 of the chip's HBM rate, so with a 2x
    //    margin it then ends before the phase does, instead of forming its tail
    //    (a shared expert wider than the routed ones, or few wide experts);
    // while every wave keeps >= 8 K steps of 32.
    const long long groups_r = max_routed_groups(s);
    const long long groups = groups_r + s.S;
    if (groups == 0) return 1;
    int steps = s.F / 32;
    if (s.S > 0 && s.Fs / 32 < steps) steps = s.Fs / 32;
    const long long kmax = (s.S > 0 && s.Fs > s.F) ? s.Fs : s.F;
    const long long weights = (groups_r * s.F + (long long)s.S * s.Fs) * s.H;  // elements, worst case
    const long long rows = 16 * stream_mt((s.T + 15) / 16);
    auto balanced = [&](int ks) { return groups * (s.H / rows) * ks >= 512 && rows * kmax / ks * 400 <= weights; };
    int ks = 1;
    while (ks < 16 && !balanced(ks) && steps / (ks * 2) >= 16) ks *= 2;
    return ks;
}

hipError_t launch_grouped_ffn(const Shape& s, const FfnArgs& fa, hipStream_t st, hipEvent_t between) {
    if (s.T == 0) return hipSuccess;
    auto mark = [&]() -> hipError_t {
        hipError_t e = hipGetLastError();
        if (e == hipSuccess && between) e = hipEventRecord(between, st);
        return e;
    };
    Args a;
    a.T = s.T; a.H = s.H; a.E = s.E; a.F = s.F; a.k = s.k; a.S = s.S; a.Fs = s.Fs; a.slots = s.slots;
    a.x = fa.x; a.perm = fa.perm; a.counts = fa.counts; a.seg_start = fa.seg_start; a.expert_slot = fa.expert_slot;
    a.w13 = fa.w13; a.w2 = fa.w2; a.ws13 = fa.ws13; a.ws2 = fa.ws2;
    a.act = fa.act; a.Fa = fa.Fa; a.y = fa.y; a.ks = fa.ks; a.y_ks_stride = fa.y_ks_stride;
    a.max_routed = max_routed_groups(s);
    a.topk_w = fa.topk_w;
    a.n_res = fa.n_res;
    a.off_rows = fa.off_rows;
    a.off_w = fa.off_w;
    if (!s.bf16 && !use_stream(s)) {  // fp32 prefill: plain FMA kernels
        a.ipg_r = a.ipg_s = 1;
        const int groups = a.max_routed + s.S;
        if (groups == 0) return hipSuccess;
        const int fmax = s.S > 0 && s.Fs > s.F ? s.Fs : s.F;
        hipLaunchKernelGGL(k_ffn1_f32, dim3(groups, fmax / 64), dim3(256), 0, st, a);
        if (hipError_t e = mark(); e != hipSuccess) return e;
        hipLaunchKernelGGL(k_ffn2_f32, dim3(groups, s.H / 64), dim3(256), 0, st, a);
        return hipGetLastError();
    }
    if (use_stream(s)) {
        const int nt = (s.T + 15) / 16;
        const bool sw = stream_weights(s);
        // phase 1: 32 features per workgroup
        const int mt = stream_mt(nt);
        a.ipg_r = s.F / (8 * mt);
        a.ipg_s = s.S > 0 ? s.Fs / (8 * mt) : 1;
        int grid = a.max_routed * a.ipg_r + s.S * a.ipg_s;
        if (fa.off_rows || fa.off_w) {
            const int P = s.T * s.k;
            grid += P < 64 ? P : 64;  // pack workgroups (P >= 1 here)
        }
        if (grid > 0) {
            if (s.bf16) launch_stream<uint16_t, false>(nt, sw, grid, a, st);
            else launch_stream<float, false>(nt, sw, grid, a, st);
        }
        if (hipError_t e = mark(); e != hipSuccess) return e;
        // phase 2: 64 output rows x one K chunk per workgroup
        a.ipg_r = (s.H / (16 * mt)) * a.ks;
        a.ipg_s = (s.H / (16 * mt)) * a.ks;
        grid = a.max_routed * a.ipg_r + s.S * a.ipg_s;
        if (grid > 0) {
            if (s.bf16) launch_stream<uint16_t, true>(nt, sw, grid, a, st);
            else launch_stream<float, true>(nt, sw, grid, a, st);
        }
        return hipGetLastError();
    }
    // tiled: worst-case number of kTn-token tiles over the routed groups
    const int P = s.T * s.k;
    const int max_rtiles = (a.max_routed == 0) ? 0 : (P + kTn - 1) / kTn + a.max_routed;
    const int tps = (s.T + kTn - 1) / kTn;
    a.ipg_r = a.ipg_s = 0;
    auto round8 = [](long long n) { return (n + 7) / 8 * 8; };
    {
        const int ntn_r = s.F / 64, ntn_s = s.S > 0 ? s.Fs / 64 : 1;
        const long long grid = round8((long long)max_rtiles * ntn_r + (long long)s.S * tps * ntn_s);
        // pack workgroups after the items: dispatched last, they overlap the phase's tail
        const int n_pack = (fa.off_rows || fa.off_w) ? (P < 256 ? P : 256) : 0;
        if (grid + n_pack > 0)
            hipLaunchKernelGGL((k_ffn_tiled<false>), dim3((unsigned)(grid + n_pack)), dim3(256), 0, st, a, max_rtiles,
                               ntn_r, ntn_s, (int)grid);
    }
    if (hipError_t e = mark(); e != hipSuccess) return e;
    {
        const int ntn = (s.H + 127) / 128;
        const long long grid = round8((long long)max_rtiles * ntn + (long long)s.S * tps * ntn);
        if (grid > 0)
            hipLaunchKernelGGL((k_ffn_tiled<true>), dim3((unsigned)grid), dim3(256), 0, st, a, max_rtiles, ntn, ntn,
                               (int)grid);
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
